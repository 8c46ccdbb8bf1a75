// Support and per-HCU activation: s = b + x w over the active input HCUs, then softmax (or
// argmax) within every hidden HCU (Alg. 1 support and softmax lines; Sec. 2).
//
// Design (gfx950):
//  * The weights are stored masked, so a hidden HCU only needs the rows of its active input
//    HCUs.  Each hidden HCU keeps an ascending list of them; the contraction for one hidden
//    HCU is a dense [B x K_h] . [K_h x M_out] product with K_h = n_active * M_in.  Silent
//    blocks are never read.
//  * The products accumulate in fp64 on the matrix cores (v_mfma_f64_16x16x4f64).  x and w are
//    fp32, so every product is exact in fp64 and the sum's rounding error stays far below the
//    fp32 rounding of the stored support.  (An fp32 accumulation of a few hundred terms of
//    magnitude ~10 drifts by ~1e-5, the size of the tolerance on the activities.)
//  * One workgroup (8 waves) owns one hidden HCU and 16 batch rows, i.e. complete softmax
//    segments, so the softmax runs in the epilogue from LDS and the support never round-trips
//    through HBM.  Wave w computes the 16-column output tiles w, w + 8, ...
//  * The K dimension is staged through LDS in chunks: the workgroup's weight rows (the active
//    units' row segments, contiguous M_out floats each) and its 16 x K input panel are loaded
//    cooperatively, all loads of a chunk in flight together, the next chunk into registers
//    while the current one feeds the matrix cores.  The chunk is as large as the register and
//    LDS budget allow (the whole K of the MNIST-shaped layer fits in one).
//  * Work items (row tile, hidden HCU) are spread over the XCDs so that the row tiles of one
//    hidden HCU share one XCD's L2 (they read the same weight block).
//
// MFMA f64 16x16x4 lane layout (verified on gfx950): A[i][k] from lane i + 16 k, B[k][j] from
// lane j + 16 k, and lane l holds D[l / 16 + 4 r][l % 16] in result register r.
#include <mutex>
#include <type_traits>

#include "bcpnn_internal.h"
#include "device_common.h"

namespace bcpnn {
namespace {

typedef double d4 __attribute__((ext_vector_type(4)));

// Buffer resource over [p, p + bytes): loads past the range return zero.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t input_rsrc(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

constexpr int kRows = 16;          // batch rows per workgroup
constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kMaxTilesPerWave = 8;   // kWaves * 8 * 16 = 1024 = largest out_mcu
// Weight vectors staged per thread per chunk (each holds its own address while in flight).
constexpr int stage_slots(int tiles_per_wave, int vec) {
    // at least one widest row per thread: M_out <= 128 * tiles_per_wave, 32 lanes per row
    return vec == 4 ? (tiles_per_wave >= 4 ? 8 : 12) : (tiles_per_wave >= 8 ? 32 : 16);
}
constexpr int kXRegs = 8;             // input elements staged per thread per chunk
constexpr int kLeanSlots = 8;         // weight vectors per thread in the lean variant (see launch)
constexpr int kRowGroups = kThreads / 32;   // weight rows staged side by side (32 lanes each)
static_assert(kRowGroups == kRows, "one row group per batch row of the input panel");

struct SupportLayout {
    int n_tiles, mpad, n_row_tiles;
    int kc;                        // units per chunk (multiple of 4)
    int k_alloc;                   // LDS entries of the unit table (>= the largest K_h)
    int xstride;                   // LDS row stride of the input panel (2 mod 32, see below)
    bool fits;                     // every thread's share of a chunk fits its staging slots
};

// Writes the 16 batch entries of unit u in k-step ks (one row tile) as bf16 hi and lo parts
// (hi = bf16(v), lo = bf16(v - hi), round to nearest even): two 16-byte fragment chunks each.
__device__ __forceinline__ void write_split_column(const float (&v)[kRows], uint16_t* hi,
                                                   uint16_t* lo, int64_t u, int ks, int32_t n_ks) {
    uint32_t h[kRows / 2], l[kRows / 2];
#pragma unroll
    for (int q = 0; q < kRows / 2; ++q) {
        const __bf16 h0 = (__bf16)v[2 * q], h1 = (__bf16)v[2 * q + 1];
        const __bf16 l0 = (__bf16)(v[2 * q] - (float)h0), l1 = (__bf16)(v[2 * q + 1] - (float)h1);
        h[q] = (uint32_t)__builtin_bit_cast(uint16_t, h0) | ((uint32_t)__builtin_bit_cast(uint16_t, h1) << 16);
        l[q] = (uint32_t)__builtin_bit_cast(uint16_t, l0) | ((uint32_t)__builtin_bit_cast(uint16_t, l1) << 16);
    }
    const int64_t c0 = frag_chunk(u, ks, 0, n_ks), c1 = frag_chunk(u, ks, 1, n_ks);
    *reinterpret_cast<uint4*>(hi + c0) = make_uint4(h[0], h[1], h[2], h[3]);
    *reinterpret_cast<uint4*>(hi + c1) = make_uint4(h[4], h[5], h[6], h[7]);
    *reinterpret_cast<uint4*>(lo + c0) = make_uint4(l[0], l[1], l[2], l[3]);
    *reinterpret_cast<uint4*>(lo + c1) = make_uint4(l[4], l[5], l[6], l[7]);
}

// The same for one half (rows 8 h .. 8 h + 7) of the 16 entries: one 16-byte chunk each.
__device__ __forceinline__ void write_split_half(const float (&v)[kRows / 2], uint16_t* hi,
                                                 uint16_t* lo, int64_t u, int ks, int h,
                                                 int32_t n_ks) {
    uint32_t hh[kRows / 4], ll[kRows / 4];
#pragma unroll
    for (int q = 0; q < kRows / 4; ++q) {
        const __bf16 h0 = (__bf16)v[2 * q], h1 = (__bf16)v[2 * q + 1];
        const __bf16 l0 = (__bf16)(v[2 * q] - (float)h0), l1 = (__bf16)(v[2 * q + 1] - (float)h1);
        hh[q] = (uint32_t)__builtin_bit_cast(uint16_t, h0) | ((uint32_t)__builtin_bit_cast(uint16_t, h1) << 16);
        ll[q] = (uint32_t)__builtin_bit_cast(uint16_t, l0) | ((uint32_t)__builtin_bit_cast(uint16_t, l1) << 16);
    }
    const int64_t c = frag_chunk(u, ks, h, n_ks);
    *reinterpret_cast<uint4*>(hi + c) = make_uint4(hh[0], hh[1], hh[2], hh[3]);
    *reinterpret_cast<uint4*>(lo + c) = make_uint4(ll[0], ll[1], ll[2], ll[3]);
}

// kTilesPerWave: 16-column output tiles per wave, ceil(ceil(M_out / 16) / 8).
// kVec: 4 when weight row segments can be read as float4 (M_out and N_out multiples of 4).
// kOps: training (the contraction operands are written); the forward pass is a variant of its
// own, without that code (and, in a kernel trace, under a name of its own).  kStamp: the
// launch stamps its start and end (training launches that profiling times).
template <int kTilesPerWave, int kVec, int kLeanSlots, bool kOps, bool kStamp>
__global__ void __launch_bounds__(kThreads)
support_kernel(Geometry g, SupportLayout lay, const float* __restrict__ x, int32_t B,
               const float* __restrict__ w, const float* __restrict__ bias,
               const int32_t* __restrict__ act_list, const int32_t* __restrict__ act_count,
               float gain, int mode, float* __restrict__ y, float* __restrict__ s,
               int32_t* __restrict__ winner, const float* __restrict__ target,
               TraceOperands ops, unsigned long long* stamp) {
    constexpr bool has_ops = kOps;
    stamp_start<kStamp>(stamp);
    // Highest wave priority: on a CU shared with the silent sweep (second stream), the SIMD
    // arbiter issues this kernel's instructions first.
    __builtin_amdgcn_s_setprio(3);
    typedef float vec_t __attribute__((ext_vector_type(kVec)));
    constexpr int kSlots = kLeanSlots > 0 ? kLeanSlots : stage_slots(kTilesPerWave, kVec);
    extern __shared__ float lds[];
    const int kc = lay.kc, mpad = lay.mpad, xstride = lay.xstride;
    int32_t* units = reinterpret_cast<int32_t*>(lds);               // [k_alloc]
    float* ws = lds + ((lay.k_alloc + 3) & ~3);                      // [kc][mpad]
    float* xs = ws + (size_t)kc * mpad;                              // [kRows][xstride]
    float* stile = ws;                                               // [kRows][mpad] afterwards

    const int64_t work = xcd_linear_index(blockIdx.x, (int64_t)lay.n_row_tiles * g.out_hcu);
    const int hj = (int)(work / lay.n_row_tiles);
    const int row0 = (int)(work % lay.n_row_tiles) * kRows;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int sub = tid & 31;          // lane within a row group
    const int grp = tid >> 5;          // row group

    const int32_t k_total = act_count[hj] * g.in_mcu;
    const int32_t* alist = act_list + (int64_t)hj * g.in_hcu;
    const int64_t col_base = (int64_t)hj * g.out_mcu;
    // The table is filled up to the largest K_h of the layer, so its loads do not wait for the
    // count; entries past k_total are never used.
    for (int32_t k = tid; k < lay.k_alloc; k += kThreads)
        units[k] = (int32_t)((uint32_t)alist[k / g.in_mcu] * (uint32_t)g.in_mcu +
                             (uint32_t)(k % g.in_mcu));
    lds_barrier();

    // Weight rows: row group grp takes chunk rows grp, grp + 16, ...; its 32 lanes take the
    // vectors sub, sub + 32, ... of each row.  Input panel: row r = grp, units sub, sub + 32, ...
    const int nvec = g.out_mcu / kVec;
    vec_t wr[kSlots];
    float xr[kXRegs];
    // Each thread walks its weight slots in a fixed order: rows grp, grp + 16, ..., and within
    // a row the vectors sub, sub + 32, ... below nvec (lanes with sub >= nvec stay idle).  The
    // walk is unrolled over the slots, so every load of a chunk is issued before any is used.
    auto load_chunk = [&](int32_t k0) {
        int u = grp, v = sub;
#pragma unroll
        for (int q = 0; q < kSlots; ++q) {
            wr[q] = vec_t(0.0f);
            if (v < nvec && u < kc && k0 + u < k_total) {
                const vec_t* src =
                    reinterpret_cast<const vec_t*>(w + (int64_t)units[k0 + u] * g.n_out + col_base);
                wr[q] = src[v];
            }
            v += 32;
            if (v >= nvec) { v = sub; u += kRowGroups; }
        }
        const int64_t xrow = (int64_t)(row0 + grp) * g.n_in;
        const bool rok = row0 + grp < B;
#pragma unroll
        for (int q = 0; q < kXRegs; ++q) {
            const int uu = sub + 32 * q;
            xr[q] = (rok && uu < kc && k0 + uu < k_total) ? x[xrow + units[k0 + uu]] : 0.0f;
        }
    };
    auto store_chunk = [&]() {
        int u = grp, v = sub;
#pragma unroll
        for (int q = 0; q < kSlots; ++q) {
            if (v < nvec && u < kc) reinterpret_cast<vec_t*>(ws + u * mpad)[v] = wr[q];
            v += 32;
            if (v >= nvec) { v = sub; u += kRowGroups; }
        }
#pragma unroll
        for (int q = 0; q < kXRegs; ++q) {
            const int uu = sub + 32 * q;
            if (uu < kc) xs[grp * xstride + uu] = xr[q];
        }
    };

    // With one tile per wave, two accumulator chains (even and odd k-steps) keep consecutive
    // MFMAs independent; with more tiles, the tiles do.
    constexpr int kChains = kTilesPerWave == 1 ? 2 : 1;
    d4 acc[kChains][kTilesPerWave];
#pragma unroll
    for (int c = 0; c < kChains; ++c)
#pragma unroll
        for (int t = 0; t < kTilesPerWave; ++t) acc[c][t] = d4{0.0, 0.0, 0.0, 0.0};
    // Output tile t of this wave is wave + 8 t; a wave with fewer tiles than kTilesPerWave
    // repeats its last valid one (same reads, result discarded), so the loop has no branches.
    int col_of[kTilesPerWave];
#pragma unroll
    for (int t = 0; t < kTilesPerWave; ++t) {
        const int nt = wave + t * kWaves;
        col_of[t] = (nt < lay.n_tiles ? nt : lay.n_tiles - 1) * 16 + (lane & 15);
    }


    // The input columns [c0, c1) of this workgroup's share of the x operand (see the epilogue),
    // in passes of 64 columns (lane = column): wave w takes passes 7 - w, 15 - w, ...  A pass
    // reads each of the 16 rows with one coalesced load (clamped in bounds, zero past the batch
    // or the range); the first pass is fetched before the softmax so that its latency hides.
    // (whole input HCUs: with complement pairs both units of a pair fall in one pass)
    const int64_t c0 = (int64_t)hj * g.in_hcu / g.out_hcu * g.in_mcu;
    const int64_t c1 = (int64_t)(hj + 1) * g.in_hcu / g.out_hcu * g.in_mcu;
    const int rows = B - row0 < kRows ? B - row0 : kRows;
    const int rt = row0 / kRows;
    const int n_pass = (int)((c1 - c0 + 63) / 64);
    const int pass0 = kWaves - 1 - wave;
    float xcol[kRows];
    // The rows are read through a buffer resource over the batch, so the rows past B read as
    // zero and all 16 loads are unconditional.  (Clamped to a valid row instead, the loads of
    // the rows past B shared one value, and the compiler loaded that row first and issued the
    // others only after it arrived.)  The launch checks that the offsets fit in 32 bits.
    const __amdgpu_buffer_rsrc_t xrs = input_rsrc(x, (uint32_t)((int64_t)B * g.n_in * 4));
    auto split_load = [&](int p) {
        const int64_t i = c0 + (int64_t)p * 64 + lane;
        const int64_t ic = i < c1 ? i : c1 - 1;
#pragma unroll
        for (int r = 0; r < kRows; ++r)
            xcol[r] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
                xrs, (uint32_t)(((int64_t)(row0 + r) * g.n_in + ic) * 4), 0, 0));
    };
    // With complement pairs every pair (x_2p, x_2p+1) of these rows must add up to 1.  The
    // range starts at an even column and passes are 64 columns wide, so the partner of an even
    // column is the next lane's column.  A violation sets the layer's flag.
    auto check_pairs = [&](int p) {
        const int64_t i = c0 + (int64_t)p * 64 + lane;
        const bool first = i < c1 && (i & 1) == 0;
        bool bad = false;
#pragma unroll
        for (int r = 0; r < kRows; ++r) {
            const float nb = __shfl_down(xcol[r], 1, 64);
            bad |= first && r < rows && !(fabsf(xcol[r] + nb - 1.0f) <= kPairTolerance);
        }
        if (bad) *ops.pair_error = 1;
    };
    auto split_store = [&](int p) {
        const int64_t i = c0 + (int64_t)p * 64 + lane;
        float sum = 0.0f;
#pragma unroll
        for (int r = 0; r < kRows; ++r) {
            xcol[r] = r < rows ? xcol[r] : 0.0f;
            sum += xcol[r];
        }
        if (ops.paired) check_pairs(p);
        if (i < c1) {
            // with complement pairs only the first unit of each input HCU enters the
            // contraction, at the HCU's index; every unit keeps its column sum
            if (!ops.paired) write_split_column(xcol, ops.x_hi, ops.x_lo, i, rt, ops.n_ks);
            else if ((i & 1) == 0) write_split_column(xcol, ops.x_hi, ops.x_lo, i >> 1, rt, ops.n_ks);
            ops.x_sum[(int64_t)rt * g.n_in + i] = sum;
        }
    };
    // With at most kWaves / 2 passes, each pass is split by two waves, rows 0-7 and 8-15 (task
    // q = kWaves - 1 - wave: pass q / 2, half q % 2): half the pair checks, conversions and
    // stores per wave.  The column sum is the two half sums added (as for t), exchanged through
    // the input panel's LDS, free by then.
    // (the panel lies past the support tile, which the t split reads meanwhile, when kc >= 16)
    const bool halves = has_ops && n_pass <= kWaves / 2 && kc >= kRows;
    const int hq = kWaves - 1 - wave, hpass = hq >> 1, hhalf = hq & 1;
    const bool hlive = halves && hpass < n_pass;
    float xh[kRows / 2];
    auto half_load = [&]() {
        const int64_t i = c0 + (int64_t)hpass * 64 + lane;
        const int64_t ic = i < c1 ? i : c1 - 1;
#pragma unroll
        for (int r = 0; r < kRows / 2; ++r)
            xh[r] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
                xrs, (uint32_t)(((int64_t)(row0 + 8 * hhalf + r) * g.n_in + ic) * 4), 0, 0));
    };
    float* hsum = xs;                                    // [n_pass][2][64] after the products
    auto half_store = [&]() {
        const int64_t i = c0 + (int64_t)hpass * 64 + lane;
        float sum = 0.0f;
#pragma unroll
        for (int r = 0; r < kRows / 2; ++r) {
            xh[r] = 8 * hhalf + r < rows ? xh[r] : 0.0f;
            sum += xh[r];
        }
        if (ops.paired) {
            const bool first = i < c1 && (i & 1) == 0;
            bool bad = false;
#pragma unroll
            for (int r = 0; r < kRows / 2; ++r) {
                const float nb = __shfl_down(xh[r], 1, 64);
                bad |= first && 8 * hhalf + r < rows && !(fabsf(xh[r] + nb - 1.0f) <= kPairTolerance);
            }
            if (bad) *ops.pair_error = 1;
        }
        if (i < c1) {
            if (!ops.paired) write_split_half(xh, ops.x_hi, ops.x_lo, i, rt, hhalf, ops.n_ks);
            else if ((i & 1) == 0) write_split_half(xh, ops.x_hi, ops.x_lo, i >> 1, rt, hhalf, ops.n_ks);
        }
        hsum[(hpass * 2 + hhalf) * 64 + lane] = sum;
    };

    if (k_total > 0) load_chunk(0);
    // Bias of this wave's columns, fetched now so that its latency hides behind the contraction
    // (after the first chunk's loads, which complete first).
    float bias_r[kTilesPerWave];
#pragma unroll
    for (int t = 0; t < kTilesPerWave; ++t) {
        const int c = col_of[t] < g.out_mcu ? col_of[t] : g.out_mcu - 1;
        bias_r[t] = bias[col_base + c];
    }
    for (int32_t k0 = 0; k0 < k_total; k0 += kc) {
        lds_barrier();                          // the previous chunk has been consumed
        store_chunk();
        lds_barrier();
        if (k0 + kc < k_total) load_chunk(k0 + kc);   // in flight during the MFMAs below
        // k-steps of 4 units (the rows beyond k_total hold zeros): groups of 8, then the rest
        const int rem = k_total - k0 < kc ? k_total - k0 : kc;
        const int ksteps = (rem + 3) / 4;
        int ks = 0;
        for (; ks + 8 <= ksteps; ks += 8) {
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int kk = (ks + u) * 4 + (lane >> 4);
                const double av = (double)xs[(lane & 15) * xstride + kk];
#pragma unroll
                for (int t = 0; t < kTilesPerWave; ++t) {
                    const double bv = (double)ws[kk * mpad + col_of[t]];
                    acc[u % kChains][t] =
                        __builtin_amdgcn_mfma_f64_16x16x4f64(av, bv, acc[u % kChains][t], 0, 0, 0);
                }
            }
        }
        for (; ks < ksteps; ++ks) {
            const int kk = ks * 4 + (lane >> 4);
            const double av = (double)xs[(lane & 15) * xstride + kk];
#pragma unroll
            for (int t = 0; t < kTilesPerWave; ++t) {
                const double bv = (double)ws[kk * mpad + col_of[t]];
                acc[0][t] = __builtin_amdgcn_mfma_f64_16x16x4f64(av, bv, acc[0][t], 0, 0, 0);
            }
        }
    }

    lds_barrier();   // done with the panels; the support tile reuses their LDS
#pragma unroll
    for (int t = 0; t < kTilesPerWave; ++t) {
        const int nt = wave + t * kWaves;
        if (nt < lay.n_tiles) {
            const int c = nt * 16 + (lane & 15);
            if (c < g.out_mcu) {
                const double bj = (double)bias_r[t];
#pragma unroll
                for (int r = 0; r < 4; ++r)
                {
                    double v = acc[0][t][r];
                    if constexpr (kChains == 2) v += acc[1][t][r];
                    stile[((lane >> 4) + 4 * r) * mpad + c] = (float)(v + bj);
                }
            }
        }
    }
    lds_barrier();

    if (hlive) half_load();
    else if (has_ops && !halves && pass0 < n_pass) split_load(pass0);

    // Each wave takes rows wave and wave + 8 together (independent reduction chains), one LDS
    // read per element: lane l holds columns l, l + 64, ... of both rows in registers
    // (M_out <= 128 kTilesPerWave, so 2 kTilesPerWave of them).
    static_assert(kRows == 2 * kWaves, "two softmax rows per wave");
    {
        constexpr int kPer = 2 * kTilesPerWave;
        const int ra = wave, rb = wave + kWaves;
        const bool va = row0 + ra < B, vb = row0 + rb < B;
        float* sa = stile + ra * mpad;
        float* sb = stile + rb * mpad;
        const int64_t oa = (int64_t)(row0 + ra) * g.n_out + col_base;
        const int64_t ob = (int64_t)(row0 + rb) * g.n_out + col_base;
        float ea[kPer], eb[kPer];
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            const int m = lane + 64 * q;
            ea[q] = m < g.out_mcu ? sa[m] : -INFINITY;
            eb[q] = m < g.out_mcu ? sb[m] : -INFINITY;
        }
        if (s) {
#pragma unroll
            for (int q = 0; q < kPer; ++q) {
                const int m = lane + 64 * q;
                if (m < g.out_mcu) {
                    if (va) s[oa + m] = ea[q];
                    if (vb) s[ob + m] = eb[q];
                }
            }
        }
        if (mode == 0) {
            float ma = -INFINITY, mb = -INFINITY;
#pragma unroll
            for (int q = 0; q < kPer; ++q) {
                ma = fmaxf(ma, ea[q]);
                mb = fmaxf(mb, eb[q]);
            }
            ma = wave_max_dpp(ma);
            mb = wave_max_dpp(mb);
            float da = 0.0f, db = 0.0f;
#pragma unroll
            for (int q = 0; q < kPer; ++q) {
                const bool in = lane + 64 * q < g.out_mcu;
                ea[q] = in ? expf(gain * (ea[q] - ma)) : 0.0f;
                eb[q] = in ? expf(gain * (eb[q] - mb)) : 0.0f;
                da += ea[q];
                db += eb[q];
            }
            da = wave_sum_dpp(da);
            db = wave_sum_dpp(db);
            const float ia = 1.0f / da, ib = 1.0f / db;
#pragma unroll
            for (int q = 0; q < kPer; ++q) {
                const int m = lane + 64 * q;
                if (m < g.out_mcu) {
                    const float ya = ea[q] * ia, yb = eb[q] * ib;
                    sa[m] = ya;                       // kept for the contraction operands
                    sb[m] = yb;
                    if (y && va) y[oa + m] = ya;   // training may not ask for them
                    if (y && vb) y[ob + m] = yb;
                }
            }
        } else {
            float bva = -INFINITY, bvb = -INFINITY;
            int bia = 0x7fffffff, bib = 0x7fffffff;
#pragma unroll
            for (int q = 0; q < kPer; ++q) {
                const int m = lane + 64 * q;
                if (m < g.out_mcu && ea[q] > bva) { bva = ea[q]; bia = m; }
                if (m < g.out_mcu && eb[q] > bvb) { bvb = eb[q]; bib = m; }
            }
            for (int off = 32; off > 0; off >>= 1) {
                const float ova = __shfl_xor(bva, off, 64), ovb = __shfl_xor(bvb, off, 64);
                const int oia = __shfl_xor(bia, off, 64), oib = __shfl_xor(bib, off, 64);
                if (ova > bva || (ova == bva && oia < bia)) { bva = ova; bia = oia; }
                if (ovb > bvb || (ovb == bvb && oib < bib)) { bvb = ovb; bib = oib; }
            }
            if (lane == 0) {
                if (va) winner[(int64_t)(row0 + ra) * g.out_hcu + hj] = bia;
                if (vb) winner[(int64_t)(row0 + rb) * g.out_hcu + hj] = bib;
            }
        }
    }
    if (!has_ops) {
        stamp_end<kStamp>(stamp);
        return;
    }

    // Contraction operands of this workgroup's share of the batch (rows row0 .. row0 + 15, one
    // k-step): the hidden HCU's columns of t (the activity above, or the target) and the input
    // columns [c0, c1) of x, each column split into bf16 hi / lo parts and written in fragment
    // order (of x, with complement pairs, the first unit of each input HCU), plus the column
    // sums over these rows.  Rows past B are written as zeros.
    // The t columns go out in halves of 8 rows (one 16-byte fragment chunk of hi and of lo per
    // half), so that 2 M_out threads share the work; the two halves of a column sit in
    // neighbouring lanes and add their row sums with one lane exchange.
    lds_barrier();
    const int n_half = 2 * g.out_mcu;
    for (int base = 0; base < n_half; base += kThreads) {          // uniform trip count
        const int q = base + tid;
        const bool live = q < n_half;
        const int m = live ? q >> 1 : 0;
        const int half = q & 1;
        float v[kRows / 2];
        float sum = 0.0f;
#pragma unroll
        for (int i = 0; i < kRows / 2; ++i) {
            const int r = 8 * half + i;
            v[i] = live && r < rows
                       ? (target ? target[(int64_t)(row0 + r) * g.n_out + col_base + m]
                                 : stile[r * mpad + m])
                       : 0.0f;
            sum += v[i];
        }
        const float total = sum + __shfl_xor(sum, 1, 64);           // same bits in both lanes
        if (live) {
            const int64_t col = col_base + m;
            write_split_half(v, ops.t_hi, ops.t_lo, col, rt, half, ops.n_ks);
            if (half == 0) ops.t_sum[(int64_t)rt * g.n_out + col] = total;
        }
    }
    if (halves) {
        if (hlive) half_store();
        lds_barrier();
        if (hlive && hhalf == 0) {
            const int64_t i = c0 + (int64_t)hpass * 64 + lane;
            if (i < c1)
                ops.x_sum[(int64_t)rt * g.n_in + i] =
                    hsum[(hpass * 2) * 64 + lane] + hsum[(hpass * 2 + 1) * 64 + lane];
        }
    } else {
        for (int p = pass0; p < n_pass; p += kWaves) {
            if (p != pass0) split_load(p);
            split_store(p);
        }
    }
    stamp_end<kStamp>(stamp);
}

constexpr size_t kLdsBudget = 120 * 1024;
constexpr size_t kLdsLimit = 160 * 1024;   // LDS of one gfx950 workgroup

SupportLayout make_layout(const Geometry& g, int32_t B, int32_t max_k, int vec, int lean_slots = 0) {
    SupportLayout L;
    L.n_tiles = (g.out_mcu + 15) / 16;
    // LDS row strides chosen so that the matrix-core operand reads of one half-wave (32 lanes:
    // 16 rows or columns at two consecutive k) fall on 32 distinct banks: the weight rows at a
    // stride of 16 mod 32 words, the input panel rows at 2 mod 32.
    L.mpad = L.n_tiles * 16 + (L.n_tiles % 2 == 0 ? 16 : 0);
    L.n_row_tiles = (B + kRows - 1) / kRows;
    L.k_alloc = max_k > 0 ? max_k : 1;
    // chunk rows such that every thread holds at most `slots` weight vectors
    const int vec_per_row = (g.out_mcu / vec + 31) / 32;
    const int tpw = (L.n_tiles + kWaves - 1) / kWaves;
    const int slots = lean_slots > 0 ? lean_slots
                                     : stage_slots(tpw <= 1 ? 1 : tpw <= 2 ? 2 : tpw <= 4 ? 4
                                                                             : kMaxTilesPerWave,
                                                   vec);
    const int by_regs_w = kRowGroups * (slots / vec_per_row);
    const int by_regs_x = 32 * kXRegs;
    const size_t fixed = (size_t)((L.k_alloc + 3) & ~3) * sizeof(int32_t);
    const size_t per_unit = (size_t)L.mpad * sizeof(float) + (size_t)kRows * sizeof(float);
    const int by_lds = (int)((kLdsBudget - fixed - kRows * sizeof(float)) / per_unit);
    int kc = by_regs_w < by_regs_x ? by_regs_w : by_regs_x;
    if (by_lds < kc) kc = by_lds;
    const int need = (max_k + 3) & ~3;
    if (need < kc) kc = need;
    kc &= ~3;
    if (kc < 4) kc = 4;
    // every thread must hold its share of a chunk: ceil(kc / 16) rows x vec_per_row vectors
    while (kc > 4 && ((kc + kRowGroups - 1) / kRowGroups) * vec_per_row > slots) kc -= 4;
    L.kc = kc;
    L.xstride = ((L.kc + 31) & ~31) + 2;
    L.fits = ((kc + kRowGroups - 1) / kRowGroups) * vec_per_row <= slots;
    return L;
}

size_t lds_bytes(const SupportLayout& L) {
    const size_t table = (size_t)((L.k_alloc + 3) & ~3) * sizeof(int32_t);
    const size_t panels = (size_t)L.kc * L.mpad * sizeof(float) +
                          (size_t)kRows * L.xstride * sizeof(float);
    const size_t tile = (size_t)kRows * L.mpad * sizeof(float);
    return table + (panels > tile ? panels : tile);
}

// Lets every support variant of one mode take dynamic LDS up to the workgroup's limit.
template <bool kOps, bool kStamp>
void raise_lds_limit() {
    const void* all[] = {(const void*)support_kernel<1, 4, kLeanSlots, kOps, kStamp>,
                         (const void*)support_kernel<1, 4, 0, kOps, kStamp>,
                         (const void*)support_kernel<2, 4, 0, kOps, kStamp>,
                         (const void*)support_kernel<4, 4, 0, kOps, kStamp>,
                         (const void*)support_kernel<kMaxTilesPerWave, 4, 0, kOps, kStamp>,
                         (const void*)support_kernel<1, 1, 0, kOps, kStamp>,
                         (const void*)support_kernel<2, 1, 0, kOps, kStamp>,
                         (const void*)support_kernel<4, 1, 0, kOps, kStamp>,
                         (const void*)support_kernel<kMaxTilesPerWave, 1, 0, kOps, kStamp>};
    for (const void* k : all)
        (void)hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsLimit);
}

}  // namespace

hipError_t launch_support(hipStream_t stream, const Geometry& g, const float* x, int32_t B,
                          const float* w, const float* bias, const int32_t* act_list,
                          const int32_t* act_count, int32_t max_active, float gain, int mode,
                          float* y, float* s, int32_t* winner, const float* target,
                          const TraceOperands* ops, hipEvent_t start, hipEvent_t stop,
                          unsigned long long* stamp) {
    const int vec = (g.out_mcu % 4 == 0 && g.n_out % 4 == 0) ? 4 : 1;
    SupportLayout lay = make_layout(g, B, max_active * g.in_mcu, vec);
    // A layer whose active rows take several chunks anyway stages fewer weight vectors per
    // thread (kLeanSlots): the kernel then needs few enough registers to share a SIMD with a
    // workgroup of the tiled silent sweep, which runs beside it on large layers.
    const bool lean = vec == 4 && lay.n_tiles <= kWaves && lay.kc < max_active * g.in_mcu;
    if (lean) lay = make_layout(g, B, max_active * g.in_mcu, vec, kLeanSlots);
    if (!lay.fits) return hipErrorInvalidValue;
    // the input rows of the last row tile (up to 15 past B) must have 32-bit byte offsets
    if ((int64_t)lay.n_row_tiles * kRows * g.n_in * 4 > (int64_t)UINT32_MAX) return hipErrorInvalidValue;
    const size_t lds = lds_bytes(lay);
    const int tpw = (lay.n_tiles + kWaves - 1) / kWaves;
    const int64_t blocks = (int64_t)lay.n_row_tiles * g.out_hcu;
    // allow dynamic LDS beyond 64 KB (gfx950 has 160 KB per workgroup): raised once, for
    // every variant a launch can pick, to the largest size a launch can ask for
    static std::once_flag raised;
    std::call_once(raised, [] {
        raise_lds_limit<false, false>();
        raise_lds_limit<true, false>();
        raise_lds_limit<true, true>();
        (void)hipGetLastError();
    });
    auto pick = [&](auto ops_c, auto stamp_c) -> hipError_t {
        constexpr bool O = decltype(ops_c)::value, S = decltype(stamp_c)::value;
        auto go = [&](auto kernel) {
            const TraceOperands o = ops ? *ops : TraceOperands{};
            // the events (when given) are recorded around the launch
            return launch_timed(kernel, dim3((unsigned)blocks), dim3(kThreads), lds, stream,
                                start, stop, g, lay, x, B, w, bias, act_list, act_count, gain,
                                mode, y, s, winner, target, o, stamp);
        };
        if (vec == 4) {
            if (lean) return go(support_kernel<1, 4, kLeanSlots, O, S>);
            if (tpw <= 1) return go(support_kernel<1, 4, 0, O, S>);
            if (tpw <= 2) return go(support_kernel<2, 4, 0, O, S>);
            if (tpw <= 4) return go(support_kernel<4, 4, 0, O, S>);
            return go(support_kernel<kMaxTilesPerWave, 4, 0, O, S>);
        }
        if (tpw <= 1) return go(support_kernel<1, 1, 0, O, S>);
        if (tpw <= 2) return go(support_kernel<2, 1, 0, O, S>);
        if (tpw <= 4) return go(support_kernel<4, 1, 0, O, S>);
        return go(support_kernel<kMaxTilesPerWave, 1, 0, O, S>);
    };
    if (!ops) return stamp ? hipErrorInvalidValue : pick(std::false_type{}, std::false_type{});
    return stamp ? pick(std::true_type{}, std::true_type{})
                 : pick(std::true_type{}, std::false_type{});
}

}  // namespace bcpnn
