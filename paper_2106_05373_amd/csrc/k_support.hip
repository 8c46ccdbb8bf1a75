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
#include "bcpnn_internal.h"
#include "device_common.h"

namespace bcpnn {
namespace {

typedef double d4 __attribute__((ext_vector_type(4)));

constexpr int kRows = 16;          // batch rows per workgroup
constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kMaxTilesPerWave = 8;   // kWaves * 8 * 16 = 1024 = largest out_mcu
// Weight elements staged per thread per chunk: fewer when the accumulators need the registers.
constexpr int weight_regs(int tiles_per_wave) { return tiles_per_wave <= 2 ? 32 : 16; }
constexpr int kXRegs = 8;          // input elements staged per thread per chunk

struct SupportLayout {
    int n_tiles, mpad, n_row_tiles;
    int kc;                        // units per chunk (multiple of 4)
    int k_alloc;                   // LDS entries of the unit table (>= the largest K_h)
    int xstride;                   // LDS row stride of the input panel (kc + 1: no bank aliasing)
};

// kTilesPerWave: 16-column output tiles per wave, ceil(ceil(M_out / 16) / 8).
template <int kTilesPerWave>
__global__ void __launch_bounds__(kThreads)
support_kernel(Geometry g, SupportLayout lay, const float* __restrict__ x, int32_t B,
               const float* __restrict__ w, const float* __restrict__ bias,
               const int32_t* __restrict__ act_list, const int32_t* __restrict__ act_count,
               float gain, int mode, float* __restrict__ y, float* __restrict__ s,
               int32_t* __restrict__ winner) {
    extern __shared__ float lds[];
    const int kc = lay.kc, mpad = lay.mpad, xstride = lay.xstride;
    int32_t* units = reinterpret_cast<int32_t*>(lds);               // [k_alloc]
    float* ws = lds + lay.k_alloc;                                   // [kc][mpad]
    float* xs = ws + (size_t)kc * mpad;                              // [kRows][xstride]
    float* stile = ws;                                               // [kRows][mpad] afterwards

    const int64_t work = xcd_linear_index(blockIdx.x, (int64_t)lay.n_row_tiles * g.out_hcu);
    const int hj = (int)(work / lay.n_row_tiles);
    const int row0 = (int)(work % lay.n_row_tiles) * kRows;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;

    const int32_t k_total = act_count[hj] * g.in_mcu;
    const int32_t* alist = act_list + (int64_t)hj * g.in_hcu;
    const int64_t col_base = (int64_t)hj * g.out_mcu;
    for (int32_t k = tid; k < k_total; k += kThreads)
        units[k] = alist[k / g.in_mcu] * g.in_mcu + k % g.in_mcu;
    __syncthreads();

    constexpr int kWRegs = weight_regs(kTilesPerWave);
    const int w_elems = kc * g.out_mcu;
    const int x_elems = kRows * kc;
    float wr[kWRegs], xr[kXRegs];
    auto load_chunk = [&](int32_t k0) {
#pragma unroll
        for (int q = 0; q < kWRegs; ++q) {
            const int e = q * kThreads + tid;
            const int u = e / g.out_mcu, c = e - u * g.out_mcu;
            wr[q] = (e < w_elems && k0 + u < k_total)
                        ? w[(int64_t)units[k0 + u] * g.n_out + col_base + c] : 0.0f;
        }
#pragma unroll
        for (int q = 0; q < kXRegs; ++q) {
            const int e = q * kThreads + tid;
            const int r = e / kc, u = e - r * kc;
            xr[q] = (e < x_elems && k0 + u < k_total && row0 + r < B)
                        ? x[(int64_t)(row0 + r) * g.n_in + units[k0 + u]] : 0.0f;
        }
    };
    auto store_chunk = [&]() {
#pragma unroll
        for (int q = 0; q < kWRegs; ++q) {
            const int e = q * kThreads + tid;
            if (e < w_elems) {
                const int u = e / g.out_mcu, c = e - u * g.out_mcu;
                ws[u * mpad + c] = wr[q];
            }
        }
#pragma unroll
        for (int q = 0; q < kXRegs; ++q) {
            const int e = q * kThreads + tid;
            if (e < x_elems) {
                const int r = e / kc, u = e - r * kc;
                xs[r * xstride + u] = xr[q];
            }
        }
    };

    d4 acc[kTilesPerWave];
#pragma unroll
    for (int t = 0; t < kTilesPerWave; ++t) acc[t] = d4{0.0, 0.0, 0.0, 0.0};

    if (k_total > 0) load_chunk(0);
    for (int32_t k0 = 0; k0 < k_total; k0 += kc) {
        __syncthreads();                          // the previous chunk has been consumed
        store_chunk();
        __syncthreads();
        if (k0 + kc < k_total) load_chunk(k0 + kc);   // in flight during the MFMAs below
        const int ksteps = (k_total - k0 < kc ? k_total - k0 + 3 : kc) / 4;
        for (int ks = 0; ks < ksteps; ++ks) {
            const int kk = ks * 4 + (lane >> 4);
            const double av = (double)xs[(lane & 15) * xstride + kk];
#pragma unroll
            for (int t = 0; t < kTilesPerWave; ++t) {
                const int nt = wave + t * kWaves;
                if (nt < lay.n_tiles) {           // uniform across the wave
                    const double bv = (double)ws[kk * mpad + nt * 16 + (lane & 15)];
                    acc[t] = __builtin_amdgcn_mfma_f64_16x16x4f64(av, bv, acc[t], 0, 0, 0);
                }
            }
        }
    }

    __syncthreads();   // done with the panels; the support tile reuses their LDS
#pragma unroll
    for (int t = 0; t < kTilesPerWave; ++t) {
        const int nt = wave + t * kWaves;
        if (nt < lay.n_tiles) {
            const int c = nt * 16 + (lane & 15);
            if (c < g.out_mcu) {
                const double bj = (double)bias[col_base + c];
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    stile[((lane >> 4) + 4 * r) * mpad + c] = (float)(acc[t][r] + bj);
            }
        }
    }
    __syncthreads();

    for (int r = wave; r < kRows; r += kWaves) {
        const int row = row0 + r;
        if (row >= B) break;                          // uniform across the wave
        const float* srow = stile + r * mpad;
        const int64_t out = (int64_t)row * g.n_out + col_base;
        if (s)
            for (int m = lane; m < g.out_mcu; m += 64) s[out + m] = srow[m];
        if (mode == 0) {
            float mx = -INFINITY;
            for (int m = lane; m < g.out_mcu; m += 64) mx = fmaxf(mx, srow[m]);
            mx = wave_max(mx);
            float den = 0.0f;
            for (int m = lane; m < g.out_mcu; m += 64) den += expf(gain * (srow[m] - mx));
            den = wave_sum(den);
            const float inv = 1.0f / den;
            for (int m = lane; m < g.out_mcu; m += 64) y[out + m] = expf(gain * (srow[m] - mx)) * inv;
        } else {
            float bv = -INFINITY;
            int bi = 0x7fffffff;
            for (int m = lane; m < g.out_mcu; m += 64)
                if (srow[m] > bv) { bv = srow[m]; bi = m; }
            for (int off = 32; off > 0; off >>= 1) {
                const float ov = __shfl_xor(bv, off, 64);
                const int oi = __shfl_xor(bi, off, 64);
                if (ov > bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
            }
            if (lane == 0) winner[(int64_t)row * g.out_hcu + hj] = bi;
        }
    }
}

constexpr size_t kLdsBudget = 120 * 1024;

SupportLayout make_layout(const Geometry& g, int32_t B, int32_t max_k) {
    SupportLayout L;
    L.n_tiles = (g.out_mcu + 15) / 16;
    const int kWRegs = weight_regs((L.n_tiles + kWaves - 1) / kWaves);
    L.mpad = L.n_tiles * 16;
    L.n_row_tiles = (B + kRows - 1) / kRows;
    L.k_alloc = max_k > 0 ? max_k : 1;
    const int by_regs_w = kWRegs * kThreads / g.out_mcu;
    const int by_regs_x = kXRegs * kThreads / kRows;
    const size_t fixed = (size_t)L.k_alloc * sizeof(int32_t);
    const size_t per_unit = (size_t)L.mpad * sizeof(float) + (size_t)kRows * sizeof(float);
    const int by_lds = (int)((kLdsBudget - fixed - kRows * sizeof(float)) / per_unit);
    int kc = by_regs_w < by_regs_x ? by_regs_w : by_regs_x;
    if (by_lds < kc) kc = by_lds;
    const int need = (max_k + 3) & ~3;
    if (need < kc) kc = need;
    kc &= ~3;
    L.kc = kc < 4 ? 4 : kc;
    L.xstride = L.kc + 1;
    return L;
}

size_t lds_bytes(const SupportLayout& L) {
    const size_t panels = (size_t)L.k_alloc * sizeof(int32_t) +
                          (size_t)L.kc * L.mpad * sizeof(float) +
                          (size_t)kRows * L.xstride * sizeof(float);
    const size_t tile = (size_t)L.k_alloc * sizeof(int32_t) + (size_t)kRows * L.mpad * sizeof(float);
    return panels > tile ? panels : tile;
}

}  // namespace

hipError_t launch_support(hipStream_t stream, const Geometry& g, const float* x, int32_t B,
                          const float* w, const float* bias, const int32_t* act_list,
                          const int32_t* act_count, int32_t max_active, float gain, int mode,
                          float* y, float* s, int32_t* winner) {
    const SupportLayout lay = make_layout(g, B, max_active * g.in_mcu);
    const size_t lds = lds_bytes(lay);
    const int tpw = (lay.n_tiles + kWaves - 1) / kWaves;
    const int64_t blocks = (int64_t)lay.n_row_tiles * g.out_hcu;
    auto go = [&](auto kernel) {
        if (lds > 64 * 1024) {
            // allow dynamic LDS beyond 64 KB (gfx950 has 160 KB per workgroup)
            (void)hipFuncSetAttribute((const void*)kernel,
                                      hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
            (void)hipGetLastError();
        }
        kernel<<<(unsigned)blocks, kThreads, lds, stream>>>(g, lay, x, B, w, bias, act_list,
                                                            act_count, gain, mode, y, s, winner);
        return hipGetLastError();
    };
    if (tpw <= 1) return go(support_kernel<1>);
    if (tpw <= 2) return go(support_kernel<2>);
    if (tpw <= 4) return go(support_kernel<4>);
    return go(support_kernel<kMaxTilesPerWave>);
}

}  // namespace bcpnn
