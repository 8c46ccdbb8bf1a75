// Joint-trace contraction with the fused trace, weight and bias updates (Alg. 1 cycle loop):
//
//   T[i][j]  = sum_b x[b][i] t[b][j]                       (the batch sum of a_i (x) a_j)
//   Pij     <- c1 Pij + c2 T[i][j]                         c1 = 1 - a_eff, c2 = a_eff / B
//   Pi, Pj  <- c1 P + a_eff mean_b(.)                      (redundantly per block, see below)
//   w[i][j]  = log max(Pij,eps) - log max(Pi,eps) - log max(Pj,eps)   on active blocks only
//   b[j]     = k_B log max(Pj, eps)
//
// a_eff = 1 - (1 - alpha)^n_cycles folds the paper's n_cycles repetitions with the same batch
// means into one update (exact in real arithmetic).
//
// Design (gfx950):
//  * T is a dense [N_in x N_out] product with K = B (the batch).  Every Pij is needed (silent
//    connections are scored for plasticity), so the contraction is dense.
//  * T runs on the bf16 matrix cores with a two-term split of both operands: v = hi + lo with
//    hi = bf16(v), lo = bf16(v - hi), and T ~ lo.hi' + hi.lo' + hi.hi' (three
//    v_mfma_f32_32x32x16_bf16, fp32 accumulation).  Each product is then exact to about 3
//    parts in 2^17 (the dropped lo.lo' term and the rounding of lo), so T carries a relative
//    error of order 1e-5; the trace update scales it by a_eff / B, which puts it near 1e-8 in
//    Pij.  Three bf16 MFMAs cost 3/16 of the fp32 MFMA time of the same product, so the kernel
//    is bound by memory: 8 bytes of Pij per element plus 4 per active weight from HBM, and the
//    operands from L2.
//  * The support kernel of the same batch has already written x^T and t^T split, in MFMA
//    fragment order (one 1 KiB chunk per 32 units and 16 batch rows), and the column sums of x
//    and t per 16-row tile.
//  * Every wave owns one 32 x 32 block of Pij and works alone: no LDS staging, no barrier.  It
//    requests its Pij values, the inputs of its rows' and columns' marginal traces and its mask
//    bytes first, then streams the operands straight into registers (each k-step of each
//    operand is one contiguous 1 KiB read), four k-steps at a time, and runs the MFMAs.  The
//    many independent waves in flight hide the memory latency; measured per wave, a block is
//    two operand round trips plus the epilogue.
//  * A workgroup is four waves on one row block and four neighbouring column blocks: they read
//    the same x fragments (L1 hits after the first) and write 512 contiguous bytes of each row.
//    Workgroups are ordered so that those of one XCD cover one contiguous stretch of blocks.
//  * The marginal traces of the block's 32 rows (lanes 0..31) and 32 columns (lanes 32..63) are
//    computed by the wave itself from the column sums (same code and order in every block,
//    hence identical values) and spread to the lanes that need them with cross-lane reads; the
//    blocks of the first block column / row store the new Pi / Pj and b.  Pi and Pj are read
//    from one buffer and written to another (the host alternates them).
//  * Pij values are buffer loads over the block's rows (rows past the layer read as zero); all
//    stores are unconditional buffer stores, a store that must not happen getting an offset
//    past the buffer range, which the hardware drops.  w is written on active blocks only.
//
// MFMA 32x32x16 bf16 lane layout (verified on gfx950): A[i][k] for k = 8 (l / 32) + 0..7 from
// lane l = i + 32 (k / 8), B[k][j] likewise with j = l % 32, and lane l holds
// D[8 (r / 4) + 4 (l / 32) + r % 4][l % 32] in result register r.
#include <hip/hip_ext.h>

#include "bcpnn_internal.h"
#include "device_common.h"

namespace bcpnn {
namespace {

typedef float f16v __attribute__((ext_vector_type(16)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __amdgpu_buffer_rsrc_t rsrc_t;

constexpr int kWaves = 4;           // waves (32 x 32 blocks) per workgroup, along the columns
constexpr int kChunk = 4;           // k-steps (16 batch rows each) of operands per round trip
constexpr int kSums = 8;            // column-sum tiles requested up front (the batch for B <= 128)
constexpr int kSweepRows = 16;      // row blocks per sweep over the column groups (see below)
constexpr uint32_t kDrop = 0x80000000u;   // byte offset past every block's buffer range

// Buffer resource over [p, p + bytes): raw (stride 0) addressing, 32-bit data format.  A load
// at an offset >= bytes returns zero and a store there is discarded by the hardware.
__device__ __forceinline__ rsrc_t make_rsrc(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

// Round-to-nearest-even to the storage mantissa (kDropBits low bits cleared); Inf / NaN kept.
template <int kDropBits>
__device__ __forceinline__ float to_storage(float v) {
    if constexpr (kDropBits == 0) {
        return v;
    } else {
        const uint32_t u = __float_as_uint(v);
        const uint32_t r = (u + ((1u << (kDropBits - 1)) - 1u) + ((u >> kDropBits) & 1u)) &
                           ~((1u << kDropBits) - 1u);
        return (u & 0x7f800000u) == 0x7f800000u ? v : __uint_as_float(r);
    }
}

template <int kDropBits>
__global__ void __launch_bounds__(kWaves * 64) __attribute__((amdgpu_waves_per_eu(3, 3)))
trace_kernel(Geometry g, TraceArgs a, int n_cg) {
    const int lane = threadIdx.x & 63;
    const int n_in = (int)g.n_in, n_out = (int)g.n_out;
    // workgroup -> (row block, group of kWaves column blocks).  The workgroups of one XCD take
    // one contiguous stretch of this order, which sweeps kSweepRows row blocks over every column
    // group, column group by column group: the x fragments of the sweep (kSweepRows blocks) stay
    // in the XCD's L2 while the t fragments stream through it once per sweep.
    const int n_rb = (n_in + 31) / 32;
    const int wg = (int)xcd_linear_index(blockIdx.x, gridDim.x);
    const int sweep = wg / (kSweepRows * n_cg);
    const int in_sweep = wg % (kSweepRows * n_cg);
    const int rows_here = n_rb - sweep * kSweepRows < kSweepRows ? n_rb - sweep * kSweepRows
                                                                  : kSweepRows;
    const int bi = sweep * kSweepRows + in_sweep % rows_here;
    const int bj = (in_sweep / rows_here) * kWaves + (threadIdx.x >> 6);
    const int i0 = bi * 32, j0 = bj * 32;
    if (j0 >= n_out) return;                                   // wave-uniform; no barriers
    const int rows = n_in - i0 < 32 ? n_in - i0 : 32;
    const int cols = n_out - j0 < 32 ? n_out - j0 : 32;
    const int nk = (a.B + 15) / 16;                            // k-steps = 16-row tiles
    const int n_ks = a.ops.n_ks;
    const int jl = lane & 31;
    const int il0 = 4 * (lane >> 5);

    // ---- requests that do not depend on the contraction -----------------------------------
    const rsrc_t rp = make_rsrc(a.pij + (int64_t)i0 * n_out, (uint32_t)rows * n_out * 4u);
    const uint32_t o0 = ((uint32_t)il0 * n_out + j0 + jl) * 4u;
    float pold[16];
#pragma unroll
    for (int r = 0; r < 16; ++r)
        pold[r] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
            rp, o0 + (uint32_t)(8 * (r >> 2) + (r & 3)) * n_out * 4u, 0, 0));
    // marginal inputs: lanes 0..31 the block's row units, 32..63 its column units (clamped)
    const bool is_row = lane < 32;
    const int u = is_row ? i0 + (lane < rows ? lane : rows - 1)
                         : j0 + (lane - 32 < cols ? lane - 32 : cols - 1);
    const float* sums = is_row ? a.ops.x_sum : a.ops.t_sum;
    const int64_t st = is_row ? n_in : n_out;
    float part[kSums];
#pragma unroll
    for (int q = 0; q < kSums; ++q) part[q] = sums[(q < nk ? q : nk - 1) * st + u];
    const float p_old = is_row ? a.pi_old[u] : a.pj_old[u];
    // Mask of the lane's column over the block's 32 rows, one bit per row.  HCU of every row /
    // column unit, spread by lane reads.  When the block's columns fall in at most two hidden
    // HCUs (always for M_out >= 32), lane l reads the byte of row l % 32 and hidden HCU
    // hc0 + l / 32, and one ballot gives both HCUs' row masks; otherwise every lane reads the
    // bytes of its 16 elements.
    const int hu = is_row ? u / g.in_mcu : u / g.out_mcu;
    const int hj = __shfl(hu, 32 + jl, 64);
    const int hc0 = __shfl(hu, 32, 64), hc1 = __shfl(hu, 63, 64);
    uint32_t act_bits = 0;
    if (hc1 - hc0 <= 1) {                                      // wave-uniform
        const int hr = __shfl(hu, jl, 64);
        const int hc = hc0 + (lane >> 5) < hc1 ? hc0 + (lane >> 5) : hc1;
        const uint64_t bits = __ballot(a.mask[(int64_t)hr * g.out_hcu + hc] != 0);
        act_bits = hj == hc0 ? (uint32_t)bits : (uint32_t)(bits >> 32);
    } else {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int il = il0 + 8 * (r >> 2) + (r & 3);
            const int hi = __shfl(hu, il, 64);
            act_bits |= (a.mask[(int64_t)hi * g.out_hcu + hj] != 0 ? 1u : 0u) << il;
        }
    }

    // ---- contraction: operands straight from the fragment-order arrays -----------------------
    const int64_t fa = ((int64_t)bi * n_ks * 64 + lane) * 8;
    const int64_t fb = ((int64_t)bj * n_ks * 64 + lane) * 8;
    f16v acc = {};
    for (int k0 = 0; k0 < nk; k0 += kChunk) {
        u32x4 op[kChunk][4];
#pragma unroll
        for (int c = 0; c < kChunk; ++c) {
            const int64_t ks = (int64_t)(k0 + c < nk ? k0 + c : nk - 1) * 512;
            op[c][0] = *reinterpret_cast<const u32x4*>(a.ops.x_hi + fa + ks);
            op[c][1] = *reinterpret_cast<const u32x4*>(a.ops.x_lo + fa + ks);
            op[c][2] = *reinterpret_cast<const u32x4*>(a.ops.t_hi + fb + ks);
            op[c][3] = *reinterpret_cast<const u32x4*>(a.ops.t_lo + fb + ks);
        }
#pragma unroll
        for (int c = 0; c < kChunk; ++c) {
            if (k0 + c < nk) {
                const bf8 ah = __builtin_bit_cast(bf8, op[c][0]);
                const bf8 al = __builtin_bit_cast(bf8, op[c][1]);
                const bf8 bh = __builtin_bit_cast(bf8, op[c][2]);
                const bf8 bl = __builtin_bit_cast(bf8, op[c][3]);
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, bh, acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bl, acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bh, acc, 0, 0, 0);
            }
        }
    }

    // ---- marginal traces of the block's rows and columns, and their logs --------------------
    float colsum = 0.0f;
#pragma unroll
    for (int q = 0; q < kSums; ++q)
        if (q < nk) colsum += part[q];
    for (int q = kSums; q < nk; ++q) colsum += sums[q * st + u];     // batches above 128
    const float p = fmaf(a.a_eff, colsum * a.inv_b, a.c1 * p_old);
    const float lp = fast_log(fmaxf(p, a.eps));
    if (is_row && lane < rows && bj == 0) a.pi_new[u] = p;
    if (!is_row && lane - 32 < cols && bi == 0) {
        a.pj_new[u] = p;
        a.b[u] = a.bias_gain * lp;
    }
    const float lpj = __shfl(lp, 32 + jl, 64);

    // ---- epilogue: joint trace and masked weights, 32 unconditional buffer stores per lane ----
    const bool jok = jl < cols;
    const rsrc_t rw = make_rsrc(a.w + (int64_t)i0 * n_out, (uint32_t)rows * n_out * 4u);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int il = il0 + 8 * (r >> 2) + (r & 3);
        const float lpi = __shfl(lp, il, 64);
        const uint32_t off = o0 + (uint32_t)(8 * (r >> 2) + (r & 3)) * n_out * 4u;
        const float pn = to_storage<kDropBits>(fmaf(a.c2, acc[r], a.c1 * pold[r]));
        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(pn), rp, jok ? off : kDrop, 0, 0);
        const float wv = to_storage<kDropBits>(fast_log(fmaxf(pn, a.eps)) - lpi - lpj);
        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(wv), rw,
                                              jok && ((act_bits >> il) & 1u) ? off : kDrop, 0, 0);
    }
}

}  // namespace

hipError_t launch_trace_update(hipStream_t stream, const Geometry& g, const TraceArgs& a,
                               hipEvent_t start, hipEvent_t stop) {
    const int64_t n_rb = (g.n_in + 31) / 32, n_cb = (g.n_out + 31) / 32;
    const int64_t n_cg = (n_cb + kWaves - 1) / kWaves;
    void (*kernel)(Geometry, TraceArgs, int) = nullptr;
    switch (a.drop_bits) {
        case 0: kernel = trace_kernel<0>; break;
        case 13: kernel = trace_kernel<13>; break;
        case 16: kernel = trace_kernel<16>; break;
        default: return hipErrorInvalidValue;
    }
    // the events (when given) are stamped by the dispatch itself, so they time the kernel alone
    hipExtLaunchKernelGGL(kernel, dim3((unsigned)(n_rb * n_cg)), dim3(kWaves * 64), 0, stream,
                          start, stop, 0, g, a, (int)n_cg);
    return hipGetLastError();
}

}  // namespace bcpnn
