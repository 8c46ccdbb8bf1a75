// Joint-trace contraction with the fused trace, weight and bias updates (Alg. 1 cycle loop):
//
//   T[i][j]  = sum_b x[b][i] t[b][j]                       (the batch sum of a_i (x) a_j)
//   Pij     <- c1 Pij + c2 T[i][j]                         c1 = 1 - a_eff, c2 = a_eff / B
//   Pi, Pj  <- c1 P + a_eff mean_b(.)                      (redundantly per tile, see below)
//   w[i][j]  = log(max(Pij,eps) / (max(Pi,eps) max(Pj,eps)))   on active blocks only
//   b[j]     = k_B log(max(Pj, eps))
//
// a_eff = 1 - (1 - alpha)^n_cycles folds the paper's n_cycles repetitions with the same batch
// means into one update (exact in real arithmetic).
//
// Design (gfx950):
//  * T is a dense [N_in x N_out] product with K = B (the batch).  Every Pij is needed (silent
//    connections are scored for plasticity), so the contraction is dense.
//  * T runs on the bf16 matrix cores with a two-term split of both operands: v = hi + lo with
//    hi = bf16(v), lo = bf16(v - hi), and T ~ hi.hi' + hi.lo' + lo.hi' (three
//    v_mfma_f32_32x32x16_bf16, fp32 accumulation).  Each product is then exact to about 3
//    parts in 2^17 (the dropped lo.lo' term and the rounding of lo), so T carries a relative
//    error of order 1e-5; the trace update scales it by a_eff / B, which puts it near 1e-8 in
//    Pij.  Three bf16 MFMAs cost 3/16 of the fp32 MFMA time of the same product.
//  * The support kernel of the same batch has already written x^T and t^T split and
//    transposed ([unit][batch] bf16, the MFMA operand order) and the column sums of x and t
//    per 16-row tile.  Splitting here would repeat the work for every tile that shares a row or
//    column panel (47 and 25 times on the MNIST-shaped layer).
//  * A workgroup owns a 64 x 64 tile of Pij; each of its four waves one 32 x 32 block.  Small
//    tiles give ~1200 workgroups for the MNIST-shaped layer, so 256 CUs receive near-equal
//    shares.  The batch is streamed in chunks of 32 rows: every thread copies four 16-byte
//    fragments per chunk into LDS (one per operand half), the next chunk's through registers
//    while the current one feeds the matrix cores.  In LDS each 64-byte row holds four 16-byte
//    groups, placed at slot group ^ ((row / 4) % 4): the 16 lanes of one phase of a 128-bit
//    operand read then hit 16 different bank groups.
//  * A workgroup's life is a few microseconds, mostly memory latency, so the loads it needs
//    later (its 16 Pij values per lane, the old Pi / Pj, the column sums, the mask block) are
//    issued at its start and overlap the contraction.  Few registers are held, so several
//    workgroups share each CU and hide one another's latency.
//  * Every workgroup computes the new Pi / Pj of its rows / columns itself from the column
//    sums (same code, same order, hence identical values) and the tiles of the first column /
//    row store them.  Pi and Pj are read from one buffer and written to another (the host
//    alternates them), so no workgroup reads an updated value.
//  * Each Pij is read once and written once; w is written only on active blocks (silent blocks
//    of w stay zero), so the HBM traffic that scales with N_in * N_out is 8 bytes per element
//    plus 4 per active element.
//
// MFMA 32x32x16 bf16 lane layout (verified on gfx950): A[i][k] for k = 8 (l / 32) + 0..7 from
// lane l = i + 32 (k / 8), B[k][j] likewise with j = l % 32, and lane l holds
// D[8 (r / 4) + 4 (l / 32) + r % 4][l % 32] in result register r.
#include "bcpnn_internal.h"
#include "device_common.h"

namespace bcpnn {
namespace {

typedef float f16v __attribute__((ext_vector_type(16)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));

constexpr int kTM = 64;            // Pij rows (input units) per tile
constexpr int kTN = 64;            // Pij columns (hidden units) per tile
constexpr int kTK = 32;            // batch rows per staged chunk (one 64-byte bf16 row)
constexpr int kThreads = 256;
constexpr int kSums = 16;          // column-sum tiles loaded together

// LDS slot of 16-byte group g (0..3) of row r.
__device__ __forceinline__ int slot(int r, int g) { return g ^ ((r >> 2) & 3); }

__global__ void __launch_bounds__(kThreads)
trace_kernel(Geometry g, TraceArgs a) {
    __shared__ uint4 pan[4][kTM][4];          // x hi, x lo, t hi, t lo: [row][16-byte slot]
    __shared__ float pi_t[kTM];
    __shared__ float pj_t[kTN];
    __shared__ int32_t row_h[kTM];
    __shared__ int32_t col_h[kTN];
    __shared__ uint8_t mtile[kTM * kTN];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int64_t j0 = (int64_t)blockIdx.x * kTN;
    const int64_t i0 = (int64_t)blockIdx.y * kTM;
    const int64_t kp = a.ops.kp;

    // Loads are issued in the order their data is needed: waiting for one load also waits for
    // every load issued before it.

    // ---- mask block of the tile (indexed by row HCU - first, column HCU - first) ------------
    const bool is_row = tid < kTM, is_col = tid >= kTM && tid < kTM + kTN;
    const int64_t hi0 = i0 / g.in_mcu;
    const int64_t hj0 = j0 / g.out_mcu;
    const int64_t i_last = (i0 + kTM < g.n_in ? i0 + kTM : g.n_in) - 1;
    const int64_t j_last = (j0 + kTN < g.n_out ? j0 + kTN : g.n_out) - 1;
    const int nhi = (int)(i_last / g.in_mcu - hi0 + 1);
    const int nhj = (int)(j_last / g.out_mcu - hj0 + 1);
    if (is_row) row_h[tid] = (int32_t)((i0 + tid) / g.in_mcu - hi0);
    else if (is_col) col_h[tid - kTM] = (int32_t)((j0 + tid - kTM) / g.out_mcu - hj0);
    for (int e = tid; e < nhi * nhj; e += kThreads)
        mtile[e] = a.mask[(hi0 + e / nhj) * g.out_hcu + hj0 + e % nhj];

    // ---- first chunk of the contraction operands ---------------------------------------------
    // Thread -> (row r = tid / 4, slot s = tid % 4) of each of the four operand halves; it
    // fetches group slot(r, s) of that row so that the group lands in slot s.
    const int sr = tid >> 2, ss = tid & 3;
    const int sg = slot(sr, ss);
    const bool a_ok = i0 + sr < g.n_in, b_ok = j0 + sr < g.n_out;
    const uint4* xh = reinterpret_cast<const uint4*>(a.ops.x_hi + (i0 + sr) * kp + sg * 8);
    const uint4* xl = reinterpret_cast<const uint4*>(a.ops.x_lo + (i0 + sr) * kp + sg * 8);
    const uint4* th = reinterpret_cast<const uint4*>(a.ops.t_hi + (j0 + sr) * kp + sg * 8);
    const uint4* tl = reinterpret_cast<const uint4*>(a.ops.t_lo + (j0 + sr) * kp + sg * 8);
    uint4 st0 = make_uint4(0u, 0u, 0u, 0u), st1 = st0, st2 = st0, st3 = st0;
    // k0: a multiple of 32 batch rows = 4 uint4 of a row; rows outside the tile stay zero
#define BCPNN_FETCH(k0)                 \
    if (a_ok) {                         \
        st0 = xh[(k0) / 8];             \
        st1 = xl[(k0) / 8];             \
    }                                   \
    if (b_ok) {                         \
        st2 = th[(k0) / 8];             \
        st3 = tl[(k0) / 8];             \
    }
    BCPNN_FETCH(0);

    // ---- requests for the epilogue: the lane's Pij values, the old Pi / Pj and the column
    // sums of the first row tiles (threads 0..63: row i0 + tid of x; 64..127: column
    // j0 + tid - 64 of t) ---------------------------------------------------------------------
    const int jl = wn * 32 + (lane & 31);
    const int64_t j = j0 + jl;
    const bool jok = j < g.n_out;
    const int il0 = wm * 32 + 4 * (lane >> 5);
    float* __restrict__ pij = a.pij + (i0 + il0) * g.n_out + j;
    float pold[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const bool ok = jok && i0 + il0 + 8 * (r >> 2) + (r & 3) < g.n_in;
        pold[r] = ok ? pij[(int64_t)(8 * (r >> 2) + (r & 3)) * g.n_out] : 0.0f;
    }
    const int64_t unit = is_row ? i0 + tid : j0 + (tid - kTM);
    const bool unit_ok = (is_row && unit < g.n_in) || (is_col && unit < g.n_out);
    const float* sums = is_row ? a.ops.x_sum : a.ops.t_sum;
    const int64_t sum_stride = is_row ? g.n_in : g.n_out;
    const int n_rt = (a.B + 15) / 16;
    float part[kSums];
#pragma unroll
    for (int q = 0; q < kSums; ++q)
        part[q] = (unit_ok && q < n_rt) ? sums[(int64_t)q * sum_stride + unit] : 0.0f;
    const float p_old = unit_ok ? (is_row ? a.pi_old[unit] : a.pj_old[unit]) : 0.0f;

    // ---- contraction ------------------------------------------------------------------------
    f16v acc0, acc1;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc0[r] = acc1[r] = 0.0f;
    const int kc = (a.B + kTK - 1) / kTK * kTK;       // rows B .. kc - 1 of the operands are zero
    const int ar = wm * 32 + (lane & 31), br = wn * 32 + (lane & 31);
    for (int k0 = 0; k0 < kc; k0 += kTK) {
        __syncthreads();                               // the previous chunk has been consumed
        pan[0][sr][ss] = st0;
        pan[1][sr][ss] = st1;
        pan[2][sr][ss] = st2;
        pan[3][sr][ss] = st3;
        __syncthreads();
        if (k0 + kTK < kc) {                           // in flight during the MFMAs below
            BCPNN_FETCH(k0 + kTK);
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {                  // two k-steps of 16
            const int gq = 2 * h + (lane >> 5);        // this lane's 16-byte group
            const bf8 ah = __builtin_bit_cast(bf8, pan[0][ar][slot(ar, gq)]);
            const bf8 al = __builtin_bit_cast(bf8, pan[1][ar][slot(ar, gq)]);
            const bf8 bh = __builtin_bit_cast(bf8, pan[2][br][slot(br, gq)]);
            const bf8 bl = __builtin_bit_cast(bf8, pan[3][br][slot(br, gq)]);
            acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bh, acc0, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bl, acc1, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, bh, acc1, 0, 0, 0);
        }
    }

#undef BCPNN_FETCH

    // ---- new marginal traces of the tile's rows and columns ---------------------------------
    if (unit_ok) {
        float colsum = 0.0f;
#pragma unroll
        for (int q = 0; q < kSums; ++q) colsum += part[q];
        for (int r0 = kSums; r0 < n_rt; r0 += kSums) {   // batches of more than 16 * kSums rows
#pragma unroll
            for (int q = 0; q < kSums; ++q)
                part[q] = r0 + q < n_rt ? sums[(int64_t)(r0 + q) * sum_stride + unit] : 0.0f;
#pragma unroll
            for (int q = 0; q < kSums; ++q) colsum += part[q];
        }
        const float p = fmaf(a.a_eff, colsum * a.inv_b, a.c1 * p_old);
        if (is_row) {
            pi_t[tid] = p;
            if (blockIdx.x == 0) a.pi_new[unit] = p;
        } else {
            pj_t[tid - kTM] = p;
            if (blockIdx.y == 0) {
                a.pj_new[unit] = p;
                a.b[unit] = a.bias_gain * __logf(fmaxf(p, a.eps));
            }
        }
    }
    __syncthreads();

    // ---- epilogue: joint trace from the prefetched values, then the masked weights ----------
    const float pjv = jok ? pj_t[jl] : 1.0f;
    float* __restrict__ wp = a.w + (i0 + il0) * g.n_out + j;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int il = il0 + 8 * (r >> 2) + (r & 3);
        if (!jok || i0 + il >= g.n_in) continue;
        const int64_t off = (int64_t)(8 * (r >> 2) + (r & 3)) * g.n_out;
        float p = fmaf(a.c2, acc0[r] + acc1[r], a.c1 * pold[r]);
        p = round_storage(p, a.drop_bits);
        pij[off] = p;
        if (mtile[row_h[il] * nhj + col_h[jl]])
            wp[off] = round_storage(log_ratio(p, pi_t[il], pjv, a.eps), a.drop_bits);
    }
}

}  // namespace

hipError_t launch_trace_update(hipStream_t stream, const Geometry& g, const TraceArgs& a) {
    dim3 grid((unsigned)((g.n_out + kTN - 1) / kTN), (unsigned)((g.n_in + kTM - 1) / kTM));
    trace_kernel<<<grid, kThreads, 0, stream>>>(g, a);
    return hipGetLastError();
}

}  // namespace bcpnn
