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
//  * T is a dense [N_in x N_out] product with K = B (the batch), on fp32 MFMA
//    (v_mfma_f32_32x32x2f32).  Every Pij is needed (silent connections are scored for
//    plasticity), so the contraction is dense.  A workgroup owns a 128 x 128 tile of Pij and
//    streams K through LDS in chunks of 32 batch rows; its four waves each hold a 64 x 64
//    accumulator (2 x 2 MFMA blocks).
//  * The epilogue reads each Pij once, writes it once, and writes w only on active blocks
//    (silent blocks of w stay zero), so the tile is the only HBM traffic of the step that
//    scales with N_in * N_out: 8 bytes per element plus 4 per active element.
//  * The batch means of the tile's rows and columns are summed from the staged LDS panels;
//    every workgroup computes the new Pi / Pj of its rows / columns itself (same code, same
//    order, hence identical values) and the tiles of the first column / row store them.  Pi and
//    Pj are therefore read from one buffer and written to another (the host alternates them),
//    so no workgroup can read a value already updated by another.
//
// MFMA f32 32x32x2 lane layout (verified on gfx950): A[i][k] from lane i + 32 k, B[k][j] from
// lane j + 32 k, lane l holds D[8 (r / 4) + 4 (l / 32) + r % 4][l % 32] in result register r.
#include "bcpnn_internal.h"
#include "device_common.h"

namespace bcpnn {
namespace {

typedef float f16v __attribute__((ext_vector_type(16)));

constexpr int kTM = 128;   // Pij rows (input units) per tile
constexpr int kTN = 128;   // Pij columns (hidden units) per tile
constexpr int kTK = 32;    // batch rows per staged chunk
constexpr int kThreads = 256;

__global__ void __launch_bounds__(kThreads)
trace_kernel(Geometry g, TraceArgs a) {
    __shared__ float As[kTK][kTM];
    __shared__ float Bs[kTK][kTN];
    __shared__ float pi_t[kTM];
    __shared__ float pj_t[kTN];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int64_t j0 = (int64_t)blockIdx.x * kTN;
    const int64_t i0 = (int64_t)blockIdx.y * kTM;

    f16v acc[2][2];
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[mi][ni][r] = 0.0f;

    float colsum = 0.0f;   // threads < 128: sum of x over the column i0 + tid; else t over j0 + tid - 128

    for (int k0 = 0; k0 < a.B; k0 += kTK) {
        __syncthreads();
        for (int e = tid; e < kTK * kTM; e += kThreads) {
            const int r = e / kTM, c = e % kTM;
            const int64_t k = k0 + r;
            const int64_t i = i0 + c, j = j0 + c;
            As[r][c] = (k < a.B && i < g.n_in) ? a.x[k * g.n_in + i] : 0.0f;
            Bs[r][c] = (k < a.B && j < g.n_out) ? a.t[k * g.n_out + j] : 0.0f;
        }
        __syncthreads();
        if (tid < kTM) {
            for (int r = 0; r < kTK; ++r) colsum += As[r][tid];
        } else {
            for (int r = 0; r < kTK; ++r) colsum += Bs[r][tid - kTM];
        }
#pragma unroll 4
        for (int kk = 0; kk < kTK; kk += 2) {
            float av[2], bv[2];
#pragma unroll
            for (int mi = 0; mi < 2; ++mi) av[mi] = As[kk + (lane >> 5)][wm * 64 + mi * 32 + (lane & 31)];
#pragma unroll
            for (int ni = 0; ni < 2; ++ni) bv[ni] = Bs[kk + (lane >> 5)][wn * 64 + ni * 32 + (lane & 31)];
#pragma unroll
            for (int mi = 0; mi < 2; ++mi)
#pragma unroll
                for (int ni = 0; ni < 2; ++ni)
                    acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[mi], bv[ni], acc[mi][ni], 0, 0, 0);
        }
    }

    // New marginal traces of this tile's rows and columns.
    if (tid < kTM) {
        const int64_t i = i0 + tid;
        if (i < g.n_in) {
            const float p = fmaf(a.a_eff, colsum * a.inv_b, a.c1 * a.pi_old[i]);
            pi_t[tid] = p;
            if (blockIdx.x == 0) a.pi_new[i] = p;
        }
    } else {
        const int64_t j = j0 + (tid - kTM);
        if (j < g.n_out) {
            const float p = fmaf(a.a_eff, colsum * a.inv_b, a.c1 * a.pj_old[j]);
            pj_t[tid - kTM] = p;
            if (blockIdx.y == 0) {
                a.pj_new[j] = p;
                a.b[j] = a.bias_gain * __logf(fmaxf(p, a.eps));
            }
        }
    }
    __syncthreads();

    // Epilogue: joint trace, then the masked log-ratio weight.
#pragma unroll
    for (int ni = 0; ni < 2; ++ni) {
        const int jl = wn * 64 + ni * 32 + (lane & 31);
        const int64_t j = j0 + jl;
        if (j >= g.n_out) continue;
        const int32_t hj = (int32_t)(j / g.out_mcu);
        const float pjv = pj_t[jl];
#pragma unroll
        for (int mi = 0; mi < 2; ++mi) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int il = wm * 64 + mi * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                const int64_t i = i0 + il;
                if (i >= g.n_in) continue;
                const int64_t idx = i * g.n_out + j;
                float p = fmaf(a.c2, acc[mi][ni][r], a.c1 * a.pij[idx]);
                p = round_storage(p, a.drop_bits);
                a.pij[idx] = p;
                if (a.mask[(i / g.in_mcu) * g.out_hcu + hj])
                    a.w[idx] = round_storage(log_ratio(p, pi_t[il], pjv, a.eps), a.drop_bits);
            }
        }
    }
}

}  // namespace

hipError_t launch_trace_update(hipStream_t stream, const Geometry& g, const TraceArgs& a) {
    dim3 grid((unsigned)((g.n_out + kTN - 1) / kTN), (unsigned)((g.n_in + kTM - 1) / kTM));
    trace_kernel<<<grid, kThreads, 0, stream>>>(g, a);
    return hipGetLastError();
}

}  // namespace bcpnn
