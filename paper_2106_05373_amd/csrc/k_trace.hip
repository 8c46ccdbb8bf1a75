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
//    plasticity), so the contraction is dense.  A workgroup owns a 64 x 64 tile of Pij; each
//    of its four waves one 32 x 32 block.  Small tiles give ~1200 workgroups for the
//    MNIST-shaped layer, so 256 CUs receive near-equal shares (with 128 x 128 tiles, 312
//    tiles leave a fifth of the CUs with twice the work of the rest).
//  * K is streamed through LDS in chunks of 32 batch rows; the next chunk is loaded into
//    registers while the current one feeds the matrix cores.  Two accumulators alternate
//    over k so consecutive MFMAs are independent.
//  * The epilogue first loads every Pij of the lane and the mask bits (from an LDS copy of the
//    tile's mask block), then computes and stores: no load waits behind a store.  Each Pij is
//    read once and written once; w is written only on active blocks (silent blocks of w stay
//    zero), so the HBM traffic of the step that scales with N_in * N_out is 8 bytes per
//    element plus 4 per active element.
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

constexpr int kTM = 64;    // Pij rows (input units) per tile
constexpr int kTN = 64;    // Pij columns (hidden units) per tile
constexpr int kTK = 32;    // batch rows per staged chunk
constexpr int kThreads = 256;
constexpr int kLoads = kTK * kTM / kThreads;   // elements of each operand per thread per chunk

__global__ void __launch_bounds__(kThreads)
trace_kernel(Geometry g, TraceArgs a) {
    __shared__ float As[kTK][kTM];
    __shared__ float Bs[kTK][kTN];
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
    const float* __restrict__ x = a.x;
    const float* __restrict__ t = a.t;

    // Mask block of the tile, indexed by (row's input HCU - first, column's hidden HCU - first).
    const int64_t hi0 = i0 / g.in_mcu;
    const int64_t hj0 = j0 / g.out_mcu;
    const int64_t i_last = (i0 + kTM < g.n_in ? i0 + kTM : g.n_in) - 1;
    const int64_t j_last = (j0 + kTN < g.n_out ? j0 + kTN : g.n_out) - 1;
    const int nhi = (int)(i_last / g.in_mcu - hi0 + 1);
    const int nhj = (int)(j_last / g.out_mcu - hj0 + 1);
    if (tid < kTM) row_h[tid] = (int32_t)((i0 + tid) / g.in_mcu - hi0);
    else if (tid < kTM + kTN) col_h[tid - kTM] = (int32_t)((j0 + tid - kTM) / g.out_mcu - hj0);
    for (int e = tid; e < nhi * nhj; e += kThreads)
        mtile[e] = a.mask[(hi0 + e / nhj) * g.out_hcu + hj0 + e % nhj];

    // Chunk loads: element q of this thread is row (q * kThreads + tid) / 64, column tid % 64.
    const int col = tid % kTM;
    const int64_t ia = i0 + col, jb = j0 + col;
    float ra[kLoads], rb[kLoads];
    auto load_chunk = [&](int k0) {
#pragma unroll
        for (int q = 0; q < kLoads; ++q) {
            const int64_t k = k0 + (q * kThreads + tid) / kTM;
            ra[q] = (k < a.B && ia < g.n_in) ? x[k * g.n_in + ia] : 0.0f;
            rb[q] = (k < a.B && jb < g.n_out) ? t[k * g.n_out + jb] : 0.0f;
        }
    };

    f16v acc0, acc1;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc0[r] = acc1[r] = 0.0f;
    float colsum = 0.0f;   // tid < 64: sum of x over column i0 + tid; 64..127: t over j0 + tid - 64

    load_chunk(0);
    for (int k0 = 0; k0 < a.B; k0 += kTK) {
        __syncthreads();   // the previous chunk has been consumed
#pragma unroll
        for (int q = 0; q < kLoads; ++q) {
            const int r = (q * kThreads + tid) / kTM;
            As[r][col] = ra[q];
            Bs[r][col] = rb[q];
        }
        __syncthreads();
        if (k0 + kTK < a.B) load_chunk(k0 + kTK);   // in flight during the MFMAs below
        if (tid < kTM) {
            for (int r = 0; r < kTK; ++r) colsum += As[r][tid];
        } else if (tid < kTM + kTN) {
            for (int r = 0; r < kTK; ++r) colsum += Bs[r][tid - kTM];
        }
#pragma unroll
        for (int kk = 0; kk < kTK; kk += 4) {
            const float a0 = As[kk + (lane >> 5)][wm * 32 + (lane & 31)];
            const float b0 = Bs[kk + (lane >> 5)][wn * 32 + (lane & 31)];
            const float a1 = As[kk + 2 + (lane >> 5)][wm * 32 + (lane & 31)];
            const float b1 = Bs[kk + 2 + (lane >> 5)][wn * 32 + (lane & 31)];
            acc0 = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b0, acc0, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b1, acc1, 0, 0, 0);
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
    } else if (tid < kTM + kTN) {
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

    // Epilogue.  Phase 1: every load of the lane; phase 2: compute and store.
    const int jl = wn * 32 + (lane & 31);
    const int64_t j = j0 + jl;
    const bool jok = j < g.n_out;
    float pold[16];
    bool act[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int il = wm * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        const int64_t i = i0 + il;
        const bool ok = jok && i < g.n_in;
        pold[r] = ok ? a.pij[i * g.n_out + j] : 0.0f;
        act[r] = ok && mtile[row_h[il] * nhj + col_h[jl]];
    }
    const float pjv = jok ? pj_t[jl] : 1.0f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int il = wm * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        const int64_t i = i0 + il;
        if (!jok || i >= g.n_in) continue;
        const int64_t idx = i * g.n_out + j;
        float p = fmaf(a.c2, acc0[r] + acc1[r], a.c1 * pold[r]);
        p = round_storage(p, a.drop_bits);
        a.pij[idx] = p;
        if (act[r]) a.w[idx] = round_storage(log_ratio(p, pi_t[il], pjv, a.eps), a.drop_bits);
    }
}

}  // namespace

hipError_t launch_trace_update(hipStream_t stream, const Geometry& g, const TraceArgs& a) {
    dim3 grid((unsigned)((g.n_out + kTN - 1) / kTN), (unsigned)((g.n_in + kTM - 1) / kTM));
    trace_kernel<<<grid, kThreads, 0, stream>>>(g, a);
    return hipGetLastError();
}

}  // namespace bcpnn
