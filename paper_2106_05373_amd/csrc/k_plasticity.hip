// Structural plasticity (Alg. 1 "update plasticity mask"; Sec. 2): score every
// (input HCU, hidden HCU) connection by the mutual information of its block of the joint trace,
// then let every hidden HCU swap its weakest active connection for its strongest silent one.
//
//   MI[hi][hj] = sum_{i in hi} sum_{j in hj} Pij log(Pij / (Pi Pj))   (0 log 0 = 0), in fp64
//
// Scores are fp64 so that the selection below, an exact comparison of scores, matches a host
// computation of the same definition: different summation orders move an fp64 score by about
// 1e-16 relative, far below the gaps between distinct scores.  Blocks holding identical data
// (e.g. inputs that never change) get bit-identical scores because every block is reduced by
// the same lane pattern wherever it sits, and such ties go to the lowest HCU index.
#include <climits>

#include "bcpnn_internal.h"
#include "device_common.h"
#include "fp64_log.h"

namespace bcpnn {
namespace {

constexpr int kThreads = 256;
constexpr int kMaxSwaps = 256;

// kGroup lanes per block, 64 / kGroup blocks per wave (consecutive blocks: neighbouring hidden
// HCUs of one input HCU, i.e. neighbouring column spans of the same Pij rows).  Lane k of a
// group sums the block's columns k, k + kGroup, ..., kColChunk columns at a time (their loads
// issued together), each chunk row by row; an xor butterfly over the group then adds the
// partial sums, leaving the same bits in every lane of the group.  The pattern depends only on
// positions inside the block.  Few lanes per block keep the lanes busy with fp64 log terms
// (M_out = 100: 13 columns per lane for 8 lanes) rather than with per-block reductions; the log
// is log_positive (fp64_log.h), a third of the instructions of the general library log.
constexpr int kGroup = 8;
constexpr int kColChunk = 4;

__global__ void __launch_bounds__(kThreads)
mi_kernel(Geometry g, const float* __restrict__ pi, const float* __restrict__ pj,
          const float* __restrict__ pij, float eps, double* __restrict__ mi) {
    const int lane = threadIdx.x & 63;
    const int sub = lane % kGroup;
    const int64_t n_blk = (int64_t)g.in_hcu * g.out_hcu;
    const int64_t blk = ((int64_t)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6)) *
                            (64 / kGroup) + lane / kGroup;
    if (((int64_t)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6)) * (64 / kGroup) >= n_blk)
        return;                                                   // whole wave
    const bool live = blk < n_blk;
    const int64_t b = live ? blk : n_blk - 1;                     // clamped lanes still reduce
    const int64_t hi = b / g.out_hcu;
    const int64_t hj = b - hi * g.out_hcu;
    const double e = (double)eps;
    double part = 0.0;
    for (int c0 = sub; c0 < g.out_mcu; c0 += kGroup * kColChunk) {
        double pjc[kColChunk];
#pragma unroll
        for (int k = 0; k < kColChunk; ++k) {
            const int c = c0 + k * kGroup;
            pjc[k] = c < g.out_mcu ? fmax((double)pj[hj * g.out_mcu + c], e) : 1.0;
        }
        for (int m = 0; m < g.in_mcu; ++m) {
            const int64_t i = hi * g.in_mcu + m;
            const double pim = fmax((double)pi[i], e);
            float q[kColChunk];
#pragma unroll
            for (int k = 0; k < kColChunk; ++k) {
                const int c = c0 + k * kGroup;
                q[k] = c < g.out_mcu ? pij[i * g.n_out + hj * g.out_mcu + c] : 0.0f;
            }
#pragma unroll
            for (int k = 0; k < kColChunk; ++k) {
                if (q[k] != 0.0f) {
                    const double den = pim * pjc[k];
                    part += (double)q[k] * log_positive(fmax((double)q[k], e) / den);
                }
            }
        }
    }
#pragma unroll
    for (int off = kGroup / 2; off > 0; off >>= 1) part += __shfl_xor(part, off, 64);
    if (live && sub == 0) mi[blk] = part;
}

struct Pick {
    double v;
    int32_t i;
};

// Lowest score first, ties to the lowest index.
__device__ __forceinline__ bool better_low(double v, int32_t i, const Pick& p) {
    return v < p.v || (v == p.v && i < p.i);
}
// Highest score first, ties to the lowest index.
__device__ __forceinline__ bool better_high(double v, int32_t i, const Pick& p) {
    return v > p.v || (v == p.v && i < p.i);
}

// One workgroup per hidden HCU.  The HCU's mask column lives in LDS while it is edited:
// 1 = active, 0 = silent, 2 = silenced now, 3 = activated now (2 and 3 are excluded from the
// later swaps of this update).
__global__ void __launch_bounds__(kThreads)
swap_kernel(Geometry g, const double* __restrict__ mi, int32_t n_swaps,
            const float* __restrict__ pi, const float* __restrict__ pj,
            const float* __restrict__ pij, float eps, int drop, uint8_t* __restrict__ mask,
            float* __restrict__ w, int32_t* __restrict__ act_list,
            int32_t* __restrict__ act_count, int32_t* __restrict__ swap_count) {
    extern __shared__ uint8_t mcol[];                 // [in_hcu]
    __shared__ Pick red_lo[kThreads / 64], red_hi[kThreads / 64];
    __shared__ int32_t sw_a[kMaxSwaps], sw_s[kMaxSwaps];
    __shared__ int32_t n_done, stop;
    __shared__ int32_t scan[kThreads];

    const int hj = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int32_t hin = g.in_hcu;

    for (int32_t h = tid; h < hin; h += kThreads) mcol[h] = mask[(int64_t)h * g.out_hcu + hj];
    if (tid == 0) n_done = 0;
    __syncthreads();

    for (int32_t t = 0; t < n_swaps; ++t) {
        Pick lo{INFINITY, INT_MAX}, hi{-INFINITY, INT_MAX};
        for (int32_t h = tid; h < hin; h += kThreads) {
            const uint8_t m = mcol[h];
            const double v = mi[(int64_t)h * g.out_hcu + hj];
            if (m == 1 && better_low(v, h, lo)) lo = Pick{v, h};
            if (m == 0 && better_high(v, h, hi)) hi = Pick{v, h};
        }
        for (int off = 32; off > 0; off >>= 1) {
            const double lv = __shfl_xor(lo.v, off, 64);
            const int32_t li = __shfl_xor(lo.i, off, 64);
            if (better_low(lv, li, lo)) lo = Pick{lv, li};
            const double hv = __shfl_xor(hi.v, off, 64);
            const int32_t hix = __shfl_xor(hi.i, off, 64);
            if (better_high(hv, hix, hi)) hi = Pick{hv, hix};
        }
        if (lane == 0) {
            red_lo[wave] = lo;
            red_hi[wave] = hi;
        }
        __syncthreads();
        if (tid == 0) {
            Pick L = red_lo[0], H = red_hi[0];
            for (int q = 1; q < kThreads / 64; ++q) {
                if (better_low(red_lo[q].v, red_lo[q].i, L)) L = red_lo[q];
                if (better_high(red_hi[q].v, red_hi[q].i, H)) H = red_hi[q];
            }
            stop = 1;
            if (L.i != INT_MAX && H.i != INT_MAX && H.v > L.v) {
                mcol[L.i] = 2;
                mcol[H.i] = 3;
                sw_a[n_done] = L.i;
                sw_s[n_done] = H.i;
                ++n_done;
                stop = 0;
            }
        }
        __syncthreads();
        if (stop) break;
    }

    const int32_t done = n_done;
    for (int32_t q = tid; q < done; q += kThreads) {
        mcol[sw_a[q]] = 0;
        mcol[sw_s[q]] = 1;
        mask[(int64_t)sw_a[q] * g.out_hcu + hj] = 0;
        mask[(int64_t)sw_s[q] * g.out_hcu + hj] = 1;
    }

    // Rewrite the changed blocks of w: 0 where silenced, the log-ratio weight where activated.
    const int32_t blk_elems = g.in_mcu * g.out_mcu;
    for (int32_t q = 0; q < done; ++q) {
        for (int side = 0; side < 2; ++side) {
            const int64_t h = side ? sw_s[q] : sw_a[q];
            for (int32_t e = tid; e < blk_elems; e += kThreads) {
                const int64_t i = h * g.in_mcu + e / g.out_mcu;
                const int64_t j = (int64_t)hj * g.out_mcu + e % g.out_mcu;
                const int64_t idx = i * g.n_out + j;
                w[idx] = side ? round_storage(log_ratio(pij[idx], pi[i], pj[j], eps), drop) : 0.0f;
            }
        }
    }
    __syncthreads();

    // Rebuild the ascending list of active input HCUs: each thread counts a contiguous range,
    // an exclusive scan over the threads gives the output offsets.
    const int32_t per = (hin + kThreads - 1) / kThreads;
    const int32_t lo_h = tid * per;
    const int32_t hi_h = lo_h + per < hin ? lo_h + per : hin;
    int32_t cnt = 0;
    for (int32_t h = lo_h; h < hi_h; ++h) cnt += mcol[h] == 1;
    scan[tid] = cnt;
    __syncthreads();
    if (tid == 0) {
        int32_t run = 0;
        for (int q = 0; q < kThreads; ++q) {
            const int32_t c = scan[q];
            scan[q] = run;
            run += c;
        }
        act_count[hj] = run;
        swap_count[hj] = done;
    }
    __syncthreads();
    int32_t pos = scan[tid];
    int32_t* list = act_list + (int64_t)hj * hin;
    for (int32_t h = lo_h; h < hi_h; ++h)
        if (mcol[h] == 1) list[pos++] = h;
}

// total[0] = sum of counts[0 .. n) (0 for n = 0), in one workgroup, in a fixed order.
__global__ void __launch_bounds__(kThreads)
count_sum_kernel(const int32_t* __restrict__ counts, int32_t n, int32_t* __restrict__ total) {
    __shared__ int32_t part[kThreads / 64];
    int32_t v = 0;
    for (int32_t k = threadIdx.x; k < n; k += kThreads) v += counts[k];
    v = wave_sum(v);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = v;
    __syncthreads();
    if (threadIdx.x == 0) {
        int32_t t = 0;
        for (int q = 0; q < kThreads / 64; ++q) t += part[q];
        total[0] = t;
    }
}

}  // namespace

hipError_t launch_count_sum(hipStream_t stream, const int32_t* counts, int32_t n,
                            int32_t* total) {
    count_sum_kernel<<<1, kThreads, 0, stream>>>(counts, n, total);
    return hipGetLastError();
}

hipError_t launch_mutual_information(hipStream_t stream, const Geometry& g, const float* pi,
                                     const float* pj, const float* pij, float eps, double* mi,
                                     hipEvent_t start) {
    const int64_t per_wg = (int64_t)(kThreads / 64) * (64 / kGroup);
    const int64_t blocks = ((int64_t)g.in_hcu * g.out_hcu + per_wg - 1) / per_wg;
    return launch_timed(mi_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, stream, start,
                        nullptr, g, pi, pj, pij, eps, mi);
}

hipError_t launch_plasticity_swap(hipStream_t stream, const Geometry& g, const double* mi,
                                  int32_t n_swaps, const float* pi, const float* pj,
                                  const float* pij, float eps, int drop_bits, uint8_t* mask,
                                  float* w, int32_t* act_list, int32_t* act_count,
                                  int32_t* swap_count, hipEvent_t stop) {
    if (n_swaps > kMaxSwaps) return hipErrorInvalidValue;
    return launch_timed(swap_kernel, dim3((unsigned)g.out_hcu), dim3(kThreads),
                        (size_t)g.in_hcu, stream, nullptr, stop, g, mi, n_swaps, pi, pj,
                        pij, eps, drop_bits, mask, w, act_list, act_count, swap_count);
}

}  // namespace bcpnn
