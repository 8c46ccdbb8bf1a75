// Whole-matrix sweeps over Pij / w: initial state, weight recompute, mask application.
//
// These are bandwidth-bound passes (one read and/or one write of 4 bytes per element).  Each
// workgroup takes one row i of the [N_in][N_out] matrices per iteration of a grid-stride loop
// over rows; within a row the lanes walk consecutive columns, so every wave touches
// contiguous 256-byte spans.  The mask row [out_hcu] of the row's input HCU is read through
// the cache.
#include "bcpnn_internal.h"
#include "device_common.h"

namespace bcpnn {
namespace {

constexpr int kSweepThreads = 256;

__global__ void __launch_bounds__(kSweepThreads)
init_state_kernel(Geometry g, const uint8_t* __restrict__ mask, float pij0, float noise,
                  uint64_t seed, int drop, float* __restrict__ pij, float* __restrict__ w) {
    const float p0 = round_storage(pij0, drop);
    for (int64_t i = blockIdx.x; i < g.n_in; i += gridDim.x) {
        const uint8_t* mrow = mask + (int64_t)(i / g.in_mcu) * g.out_hcu;
        float* prow = pij + i * g.n_out;
        float* wrow = w + i * g.n_out;
        for (int64_t j = threadIdx.x; j < g.n_out; j += kSweepThreads) {
            prow[j] = p0;
            float v = 0.0f;
            if (mrow[j / g.out_mcu]) {
                const float u = splitmix_uniform(seed, (uint64_t)(i * g.n_out + j));
                v = __fmul_rn(noise, 2.0f * u - 1.0f);   // 2u - 1 is exact in fp32
            }
            wrow[j] = round_storage(v, drop);
        }
    }
}

__global__ void __launch_bounds__(kSweepThreads)
recompute_weights_kernel(Geometry g, const uint8_t* __restrict__ mask,
                         const float* __restrict__ pi, const float* __restrict__ pj,
                         const float* __restrict__ pij, float eps, int drop,
                         float* __restrict__ w) {
    for (int64_t i = blockIdx.x; i < g.n_in; i += gridDim.x) {
        const uint8_t* mrow = mask + (int64_t)(i / g.in_mcu) * g.out_hcu;
        const float pii = pi[i];
        const float* prow = pij + i * g.n_out;
        float* wrow = w + i * g.n_out;
        for (int64_t j = threadIdx.x; j < g.n_out; j += kSweepThreads) {
            float v = 0.0f;
            if (mrow[j / g.out_mcu]) v = log_ratio(prow[j], pii, pj[j], eps);
            wrow[j] = round_storage(v, drop);
        }
    }
}

__global__ void __launch_bounds__(kSweepThreads)
bias_kernel(int64_t n_out, const float* __restrict__ pj, float eps, float bias_gain,
            float* __restrict__ b) {
    const int64_t j = (int64_t)blockIdx.x * kSweepThreads + threadIdx.x;
    if (j < n_out) b[j] = bias_gain * __logf(fmaxf(pj[j], eps));
}

__global__ void __launch_bounds__(kSweepThreads)
apply_mask_kernel(Geometry g, const uint8_t* __restrict__ mask, float* __restrict__ w) {
    for (int64_t i = blockIdx.x; i < g.n_in; i += gridDim.x) {
        const uint8_t* mrow = mask + (int64_t)(i / g.in_mcu) * g.out_hcu;
        float* wrow = w + i * g.n_out;
        for (int64_t j = threadIdx.x; j < g.n_out; j += kSweepThreads)
            if (!mrow[j / g.out_mcu]) wrow[j] = 0.0f;
    }
}

unsigned sweep_blocks(const Geometry& g) {
    const int64_t cap = 8192;
    return (unsigned)(g.n_in < cap ? g.n_in : cap);
}

}  // namespace

hipError_t launch_init_state(hipStream_t stream, const Geometry& g, const uint8_t* mask,
                             float pij0, float init_noise, uint64_t seed, int drop_bits,
                             float* pij, float* w) {
    init_state_kernel<<<sweep_blocks(g), kSweepThreads, 0, stream>>>(g, mask, pij0, init_noise,
                                                                      seed, drop_bits, pij, w);
    return hipGetLastError();
}

hipError_t launch_recompute_weights(hipStream_t stream, const Geometry& g, const uint8_t* mask,
                                    const float* pi, const float* pj, const float* pij,
                                    float eps, float bias_gain, int drop_bits, float* w,
                                    float* b) {
    recompute_weights_kernel<<<sweep_blocks(g), kSweepThreads, 0, stream>>>(
        g, mask, pi, pj, pij, eps, drop_bits, w);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_bias(stream, g, pj, eps, bias_gain, b);
}

hipError_t launch_bias(hipStream_t stream, const Geometry& g, const float* pj, float eps,
                       float bias_gain, float* b) {
    bias_kernel<<<(unsigned)((g.n_out + kSweepThreads - 1) / kSweepThreads), kSweepThreads, 0,
                  stream>>>(g.n_out, pj, eps, bias_gain, b);
    return hipGetLastError();
}

hipError_t launch_apply_mask(hipStream_t stream, const Geometry& g, const uint8_t* mask,
                             float* w) {
    apply_mask_kernel<<<sweep_blocks(g), kSweepThreads, 0, stream>>>(g, mask, w);
    return hipGetLastError();
}

}  // namespace bcpnn
