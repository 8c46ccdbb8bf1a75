// Whole-matrix sweeps over Pij / w: initial state, weight recompute, mask application.
//
// These are bandwidth-bound passes (one read and/or one write of 4 bytes per element).  Each
// workgroup takes one row i of the [N_in][N_out] matrices per iteration of a grid-stride loop
// over rows; within a row the lanes walk consecutive columns, so every wave touches
// contiguous spans.  The mask row [out_hcu] of the row's input HCU is read through the cache.
//
// The weight recompute (Alg. 1 weight and mask lines) writes every w but reads Pij only where
// the mask is set: a silent weight is 0 whatever its trace.  When N_out is a multiple of 4
// (16-byte rows) each lane moves 16 bytes per access, eight accesses in flight, finds a column's
// hidden HCU by a multiply-high instead of a division, and stores w with the non-temporal hint.
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

constexpr int kWeightUnroll = 8;    // 16-byte accesses per lane in flight

typedef float f32x4 __attribute__((ext_vector_type(4)));

// Streaming store: w is not read again by this pass, so it need not stay in the caches.
__device__ __forceinline__ void store_streaming(float4* p, float4 v) {
    const f32x4 x = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(x, reinterpret_cast<f32x4*>(p));
}

// Hidden HCU of column j: floor(j / out_mcu) as the high word of j * ceil(2^32 / out_mcu),
// exact for out_mcu >= 2 while j * out_mcu < 2^32 (both checked by the launcher).
__device__ __forceinline__ uint32_t column_hcu(uint32_t j, uint32_t magic) {
    return __umulhi(j, magic);
}

__device__ __forceinline__ float weight_of(bool live, float pij, float pi, float pj, float eps,
                                           int drop) {
    return live ? round_storage(log_ratio(pij, pi, pj, eps), drop) : 0.0f;
}

__global__ void __launch_bounds__(kSweepThreads)
recompute_weights_vec_kernel(Geometry g, const uint8_t* __restrict__ mask,
                             const float* __restrict__ pi, const float* __restrict__ pj,
                             const float* __restrict__ pij, float eps, int drop, uint32_t magic,
                             float* __restrict__ w) {
    const uint32_t n4 = (uint32_t)(g.n_out >> 2);
    const float4* pj4 = reinterpret_cast<const float4*>(pj);
    for (int64_t i = blockIdx.x; i < g.n_in; i += gridDim.x) {
        const uint8_t* mrow = mask + (int64_t)(i / g.in_mcu) * g.out_hcu;
        const float pii = pi[i];
        const float4* prow = reinterpret_cast<const float4*>(pij + i * g.n_out);
        float4* wrow = reinterpret_cast<float4*>(w + i * g.n_out);
        for (uint32_t q0 = threadIdx.x; q0 < n4; q0 += kSweepThreads * kWeightUnroll) {
            float4 p[kWeightUnroll], pq[kWeightUnroll];
            uint32_t live[kWeightUnroll];     // bit e: column 4q + e is in an active block
#pragma unroll
            for (int u = 0; u < kWeightUnroll; ++u) {
                const uint32_t q = q0 + u * kSweepThreads;
                live[u] = 0;
                p[u] = pq[u] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
                if (q < n4) {
                    const uint32_t j = 4 * q;
                    const uint32_t h0 = column_hcu(j, magic), h3 = column_hcu(j + 3, magic);
                    const uint32_t m0 = mrow[h0] != 0, m3 = mrow[h3] != 0;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const uint32_t h = column_hcu(j + e, magic);
                        const uint32_t m = h == h0 ? m0 : h == h3 ? m3 : (mrow[h] != 0);
                        live[u] |= m << e;
                    }
                    if (live[u]) {
                        p[u] = prow[q];
                        pq[u] = pj4[q];
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < kWeightUnroll; ++u) {
                const uint32_t q = q0 + u * kSweepThreads;
                if (q >= n4) continue;
                float4 v;
                v.x = weight_of(live[u] & 1u, p[u].x, pii, pq[u].x, eps, drop);
                v.y = weight_of(live[u] & 2u, p[u].y, pii, pq[u].y, eps, drop);
                v.z = weight_of(live[u] & 4u, p[u].z, pii, pq[u].z, eps, drop);
                v.w = weight_of(live[u] & 8u, p[u].w, pii, pq[u].w, eps, drop);
                store_streaming(&wrow[q], v);
            }
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
                                    float* b, hipEvent_t start, hipEvent_t stop) {
    // 16-byte rows and an exact multiply-high HCU lookup (out_mcu >= 2, so that the multiplier
    // fits 32 bits): the vector kernel; else the scalar one
    hipError_t e;
    if (g.n_out % 4 == 0 && g.out_mcu >= 2 &&
        (uint64_t)g.n_out * (uint64_t)g.out_mcu < (1ull << 32)) {
        const uint32_t magic =
            (uint32_t)(((1ull << 32) + (uint64_t)g.out_mcu - 1) / (uint64_t)g.out_mcu);
        // one row per workgroup: short-lived workgroups keep the stores streaming (a
        // grid-stride loop over rows with fewer workgroups writes at about 5.5 against 6.3 TB/s)
        const int64_t rows = g.n_in < (int64_t)1 << 30 ? g.n_in : (int64_t)1 << 30;
        e = launch_timed(recompute_weights_vec_kernel, dim3((unsigned)rows),
                         dim3(kSweepThreads), 0, stream, start, stop, g, mask, pi, pj,
                         pij, eps, drop_bits, magic, w);
    } else {
        e = launch_timed(recompute_weights_kernel, dim3(sweep_blocks(g)),
                         dim3(kSweepThreads), 0, stream, start, stop, g, mask, pi, pj,
                         pij, eps, drop_bits, w);
    }
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
