// Device helpers shared by the kernels of libbcpnn.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bcpnn {

// Round-to-nearest-even of an fp32 value to (23 - drop) mantissa bits, done on the bit
// pattern: add half of the dropped range minus one plus the lowest kept bit, then truncate.
// A carry out of the mantissa moves into the exponent (and to infinity past the largest
// finite value), as rounding requires.  NaN and infinity are returned unchanged.
__device__ __forceinline__ float round_storage(float v, int drop) {
    if (drop == 0) return v;
    uint32_t u = __float_as_uint(v);
    if ((u & 0x7f800000u) == 0x7f800000u) return v;
    const uint32_t lsb = (u >> drop) & 1u;
    u += ((1u << (drop - 1)) - 1u) + lsb;
    u &= ~((1u << drop) - 1u);
    return __uint_as_float(u);
}

// Weight of one connection, w = log(Pij / (Pi Pj)) with every probability clamped at eps.
__device__ __forceinline__ float log_ratio(float pij, float pi, float pj, float eps) {
    const float den = fmaxf(pi, eps) * fmaxf(pj, eps);
    return __logf(fmaxf(pij, eps) / den);
}

// Natural log through the hardware base-2 log (v_log_f32, about one ulp for normal inputs)
// times ln 2; callers pass normal floats only (every argument here is clamped to eps >= FLT_MIN).
__device__ __forceinline__ float fast_log(float x) {
    return __builtin_amdgcn_logf(x) * 0.6931471805599453f;
}

// Uniform draw in [0, 1) with 24 bits: the SplitMix64 output function (Steele, Lea, Flood,
// OOPSLA 2014) applied to state seed + (idx + 1) * golden-ratio increment.
__device__ __forceinline__ float splitmix_uniform(uint64_t seed, uint64_t idx) {
    uint64_t z = seed + (idx + 1ull) * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    z ^= z >> 31;
    return (float)(uint32_t)(z >> 40) * (1.0f / 16777216.0f);
}

// Workgroups of a 1-D grid are dealt to the 8 XCDs round-robin (id % 8).  This maps the id
// to a linear work index so that each XCD receives one contiguous range of work indices:
// neighbouring work items (which share operands) then share that XCD's L2.  It is a
// bijection of [0, total).
__device__ __forceinline__ int64_t xcd_linear_index(int64_t bid, int64_t total) {
    const int64_t q = total / 8, rem = total % 8;
    const int64_t xcd = bid % 8, slot = bid / 8;
    return xcd * q + (xcd < rem ? xcd : rem) + slot;
}

// Workgroup barrier that orders LDS only: the fences are limited to the local address space, so
// the barrier waits for this wave's LDS operations (lgkmcnt) but leaves its global loads and
// stores in flight (a plain __syncthreads also drains vmcnt).  For kernels whose waves exchange
// data through LDS alone.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Wave-wide reductions over data-parallel-primitive lane moves (no LDS round trips): partial
// results climb the lanes of each 16-lane row (shift right by 1, 2, 4, 8), then rows 0 / 2
// feed rows 1 / 3 (broadcast of lane 15) and rows 0-1 feed rows 2-3 (broadcast of lane 31);
// lane 63 ends with the total, which is then read back to every lane.  Lanes a move cannot
// fill keep the identity (`idle`).
template <int kCtrl, int kRowMask>
__device__ __forceinline__ float dpp_move(float v, float idle) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(
        __builtin_bit_cast(int, idle), __builtin_bit_cast(int, v), kCtrl, kRowMask, 0xf, false));
}

template <typename Op>
__device__ __forceinline__ float wave_reduce_dpp(float v, float idle, Op op) {
    v = op(v, dpp_move<0x111, 0xf>(v, idle));   // row_shr:1
    v = op(v, dpp_move<0x112, 0xf>(v, idle));   // row_shr:2
    v = op(v, dpp_move<0x114, 0xf>(v, idle));   // row_shr:4
    v = op(v, dpp_move<0x118, 0xf>(v, idle));   // row_shr:8
    v = op(v, dpp_move<0x142, 0xa>(v, idle));   // row_bcast:15 into rows 1 and 3
    v = op(v, dpp_move<0x143, 0xc>(v, idle));   // row_bcast:31 into rows 2 and 3
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}

__device__ __forceinline__ float wave_max_dpp(float v) {
    return wave_reduce_dpp(v, -INFINITY, [](float a, float b) { return fmaxf(a, b); });
}

__device__ __forceinline__ float wave_sum_dpp(float v) {
    return wave_reduce_dpp(v, 0.0f, [](float a, float b) { return a + b; });
}

template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

__device__ __forceinline__ float wave_max(float v) {
    for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
    return v;
}

}  // namespace bcpnn
