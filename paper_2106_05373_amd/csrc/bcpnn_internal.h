// Internal declarations shared by the HIP translation units of libbcpnn (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bcpnn.h"

namespace bcpnn {

// Device-side description of the layer geometry and learning constants.
struct Geometry {
    int32_t in_hcu, in_mcu, out_hcu, out_mcu;
    int64_t n_in, n_out;
};

// Storage rounding of Pij and W (bcpnn_storage): number of fp32 mantissa bits dropped.
inline int storage_drop_bits(int32_t storage) {
    return storage == BCPNN_STORE_BF16 ? 16 : (storage == BCPNN_STORE_M10 ? 13 : 0);
}

// ---- launchers (each enqueues on `stream` and returns hipGetLastError()) ----

// Launches kernel<<<grid, block, lds, stream>>>(args...), with start / stop (each nullable)
// recorded on the stream right before and after it: the elapsed time between them is the
// kernel's, with the event records' own short passage through the stream.
template <typename... Params, typename... Args>
hipError_t launch_timed(void (*kernel)(Params...), dim3 grid, dim3 block, size_t lds,
                        hipStream_t stream, hipEvent_t start, hipEvent_t stop, Args&&... args) {
    if (start) {
        const hipError_t e = hipEventRecord(start, stream);
        if (e != hipSuccess) return e;
    }
    kernel<<<grid, block, lds, stream>>>(static_cast<Args&&>(args)...);
    hipError_t e = hipGetLastError();
    if (e == hipSuccess && stop) e = hipEventRecord(stop, stream);
    return e;
}

// Launch-duration stamps (profiling of the short kernels of the caller's stream), on the
// device's constant-rate clock (s_memrealtime): a launch's stamp holds kStampLanes start words
// and as many end words; workgroup b takes the 64-bit atomic min of its start into start word
// b % kStampLanes and the max of its end into end word b % kStampLanes (spread over many words,
// so that the atomics of a large grid do not queue on one address).  The host initialises the
// starts to the largest value and the ends to 0; the launch's span is the least start to the
// greatest end.  A kernel stamps in a variant of its own (kOn): even a test of a null pointer
// at both ends slows the short kernels measurably.  The end waits for the workgroup's memory
// operations and all its waves; call it where every thread of the workgroup arrives.
constexpr int kStampLanes = 64;
template <bool kOn>
__device__ __forceinline__ void stamp_start(unsigned long long* stamp) {
    if constexpr (kOn) {
        if (threadIdx.x == 0)
            atomicMin(stamp + blockIdx.x % kStampLanes,
                      (unsigned long long)__builtin_amdgcn_s_memrealtime());
    }
}
template <bool kOn>
__device__ __forceinline__ void stamp_end(unsigned long long* stamp) {
    if constexpr (kOn) {
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        if (threadIdx.x == 0)
            atomicMax(stamp + kStampLanes + blockIdx.x % kStampLanes,
                      (unsigned long long)__builtin_amdgcn_s_memrealtime());
    }
}

// Initial state: Pij = pij0, w = mask ? noise * (2u - 1) : 0 with u from SplitMix64.
hipError_t launch_init_state(hipStream_t stream, const Geometry& g, const uint8_t* mask,
                             float pij0, float init_noise, uint64_t seed, int drop_bits,
                             float* pij, float* w);

// b = bias_gain * log(max(pj, eps)).
hipError_t launch_bias(hipStream_t stream, const Geometry& g, const float* pj, float eps,
                       float bias_gain, float* b);

// w = mask ? log(max(pij,eps) / (max(pi,eps) max(pj,eps))) : 0 over the whole matrix, and
// b = bias_gain * log(max(pj, eps)).
hipError_t launch_recompute_weights(hipStream_t stream, const Geometry& g, const uint8_t* mask,
                                    const float* pi, const float* pj, const float* pij,
                                    float eps, float bias_gain, int drop_bits, float* w,
                                    float* b, hipEvent_t start = nullptr,
                                    hipEvent_t stop = nullptr);

// Zeroes the silent blocks of w (used after a host upload of w).
hipError_t launch_apply_mask(hipStream_t stream, const Geometry& g, const uint8_t* mask,
                             float* w);

// Support over the active input HCUs (fp64 MFMA) followed by, per (sample, hidden HCU):
//   mode 0: softmax with gain -> y if non-null (and s if non-null);
//   mode 1: argmax -> winner (and s if non-null).
// max_active is the largest number of active input HCUs of any hidden HCU (swaps keep it).
// With ops non-null (training), the kernel also writes the contraction operands: the split
// x^T from x, the split t^T from target (or from y when target is null), and the column sums.
// The contraction operands are stored in MFMA fragment order: per block of 32 units and k-step of
// 16 batch rows, 64 lanes x 8 bf16 (1 KiB), lane l holding rows 8 (l / 32) .. + 7 of unit
// l % 32 -- exactly the A / B operand of v_mfma_f32_32x32x16_bf16, so a wave loads one step of
// one operand as a single contiguous 1 KiB read.  Units past the layer stay zero.
// With complement pairs (every input HCU holds x and 1 - x), x^T holds the first unit of each
// input HCU only, indexed by the HCU: [ceil(in_hcu / 32)][n_ks][64][8]; x_sum still has every
// unit.
struct TraceOperands {
    uint16_t* x_hi;   // [ceil(n_in / 32)][n_ks][64][8] bf16 bits
    uint16_t* x_lo;
    uint16_t* t_hi;   // [ceil(n_out / 32)][n_ks][64][8]
    uint16_t* t_lo;
    float* x_sum;     // [ceil(B / 16)][n_in]
    float* t_sum;     // [ceil(B / 16)][n_out]
    int32_t n_ks;     // k-steps per unit block: ceil(max_batch / 16)
    int32_t paired;   // PairMode: with complement pairs, x^T over input HCUs (see above)
    // With complement pairs: set to 1 by the support kernel when a pair of the batch input is
    // not (x, 1 - x) (|x_2p + x_2p+1 - 1| > kPairTolerance, or NaN); never cleared on the device.
    int32_t* pair_error;
};

constexpr float kPairTolerance = 1e-6f;

// How the trace kernels treat the input units.  kPairsSplit is kPairs for a small layer: the
// active-block kernel then runs each contraction twice, in two waves that store the first and
// the second rows of the pairs (see trace_active_pair_kernel).
enum PairMode { kUnpaired = 0, kPairs = 1, kPairsSplit = 2 };

// Element offset (bf16 units) of the fragment chunk that holds batch rows 8 h .. 8 h + 7 of unit
// u in k-step ks (16 bytes, 8 consecutive rows).
__host__ __device__ inline int64_t frag_chunk(int64_t u, int64_t ks, int h, int32_t n_ks) {
    return (((u >> 5) * n_ks + ks) * 64 + (u & 31) + 32 * h) * 8;
}

hipError_t launch_support(hipStream_t stream, const Geometry& g, const float* x, int32_t B,
                          const float* w, const float* bias, const int32_t* act_list,
                          const int32_t* act_count, int32_t max_active, float gain, int mode,
                          float* y, float* s, int32_t* winner, const float* target,
                          const TraceOperands* ops, hipEvent_t start = nullptr,
                          hipEvent_t stop = nullptr, unsigned long long* stamp = nullptr);

// Largest number of active input units (active HCUs * in_mcu) of one hidden HCU that the
// support kernel keeps in its LDS unit table.
constexpr int32_t kMaxActiveUnits = 12288;

// Joint-trace contraction with the trace, weight and bias updates, in two kernels that touch
// disjoint elements of Pij:
//   Pij <- c1 Pij + c2 sum_b x[b,i] t[b,j];  Pi, Pj from the batch means (read *_old, write
//   *_new); w on active blocks; b = bias_gain log(max(Pj_new, eps)).  The batch enters as the
//   split operands and column sums written by the support kernel.  With complement pairs the
//   contraction covers the first unit 2p of each input HCU, and the second takes
//   sum_b x[b,2p+1] t[b,j] = sum_b t[b,j] - sum_b x[b,2p] t[b,j].
struct TraceArgs {
    TraceOperands ops;
    int32_t B;
    float c1, a_eff, inv_b, c2;
    const float* pi_old;
    const float* pj_old;
    float* pi_new;
    float* pj_new;
    float* pij;
    float* w;
    float* b;
    const uint8_t* mask;
    float eps, bias_gain;
    int drop_bits;
    unsigned long long* stamp;   // launch-duration stamp (stamp_start / stamp_end), or null
};
// The elements of active blocks (the rows of each hidden HCU's active input units), their
// weights, and Pi, Pj, b of every unit.  max_active as for launch_support.
hipError_t launch_trace_active(hipStream_t stream, const Geometry& g, const TraceArgs& a,
                               const int32_t* act_list, const int32_t* act_count,
                               int32_t max_active, hipEvent_t start = nullptr,
                               hipEvent_t stop = nullptr);
// Workgroups of that launch (for the launch-size check); paired is a PairMode.
int64_t trace_active_workgroups(const Geometry& g, int32_t max_active, int paired);
// The elements of silent blocks over several consecutive batches: each element is read once,
// takes the batches' updates Pij <- c1 Pij + c2 T in order (rounded to the storage format after
// each, exactly as per-batch updates), and is written once.  Reads the mask; Pi, Pj, w and b
// are untouched.  start / stop (nullable) are recorded on the stream around the launch.
constexpr int kMaxSweepBatches = 8;
struct SweepBatch {
    const uint16_t* x_hi;
    const uint16_t* x_lo;
    const uint16_t* t_hi;
    const uint16_t* t_lo;
    const float* t_sum;   // column sums of t per 16-row tile (read with complement pairs)
    int32_t nk;       // k-steps of this batch: ceil(B / 16)
    float c1, c2;     // 1 - a_eff and a_eff / B
};
struct SweepArgs {
    SweepBatch bt[kMaxSweepBatches];
    int32_t n_batches;
    int32_t n_ks;     // k-steps per unit block of the operand arrays
    int32_t paired;   // PairMode (the sweep treats kPairs and kPairsSplit alike)
    float* pij;
    const uint8_t* mask;
    int drop_bits;
};
// resident_wgs > 0 caps the grid at that many workgroups (rounded up to a multiple of 8), each
// looping over the 32 x 128 block groups; 0 launches one workgroup per group; < 0 selects the
// 128 x 128 LDS-staged tiles of a large layer.
hipError_t launch_trace_sweep(hipStream_t stream, const Geometry& g, const SweepArgs& a,
                              int64_t resident_wgs, hipEvent_t start = nullptr,
                              hipEvent_t stop = nullptr);

// Mutual information of every (input HCU, hidden HCU) block, fp64, [in_hcu][out_hcu].
// start (nullable) is recorded on the stream right before the launch.
hipError_t launch_mutual_information(hipStream_t stream, const Geometry& g, const float* pi,
                                     const float* pj, const float* pij, float eps, double* mi,
                                     hipEvent_t start = nullptr);

// Greedy swap per hidden HCU, patch of the swapped blocks of w, rebuild of the active lists.
// stop (nullable) is recorded on the stream right after the launch.
hipError_t launch_plasticity_swap(hipStream_t stream, const Geometry& g, const double* mi,
                                  int32_t n_swaps, const float* pi, const float* pj,
                                  const float* pij, float eps, int drop_bits, uint8_t* mask,
                                  float* w, int32_t* act_list, int32_t* act_count,
                                  int32_t* swap_count, hipEvent_t stop = nullptr);

// total[0] = counts[0] + ... + counts[n - 1] (one workgroup; 0 for n = 0).
hipError_t launch_count_sum(hipStream_t stream, const int32_t* counts, int32_t n,
                            int32_t* total);

}  // namespace bcpnn
