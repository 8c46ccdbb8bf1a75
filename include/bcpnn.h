/*
 * bcpnn.h -- C ABI of the BCPNN hidden-layer training library for AMD MI355X (gfx950).
 *
 * The library implements one layer of the Bayesian Confidence Propagation Neural Network as
 * trained by StreamBrain (Podobas et al., HEART 2021, Sec. 2, Algorithm 1):
 *
 *   support      s_j  = b_j + sum_i a_i w_ij          (w already masked)      Alg. 1, support line
 *   activation   a_j  = softmax over the hidden HCU of g * s_j                 Alg. 1; Sec. 2
 *   traces       C_i  <- (1-l) C_i  + l <a_i>                                 Alg. 1, cycle loop
 *                C_j  <- (1-l) C_j  + l <a_j>
 *                C_ij <- (1-l) C_ij + l <a_i a_j>   (<.> = mean over the batch)
 *   weights      w_ij = log(C_ij / (C_i C_j)),  b_j = k_B log C_j,  w *= mask   Alg. 1
 *   plasticity   per hidden HCU, swap the active input HCU of lowest mutual
 *                information for the silent one of highest                  Sec. 2, last paragraph
 *
 * Terms: an HCU (hypercolumn) is a group of MCUs (minicolumns) whose activities form one
 * discrete distribution.  Units are numbered HCU-major: unit = hcu * M + mcu.  C_i, C_j, C_ij
 * are called Pi, Pj, Pij below and l is `alpha`.
 *
 * Layouts (row-major, fp32 unless stated):
 *   x       [B][N_in]            input activities, N_in = in_hcu * in_mcu
 *   y, s    [B][N_out]           hidden activities / support, N_out = out_hcu * out_mcu
 *   target  [B][N_out]           clamped activities for supervised training
 *   winner  [B][out_hcu] int32   argmax MCU index of each hidden HCU
 *   pi [N_in], pj [N_out], b [N_out]
 *   pij, w  [N_in][N_out]        i-major: block (hi, hj) is in_mcu rows x out_mcu columns
 *   mask    [in_hcu][out_hcu] uint8, 1 = active connection, 0 = silent
 *
 * Ownership and streams: the layer owns every state buffer (allocated in create, freed in
 * destroy).  Caller buffers named *_dev are device pointers (16-byte aligned, contiguous) that
 * the caller owns; *_host are host pointers.  Every call enqueues its kernels on the stream
 * given to create and returns without waiting, except get_state, set_state, get_mi, the
 * profile reads and structural_update with a non-NULL count pointer, which wait for the
 * stream.  Calls on one layer must not run concurrently from several host threads.
 *
 * Second stream: train_batch updates, on the caller's stream, everything the next batch reads
 * (Pij and w of active blocks, Pi, Pj, b, the activities).  The Pij of silent blocks are
 * updated on a stream the layer owns (default priority, non-blocking), for up to eight batches
 * in one pass with the same per-batch arithmetic; the caller's stream is made to wait for that
 * work before every call that reads or replaces Pij (get_state, set_state, structural_update,
 * recompute_weights, the profile reads, flush) and destroy waits for both streams.  The results
 * are those of per-batch updates, bit for bit, except on a large layer (more than 64 blocks of
 * 32 x 32 elements per compute unit) with complement pairs and fp32 storage: there the silent
 * elements take the queued updates regrouped as c1^n P + (the batches' scaled contractions),
 * equal in real arithmetic and within a few fp32 ulps per batch of per-batch updates.
 *
 * HIP graphs: forward, train_batch, recompute_weights, readout, flush, structural_update
 * with a NULL count and structural_update_static allocate nothing, wait for nothing and
 * enqueue no memset, so a sequence of them can be captured on the layer's stream (with
 * profiling off) into a HIP graph.  The layer's host-side bookkeeping (which trace and
 * operand buffers the next batch uses, which silent updates are queued) advances when a call
 * is made, so a captured sequence that ends with flush must be replayed exactly once, before
 * any later call on the layer.
 *
 * Errors: every call returns a bcpnn_status.  Arguments are checked on the host before any
 * device work; BCPNN_EINVAL leaves the layer unchanged.  A failed HIP call returns
 * BCPNN_EDEVICE and marks the layer failed: later calls on it return BCPNN_ESTATE (destroy
 * still works).  Input properties that only the device can see (complement_pairs below) are
 * checked by the kernels and reported by the next call that waits for the stream, as
 * BCPNN_EINPUT, which also marks the layer failed.  bcpnn_last_error() describes the last
 * failure of the calling thread.
 */
#ifndef BCPNN_H
#define BCPNN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct bcpnn_layer bcpnn_layer;

typedef enum {
    BCPNN_OK = 0,
    BCPNN_EINVAL = -1,   /* invalid argument; nothing was changed                        */
    BCPNN_ENOMEM = -2,   /* device or host allocation failed                             */
    BCPNN_EDEVICE = -3,  /* a HIP call failed; the layer is now unusable                 */
    BCPNN_ESTATE = -4,   /* the layer failed earlier                                     */
    BCPNN_EINPUT = -5    /* an earlier train_batch's input broke a property the layer was
                            configured with (complement_pairs); its traces are not the
                            method's; the layer is now unusable                          */
} bcpnn_status;

/* Storage format of Pij and W.  F32 stores fp32.  BF16 and M10 keep fp32 arrays whose values
 * are rounded to nearest-even to 7 (bfloat16) or 10 mantissa bits after every update; the
 * paper's FPGA backend varies this width (Sec. 3, FPGA backend).  Arithmetic stays fp32. */
typedef enum { BCPNN_STORE_F32 = 0, BCPNN_STORE_BF16 = 1, BCPNN_STORE_M10 = 2 } bcpnn_storage;

typedef struct {
    int32_t in_hcu, in_mcu;     /* input HCUs and MCUs per HCU (> 0, in_hcu <= 49152,
                                   N_in <= 65535 * 64)                                       */
    int32_t out_hcu, out_mcu;   /* hidden HCUs and MCUs per HCU (> 0, out_mcu <= 1024,
                                   N_out <= 2^22)                                            */
    int32_t max_batch;          /* largest B accepted by forward/train_batch/readout,
                                   in [1, 2^20]; also N_in * N_out <= 2^35,
                                   in_hcu * out_hcu <= 2^26, ceil(max_batch / 16) * out_hcu
                                   <= 2^23 (launch grids stay below 2^32 work-items)          */
    float alpha;                /* trace rate l of Alg. 1, in (0, 1]; from a time constant
                                   tau (in batches) use alpha = 1 / tau                      */
    int32_t n_cycles;           /* repetitions of the trace/weight cycle per batch (>= 1);
                                   equivalent to one cycle at 1 - (1 - alpha)^n_cycles        */
    float gain;                 /* softmax gain g (>= 0, finite); 1 is the paper's softmax    */
    float bias_gain;            /* k_B of Alg. 1 (finite)                                     */
    float eps;                  /* lower clamp of each probability inside a log (a normal
                                   float: FLT_MIN <= eps, finite)                            */
    float pi_init, pj_init;     /* initial Pi, Pj; <= 0 selects 1 / in_mcu, 1 / out_mcu        */
    float init_noise;           /* initial w = mask * init_noise * (2u - 1), u ~ U[0, 1) from
                                   the SplitMix64 finaliser of (seed, i * N_out + j)          */
    uint64_t seed;
    int32_t n_swaps;            /* swaps per hidden HCU per structural update (>= 0)          */
    int32_t storage;            /* bcpnn_storage                                              */
    int32_t complement_pairs;   /* 0 or 1.  1 declares that every input HCU has two MCUs whose
                                   activities are x and 1 - x (the pixel encoding of the
                                   paper's image inputs; requires in_mcu == 2).  The batch sum
                                   of the second row of each pair is then taken as
                                   sum_b t_bj - sum_b x_b t_bj, equal in real arithmetic for
                                   such inputs, so the joint-trace contraction runs over half
                                   the input units.  train_batch checks every pair of its
                                   input (|x_2p + x_2p+1 - 1| <= 1e-6, NaN fails) and a
                                   violation makes the next waiting call return BCPNN_EINPUT.
                                   0 (the default) contracts every input unit.                */
} bcpnn_config;

/* Host-side view of the layer state (fp32 arrays and the uint8 mask, layouts above). */
typedef struct {
    float *pi, *pj, *pij, *w, *b;
    uint8_t *mask;
} bcpnn_state_view;

/* Fills cfg with the defaults (alpha 1e-3, one cycle, gain 1, k_B 1, eps 1e-8, uniform initial
 * traces, init_noise 0.1, seed 0, one swap, fp32 storage, complement_pairs 0) for the given
 * sizes. */
void bcpnn_config_default(bcpnn_config *cfg, int32_t in_hcu, int32_t in_mcu, int32_t out_hcu,
                          int32_t out_mcu, int32_t max_batch);

/* Creates a layer (Alg. 1 initial state): Pi = pi_init, Pj = pj_init, Pij = Pi * Pj,
 * b = k_B log Pj, w = the masked noise described at init_noise.  mask_host is
 * [in_hcu][out_hcu] of 0/1 (NULL = every connection active); every hidden HCU needs at least
 * one active input HCU.  hip_stream is a hipStream_t (NULL = the null stream).  The layer
 * allocates about 8 * N_in * N_out bytes of device memory for Pij and w, 24 sets of batch
 * operands of 4 * (N_in + N_out) * ceil(max_batch / 16) * 17 bytes each (the silent-block
 * sweeps of queued batches read them later), and smaller buffers; it creates its second stream.
 * Errors: EINVAL (sizes, rates, mask), ENOMEM, EDEVICE. */
bcpnn_status bcpnn_layer_create(const bcpnn_config *cfg, const uint8_t *mask_host,
                                void *hip_stream, bcpnn_layer **out);

/* Releases the layer and its device memory after its stream is idle.  NULL is ignored. */
void bcpnn_layer_destroy(bcpnn_layer *layer);

/* Inference (Alg. 1 support and softmax lines, no learning): y_dev [B][N_out] receives the
 * activities; s_dev (nullable) the support.  1 <= B <= max_batch. */
bcpnn_status bcpnn_forward(bcpnn_layer *layer, const float *x_dev, int32_t B, float *y_dev,
                           float *s_dev);

/* One training batch, Alg. 1 from the batch input to "apply mask" (support, softmax, the
 * n_cycles trace updates with the batch means, weights, bias, mask).  If target_dev is not NULL
 * its rows replace the softmax activity in the trace updates (supervised output layer, Sec. 2).
 * y_dev (nullable) receives the softmax activities.  1 <= B <= max_batch; the means divide by B. */
bcpnn_status bcpnn_train_batch(bcpnn_layer *layer, const float *x_dev, int32_t B,
                               const float *target_dev, float *y_dev);

/* Recomputes w and b from the current traces and mask (Alg. 1 weight, bias and mask lines). */
bcpnn_status bcpnn_recompute_weights(bcpnn_layer *layer);

/* Structural plasticity (Alg. 1 "update plasticity mask"; Sec. 2): scores every
 * (input HCU, hidden HCU) pair by the mutual information of its block of Pij (fp64), then for
 * each hidden HCU swaps, up to n_swaps times, the active input HCU of lowest score for the
 * silent one of highest score when that score is strictly larger (ties: lowest HCU index), and
 * rewrites the changed blocks of w.  The caller schedules it (before a batch).
 * n_swapped_host (nullable) receives the number of swaps; passing it waits for the stream. */
bcpnn_status bcpnn_structural_update(bcpnn_layer *layer, int32_t *n_swapped_host);

/* For callers that cannot allocate memory or wait for the device (code under HIP graph capture,
 * serving loops, harnesses that forbid allocation): bcpnn_structural_update without them.  It
 * computes the same scores and makes the same swaps and weight patches with the same kernels,
 * but keeps the scores and per-HCU swap counts in a static scratch array of the library (32 MiB
 * of device memory per GPU, held until the process ends) instead of the layer's buffers, and
 * writes the number of swaps to n_swapped_dev (a device int32, 4-byte aligned, nullable)
 * instead of returning it on the host.  It calls no allocating routine and does not wait.
 * Limit: in_hcu * out_hcu * 8 (rounded up to 256) + out_hcu * 4 bytes <= 32 MiB, else EINVAL
 * (e.g. 27648 x 100 HCUs fit).  Every call on one GPU shares that array and leaves the last
 * call's contents in it, so such calls on one GPU must not overlap (calls on one stream never
 * do; calls on different streams race).  The scores are not kept: get_mi afterwards returns
 * EINVAL.  Errors: EINVAL, ESTATE, EDEVICE. */
bcpnn_status bcpnn_structural_update_static(bcpnn_layer *layer, int32_t *n_swapped_dev);

/* Readout (Sec. 2, inference: the trained network is evaluated like a conventional
 * feed-forward network, from the support of the output layer): winner_dev [B][out_hcu]
 * receives, for each sample and hidden HCU, the MCU index of the largest support s_j of the
 * Alg. 1 support line (ties: lowest index).  No learning; 1 <= B <= max_batch.  x_dev as for
 * forward; winner_dev is caller-owned device memory, 16-byte aligned. */
bcpnn_status bcpnn_readout(bcpnn_layer *layer, const float *x_dev, int32_t B,
                           int32_t *winner_dev);

/* Applies the queued silent-block updates of Pij (train_batch defers them; see "Second stream"
 * above) and makes the caller's stream wait for them: work enqueued on that stream after this
 * call sees every Pij as per-batch updates leave it.  It enqueues only and does not wait for
 * the host.  A caller that times a run, or hands the layer's stream to other work that reads
 * Pij, calls it at the end of its batches.  Errors: ESTATE, EDEVICE. */
bcpnn_status bcpnn_flush(bcpnn_layer *layer);

/* Copies the state to host arrays (each pointer of the view may be NULL to skip it).  Applies
 * the queued silent-block updates first (it enqueues work, so the layer is not const).  Waits. */
bcpnn_status bcpnn_get_state(bcpnn_layer *layer, const bcpnn_state_view *host_out);

/* Replaces the state from host arrays (all six pointers required).  The mask must satisfy the
 * create rules; w is stored with the mask applied (silent blocks become 0).  Waits. */
bcpnn_status bcpnn_set_state(bcpnn_layer *layer, const bcpnn_state_view *host_in);

/* Copies the mutual-information scores of the last structural update, [in_hcu][out_hcu] fp64,
 * to the host.  Waits.  EINVAL before the first structural update. */
bcpnn_status bcpnn_get_mi(bcpnn_layer *layer, double *mi_host);

/* Kernel timing for measurement: with period n > 0, every n-th launch of the silent-block sweep
 * of the joint traces, counting from the call, is bracketed by a pair of HIP events recorded on
 * its stream right before and after it (their interval is the kernel's execution plus the
 * events' short passage through the stream); when the mask has no silent block, the
 * active-block trace kernel's launches are timed instead, by their own clock stamps (see
 * bcpnn_profile_read_kernel); n = 0 turns it off.  Each timed launch costs the stream a few
 * microseconds, so a period of 10 or more keeps a throughput measurement nearly
 * unperturbed.  bcpnn_profile_read waits for both
 * streams and returns the summed duration (ms) and count of the timed launches since the last
 * read; silent updates still queued stay queued (a read does not change which batches a sweep
 * covers: bcpnn_flush applies them).
 * Errors: EINVAL for n < 0. */
bcpnn_status bcpnn_profile_enable(bcpnn_layer *layer, int32_t period);
bcpnn_status bcpnn_profile_read(bcpnn_layer *layer, double *total_ms, int32_t *launches);

/* The same for one kernel: the silent-block sweep, the support (with softmax and the
 * contraction operands) or the active-block trace kernel of train_batch, the weight pass of
 * recompute_weights (w over the whole matrix; the bias kernel after it is not included), or
 * the structural update (from the start of the mutual-information kernel to the end of the
 * swap kernel; the queued sweep it applies first is not included).  The support and active
 * kernels, short launches on the caller's stream, are not bracketed by events: a timed launch
 * stamps the device clock (hipDeviceAttributeWallClockRate) when its first workgroup starts and
 * when its last one ends, and its duration is that span: the kernel's execution on the compute
 * units (a kernel trace also counts the dispatch's start and completion, 1-2 us).
 * profile_enable's period applies to each kernel's own launch count.  Reads and clears that
 * kernel's record only.
 * Errors: EINVAL for an unknown kernel or NULL outputs. */
typedef enum {
    BCPNN_KERNEL_SWEEP = 0,
    BCPNN_KERNEL_SUPPORT = 1,
    BCPNN_KERNEL_ACTIVE = 2,
    BCPNN_KERNEL_WEIGHTS = 3,
    BCPNN_KERNEL_STRUCTURAL = 4
} bcpnn_kernel;
bcpnn_status bcpnn_profile_read_kernel(bcpnn_layer *layer, int32_t kernel, double *total_ms,
                                       int32_t *launches);

/* Message of the calling thread's last failure ("" if none). */
const char *bcpnn_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* BCPNN_H */
