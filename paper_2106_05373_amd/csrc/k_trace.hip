// Joint-trace contraction with the trace, weight and bias updates (Alg. 1 cycle loop):
//
//   T[i][j]  = sum_b x[b][i] t[b][j]                       (the batch sum of a_i (x) a_j)
//   Pij     <- c1 Pij + c2 T[i][j]                         c1 = 1 - a_eff, c2 = a_eff / B
//   Pi, Pj  <- c1 P + a_eff mean_b(.)
//   w[i][j]  = log max(Pij,eps) - log max(Pi,eps) - log max(Pj,eps)   on active blocks only
//   b[j]     = k_B log max(Pj, eps)
//
// a_eff = 1 - (1 - alpha)^n_cycles folds the paper's n_cycles repetitions with the same batch
// means into one update (exact in real arithmetic).
//
// Design (gfx950):
//  * T is a dense [N_in x N_out] product with K = B (the batch).  Every Pij is needed (silent
//    connections are scored for plasticity), so the contraction is dense.
//  * The update is split by the mask into two kernels that touch disjoint elements:
//      - the active kernel updates the elements of active blocks (the rows of each hidden
//        HCU's active input units, gathered) together with their weights, and the marginal
//        traces and bias of every unit: everything the next batch's support reads;
//      - the silent kernel sweeps the whole matrix and stores the elements of silent blocks.
//    For a small layer the library runs the silent kernel on a second stream, where it overlaps
//    the next batch's support kernel (which never reads silent elements); every state access
//    waits for it.  A large layer's sweep runs in order on the caller's stream.
//  * With complement pairs (every input HCU holds x and 1 - x) the contraction covers the first
//    unit of each pair and the second row takes the column total minus it (the *_pair_*
//    kernels below), halving the matrix work and the x operand traffic.
//  * T runs on the bf16 matrix cores with a two-term split of both operands: v = hi + lo with
//    hi = bf16(v), lo = bf16(v - hi), and T ~ lo.hi' + hi.lo' + hi.hi' (three
//    v_mfma_f32_32x32x16_bf16, fp32 accumulation).  Each product is then exact to about 3
//    parts in 2^17 (the dropped lo.lo' term and the rounding of lo), so T carries a relative
//    error of order 1e-5; the trace update scales it by a_eff / B, which puts it near 1e-8 in
//    Pij.  Three bf16 MFMAs cost 3/16 of the fp32 MFMA time of the same product, so the
//    kernels are bound by memory: 8 bytes of Pij per element plus 4 per active weight from
//    HBM, and the operands from L2.
//  * The support kernel of the same batch has already written x^T and t^T split, in MFMA
//    fragment order (one 1 KiB chunk per 32 units and 16 batch rows), and the column sums of x
//    and t per 16-row tile.
//  * The sweep of a large layer (more than 64 blocks per CU) uses 128 x 128 workgroup tiles
//    whose operands are staged through LDS (see trace_sweep_tile_kernel); everything else
//    below describes the one-wave-per-block kernels.
//  * Every wave owns one 32 x 32 block and works alone: no LDS staging, no barrier.  It
//    requests its Pij values (and, in the active kernel, the inputs of its rows' and columns'
//    marginal traces) first, then streams the operands straight into registers (each k-step of
//    each operand is one contiguous 1 KiB read in the sweep, 32 16-byte pieces when the rows
//    are gathered), four k-steps at a time, and runs the MFMAs.  The many independent waves in
//    flight hide the memory latency.
//  * Sweep: a workgroup is four waves on one row block and four neighbouring column blocks:
//    they read the same x fragments (L1 hits after the first) and write 512 contiguous bytes
//    of each row.  Workgroups are ordered so that those of one XCD cover one contiguous
//    stretch of blocks.  Pij values are buffer loads over the block's rows (rows past the
//    layer read as zero); all stores are unconditional buffer stores, a store that must not
//    happen (an element of an active block, a column past the layer) getting an offset past
//    the buffer range, which the hardware drops.
//  * Marginals: Pi of a row and Pj of a column are computed from the column sums by the same
//    code wherever they are needed (hence identical values); dedicated workgroups of the
//    active kernel store Pi, Pj and b for every unit.  Pi and Pj are read from one buffer and
//    written to another (the host alternates them).
//
// MFMA 32x32x16 bf16 lane layout (verified on gfx950): A[i][k] for k = 8 (l / 32) + 0..7 from
// lane l = i + 32 (k / 8), B[k][j] likewise with j = l % 32, and lane l holds
// D[8 (r / 4) + 4 (l / 32) + r % 4][l % 32] in result register r.
#include <type_traits>

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
constexpr int kActiveChunk = 8;     // the same in the active kernel (few waves: one round trip
                                    // covers a batch of 128)
constexpr int kPairChunk = 2;       // the same in the small sweep with complement pairs (its
                                    // registers also hold both rows of each input HCU)
constexpr int kSums = 8;            // column-sum tiles requested up front (the batch for B <= 128)
constexpr int kSweepRows = 16;      // row blocks per sweep over the column groups (tiled sweep)
constexpr int64_t kStripeBytes = 3 << 19;  // t fragments an XCD keeps in L2 (persistent sweep)
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

// Value of lane src in lanes 0..31 and of lane src + 4 in lanes 32..63 (src a constant).
template <typename T>
__device__ __forceinline__ T half_broadcast(T v, int src, int lane) {
    const int bits = __builtin_bit_cast(int, v);
    const int lo = __builtin_amdgcn_readlane(bits, src);
    const int hi = __builtin_amdgcn_readlane(bits, src + 4);
    return __builtin_bit_cast(T, lane < 32 ? lo : hi);
}

// Inputs of one unit's marginal trace: its column sums over the batch's 16-row tiles (the
// first kSums requested up front) and its previous value.
struct MarginalIn {
    float part[kSums];
    float p_old;
};

__device__ __forceinline__ void marginal_request(MarginalIn& m, const float* sums, int64_t st,
                                                 int u, int nk, const float* p_old) {
#pragma unroll
    for (int q = 0; q < kSums; ++q) m.part[q] = sums[(q < nk ? q : nk - 1) * st + u];
    m.p_old = p_old[u];
}

// Column sum over the batch: the 16-row tile sums added in tile order, starting from zero.
// Every kernel forms a column's sum in this order, so all of them get the same bits.
__device__ __forceinline__ float marginal_colsum(const MarginalIn& m, const float* sums,
                                                 int64_t st, int u, int nk) {
    float colsum = 0.0f;
#pragma unroll
    for (int q = 0; q < kSums; ++q)
        if (q < nk) colsum += m.part[q];
    for (int q = kSums; q < nk; ++q) colsum += sums[q * st + u];     // batches above 128
    return colsum;
}

// P = c1 P_old + a_eff * (column sum / B); the same operations in the same order everywhere.
__device__ __forceinline__ float marginal_from_colsum(const MarginalIn& m, float colsum,
                                                      const TraceArgs& a) {
    return fmaf(a.a_eff, colsum * a.inv_b, a.c1 * m.p_old);
}

__device__ __forceinline__ float marginal_value(const MarginalIn& m, const float* sums, int64_t st,
                                                int u, int nk, const TraceArgs& a) {
    return marginal_from_colsum(m, marginal_colsum(m, sums, st, u, nk), a);
}

// Marginal traces and bias of unit v of the layer (rows first, then columns): the work of the
// workgroups past the blocks in the active-block kernels.
__device__ __forceinline__ void store_marginal(const Geometry& g, const TraceArgs& a, int64_t v,
                                               int nk) {
    const int n_in = (int)g.n_in, n_out = (int)g.n_out;
    if (v >= (int64_t)n_in + n_out) return;
    const bool is_row = v < n_in;
    const int u = is_row ? (int)v : (int)(v - n_in);
    const float* sums = is_row ? a.ops.x_sum : a.ops.t_sum;
    const int64_t st = is_row ? n_in : n_out;
    MarginalIn m;
    marginal_request(m, sums, st, u, nk, is_row ? a.pi_old : a.pj_old);
    const float p = marginal_value(m, sums, st, u, nk, a);
    if (is_row) {
        a.pi_new[u] = p;
    } else {
        a.pj_new[u] = p;
        a.b[u] = a.bias_gain * fast_log(fmaxf(p, a.eps));
    }
}

// Silent sweep: every 32 x 32 block of Pij, updated by the contractions of a.n_batches
// consecutive batches in order, storing the elements whose block is silent.
template <int kDropBits>
__global__ void __launch_bounds__(kWaves * 64) __attribute__((amdgpu_waves_per_eu(3, 3)))
trace_sweep_kernel(Geometry g, SweepArgs a, int n_cg, int n_work, int stripe) {
    const int lane = threadIdx.x & 63;
    const int n_in = (int)g.n_in, n_out = (int)g.n_out;
    // Persistent: workgroup b takes work items b, b + G, ... (G = gridDim.x, a multiple of 8, so
    // they all lie on the workgroup's XCD).
    for (int item = blockIdx.x; item < n_work; item += gridDim.x) {
        // work item -> (row block, group of kWaves column blocks).  The items of one XCD form
        // one contiguous stretch of this order: stripes of `stripe` column groups, each walked
        // row block by row block.  The t fragments of a stripe (all queued batches) stay in the
        // XCD's L2 while the x fragments of each row block are read once per stripe, by the
        // stripe's column groups one after another.
        const int n_rb = (n_in + 31) / 32;
        const int wg = (int)xcd_linear_index(item, n_work);
        const int s0 = wg / (n_rb * stripe) * stripe;             // first column group
        const int in_stripe = wg - s0 * n_rb;
        const int groups_here = n_cg - s0 < stripe ? n_cg - s0 : stripe;
        const int bi = in_stripe / groups_here;
        const int bj = (s0 + in_stripe % groups_here) * kWaves + (threadIdx.x >> 6);
        const int i0 = bi * 32, j0 = bj * 32;
        if (j0 >= n_out) continue;                                 // wave-uniform; no barriers
        const int rows = n_in - i0 < 32 ? n_in - i0 : 32;
        const int cols = n_out - j0 < 32 ? n_out - j0 : 32;
        const int n_ks = a.n_ks;
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
        // lanes 0..31 the block's row units, 32..63 its column units (clamped)
        const bool is_row = lane < 32;
        const int u = is_row ? i0 + (lane < rows ? lane : rows - 1)
                             : j0 + (lane - 32 < cols ? lane - 32 : cols - 1);
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

        // ---- per batch: contraction (operands straight from the fragment-order arrays), update --
        const int64_t fa = ((int64_t)bi * n_ks * 64 + lane) * 8;
        const int64_t fb = ((int64_t)bj * n_ks * 64 + lane) * 8;
        for (int t = 0; t < a.n_batches; ++t) {
            const SweepBatch bt = a.bt[t];
            const int nk = bt.nk;
            f16v acc = {};
            for (int k0 = 0; k0 < nk; k0 += kChunk) {
                u32x4 op[kChunk][4];
#pragma unroll
                for (int c = 0; c < kChunk; ++c) {
                    const int64_t ks = (int64_t)(k0 + c < nk ? k0 + c : nk - 1) * 512;
                    op[c][0] = *reinterpret_cast<const u32x4*>(bt.x_hi + fa + ks);
                    op[c][1] = *reinterpret_cast<const u32x4*>(bt.x_lo + fa + ks);
                    op[c][2] = *reinterpret_cast<const u32x4*>(bt.t_hi + fb + ks);
                    op[c][3] = *reinterpret_cast<const u32x4*>(bt.t_lo + fb + ks);
                }
                // every load of the chunk issued before the first product waits on one
                __builtin_amdgcn_sched_barrier(0);
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
#pragma unroll
            for (int r = 0; r < 16; ++r)
                pold[r] = to_storage<kDropBits>(fmaf(bt.c2, acc[r], bt.c1 * pold[r]));
        }

        // ---- epilogue: the elements of silent blocks, 16 unconditional buffer stores ----------
        const bool jok = jl < cols;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int il = il0 + 8 * (r >> 2) + (r & 3);
            const uint32_t off = o0 + (uint32_t)(8 * (r >> 2) + (r & 3)) * n_out * 4u;
            const bool keep = jok && !((act_bits >> il) & 1u);
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(pold[r]), rp,
                                                  keep ? off : kDrop, 0, 0);
        }
    }
}
// Mask of the lane's column over a 32 x 32 block's rows, one bit per row (rows i0 .. i0 + rows - 1,
// columns j0 .. j0 + cols - 1), as in the sweep below: one byte per lane and one ballot when the
// block's columns fall in at most two hidden HCUs, else the bytes of the lane's 16 elements.
// hu: in lanes 0..31 the input HCU of block row lane, in lanes 32..63 the hidden HCU of block
// column lane - 32 (both clamped into the layer).
__device__ __forceinline__ uint32_t block_mask_bits_hu(const Geometry& g, const uint8_t* mask,
                                                       int hu, int lane) {
    const int jl = lane & 31;
    const int il0 = 4 * (lane >> 5);
    const int hj = __shfl(hu, 32 + jl, 64);
    const int hc0 = __shfl(hu, 32, 64), hc1 = __shfl(hu, 63, 64);
    uint32_t bits32 = 0;
    if (hc1 - hc0 <= 1) {                                          // wave-uniform
        const int hr = __shfl(hu, jl, 64);
        const int hc = hc0 + (lane >> 5) < hc1 ? hc0 + (lane >> 5) : hc1;
        const uint64_t bits = __ballot(mask[(int64_t)hr * g.out_hcu + hc] != 0);
        bits32 = hj == hc0 ? (uint32_t)bits : (uint32_t)(bits >> 32);
    } else {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int il = il0 + 8 * (r >> 2) + (r & 3);
            const int hi = __shfl(hu, il, 64);
            bits32 |= (mask[(int64_t)hi * g.out_hcu + hj] != 0 ? 1u : 0u) << il;
        }
    }
    return bits32;
}

__device__ __forceinline__ uint32_t block_mask_bits(const Geometry& g, const uint8_t* mask,
                                                    int i0, int rows, int j0, int cols,
                                                    int lane) {
    const bool is_row = lane < 32;
    const int u = is_row ? i0 + (lane < rows ? lane : rows - 1)
                         : j0 + (lane - 32 < cols ? lane - 32 : cols - 1);
    return block_mask_bits_hu(g, mask, is_row ? u / g.in_mcu : u / g.out_mcu, lane);
}

// Silent sweep of a large layer: one 128 x 128 tile (4 x 4 blocks) per workgroup of four waves,
// wave w on row block w of the tile and all four column blocks (64 accumulators).  The t
// fragments of the four column blocks, which every wave reads, are copied straight into LDS by
// the memory unit (global_load_lds, 16 bytes per lane, 1 KiB per fragment chunk) into one of
// two stage buffers of kKC k-steps; each wave's x fragments (its own row block, read by no other
// wave) go straight into registers; both one chunk ahead of the matrix cores, one barrier per
// chunk.  The chunk sequence runs over all the queued batches; after a batch's last chunk the
// wave applies that batch's update to its Pij values in registers.  Operand traffic from L2 is
// 16 bytes per element per batch of 256 (40 with one wave per block); every wave takes part in
// every barrier (waves past the layer compute on clamped data and store nothing).
// Measured on the STL-shaped layer (4 batches per launch): 3.44-3.52 ms; x through LDS as well
// 3.57-3.62 ms (deeper stages: four of one k-step 3.74 ms, three of two at one workgroup per CU
// 6.85 ms); the one-wave-per-block sweep 5.21 ms.
__device__ __forceinline__ void stage_barrier() {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// s_waitcnt immediate with vmcnt = n (6 bits) and the other counters left alone.
constexpr int vm_wait(int n) { return (n & 0xF) | ((n >> 4) << 14) | (0x7 << 4) | (0xF << 8); }

// Stage buffer index as a type.  The two stage buffers of a tiled sweep are separate LDS arrays
// and the chunk loop is unrolled by two, so that every access names its buffer at compile time:
// the compiler then knows that a chunk's LDS reads do not touch the buffer that the next
// chunk's direct-to-LDS loads are filling, and lets those loads run under the chunk's products.
// (With one array indexed by the chunk's parity it cannot tell the buffers apart and waits for
// the next chunk's loads before the first read of the current one.)
template <int V>
struct StageIx { static constexpr int value = V; };

constexpr int kTileKC = 2;
constexpr int kPairTileCB = 3;   // column blocks per workgroup of the tiled sweep with pairs
constexpr int kSumTileCB = 8;    // column blocks per workgroup of the sum-form sweep
constexpr int kSumTileWaves = 4; // waves (blocks of 32 input HCUs) per workgroup of it
constexpr int kSumTileKC = 1;    // k-steps per chunk of it
constexpr int kSumTileStages = 4;   // its stage buffers: chunks in flight + 1

template <int kDropBits, int kKC>
__global__ void __launch_bounds__(kWaves * 64) __attribute__((amdgpu_waves_per_eu(2, 2)))
trace_sweep_tile_kernel(Geometry g, SweepArgs a, int n_tj) {
    constexpr int kItems = 8 * kKC;                 // 1 KiB t items per chunk
    constexpr int kPerWave = kItems / kWaves;
    __shared__ u32x4 stage0[kItems][64];
    __shared__ u32x4 stage1[kItems][64];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int n_in = (int)g.n_in, n_out = (int)g.n_out;
    const int n_rb = (n_in + 31) / 32, n_cb = (n_out + 31) / 32;
    const int n_ti = (n_rb + 3) / 4;
    constexpr int kSweepTiles = kSweepRows / 4;
    const int wg = (int)xcd_linear_index(blockIdx.x, gridDim.x);
    const int sweep = wg / (kSweepTiles * n_tj);
    const int in_sweep = wg % (kSweepTiles * n_tj);
    const int here = n_ti - sweep * kSweepTiles < kSweepTiles ? n_ti - sweep * kSweepTiles
                                                              : kSweepTiles;
    const int ti = sweep * kSweepTiles + in_sweep % here;
    const int tj = in_sweep / here;
    const int n_ks = a.n_ks;

    const int bi = 4 * ti + wave;
    const int bic = bi < n_rb ? bi : n_rb - 1;
    const int i0 = bic * 32;
    const int rows = n_in - i0 < 32 ? n_in - i0 : 32;
    const bool live = bi < n_rb;                           // wave-uniform
    const int j00 = 4 * tj * 32;
    const int jl = lane & 31, il0 = 4 * (lane >> 5);
    const rsrc_t rp = make_rsrc(a.pij + (int64_t)i0 * n_out, (uint32_t)rows * n_out * 4u);
    const uint32_t o0 = ((uint32_t)il0 * n_out + j00 + jl) * 4u;
    float pold[4][16];
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r)
            pold[c][r] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
                rp, o0 + (uint32_t)((8 * (r >> 2) + (r & 3)) * n_out + 32 * c) * 4u, 0, 0));
    uint32_t act_bits[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const int j0 = j00 + 32 * c;
        const int jc = j0 < n_out ? j0 : (n_cb - 1) * 32;
        act_bits[c] = block_mask_bits(g, a.mask, i0, rows, jc, n_out - jc < 32 ? n_out - jc : 32,
                                      lane);
    }

    int n_ch = 0;
    for (int t = 0; t < a.n_batches; ++t) n_ch += (a.bt[t].nk + kKC - 1) / kKC;
    // requests of the chunk at (batch t, first k-step k0): the t items into stage buffer sb
    // (item = (k-step in chunk * 4 + column block) * 2 + {hi, lo}, wave w issuing w, w + 4, ...)
    // and this wave's x fragments into xn
    u32x4 xc[kKC][2], xn[kKC][2];
    auto request = [&](int t, int k0, auto sb_c) {
        u32x4 (*const st)[64] = decltype(sb_c)::value == 0 ? stage0 : stage1;
        const SweepBatch bt = a.bt[t];
#pragma unroll
        for (int q = 0; q < kPerWave; ++q) {
            const int item = wave + kWaves * q;
            const int half = item & 1, cb = (item >> 1) & 3, kq = item >> 3;
            int blk = 4 * tj + cb;
            blk = blk < n_cb ? blk : n_cb - 1;
            const int ks = k0 + kq < bt.nk ? k0 + kq : bt.nk - 1;
            const uint16_t* src = (half ? bt.t_lo : bt.t_hi) +
                                  (((int64_t)blk * n_ks + ks) * 64 + lane) * 8;
            __builtin_amdgcn_global_load_lds((const void*)src,
                (void __attribute__((address_space(3)))*)&st[item][0], 16, 0, 0);
        }
#pragma unroll
        for (int kq = 0; kq < kKC; ++kq) {
            const int ks = k0 + kq < bt.nk ? k0 + kq : bt.nk - 1;
            const int64_t fa = (((int64_t)bic * n_ks + ks) * 64 + lane) * 8;
            xn[kq][0] = *reinterpret_cast<const u32x4*>(bt.x_hi + fa);
            xn[kq][1] = *reinterpret_cast<const u32x4*>(bt.x_lo + fa);
        }
    };
    auto next = [&](int& t, int& k0) {
        k0 += kKC;
        if (k0 >= a.bt[t].nk) { k0 = 0; ++t; }
    };

    int dt = 0, dk = 0;
    request(dt, dk, StageIx<0>{});
    next(dt, dk);

    f16v acc[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[c] = f16v{};
    int ct = 0, ck = 0;
    // chunk lc, its t items in stage buffer sb_c (lc's parity)
    auto chunk = [&](int lc, auto sb_c) {
        constexpr int sb = decltype(sb_c)::value;
        const u32x4 (*const st)[64] = sb == 0 ? stage0 : stage1;
        // chunk lc's requests were the last issued: wait for all, then the barrier makes its t
        // items visible to every wave and tells that every wave is done with the other buffer
        __builtin_amdgcn_s_waitcnt(vm_wait(0));
#pragma unroll
        for (int kq = 0; kq < kKC; ++kq) {
            xc[kq][0] = xn[kq][0];
            xc[kq][1] = xn[kq][1];
        }
        stage_barrier();
        if (lc + 1 < n_ch) {
            request(dt, dk, StageIx<1 - sb>{});
            next(dt, dk);
        }
        const int nk = a.bt[ct].nk;
#pragma unroll
        for (int kq = 0; kq < kKC; ++kq) {
            if (ck + kq < nk) {
                const bf8 ah = __builtin_bit_cast(bf8, xc[kq][0]);
                const bf8 al = __builtin_bit_cast(bf8, xc[kq][1]);
                bf8 bh[4], bl[4];
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    bh[c] = __builtin_bit_cast(bf8, st[(kq * 4 + c) * 2][lane]);
                    bl[c] = __builtin_bit_cast(bf8, st[(kq * 4 + c) * 2 + 1][lane]);
                }
#pragma unroll
                for (int c = 0; c < 4; ++c)
                    acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, bh[c], acc[c], 0, 0, 0);
#pragma unroll
                for (int c = 0; c < 4; ++c)
                    acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bl[c], acc[c], 0, 0, 0);
#pragma unroll
                for (int c = 0; c < 4; ++c)
                    acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bh[c], acc[c], 0, 0, 0);
            }
        }
        if (ck + kKC >= nk) {
            const float c1 = a.bt[ct].c1, c2 = a.bt[ct].c2;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    pold[c][r] = to_storage<kDropBits>(fmaf(c2, acc[c][r], c1 * pold[c][r]));
                acc[c] = f16v{};
            }
        }
        next(ct, ck);
    };
    for (int lc = 0; lc < n_ch; lc += 2) {
        chunk(lc, StageIx<0>{});
        if (lc + 1 < n_ch) chunk(lc + 1, StageIx<1>{});
    }
    if (!live) return;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const bool jok = j00 + 32 * c + jl < n_out;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int il = il0 + 8 * (r >> 2) + (r & 3);
            const uint32_t off = o0 + (uint32_t)((8 * (r >> 2) + (r & 3)) * n_out + 32 * c) * 4u;
            const bool keep = jok && !((act_bits[c] >> il) & 1u);
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(pold[c][r]), rp,
                                                  keep ? off : kDrop, 0, 0);
        }
    }
}

// Active blocks: one workgroup per (hidden HCU, 32 of its active input units, 4 column blocks
// of the HCU), one wave per 32 x 32 block; workgroups past n_work store the marginal traces and
// bias of every unit instead.
template <int kDropBits, bool kStamp>
__global__ void __launch_bounds__(kWaves * 64) __attribute__((amdgpu_waves_per_eu(2, 2)))
trace_active_kernel(Geometry g, TraceArgs a, const int32_t* __restrict__ act_list,
                    const int32_t* __restrict__ act_count, int n_rt, int n_cgr, int n_work) {
    // Highest wave priority, as in the support kernel: it shares CUs with the silent sweep.
    __builtin_amdgcn_s_setprio(3);
    stamp_start<kStamp>(a.stamp);
    const int n_in = (int)g.n_in, n_out = (int)g.n_out;
    const int nk = (a.B + 15) / 16;
    const int n_ks = a.ops.n_ks;
    if ((int)blockIdx.x >= n_work) {
        store_marginal(g, a, (int64_t)(blockIdx.x - n_work) * blockDim.x + threadIdx.x, nk);
        stamp_end<kStamp>(a.stamp);
        return;
    }
    // The x fragment pieces of the block rows (32 gathered units), the same for the four waves,
    // are gathered once per workgroup into LDS, kActiveChunk k-steps at a time:
    // xs[k-step][hi, lo][lane], lane = unit slot + 32 * half, exactly the A operand of a wave.
    __shared__ u32x4 xs[kActiveChunk][2][64];
    const int lane = threadIdx.x & 63;
    const int wg = (int)xcd_linear_index(blockIdx.x, n_work);
    const int per_hcu = n_rt * n_cgr;
    const int hj = wg / per_hcu;
    const int rt = (wg - hj * per_hcu) / n_cgr;
    const int c0 = ((wg - hj * per_hcu - rt * n_cgr) * kWaves + (threadIdx.x >> 6)) * 32;
    // waves past the HCU's columns only help gather the x pieces (every wave takes part in
    // every barrier); they compute on clamped columns and store nothing
    const bool col_live = c0 < g.out_mcu;                      // wave-uniform
    const int cols = col_live ? (g.out_mcu - c0 < 32 ? g.out_mcu - c0 : 32) : 1;
    const int j0 = hj * g.out_mcu + (col_live ? c0 : 0);
    const int jl = lane & 31;
    const int il0 = 4 * (lane >> 5);
    const int h = lane >> 5;
    const int jb = j0 + (jl < cols ? jl : cols - 1);          // the lane's column (clamped)

    // ---- requests, in order of dependence -------------------------------------------------
    // The active count and the list entry of block row jl are requested together (rows past
    // the count read an in-bounds entry and are never stored), then everything on the column
    // side, which needs neither.
    const int k_total = act_count[hj] * g.in_mcu;
    const int n_units = g.in_hcu * g.in_mcu;
    const int kr = rt * 32 + jl < n_units ? rt * 32 + jl : n_units - 1;
    const int hsel = act_list[(int64_t)hj * g.in_hcu + kr / g.in_mcu];
    u32x4 opt[kActiveChunk][2], opx[kActiveChunk][2];
    auto load_t = [&](int k0) {
#pragma unroll
        for (int c = 0; c < kActiveChunk; ++c) {
            const int64_t fb = frag_chunk(jb, k0 + c < nk ? k0 + c : nk - 1, h, n_ks);
            opt[c][0] = *reinterpret_cast<const u32x4*>(a.ops.t_hi + fb);
            opt[c][1] = *reinterpret_cast<const u32x4*>(a.ops.t_lo + fb);
        }
    };
    // thread t gathers the pieces P = t + 256 q (unit slot P % 32 = lane % 32, half P / 32 % 2,
    // hi / lo P / 64 % 2, k-step P / 128) of the chunk at k0; then the wave reads its operands
    constexpr int kGather = kActiveChunk * 2 * 64 / (kWaves * 64);
    auto gather_x = [&](int k0, int ua) {
        u32x4 v[kGather];
#pragma unroll
        for (int q = 0; q < kGather; ++q) {
            const int P = threadIdx.x + kWaves * 64 * q;
            const int hp = (P >> 5) & 1, hl = (P >> 6) & 1, kq = P >> 7;
            const int ks = k0 + kq < nk ? k0 + kq : nk - 1;
            const int64_t fa = frag_chunk(ua, ks, hp, n_ks);
            v[q] = *reinterpret_cast<const u32x4*>((hl ? a.ops.x_lo : a.ops.x_hi) + fa);
        }
#pragma unroll
        for (int q = 0; q < kGather; ++q) {
            const int P = threadIdx.x + kWaves * 64 * q;
            xs[P >> 7][(P >> 6) & 1][P & 63] = v[q];
        }
    };
    auto load_x = [&]() {
#pragma unroll
        for (int c = 0; c < kActiveChunk; ++c) {
            opx[c][0] = xs[c][0][lane];
            opx[c][1] = xs[c][1][lane];
        }
    };
    f16v acc = {};
    auto contract = [&](int k0) {
#pragma unroll
        for (int c = 0; c < kActiveChunk; ++c) {
            if (k0 + c < nk) {
                const bf8 ah = __builtin_bit_cast(bf8, opx[c][0]);
                const bf8 al = __builtin_bit_cast(bf8, opx[c][1]);
                const bf8 bh = __builtin_bit_cast(bf8, opt[c][0]);
                const bf8 bl = __builtin_bit_cast(bf8, opt[c][1]);
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, bh, acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bl, acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bh, acc, 0, 0, 0);
            }
        }
    };
    load_t(0);

    // unit of block row jl (the A-operand row of this lane), clamped into the layer
    const int hs = hsel < 0 ? 0 : (hsel < g.in_hcu ? hsel : g.in_hcu - 1);
    const int ua = hs * g.in_mcu + kr % g.in_mcu;
    // Row of result register r: 8 (r / 4) + r % 4 in lanes 0..31, 4 more in lanes 32..63, so
    // its unit is a broadcast of one lane per half-wave (two lane reads, no permute).
    int ur[16];
    float pold[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        ur[r] = half_broadcast(ua, 8 * (r >> 2) + (r & 3), lane);
        pold[r] = a.pij[(int64_t)ur[r] * n_out + jb];
    }
    gather_x(0, ua);
    // marginal inputs: lanes 0..31 the block's row units, 32..63 its column units
    const bool is_row = lane < 32;
    const int u = is_row ? ua : jb;
    const float* sums = is_row ? a.ops.x_sum : a.ops.t_sum;
    const int64_t st = is_row ? n_in : n_out;
    MarginalIn m;
    marginal_request(m, sums, st, u, nk, is_row ? a.pi_old : a.pj_old);

    // ---- contraction: x pieces from LDS, t pieces of the columns from memory -----------------
    lds_barrier();
    load_x();
    contract(0);
    for (int k0 = kActiveChunk; k0 < nk; k0 += kActiveChunk) {   // batches above 128 rows
        lds_barrier();                                          // every wave has read its x
        load_t(k0);
        gather_x(k0, ua);
        lds_barrier();
        load_x();
        contract(k0);
    }
    if (col_live) {                                    // wave-uniform
        const int rows = k_total - rt * 32 < 32 ? k_total - rt * 32 : 32;   // may be <= 0

        // ---- marginal traces of the block's rows and columns, and their logs --------------------
        const float lp = fast_log(fmaxf(marginal_value(m, sums, st, u, nk, a), a.eps));
        const float lpj = __shfl(lp, 32 + jl, 64);

        // ---- epilogue: joint trace and weight of every element of the block ---------------------
        const bool jok = jl < cols;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int il = il0 + 8 * (r >> 2) + (r & 3);
            const float lpi = half_broadcast(lp, 8 * (r >> 2) + (r & 3), lane);
            const float pn = to_storage<kDropBits>(fmaf(a.c2, acc[r], a.c1 * pold[r]));
            const float wv = to_storage<kDropBits>(fast_log(fmaxf(pn, a.eps)) - lpi - lpj);
            if (jok && il < rows) {
                const int64_t e = (int64_t)ur[r] * n_out + jb;
                a.pij[e] = pn;
                a.w[e] = wv;
            }
        }
    }
    stamp_end<kStamp>(a.stamp);
}


// ---- complement pairs ----------------------------------------------------------------------
// Every input HCU p holds units 2p (x) and 2p + 1 (1 - x).  The kernels below contract only the
// first units, whose split operands the support kernel wrote indexed by p, and update both rows:
//   Pij[2p][j]     <- c1 Pij + c2 T[p][j]
//   Pij[2p + 1][j] <- c1 Pij + c2 (S[j] - T[p][j]),   S[j] = sum_b t[b][j]
// S is the column total in tile order (marginal_colsum).  A wave's 32 x 32 contraction over 32
// input HCUs and 32 columns then updates 64 x 32 elements: half the matrix-core work and half
// the x operand traffic per element.  Result register r of lane l belongs to input HCU
// 8 (r / 4) + 4 (l / 32) + r % 4 of the block, as in the kernels above.

// Silent sweep with complement pairs (small layers): trace_sweep_kernel over blocks of 32 input
// HCUs (64 rows).
template <int kDropBits>
__global__ void __launch_bounds__(kWaves * 64) __attribute__((amdgpu_waves_per_eu(3, 3)))
trace_sweep_pair_kernel(Geometry g, SweepArgs a, int n_cg, int n_work, int stripe) {
    const int lane = threadIdx.x & 63;
    const int n_out = (int)g.n_out;
    const int n_pb = (g.in_hcu + 31) / 32;
    for (int item = blockIdx.x; item < n_work; item += gridDim.x) {
        // the order of trace_sweep_kernel, over blocks of input HCUs
        const int wg = (int)xcd_linear_index(item, n_work);
        const int s0 = wg / (n_pb * stripe) * stripe;
        const int in_stripe = wg - s0 * n_pb;
        const int groups_here = n_cg - s0 < stripe ? n_cg - s0 : stripe;
        const int bi = in_stripe / groups_here;
        const int bj = (s0 + in_stripe % groups_here) * kWaves + (threadIdx.x >> 6);
        const int p0 = bi * 32, j0 = bj * 32;
        if (j0 >= n_out) continue;                                 // wave-uniform; no barriers
        const int prs = g.in_hcu - p0 < 32 ? g.in_hcu - p0 : 32;   // input HCUs of the block
        const int cols = n_out - j0 < 32 ? n_out - j0 : 32;
        const int n_ks = a.n_ks;
        const int jl = lane & 31;
        const int il0 = 4 * (lane >> 5);
        const int jc = j0 + (jl < cols ? jl : cols - 1);           // the lane's column (clamped)

        // rows 2 p0 .. 2 (p0 + prs) - 1; a row past them is out of the buffer range
        const rsrc_t rp = make_rsrc(a.pij + (int64_t)(2 * p0) * n_out,
                                    (uint32_t)(2 * prs) * n_out * 4u);
        const uint32_t o0 = ((uint32_t)(2 * il0) * n_out + j0 + jl) * 4u;
        const uint32_t odd = (uint32_t)n_out * 4u;
        float pe[16], po[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const uint32_t off = o0 + (uint32_t)(2 * (8 * (r >> 2) + (r & 3))) * n_out * 4u;
            pe[r] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rp, off, 0, 0));
            po[r] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rp, off + odd, 0, 0));
        }
        const int hu = lane < 32 ? p0 + (lane < prs ? lane : prs - 1) : jc / g.out_mcu;
        const uint32_t act_bits = block_mask_bits_hu(g, a.mask, hu, lane);

        const int64_t fa = ((int64_t)bi * n_ks * 64 + lane) * 8;
        const int64_t fb = ((int64_t)bj * n_ks * 64 + lane) * 8;
        for (int t = 0; t < a.n_batches; ++t) {
            const SweepBatch bt = a.bt[t];
            const int nk = bt.nk;
            // the column total's first tile sums, requested ahead of the contraction
            MarginalIn m;
#pragma unroll
            for (int q = 0; q < kSums; ++q)
                m.part[q] = bt.t_sum[(int64_t)(q < nk ? q : nk - 1) * n_out + jc];
            f16v acc = {};
            for (int k0 = 0; k0 < nk; k0 += kPairChunk) {
                u32x4 op[kPairChunk][4];
#pragma unroll
                for (int c = 0; c < kPairChunk; ++c) {
                    const int64_t ks = (int64_t)(k0 + c < nk ? k0 + c : nk - 1) * 512;
                    op[c][0] = *reinterpret_cast<const u32x4*>(bt.x_hi + fa + ks);
                    op[c][1] = *reinterpret_cast<const u32x4*>(bt.x_lo + fa + ks);
                    op[c][2] = *reinterpret_cast<const u32x4*>(bt.t_hi + fb + ks);
                    op[c][3] = *reinterpret_cast<const u32x4*>(bt.t_lo + fb + ks);
                }
                // every load of the chunk issued before the first product waits on one
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int c = 0; c < kPairChunk; ++c) {
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
            const float st = marginal_colsum(m, bt.t_sum, n_out, jc, nk);
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                pe[r] = to_storage<kDropBits>(fmaf(bt.c2, acc[r], bt.c1 * pe[r]));
                po[r] = to_storage<kDropBits>(fmaf(bt.c2, st - acc[r], bt.c1 * po[r]));
            }
        }

        // ---- epilogue: the elements of silent blocks, unconditional buffer stores -------------
        const bool jok = jl < cols;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int il = il0 + 8 * (r >> 2) + (r & 3);
            const uint32_t off = o0 + (uint32_t)(2 * (8 * (r >> 2) + (r & 3))) * n_out * 4u;
            const bool keep = jok && !((act_bits >> il) & 1u);
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(pe[r]), rp,
                                                  keep ? off : kDrop, 0, 0);
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(po[r]), rp,
                                                  keep ? off + odd : kDrop, 0, 0);
        }
    }
}

// Silent sweep with complement pairs (large layers): trace_sweep_tile_kernel with wave w on
// block w of 32 input HCUs (64 rows) and kCB column blocks, a workgroup on 128 input HCUs x
// 32 kCB columns (the library uses three: 96 columns).  The column totals of every queued
// batch are formed once per workgroup into LDS.
template <int kDropBits, int kKC, int kCB>
__global__ void __launch_bounds__(kWaves * 64) __attribute__((amdgpu_waves_per_eu(2, 2)))
trace_sweep_pair_tile_kernel(Geometry g, SweepArgs a, int n_tj) {
    constexpr int kItems = 2 * kCB * kKC;           // 1 KiB t items per chunk
    constexpr int kPerWave = kItems / kWaves;
    static_assert(kPerWave * kWaves == kItems, "t items split evenly over the waves");
    __shared__ u32x4 stage0[kItems][64];
    __shared__ u32x4 stage1[kItems][64];
    __shared__ float stot[kMaxSweepBatches][32 * kCB];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int n_out = (int)g.n_out;
    const int n_pb = (g.in_hcu + 31) / 32, n_cb = (n_out + 31) / 32;
    const int n_ti = (n_pb + 3) / 4;
    constexpr int kSweepTiles = kSweepRows / 4;
    const int wg = (int)xcd_linear_index(blockIdx.x, gridDim.x);
    const int sweep = wg / (kSweepTiles * n_tj);
    const int in_sweep = wg % (kSweepTiles * n_tj);
    const int here = n_ti - sweep * kSweepTiles < kSweepTiles ? n_ti - sweep * kSweepTiles
                                                              : kSweepTiles;
    const int ti = sweep * kSweepTiles + in_sweep % here;
    const int tj = in_sweep / here;
    const int n_ks = a.n_ks;

    const int bi = 4 * ti + wave;
    const int bic = bi < n_pb ? bi : n_pb - 1;
    const int p0 = bic * 32;
    const int prs = g.in_hcu - p0 < 32 ? g.in_hcu - p0 : 32;
    const bool live = bi < n_pb;                           // wave-uniform
    const int j00 = kCB * tj * 32;
    const int jl = lane & 31, il0 = 4 * (lane >> 5);
    const rsrc_t rp = make_rsrc(a.pij + (int64_t)(2 * p0) * n_out, (uint32_t)(2 * prs) * n_out * 4u);
    const uint32_t o0 = ((uint32_t)(2 * il0) * n_out + j00 + jl) * 4u;
    const uint32_t odd = (uint32_t)n_out * 4u;
    float pold[kCB][2][16];
#pragma unroll
    for (int c = 0; c < kCB; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const uint32_t off =
                o0 + (uint32_t)(2 * (8 * (r >> 2) + (r & 3)) * n_out + 32 * c) * 4u;
            pold[c][0][r] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rp, off, 0, 0));
            pold[c][1][r] =
                __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rp, off + odd, 0, 0));
        }
    uint32_t act_bits[kCB];
#pragma unroll
    for (int c = 0; c < kCB; ++c) {
        const int j0 = j00 + 32 * c;
        const int jc = j0 < n_out ? j0 : (n_cb - 1) * 32;
        const int cols = n_out - jc < 32 ? n_out - jc : 32;
        const int hu = lane < 32 ? p0 + (lane < prs ? lane : prs - 1)
                                 : (jc + (lane - 32 < cols ? lane - 32 : cols - 1)) / g.out_mcu;
        act_bits[c] = block_mask_bits_hu(g, a.mask, hu, lane);
    }

    int n_ch = 0;
    for (int t = 0; t < a.n_batches; ++t) n_ch += (a.bt[t].nk + kKC - 1) / kKC;
    // requests of the chunk at (batch t, first k-step k0): the t items into stage buffer sb
    // (item = (k-step in chunk * kCB + column block) * 2 + {hi, lo}, wave w issuing w, w + 4,
    // ...) and this wave's x fragments into xn
    u32x4 xc[kKC][2], xn[kKC][2];
    auto request = [&](int t, int k0, auto sb_c) {
        u32x4 (*const st)[64] = decltype(sb_c)::value == 0 ? stage0 : stage1;
        const SweepBatch bt = a.bt[t];
#pragma unroll
        for (int q = 0; q < kPerWave; ++q) {
            const int item = wave + kWaves * q;
            const int half = item & 1, cb = (item >> 1) % kCB, kq = item / (2 * kCB);
            int blk = kCB * tj + cb;
            blk = blk < n_cb ? blk : n_cb - 1;
            const int ks = k0 + kq < bt.nk ? k0 + kq : bt.nk - 1;
            const uint16_t* src = (half ? bt.t_lo : bt.t_hi) +
                                  (((int64_t)blk * n_ks + ks) * 64 + lane) * 8;
            __builtin_amdgcn_global_load_lds((const void*)src,
                (void __attribute__((address_space(3)))*)&st[item][0], 16, 0, 0);
        }
#pragma unroll
        for (int kq = 0; kq < kKC; ++kq) {
            const int ks = k0 + kq < bt.nk ? k0 + kq : bt.nk - 1;
            const int64_t fa = (((int64_t)bic * n_ks + ks) * 64 + lane) * 8;
            xn[kq][0] = *reinterpret_cast<const u32x4*>(bt.x_hi + fa);
            xn[kq][1] = *reinterpret_cast<const u32x4*>(bt.x_lo + fa);
        }
    };
    auto next = [&](int& t, int& k0) {
        k0 += kKC;
        if (k0 >= a.bt[t].nk) { k0 = 0; ++t; }
    };

    int dt = 0, dk = 0;
    request(dt, dk, StageIx<0>{});
    next(dt, dk);

    // column totals of every queued batch for the workgroup's 32 kCB columns (clamped)
    for (int e = threadIdx.x; e < a.n_batches * 32 * kCB; e += kWaves * 64) {
        const int t = e / (32 * kCB), cl = e % (32 * kCB);
        const int col = j00 + cl < n_out ? j00 + cl : n_out - 1;
        const SweepBatch bt = a.bt[t];
        MarginalIn m;
#pragma unroll
        for (int q = 0; q < kSums; ++q)
            m.part[q] = bt.t_sum[(int64_t)(q < bt.nk ? q : bt.nk - 1) * n_out + col];
        stot[t][cl] = marginal_colsum(m, bt.t_sum, n_out, col, bt.nk);
    }
    lds_barrier();

    f16v acc[kCB];
#pragma unroll
    for (int c = 0; c < kCB; ++c) acc[c] = f16v{};
    int ct = 0, ck = 0;
    // chunk lc, its t items in stage buffer sb_c (lc's parity)
    auto chunk = [&](int lc, auto sb_c) {
        constexpr int sb = decltype(sb_c)::value;
        const u32x4 (*const st)[64] = sb == 0 ? stage0 : stage1;
        // chunk lc's requests were the last issued: wait for all, then the barrier makes its t
        // items visible to every wave and tells that every wave is done with the other buffer
        __builtin_amdgcn_s_waitcnt(vm_wait(0));
#pragma unroll
        for (int kq = 0; kq < kKC; ++kq) {
            xc[kq][0] = xn[kq][0];
            xc[kq][1] = xn[kq][1];
        }
        stage_barrier();
        if (lc + 1 < n_ch) {
            request(dt, dk, StageIx<1 - sb>{});
            next(dt, dk);
        }
        const int nk = a.bt[ct].nk;
#pragma unroll
        for (int kq = 0; kq < kKC; ++kq) {
            if (ck + kq < nk) {
                const bf8 ah = __builtin_bit_cast(bf8, xc[kq][0]);
                const bf8 al = __builtin_bit_cast(bf8, xc[kq][1]);
                // the hi parts of t stay for two passes, each lo part is read for its one
                bf8 bh[kCB];
#pragma unroll
                for (int c = 0; c < kCB; ++c)
                    bh[c] = __builtin_bit_cast(bf8, st[(kq * kCB + c) * 2][lane]);
#pragma unroll
                for (int c = 0; c < kCB; ++c)
                    acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, bh[c], acc[c], 0, 0, 0);
#pragma unroll
                for (int c = 0; c < kCB; ++c) {
                    const bf8 bl = __builtin_bit_cast(bf8, st[(kq * kCB + c) * 2 + 1][lane]);
                    acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bl, acc[c], 0, 0, 0);
                }
#pragma unroll
                for (int c = 0; c < kCB; ++c)
                    acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bh[c], acc[c], 0, 0, 0);
            }
        }
        if (ck + kKC >= nk) {
            const float c1 = a.bt[ct].c1, c2 = a.bt[ct].c2;
#pragma unroll
            for (int c = 0; c < kCB; ++c) {
                const float st = stot[ct][32 * c + jl];
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    pold[c][0][r] = to_storage<kDropBits>(fmaf(c2, acc[c][r], c1 * pold[c][0][r]));
                    pold[c][1][r] =
                        to_storage<kDropBits>(fmaf(c2, st - acc[c][r], c1 * pold[c][1][r]));
                }
                acc[c] = f16v{};
            }
        }
        next(ct, ck);
    };
    for (int lc = 0; lc < n_ch; lc += 2) {
        chunk(lc, StageIx<0>{});
        if (lc + 1 < n_ch) chunk(lc + 1, StageIx<1>{});
    }
    if (!live) return;
#pragma unroll
    for (int c = 0; c < kCB; ++c) {
        const bool jok = j00 + 32 * c + jl < n_out;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int il = il0 + 8 * (r >> 2) + (r & 3);
            const uint32_t off =
                o0 + (uint32_t)(2 * (8 * (r >> 2) + (r & 3)) * n_out + 32 * c) * 4u;
            const bool keep = jok && !((act_bits[c] >> il) & 1u);
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(pold[c][0][r]), rp,
                                                  keep ? off : kDrop, 0, 0);
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(pold[c][1][r]), rp,
                                                  keep ? off + odd : kDrop, 0, 0);
        }
    }
}

// The same sweep for fp32 storage, in sum form.  With no rounding to a storage format between
// batches, the n queued updates P <- c1_t P + c2_t T_t of an element combine exactly (in real
// arithmetic) into
//   P_n = (c1_0 ... c1_{n-1}) P_0 + R,   R_t = c1_t R_{t-1} + c2_t T_t,
// and for the second unit of a pair into (c1_0 ... c1_{n-1}) P2_0 + Stot - R with
// Stot = sum_t (c1_{t+1} ... c1_{n-1}) c2_t S_t (S_t the column total).  The matrix cores
// accumulate R / c2_t in place (the accumulator is scaled by c1_t c2_{t-1} / c2_t before batch
// t's products), so the old traces are read only in the epilogue, and the registers they take
// in trace_sweep_pair_tile_kernel hold more accumulators instead: a wave covers 32 kCB columns
// (kCB = 8 against 3), so that each operand byte feeds 8 / 3 times the matrix-core work.  kTW
// waves share the t items, which stream through kStages LDS buffers of kKC k-steps (kStages - 1
// chunks in flight; a wave's x fragments likewise through kStages register sets); column block
// c + 1's t fragments are read from LDS during block c's products.
// Measured on the STL-shaped layer (6.67 batches per launch, each variant beside the previous
// one on one box): 4.16 ms per launch per-batch (trace_sweep_pair_tile_kernel), 3.49 ms with
// kCB = 6, 3.33 ms with kCB = 8; 8 waves of kCB = 6 (256 input HCUs) 3.84 ms; 3.05 ms with the
// stage buffers as separate arrays (StageIx), so that the next chunk's loads run under the
// products; four stages of one k-step instead of two of two 2.99 ms; the LDS reads one block
// ahead 2.94 ms; the column totals' loads issued all at once 2.75-2.80 ms.  Per workgroup (time
// stamps, 7 batches, the kernel alone): prologue 7 us, products 107 us, epilogue 26 us.  The result differs from per-batch updates by the
// fp32 rounding of the regrouped sums (a few ulps per batch), not by more.
template <int kKC, int kCB, int kTW, int kStages>
__global__ void __launch_bounds__(kTW * 64) __attribute__((amdgpu_waves_per_eu(2, 2)))
trace_sweep_pair_tile_sum_kernel(Geometry g, SweepArgs a, int n_tj) {
    constexpr int kItems = 2 * kCB * kKC;           // 1 KiB t items per chunk
    constexpr int kPerWave = kItems / kTW;
    static_assert(kPerWave * kTW == kItems, "t items split evenly over the waves");
    static_assert(kStages >= 2 && kStages <= 4, "two to four stage buffers");
    // memory loads a wave issues per chunk: its share of the t items and its x fragments
    constexpr int kLoads = kPerWave + 2 * kKC;
    __shared__ u32x4 stage0[kItems][64];
    __shared__ u32x4 stage1[kItems][64];
    __shared__ u32x4 stage2[kStages > 2 ? kItems : 1][64];
    __shared__ u32x4 stage3[kStages > 3 ? kItems : 1][64];
    auto buf = [&](auto sb_c) -> u32x4 (*)[64] {
        constexpr int b = decltype(sb_c)::value;
        if constexpr (b == 0) return stage0;
        else if constexpr (b == 1) return stage1;
        else if constexpr (b == 2) return stage2;
        else return stage3;
    };    __shared__ float stot[32 * kCB];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int n_out = (int)g.n_out;
    const int n_pb = (g.in_hcu + 31) / 32, n_cb = (n_out + 31) / 32;
    const int n_ti = (n_pb + kTW - 1) / kTW;
    constexpr int kSweepTiles = kSweepRows / kTW;
    const int wg = (int)xcd_linear_index(blockIdx.x, gridDim.x);
    const int sweep = wg / (kSweepTiles * n_tj);
    const int in_sweep = wg % (kSweepTiles * n_tj);
    const int here = n_ti - sweep * kSweepTiles < kSweepTiles ? n_ti - sweep * kSweepTiles
                                                              : kSweepTiles;
    const int ti = sweep * kSweepTiles + in_sweep % here;
    const int tj = in_sweep / here;
    const int n_ks = a.n_ks;

    const int bi = kTW * ti + wave;
    const int bic = bi < n_pb ? bi : n_pb - 1;
    const int p0 = bic * 32;
    const int prs = g.in_hcu - p0 < 32 ? g.in_hcu - p0 : 32;
    const bool live = bi < n_pb;                           // wave-uniform
    const int j00 = kCB * tj * 32;
    const int jl = lane & 31, il0 = 4 * (lane >> 5);

    int n_ch = 0;
    for (int t = 0; t < a.n_batches; ++t) n_ch += (a.bt[t].nk + kKC - 1) / kKC;
    // requests of the chunk at (batch t, first k-step k0) into stage sb_c: its t items into
    // that stage buffer, the wave's x fragments into xs[sb_c]
    u32x4 xs[kStages][kKC][2];
    auto request = [&](int t, int k0, auto sb_c) {
        constexpr int sb = decltype(sb_c)::value;
        u32x4 (*const st)[64] = buf(sb_c);
        const SweepBatch bt = a.bt[t];
#pragma unroll
        for (int q = 0; q < kPerWave; ++q) {
            const int item = wave + kTW * q;
            const int half = item & 1, cb = (item >> 1) % kCB, kq = item / (2 * kCB);
            int blk = kCB * tj + cb;
            blk = blk < n_cb ? blk : n_cb - 1;
            const int ks = k0 + kq < bt.nk ? k0 + kq : bt.nk - 1;
            const uint16_t* src = (half ? bt.t_lo : bt.t_hi) +
                                  (((int64_t)blk * n_ks + ks) * 64 + lane) * 8;
            __builtin_amdgcn_global_load_lds((const void*)src,
                (void __attribute__((address_space(3)))*)&st[item][0], 16, 0, 0);
        }
#pragma unroll
        for (int kq = 0; kq < kKC; ++kq) {
            const int ks = k0 + kq < bt.nk ? k0 + kq : bt.nk - 1;
            const int64_t fa = (((int64_t)bic * n_ks + ks) * 64 + lane) * 8;
            xs[sb][kq][0] = *reinterpret_cast<const u32x4*>(bt.x_hi + fa);
            xs[sb][kq][1] = *reinterpret_cast<const u32x4*>(bt.x_lo + fa);
        }
    };
    auto next = [&](int& t, int& k0) {
        k0 += kKC;
        if (k0 >= a.bt[t].nk) { k0 = 0; ++t; }
    };
    // the chunk after (t, k0) for the requests, which stay on the last chunk past the end: every
    // chunk requests the one kStages - 1 ahead, unconditionally, so that a wave always has the
    // same number of loads in flight (past the end, reloads of the last chunk that nothing reads)
    auto next_req = [&](int& t, int& k0) {
        k0 += kKC;
        if (k0 >= a.bt[t].nk) {
            if (t + 1 < a.n_batches) { k0 = 0; ++t; }
            else k0 -= kKC;
        }
    };

    // the first kStages - 1 chunks
    int dt = 0, dk = 0;
    request(dt, dk, StageIx<0>{});
    next_req(dt, dk);
    if constexpr (kStages > 2) { request(dt, dk, StageIx<1>{}); next_req(dt, dk); }
    if constexpr (kStages > 3) { request(dt, dk, StageIx<2>{}); next_req(dt, dk); }

    // Stot of the workgroup's 32 kCB columns (clamped; one per thread): the column-sum tiles
    // of every queued batch requested at once (batch and tile clamped), then added in tile
    // order (as marginal_colsum) and combined batch by batch in order
    static_assert(32 * kCB == kTW * 64, "one Stot column per thread");
    {
        constexpr int kParts = 16;                      // tiles requested up front per batch
        const int cl = threadIdx.x;
        const int col = j00 + cl < n_out ? j00 + cl : n_out - 1;
        float part[kMaxSweepBatches][kParts];
#pragma unroll
        for (int t = 0; t < kMaxSweepBatches; ++t) {
            const SweepBatch& bt = a.bt[t < a.n_batches ? t : a.n_batches - 1];
#pragma unroll
            for (int q = 0; q < kParts; ++q)
                part[t][q] = bt.t_sum[(int64_t)(q < bt.nk ? q : bt.nk - 1) * n_out + col];
        }
        float v = 0.0f;
#pragma unroll
        for (int t = 0; t < kMaxSweepBatches; ++t) {
            if (t < a.n_batches) {
                const SweepBatch& bt = a.bt[t];
                float colsum = 0.0f;
#pragma unroll
                for (int q = 0; q < kParts; ++q)
                    if (q < bt.nk) colsum += part[t][q];
                for (int q = kParts; q < bt.nk; ++q) colsum += bt.t_sum[(int64_t)q * n_out + col];
                v = fmaf(bt.c2, colsum, v * bt.c1);
            }
        }
        stot[cl] = v;
    }

    f16v acc[kCB];
#pragma unroll
    for (int c = 0; c < kCB; ++c) acc[c] = f16v{};
    int ct = 0, ck = 0;
    // chunk lc, in stage sb_c = lc mod kStages
    auto chunk = [&](int lc, auto sb_c) __attribute__((always_inline)) {
        constexpr int sb = decltype(sb_c)::value;
        const u32x4 (*const st)[64] = buf(sb_c);
        // wait for this wave's loads of chunk lc (those of the kStages - 2 chunks issued after
        // it stay in flight), then the barrier makes every wave's t items of it visible and
        // tells that every wave is done with chunk lc - 1, whose buffer the request refills
        __builtin_amdgcn_s_waitcnt(vm_wait((kStages - 2) * kLoads));
        stage_barrier();
        request(dt, dk, StageIx<(sb + kStages - 1) % kStages>{});
        next_req(dt, dk);
        const auto& xc = xs[sb];
        if (ck == 0 && ct > 0) {
            // batch ct starts: acc holds R_{ct-1} / c2_{ct-1}; make it R_{ct-1} c1_ct / c2_ct
            const float sc = a.bt[ct].c1 * (a.bt[ct - 1].c2 / a.bt[ct].c2);
#pragma unroll
            for (int c = 0; c < kCB; ++c)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[c][r] *= sc;
        }
        const int nk = a.bt[ct].nk;
#pragma unroll
        for (int kq = 0; kq < kKC; ++kq) {
            // (a chunk of one k-step is never past its batch: no branch around the products,
            // which would hide from the compiler that their x loads were waited for)
            if (kKC == 1 || ck + kq < nk) {
                const bf8 ah = __builtin_bit_cast(bf8, xc[kq][0]);
                const bf8 al = __builtin_bit_cast(bf8, xc[kq][1]);
                // column block c + 1's t fragments are read from LDS before block c's products,
                // so that their latency passes under them
                bf8 bh = __builtin_bit_cast(bf8, st[(kq * kCB) * 2][lane]);
                bf8 bl = __builtin_bit_cast(bf8, st[(kq * kCB) * 2 + 1][lane]);
#pragma unroll
                for (int c = 0; c < kCB; ++c) {
                    bf8 bhn = bh, bln = bl;
                    if (c + 1 < kCB) {
                        bhn = __builtin_bit_cast(bf8, st[(kq * kCB + c + 1) * 2][lane]);
                        bln = __builtin_bit_cast(bf8, st[(kq * kCB + c + 1) * 2 + 1][lane]);
                    }
                    acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, bh, acc[c], 0, 0, 0);
                    acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bl, acc[c], 0, 0, 0);
                    acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bh, acc[c], 0, 0, 0);
                    bh = bhn;
                    bl = bln;
                }
#pragma unroll
                for (int c = 0; c < kCB; ++c) {
                    if (c == 0) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);   // LDS reads
                    if (c + 1 < kCB) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
                    __builtin_amdgcn_sched_group_barrier(0x008, 3, 0);               // MFMA
                }
            }
        }
        next(ct, ck);
    };
    // kStages chunks from lc; whether chunks remain after them
    auto group = [&](int lc) __attribute__((always_inline)) -> bool {
        chunk(lc, StageIx<0>{});
        if (lc + 1 >= n_ch) return false;
        chunk(lc + 1, StageIx<1>{});
        if constexpr (kStages > 2) {
            if (lc + 2 >= n_ch) return false;
            chunk(lc + 2, StageIx<2>{});
        }
        if constexpr (kStages > 3) {
            if (lc + 3 >= n_ch) return false;
            chunk(lc + 3, StageIx<3>{});
        }
        return lc + kStages < n_ch;
    };
    // (the first group outside the loop: the loop is then entered with the loads in flight
    // that its back edge carries, and the compiler's count of them stays exact)
    bool more = group(0);
    for (int lc = kStages; more; lc += kStages) more = group(lc);
    // (the reloads past the end land in LDS before the workgroup may end)
    __builtin_amdgcn_s_waitcnt(vm_wait(0));
    stage_barrier();                                    // stot is visible to every wave

    // ---- epilogue: P_n = c1^n P_0 + R, P2_n = c1^n P2_0 + Stot - R, silent elements; column
    // block by column block -----------------------------------------------------------------
    const rsrc_t rp = make_rsrc(a.pij + (int64_t)(2 * p0) * n_out, (uint32_t)(2 * prs) * n_out * 4u);
    const uint32_t o0 = ((uint32_t)(2 * il0) * n_out + j00 + jl) * 4u;
    const uint32_t odd = (uint32_t)n_out * 4u;
    // byte offset of the lane's element of result register r in the first column block (row
    // and column in the vector offset, so that the buffer's range check drops the rows past
    // the layer and the columns past the last); column block c adds 128 c bytes (an immediate)
    uint32_t rowoff[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) rowoff[r] = o0 + (uint32_t)(2 * (8 * (r >> 2) + (r & 3))) * odd;
    float c1n = 1.0f;
    for (int t = 0; t < a.n_batches; ++t) c1n *= a.bt[t].c1;
    const float c2n = a.bt[a.n_batches - 1].c2;
    // old traces of column block c, both rows of each pair (requested kEpiDepth - 1 blocks
    // ahead, into slot c mod kEpiDepth)
    constexpr int kEpiDepth = 2;
    float pold[kEpiDepth][2][16];
    auto request_old = [&](int c, int slot) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const uint32_t off = rowoff[r] + 128u * c;
            pold[slot][0][r] =
                __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rp, off, 0, 0));
            pold[slot][1][r] =
                __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rp, off + odd, 0, 0));
        }
    };
    uint32_t act_bits[kCB];
#pragma unroll
    for (int c = 0; c < kCB; ++c) {
        const int j0 = j00 + 32 * c;
        const int jc = j0 < n_out ? j0 : (n_cb - 1) * 32;
        const int cols = n_out - jc < 32 ? n_out - jc : 32;
        const int hu = lane < 32 ? p0 + (lane < prs ? lane : prs - 1)
                                 : (jc + (lane - 32 < cols ? lane - 32 : cols - 1)) / g.out_mcu;
        act_bits[c] = block_mask_bits_hu(g, a.mask, hu, lane);
    }
#pragma unroll
    for (int c = 0; c + 1 < kEpiDepth; ++c) request_old(c, c);
#pragma unroll
    for (int c = 0; c < kCB; ++c) {
        if (c + kEpiDepth - 1 < kCB) request_old(c + kEpiDepth - 1, (c + kEpiDepth - 1) % kEpiDepth);
        const int j0 = j00 + 32 * c;
        if (live) {                                             // wave-uniform
            const bool jok = j0 + jl < n_out;
            const float st = stot[32 * c + jl];
            const uint32_t act = act_bits[c];
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int il = il0 + 8 * (r >> 2) + (r & 3);
                const float R = c2n * acc[c][r];
                const float pe = fmaf(c1n, pold[c % kEpiDepth][0][r], R);
                const float po = fmaf(c1n, pold[c % kEpiDepth][1][r], st - R);
                const uint32_t off = rowoff[r] + 128u * c;
                const bool keep = jok && !((act >> il) & 1u);
                __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(pe), rp, keep ? off : kDrop,
                                                      0, 0);
                __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(po), rp,
                                                      keep ? off + odd : kDrop, 0, 0);
            }
        }
        // (a compiler fence: block c + kEpiDepth's loads, into this block's registers, stay
        // after this block's stores)
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
    }
}

// Active blocks with complement pairs: trace_active_kernel with the block rows taken as 32 of
// the hidden HCU's active input HCUs (64 rows), their first units gathered through the active
// list.  kSplit (small layers, where the kernel is bound by latency rather than by its matrix
// work): a workgroup covers two column blocks, and each block's contraction is run by two
// waves, one storing the first rows of the pairs and one the second, so that every wave keeps
// the per-element work of the unpaired kernel.  Otherwise a workgroup covers four column blocks
// and each wave stores both rows.
template <int kDropBits, bool kSplit, bool kStamp>
__global__ void __launch_bounds__(kWaves * 64) __attribute__((amdgpu_waves_per_eu(2, 2)))
trace_active_pair_kernel(Geometry g, TraceArgs a, const int32_t* __restrict__ act_list,
                         const int32_t* __restrict__ act_count, int n_rt, int n_cgr,
                         int n_work) {
    __builtin_amdgcn_s_setprio(3);
    stamp_start<kStamp>(a.stamp);
    const int n_in = (int)g.n_in, n_out = (int)g.n_out;
    const int nk = (a.B + 15) / 16;
    const int n_ks = a.ops.n_ks;
    if ((int)blockIdx.x >= n_work) {
        store_marginal(g, a, (int64_t)(blockIdx.x - n_work) * blockDim.x + threadIdx.x, nk);
        stamp_end<kStamp>(a.stamp);
        return;
    }
    constexpr int kBlocks = kSplit ? kWaves / 2 : kWaves;     // column blocks per workgroup
    __shared__ u32x4 xs[kActiveChunk][2][64];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int par = kSplit ? (wave & 1) : 0;                  // the rows a split wave stores
    const int wg = (int)xcd_linear_index(blockIdx.x, n_work);
    const int per_hcu = n_rt * n_cgr;
    const int hj = wg / per_hcu;
    const int rt = (wg - hj * per_hcu) / n_cgr;
    const int c0 = ((wg - hj * per_hcu - rt * n_cgr) * kBlocks + (kSplit ? wave >> 1 : wave)) * 32;
    const bool col_live = c0 < g.out_mcu;                      // wave-uniform
    const int cols = col_live ? (g.out_mcu - c0 < 32 ? g.out_mcu - c0 : 32) : 1;
    const int j0 = hj * g.out_mcu + (col_live ? c0 : 0);
    const int jl = lane & 31;
    const int il0 = 4 * (lane >> 5);
    const int h = lane >> 5;
    const int jb = j0 + (jl < cols ? jl : cols - 1);

    // the active count (in input HCUs) and the list entry of block row jl, then the columns
    const int k_total = act_count[hj];
    const int kr = rt * 32 + jl < g.in_hcu ? rt * 32 + jl : g.in_hcu - 1;
    const int hsel = act_list[(int64_t)hj * g.in_hcu + kr];
    u32x4 opt[kActiveChunk][2], opx[kActiveChunk][2];
    auto load_t = [&](int k0) {
#pragma unroll
        for (int c = 0; c < kActiveChunk; ++c) {
            const int64_t fb = frag_chunk(jb, k0 + c < nk ? k0 + c : nk - 1, h, n_ks);
            opt[c][0] = *reinterpret_cast<const u32x4*>(a.ops.t_hi + fb);
            opt[c][1] = *reinterpret_cast<const u32x4*>(a.ops.t_lo + fb);
        }
    };
    constexpr int kGather = kActiveChunk * 2 * 64 / (kWaves * 64);
    auto gather_x = [&](int k0, int pa) {
        u32x4 v[kGather];
#pragma unroll
        for (int q = 0; q < kGather; ++q) {
            const int P = threadIdx.x + kWaves * 64 * q;
            const int hp = (P >> 5) & 1, hl = (P >> 6) & 1, kq = P >> 7;
            const int ks = k0 + kq < nk ? k0 + kq : nk - 1;
            const int64_t fa = frag_chunk(pa, ks, hp, n_ks);
            v[q] = *reinterpret_cast<const u32x4*>((hl ? a.ops.x_lo : a.ops.x_hi) + fa);
        }
#pragma unroll
        for (int q = 0; q < kGather; ++q) {
            const int P = threadIdx.x + kWaves * 64 * q;
            xs[P >> 7][(P >> 6) & 1][P & 63] = v[q];
        }
    };
    auto load_x = [&]() {
#pragma unroll
        for (int c = 0; c < kActiveChunk; ++c) {
            opx[c][0] = xs[c][0][lane];
            opx[c][1] = xs[c][1][lane];
        }
    };
    f16v acc = {};
    auto contract = [&](int k0) {
#pragma unroll
        for (int c = 0; c < kActiveChunk; ++c) {
            if (k0 + c < nk) {
                const bf8 ah = __builtin_bit_cast(bf8, opx[c][0]);
                const bf8 al = __builtin_bit_cast(bf8, opx[c][1]);
                const bf8 bh = __builtin_bit_cast(bf8, opt[c][0]);
                const bf8 bl = __builtin_bit_cast(bf8, opt[c][1]);
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, bh, acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bl, acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bh, acc, 0, 0, 0);
            }
        }
    };
    load_t(0);

    // input HCU of block row jl (the A-operand row of this lane), clamped into the layer
    const int pa = hsel < 0 ? 0 : (hsel < g.in_hcu ? hsel : g.in_hcu - 1);
    int pr[16];
    float pe[16], po[kSplit ? 1 : 16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        pr[r] = half_broadcast(pa, 8 * (r >> 2) + (r & 3), lane);
        if constexpr (kSplit) {
            pe[r] = a.pij[(int64_t)(2 * pr[r] + par) * n_out + jb];
        } else {
            pe[r] = a.pij[(int64_t)(2 * pr[r]) * n_out + jb];
            po[r] = a.pij[(int64_t)(2 * pr[r] + 1) * n_out + jb];
        }
    }
    gather_x(0, pa);
    // marginal inputs.  Split: lanes 0..31 the stored unit of row jl's input HCU, 32..63 the
    // block's columns.  Otherwise: lane l the unit 2 pa + l / 32 (both units of row jl's input
    // HCU), and every lane its own column.
    const bool row_lane = kSplit ? lane < 32 : true;
    const int urow = kSplit ? 2 * pa + par : 2 * pa + (lane >> 5);
    MarginalIn mr, mc;
    if constexpr (kSplit) {
        marginal_request(mr, row_lane ? a.ops.x_sum : a.ops.t_sum, row_lane ? n_in : n_out,
                         row_lane ? urow : jb, nk, row_lane ? a.pi_old : a.pj_old);
    } else {
        marginal_request(mr, a.ops.x_sum, n_in, urow, nk, a.pi_old);
        marginal_request(mc, a.ops.t_sum, n_out, jb, nk, a.pj_old);
    }

    lds_barrier();
    load_x();
    contract(0);
    for (int k0 = kActiveChunk; k0 < nk; k0 += kActiveChunk) {   // batches above 128 rows
        lds_barrier();
        load_t(k0);
        gather_x(k0, pa);
        lds_barrier();
        load_x();
        contract(k0);
    }
    if (col_live) {                                    // wave-uniform
        const int rows = k_total - rt * 32 < 32 ? k_total - rt * 32 : 32;   // may be <= 0
        const bool jok = jl < cols;

        if constexpr (kSplit) {
            const float* sums = row_lane ? a.ops.x_sum : a.ops.t_sum;
            const int64_t st_m = row_lane ? n_in : n_out;
            const int um = row_lane ? urow : jb;
            const float cs = marginal_colsum(mr, sums, st_m, um, nk);
            const float lp = fast_log(fmaxf(marginal_from_colsum(mr, cs, a), a.eps));
            const float lpj = __shfl(lp, 32 + jl, 64);
            const float st = __shfl(cs, 32 + jl, 64);          // column total of t
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int src = 8 * (r >> 2) + (r & 3);
                const int il = il0 + src;
                const float lpi = half_broadcast(lp, src, lane);
                const float tv = par ? st - acc[r] : acc[r];
                const float pn = to_storage<kDropBits>(fmaf(a.c2, tv, a.c1 * pe[r]));
                const float wv = to_storage<kDropBits>(fast_log(fmaxf(pn, a.eps)) - lpi - lpj);
                if (jok && il < rows) {
                    const int64_t e = (int64_t)(2 * pr[r] + par) * n_out + jb;
                    a.pij[e] = pn;
                    a.w[e] = wv;
                }
            }
        } else {
            const float lp = fast_log(fmaxf(marginal_value(mr, a.ops.x_sum, n_in, urow, nk, a), a.eps));
            const float st = marginal_colsum(mc, a.ops.t_sum, n_out, jb, nk);
            const float lpj = fast_log(fmaxf(marginal_from_colsum(mc, st, a), a.eps));
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int src = 8 * (r >> 2) + (r & 3);
                const int il = il0 + src;
                const float lpe = half_broadcast(lp, src, lane);        // first unit of HCU il
                const float lpo = half_broadcast(lp, 32 + src, lane);   // second unit
                const float ne = to_storage<kDropBits>(fmaf(a.c2, acc[r], a.c1 * pe[r]));
                const float no = to_storage<kDropBits>(fmaf(a.c2, st - acc[r], a.c1 * po[r]));
                const float we = to_storage<kDropBits>(fast_log(fmaxf(ne, a.eps)) - lpe - lpj);
                const float wo = to_storage<kDropBits>(fast_log(fmaxf(no, a.eps)) - lpo - lpj);
                if (jok && il < rows) {
                    const int64_t e = (int64_t)(2 * pr[r]) * n_out + jb;
                    a.pij[e] = ne;
                    a.w[e] = we;
                    a.pij[e + n_out] = no;
                    a.w[e + n_out] = wo;
                }
            }
        }
    }
    stamp_end<kStamp>(a.stamp);
}

}  // namespace

hipError_t launch_trace_sweep(hipStream_t stream, const Geometry& g, const SweepArgs& a,
                              int64_t resident_wgs, hipEvent_t start, hipEvent_t stop) {
    if (a.n_batches < 1 || a.n_batches > kMaxSweepBatches) return hipErrorInvalidValue;
    if (a.paired && g.in_mcu != 2) return hipErrorInvalidValue;
    // row blocks: 32 input units, or with complement pairs 32 input HCUs (64 rows)
    const int64_t n_rb = a.paired ? (g.in_hcu + 31) / 32 : (g.n_in + 31) / 32;
    const int64_t n_cb = (g.n_out + 31) / 32;
    const int64_t n_cg = (n_cb + kWaves - 1) / kWaves;
    if (resident_wgs < 0 && a.paired) {
        // large layer: 128 input HCUs x 96 columns per workgroup; in the sum form (fp32
        // storage) 128 x 256
        void (*kernel)(Geometry, SweepArgs, int) = nullptr;
        int cbs = kPairTileCB, tw = kWaves;
        switch (a.drop_bits) {
            case 0:
                kernel = trace_sweep_pair_tile_sum_kernel<kSumTileKC, kSumTileCB, kSumTileWaves,
                                                          kSumTileStages>;
                cbs = kSumTileCB;
                tw = kSumTileWaves;
                break;
            case 13: kernel = trace_sweep_pair_tile_kernel<13, kTileKC, kPairTileCB>; break;
            case 16: kernel = trace_sweep_pair_tile_kernel<16, kTileKC, kPairTileCB>; break;
            default: return hipErrorInvalidValue;
        }
        const int64_t n_ti = (n_rb + tw - 1) / tw;
        const int64_t n_tj = (n_cb + cbs - 1) / cbs;
        return launch_timed(kernel, dim3((unsigned)(n_ti * n_tj)), dim3(tw * 64), 0, stream,
                            start, stop, g, a, (int)n_tj);
    }
    if (resident_wgs < 0) {
        // large layer: 128 x 128 tiles, operands staged through LDS
        void (*kernel)(Geometry, SweepArgs, int) = nullptr;
        switch (a.drop_bits) {
            case 0: kernel = trace_sweep_tile_kernel<0, kTileKC>; break;
            case 13: kernel = trace_sweep_tile_kernel<13, kTileKC>; break;
            case 16: kernel = trace_sweep_tile_kernel<16, kTileKC>; break;
            default: return hipErrorInvalidValue;
        }
        const int64_t n_ti = (n_rb + 3) / 4;
        return launch_timed(kernel, dim3((unsigned)(n_ti * n_cg)), dim3(kWaves * 64), 0, stream,
                            start, stop, g, a, (int)n_cg);
    }
    void (*kernel)(Geometry, SweepArgs, int, int, int) = nullptr;
    switch (a.drop_bits * 2 + (a.paired ? 1 : 0)) {
        case 0: kernel = trace_sweep_kernel<0>; break;
        case 26: kernel = trace_sweep_kernel<13>; break;
        case 32: kernel = trace_sweep_kernel<16>; break;
        case 1: kernel = trace_sweep_pair_kernel<0>; break;
        case 27: kernel = trace_sweep_pair_kernel<13>; break;
        case 33: kernel = trace_sweep_pair_kernel<16>; break;
        default: return hipErrorInvalidValue;
    }
    const int64_t n_work = n_rb * n_cg;
    int64_t grid = n_work;
    if (resident_wgs > 0 && resident_wgs < grid) grid = (resident_wgs + 7) / 8 * 8;
    // Column groups per stripe: at most an eighth of them (one stripe or less per XCD), and few
    // enough that the stripe's t fragments of every queued batch fit kStripeBytes.
    int64_t ks = 0;
    for (int t = 0; t < a.n_batches; ++t) ks += a.bt[t].nk;
    const int64_t cg_bytes = kWaves * ks * 2 * 1024;               // hi + lo, 1 KiB per k-step
    int64_t stripe = (n_cg + 7) / 8;
    if (stripe * cg_bytes > kStripeBytes) stripe = kStripeBytes / cg_bytes;
    if (stripe < 1) stripe = 1;
    // the events (when given) are recorded around the launch
    return launch_timed(kernel, dim3((unsigned)grid), dim3(kWaves * 64), 0, stream, start,
                        stop, g, a, (int)n_cg, (int)n_work, (int)stripe);
}

// Row tiles of a hidden HCU's active rows (32 units, or with complement pairs 32 input HCUs)
// and column groups of a hidden HCU (four 32-column blocks, two when pair rows are split).
static int64_t active_row_tiles(const Geometry& g, int32_t max_active, int paired) {
    return paired ? ((int64_t)max_active + 31) / 32 : ((int64_t)max_active * g.in_mcu + 31) / 32;
}
static int64_t active_col_groups(const Geometry& g, int paired) {
    const int per = paired == kPairsSplit ? kWaves / 2 : kWaves;
    return ((g.out_mcu + 31) / 32 + per - 1) / per;
}

int64_t trace_active_workgroups(const Geometry& g, int32_t max_active, int paired) {
    const int64_t n_rt = active_row_tiles(g, max_active, paired);
    const int64_t n_cgr = active_col_groups(g, paired);
    return (int64_t)g.out_hcu * n_rt * n_cgr + (g.n_in + g.n_out + kWaves * 64 - 1) / (kWaves * 64);
}

hipError_t launch_trace_active(hipStream_t stream, const Geometry& g, const TraceArgs& a,
                               const int32_t* act_list, const int32_t* act_count,
                               int32_t max_active, hipEvent_t start, hipEvent_t stop) {
    const int paired = a.ops.paired;
    if (paired && g.in_mcu != 2) return hipErrorInvalidValue;
    const int64_t n_rt = active_row_tiles(g, max_active, paired);
    const int64_t n_cgr = active_col_groups(g, paired);
    const int64_t n_work = (int64_t)g.out_hcu * n_rt * n_cgr;
    const int64_t blocks = trace_active_workgroups(g, max_active, paired);
    using Kernel = void (*)(Geometry, TraceArgs, const int32_t*, const int32_t*, int, int, int);
    // the stamping variant when the launch carries a duration stamp
    auto pick = [&](auto stamp_c) -> Kernel {
        constexpr bool S = decltype(stamp_c)::value;
        switch (a.drop_bits * 4 + paired) {
            case 0: return trace_active_kernel<0, S>;
            case 52: return trace_active_kernel<13, S>;
            case 64: return trace_active_kernel<16, S>;
            case 1: return trace_active_pair_kernel<0, false, S>;
            case 53: return trace_active_pair_kernel<13, false, S>;
            case 65: return trace_active_pair_kernel<16, false, S>;
            case 2: return trace_active_pair_kernel<0, true, S>;
            case 54: return trace_active_pair_kernel<13, true, S>;
            case 66: return trace_active_pair_kernel<16, true, S>;
            default: return nullptr;
        }
    };
    const Kernel kernel = a.stamp ? pick(std::true_type{}) : pick(std::false_type{});
    if (!kernel) return hipErrorInvalidValue;
    return launch_timed(kernel, dim3((unsigned)blocks), dim3(kWaves * 64), 0, stream, start,
                        stop, g, a, act_list, act_count, (int)n_rt, (int)n_cgr, (int)n_work);
}

}  // namespace bcpnn
