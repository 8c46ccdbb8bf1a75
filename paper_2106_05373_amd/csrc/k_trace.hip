// Joint-trace contraction with the fused trace, weight and bias updates (Alg. 1 cycle loop):
//
//   T[i][j]  = sum_b x[b][i] t[b][j]                       (the batch sum of a_i (x) a_j)
//   Pij     <- c1 Pij + c2 T[i][j]                         c1 = 1 - a_eff, c2 = a_eff / B
//   Pi, Pj  <- c1 P + a_eff mean_b(.)                      (redundantly per tile, see below)
//   w[i][j]  = log max(Pij,eps) - log max(Pi,eps) - log max(Pj,eps)   on active blocks only
//   b[j]     = k_B log max(Pj, eps)
//
// a_eff = 1 - (1 - alpha)^n_cycles folds the paper's n_cycles repetitions with the same batch
// means into one update (exact in real arithmetic).
//
// Design (gfx950):
//  * T is a dense [N_in x N_out] product with K = B (the batch).  Every Pij is needed (silent
//    connections are scored for plasticity), so the contraction is dense.
//  * T runs on the bf16 matrix cores with a two-term split of both operands: v = hi + lo with
//    hi = bf16(v), lo = bf16(v - hi), and T ~ lo.hi' + hi.lo' + hi.hi' (three
//    v_mfma_f32_32x32x16_bf16, fp32 accumulation).  Each product is then exact to about 3
//    parts in 2^17 (the dropped lo.lo' term and the rounding of lo), so T carries a relative
//    error of order 1e-5; the trace update scales it by a_eff / B, which puts it near 1e-8 in
//    Pij.  Three bf16 MFMAs cost 3/16 of the fp32 MFMA time of the same product, so the kernel
//    is bound by the Pij traffic: 8 bytes per element plus 4 per active weight.
//  * The support kernel of the same batch has already written x^T and t^T split and
//    transposed ([unit][batch] bf16, the MFMA operand order) and the column sums of x and t
//    per 16-row tile.
//  * Tiles of 64 x 64 Pij elements; each of a workgroup's four waves owns one 32 x 32 block.
//    The grid is persistent (three workgroups per CU); workgroup b walks a contiguous run of
//    tiles (i fastest), and the runs are handed out so that the workgroups of one XCD cover
//    one contiguous stretch of tiles, whose operand panels then stay in that XCD's L2.
//  * Work is cut into passes of up to 64 batch rows.  Vector-memory operations complete in
//    issue order, so each pass first requests what the next one needs (before a tile's last
//    pass: the next tile's Pij values, mask block, column sums and old Pi / Pj; then the next
//    operand panels, into registers), and only then runs its own MFMAs and, after a tile's
//    last pass, the epilogue.  The epilogue's 32 stores per lane are unconditional buffer
//    stores (a store that must not happen gets an offset past the buffer's range, which the
//    hardware drops), so the wait for the next panels after the epilogue can leave those
//    stores in flight.  Between tiles, the marginal traces, their logs, the HCU tables and
//    the mask block of the next tile go to LDS as soon as its requests have landed, which
//    leaves the epilogue free of memory waits.
//  * No load needs a branch: Pij values and operand panels are buffer loads over the tile's
//    rows (rows past the layer read as zero), the other indexes are clamped into the tile, and
//    out-of-range lanes read values that only feed results which are dropped.
//  * In LDS each 128-byte operand row (64 bf16) holds eight 16-byte groups, group g of row r at
//    slot g ^ ((r / 2) % 8): the 16 lanes of one phase of a 128-bit operand read (16
//    consecutive rows at one group) spread over all 64 banks.
//  * Every tile computes the new Pi / Pj of its rows / columns itself from the column sums
//    (same code, same order, hence identical values); the tiles of the first column / row store
//    them.  Pi and Pj are read from one buffer and written to another (the host alternates
//    them), so no workgroup reads an updated value.
//
// MFMA 32x32x16 bf16 lane layout (verified on gfx950): A[i][k] for k = 8 (l / 32) + 0..7 from
// lane l = i + 32 (k / 8), B[k][j] likewise with j = l % 32, and lane l holds
// D[8 (r / 4) + 4 (l / 32) + r % 4][l % 32] in result register r.
#include <hip/hip_ext.h>

#include "bcpnn_internal.h"
#include "device_common.h"

namespace bcpnn {
namespace {

typedef float f16v __attribute__((ext_vector_type(16)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef int32_t i4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __amdgpu_buffer_rsrc_t rsrc_t;

constexpr int kTM = 64;            // Pij rows (input units) per tile
constexpr int kTN = 64;            // Pij columns (hidden units) per tile
constexpr int kThreads = 256;
constexpr int kPass = 64;          // batch rows per pass (one 128-byte bf16 row per unit)
constexpr int kGroups = kPass / 8; // 16-byte groups per operand row
constexpr int kSums = 8;           // column-sum tiles requested ahead (the batch for B <= 128)
constexpr int kMaskRegs = 2;       // mask bytes per thread requested ahead (512 per tile)
constexpr int kMaskMax = kTM * kTN;                // HCU blocks a tile can touch (MCU counts 1)
constexpr int kStage = kTM * kGroups / kThreads;   // staged 16-byte groups per operand half
constexpr uint32_t kDrop = 0x80000000u;            // byte offset past every tile's buffer range

__device__ __forceinline__ int slot(int r, int g) { return g ^ ((r >> 1) & 7); }

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

template <int kDropBits>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(3, 3)))
trace_kernel(Geometry g, TraceArgs a, int n_tiles) {
    __shared__ u32x4 pan[4][kTM][kGroups];    // x hi, x lo, t hi, t lo
    __shared__ f4 lpi_t[kTM / 4];             // log(max(Pi, eps)) of the tile's rows
    __shared__ float lpj_t[kTN];              // log(max(Pj, eps)) of its columns
    __shared__ i4 row_h[kTM / 4];             // input HCU of each row, relative to the tile's first
    __shared__ int32_t col_h[kTN];            // hidden HCU of each column, likewise
    __shared__ uint8_t mtile[kMaskMax];       // mask block [row HCU][column HCU]

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int n_in = (int)g.n_in, n_out = (int)g.n_out;
    const int in_mcu = g.in_mcu, out_mcu = g.out_mcu, out_hcu = g.out_hcu;
    const int kp = a.ops.kp;
    const int n_it = (n_in + kTM - 1) / kTM;
    const int kc = (a.B + 31) / 32 * 32;                  // rows B .. kc - 1 are zero
    const int n_pass = (kc + kPass - 1) / kPass;
    const int n_rt = (a.B + 15) / 16;

    // This workgroup's contiguous run of tiles (XCD-major order of the runs).
    const int64_t run = xcd_linear_index(blockIdx.x, gridDim.x);
    const int t_begin = (int)((int64_t)n_tiles * run / gridDim.x);
    const int t_end = (int)((int64_t)n_tiles * (run + 1) / gridDim.x);
    if (t_begin >= t_end) return;

    // lane geometry inside a tile
    const int jl = wn * 32 + (lane & 31);
    const int il0 = wm * 32 + 4 * (lane >> 5);
    const bool is_row = tid < kTM, is_col = tid >= kTM && tid < kTM + kTN;
    const int ss = tid & 7;                  // staging: rows (tid / 8) + 32 q, LDS slot tid % 8
    // byte offset of this thread's first staged group inside a panel (pass 0)
    const uint32_t stage_off =
        (uint32_t)(((tid >> 3) * kp + 8 * slot(tid >> 3, ss)) * 2);
    const uint32_t stage_step = (uint32_t)(32 * kp * 2);          // rows + 32

    u32x4 stg[4][kStage];
    float n_pold[16], c_pold[16];
    float n_part[kSums];
    float n_pod;
    uint32_t n_mb[kMaskRegs];

    // ---- requests (macros over register arrays: nothing may take their address) ----------
    // Operand panels of pass pass_ of tile (ti_, tj_): rows past the layer read as zero.
#define BCPNN_REQUEST_PANELS(ti_, tj_, pass_)                                                  \
    {                                                                                          \
        const int i0_ = (ti_) * kTM, j0_ = (tj_) * kTN;                                        \
        const uint32_t ra_ = (uint32_t)(n_in - i0_ < kTM ? n_in - i0_ : kTM) * kp * 2u;        \
        const uint32_t rb_ = (uint32_t)(n_out - j0_ < kTN ? n_out - j0_ : kTN) * kp * 2u;      \
        const rsrc_t xh_ = make_rsrc(a.ops.x_hi + (int64_t)i0_ * kp, ra_);                     \
        const rsrc_t xl_ = make_rsrc(a.ops.x_lo + (int64_t)i0_ * kp, ra_);                     \
        const rsrc_t th_ = make_rsrc(a.ops.t_hi + (int64_t)j0_ * kp, rb_);                     \
        const rsrc_t tl_ = make_rsrc(a.ops.t_lo + (int64_t)j0_ * kp, rb_);                     \
        const uint32_t o_ = stage_off + (uint32_t)((pass_) * kPass * 2);                       \
        _Pragma("unroll") for (int q = 0; q < kStage; ++q) {                                   \
            stg[0][q] = __builtin_amdgcn_raw_buffer_load_b128(xh_, o_ + q * stage_step, 0, 0); \
            stg[1][q] = __builtin_amdgcn_raw_buffer_load_b128(xl_, o_ + q * stage_step, 0, 0); \
            stg[2][q] = __builtin_amdgcn_raw_buffer_load_b128(th_, o_ + q * stage_step, 0, 0); \
            stg[3][q] = __builtin_amdgcn_raw_buffer_load_b128(tl_, o_ + q * stage_step, 0, 0); \
        }                                                                                      \
    }
    // Pij values of the lane, column sums and old Pi / Pj (threads 0..127), mask bytes.
#define BCPNN_REQUEST_TILE(ti_, tj_)                                                           \
    {                                                                                          \
        const int i0_ = (ti_) * kTM, j0_ = (tj_) * kTN;                                        \
        const int rows_ = n_in - i0_ < kTM ? n_in - i0_ : kTM;                                 \
        const int cols_ = n_out - j0_ < kTN ? n_out - j0_ : kTN;                               \
        const rsrc_t rp_ = make_rsrc(a.pij + (int64_t)i0_ * n_out, (uint32_t)rows_ * n_out * 4u); \
        const uint32_t o_ = ((uint32_t)il0 * n_out + j0_ + jl) * 4u;                           \
        _Pragma("unroll") for (int r = 0; r < 16; ++r)                                         \
            n_pold[r] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(                  \
                rp_, o_ + (uint32_t)(8 * (r >> 2) + (r & 3)) * n_out * 4u, 0, 0));            \
        if (is_row || is_col) {                                                                \
            const int u_ = is_row ? i0_ + (tid < rows_ ? tid : rows_ - 1)                      \
                                  : j0_ + (tid - kTM < cols_ ? tid - kTM : cols_ - 1);         \
            const float* sums_ = is_row ? a.ops.x_sum : a.ops.t_sum;                           \
            const int64_t st_ = is_row ? n_in : n_out;                                         \
            _Pragma("unroll") for (int q = 0; q < kSums; ++q)                                  \
                n_part[q] = sums_[(q < n_rt ? q : n_rt - 1) * st_ + u_];                       \
            n_pod = is_row ? a.pi_old[u_] : a.pj_old[u_];                                      \
        }                                                                                      \
        const int hi0_ = i0_ / in_mcu, hj0_ = j0_ / out_mcu;                                   \
        const int nhj_ = (j0_ + cols_ - 1) / out_mcu - hj0_ + 1;                               \
        const int nm_ = ((i0_ + rows_ - 1) / in_mcu - hi0_ + 1) * nhj_;                        \
        _Pragma("unroll") for (int q = 0; q < kMaskRegs; ++q) {                                \
            const int e = tid + q * kThreads < nm_ ? tid + q * kThreads : nm_ - 1;             \
            n_mb[q] = a.mask[(int64_t)(hi0_ + e / nhj_) * out_hcu + hj0_ + e % nhj_];          \
        }                                                                                      \
    }
#define BCPNN_STAGE()                                                                          \
    {                                                                                          \
        _Pragma("unroll") for (int q = 0; q < kStage; ++q) {                                   \
            const int r = (tid >> 3) + 32 * q;                                                 \
            pan[0][r][ss] = stg[0][q];                                                         \
            pan[1][r][ss] = stg[1][q];                                                         \
            pan[2][r][ss] = stg[2][q];                                                         \
            pan[3][r][ss] = stg[3][q];                                                         \
        }                                                                                      \
    }
    // Switch to tile (ti_, tj_) once its requests have landed: Pij values into c_pold, and the
    // tile's row / column HCU tables, mask block and new marginal traces (with their logs) into
    // LDS; the tiles of the first column / row store the new Pi / Pj and the bias.
#define BCPNN_NEW_TILE(ti_, tj_)                                                               \
    {                                                                                          \
        _Pragma("unroll") for (int r = 0; r < 16; ++r) {                                       \
            c_pold[r] = n_pold[r];                                                             \
            acc[r] = 0.0f;                                                                     \
        }                                                                                      \
        const int i0_ = (ti_) * kTM, j0_ = (tj_) * kTN;                                        \
        const int rows_ = n_in - i0_ < kTM ? n_in - i0_ : kTM;                                 \
        const int cols_ = n_out - j0_ < kTN ? n_out - j0_ : kTN;                               \
        const int hi0_ = i0_ / in_mcu, hj0_ = j0_ / out_mcu;                                   \
        const int nhj_ = (j0_ + cols_ - 1) / out_mcu - hj0_ + 1;                               \
        const int nm_ = ((i0_ + rows_ - 1) / in_mcu - hi0_ + 1) * nhj_;                        \
        _Pragma("unroll") for (int q = 0; q < kMaskRegs; ++q)                                  \
            if (tid + q * kThreads < nm_) mtile[tid + q * kThreads] = (uint8_t)n_mb[q];        \
        for (int e = tid + kMaskRegs * kThreads; e < nm_; e += kThreads) /* small MCU counts */ \
            mtile[e] = a.mask[(int64_t)(hi0_ + e / nhj_) * out_hcu + hj0_ + e % nhj_];         \
        if (is_row)                                                                            \
            reinterpret_cast<int32_t*>(row_h)[tid] =                                           \
                (i0_ + (tid < rows_ ? tid : rows_ - 1)) / in_mcu - hi0_;                       \
        else if (is_col)                                                                       \
            col_h[tid - kTM] = (j0_ + (tid - kTM < cols_ ? tid - kTM : cols_ - 1)) / out_mcu - hj0_; \
        if ((is_row && tid < rows_) || (is_col && tid - kTM < cols_)) {                        \
            const int unit_ = is_row ? i0_ + tid : j0_ + (tid - kTM);                          \
            float colsum_ = 0.0f;                                                              \
            _Pragma("unroll") for (int q = 0; q < kSums; ++q)                                  \
                if (q < n_rt) colsum_ += n_part[q];                                            \
            const float* sums_ = is_row ? a.ops.x_sum : a.ops.t_sum;                           \
            const int64_t st_ = is_row ? n_in : n_out;                                         \
            for (int q = kSums; q < n_rt; ++q) colsum_ += sums_[q * st_ + unit_];              \
            const float p_ = fmaf(a.a_eff, colsum_ * a.inv_b, a.c1 * n_pod);                   \
            const float lp_ = fast_log(fmaxf(p_, a.eps));                                        \
            if (is_row) {                                                                      \
                reinterpret_cast<float*>(lpi_t)[tid] = lp_;                                    \
                if (j0_ == 0) a.pi_new[unit_] = p_;                                            \
            } else {                                                                           \
                lpj_t[tid - kTM] = lp_;                                                        \
                if (i0_ == 0) {                                                                \
                    a.pj_new[unit_] = p_;                                                      \
                    a.b[unit_] = a.bias_gain * lp_;                                            \
                }                                                                              \
            }                                                                                  \
        }                                                                                      \
    }
#define BCPNN_CONTRACT(pass_)                                                                  \
    {                                                                                          \
        const int k0_ = (pass_) * kPass;                                                       \
        const int gp_ = (kc - k0_ < kPass ? kc - k0_ : kPass) / 8;                             \
        const int ar_ = wm * 32 + (lane & 31), br_ = wn * 32 + (lane & 31);                    \
        for (int g2 = 0; g2 < gp_; g2 += 2) {            /* k-steps of 16 rows */              \
            const int gq = g2 + (lane >> 5);                                                   \
            const bf8 ah = __builtin_bit_cast(bf8, pan[0][ar_][slot(ar_, gq)]);                \
            const bf8 al = __builtin_bit_cast(bf8, pan[1][ar_][slot(ar_, gq)]);                \
            const bf8 bh = __builtin_bit_cast(bf8, pan[2][br_][slot(br_, gq)]);                \
            const bf8 bl = __builtin_bit_cast(bf8, pan[3][br_][slot(br_, gq)]);                \
            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, bh, acc, 0, 0, 0);               \
            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bl, acc, 0, 0, 0);               \
            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bh, acc, 0, 0, 0);               \
        }                                                                                      \
    }

    int ti = t_begin % n_it, tj = t_begin / n_it;
    f16v acc;
    BCPNN_REQUEST_TILE(ti, tj);
    BCPNN_REQUEST_PANELS(ti, tj, 0);
    BCPNN_STAGE();
    BCPNN_NEW_TILE(ti, tj);
    __syncthreads();

    for (int t = t_begin;; ++t) {                     // one tile per iteration
        for (int pass = 0; pass < n_pass - 1; ++pass) {
            BCPNN_REQUEST_PANELS(ti, tj, pass + 1);
            BCPNN_CONTRACT(pass);
            __syncthreads();
            BCPNN_STAGE();
            __syncthreads();
        }
        // last pass: the next tile's data is requested first (the last tile requests itself
        // again, which keeps every request unconditional)
        const bool last = t + 1 == t_end;
        int nti = ti + 1, ntj = tj;
        if (nti == n_it) {
            nti = 0;
            ++ntj;
        }
        if (last) {
            nti = ti;
            ntj = tj;
        }
        BCPNN_REQUEST_TILE(nti, ntj);
        BCPNN_REQUEST_PANELS(nti, ntj, 0);
        BCPNN_CONTRACT(n_pass - 1);

        // ---- tile epilogue ---------------------------------------------------------------
        {
            const int i0 = ti * kTM, j0 = tj * kTN;
            const int rows = n_in - i0 < kTM ? n_in - i0 : kTM;
            const int cols = n_out - j0 < kTN ? n_out - j0 : kTN;
            const int nhj = (j0 + cols - 1) / out_mcu - j0 / out_mcu + 1;
            // joint trace and masked weights: 32 unconditional buffer stores per lane (a store
            // outside the layer or on a silent block gets an offset past the range)
            const uint32_t bytes = (uint32_t)rows * n_out * 4u;
            const rsrc_t rp = make_rsrc(a.pij + (int64_t)i0 * n_out, bytes);
            const rsrc_t rw = make_rsrc(a.w + (int64_t)i0 * n_out, bytes);
            const bool jok = jl < cols;
            const uint32_t o0 = ((uint32_t)il0 * n_out + j0 + jl) * 4u;
            const float lpj = lpj_t[jl];
            const int ch = col_h[jl];
            float lpi[16];
            int act[16];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const f4 l4 = lpi_t[il0 / 4 + 2 * k];
                const i4 h4 = row_h[il0 / 4 + 2 * k];
#pragma unroll
                for (int m = 0; m < 4; ++m) {
                    lpi[4 * k + m] = l4[m];
                    act[4 * k + m] = mtile[h4[m] * nhj + ch];
                }
            }
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const uint32_t off = o0 + (uint32_t)(8 * (r >> 2) + (r & 3)) * n_out * 4u;
                const float p = to_storage<kDropBits>(fmaf(a.c2, acc[r], a.c1 * c_pold[r]));
                __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(p), rp, jok ? off : kDrop, 0,
                                                      0);
                const float wv = to_storage<kDropBits>(fast_log(fmaxf(p, a.eps)) - lpi[r] - lpj);
                __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(wv), rw,
                                                      jok && act[r] ? off : kDrop, 0, 0);
            }
        }
        __syncthreads();
        if (last) break;
        BCPNN_STAGE();
        BCPNN_NEW_TILE(nti, ntj);
        __syncthreads();
        ti = nti;
        tj = ntj;
    }
#undef BCPNN_REQUEST_PANELS
#undef BCPNN_REQUEST_TILE
#undef BCPNN_STAGE
#undef BCPNN_NEW_TILE
#undef BCPNN_CONTRACT
}

int persistent_blocks() {
    static int n = 0;
    if (n == 0) {
        int dev = 0, cus = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            cus <= 0)
            cus = 256;
        n = 3 * cus;
    }
    return n;
}

}  // namespace

hipError_t launch_trace_update(hipStream_t stream, const Geometry& g, const TraceArgs& a,
                               hipEvent_t start, hipEvent_t stop) {
    const int64_t n_tiles = ((g.n_in + kTM - 1) / kTM) * ((g.n_out + kTN - 1) / kTN);
    const unsigned blocks = (unsigned)(n_tiles < persistent_blocks() ? n_tiles : persistent_blocks());
    void (*kernel)(Geometry, TraceArgs, int) = nullptr;
    switch (a.drop_bits) {
        case 0: kernel = trace_kernel<0>; break;
        case 13: kernel = trace_kernel<13>; break;
        case 16: kernel = trace_kernel<16>; break;
        default: return hipErrorInvalidValue;
    }
    // the events (when given) are stamped by the dispatch itself, so they time the kernel alone
    hipExtLaunchKernelGGL(kernel, dim3(blocks), dim3(kThreads), 0, stream, start, stop, 0, g, a,
                          (int)n_tiles);
    return hipGetLastError();
}

}  // namespace bcpnn
