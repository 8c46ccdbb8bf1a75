// Support and per-HCU activation: s = b + x w over the active input HCUs, then softmax (or
// argmax) within every hidden HCU (Alg. 1 support and softmax lines; Sec. 2).
//
// Design (gfx950):
//  * The weights are stored masked, so a hidden HCU only needs the rows of its active input
//    HCUs.  Each hidden HCU keeps an ascending list of them; the contraction for one hidden
//    HCU is a dense [B x K_h] . [K_h x M_out] product with K_h = n_active * M_in.  Silent
//    blocks are never read.
//  * The products accumulate in fp64 on the matrix cores (v_mfma_f64_16x16x4f64).  x and w are
//    fp32, so every product is exact in fp64 and the sum's rounding error stays far below the
//    fp32 rounding of the stored support.  (An fp32 accumulation of a few hundred terms of
//    magnitude ~10 drifts by ~1e-5, the size of the tolerance on the activities.)
//  * One workgroup owns one hidden HCU and 16 batch rows, i.e. complete softmax segments, so
//    the softmax runs in the epilogue from LDS and the support never round-trips through HBM.
//    Wave w computes the 16-column output tiles w, w + n_waves, ...; the 16 x K_h input panel
//    is gathered into LDS once per chunk and shared by all waves; each weight row segment is
//    read once per workgroup straight into the MFMA B operand.
//  * Work items (row tile, hidden HCU) are spread over the XCDs so that the row tiles of one
//    hidden HCU share one XCD's L2 (they read the same weight block).
//
// MFMA f64 16x16x4 lane layout (verified on gfx950): A[i][k] from lane i + 16 k, B[k][j] from
// lane j + 16 k, and lane l holds D[l / 16 + 4 r][l % 16] in result register r.
#include "bcpnn_internal.h"
#include "device_common.h"

namespace bcpnn {
namespace {

typedef double d4 __attribute__((ext_vector_type(4)));

constexpr int kRows = 16;         // batch rows per workgroup
constexpr int kChunk = 256;       // active input units staged per chunk
constexpr int kMaxWaves = 8;
constexpr int kTilesPerWave = 8;  // kMaxWaves * kTilesPerWave * 16 = 1024 = largest out_mcu

__global__ void __launch_bounds__(64 * kMaxWaves)
support_kernel(Geometry g, const float* __restrict__ x, int32_t B, const float* __restrict__ w,
               const float* __restrict__ bias, const int32_t* __restrict__ act_list,
               const int32_t* __restrict__ act_count, float gain, int mode, int n_tiles,
               int mpad, int n_row_tiles, float* __restrict__ y, float* __restrict__ s,
               int32_t* __restrict__ winner) {
    // LDS: the staged input panel during the contraction, the support tile afterwards.
    extern __shared__ float lds[];
    float* xs = lds;                                            // [kRows][kChunk]
    int32_t* units = reinterpret_cast<int32_t*>(lds + kRows * kChunk);   // [kChunk]
    float* stile = lds;                                         // [kRows][mpad]

    const int64_t work = xcd_linear_index(blockIdx.x, (int64_t)n_row_tiles * g.out_hcu);
    const int hj = (int)(work / n_row_tiles);
    const int row0 = (int)(work % n_row_tiles) * kRows;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int n_waves = blockDim.x >> 6;

    const int64_t k_total = (int64_t)act_count[hj] * g.in_mcu;
    const int32_t* alist = act_list + (int64_t)hj * g.in_hcu;
    const int64_t col_base = (int64_t)hj * g.out_mcu;

    d4 acc[kTilesPerWave];
#pragma unroll
    for (int t = 0; t < kTilesPerWave; ++t) acc[t] = d4{0.0, 0.0, 0.0, 0.0};

    for (int64_t k0 = 0; k0 < k_total; k0 += kChunk) {
        const int kc = (int)((k_total - k0) < kChunk ? (k_total - k0) : kChunk);
        __syncthreads();   // the previous chunk has been consumed
        for (int t = threadIdx.x; t < kChunk; t += blockDim.x) {
            int32_t unit = -1;
            if (t < kc) {
                const int64_t k = k0 + t;
                unit = alist[k / g.in_mcu] * g.in_mcu + (int32_t)(k % g.in_mcu);
            }
            units[t] = unit;
        }
        __syncthreads();
        for (int t = threadIdx.x; t < kRows * kChunk; t += blockDim.x) {
            const int r = t / kChunk, c = t % kChunk;
            const int32_t unit = units[c];
            float v = 0.0f;
            if (unit >= 0 && row0 + r < B) v = x[(int64_t)(row0 + r) * g.n_in + unit];
            xs[t] = v;
        }
        __syncthreads();

        const int ksteps = (kc + 3) / 4;
        for (int ks = 0; ks < ksteps; ++ks) {
            const int kk = ks * 4 + (lane >> 4);
            const double a = (double)xs[(lane & 15) * kChunk + kk];
            const int32_t unit = units[kk];
            const float* wrow = w + (int64_t)(unit < 0 ? 0 : unit) * g.n_out + col_base;
#pragma unroll
            for (int t = 0; t < kTilesPerWave; ++t) {
                const int nt = wave + t * n_waves;
                if (nt < n_tiles) {                       // uniform across the wave
                    const int col = nt * 16 + (lane & 15);
                    const double bv = (unit >= 0 && col < g.out_mcu) ? (double)wrow[col] : 0.0;
                    acc[t] = __builtin_amdgcn_mfma_f64_16x16x4f64(a, bv, acc[t], 0, 0, 0);
                }
            }
        }
    }

    __syncthreads();   // done with the input panel; reuse LDS for the support tile
#pragma unroll
    for (int t = 0; t < kTilesPerWave; ++t) {
        const int nt = wave + t * n_waves;
        if (nt < n_tiles) {
            const int col = nt * 16 + (lane & 15);
            if (col < g.out_mcu) {
                const double bj = (double)bias[col_base + col];
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    stile[((lane >> 4) + 4 * r) * mpad + col] = (float)(acc[t][r] + bj);
            }
        }
    }
    __syncthreads();

    for (int r = wave; r < kRows; r += n_waves) {
        const int row = row0 + r;
        if (row >= B) break;                          // uniform across the wave
        const float* srow = stile + r * mpad;
        const int64_t out = (int64_t)row * g.n_out + col_base;
        if (s)
            for (int m = lane; m < g.out_mcu; m += 64) s[out + m] = srow[m];
        if (mode == 0) {
            float mx = -INFINITY;
            for (int m = lane; m < g.out_mcu; m += 64) mx = fmaxf(mx, srow[m]);
            mx = wave_max(mx);
            float den = 0.0f;
            for (int m = lane; m < g.out_mcu; m += 64) den += expf(gain * (srow[m] - mx));
            den = wave_sum(den);
            const float inv = 1.0f / den;
            for (int m = lane; m < g.out_mcu; m += 64) y[out + m] = expf(gain * (srow[m] - mx)) * inv;
        } else {
            float bv = -INFINITY;
            int bi = 0x7fffffff;
            for (int m = lane; m < g.out_mcu; m += 64)
                if (srow[m] > bv) { bv = srow[m]; bi = m; }
            for (int off = 32; off > 0; off >>= 1) {
                const float ov = __shfl_xor(bv, off, 64);
                const int oi = __shfl_xor(bi, off, 64);
                if (ov > bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
            }
            if (lane == 0) winner[(int64_t)row * g.out_hcu + hj] = bi;
        }
    }
}

}  // namespace

hipError_t launch_support(hipStream_t stream, const Geometry& g, const float* x, int32_t B,
                          const float* w, const float* bias, const int32_t* act_list,
                          const int32_t* act_count, float gain, int mode, float* y, float* s,
                          int32_t* winner) {
    const int n_tiles = (g.out_mcu + 15) / 16;
    const int mpad = n_tiles * 16;
    const int n_waves = n_tiles < kMaxWaves ? n_tiles : kMaxWaves;
    const int n_row_tiles = (B + kRows - 1) / kRows;
    const size_t panel = (size_t)kRows * kChunk * sizeof(float) + kChunk * sizeof(int32_t);
    const size_t tile = (size_t)kRows * mpad * sizeof(float);
    const size_t lds = panel > tile ? panel : tile;
    const int64_t blocks = (int64_t)n_row_tiles * g.out_hcu;
    support_kernel<<<(unsigned)blocks, 64 * n_waves, lds, stream>>>(
        g, x, B, w, bias, act_list, act_count, gain, mode, n_tiles, mpad, n_row_tiles, y, s,
        winner);
    return hipGetLastError();
}

}  // namespace bcpnn
