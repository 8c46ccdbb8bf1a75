/*
 * CPU oracle of the BCPNN hidden-layer training step (Podobas et al., "StreamBrain: An HPC
 * Framework for Brain-like Neural Networks on CPUs, GPUs and FPGAs", HEART 2021).
 *
 * TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's CPU-baseline leg
 * may load this library.  It shares no code, header, table or constant with the GPU library:
 * everything below is written out from the paper's update equations.
 *
 * Conventions (all functions):
 *   - units are numbered HCU-major: unit = h * M + m;
 *   - x is [B][N_in], y and s are [B][N_out], pij and w are [N_in][N_out] (i-major), pi is
 *     [N_in], pj and b are [N_out], mask is [H_in][H_out] uint8 (1 = active connection);
 *   - state is stored as fp32; every result is computed in fp64 from the stored fp32 values
 *     and rounded to fp32 once when it is stored (unless the storage format says otherwise);
 *   - sums run over their index in increasing order; no blocking, fusion or reordering.
 *
 * Readings of points the paper leaves open (each one is listed with its reason in the design
 * notes of the repository):
 *   - initial traces pi_init, pj_init (<= 0 selects 1/M_in, 1/M_out) and Pij = fl(Pi * Pj);
 *   - initial weights w = mask * init_noise * (2u - 1), u from the SplitMix64 finaliser keyed by
 *     (seed, i * N_out + j), so that the softmax is not uniform at the first batch;
 *   - logs take max(P, eps) of every probability; the stored traces are not clamped;
 *   - softmax carries a gain g: a_j = exp(g s_j) / sum_m exp(g s_m) (g = 1 is the paper's);
 *   - mutual information is the textbook MI of the joint table {Pij : i in h_i, j in h_j}
 *     with marginals Pi, Pj, in fp64, 0 * log(.) = 0;
 *   - the greedy swap exchanges, per hidden HCU, the lowest-MI active input HCU with the
 *     highest-MI silent one if the latter is strictly larger, ties to the lowest HCU index,
 *     n_swaps times over HCUs not yet swapped in this update;
 *   - Pij and W may be stored rounded to bf16 or to a 10-bit mantissa (round to nearest even).
 */
#include "bcpnn_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int oracle_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void oracle_set_threads(int n) {
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* ------------------------------------------------------------------------------------------
 * Storage rounding.  bf16 keeps 1 sign + 8 exponent + 7 mantissa bits of an fp32 value; the
 * "M10" format keeps 10 mantissa bits (the paper's BFn naming: n = 1 + 8 + mantissa, Sec. 3,
 * FPGA backend).  Rounding is IEEE-754 round-to-nearest, ties to even, written from the
 * definition: the value is the fp32 value v; the two neighbours in the target format are the
 * truncation t and t + ulp; pick the nearer, and on an exact tie the one with an even last kept
 * bit.  NaN and infinities pass through.  Evaluated in fp64, where every quantity is exact.
 * ------------------------------------------------------------------------------------------ */
static float round_to_mantissa(float v, int mant_bits) {
    if (!isfinite(v) || v == 0.0f) return v;
    int e;
    (void)frexp((double)fabsf(v), &e);              /* |v| = m 2^e, m in [0.5, 1) */
    int exp2 = e - 1;                                /* |v| = 1.f * 2^exp2 */
    if (exp2 < -126) exp2 = -126;                    /* below fp32's normal range the step is fixed */
    const double quantum = ldexp(1.0, exp2 - mant_bits);
    const double scaled = (double)fabsf(v) / quantum;          /* exact: a power-of-two scale */
    const double lo = floor(scaled);
    const double frac = scaled - lo;
    double kept;
    if (frac > 0.5) kept = lo + 1.0;
    else if (frac < 0.5) kept = lo;
    else kept = (fmod(lo, 2.0) == 0.0) ? lo : lo + 1.0;   /* tie: even last kept bit */
    const float out = (float)(kept * quantum);       /* exact, or +inf past the largest finite */
    return signbit(v) ? -out : out;
}

static float store(double v, int32_t storage) {
    float f = (float)v;
    if (storage == ORACLE_STORE_BF16) return round_to_mantissa(f, 7);
    if (storage == ORACLE_STORE_M10) return round_to_mantissa(f, 10);
    return f;
}

float oracle_round_storage(float v, int32_t storage) { return store((double)v, storage); }

/* ------------------------------------------------------------------------------------------
 * SplitMix64 finaliser (Steele, Lea, Flood, "Fast splittable pseudorandom number generators",
 * OOPSLA 2014), used as a counter-based generator: draw idx of stream seed.
 * ------------------------------------------------------------------------------------------ */
double oracle_splitmix_uniform(uint64_t seed, uint64_t idx) {
    uint64_t z = seed + (idx + 1u) * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    z = z ^ (z >> 31);
    return (double)(z >> 40) * (1.0 / 16777216.0);   /* 24 bits: exact in fp32 */
}

static double clamp_eps(float p, double eps) { return (double)p > eps ? (double)p : eps; }

/* log(Pij / (Pi Pj)) with every probability clamped below at eps (Alg. 1, weight line). */
static double log_ratio(float pij, float pi, float pj, double eps) {
    return log(clamp_eps(pij, eps) / (clamp_eps(pi, eps) * clamp_eps(pj, eps)));
}

static double initial_pi(const oracle_params *p) {
    return p->pi_init > 0.0f ? (double)p->pi_init : 1.0 / (double)p->in_mcu;
}

static double initial_pj(const oracle_params *p) {
    return p->pj_init > 0.0f ? (double)p->pj_init : 1.0 / (double)p->out_mcu;
}

/* Initial state.  Sec. 2 says only that the connectivity (mask) starts random; it gives no
 * initial trace values.  The reading taken here: the traces start at the uniform distribution
 * of each HCU and the joint at the product of its marginals, and the weights as masked
 * SplitMix64 noise (with traces in product form alone every weight would be 0 and stay 0). */
void oracle_init_state(const oracle_params *p, const uint8_t *mask, float *pi, float *pj,
                       float *pij, float *w, float *b) {
    const int64_t n_in = (int64_t)p->in_hcu * p->in_mcu;
    const int64_t n_out = (int64_t)p->out_hcu * p->out_mcu;
    const float pi0 = (float)initial_pi(p);
    const float pj0 = (float)initial_pj(p);
    const double eps = (double)p->eps;
    for (int64_t i = 0; i < n_in; ++i) pi[i] = pi0;
    for (int64_t j = 0; j < n_out; ++j) {
        pj[j] = pj0;
        b[j] = (float)((double)p->bias_gain * log(clamp_eps(pj0, eps)));
    }
    const float pij0 = (float)((double)pi0 * (double)pj0);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n_in; ++i) {
        const int64_t hi = i / p->in_mcu;
        for (int64_t j = 0; j < n_out; ++j) {
            const int64_t hj = j / p->out_mcu;
            pij[i * n_out + j] = store((double)pij0, p->storage);
            double v = 0.0;
            if (mask[hi * p->out_hcu + hj]) {
                double u = oracle_splitmix_uniform(p->seed, (uint64_t)(i * n_out + j));
                v = (double)p->init_noise * (2.0 * u - 1.0);
            }
            w[i * n_out + j] = store(v, p->storage);
        }
    }
}

/* Support, Alg. 1 (s_j <- a_i w_0 + b_0): s[b][j] = b_j + sum_i x[b][i] w[i][j].  The weights
 * are stored with the mask already applied (Alg. 1, last line of the cycle). */
void oracle_support(const oracle_params *p, int32_t B, const float *x, const float *w,
                    const float *b, float *s) {
    const int64_t n_in = (int64_t)p->in_hcu * p->in_mcu;
    const int64_t n_out = (int64_t)p->out_hcu * p->out_mcu;
#pragma omp parallel for schedule(static)
    for (int32_t r = 0; r < B; ++r) {
        double *acc = (double *)malloc((size_t)n_out * sizeof(double));
        for (int64_t j = 0; j < n_out; ++j) acc[j] = (double)b[j];
        for (int64_t i = 0; i < n_in; ++i) {               /* i ascending for every j */
            const double xi = (double)x[(int64_t)r * n_in + i];
            const float *wrow = w + i * n_out;
            for (int64_t j = 0; j < n_out; ++j) acc[j] += xi * (double)wrow[j];
        }
        for (int64_t j = 0; j < n_out; ++j) s[(int64_t)r * n_out + j] = (float)acc[j];
        free(acc);
    }
}

/* Softmax within each hidden HCU, Alg. 1 and Sec. 2: a_j = exp(g s_j) / sum_{m in HCU} exp(g s_m),
 * evaluated as exp(g (s_j - max)) / sum exp(g (s_m - max)), an identity in exact arithmetic. */
void oracle_softmax(const oracle_params *p, int32_t B, const float *s, float *y) {
    const int64_t n_out = (int64_t)p->out_hcu * p->out_mcu;
    const double g = (double)p->gain;
    for (int32_t r = 0; r < B; ++r) {
        for (int32_t h = 0; h < p->out_hcu; ++h) {
            const float *sr = s + (int64_t)r * n_out + (int64_t)h * p->out_mcu;
            float *yr = y + (int64_t)r * n_out + (int64_t)h * p->out_mcu;
            double mx = (double)sr[0];
            for (int32_t m = 1; m < p->out_mcu; ++m)
                if ((double)sr[m] > mx) mx = (double)sr[m];
            double den = 0.0;
            for (int32_t m = 0; m < p->out_mcu; ++m) den += exp(g * ((double)sr[m] - mx));
            for (int32_t m = 0; m < p->out_mcu; ++m)
                yr[m] = (float)(exp(g * ((double)sr[m] - mx)) / den);
        }
    }
}

/* Trace updates, Alg. 1 cycle loop (repeated n_cycles times with the same batch averages):
 *   C_i  <- (1 - lambda) C_i  + lambda <a_i>
 *   C_j  <- (1 - lambda) C_j  + lambda <a_j>
 *   C_ij <- (1 - lambda) C_ij + lambda <a_i (x) a_j>
 * where <.> is the mean over the batch (Sec. 2).  The traces stay in fp64 across the cycles
 * and are rounded once on store. */
void oracle_update_traces(const oracle_params *p, int32_t B, const float *x, const float *y,
                          float *pi, float *pj, float *pij) {
    const int64_t n_in = (int64_t)p->in_hcu * p->in_mcu;
    const int64_t n_out = (int64_t)p->out_hcu * p->out_mcu;
    const double lam = (double)p->alpha;
    const double invB = 1.0 / (double)B;

    for (int64_t i = 0; i < n_in; ++i) {
        double sum = 0.0;
        for (int32_t r = 0; r < B; ++r) sum += (double)x[(int64_t)r * n_in + i];
        double c = (double)pi[i];
        for (int32_t cyc = 0; cyc < p->n_cycles; ++cyc) c = (1.0 - lam) * c + lam * (sum * invB);
        pi[i] = (float)c;
    }
    for (int64_t j = 0; j < n_out; ++j) {
        double sum = 0.0;
        for (int32_t r = 0; r < B; ++r) sum += (double)y[(int64_t)r * n_out + j];
        double c = (double)pj[j];
        for (int32_t cyc = 0; cyc < p->n_cycles; ++cyc) c = (1.0 - lam) * c + lam * (sum * invB);
        pj[j] = (float)c;
    }
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n_in; ++i) {
        double *acc = (double *)calloc((size_t)n_out, sizeof(double));
        for (int32_t r = 0; r < B; ++r) {                   /* r ascending for every j */
            const double xi = (double)x[(int64_t)r * n_in + i];
            const float *yr = y + (int64_t)r * n_out;
            for (int64_t j = 0; j < n_out; ++j) acc[j] += xi * (double)yr[j];
        }
        float *prow = pij + i * n_out;
        for (int64_t j = 0; j < n_out; ++j) {
            double c = (double)prow[j];
            for (int32_t cyc = 0; cyc < p->n_cycles; ++cyc)
                c = (1.0 - lam) * c + lam * (acc[j] * invB);
            prow[j] = store(c, p->storage);
        }
        free(acc);
    }
}

/* Weights and bias, Alg. 1: w_0 <- log(C_ij / (C_i (x) C_j)), b_0 <- k_B log C_j, then the
 * mask is applied element by element (Sec. 2, structural plasticity paragraph). */
void oracle_update_weights(const oracle_params *p, const uint8_t *mask, const float *pi,
                           const float *pj, const float *pij, float *w, float *b) {
    const int64_t n_in = (int64_t)p->in_hcu * p->in_mcu;
    const int64_t n_out = (int64_t)p->out_hcu * p->out_mcu;
    const double eps = (double)p->eps;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n_in; ++i) {
        const int64_t hi = i / p->in_mcu;
        for (int64_t j = 0; j < n_out; ++j) {
            const int64_t hj = j / p->out_mcu;
            double v = 0.0;
            if (mask[hi * p->out_hcu + hj]) v = log_ratio(pij[i * n_out + j], pi[i], pj[j], eps);
            w[i * n_out + j] = store(v, p->storage);
        }
    }
    for (int64_t j = 0; j < n_out; ++j)
        b[j] = (float)((double)p->bias_gain * log(clamp_eps(pj[j], eps)));
}

/* Mutual-information score of every (input HCU, hidden HCU) connection (Sec. 2, structural
 * plasticity paragraph): MI[hi][hj] = sum_{i in hi} sum_{j in hj} Pij log(Pij / (Pi Pj)).
 * Output [H_in][H_out] fp64. */
void oracle_mutual_information(const oracle_params *p, const float *pi, const float *pj,
                               const float *pij, double *mi) {
    const int64_t n_out = (int64_t)p->out_hcu * p->out_mcu;
    const double eps = (double)p->eps;
#pragma omp parallel for schedule(static)
    for (int32_t hi = 0; hi < p->in_hcu; ++hi) {
        for (int32_t hj = 0; hj < p->out_hcu; ++hj) {
            double sum = 0.0;
            for (int32_t a = 0; a < p->in_mcu; ++a) {
                const int64_t i = (int64_t)hi * p->in_mcu + a;
                for (int32_t c = 0; c < p->out_mcu; ++c) {
                    const int64_t j = (int64_t)hj * p->out_mcu + c;
                    const float q = pij[i * n_out + j];
                    if (q == 0.0f) continue;                 /* 0 log 0 := 0 */
                    sum += (double)q * log_ratio(q, pi[i], pj[j], eps);
                }
            }
            mi[(int64_t)hi * p->out_hcu + hj] = sum;
        }
    }
}

/* Greedy swap (Sec. 2): for each hidden HCU, silence the active connection with the lowest MI
 * and activate the silent one with the highest, if that raises the HCU's received MI.  The
 * number of active connections stays fixed.  swaps (nullable) receives, per hidden HCU and
 * swap slot, the (silenced, activated) input HCU pair or (-1, -1).  Returns the swap count. */
int32_t oracle_plasticity_swap(const oracle_params *p, const double *mi, uint8_t *mask,
                               int32_t *swaps) {
    const int32_t hin = p->in_hcu, hout = p->out_hcu;
    uint8_t *used = (uint8_t *)malloc((size_t)hin);
    int32_t count = 0;
    if (swaps)
        for (int64_t t = 0; t < (int64_t)hout * p->n_swaps * 2; ++t) swaps[t] = -1;
    for (int32_t hj = 0; hj < hout; ++hj) {
        memset(used, 0, (size_t)hin);
        for (int32_t t = 0; t < p->n_swaps; ++t) {
            int32_t a = -1, s = -1;
            for (int32_t hi = 0; hi < hin; ++hi) {
                if (used[hi]) continue;
                const double v = mi[(int64_t)hi * hout + hj];
                if (mask[(int64_t)hi * hout + hj]) {
                    if (a < 0 || v < mi[(int64_t)a * hout + hj]) a = hi;
                } else {
                    if (s < 0 || v > mi[(int64_t)s * hout + hj]) s = hi;
                }
            }
            if (a < 0 || s < 0) break;
            if (!(mi[(int64_t)s * hout + hj] > mi[(int64_t)a * hout + hj])) break;
            mask[(int64_t)a * hout + hj] = 0;
            mask[(int64_t)s * hout + hj] = 1;
            used[a] = used[s] = 1;
            if (swaps) {
                swaps[((int64_t)hj * p->n_swaps + t) * 2 + 0] = a;
                swaps[((int64_t)hj * p->n_swaps + t) * 2 + 1] = s;
            }
            ++count;
        }
    }
    free(used);
    return count;
}

/* Structural update, Alg. 1 "update plasticity mask": score, swap, then give the changed
 * blocks of w their masked values (0 for a silenced block, the log-ratio for an activated one)
 * so that the same batch's support already uses the new mask.  mi_out and swaps nullable. */
int32_t oracle_structural_update(const oracle_params *p, const float *pi, const float *pj,
                                 const float *pij, uint8_t *mask, float *w, double *mi_out,
                                 int32_t *swaps_out) {
    const int64_t n_out = (int64_t)p->out_hcu * p->out_mcu;
    const double eps = (double)p->eps;
    double *mi = mi_out ? mi_out
                        : (double *)malloc((size_t)p->in_hcu * p->out_hcu * sizeof(double));
    int32_t *swaps = (int32_t *)malloc((size_t)p->out_hcu * p->n_swaps * 2 * sizeof(int32_t));
    oracle_mutual_information(p, pi, pj, pij, mi);
    int32_t count = oracle_plasticity_swap(p, mi, mask, swaps);
    for (int32_t hj = 0; hj < p->out_hcu; ++hj) {
        for (int32_t t = 0; t < p->n_swaps; ++t) {
            for (int side = 0; side < 2; ++side) {
                const int32_t hi = swaps[((int64_t)hj * p->n_swaps + t) * 2 + side];
                if (hi < 0) continue;
                for (int32_t a = 0; a < p->in_mcu; ++a) {
                    const int64_t i = (int64_t)hi * p->in_mcu + a;
                    for (int32_t c = 0; c < p->out_mcu; ++c) {
                        const int64_t j = (int64_t)hj * p->out_mcu + c;
                        double v = side ? log_ratio(pij[i * n_out + j], pi[i], pj[j], eps) : 0.0;
                        w[i * n_out + j] = store(v, p->storage);
                    }
                }
            }
        }
    }
    if (swaps_out) memcpy(swaps_out, swaps, (size_t)p->out_hcu * p->n_swaps * 2 * sizeof(int32_t));
    free(swaps);
    if (!mi_out) free(mi);
    return count;
}

/* Inference readout: the winning MCU of each (sample, HCU), the argmax of the support, ties to
 * the lowest MCU index.  winner is [B][H_out]. */
void oracle_readout(const oracle_params *p, int32_t B, const float *s, int32_t *winner) {
    const int64_t n_out = (int64_t)p->out_hcu * p->out_mcu;
    for (int32_t r = 0; r < B; ++r)
        for (int32_t h = 0; h < p->out_hcu; ++h) {
            const float *sr = s + (int64_t)r * n_out + (int64_t)h * p->out_mcu;
            int32_t best = 0;
            for (int32_t m = 1; m < p->out_mcu; ++m)
                if (sr[m] > sr[best]) best = m;
            winner[(int64_t)r * p->out_hcu + h] = best;
        }
}

/* One batch of Alg. 1 (activations, then the cycle loop): support, softmax, traces, weights.
 * target (nullable, [B][N_out]) replaces the softmax activity in the trace update, as in the
 * supervised output layer.  s and y receive the support and the softmax. */
void oracle_train_batch(const oracle_params *p, int32_t B, const float *x, const float *target,
                        float *s, float *y, float *pi, float *pj, float *pij, float *w,
                        float *b, const uint8_t *mask) {
    oracle_support(p, B, x, w, b, s);
    oracle_softmax(p, B, s, y);
    oracle_update_traces(p, B, x, target ? target : y, pi, pj, pij);
    oracle_update_weights(p, mask, pi, pj, pij, w, b);
}
