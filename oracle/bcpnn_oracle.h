/*
 * CPU oracle of the BCPNN hidden-layer training step: declarations.
 *
 * TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's CPU-baseline leg
 * may use this library.  Host pointers only; layouts are described in bcpnn_oracle.c.
 */
#ifndef BCPNN_ORACLE_H
#define BCPNN_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { ORACLE_STORE_F32 = 0, ORACLE_STORE_BF16 = 1, ORACLE_STORE_M10 = 2 };

typedef struct {
    int32_t in_hcu, in_mcu, out_hcu, out_mcu;
    float alpha;        /* lambda of Alg. 1: the trace update rate                      */
    int32_t n_cycles;   /* repetitions of the trace/weight cycle per batch (Alg. 1)      */
    float gain;         /* softmax gain g                                                */
    float bias_gain;    /* k_B of Alg. 1                                                 */
    float eps;          /* lower clamp of every probability inside a log                  */
    float pi_init;      /* initial Pi (<= 0: 1 / M_in)                                    */
    float pj_init;      /* initial Pj (<= 0: 1 / M_out)                                   */
    float init_noise;   /* amplitude of the initial weights                               */
    uint64_t seed;      /* stream of the initial weights                                  */
    int32_t n_swaps;    /* swaps per hidden HCU per structural update                     */
    int32_t storage;    /* ORACLE_STORE_* format of Pij and W                             */
} oracle_params;

int oracle_threads(void);
/* Worker threads of the OpenMP loops from now on (n > 0); only timing depends on it. */
void oracle_set_threads(int n);
float oracle_round_storage(float v, int32_t storage);
double oracle_splitmix_uniform(uint64_t seed, uint64_t idx);

void oracle_init_state(const oracle_params *p, const uint8_t *mask, float *pi, float *pj,
                       float *pij, float *w, float *b);
void oracle_support(const oracle_params *p, int32_t B, const float *x, const float *w,
                    const float *b, float *s);
void oracle_softmax(const oracle_params *p, int32_t B, const float *s, float *y);
void oracle_update_traces(const oracle_params *p, int32_t B, const float *x, const float *y,
                          float *pi, float *pj, float *pij);
void oracle_update_weights(const oracle_params *p, const uint8_t *mask, const float *pi,
                           const float *pj, const float *pij, float *w, float *b);
void oracle_mutual_information(const oracle_params *p, const float *pi, const float *pj,
                               const float *pij, double *mi);
int32_t oracle_plasticity_swap(const oracle_params *p, const double *mi, uint8_t *mask,
                               int32_t *swaps);
int32_t oracle_structural_update(const oracle_params *p, const float *pi, const float *pj,
                                 const float *pij, uint8_t *mask, float *w, double *mi_out,
                                 int32_t *swaps_out);
void oracle_readout(const oracle_params *p, int32_t B, const float *s, int32_t *winner);
void oracle_train_batch(const oracle_params *p, int32_t B, const float *x, const float *target,
                        float *s, float *y, float *pi, float *pj, float *pij, float *w,
                        float *b, const uint8_t *mask);

#ifdef __cplusplus
}
#endif
#endif
