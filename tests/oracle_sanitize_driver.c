/*
 * Drives every entry point of the CPU oracle on small layers (ragged batches, a partial mask,
 * reduced storage, supervised targets, several swaps), for a build with the address and
 * undefined-behaviour sanitizers (tests/test_oracle_sanitizers.py).  Exit status 0 and no
 * sanitizer report mean no out-of-bounds access, leak or undefined operation was seen.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "bcpnn_oracle.h"

static uint64_t lcg = 12345;
static float urand(void) {
    lcg = lcg * 6364136223846793005ull + 1442695040888963407ull;
    return (float)((lcg >> 40) & 0xffffff) / 16777216.0f;
}

static int run(int in_hcu, int in_mcu, int out_hcu, int out_mcu, int storage, int n_swaps,
               int active, int supervised) {
    oracle_params p;
    memset(&p, 0, sizeof p);
    p.in_hcu = in_hcu; p.in_mcu = in_mcu; p.out_hcu = out_hcu; p.out_mcu = out_mcu;
    p.alpha = 0.05f; p.n_cycles = 2; p.gain = 2.0f; p.bias_gain = 1.0f; p.eps = 1e-8f;
    p.init_noise = 0.1f; p.seed = 7; p.n_swaps = n_swaps; p.storage = storage;
    const int n_in = in_hcu * in_mcu, n_out = out_hcu * out_mcu, max_b = 19;
    const size_t E = (size_t)n_in * n_out, H = (size_t)in_hcu * out_hcu;
    float *pi = malloc(n_in * sizeof(float)), *pj = malloc(n_out * sizeof(float));
    float *pij = malloc(E * sizeof(float)), *w = malloc(E * sizeof(float));
    float *b = malloc(n_out * sizeof(float));
    float *x = malloc((size_t)max_b * n_in * sizeof(float));
    float *t = malloc((size_t)max_b * n_out * sizeof(float));
    float *s = malloc((size_t)max_b * n_out * sizeof(float));
    float *y = malloc((size_t)max_b * n_out * sizeof(float));
    int32_t *win = malloc((size_t)max_b * out_hcu * sizeof(int32_t));
    uint8_t *mask = malloc(H);
    double *mi = malloc(H * sizeof(double));
    int32_t *sw = malloc((size_t)out_hcu * n_swaps * 2 * sizeof(int32_t) + 1);
    for (int hi = 0; hi < in_hcu; ++hi)
        for (int hj = 0; hj < out_hcu; ++hj)
            mask[(size_t)hi * out_hcu + hj] = (uint8_t)((hi + hj) % in_hcu < active);
    oracle_init_state(&p, mask, pi, pj, pij, w, b);
    const int sizes[] = {19, 7, 1, 19, 13};
    int swapped = 0;
    for (int k = 0; k < 5; ++k) {
        const int B = sizes[k];
        for (int r = 0; r < B; ++r)
            for (int h = 0; h < in_hcu; ++h) {
                float tot = 0.0f;
                for (int m = 0; m < in_mcu; ++m) tot += (x[(size_t)r * n_in + h * in_mcu + m] = urand() + 0.01f);
                for (int m = 0; m < in_mcu; ++m) x[(size_t)r * n_in + h * in_mcu + m] /= tot;
            }
        for (int r = 0; r < B; ++r)
            for (int j = 0; j < n_out; ++j) t[(size_t)r * n_out + j] = (j % out_mcu == (r + k) % out_mcu);
        if (k == 3) swapped += oracle_structural_update(&p, pi, pj, pij, mask, w, mi, sw);
        oracle_train_batch(&p, B, x, supervised ? t : NULL, s, y, pi, pj, pij, w, b, mask);
        oracle_readout(&p, B, s, win);
    }
    oracle_support(&p, 7, x, w, b, s);
    oracle_softmax(&p, 7, s, y);
    oracle_update_traces(&p, 7, x, y, pi, pj, pij);
    oracle_update_weights(&p, mask, pi, pj, pij, w, b);
    oracle_mutual_information(&p, pi, pj, pij, mi);
    swapped += oracle_plasticity_swap(&p, mi, mask, sw);
    (void)oracle_round_storage(1.5f, storage);
    (void)oracle_splitmix_uniform(7, 3);
    int active_left = 0;
    for (size_t q = 0; q < H; ++q) active_left += mask[q];
    free(pi); free(pj); free(pij); free(w); free(b); free(x); free(t); free(s); free(y);
    free(win); free(mask); free(mi); free(sw);
    printf("layer %dx%d -> %dx%d storage %d: %d swaps, %d active\n", in_hcu, in_mcu, out_hcu,
           out_mcu, storage, swapped, active_left);
    return active_left == active * out_hcu ? 0 : 1;
}

int main(void) {
    int bad = 0;
    bad |= run(9, 2, 3, 5, 0, 1, 4, 0);
    bad |= run(7, 3, 4, 1, 1, 2, 3, 1);
    bad |= run(5, 1, 2, 33, 2, 3, 2, 0);
    bad |= run(6, 2, 5, 4, 0, 1, 6, 1);
    printf("oracle threads %d\n", oracle_threads());
    return bad;
}
