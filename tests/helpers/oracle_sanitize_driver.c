/* Calls every entry point of the oracle on small models, including its
 * argument-error paths, so that a build with AddressSanitizer and
 * UndefinedBehaviorSanitizer can check the oracle's memory accesses. Exits 0
 * when every call returns what it should. */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "zo_oracle.h"

#define CHECK(x)                                                   \
    do {                                                           \
        if (!(x)) {                                                \
            fprintf(stderr, "check failed: %s (line %d)\n", #x, __LINE__); \
            return 1;                                              \
        }                                                          \
    } while (0)

static double quad(const double* w, uint64_t P, void* ctx) {
    (void)ctx;
    double s = 0.0;
    for (uint64_t j = 0; j < P; ++j) s += 0.5 * w[j] * w[j] + (double)j * w[j];
    return s;
}

static int run(const zo_ref_config* cfg) {
    const uint64_t P = zo_ref_param_count(cfg);
    CHECK(P > 0);
    uint64_t off[64];
    CHECK(zo_ref_layout(cfg, off, 3 * cfg->n_layers + 4) == ZO_REF_OK);
    CHECK(off[3 * cfg->n_layers + 3] == P);
    const size_t el = cfg->wdtype ? 2 : 4;
    void* theta = malloc(P * el);
    void* t2 = malloc(P * el);
    double* w = malloc(sizeof(double) * P);
    CHECK(theta && t2 && w);
    CHECK(zo_ref_init(cfg, theta, 11) == ZO_REF_OK);
    enum { B = 3, C = 5, N = 3 };
    int32_t tokens[B * (C + 1)];
    uint8_t mask[B * C];
    for (int k = 0; k < B * (C + 1); ++k) tokens[k] = (k * 7 + 3) % cfg->vocab;
    for (int k = 0; k < B * C; ++k) mask[k] = (uint8_t)(k % 3 != 0);
    CHECK(zo_ref_materialise(cfg, theta, 5, 1, 1e-2, 0, w) == ZO_REF_OK);
    double ell[B * C];
    const double L = zo_ref_lstm_loss(cfg, w, tokens, mask, B, C, C + 1, ell);
    CHECK(isfinite(L) && L > 0.0);
    float lp[N], lm[N];
    double dp[N], dm[N], fl[N], f0;
    CHECK(zo_ref_perturbed_losses(cfg, theta, 5, 1e-2f, N, 2, tokens, mask, B, C, lp, lm) == ZO_REF_OK);
    CHECK(zo_ref_perturbed_losses_ex(cfg, theta, 5, 1e-2f, N, 2, tokens, NULL, B, C, 1, dp, dm) == ZO_REF_OK);
    CHECK(zo_ref_fd_losses(cfg, theta, 5, 1e-2f, N, 2, tokens, mask, B, C, fl, &f0) == ZO_REF_OK);
    memcpy(t2, theta, P * el);
    CHECK(zo_ref_update(cfg, t2, 5, 1e-2f, 1e-2f, N, 2, lp, lm) == ZO_REF_OK);
    const float lf[N] = {(float)fl[0], (float)fl[1], (float)fl[2]};
    CHECK(zo_ref_fd_update(cfg, t2, 5, 1e-2f, 1e-2f, N, 2, lf, (float)f0) == ZO_REF_OK);
    uint64_t idx[3] = {0, P / 2, P - 1};
    unsigned char out[3 * 4];
    CHECK(zo_ref_update_sampled(cfg, theta, 5, 1e-2f, 1e-2f, N, 2, lp, lm, idx, 3, out) == ZO_REF_OK);
    /* error paths: nothing written */
    memcpy(t2, theta, P * el);
    float bad[N] = {1.0f, NAN, 2.0f};
    CHECK(zo_ref_update(cfg, t2, 5, 1e-2f, 1e-2f, N, 2, bad, lm) == ZO_REF_ENONFINITE);
    CHECK(memcmp(t2, theta, P * el) == 0);
    CHECK(zo_ref_update(cfg, NULL, 5, 1e-2f, 1e-2f, N, 2, lp, lm) == ZO_REF_EINVAL);
    CHECK(zo_ref_perturbed_losses(cfg, theta, 5, 0.0f, N, 0, tokens, mask, B, C, lp, lm) == ZO_REF_EINVAL);
    int32_t badtok[B * (C + 1)];
    memcpy(badtok, tokens, sizeof badtok);
    badtok[4] = cfg->vocab;
    CHECK(zo_ref_perturbed_losses(cfg, theta, 5, 1e-2f, N, 0, badtok, mask, B, C, lp, lm) == ZO_REF_EINVAL);
    CHECK(zo_ref_fd_update(cfg, t2, 5, 1e-2f, 1e-2f, N, 0, lf, NAN) == ZO_REF_ENONFINITE);
    free(theta);
    free(t2);
    free(w);
    return 0;
}

int main(void) {
    const zo_ref_config cfgs[3] = {
        {1, 11, 4, 4, 0, 0},
        {2, 7, 6, 5, 0, 1},
        {2, 9, 8, 8, 1, 0},
    };
    for (int k = 0; k < 3; ++k)
        if (run(&cfgs[k])) return 1;
    /* probe stream, transforms and the generic estimator */
    float z[1000];
    zo_ref_probe(0, 3, 1, 5, 1000, z);
    zo_ref_probe(1, 3, 1, 7, 1000, z);
    uint32_t words[64];
    for (int k = 0; k < 64; ++k) words[k] = 2654435761u * (uint32_t)k;
    zo_ref_gauss_pairs(words, 32, z);
    float u[16], s[16], c[16];
    uint32_t k24[16];
    for (int k = 0; k < 16; ++k) {
        u[k] = (float)(k + 1) / 16.0f;
        k24[k] = (uint32_t)k << 20;
    }
    zo_ref_log_f32_array(u, 16, z);
    zo_ref_sincos_2pi_array(k24, 16, s, c);
    double th[10], gp[4], gm[4], g[10];
    for (int k = 0; k < 10; ++k) th[k] = 0.1 * k;
    CHECK(zo_ref_cd_losses_generic(10, th, 0, 9, 1e-3, 4, 0, 0, quad, NULL, gp, gm) == ZO_REF_OK);
    zo_ref_cd_gradient(10, 0, 9, 1e-3, 4, 0, gp, gm, g);
    printf("oracle sanitizer driver ok\n");
    return 0;
}
