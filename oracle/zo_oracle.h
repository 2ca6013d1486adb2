/*
 * CPU oracle for one CD-RGE training step of a stacked-LSTM language model.
 *
 * TEST INFRASTRUCTURE ONLY. This library is the independent, slow, obviously
 * correct reference that the GPU path is checked against. Only the tests, the
 * smoke check and the benchmark's CPU-baseline leg may load it; the product
 * path never calls it and shares no code with it.
 *
 * Everything here follows the paper directly:
 *   - central-difference estimator, Eq. 2 (Section 2);
 *   - the step of Algorithm 1 (evaluate L(theta + eps z_i) and L(theta - eps z_i)
 *     for every probe, then step along the difference-weighted probes);
 *   - the update of Eq. 7 in its general form
 *         theta <- theta - lr * (1/N) * sum_i (L+_i - L-_i) / (2 eps) * z_i
 *     which is Eq. 7 exactly when lr == eps (Section 2 ties eta = eps);
 *   - Rademacher probes (Section 2, Algorithm 2) and normal probes (Section 2).
 * Every perturbed weight set is materialised in full, in double precision,
 * from the pristine theta, and the LSTM forward runs naively in double.
 *
 * The random numbers are fixed by a counter-based Philox4x32-10 stream
 * (Salmon, Moraes, Dror, Shaw, SC'11), keyed by the 64-bit seed, with the
 * counter (block_lo, block_hi, probe index i, tag). The transforms from
 * Philox words to probe values are stated in zo_oracle.c next to the code.
 *
 * Parity status of each function is stated in its comment in zo_oracle.c.
 */
#ifndef ZO_ORACLE_H
#define ZO_ORACLE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
    int32_t n_layers;
    int32_t vocab;
    int32_t embed;
    int32_t hidden;
    int32_t wdtype; /* 0 = fp32 weights, 1 = bf16 weights */
    int32_t probe;  /* 0 = Rademacher, 1 = Gaussian */
} zo_ref_config;

enum {
    ZO_REF_OK = 0,
    ZO_REF_EINVAL = -1,
    ZO_REF_ESHAPE = -2,
    ZO_REF_ENOMEM = -4,
    ZO_REF_ENONFINITE = -5
};

/* Philox tags (fourth counter word). */
enum { ZO_REF_TAG_RADEMACHER = 0, ZO_REF_TAG_GAUSSIAN = 1, ZO_REF_TAG_INIT = 2 };

int zo_ref_threads(void);

/* ---- random stream ---------------------------------------------------- */
void zo_ref_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);
float zo_ref_log_f32(float u);
void zo_ref_sincos_2pi_f32(uint32_t k24, float* s, float* c);
void zo_ref_gauss_pair(uint32_t x0, uint32_t x1, float* z0, float* z1);
void zo_ref_gauss_pairs(const uint32_t* x, uint64_t n_pairs, float* z);
void zo_ref_log_f32_array(const float* u, uint64_t n, float* out);
void zo_ref_sincos_2pi_array(const uint32_t* k24, uint64_t n, float* s, float* c);
float zo_ref_probe_value(int32_t kind, uint64_t seed, uint32_t i, uint64_t j);
void zo_ref_probe(int32_t kind, uint64_t seed, uint32_t i, uint64_t j0, uint64_t n, float* out);

/* ---- model layout ----------------------------------------------------- */
uint64_t zo_ref_param_count(const zo_ref_config* cfg);
/* offsets[0] = EMB; for layer l: offsets[1+3l] = W_ih, [2+3l] = W_hh, [3+3l] = b;
 * offsets[1+3L] = W_out, offsets[2+3L] = b_out, offsets[3+3L] = P. */
int zo_ref_layout(const zo_ref_config* cfg, uint64_t* offsets, int32_t n_offsets);

/* ---- the step ---------------------------------------------------------- */
int zo_ref_init(const zo_ref_config* cfg, void* theta, uint64_t seed);
int zo_ref_materialise(const zo_ref_config* cfg, const void* theta, uint64_t seed, uint32_t i,
                       double signed_eps, int32_t negate, double* w_out);
double zo_ref_lstm_loss(const zo_ref_config* cfg, const double* w, const int32_t* tokens,
                        const uint8_t* mask, int32_t B, int32_t C, int32_t tok_stride,
                        double* token_losses);
int zo_ref_perturbed_losses_ex(const zo_ref_config* cfg, const void* theta, uint64_t seed,
                               float eps, int32_t N, uint32_t i0, const int32_t* tokens,
                               const uint8_t* mask, int32_t B, int32_t C, int32_t negate,
                               double* Lplus, double* Lminus);
int zo_ref_perturbed_losses(const zo_ref_config* cfg, const void* theta, uint64_t seed, float eps,
                            int32_t N, uint32_t i0, const int32_t* tokens, const uint8_t* mask,
                            int32_t B, int32_t C, float* Lplus, float* Lminus);
float zo_ref_update_coeff(float lr, int32_t N, float Lplus, float Lminus, float eps);
int zo_ref_update(const zo_ref_config* cfg, void* theta, uint64_t seed, float eps, float lr,
                  int32_t N, uint32_t i0, const float* Lplus, const float* Lminus);

/* Forward differences (Eq. 1): L[n] = L(theta + eps z_{i0+n}), *L0 = L(theta)
 * (double). Update: c_n = fp32((lr/N)(L[n] - L0)/eps), then as zo_ref_update. */
int zo_ref_fd_losses(const zo_ref_config* cfg, const void* theta, uint64_t seed, float eps, int32_t N,
                     uint32_t i0, const int32_t* tokens, const uint8_t* mask, int32_t B, int32_t C,
                     double* L, double* L0);
float zo_ref_fd_update_coeff(float lr, int32_t N, float L, float L0, float eps);
int zo_ref_fd_update(const zo_ref_config* cfg, void* theta, uint64_t seed, float eps, float lr, int32_t N,
                     uint32_t i0, const float* L, float L0);
int zo_ref_update_sampled(const zo_ref_config* cfg, const void* theta, uint64_t seed, float eps,
                          float lr, int32_t N, uint32_t i0, const float* Lplus,
                          const float* Lminus, const uint64_t* idx, uint64_t n_idx, void* out);

/* ---- the estimator over an arbitrary loss (for closed-form checks) ---- */
typedef double (*zo_ref_loss_fn)(const double* w, uint64_t P, void* ctx);
int zo_ref_cd_losses_generic(uint64_t P, const double* theta, int32_t kind, uint64_t seed,
                             double eps, int32_t N, uint32_t i0, int32_t negate, zo_ref_loss_fn f,
                             void* ctx, double* Lplus, double* Lminus);
void zo_ref_cd_gradient(uint64_t P, int32_t kind, uint64_t seed, double eps, int32_t N,
                        uint32_t i0, const double* Lplus, const double* Lminus, double* g);

#ifdef __cplusplus
}
#endif
#endif
