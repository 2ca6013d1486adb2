/*
 * CPU oracle for one CD-RGE training step of a stacked-LSTM language model.
 *
 * TEST INFRASTRUCTURE ONLY: loaded by the tests, the smoke check and the
 * benchmark's CPU-baseline leg, never by the product path. It shares no code,
 * header, table or constant generator with the GPU path.
 *
 * Build: plain C11, -O2 -ffp-contract=off, no fast-math (see build.py next to
 * this file). Floating point is double except where the random-number
 * contract fixes fp32 operations (the probe and init transforms), which are
 * written out as single fp32 operations so that each one rounds once.
 *
 * Parity pins (tests/test_oracle_*.py):
 *   Philox4x32-10 ........ two independent installed implementations
 *                          (PyTorch's and rocRAND's source headers), live.
 *   log / sincos / sqrt .. libm in double, exhaustive over all 2^24 inputs.
 *   Rademacher probe ..... values exactly +-1, |z|^2 == P, moments.
 *   Gaussian probe ....... moments and a Kolmogorov-Smirnov test.
 *   init ................. range and moments of U(-1/sqrt(H), 1/sqrt(H)).
 *   forward + loss ....... zero weights give ln V; a bias-only closed-form
 *                          recurrence; torch.nn.LSTM / cross_entropy (CPU, fp64).
 *   estimator ............ exactness on a quadratic (Eq. 2: the even terms
 *                          cancel); convergence to a brute-force gradient as
 *                          N grows with the variance (P-1)/N of Section 2;
 *                          z -> -z swaps L+ and L- bit-exactly.
 *   update ............... L+ == L- leaves theta unchanged; N == 1 closed form;
 *                          linearity in the coefficients.
 */
#include "zo_oracle.h"

#include <math.h>
#include <omp.h>
#include <stdlib.h>
#include <string.h>

/* Threads the OpenMP loops of this library use (for reporting timings). */
int zo_ref_threads(void) { return omp_get_max_threads(); }

/* ======================================================================= */
/* Philox4x32-10 (Salmon et al., SC'11): 10 rounds of the 4x32 S-box with   */
/* multipliers 0xD2511F53 and 0xCD9E8D57 and Weyl key increments            */
/* 0x9E3779B9 and 0xBB67AE85.                                                */
/* ======================================================================= */
void zo_ref_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
    uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; ++round) {
        uint64_t p0 = (uint64_t)0xD2511F53u * (uint64_t)c0;
        uint64_t p1 = (uint64_t)0xCD9E8D57u * (uint64_t)c2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t n0 = hi1 ^ c1 ^ k0;
        uint32_t n1 = lo1;
        uint32_t n2 = hi0 ^ c3 ^ k1;
        uint32_t n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

static void philox_block(uint64_t seed, uint64_t blk, uint32_t i, uint32_t tag, uint32_t out[4]) {
    uint32_t ctr[4] = {(uint32_t)blk, (uint32_t)(blk >> 32), i, tag};
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    zo_ref_philox4x32_10(ctr, key, out);
}

/* ======================================================================= */
/* Normal probes (Section 2 evaluates N(0,1) probes). Box-Muller (1958):     */
/*   z0 = sqrt(-2 ln u1) cos(2 pi u2),  z1 = sqrt(-2 ln u1) sin(2 pi u2),    */
/* with u1 = ((x0 >> 8) + 1) 2^-24 in (0, 1] and u2 = (x1 >> 8) 2^-24 in     */
/* [0, 1). ln and sin/cos are fixed fp32 operation sequences so that every   */
/* implementation of the contract produces the same bits.                   */
/* ======================================================================= */
static float f32_from_bits(uint32_t b) { float f; memcpy(&f, &b, 4); return f; }
static uint32_t bits_from_f32(float f) { uint32_t b; memcpy(&b, &f, 4); return b; }

/* ln(u) for normal u in (0, 1]: u = 2^e m with m in (sqrt(1/2), sqrt(2)],
 * ln m = 2 atanh(s), s = (m - 1)/(m + 1), atanh series through s^9. */
float zo_ref_log_f32(float u) {
    uint32_t b = bits_from_f32(u);
    int e = (int)((b >> 23) & 0xFFu) - 127;
    float m = f32_from_bits((b & 0x007FFFFFu) | 0x3F800000u);
    /* 0x3FB504F3 is the largest float not above sqrt(2). */
    if (m > f32_from_bits(0x3FB504F3u)) {
        m = m * 0.5f;
        e = e + 1;
    }
    float num = m - 1.0f;
    float den = m + 1.0f;
    float s = num / den;
    float s2 = s * s;
    float p = (float)(2.0 / 9.0);
    p = p * s2;
    p = p + (float)(2.0 / 7.0);
    p = p * s2;
    p = p + (float)(2.0 / 5.0);
    p = p * s2;
    p = p + (float)(2.0 / 3.0);
    p = p * s2;
    p = p + 2.0f;
    float lnm = s * p;
    float ef = (float)e;
    const float ln2_hi = f32_from_bits(0x3F317200u); /* 0.693145751953125, 16 significant bits */
    const float ln2_lo = (float)(0.6931471805599453094 - 0.693145751953125);
    float lo = ef * ln2_lo;
    lo = lo + lnm;
    float hi = ef * ln2_hi;
    return hi + lo;
}

/* sin and cos of 2 pi k 2^-24 for a 24-bit integer k. The angle is split as
 * q quarter turns plus d quarter turns, d in [-1/2, 1/2) (exact integer
 * arithmetic), phi = d * (pi/2) in [-pi/4, pi/4), then Taylor series:
 * sin through phi^9, cos through phi^10. */
void zo_ref_sincos_2pi_f32(uint32_t k24, float* s_out, float* c_out) {
    int32_t k = (int32_t)(k24 & 0xFFFFFFu);
    int32_t qn = (k + (1 << 21)) >> 22;      /* nearest quarter turn, 0..4 */
    int32_t dk = k - (qn << 22);             /* in [-2^21, 2^21) */
    int q = qn & 3;
    float d = (float)dk * f32_from_bits(0x34800000u); /* * 2^-22, exact */
    float phi = d * (float)1.57079632679489661923;
    float p2 = phi * phi;
    /* sin(phi) = phi + phi*p2*(-1/3! + p2*(1/5! + p2*(-1/7! + p2/9!))) */
    float sp = (float)(1.0 / 362880.0);
    sp = sp * p2;
    sp = sp + (float)(-1.0 / 5040.0);
    sp = sp * p2;
    sp = sp + (float)(1.0 / 120.0);
    sp = sp * p2;
    sp = sp + (float)(-1.0 / 6.0);
    sp = sp * p2;
    sp = sp * phi;
    float sn = phi + sp;
    /* cos(phi) = 1 + p2*(-1/2! + p2*(1/4! + p2*(-1/6! + p2*(1/8! - p2/10!)))) */
    float cp = (float)(-1.0 / 3628800.0);
    cp = cp * p2;
    cp = cp + (float)(1.0 / 40320.0);
    cp = cp * p2;
    cp = cp + (float)(-1.0 / 720.0);
    cp = cp * p2;
    cp = cp + (float)(1.0 / 24.0);
    cp = cp * p2;
    cp = cp + -0.5f;
    cp = cp * p2;
    float cs = 1.0f + cp;
    /* rotate by q quarter turns */
    float s, c;
    switch (q) {
        case 0: s = sn; c = cs; break;
        case 1: s = cs; c = -sn; break;
        case 2: s = -sn; c = -cs; break;
        default: s = -cs; c = sn; break;
    }
    *s_out = s;
    *c_out = c;
}

void zo_ref_gauss_pair(uint32_t x0, uint32_t x1, float* z0, float* z1) {
    float u1 = (float)((x0 >> 8) + 1u) * f32_from_bits(0x33800000u); /* * 2^-24 */
    float l = zo_ref_log_f32(u1);
    float r2 = -2.0f * l;
    float r = sqrtf(r2);
    float s, c;
    zo_ref_sincos_2pi_f32(x1 >> 8, &s, &c);
    *z0 = r * c;
    *z1 = r * s;
}

void zo_ref_gauss_pairs(const uint32_t* x, uint64_t n_pairs, float* z) {
    for (uint64_t p = 0; p < n_pairs; ++p) zo_ref_gauss_pair(x[2 * p], x[2 * p + 1], &z[2 * p], &z[2 * p + 1]);
}

void zo_ref_log_f32_array(const float* u, uint64_t n, float* out) {
    for (uint64_t t = 0; t < n; ++t) out[t] = zo_ref_log_f32(u[t]);
}

void zo_ref_sincos_2pi_array(const uint32_t* k24, uint64_t n, float* s, float* c) {
    for (uint64_t t = 0; t < n; ++t) zo_ref_sincos_2pi_f32(k24[t], &s[t], &c[t]);
}

/* ======================================================================= */
/* Probe element z_i[j] (Algorithm 2 draws one Bernoulli(1/2) sign per      */
/* parameter; here the sign is one Philox bit).                              */
/*   Rademacher: block j >> 7, word (j >> 5) & 3, bit j & 31; 1 -> +1.       */
/*   Gaussian:   block j >> 2, pair (j >> 1) & 1 uses words (2p, 2p+1),      */
/*               even j -> z0 (cosine), odd j -> z1 (sine).                  */
/* ======================================================================= */
static float probe_from_block(int32_t kind, const uint32_t x[4], uint64_t j) {
    if (kind == 0) {
        uint32_t w = x[(j >> 5) & 3u];
        return ((w >> (j & 31u)) & 1u) ? 1.0f : -1.0f;
    }
    uint32_t p = (uint32_t)((j >> 1) & 1u);
    float z0, z1;
    zo_ref_gauss_pair(x[2 * p], x[2 * p + 1], &z0, &z1);
    return (j & 1u) ? z1 : z0;
}

float zo_ref_probe_value(int32_t kind, uint64_t seed, uint32_t i, uint64_t j) {
    uint32_t x[4];
    if (kind == 0) philox_block(seed, j >> 7, i, ZO_REF_TAG_RADEMACHER, x);
    else philox_block(seed, j >> 2, i, ZO_REF_TAG_GAUSSIAN, x);
    return probe_from_block(kind, x, j);
}

/* Fills z_i[j0 .. j0+n). One Philox call per block, shared by the elements
 * of that block; elementwise the same as zo_ref_probe_value. */
void zo_ref_probe(int32_t kind, uint64_t seed, uint32_t i, uint64_t j0, uint64_t n, float* out) {
    const unsigned shift = kind == 0 ? 7u : 2u;
    const uint32_t tag = kind == 0 ? ZO_REF_TAG_RADEMACHER : ZO_REF_TAG_GAUSSIAN;
    int64_t blk_first = (int64_t)(j0 >> shift);
    int64_t blk_last = n ? (int64_t)((j0 + n - 1) >> shift) : blk_first - 1;
#pragma omp parallel for schedule(static) if (n >= (1u << 16))
    for (int64_t blk = blk_first; blk <= blk_last; ++blk) {
        uint32_t x[4];
        philox_block(seed, (uint64_t)blk, i, tag, x);
        uint64_t lo = (uint64_t)blk << shift, hi = ((uint64_t)blk + 1) << shift;
        if (lo < j0) lo = j0;
        if (hi > j0 + n) hi = j0 + n;
        for (uint64_t j = lo; j < hi; ++j) out[j - j0] = probe_from_block(kind, x, j);
    }
}

/* ======================================================================= */
/* Parameter layout (flat, row major). The paper stores theta as one flat   */
/* vector (Algorithm 1 input theta in R^d) and perturbs all of it            */
/* (Algorithm 2 loops over every theta_i).                                    */
/*   EMB[V][E]; per layer l: W_ih[4H][E_l], W_hh[4H][H], b[4H];             */
/*   W_out[V][H]; b_out[V].  E_0 = E, E_l = H for l >= 1.                    */
/*   Gate row blocks of W_ih, W_hh, b in the order i, f, g, o.               */
/* ======================================================================= */
static int cfg_ok(const zo_ref_config* cfg) {
    if (!cfg) return 0;
    if (cfg->n_layers < 1 || cfg->vocab < 1 || cfg->embed < 1 || cfg->hidden < 1) return 0;
    if (cfg->wdtype != 0 && cfg->wdtype != 1) return 0;
    if (cfg->probe != 0 && cfg->probe != 1) return 0;
    return 1;
}

int zo_ref_layout(const zo_ref_config* cfg, uint64_t* off, int32_t n_off) {
    if (!cfg_ok(cfg)) return ZO_REF_EINVAL;
    int32_t L = cfg->n_layers;
    if (n_off < 3 * L + 4) return ZO_REF_EINVAL;
    uint64_t V = (uint64_t)cfg->vocab, E = (uint64_t)cfg->embed, H = (uint64_t)cfg->hidden;
    uint64_t p = 0;
    off[0] = p;
    p += V * E;
    for (int32_t l = 0; l < L; ++l) {
        uint64_t El = l == 0 ? E : H;
        off[1 + 3 * l] = p; p += 4 * H * El;
        off[2 + 3 * l] = p; p += 4 * H * H;
        off[3 + 3 * l] = p; p += 4 * H;
    }
    off[1 + 3 * L] = p; p += V * H;
    off[2 + 3 * L] = p; p += V;
    off[3 + 3 * L] = p;
    return ZO_REF_OK;
}

uint64_t zo_ref_param_count(const zo_ref_config* cfg) {
    if (!cfg_ok(cfg)) return 0;
    uint64_t off[3 * 64 + 4];
    if (cfg->n_layers > 64) return 0;
    zo_ref_layout(cfg, off, 3 * 64 + 4);
    return off[3 * cfg->n_layers + 3];
}

/* ---- bf16 storage ----------------------------------------------------- */
static float bf16_to_f32(uint16_t h) { return f32_from_bits((uint32_t)h << 16); }
static uint16_t f32_to_bf16_rne(float f) {
    uint32_t b = bits_from_f32(f);
    if ((b & 0x7F800000u) == 0x7F800000u && (b & 0x007FFFFFu)) return (uint16_t)((b >> 16) | 0x40u);
    uint32_t lsb = (b >> 16) & 1u;
    b += 0x7FFFu + lsb;
    return (uint16_t)(b >> 16);
}
static double theta_at(const zo_ref_config* cfg, const void* theta, uint64_t j) {
    if (cfg->wdtype == 1) return (double)bf16_to_f32(((const uint16_t*)theta)[j]);
    return (double)((const float*)theta)[j];
}

/* ======================================================================= */
/* Initialisation: every parameter ~ U(-1/sqrt(H), 1/sqrt(H)).               */
/*   Philox tag 2, block j >> 2, word j & 3; m = word >> 8 (24 bits);        */
/*   v = (2m + 1 - 2^24) 2^-24 (exact, symmetric in (-1, 1));                */
/*   a = fp32(1/sqrt(H)) (double then one rounding); theta_j = fp32(v * a);  */
/*   bf16 weights take the round-to-nearest-even of that fp32 value.         */
/* ======================================================================= */
int zo_ref_init(const zo_ref_config* cfg, void* theta, uint64_t seed) {
    if (!cfg_ok(cfg) || !theta) return ZO_REF_EINVAL;
    uint64_t P = zo_ref_param_count(cfg);
    float a = (float)(1.0 / sqrt((double)cfg->hidden));
    int64_t nblk = (int64_t)((P + 3) >> 2);
#pragma omp parallel for schedule(static) if (P >= (1u << 16))
    for (int64_t blk = 0; blk < nblk; ++blk) {
        uint32_t x[4];
        philox_block(seed, (uint64_t)blk, 0u, ZO_REF_TAG_INIT, x);
        for (uint64_t w = 0; w < 4; ++w) {
            uint64_t j = ((uint64_t)blk << 2) + w;
            if (j >= P) break;
            int32_t m = (int32_t)(x[w] >> 8);
            float v = (float)(2 * m + 1 - (1 << 24)) * f32_from_bits(0x33800000u);
            float t = v * a;
            if (cfg->wdtype == 1) ((uint16_t*)theta)[j] = f32_to_bf16_rne(t);
            else ((float*)theta)[j] = t;
        }
    }
    return ZO_REF_OK;
}

/* ======================================================================= */
/* theta^{(i,s)} = theta + s eps z_i, materialised in double from the        */
/* pristine theta (not by the in-place +eps, -2eps, +eps walk of Algorithm   */
/* 1, which is the same point in exact arithmetic). negate != 0 uses -z_i.   */
/* ======================================================================= */
int zo_ref_materialise(const zo_ref_config* cfg, const void* theta, uint64_t seed, uint32_t i,
                       double signed_eps, int32_t negate, double* w) {
    if (!cfg_ok(cfg) || !theta || !w) return ZO_REF_EINVAL;
    uint64_t P = zo_ref_param_count(cfg);
    const int32_t kind = cfg->probe;
    const unsigned shift = kind == 0 ? 7u : 2u;
    const uint32_t tag = kind == 0 ? ZO_REF_TAG_RADEMACHER : ZO_REF_TAG_GAUSSIAN;
    int64_t nblk = (int64_t)((P + ((1u << shift) - 1)) >> shift);
#pragma omp parallel for schedule(static) if (P >= (1u << 16))
    for (int64_t blk = 0; blk < nblk; ++blk) {
        uint32_t x[4];
        philox_block(seed, (uint64_t)blk, i, tag, x);
        for (uint64_t j = (uint64_t)blk << shift; j < (((uint64_t)blk + 1) << shift) && j < P; ++j) {
            double z = (double)probe_from_block(kind, x, j);
            if (negate) z = -z;
            w[j] = theta_at(cfg, theta, j) + signed_eps * z;
        }
    }
    return ZO_REF_OK;
}

/* ======================================================================= */
/* Loss of the LSTM language model at weights w (double).                    */
/* Standard LSTM with forget gate, one bias per layer, zero initial state:   */
/*   a = W_ih x + W_hh h + b;  i = sig(a_i), f = sig(a_f), g = tanh(a_g),    */
/*   o = sig(a_o);  c <- f c + i g;  h <- o tanh(c);  x <- h (next layer).  */
/* Head y = W_out h_top + b_out; per position l = logsumexp(y) - y[target]  */
/* (nats). tokens[b][0..C] (row stride tok_stride), input tokens[b][t],     */
/* target tokens[b][t+1]; mask[b][t] (NULL = all ones). Returns the masked  */
/* mean sum(m l)/sum(m) (0 if no position is masked in).                     */
/* token_losses[b][t] (optional) receives l for every position.              */
/* ======================================================================= */
static double sigmoid(double x) { return 1.0 / (1.0 + exp(-x)); }

static void lstm_sequence(const zo_ref_config* cfg, const uint64_t* off, const double* w,
                          const int32_t* tok, const uint8_t* mask, int32_t C, double* ell,
                          int inner_parallel) {
    const int32_t L = cfg->n_layers, V = cfg->vocab, E = cfg->embed, H = cfg->hidden;
    double* h = calloc((size_t)L * H, sizeof(double));
    double* c = calloc((size_t)L * H, sizeof(double));
    double* a = malloc(sizeof(double) * 4 * (size_t)H);
    double* x = malloc(sizeof(double) * (size_t)(E > H ? E : H));
    double* y = malloc(sizeof(double) * (size_t)V);
    for (int32_t t = 0; t < C; ++t) {
        const double* emb = w + off[0] + (uint64_t)tok[t] * (uint64_t)E;
        for (int32_t e = 0; e < E; ++e) x[e] = emb[e];
        int32_t xin = E;
        for (int32_t l = 0; l < L; ++l) {
            const double* Wih = w + off[1 + 3 * l];
            const double* Whh = w + off[2 + 3 * l];
            const double* bl = w + off[3 + 3 * l];
            double* hl = h + (size_t)l * H;
            double* cl = c + (size_t)l * H;
#pragma omp parallel for schedule(static) if (inner_parallel && (int64_t)H * (xin + H) >= (1 << 16))
            for (int32_t n = 0; n < 4 * H; ++n) {
                double acc = bl[n];
                const double* wr = Wih + (uint64_t)n * (uint64_t)xin;
                for (int32_t k = 0; k < xin; ++k) acc += wr[k] * x[k];
                const double* ur = Whh + (uint64_t)n * (uint64_t)H;
                for (int32_t k = 0; k < H; ++k) acc += ur[k] * hl[k];
                a[n] = acc;
            }
            for (int32_t u = 0; u < H; ++u) {
                double ig = sigmoid(a[u]);
                double fg = sigmoid(a[H + u]);
                double gg = tanh(a[2 * H + u]);
                double og = sigmoid(a[3 * H + u]);
                cl[u] = fg * cl[u] + ig * gg;
                hl[u] = og * tanh(cl[u]);
            }
            for (int32_t u = 0; u < H; ++u) x[u] = hl[u];
            xin = H;
        }
        if (mask && !mask[t]) {
            ell[t] = 0.0;
            continue;
        }
        const double* Wo = w + off[1 + 3 * L];
        const double* bo = w + off[2 + 3 * L];
#pragma omp parallel for schedule(static) if (inner_parallel && (int64_t)V * H >= (1 << 16))
        for (int32_t v = 0; v < V; ++v) {
            double acc = bo[v];
            const double* wr = Wo + (uint64_t)v * (uint64_t)H;
            for (int32_t k = 0; k < H; ++k) acc += wr[k] * x[k];
            y[v] = acc;
        }
        double ymax = -INFINITY;
        for (int32_t v = 0; v < V; ++v)
            if (y[v] > ymax) ymax = y[v];
        double se = 0.0;
        for (int32_t v = 0; v < V; ++v) se += exp(y[v] - ymax);
        ell[t] = ymax + log(se) - y[tok[t + 1]];
    }
    free(h); free(c); free(a); free(x); free(y);
}

double zo_ref_lstm_loss(const zo_ref_config* cfg, const double* w, const int32_t* tokens,
                        const uint8_t* mask, int32_t B, int32_t C, int32_t tok_stride,
                        double* token_losses) {
    uint64_t off[3 * 64 + 4];
    if (!cfg_ok(cfg) || cfg->n_layers > 64 || B < 1 || C < 1) return NAN;
    zo_ref_layout(cfg, off, 3 * 64 + 4);
    if (tok_stride <= 0) tok_stride = C + 1;
    double* ell = malloc(sizeof(double) * (size_t)B * (size_t)C);
    /* sequences are independent: spread them over threads when there are
     * enough of them, otherwise spread the rows of each matrix product */
    int outer = B >= omp_get_max_threads() && (uint64_t)B * (uint64_t)C * zo_ref_param_count(cfg) >= (1u << 20);
#pragma omp parallel for schedule(dynamic, 1) if (outer)
    for (int32_t b = 0; b < B; ++b)
        lstm_sequence(cfg, off, w, tokens + (size_t)b * tok_stride,
                      mask ? mask + (size_t)b * C : NULL, C, ell + (size_t)b * C, !outer);
    double sum = 0.0, cnt = 0.0;
    for (int32_t b = 0; b < B; ++b)
        for (int32_t t = 0; t < C; ++t) {
            int m = mask ? mask[(size_t)b * C + t] != 0 : 1;
            if (m) { sum += ell[(size_t)b * C + t]; cnt += 1.0; }
            if (token_losses) token_losses[(size_t)b * C + t] = m ? ell[(size_t)b * C + t] : 0.0;
        }
    free(ell);
    return cnt > 0.0 ? sum / cnt : 0.0;
}

/* ======================================================================= */
/* Losses of Algorithm 1: for i = i0 .. i0+N-1, L+_i = L(theta + eps z_i) and */
/* L-_i = L(theta - eps z_i).                                                */
/* ======================================================================= */
static int tokens_ok(const zo_ref_config* cfg, const int32_t* tokens, int32_t B, int32_t C) {
    for (int64_t t = 0; t < (int64_t)B * (C + 1); ++t)
        if (tokens[t] < 0 || tokens[t] >= cfg->vocab) return 0;
    return 1;
}

int zo_ref_perturbed_losses_ex(const zo_ref_config* cfg, const void* theta, uint64_t seed,
                               float eps, int32_t N, uint32_t i0, const int32_t* tokens,
                               const uint8_t* mask, int32_t B, int32_t C, int32_t negate,
                               double* Lplus, double* Lminus) {
    if (!cfg_ok(cfg) || !theta || !tokens || !Lplus || !Lminus) return ZO_REF_EINVAL;
    if (N < 1 || B < 1 || C < 1 || !(eps > 0.0f) || !isfinite(eps)) return ZO_REF_EINVAL;
    if (!tokens_ok(cfg, tokens, B, C)) return ZO_REF_EINVAL;
    uint64_t P = zo_ref_param_count(cfg);
    double* w = malloc(sizeof(double) * P);
    if (!w) return ZO_REF_ENOMEM;
    for (int32_t n = 0; n < N; ++n) {
        zo_ref_materialise(cfg, theta, seed, i0 + (uint32_t)n, (double)eps, negate, w);
        Lplus[n] = zo_ref_lstm_loss(cfg, w, tokens, mask, B, C, C + 1, NULL);
        zo_ref_materialise(cfg, theta, seed, i0 + (uint32_t)n, -(double)eps, negate, w);
        Lminus[n] = zo_ref_lstm_loss(cfg, w, tokens, mask, B, C, C + 1, NULL);
    }
    free(w);
    return ZO_REF_OK;
}

int zo_ref_perturbed_losses(const zo_ref_config* cfg, const void* theta, uint64_t seed, float eps,
                            int32_t N, uint32_t i0, const int32_t* tokens, const uint8_t* mask,
                            int32_t B, int32_t C, float* Lplus, float* Lminus) {
    if (N < 1) return ZO_REF_EINVAL;
    double* lp = malloc(sizeof(double) * (size_t)N);
    double* lm = malloc(sizeof(double) * (size_t)N);
    int st = zo_ref_perturbed_losses_ex(cfg, theta, seed, eps, N, i0, tokens, mask, B, C, 0, lp, lm);
    if (st == ZO_REF_OK)
        for (int32_t n = 0; n < N; ++n) { Lplus[n] = (float)lp[n]; Lminus[n] = (float)lm[n]; }
    free(lp); free(lm);
    return st;
}

/* ======================================================================= */
/* Update (Eq. 7 with a general step size; Algorithm 1's final loop):        */
/*   c_i = (lr / N) (L+_i - L-_i) / (2 eps), in double, rounded to fp32 once; */
/*   theta_j <- theta_j - sum_i c_i z_i[j], summed in double in ascending i, */
/*   rounded once to the storage type (bf16: round to nearest even).         */
/* A non-finite loss skips the whole update (theta unchanged).               */
/* ======================================================================= */
float zo_ref_update_coeff(float lr, int32_t N, float Lplus, float Lminus, float eps) {
    double c = ((double)lr / (double)N) * (((double)Lplus - (double)Lminus) / (2.0 * (double)eps));
    return (float)c;
}

static int update_args(const zo_ref_config* cfg, float eps, float lr, int32_t N,
                       const float* Lplus, const float* Lminus, float** coeff) {
    if (!cfg_ok(cfg) || !Lplus || !Lminus || N < 1) return ZO_REF_EINVAL;
    if (!(eps > 0.0f) || !isfinite(eps) || !isfinite(lr)) return ZO_REF_EINVAL;
    for (int32_t n = 0; n < N; ++n)
        if (!isfinite(Lplus[n]) || !isfinite(Lminus[n])) return ZO_REF_ENONFINITE;
    float* c = malloc(sizeof(float) * (size_t)N);
    for (int32_t n = 0; n < N; ++n) c[n] = zo_ref_update_coeff(lr, N, Lplus[n], Lminus[n], eps);
    *coeff = c;
    return ZO_REF_OK;
}

static void update_one(const zo_ref_config* cfg, const void* theta_in, void* theta_out,
                       uint64_t j, uint64_t o, double acc) {
    double t = theta_at(cfg, theta_in, j) - acc;
    if (cfg->wdtype == 1) ((uint16_t*)theta_out)[o] = f32_to_bf16_rne((float)t);
    else ((float*)theta_out)[o] = (float)t;
}

static int apply_update(const zo_ref_config* cfg, void* theta, uint64_t seed, int32_t N, uint32_t i0,
                        float* coeff);

int zo_ref_update(const zo_ref_config* cfg, void* theta, uint64_t seed, float eps, float lr,
                  int32_t N, uint32_t i0, const float* Lplus, const float* Lminus) {
    float* coeff = NULL;
    if (!theta) return ZO_REF_EINVAL;
    int st = update_args(cfg, eps, lr, N, Lplus, Lminus, &coeff);
    if (st != ZO_REF_OK) return st;
    return apply_update(cfg, theta, seed, N, i0, coeff);
}

/* theta_j <- theta_j - sum_n coeff[n] z_{i0+n}[j] (double, ascending n), one
 * rounding to the storage type; frees coeff. */
static int apply_update(const zo_ref_config* cfg, void* theta, uint64_t seed, int32_t N, uint32_t i0,
                        float* coeff) {
    uint64_t P = zo_ref_param_count(cfg);
    double* acc = calloc(P, sizeof(double));
    float* z = malloc(sizeof(float) * P);
    if (!acc || !z) { free(acc); free(z); free(coeff); return ZO_REF_ENOMEM; }
    for (int32_t n = 0; n < N; ++n) {
        zo_ref_probe(cfg->probe, seed, i0 + (uint32_t)n, 0, P, z);
#pragma omp parallel for schedule(static) if (P >= (1u << 16))
        for (int64_t j = 0; j < (int64_t)P; ++j) acc[j] += (double)coeff[n] * (double)z[j];
    }
#pragma omp parallel for schedule(static) if (P >= (1u << 16))
    for (int64_t j = 0; j < (int64_t)P; ++j) update_one(cfg, theta, theta, (uint64_t)j, (uint64_t)j, acc[j]);
    free(acc); free(z); free(coeff);
    return ZO_REF_OK;
}

/* The same update evaluated only at the listed indices (for checks at sizes
 * where a full pass is too slow); out[k] receives the new theta[idx[k]]. */
int zo_ref_update_sampled(const zo_ref_config* cfg, const void* theta, uint64_t seed, float eps,
                          float lr, int32_t N, uint32_t i0, const float* Lplus,
                          const float* Lminus, const uint64_t* idx, uint64_t n_idx, void* out) {
    float* coeff = NULL;
    if (!theta || !idx || !out) return ZO_REF_EINVAL;
    int st = update_args(cfg, eps, lr, N, Lplus, Lminus, &coeff);
    if (st != ZO_REF_OK) return st;
    uint64_t P = zo_ref_param_count(cfg);
    for (uint64_t k = 0; k < n_idx; ++k) {
        if (idx[k] >= P) { free(coeff); return ZO_REF_EINVAL; }
        double acc = 0.0;
        for (int32_t n = 0; n < N; ++n)
            acc += (double)coeff[n] * (double)zo_ref_probe_value(cfg->probe, seed, i0 + (uint32_t)n, idx[k]);
        update_one(cfg, theta, out, idx[k], k, acc);
    }
    free(coeff);
    return ZO_REF_OK;
}

/* ======================================================================= */
/* Forward differences (Eq. 1, the one-sided difference the paper compares  */
/* with the central one): one clean loss L0 = L(theta) and N losses          */
/* L_n = L(theta + eps z_{i0+n}); the update uses                            */
/*   c_n = (lr / N) (L_n - L0) / eps  (double, rounded to fp32)              */
/* and the same sum over probes as zo_ref_update.                            */
/* ======================================================================= */
int zo_ref_fd_losses(const zo_ref_config* cfg, const void* theta, uint64_t seed, float eps, int32_t N,
                     uint32_t i0, const int32_t* tokens, const uint8_t* mask, int32_t B, int32_t C,
                     double* L, double* L0) {
    if (!cfg_ok(cfg) || !theta || !tokens || !L || !L0) return ZO_REF_EINVAL;
    if (N < 1 || B < 1 || C < 1 || !(eps > 0.0f) || !isfinite(eps)) return ZO_REF_EINVAL;
    if (!tokens_ok(cfg, tokens, B, C)) return ZO_REF_EINVAL;
    uint64_t P = zo_ref_param_count(cfg);
    double* w = malloc(sizeof(double) * P);
    if (!w) return ZO_REF_ENOMEM;
    for (uint64_t j = 0; j < P; ++j) w[j] = theta_at(cfg, theta, j);
    *L0 = zo_ref_lstm_loss(cfg, w, tokens, mask, B, C, C + 1, NULL);
    for (int32_t n = 0; n < N; ++n) {
        zo_ref_materialise(cfg, theta, seed, i0 + (uint32_t)n, (double)eps, 0, w);
        L[n] = zo_ref_lstm_loss(cfg, w, tokens, mask, B, C, C + 1, NULL);
    }
    free(w);
    return ZO_REF_OK;
}

float zo_ref_fd_update_coeff(float lr, int32_t N, float L, float L0, float eps) {
    double c = ((double)lr / (double)N) * (((double)L - (double)L0) / (double)eps);
    return (float)c;
}

int zo_ref_fd_update(const zo_ref_config* cfg, void* theta, uint64_t seed, float eps, float lr, int32_t N,
                     uint32_t i0, const float* L, float L0) {
    if (!cfg_ok(cfg) || !theta || !L || N < 1) return ZO_REF_EINVAL;
    if (!(eps > 0.0f) || !isfinite(eps) || !isfinite(lr)) return ZO_REF_EINVAL;
    if (!isfinite(L0)) return ZO_REF_ENONFINITE;
    for (int32_t n = 0; n < N; ++n)
        if (!isfinite(L[n])) return ZO_REF_ENONFINITE;
    float* c = malloc(sizeof(float) * (size_t)N);
    if (!c) return ZO_REF_ENOMEM;
    for (int32_t n = 0; n < N; ++n) c[n] = zo_ref_fd_update_coeff(lr, N, L[n], L0, eps);
    return apply_update(cfg, theta, seed, N, i0, c);
}

/* ======================================================================= */
/* The estimator of Eq. 2 averaged over N probes (Section 2), on any loss.   */
/* ======================================================================= */
int zo_ref_cd_losses_generic(uint64_t P, const double* theta, int32_t kind, uint64_t seed,
                             double eps, int32_t N, uint32_t i0, int32_t negate, zo_ref_loss_fn f,
                             void* ctx, double* Lplus, double* Lminus) {
    if (!theta || !f || N < 1 || (kind != 0 && kind != 1)) return ZO_REF_EINVAL;
    double* w = malloc(sizeof(double) * P);
    float* z = malloc(sizeof(float) * P);
    for (int32_t n = 0; n < N; ++n) {
        zo_ref_probe(kind, seed, i0 + (uint32_t)n, 0, P, z);
        for (uint64_t j = 0; j < P; ++j) w[j] = theta[j] + eps * (negate ? -(double)z[j] : (double)z[j]);
        Lplus[n] = f(w, P, ctx);
        for (uint64_t j = 0; j < P; ++j) w[j] = theta[j] - eps * (negate ? -(double)z[j] : (double)z[j]);
        Lminus[n] = f(w, P, ctx);
    }
    free(w); free(z);
    return ZO_REF_OK;
}

/* g = (1/N) sum_i (L+_i - L-_i) / (2 eps) z_i, in double. */
void zo_ref_cd_gradient(uint64_t P, int32_t kind, uint64_t seed, double eps, int32_t N,
                        uint32_t i0, const double* Lplus, const double* Lminus, double* g) {
    float* z = malloc(sizeof(float) * P);
    for (uint64_t j = 0; j < P; ++j) g[j] = 0.0;
    for (int32_t n = 0; n < N; ++n) {
        double d = (Lplus[n] - Lminus[n]) / (2.0 * eps);
        zo_ref_probe(kind, seed, i0 + (uint32_t)n, 0, P, z);
        for (uint64_t j = 0; j < P; ++j) g[j] += d * (double)z[j];
    }
    for (uint64_t j = 0; j < P; ++j) g[j] /= (double)N;
    free(z);
}
