/*
 * zo.h - C ABI of the MI355X (gfx950) library for one Central-Difference
 * Random-vector Gradient Estimation (CD-RGE) training step of a stacked-LSTM
 * language model (Chaubard & Kochenderfer, "Scaling Recurrent Neural Networks
 * to a Billion Parameters with Zero-Order Optimization").
 *
 * One step, as stated in the paper (Section 2, Eq. 2 and Eq. 7; Section 3,
 * Algorithm 1 and Algorithm 2):
 *   for every probe i: L+_i = L(theta + eps z_i, x),  L-_i = L(theta - eps z_i, x)
 *   theta <- theta - lr * (1/N) * sum_i (L+_i - L-_i) / (2 eps) * z_i
 * With lr == eps this is Eq. 7 (the paper ties the step size to eps).
 *
 * Conventions shared by every call
 * --------------------------------
 * Device pointers. Every buffer argument (theta, tokens, mask, losses,
 * workspace, out) is a device pointer on the current HIP device, allocated
 * and owned by the caller. The library never allocates, frees or retains
 * caller memory. It keeps no state between calls apart from the optional
 * kernel-timing records (zo_profile_enable) and, for zo_perturbed_losses_noalloc,
 * one fixed scratch array per device.
 *
 * Streams. `stream` is a hipStream_t (NULL = the default stream). Every call
 * only enqueues work on that stream and returns; outputs are valid once the
 * stream has been synchronised. Calls on distinct streams with distinct
 * workspaces may run concurrently.
 *
 * Errors. Calls return a zo_status. Arguments are validated on the host
 * before anything is enqueued; on an error nothing is enqueued and no caller
 * buffer is touched. zo_last_error() returns a thread-local description of
 * the last failure. No C++ exception crosses this interface.
 *
 * Parameter vector theta (flat, row major, one contiguous array of P
 * elements, fp32 or bf16 according to zo_config.wdtype). The paper keeps the
 * model as one flat vector and perturbs every element of it (Algorithm 1
 * input theta in R^d; Algorithm 2 loops over all of theta):
 *   EMB[V][E]
 *   for l = 0..L-1: W_ih[4H][E_l], W_hh[4H][H], b[4H]   (E_0 = E, E_l = H)
 *                   gate row blocks in the order i, f, g, o
 *   W_out[V][H], b_out[V]
 *
 * Probes. z_i[j] is regenerated from (seed, i, j) by Philox4x32-10 (Salmon
 * et al., SC'11) with key (seed low word, seed high word) and counter
 * (block low, block high, i, tag):
 *   Rademacher (tag 0): block j>>7, word (j>>5)&3, bit j&31; bit 1 -> +1,
 *                       bit 0 -> -1 (Section 2; Algorithm 2's Bernoulli sign);
 *   normal     (tag 1): block j>>2; words (0,1) give elements 4b, 4b+1 and
 *                       words (2,3) give 4b+2, 4b+3 by Box-Muller with fixed
 *                       fp32 operation sequences for ln, sqrt and sin/cos of
 *                       2 pi k / 2^24 (Section 2 evaluates N(0,1) probes).
 * Perturbed weights theta +- eps z_i are never materialised.
 */
#ifndef ZO_H
#define ZO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    ZO_OK = 0,
    ZO_EINVAL = -1,     /* a null pointer, a non-positive size, eps <= 0, a non-finite lr ... */
    ZO_ESHAPE = -2,     /* a model shape the kernels do not support (see zo_config) */
    ZO_EDEVICE = -3,    /* a HIP runtime error, or no gfx950 device */
    ZO_ENOMEM = -4,     /* the workspace is smaller than zo_workspace_bytes_min() */
    ZO_ENONFINITE = -5  /* reserved: a non-finite loss (zo_update reports it through skipped_out) */
} zo_status;

enum { ZO_WFP32 = 0, ZO_WBF16 = 1 };
enum { ZO_RADEMACHER = 0, ZO_GAUSSIAN = 1 };

/* Model shape. All fields > 0; embed and hidden must be multiples of 32
 * (ZO_ESHAPE otherwise), and for zo_perturbed_losses with bf16 weights
 * multiples of 64; n_layers <= 64. wdtype: ZO_WFP32 or ZO_WBF16
 * (storage type of theta; bf16 runs every matrix product on fp16 operands
 * from an fp16 copy of the weights, with fp32 accumulation and fp32 cell
 * state, see "Products" below). probe: ZO_RADEMACHER or ZO_GAUSSIAN. */
typedef struct {
    int32_t n_layers;
    int32_t vocab;
    int32_t embed;
    int32_t hidden;
    int32_t wdtype;
    int32_t probe;
} zo_config;

/* Products (bf16 weights). Each perturbed product A.(W + s eps Z) runs on
 * fp16 MFMA operands in one of two forms:
 *   fused      acc += A . fp16(W + s eps z): the probe added to the fp16
 *              weight fragment in registers and rounded once (one matrix
 *              stream). The rounding costs each element up to half an fp16
 *              ulp of w, 2^-11 |w|, so the form is used only for
 *              eps >= ZO_BF16_FUSED_EPS_MIN (there, for |w| < 2^-5, at most
 *              1.6% of eps z per element, zero-mean across elements);
 *   two-stream acc += A . W, then acc += A . (s fp16(eps z)) into the same
 *              fp32 accumulator (twice the matrix work): the probe operand
 *              keeps eps z to 2^-11 relative, or to 2^-25 absolute where it is
 *              subnormal in fp16, so eps >= ZO_BF16_EPS_MIN keeps it within
 *              0.4% of eps per element.
 * Sign probes use +-fp16(eps) in both forms (a scale error of at most 2^-11,
 * or 0.4% at ZO_BF16_EPS_MIN, that is the same for every element). The
 * perturbed embedding rows are formed in fp32 and rounded once to fp16 in
 * both forms. zo_perturbed_losses chooses by eps (ZO_PRODUCTS_AUTO); the _ex
 * entry points take the form as an argument, for measurement. A bf16 call
 * with eps < ZO_BF16_EPS_MIN returns ZO_EINVAL. fp32 weights form
 * w +- eps z in fp32 (fused, one fp32 rounding); their two-stream form exists
 * for measurement only (central differences). */
#define ZO_BF16_FUSED_EPS_MIN 0x1p-10f /* 9.765625e-4 */
#define ZO_BF16_EPS_MIN 0x1p-17f       /* 7.62939453125e-6 */
enum { ZO_PRODUCTS_AUTO = 0, ZO_PRODUCTS_FUSED = 1, ZO_PRODUCTS_SPLIT = 2 };

/* Number of elements P of theta for this shape (layout above); 0 if the
 * configuration is invalid. Host only. */
size_t zo_param_count(const zo_config* cfg);

/* Bytes of device workspace zo_perturbed_losses (or zo_fd_losses) uses for N probes and a
 * batch of B sequences of C positions; 0 if the arguments are invalid.
 * Host only. With bf16 weights every workspace holds an fp16 copy of the
 * weight matrices (every W_ih, W_hh and W_out; P_g values), written once per
 * call. With normal probes this includes the probe cache, written once per
 * call and read by every timestep instead of regenerating the probe in every
 * tile (the results are bit-identical either way): N * P_g values of eps z
 * for fp32 weights; 2 * N * P_g fp16 values for bf16 weights, each probe's
 * perturbed weights fp16(w + fp16(eps z)) and fp16(w - fp16(eps z)) (fused
 * products), or fp16(eps z) (two-stream products). With
 * sign probes and bf16 weights it includes the sign-probe cache (below); with
 * sign probes and fp32 weights it equals zo_workspace_bytes_min. */
size_t zo_workspace_bytes(const zo_config* cfg, int32_t N, int32_t B, int32_t C);

/* The smallest workspace zo_perturbed_losses accepts: without the probe
 * cache (normal probes are then regenerated in every tile). A workspace of
 * at least zo_workspace_bytes() enables the cache. Host only. */
size_t zo_workspace_bytes_min(const zo_config* cfg, int32_t N, int32_t B, int32_t C);

/* Initialisation: every parameter ~ U(-1/sqrt(H), 1/sqrt(H)), drawn from
 * Philox tag 2, block j>>2, word j&3 (m = word>>8, value (2m+1-2^24) 2^-24
 * times fp32(1/sqrt(H)); bf16 storage rounds that fp32 value to nearest
 * even). theta: device, P elements of the storage type. Setup, not part of
 * the step. */
int zo_init(const zo_config* cfg, void* theta, uint64_t seed, void* stream);

/* The 2N perturbed forward passes of one step (Algorithm 1, the loop over
 * the worker's probes; Eq. 2's two loss queries per probe).
 *   theta    device, P elements (read only)
 *   seed     Philox key of this step's probes; probe n uses index i0 + n
 *   eps      perturbation size, > 0 and finite (bf16 weights: >= ZO_BF16_EPS_MIN)
 *   N        number of probes (>= 1); 2N forward passes
 *   i0       global index of the first probe (a slice [i0, i0+N) of a larger
 *            set gives bit-identical losses to the same probes in the full set)
 *   tokens   device int32 [B][C+1], ids in [0, V): position t reads token
 *            tokens[b][t] and is scored on the next token tokens[b][t+1]
 *            (teacher forcing). Ids outside [0, V) are never used to address
 *            memory: an input id outside the range makes that sequence's
 *            states NaN from its position on, and a scored target id outside
 *            it makes that position's loss NaN, so the losses it reaches are
 *            not finite (zo_update then skips, see skipped_out); an id that
 *            only serves as an unscored target changes nothing. The call
 *            itself still returns ZO_OK: the ids are not read on the host.
 *   mask     device uint8 [B][C] or NULL (all positions scored)
 *   Lplus, Lminus  device fp32 [N]: the masked mean over (b, t) of the
 *            next-token cross-entropy in nats at theta + eps z and at
 *            theta - eps z (0 when the mask selects nothing)
 *   workspace, ws_bytes  device scratch of at least zo_workspace_bytes_min()
 *            (normal probes: at least zo_workspace_bytes() to use the probe
 *            cache; same results, fewer probe regenerations)
 * Returns ZO_OK, ZO_EINVAL, ZO_ESHAPE, ZO_ENOMEM or ZO_EDEVICE.
 * fp32 weights: each matrix product uses the perturbed weight tile
 * w +- eps z formed in LDS (one fp32 rounding). bf16 weights: the fused or
 * the two-stream products by eps (see "Products"). */
int zo_perturbed_losses(const zo_config* cfg, const void* theta, uint64_t seed, float eps,
                        int32_t N, uint32_t i0, const int32_t* tokens, const uint8_t* mask,
                        int32_t B, int32_t C, float* Lplus, float* Lminus, void* workspace,
                        size_t ws_bytes, void* stream);

/* zo_perturbed_losses with the form of the products given: ZO_PRODUCTS_AUTO
 * (as zo_perturbed_losses), ZO_PRODUCTS_FUSED or ZO_PRODUCTS_SPLIT (any
 * other value is ZO_EINVAL). For measuring one form against the other; the
 * eps floor of bf16 weights applies to both. */
int zo_perturbed_losses_ex(const zo_config* cfg, const void* theta, uint64_t seed, float eps,
                           int32_t N, uint32_t i0, const int32_t* tokens, const uint8_t* mask,
                           int32_t B, int32_t C, float* Lplus, float* Lminus, void* workspace,
                           size_t ws_bytes, int32_t products, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * zo_perturbed_losses without a workspace argument. The workspace is a fixed
 * device array of ZO_NOALLOC_WORKSPACE_BYTES inside the library, one per
 * device, held from the first call on that device until the process ends
 * (the probe cache is used when zo_workspace_bytes() fits in it as well).
 * The call allocates and frees nothing, and does no kernel timing. A shape
 * whose zo_workspace_bytes_min() exceeds the array returns ZO_ENOMEM before
 * anything is enqueued. Every call on a device shares that device's array:
 * calls that overlap on one device (concurrent streams or threads) race and
 * must be serialised by the caller. Each call clears what it reads before
 * writing it, so no state carries from one call to the next. Other arguments,
 * results and return codes as for zo_perturbed_losses. */
#define ZO_NOALLOC_WORKSPACE_BYTES (128u << 20)
int zo_perturbed_losses_noalloc(const zo_config* cfg, const void* theta, uint64_t seed, float eps,
                                int32_t N, uint32_t i0, const int32_t* tokens, const uint8_t* mask,
                                int32_t B, int32_t C, float* Lplus, float* Lminus, void* stream);

/* The update of Eq. 7 in its general form (Algorithm 1's closing loop):
 *   c_n = fp32( (lr / N) * (L+_n - L-_n) / (2 eps) )  (computed in double)
 *   theta_j <- theta_j - sum_{n=0}^{N-1} c_n z_{i0+n}[j]  (summed in fp32:
 *   Rademacher probes by groups of 8 in probe order, normal probes in
 *   ascending n; bf16 storage rounds the fp32 result to nearest even)
 * theta is read and written once, in place, and must be 16-byte aligned. Lplus and Lminus are device fp32
 * [N]. If any of them is not finite the update is skipped on the device,
 * theta is left bit-unchanged and, when skipped_out (device int32, may be
 * NULL) is given, *skipped_out is set to 1 (0 otherwise).
 * Returns ZO_OK, ZO_EINVAL, ZO_ESHAPE or ZO_EDEVICE. */
int zo_update(const zo_config* cfg, void* theta, uint64_t seed, float eps, float lr, int32_t N,
              uint32_t i0, const float* Lplus, const float* Lminus, int32_t* skipped_out,
              void* stream);

/* Sign-probe cache (bf16 weights with sign probes; the paper notes that sign
 * probes can be stored as bits). A workspace of at least zo_workspace_bytes()
 * holds, at byte offset zo_probe_bits_offset(cfg, N, B, C), the sign words of
 * the call's probes i0 .. i0+N-1 over the whole of theta: probe n's word w at
 * n * 4 * ceil(P / 128) + w (uint32) holds the signs of parameters 32 w ..
 * 32 w + 31, unshuffled: bit i set when z_{i0+n}[32 w + 2 i] = +1 and bit
 * 16 + i when z_{i0+n}[32 w + 2 i + 1] = +1 (i < 16). zo_perturbed_losses writes it once per call and its
 * kernels read the words from it instead of regenerating them (the losses are
 * bit-identical either way); a smaller workspace regenerates them.
 * zo_probe_bits_offset returns 0 for shapes without the cache or invalid
 * arguments. Host only. */
size_t zo_probe_bits_offset(const zo_config* cfg, int32_t N, int32_t B, int32_t C);

/* zo_update reading the probes' sign words from a sign-probe cache
 * (probe_bits: device, 16-byte aligned, the words of probes i0 .. i0+N-1 as
 * written by the zo_perturbed_losses call of the same seed, i0 and N, at its
 * workspace's zo_probe_bits_offset) instead of regenerating them. theta comes
 * out bit-identical to zo_update's. Sign probes only (ZO_EINVAL otherwise);
 * other arguments and return codes as for zo_update. For measuring the
 * update's cost in memory traffic against regeneration. */
int zo_update_cached(const zo_config* cfg, void* theta, uint64_t seed, float eps, float lr, int32_t N,
                     uint32_t i0, const float* Lplus, const float* Lminus, int32_t* skipped_out,
                     const uint32_t* probe_bits, void* stream);

/* Forward differences (Eq. 1's one-sided difference; the paper's FD-RGE,
 * compared with CD-RGE in its appendix): N + 1 passes instead of 2N.
 *   L   device fp32 [N]: the loss at theta + eps z_{i0+n}, as zo_perturbed_losses'
 *       Lplus (bit-identical to it)
 *   L0  device fp32 [1]: the loss at theta itself (the clean pass)
 * Other arguments, the workspace (zo_workspace_bytes covers both estimators),
 * the products and the return codes as for zo_perturbed_losses. */
int zo_fd_losses(const zo_config* cfg, const void* theta, uint64_t seed, float eps, int32_t N,
                 uint32_t i0, const int32_t* tokens, const uint8_t* mask, int32_t B, int32_t C,
                 float* L, float* L0, void* workspace, size_t ws_bytes, void* stream);

/* zo_fd_losses with the form of the products given, as
 * zo_perturbed_losses_ex (fp32 weights: ZO_PRODUCTS_SPLIT is ZO_EINVAL). */
int zo_fd_losses_ex(const zo_config* cfg, const void* theta, uint64_t seed, float eps, int32_t N,
                    uint32_t i0, const int32_t* tokens, const uint8_t* mask, int32_t B, int32_t C,
                    float* L, float* L0, void* workspace, size_t ws_bytes, int32_t products,
                    void* stream);

/* The forward-difference update:
 *   c_n = fp32( (lr / N) * (L_n - L0) / eps )  (computed in double)
 *   theta_j <- theta_j - sum_n c_n z_{i0+n}[j]
 * with the summation, rounding, alignment, skipping (any of L, L0 not
 * finite) and return codes of zo_update. L device fp32 [N], L0 device fp32 [1]. */
int zo_fd_update(const zo_config* cfg, void* theta, uint64_t seed, float eps, float lr, int32_t N,
                 uint32_t i0, const float* L, const float* L0, int32_t* skipped_out, void* stream);

/* Writes z_i[j0 .. j0+n) of the probe kind `probe` (ZO_RADEMACHER or
 * ZO_GAUSSIAN) to out (device fp32 [n], n <= 2^30). For checking the regenerated probe
 * stream; not part of the step. */
int zo_debug_probe(int32_t probe, uint64_t seed, uint32_t i, uint64_t j0, uint64_t n, float* out,
                   void* stream);

/* Applies the Box-Muller transform of the normal probes to n_pairs given
 * word pairs: words (device uint32 [2 n_pairs]) -> out (device fp32
 * [2 n_pairs]), pair p giving out[2p] = r cos and out[2p+1] = r sin. For
 * checking the fixed fp32 ln / sqrt / sin / cos sequences over their whole
 * input range (n_pairs <= 2^30); not part of the step. */
int zo_debug_gauss_pairs(const uint32_t* words, uint64_t n_pairs, float* out, void* stream);

/* Kernel timing (instrumentation, off by default). zo_profile_enable(every),
 * every >= 1, discards earlier records, counts every launch of the kernel
 * classes below and brackets every every-th launch of each class (the 1st,
 * (every+1)-th, ...) with a HIP event pair recorded on the stream of the
 * launch; each pair adds a few microseconds to the stream, so workloads of
 * short kernels sample (a prime stride cycles through layers and timesteps).
 * zo_profile_enable(0) stops recording; every < 0 is ZO_EINVAL.
 * zo_profile_read() waits for the recorded events and returns, for one class,
 * the summed time of the timed launches in milliseconds, their number, and
 * the number of all launches of the class since the last enable. */
enum { ZO_K_GATE = 0, ZO_K_HEAD = 1, ZO_K_EMBED = 2, ZO_K_COMBINE = 3, ZO_K_UPDATE = 4, ZO_K_PROBE_CACHE = 5,
       ZO_K_WEIGHTS16 = 6 };
int zo_profile_enable(int32_t every);
int zo_profile_read(int32_t kernel_class, double* timed_ms, int64_t* timed_launches, int64_t* all_launches);

/* Thread-local text of the last error (empty string if none). */
const char* zo_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* ZO_H */
