/*
 * countdown.h -- C ABI of the MI355X (gfx950) COUNTDOWN sparse Gated-MLP FFN.
 *
 * The FFN of arXiv 2505.17701 (Sec. 3, Eq. 1) is
 *     y = ((x.W_up) (.) SiLU(x.W_gate)) . W_down^T = sum_i s[i] W_down^T[i]   (Eq. 5)
 * and the library evaluates it only on an index set IDX chosen per call by a
 * coefficient and a per-layer threshold (Eq. 2, 3, 6; Sec. 4):
 *   M-CountDown  (countdown_ffn_mono):        IDX = {i : |u[i]| > thld}, u = x.W_up;
 *   D-CountDown  (countdown_ffn_dual, ideal): IDX = {i : |s[i]| > thld}, s computed densely;
 *   D-CountDown  (countdown_ffn_dual, pred):  IDX = {i : s_hat[i] > thld},
 *                                             s_hat = (x.theta_A).theta_B (signed score);
 *   D-CountDown  (countdown_ffn_tern):        the same with the ternary predictor
 *                                             s_hat = x.theta, theta in {-1, 0, +1}.
 * For a batch of B tokens IDX is the union of the per-token sets and every
 * token uses all rows of IDX with its own coefficients.
 *
 * Data conventions (all calls):
 *  - bf16 tensors are passed as `const uint16_t *` (bf16 bit patterns);
 *    fp32 tensors as `float *`.
 *  - Every tensor pointer is a DEVICE pointer owned by the caller, 16-byte
 *    aligned; the library neither frees nor retains it beyond the call.
 *  - Weight matrices are neuron-major, row-major [d_ff][d_model]: row i is
 *    the weight vector of intermediate neuron i (W_gate[i][j] is the paper's
 *    W_gate[j][i]; W_down[i][:] is the paper's W_down^T[i]).
 *    The predictor is A_t [d_rank][d_model] (theta_A transposed) and
 *    B_t [d_ff][d_rank] (theta_B transposed).
 *  - x is [B][d_model] bf16, y is [B][d_model] fp32 and is fully
 *    overwritten (no pre-zeroing needed).
 *  - `stream` is a hipStream_t (NULL = the default stream). Every call only
 *    enqueues work on `stream` and returns without synchronising; outputs
 *    are valid once the stream reaches that point. No call but
 *    countdown_plan_create / countdown_plan_destroy / countdown_calibrate
 *    allocates device memory.
 *  - thld is one fp32 constant per layer (Sec. 4: the calibrated layerwise
 *    threshold). Selection is strict (coefficient > thld). thld = -INFINITY
 *    selects every row (the dense result); thld = +INFINITY selects none
 *    (y = 0). A NaN thld is rejected with CD_EINVAL.
 *  - Arguments are validated on the host before anything is enqueued;
 *    on error nothing is launched. A launch failure returns CD_EHIP.
 *  - A plan is not thread-safe: calls on one plan must not overlap (use one
 *    plan per stream).
 *  - A plan belongs to the device that was current when it was created:
 *    every call on it must be made with that device current (else
 *    CD_EINVAL); countdown_plan_destroy switches to it by itself.
 *  - The outputs of a call (y, and thld_out of the per-token calls) must not
 *    share memory with its inputs (x, the weights, the predictor) or with
 *    each other: CD_EINVAL. The residual step states its own rules.
 */
#ifndef COUNTDOWN_H
#define COUNTDOWN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int cd_status;
#define CD_OK 0
#define CD_EINVAL (-1)        /* bad argument (null/misaligned pointer, size, NaN thld) */
#define CD_EUNSUPPORTED (-2)  /* shape outside what the kernels implement */
#define CD_EHIP (-3)          /* a HIP runtime call or kernel launch failed */
#define CD_ENOMEM (-4)        /* device allocation failed */

/* Variants, for countdown_check_args and countdown_calibrate. */
#define CD_VARIANT_MONO 0        /* M-CountDown, coefficient |u| (Eq. 6b) */
#define CD_VARIANT_DUAL_IDEAL 1  /* D-CountDown ideal, coefficient |s| (Eq. 6c) */
#define CD_VARIANT_DUAL_PRED 2   /* D-CountDown, predictor score s_hat (Sec. 4) */
#define CD_VARIANT_DENSE 3       /* dense Gated-MLP (Eq. 1) */
#define CD_VARIANT_CATS 4        /* CATS, the comparison method: |SiLU(x.W_gate)| (Eq. 6a) */
#define CD_VARIANT_DUAL_TERN 5   /* D-CountDown, ternary predictor score x.theta (Sec. 6) */

/* Plan flags. */
#define CD_PLAN_KEEP_COEF 1u  /* also store the dense coefficient vector of each call
                                 (u for mono, s for dual ideal, s_hat for dual pred) */
#define CD_PLAN_DETERMINISTIC 2u  /* bit-reproducible y: the down projection stores one
                                 partial sum per neuron range (plan workspace, about
                                 64 x max_batch x d_model floats) and a second kernel
                                 adds them in ascending range order, instead of fp32
                                 atomics in arrival order; costs one more launch */

typedef struct cd_plan cd_plan;

/*
 * Create a plan for one FFN shape. Allocates the plan's device workspace
 * (a per-neuron active flag, the coefficients s of the active neurons, the
 * predictor latent and, with CD_PLAN_KEEP_COEF, the dense coefficients) on
 * the current device. d_model and d_ff must be positive multiples of 8 with
 * d_model <= 8192; 1 <= max_batch <= 8; d_rank is 0 (no predictor) or a
 * power of two in [8, 1024]; T * C <= 32768, where T is max_batch rounded up
 * to 1, 2, 4 or 8 and C is d_model rounded up to 512, 1024, 2048, 4096 or
 * 8192 (the widest token tile a call stages; d_model 4096 takes up to 8
 * tokens, d_model 4097..8192 up to 4). Returns CD_EINVAL
 * for malformed sizes and CD_EUNSUPPORTED for well-formed sizes beyond those
 * limits (both checked before any HIP call), CD_ENOMEM / CD_EHIP when the
 * device is missing or allocation fails. *out is set only on success.
 */
cd_status countdown_plan_create(int d_model, int d_ff, int max_batch, int d_rank,
                                unsigned flags, cd_plan **out);

/* Release a plan and its workspace (synchronises the device first). NULL is a no-op. */
cd_status countdown_plan_destroy(cd_plan *plan);

/*
 * M-CountDown (Eq. 6b; Sec. 4, layerwise threshold): u = x.W_up over all
 * rows; IDX = {i : exists b, |u_b[i]| > thld}; s_b[i] = u_b[i] SiLU(x_b.W_gate[i])
 * on IDX only (Eq. 2); y_b = sum_{i in IDX} s_b[i] W_down[i] (Eq. 5).
 * B in [1, max_batch]. W_gate, W_up, W_down: [d_ff][d_model] bf16.
 */
cd_status countdown_ffn_mono(cd_plan *plan, const uint16_t *x, int B, const uint16_t *W_gate,
                             const uint16_t *W_up, const uint16_t *W_down, float thld, float *y,
                             void *stream);

/*
 * D-CountDown (Eq. 6c; Sec. 4). With A_t == B_t == NULL (ideal): s is
 * computed over all rows and IDX = {i : exists b, |s_b[i]| > thld}. With a
 * predictor (both non-NULL, plan created with this d_rank): s_hat_b =
 * (x_b.theta_A).theta_B, IDX = {i : exists b, s_hat_b[i] > thld} (signed),
 * then gate and up are evaluated on IDX only. y by Eq. (5) over IDX.
 * Passing exactly one of A_t / B_t is CD_EINVAL.
 */
cd_status countdown_ffn_dual(cd_plan *plan, const uint16_t *x, int B, const uint16_t *W_gate,
                             const uint16_t *W_up, const uint16_t *W_down, const uint16_t *A_t,
                             const uint16_t *B_t, float thld, float *y, void *stream);

/*
 * countdown_ffn_mono without a plan, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc). It computes exactly what countdown_ffn_mono computes, with
 * the same kernels, and allocates nothing: the per-neuron workspace (active
 * flags and s) lives in a static device array of the library, 1.125 MiB per
 * device (d_ff <= 32768 at up to 8 tokens), held on each device the library
 * runs on until the process ends. Its device address is looked up on the first
 * call made with that device current.
 * x [B][d_model], W_gate / W_up / W_down [d_ff][d_model] bf16; y [B][d_model]
 * fp32, overwritten; all device pointers owned by the caller, 16-byte aligned.
 * Shape rules as countdown_plan_create with max_batch = B and d_rank = 0, plus
 * d_ff <= 32768 (CD_EUNSUPPORTED beyond); argument errors as countdown_ffn_mono.
 * All calls on one device share the array: calls that overlap in time on one
 * device (two streams, two host threads) race and must not be made. Enqueued
 * on `stream`; no host synchronisation.
 */
cd_status countdown_ffn_mono_noalloc(const uint16_t *x, int B, const uint16_t *W_gate,
                                     const uint16_t *W_up, const uint16_t *W_down, int d_model,
                                     int d_ff, float thld, float *y, void *stream);

/* Dense Gated-MLP (Eq. 1) through the same kernels with every row active:
 * the reference the sparse variants are timed against. */
cd_status countdown_ffn_dense(cd_plan *plan, const uint16_t *x, int B, const uint16_t *W_gate,
                              const uint16_t *W_up, const uint16_t *W_down, float *y,
                              void *stream);

/*
 * CATS (Eq. 6a; the comparison method of Sec. 3), through the same kernels:
 * h = SiLU(x.W_gate) over all rows; IDX = {i : exists b, |h_b[i]| > thld};
 * u_b[i] = x_b.W_up[i] on IDX only; y_b = sum_{i in IDX} u_b[i] h_b[i] W_down[i].
 * Conventions as countdown_ffn_mono (the roles of W_gate and W_up swapped).
 */
cd_status countdown_ffn_cats(cd_plan *plan, const uint16_t *x, int B, const uint16_t *W_gate,
                             const uint16_t *W_up, const uint16_t *W_down, float thld, float *y,
                             void *stream);

/*
 * Per-token threshold (the per-token form of Eq. 6: the threshold of each
 * token is the quantile of its own coefficient vector, as in the ideal
 * sparsity of Sec. 3, instead of the calibrated layer constant of Sec. 4):
 *   thld_b = Quantile(k, c_b), linear interpolation between order statistics,
 *   IDX = {i : exists b, c_b[i] > thld_b}   (strict, union over the batch),
 * c_b = |u_b| (CD_VARIANT_MONO), |s_b| (CD_VARIANT_DUAL_IDEAL), |h_b|
 * (CD_VARIANT_CATS) or the signed predictor score s_hat_b
 * (CD_VARIANT_DUAL_PRED, A_t / B_t set); then s on
 * IDX and y by Eq. (5) as in the constant-threshold calls. A batch-1 call
 * keeps exactly d_ff - 1 - floor(k (d_ff - 1)) neurons when the coefficients
 * are distinct. thld_out (DEVICE double[B], 8-byte aligned, may be NULL)
 * receives the per-token thresholds, computed in fp64 from the fp32
 * coefficients. k in [0, 1]; d_ff <= 32768 (CD_EUNSUPPORTED beyond). The
 * call runs the coefficient kernel over all neurons, a per-token selection
 * kernel, the gather of IDX and the down projection; for one token with
 * d_model <= 4096 and d_ff <= 16384 the selection and the gather are one
 * launch (ideal D, which has nothing to gather: the selection, the flags and
 * the down projection; not in a deterministic plan). Results are the same
 * either way, y to fp32 rounding.
 */
cd_status countdown_ffn_topk(cd_plan *plan, int variant, const uint16_t *x, int B,
                             const uint16_t *W_gate, const uint16_t *W_up, const uint16_t *W_down,
                             const uint16_t *A_t, const uint16_t *B_t, double k, double *thld_out,
                             float *y, void *stream);

/*
 * Ternary predictor (the TernaryLinear candidate of Sec. 6, Table 4; trained
 * by Alg. 1): s_hat_b = x_b.theta with theta in {-1, 0, +1}^{d_model x d_ff}
 * (no scale: a positive per-layer scale only rescales the threshold),
 * IDX = {i : exists b, s_hat_b[i] > thld} (signed, strict), then gate and
 * up on IDX and y by Eq. (5), as countdown_ffn_dual with a predictor.
 * theta_packed is the DEVICE buffer written by countdown_ternary_pack
 * (countdown_ternary_words(d_model, d_ff) uint32 words, 16-byte aligned).
 * The plan's d_rank is not used. s_hat is accumulated in fp32.
 */
cd_status countdown_ffn_tern(cd_plan *plan, const uint16_t *x, int B, const uint16_t *W_gate,
                             const uint16_t *W_up, const uint16_t *W_down,
                             const uint32_t *theta_packed, float thld, float *y, void *stream);

/* countdown_ffn_topk with the ternary predictor score (signed, per-token thresholds). */
cd_status countdown_ffn_tern_topk(cd_plan *plan, const uint16_t *x, int B,
                                  const uint16_t *W_gate, const uint16_t *W_up,
                                  const uint16_t *W_down, const uint32_t *theta_packed, double k,
                                  double *thld_out, float *y, void *stream);

/* countdown_calibrate for the ternary predictor score (signed s_hat = x.theta). */
cd_status countdown_calibrate_tern(cd_plan *plan, const uint16_t *X, int T,
                                   const uint32_t *theta_packed, double k, float *thld_out,
                                   double *q_out, void *stream);

/*
 * Size in uint32 words of the packed ternary predictor of a shape: d_ff rows
 * of 64 * W words, W = max(1, C / 2), C the smallest of 1, 2, 4, 8, 16 with
 * 512 C >= d_model. 0 for shapes countdown_check_shape rejects. Host only.
 */
size_t countdown_ternary_words(int d_model, int d_ff);

/*
 * Pack theta for the ternary predictor. HOST memory in and out, no device
 * call. theta_t is int8 [d_ff][d_model] (theta transposed: row i is neuron
 * i's weights), every entry -1, 0 or +1 (else CD_EINVAL, packed untouched
 * beyond the rows already written). packed receives
 * countdown_ternary_words(d_model, d_ff) words. Layout of row i (64 W words,
 * unused columns zero): lane l = 0..63 owns words [l W, (l + 1) W); its unit
 * j (j < C) holds the 8 weights of columns j * 512 + 8 l + e, e = 0..7; word
 * k of the lane holds units 2k (A) and 2k + 1 (B). In a word, byte 1 bits
 * 2m..2m+1 hold A's weight e = 2m, byte 3 A's e = 2m + 1, byte 0 B's e = 2m,
 * byte 2 B's e = 2m + 1 (m = 0..3), coded 0 -> 0, 1 -> +1, 2 -> -1.
 */
cd_status countdown_ternary_pack(const int8_t *theta_t, int d_model, int d_ff, uint32_t *packed);

/*
 * One layer of a stack of FFNs joined by a residual stream. The paper
 * evaluates single Gated-MLP layers (Sec. 3); the stack workload adds, per
 * token b, before the FFN of `variant` (CD_VARIANT_*, as in the calls above):
 *   h_out_b = h_in_b + y_prev_b                    (fp32; y_prev NULL: h_out = h_in)
 *   x_b = bf16(h_out_b / sqrt(mean_j(h_out_b[j]^2) + eps))   (RMSNorm, unit gain,
 *                                                             round to nearest even)
 * then y = FFN(x). x is written to x_out [B][d_model] bf16 (the FFN input).
 * h_in, y_prev, h_out are [B][d_model] fp32. Only y_prev and y may share
 * memory (y_prev is read before y is written); any other overlap among h_in,
 * h_out, x_out, y and y_prev, or of h_out, x_out or y with the weights or the
 * predictor, is CD_EINVAL. eps must be finite and >= 0.
 * thld is ignored for CD_VARIANT_DENSE; A_t / B_t as for countdown_ffn_dual
 * (both set exactly for CD_VARIANT_DUAL_PRED, else NULL). With the predictor
 * the normalisation is computed inside the latent product's kernel.
 */
cd_status countdown_ffn_residual(cd_plan *plan, int variant, const float *h_in,
                                 const float *y_prev, float *h_out, float eps, uint16_t *x_out,
                                 int B, const uint16_t *W_gate, const uint16_t *W_up,
                                 const uint16_t *W_down, const uint16_t *A_t, const uint16_t *B_t,
                                 float thld, float *y, void *stream);

/*
 * Layerwise threshold calibration (Sec. 4): thld = (1/T) sum_t Quantile(k, c^(t))
 * over T calibration tokens X [T][d_model], with c^(t) the variant's
 * coefficient vector (|u| mono, |s| dual ideal, signed s_hat dual pred) and
 * Quantile the linear interpolation between order statistics:
 * h = k (d_ff - 1), q = v[floor h] + (h - floor h)(v[floor h + 1] - v[floor h]).
 * Quantiles and the mean are formed in fp64; *thld_out (a DEVICE float) gets
 * the mean rounded to fp32. q_out (DEVICE double[T], may be NULL) gets the
 * per-token quantiles. k in [0, 1]. Allocates and frees temporary device
 * memory, and synchronises `stream` before returning.
 */
cd_status countdown_calibrate(cd_plan *plan, int variant, const uint16_t *X, int T,
                              const uint16_t *W_gate, const uint16_t *W_up, const uint16_t *A_t,
                              const uint16_t *B_t, double k, float *thld_out, double *q_out,
                              void *stream);

/*
 * Export the last FFN call's index set on `stream` into caller-owned DEVICE
 * buffers (any destination may be NULL): idx_dst int32[d_ff] receives the
 * ascending IDX in its first |IDX| entries, n_dst int32[1] receives |IDX|,
 * s_dst fp32[B][d_ff] receives s_b[IDX[j]] at s_dst[b * d_ff + j], and
 * coef_dst fp32[B][d_ff] the dense coefficient vector of every neuron (u for
 * mono, s for dual ideal and dense, s_hat for dual pred; CD_PLAN_KEEP_COEF
 * plans only, else CD_EINVAL). B is the batch of that call. The hot path
 * keeps the active set as per-neuron flags; this call runs a small kernel
 * that scans them in order. CD_EINVAL before the plan's first FFN call and after
 * countdown_calibrate (which reuses the workspace).
 */
cd_status countdown_export_active(const cd_plan *plan, int32_t *idx_dst, int32_t *n_dst,
                                  float *s_dst, float *coef_dst, void *stream);

/*
 * Measurement aid: choose which kernels the plan's subsequent FFN calls
 * launch. Every call runs its coefficient kernel (predictor latent, dense
 * coefficient, threshold, gathered gate or gate+up; it writes the plan's
 * per-neuron active flags and coefficients and zeroes y) and then its down
 * kernel (gathered down projection into y). CD_PHASE_COEF or CD_PHASE_DOWN
 * alone launch only that kernel, so a loop of calls times one kernel in
 * isolation; y is then not the FFN output. A down-only call uses the flags
 * and coefficients left by the plan's last coefficient kernel (CD_EINVAL if
 * there is none, or if it ran on another batch size). Plans start at
 * CD_PHASE_ALL.
 */
#define CD_PHASE_COEF 1u
#define CD_PHASE_DOWN 2u
#define CD_PHASE_ALL 3u
cd_status countdown_plan_set_phases(cd_plan *plan, unsigned phases);

/*
 * Measurement aid, not part of the method: a plain streaming read of `bytes`
 * bytes at `src` with the coefficient kernel's load pattern (one wave per
 * 8 KB, non-temporal 16-byte loads) and no arithmetic but an xor per load.
 * Timed by the caller, it gives the read bandwidth that a kernel reading the
 * same number of bytes can reach: the measured ceiling beside the 8 TB/s
 * peak. src: device, 16-byte aligned; bytes: a positive multiple of 16.
 * sink: one device uint32, written only when the xor of a lane's data equals
 * 0x9E3779B9 (which keeps the loads from being optimised away). Enqueued on
 * `stream`; CD_EINVAL for bad arguments.
 */
cd_status countdown_stream_read(const void *src, size_t bytes, uint32_t *sink, void *stream);

/*
 * Host-only validation of an FFN call's arguments against a shape, exactly
 * as the entry points perform it before launching: pointers non-NULL and
 * 16-byte aligned, 1 <= B <= max_batch, thld not NaN, predictor pointers
 * both NULL or both set (dual only, and d_rank > 0 when set). For
 * CD_VARIANT_DUAL_TERN, A_t is the packed ternary predictor and B_t must be
 * NULL. Touches no device. variant is a CD_VARIANT_*.
 */
cd_status countdown_check_args(int variant, int d_model, int d_ff, int max_batch, int d_rank,
                               const void *x, int B, const void *W_gate, const void *W_up,
                               const void *W_down, const void *A_t, const void *B_t, float thld,
                               const void *y);

/* Host-only validation of plan sizes (the checks countdown_plan_create makes first). */
cd_status countdown_check_shape(int d_model, int d_ff, int max_batch, int d_rank);

/* Static description of a status code. */
const char *countdown_status_string(cd_status status);

/* ABI version of this header (bumped on any signature change). */
#define COUNTDOWN_ABI_VERSION 9
int countdown_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* COUNTDOWN_H */
