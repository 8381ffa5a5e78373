/*
 * jab.h -- C ABI of libjab, an MI355X (gfx950) implementation of the joint
 * attention-block (JAB) loss of "From Attention Sensitivity to Layer Role:
 * Revisiting Mixed-Precision Quantization of Transformers".
 *
 * What is computed (paper, Method, "Layer-wise PTQ" and "The joint attention
 * loss", eq. joint_loss; its KL attention-map term by jab_loss_fwd_kl):
 *
 *   W_hat   = fake-quantized [W_Q | W_K | W_V]   (eq. quant, one scale -- and for
 *             the asymmetric grid one zero-point -- per (output row, group))
 *   A(X)    = softmax(Q K^T / sqrt(head_dim) + M) V,  causal mask M, grouped-query
 *             heads (query head h reads key/value head floor(h * Hkv / Hq))
 *   loss    = || A(X; W) - A(X; W_hat) ||_F^2          (sse)
 *   mse     = sse / (batch * seq_len * n_heads * head_dim)
 *   backward: straight-through estimator on the weights (dW = dW_hat) and the
 *             LSQ rule on the scales (eq. lsq), gradients of mse.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Pointers are DEVICE pointers unless the comment says (host).  The caller
 *   owns every buffer.  The one allocation the library keeps is the tile queue
 *   of its large projection GEMMs (at least 32 tiles of 256 x 256 per CU): 4 KiB
 *   per device and stream, allocated with hipMalloc on the first such launch on
 *   that stream (not while the stream is being captured, and never by
 *   jab_loss_fwd_noalloc: without a queue the GEMM keeps a static tile order,
 *   with bitwise the same results) and held until the process ends.
 * - Calls enqueue work on `stream` (a hipStream_t; NULL = the null stream) and
 *   return without synchronising.  Outputs are valid once the stream reaches
 *   the end of the call.  Scratch memory comes from the caller's workspace
 *   (`ws`, `ws_bytes`, sized by jab_workspace_size) and is not allocated here.
 * - All arguments are validated on the host before any device work; a failing
 *   call returns a negative jab_status, enqueues nothing and leaves every
 *   output untouched.  jab_last_error() returns a per-thread description.
 *   A HIP launch error returns JAB_E_HIP; asynchronous device faults surface
 *   at the caller's next synchronisation.
 * - Results are deterministic: no atomics on any reduction, fixed reduction
 *   order, so two identical calls produce bitwise-identical outputs.
 *
 * Layouts (row-major)
 * -------------------
 *   x      [batch][seq_len][d_model]              in `dtype`
 *   w      [R][d_model], R = (n_heads + 2 n_kv_heads) head_dim, in `dtype`;
 *          row = output channel: the W_Q rows, then W_K, then W_V (the
 *          nn.Linear orientation; groups run along d_model inside one row)
 *   scale  [R][d_model / group_size] fp32,  zero  [R][d_model / group_size] u8
 *   a_ref  [batch][seq_len][n_heads * head_dim] fp32, head h in columns
 *          h*head_dim .. h*head_dim + head_dim - 1 (the merged attention output)
 *   codes  [R][d_model] u8: asymmetric grid index q in 0..2^b-1, or for the
 *          symmetric grid q + q_max in 0..2 q_max.
 *   dw     [R][d_model] fp32,  dscale [R][d_model / group_size] fp32.
 */
#ifndef JAB_H
#define JAB_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    JAB_OK = 0,
    JAB_E_INVALID = -1,     /* NULL or misaligned pointer, bad size or divisibility, bad bits */
    JAB_E_UNSUPPORTED = -2, /* head_dim / group_size / dtype / GQA ratio outside what is built */
    JAB_E_WORKSPACE = -3,   /* ws_bytes smaller than jab_workspace_size() */
    JAB_E_HIP = -4          /* the HIP runtime reported an error at launch */
} jab_status;

typedef enum { JAB_F32 = 0, JAB_F16 = 1, JAB_BF16 = 2 } jab_dtype;

/* JAB_ASYM: scale + integer zero-point per group, min-max initialised with 0 in
 *           the range (codes 0..2^b-1).
 * JAB_SYM:  the symmetric grid exactly as eq. quant prints it, no zero-point
 *           (codes -q_max..q_max, q_max = 2^(b-1)-1). */
typedef enum { JAB_ASYM = 0, JAB_SYM = 1 } jab_qscheme;

/* Workspace selector for jab_workspace_size: JAB_OP_QUANTIZE covers jab_quantize
 * (only when werr is requested), JAB_OP_PROJECT covers jab_project, JAB_OP_REF
 * jab_attn_ref and jab_attn_ref_kl, JAB_OP_FWD_KL jab_loss_fwd_kl. */
typedef enum { JAB_OP_FWD = 0, JAB_OP_SWEEP = 1, JAB_OP_BWD = 2, JAB_OP_REF = 3,
               JAB_OP_QUANTIZE = 4, JAB_OP_PROJECT = 5, JAB_OP_FWD_KL = 6, JAB_OP_CURVATURE = 7,
               JAB_OP_FISHER = 8, JAB_OP_STE = 9 } jab_op;

typedef struct {
    int32_t batch, seq_len, d_model;       /* X: [batch][seq_len][d_model]            */
    int32_t n_heads, n_kv_heads, head_dim; /* n_heads % n_kv_heads == 0               */
    int32_t group_size;                    /* d_model % group_size == 0               */
    int32_t dtype;                         /* jab_dtype of x, w and of Q/K/V storage   */
    int32_t scheme;                        /* jab_qscheme                              */
    float rope_theta;                      /* > 0: rotary position embedding on Q and K
                                              (RoPE as Mistral applies it, base theta;
                                              element j of a head pairs with j + head_dim/2,
                                              position t turns it by t theta^(-2j/head_dim),
                                              every sequence from position 0), in every
                                              entry point but jab_project; 0: none        */
} jab_problem;

typedef struct {
    int32_t bits[3];      /* b_Q, b_K, b_V in {2..8}; 0 = that matrix keeps its float weights */
    const float *scale;   /* [R][d_model/group_size]                                         */
    const uint8_t *zero;  /* [R][d_model/group_size] for JAB_ASYM; must be NULL for JAB_SYM   */
} jab_quant;

/* Supported: head_dim in {16, 64, 128}; group_size in {32, 64, 128};
 * n_heads / n_kv_heads in {1, 2} or a multiple of 4; all three dtypes.
 * Pointer alignment: 16 bytes for x, w, a_ref, dw, w_hat, codes; 4 for scale,
 * dscale; 8 for out / loss buffers. */

/* Bytes of workspace `op` needs.  n_bits: number of candidate bit-widths, used by
 * JAB_OP_SWEEP only (the sweep workspace holds up to n_bits^3 triples).
 * Returns 0 for an invalid problem or op. */
size_t jab_workspace_size(const jab_problem *p, int32_t op, int32_t n_bits);

/* Min-max quantizer parameters (eq. quant; asymmetric reading: lo = min(0, min w),
 * hi = max(0, max w), s = fp32((hi-lo)/(2^b-1)), s = 1 if that is 0,
 * z = clip(round_half_even(-lo/s), 0, 2^b-1); symmetric: s = fp32(max|w| / q_max)).
 * bits (host) [3]: per matrix; rows of a matrix with bits 0 get s = 1, z = 0.
 * zero must be NULL for JAB_SYM. */
jab_status jab_quant_init(const jab_problem *p, const void *w, const int32_t *bits,
                          float *scale, uint8_t *zero, void *stream);

/* Codes and fake-quantized weights (eq. quant): v = fp32(w / s), u = round half
 * to even (v), q = clip(u + z, 0, 2^b-1), w_hat = (q - z) s in fp32.
 * codes, w_hat: NULL to skip.  werr: NULL, or [3][2] doubles (device): per
 * matrix sum (w_hat - w)^2 and sum w^2 (Metric M3, eps^W = sqrt(ratio)). */
jab_status jab_quantize(const jab_problem *p, const void *w, const jab_quant *q,
                        uint8_t *codes, float *w_hat, double *werr, void *ws, size_t ws_bytes,
                        void *stream);

/* Teacher output A(X) = softmax(Q K^T / sqrt(head_dim) + M) V of the unmodified
 * block (Method, "Layer-wise PTQ" for A(X) and the causal mask M; "The joint
 * attention loss" for its role as the target), with the float weights, written to
 * a_ref (fp32) [batch][seq_len][n_heads head_dim], head h in columns h head_dim ..
 * h head_dim + head_dim - 1 (the merged output before the output projection,
 * Appendix on metrics, M4).  The loss entry points difference the student against
 * a buffer written here with the same kernels, so quantization disabled gives a
 * loss of exactly 0.  Errors: JAB_E_INVALID for NULL or misaligned pointers;
 * JAB_E_WORKSPACE below jab_workspace_size(p, JAB_OP_REF, 0). */
jab_status jab_attn_ref(const jab_problem *p, const void *x, const void *w, float *a_ref,
                        void *ws, size_t ws_bytes, void *stream);

/* Forward loss: the squared-error term of eq. joint_loss (Method, "The joint
 * attention loss"), ||A(X) - A_hat(X; w)||_F^2 with A_hat the block at the
 * fake-quantized weights of eq. quant (per-(row, group) scale, q->bits per matrix),
 * summed in a fixed order.  out (device) [3 + batch] doubles:
 *   out[0] = sse, out[1] = mse = sse / (batch seq_len n_heads head_dim),
 *   out[2] = sum a_ref^2 (so the attention-space error of the Metrics section,
 *            eps^A = sqrt(sse / out[2])),
 *   out[3 + b] = sse of sequence b.
 * Errors: JAB_E_INVALID for NULL or misaligned pointers or invalid bits;
 * JAB_E_WORKSPACE below jab_workspace_size(p, JAB_OP_FWD, 0). */
jab_status jab_loss_fwd(const jab_problem *p, const void *x, const void *w, const jab_quant *q,
                        const float *a_ref, double *out, void *ws, size_t ws_bytes, void *stream);

/* Teacher pass for the KL attention-map term (eq. joint_loss, D_KL(P || Q(w)), P
 * the teacher's causal softmax map): as jab_attn_ref, and it also keeps what the
 * student's KL term needs of the teacher's map:
 *   qk_ref  [batch*seq_len][(n_heads + n_kv_heads) head_dim] in dtype: the
 *           teacher's query and key projections (queries first, then keys),
 *   lse_ref [batch][n_heads][seq_len] fp32: the base-2 log-sum-exp of each
 *           teacher query row, log2 sum_j 2^(c q.k_j), c = log2(e)/sqrt(head_dim).
 * Alignment: 16 bytes for qk_ref, 4 for lse_ref.  Workspace: JAB_OP_REF. */
jab_status jab_attn_ref_kl(const jab_problem *p, const void *x, const void *w, float *a_ref,
                           void *qk_ref, float *lse_ref, void *ws, size_t ws_bytes, void *stream);

/* Forward loss with the KL attention-map term of eq. joint_loss, from one
 * projection of the student: the squared error of jab_loss_fwd and
 *   kl = sum over sequences, query heads and query rows i of
 *        D_KL(P_i || Q_i) = sum_{j <= i} P_ij (log P_ij - log Q_ij),
 * P the teacher's map (from qk_ref and lse_ref of jab_attn_ref_kl on the same
 * x and float w), Q that of the quantized block; the paper's reduction divides
 * the sum by the batch size only ("batchmean"), so the joint objective is
 * out[1] + lambda_KL * out[4 + batch].
 * out (device) [2 (3 + batch)] doubles:
 *   out[0 .. 3 + batch)  exactly as jab_loss_fwd,
 *   out[3 + batch] = kl,  out[4 + batch] = kl / batch,
 *   out[5 + batch] = sum over query rows of (sum_j P_ij - 1), P rebuilt from qk_ref
 *                    and normalised by lse_ref: zero up to rounding when both come
 *                    from one jab_attn_ref_kl call (a consistency check of the cache),
 *   out[6 + batch + b] = kl of sequence b.
 * Workspace: JAB_OP_FWD_KL. */
jab_status jab_loss_fwd_kl(const jab_problem *p, const void *x, const void *w, const jab_quant *q,
                           const float *a_ref, const void *qk_ref, const float *lse_ref, double *out,
                           void *ws, size_t ws_bytes, void *stream);

/* Loss for every candidate (b_Q, b_K, b_V) triple: the squared-error term of
 * eq. joint_loss at each triple of widths from the candidate set of eq. mckp
 * (Method, "Sensitivity and allocation"), a direct per-triple evaluation that can
 * stand in for an Omega table.  Errors as jab_loss_fwd, plus JAB_E_INVALID for a
 * triple whose width is not in `bits`; workspace JAB_OP_SWEEP with n_bits.
 * bits (host) [n_bits]: the candidate bit-widths; scale_by_bits / zero_by_bits
 * (host arrays of device pointers) [n_bits]: the fused weight's scales and
 * zero-points at each candidate width (zero_by_bits entries NULL for JAB_SYM).
 * triples (host) [n_triples][3]: bit values, each one of `bits`.
 * loss (device) [n_triples] doubles: sse of each triple;
 * loss_per_seq (device) [n_triples][batch] doubles or NULL.
 * Each (matrix, bit-width) projection is computed once and each (b_Q, b_K)
 * score matrix is shared by the triples that differ only in b_V. */
jab_status jab_loss_sweep(const jab_problem *p, const void *x, const void *w, int32_t n_bits,
                          const int32_t *bits, const float *const *scale_by_bits,
                          const uint8_t *const *zero_by_bits, int32_t n_triples,
                          const int32_t *triples, const float *a_ref, double *loss,
                          double *loss_per_seq, void *ws, size_t ws_bytes, void *stream);

/* Forward loss and gradients of mse (eq. lsq):
 *   dw[r][k]     = dmse/dw_hat[r][k]                      (straight-through)
 *   dscale[r][j] = gamma_m * sum_{k in group j} dw[r][k] phi[r][k],
 *   phi = u - v if the unrounded v lies on the grid (-z <= v <= 2^b-1-z; symmetric
 *   |v| <= q_max), else the clipped offset (-z or 2^b-1-z; symmetric sign(v) q_max).
 * lsq_gscale (host) [3]: gamma per matrix (1.0 = raw gradient; LSQ's choice is
 * (n_w q_max)^(-1/2)).  Attention is recomputed in the backward from the
 * forward's log-sum-exp.  out as in jab_loss_fwd.  dscale rows of a matrix with
 * bits 0 are written 0. */
jab_status jab_loss_bwd(const jab_problem *p, const void *x, const void *w, const jab_quant *q,
                        const float *a_ref, const float *lsq_gscale, double *out, float *dw,
                        float *dscale, void *ws, size_t ws_bytes, void *stream);

/* Memory / time trade of the attention backward inside jab_loss_bwd, jab_loss_bwd_kl,
 * jab_fisher and jab_ste_finetune (16-bit dtypes, head_dim 64 or 128).  Its first pass
 * (dK, dV) forms every causal dS_ij entry of eq. lsq's chain rule; it keeps them
 * (2 bytes per (sequence, query head, query, key <= query), rounded to the dtype as
 * the dK product uses them) in the workspace when they fit in max_bytes, and the dQ
 * pass then reads them instead of recomputing the scores and dP.  Default 8 GiB;
 * 0 always recomputes.  Process-wide: set it before sizing workspaces, since
 * jab_workspace_size (JAB_OP_BWD, JAB_OP_FISHER, JAB_OP_STE) counts the buffer; a
 * workspace sized under a lower limit is then rejected with JAB_E_WORKSPACE.  Not
 * synchronised with calls running on other host threads.  Always JAB_OK. */
jab_status jab_set_bwd_ds_limit(size_t max_bytes);

/* Stage helper: the fused QKV projection of the Method's "Layer-wise PTQ"
 * section, y = x W with W = [W_Q | W_K | W_V], here Y = X W_hat^T with W_hat
 * fake-quantized by eq. quant and rounded to dtype; y [batch][seq_len][R] in dtype
 * (the W_Q rows' outputs first, then W_K, then W_V).  q == NULL projects the float
 * weights.  Errors: JAB_E_INVALID for NULL or misaligned pointers or invalid bits;
 * JAB_E_WORKSPACE below jab_workspace_size(p, JAB_OP_PROJECT, 0). */
jab_status jab_project(const jab_problem *p, const void *x, const void *w, const jab_quant *q,
                       void *y, void *ws, size_t ws_bytes, void *stream);

/* Backward of the joint objective of eq. joint_loss with its KL attention-map
 * term: the gradients of  mse + lambda_kl * kl / batch  (kl as jab_loss_fwd_kl
 * defines it, P from the teacher cache qk_ref, lse_ref of jab_attn_ref_kl), by
 * the straight-through estimator and the LSQ rule as in jab_loss_bwd.  The KL
 * term adds (lambda_kl / batch) (Q_ij - P_ij) / sqrt(head_dim) to the gradient of
 * every raw score q_i . k_j (Q the student's map), recomputing the teacher map
 * from the cache inside the attention backward.  out (device) [2 (3 + batch)] as
 * jab_loss_fwd_kl's; dw, dscale as jab_loss_bwd's.  lambda_kl = 0 gives
 * jab_loss_bwd's gradients (up to the backward kernels' summation order).
 * Errors as jab_loss_bwd, plus JAB_E_INVALID for a NULL or misaligned cache or a
 * negative or non-finite lambda_kl.  Workspace: JAB_OP_BWD. */
jab_status jab_loss_bwd_kl(const jab_problem *p, const void *x, const void *w, const jab_quant *q,
                           const float *a_ref, const void *qk_ref, const float *lse_ref,
                           const float *lsq_gscale, float lambda_kl, double *out, float *dw, float *dscale,
                           void *ws, size_t ws_bytes, void *stream);

/* Curvature scores for the bit allocation (Method, "Sensitivity and allocation", eq. gn; eq. omega
 * uses the traces).  At the float point the joint loss of eq. joint_loss,
 *   L(w) = ||A(X) - A(X; w)||_F^2 + lambda_kl * D_KL(P || Q(w))   (KL summed over every query row),
 * is 0, so its Hessian there is exactly H = 2 J_A^T J_A + lambda_kl J_Q^T I(P) J_Q (J_A: Jacobian of
 * the attention output, J_Q: of the attention logits q.k / sqrt(head_dim), I(P) = diag(P) - P P^T
 * per query row).  For each probe p (a vector v over the fused weight's rows), with v_u its part in
 * the rows of W_Q (u = 0), W_K (1), W_V (2):
 *   out[7 p + u]     = t_u = v_u^T (H v)_u, u = 0..2   (the per-unit partition of the Appendix on
 *                      per-unit traces; its mean over Rademacher probes is Tr(H_uu))
 *   out[7 p + 3]     = v^T H v = t_0 + t_1 + t_2      (the pooled Hutchinson term)
 *   out[7 p + 4 + u] = v_u^T H_uu v_u                  (the diagonal block alone)
 * computed exactly (no finite difference) from one forward-mode pass: the tangent of the
 * projection X v^T (in the storage dtype, like Q, K, V; turned by the rotary embedding with Q
 * and K) carried through the attention beside the float point's (lambda_kl = 0: the squared error
 * alone; for the objective as implemented, mse + lambda kl / batch, pass lambda * N / batch and
 * divide the forms by N = batch * seq_len * n_heads * head_dim).
 * probes (device) [n_probes][R][d_model] int8 in {-1, +1}; out (device) [n_probes][7] doubles.
 * Work per call: one projection of w; per probe one projection of the probe and one tangent
 * attention pass.  Errors: JAB_E_INVALID for NULL or misaligned pointers, n_probes < 1 or a
 * negative or non-finite lambda_kl; JAB_E_WORKSPACE below jab_workspace_size(p,
 * JAB_OP_CURVATURE, 0).  Workspace: JAB_OP_CURVATURE. */
jab_status jab_curvature(const jab_problem *p, const void *x, const void *w, float lambda_kl, int32_t n_probes,
                         const int8_t *probes, double *out, void *ws, size_t ws_bytes, void *stream);

/* Fisher-coupling scores (Appendix on Fisher-coupling; the first-order
 * alternative to the curvature scores): at a coarse round-to-nearest probe q
 * (the paper's is 2-bit: bits {2,2,2} with jab_quant_init's scales), the squared
 * straight-through gradient norm of the loss per unit,
 *   out[u] = sum over the rows of unit u of (d mse / dW)^2,  u = 0 (W_Q), 1 (W_K), 2 (W_V),
 *   out[3] = mse at the probe,
 * with the gradient exactly as jab_loss_bwd computes dW (dW = dW_hat, gradient of
 * mse).  One jab_loss_bwd pass plus a fixed-order fp64 sum of squares; dW and ds
 * stay in the workspace.  out (device) [4] doubles; a_ref from jab_attn_ref.
 * lambda_kl > 0 scores the joint objective mse + lambda_kl kl / batch instead (the
 * gradient of jab_loss_bwd_kl; qk_ref, lse_ref: the teacher cache of
 * jab_attn_ref_kl, unused when lambda_kl = 0); out[3] stays the mse.
 * Errors as jab_loss_bwd (no lsq_gscale, dw or dscale arguments), plus
 * JAB_E_INVALID for a negative or non-finite lambda_kl or a missing cache.
 * Workspace: JAB_OP_FISHER. */
jab_status jab_fisher(const jab_problem *p, const void *x, const void *w, const jab_quant *q,
                      const float *a_ref, const void *qk_ref, const float *lse_ref, float lambda_kl,
                      double *out, void *ws, size_t ws_bytes, void *stream);

/* Joint STE fine-tuning (Appendix "Joint STE fine-tuning": STE on the weights,
 * LSQ on the scales, eq. lr, the held-out commit gate, eq. flip).  Adam on the fp32
 * latent weights w_master [R][d_model] and on the per-(row, group) scales, with the
 * gradients of jab_loss_bwd at the dtype-rounded weights, learning rates
 *   eta_w = alpha_w * sbar * c_t,  eta_s = alpha_s * sbar * c_t,
 *   c_t = (1 + cos(pi (t - 1) / n_steps)) / 2 for step t = 1..n_steps,
 * sbar = the mean of the starting scales over the quantized units.  The held-out
 * batch (x_held, a_ref_held: held_batch <= batch sequences) is scored with
 * jab_loss_fwd at the start and after every eval_every-th step and the last; the
 * best checkpoint (strictly below every earlier score, the start included) is
 * written back, so the start is returned unchanged unless fine-tuning beat it.
 * Scales are kept >= scale_floor after each step.  Zero-points stay fixed. */
typedef struct {
    int32_t n_steps;          /* Adam steps (the paper: 200)                         */
    int32_t eval_every;       /* held-out evaluation period (the paper: 10)          */
    float alpha_w, alpha_s;   /* grid-relative rates (the paper: 0.05, 0.02)         */
    float beta1, beta2;       /* Adam moments (0.9, 0.999)                           */
    float adam_eps;           /* Adam denominator term (1e-8)                        */
    float scale_floor;        /* lower bound on every scale after a step (> 0 keeps
                                 the quantizer defined)                               */
    float lambda_kl;          /* > 0: the objective is mse + lambda_kl kl / batch (eq.
                                 joint_loss; the paper: 0.1), its gradient as
                                 jab_loss_bwd_kl's, the log and the held-out scores
                                 that objective; 0: the squared error alone           */
} jab_ste_config;

/* Length of the stats array: 6 + n_steps + ceil(n_steps / eval_every); 0 for
 * invalid arguments. */
int32_t jab_ste_stats_len(int32_t n_steps, int32_t eval_every);

/* In/out (device): w_master (fp32; in: the start, out: the best checkpoint), scale
 * (in/out likewise); out: w = dtype(w_master) [R][d_model].  zero: the fixed
 * zero-points (NULL for JAB_SYM).  bits, lsq_gscale (host) [3].  stats (device,
 * doubles, jab_ste_stats_len): [0] held-out mse at the start, [1] best held-out
 * mse, [2] step of the best checkpoint (0: the start), [3..5] flip rate of W_Q,
 * W_K, W_V (eq. flip: the fraction of codes that differ between the start's and
 * the returned weights, both on the returned grid; 0 for an unquantized matrix),
 * [6 .. 6 + n_steps) training mse before each step, then the held-out mse of each
 * evaluation (with lambda_kl > 0: the joint objective in every slot).  qk_ref,
 * lse_ref and qk_ref_held, lse_ref_held: the teacher caches of jab_attn_ref_kl on
 * x and x_held with the float weights, required when lambda_kl > 0 (else unused).  Asynchronous on `stream` (no host synchronisation inside).
 * Errors: JAB_E_INVALID for NULL or misaligned pointers, invalid bits, config or
 * held_batch; JAB_E_WORKSPACE below jab_workspace_size(p, JAB_OP_STE, 0). */
jab_status jab_ste_finetune(const jab_problem *p, const jab_ste_config *cfg, const void *x, const float *a_ref,
                            int32_t held_batch, const void *x_held, const float *a_ref_held,
                            const void *qk_ref, const float *lse_ref, const void *qk_ref_held,
                            const float *lse_ref_held,
                            const int32_t bits[3], const float lsq_gscale[3], float *w_master, void *w,
                            float *scale, const uint8_t *zero, double *stats, void *ws, size_t ws_bytes,
                            void *stream);

/* Bit allocation (Method, eq. mckp): each unit i (a weight matrix) picks a width
 * b_i from `widths` to minimise sum_i Omega_i(b_i) subject to
 * sum_i P_i b_i <= budget_bits * sum_i P_i (the parameter-weighted budget,
 * eq. pwbudget) and b_i >= min_bits (0: no floor; the paper's floor is 3).
 * method: JAB_ALLOC_GREEDY (start at the highest width, apply the downgrade with
 * the smallest Delta Omega / Delta c until the budget holds, then the upgrades
 * with the largest -Delta Omega / Delta c that fit and lower the objective) or
 * JAB_ALLOC_PARETO (the same walk on each unit's Pareto-efficient widths: a
 * width is kept only if its Omega is below that of every lower width); ties go
 * to the lowest unit index (Appendix "Allocators").
 * widths (host) [n_widths] strictly ascending; omega (host) [n_units][n_widths],
 * e.g. eq. omega's Tr(H_i) ||Q_b(W_i) - W_i||^2 or the sweep's losses;
 * params (host) [n_units] > 0; choice (host out) [n_units]: index into widths;
 * objective (host out, or NULL).  Host-only and synchronous; JAB_E_INVALID for
 * bad arguments or a budget below the lowest admissible widths. */
enum { JAB_ALLOC_GREEDY = 0, JAB_ALLOC_PARETO = 1 };
jab_status jab_allocate(int32_t n_units, int32_t n_widths, const int32_t *widths, const double *omega,
                        const double *params, double budget_bits, int32_t min_bits, int32_t method,
                        int32_t *choice, double *objective);

/* Sensitivity table of eq. omega (Method, "Sensitivity and allocation"; Appendix on per-unit
 * traces) for n_layers attention blocks.  Unit i = 3 l + m is matrix m (0 W_Q, 1 W_K, 2 W_V) of
 * block l, l = 0 .. n_layers - 1 in depth order, and for candidate width k:
 *   C1 (JAB_OMEGA_C1): omega[i][k] = Tr_i * ||Q_{b_k}(W_i) - W_i||_F^2
 *   C2 (JAB_OMEGA_C2): omega[i][k] = (n_layers - l) * Tr_i * ||Q_{b_k}(W_i) - W_i||_F^2
 * (C2 weights an error by the layers it passes through, block l's own included).  Tr_i is the
 * Hutchinson mean over the block's n_probes probes (summed in probe order, divided by n_probes) of
 * jab_curvature's pooled form v^T H v (JAB_TRACE_BLOCK: one trace per block, shared by its three
 * matrices, as in the Method section) or of the unit's partition term t_u (JAB_TRACE_UNIT: the
 * per-unit traces of the Appendix, unbiased for Tr(H_uu)).
 * curv (host) [n_layers][n_probes][7]: jab_curvature's out for each block, copied to the host.
 * werr (host) [n_layers][n_widths][3][2]: jab_quantize's werr for each block at each width (its
 * column 0, sum (w_hat - w)^2, is ||Q_b(W) - W||_F^2); a width kept in float has zeros there.
 * omega (host out) [3 n_layers][n_widths], the table jab_allocate takes.  Nothing is clamped: a
 * negative mean (a per-unit trace from few probes) stays negative.  Host-only and synchronous.
 * Errors: JAB_E_INVALID for NULL pointers, n_layers, n_probes or n_widths below 1, an unknown
 * trace or criterion, or a non-finite input. */
enum { JAB_TRACE_BLOCK = 0, JAB_TRACE_UNIT = 1 };
enum { JAB_OMEGA_C1 = 0, JAB_OMEGA_C2 = 1 };
jab_status jab_omega(int32_t n_layers, int32_t n_probes, const double *curv, int32_t n_widths, const double *werr,
                     int32_t trace, int32_t criterion, double *omega);

/* Allocation-free forward loss, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): exactly jab_loss_fwd (same kernels, bitwise the same out), with the
 * workspace taken from a device array inside the library instead of a caller
 * buffer.  The array holds JAB_NOALLOC_SCRATCH_BYTES per device; it is placed on
 * a device when the library's code is loaded there and is held until the process
 * ends.  Its address is looked up on the first call on each device (the current
 * device, which must be the one `stream` belongs to).  The call allocates
 * nothing and needs no clearing: it writes every scratch byte whose value can
 * reach a result.  Calls that overlap in time on one device share that device's
 * array and race: serialise them (one stream, or events).
 * Errors as jab_loss_fwd, plus JAB_E_WORKSPACE when jab_workspace_size(p,
 * JAB_OP_FWD, 0) exceeds JAB_NOALLOC_SCRATCH_BYTES (checked on the host before
 * any device work) and JAB_E_HIP when the array's address cannot be looked up. */
#define JAB_NOALLOC_SCRATCH_BYTES (64u << 20)
jab_status jab_loss_fwd_noalloc(const jab_problem *p, const void *x, const void *w, const jab_quant *q,
                                const float *a_ref, double *out, void *stream);

const char *jab_status_string(int32_t status);
const char *jab_last_error(void);

/* Kernel timing.  When enabled, every kernel launch of this thread's calls is
 * bracketed by hipEvents on the launch stream.  jab_timing_read synchronises
 * those events and returns, per kernel family (JAB_KT_*), the summed duration
 * in milliseconds and the launch count since the last reset. */
/* JAB_KT_GEMM: the projection of Q and K (or the single projection of jab_project);
 * JAB_KT_GEMM_VT: the projection that writes V transposed; JAB_KT_KL: the KL
 * attention-map kernel of jab_loss_fwd_kl. */
enum { JAB_KT_QUANT = 0, JAB_KT_GEMM = 1, JAB_KT_ATTN = 2, JAB_KT_REDUCE = 3,
       JAB_KT_ATTN_BWD = 4, JAB_KT_DW_GEMM = 5, JAB_KT_MISC = 6, JAB_KT_GEMM_VT = 7, JAB_KT_KL = 8,
       JAB_KT_COUNT = 9 };
jab_status jab_timing_enable(int32_t on);
jab_status jab_timing_read(double *ms /*host [JAB_KT_COUNT]*/, int64_t *launches /*host [JAB_KT_COUNT]*/);

#ifdef __cplusplus
}
#endif
#endif /* JAB_H */
