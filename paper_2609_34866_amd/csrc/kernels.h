// kernels.h -- host-side launchers of the libjab kernels (internal interface
// between the C ABI layer and the HIP translation units).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace jab {

// Shape of the fused weight for the quantizer kernels.
struct QuantShape {
    int rows, cols, group;   // rows = R, cols = d_model
    int row_k, row_v;        // first row of W_K and of W_V
    int bits[3];             // per matrix; 0 = not quantized
    int scheme;              // 0 asymmetric, 1 symmetric
};

int quant_blocks(const QuantShape &sh);
hipError_t launch_quant_init(const QuantShape &sh, int dtype, const void *w, float *scale,
                             uint8_t *zero, hipStream_t st);
hipError_t launch_quantize(const QuantShape &sh, int dtype, const void *w, const float *scale,
                           const uint8_t *zero, uint8_t *codes, float *w_hat, void *w_op,
                           double *werr_part, hipStream_t st);
// scratch: werr_scratch_doubles(sh) doubles, the quantizer's per-block partials first
size_t werr_scratch_doubles(const QuantShape &sh);
hipError_t launch_werr_reduce(const QuantShape &sh, double *scratch, double *out, hipStream_t st);
// The persistent GEMMs take their tiles from a per-(device, stream) queue of 4 KiB that the
// library allocates on the first launch on a stream (not while the stream is being captured) and
// holds until the process ends.  While a GemmQueueNoAlloc lives on the calling thread, a stream
// without a queue yet keeps the static tile order and nothing is allocated.
struct GemmQueueNoAlloc {
    GemmQueueNoAlloc();
    ~GemmQueueNoAlloc();
};
// C[m][n] = sum_k A[m][k] B[n][k] (both operands k-contiguous), fp32 accumulate,
// C stored in dtype with row stride ldc.
hipError_t launch_gemm_nt(int dtype, const void *A, const void *B, void *C, int M, int N, int K,
                          int lda, int ldb, int ldc, hipStream_t st);
// Transposed values for attention: A = W_V [Hkv*dh][d], B = X [B*T][d]; C[r][b*Tp + perm(t)]
// (Tp = T rounded up to 32, perm = vt_perm within blocks of 32 tokens), ldc >= B*Tp.
// [Q|K] projection with the rotary embedding in the epilogue (the persistent kernel; every
// output column in a query or key head of head_dim columns, row r at position r % seq_T, tab the
// transposed table tab_t of launch_rope_table).  gemm_rope_fuses: whether a shape
// takes this path (16-bit, head_dim 64 or 128, the persistent kernel's shape conditions);
// launch_gemm_nt_rope returns hipErrorInvalidValue where it does not.
bool gemm_rope_fuses(int dtype, int M, int N, int K, int ldc, int head_dim);
hipError_t launch_gemm_nt_rope(int dtype, const void *A, const void *B, void *C, int M, int N, int K, int lda,
                               int ldb, int ldc, int head_dim, int seq_T, const float4 *tab_t, hipStream_t st);
hipError_t launch_gemm_nt_vt(int dtype, const void *A, const void *B, void *C, int M, int N, int K,
                             int lda, int ldb, int ldc, int seq_T, hipStream_t st);
// Same product with an fp32 C = alpha * (A B^T).  With C2 (same shape) the product may be split
// in two halves of K: *ksplit_used = 2 means C holds the first half's product and C2 the
// second's (their sum is the result), 1 means C holds all of it.
hipError_t launch_gemm_nt_f32out(int dtype, const void *A, const void *B, float *C, int M, int N, int K,
                                 int lda, int ldb, int ldc, float alpha, hipStream_t st, float *C2 = nullptr,
                                 int *ksplit_used = nullptr);

// ---- backward
// zero the padding columns of transposed values (T not a multiple of 32)
hipError_t launch_zero_vt_pad(int dtype, void *vt, int rows, int64_t ld, int batch, int T, hipStream_t st);
// V [B*T][ldv] in natural token order from transposed values [rows][ldt]
hipError_t launch_vt_to_v(int dtype, const void *vt, void *v, int rows, int64_t ldt, int batch, int T, int ldv,
                          hipStream_t st);
struct AttnBwdArgs {
    const void *q, *k, *v;        // Q, K [B*T][ldq] (head-major columns), V [B*T][ldv]
    int ldq, ldv;
    const void *g;                // [B*T][Hq*dh] storage dtype: a_hat - a_ref
    const float *lse2, *D;        // [B][Hq][T]
    void *dyt;                    // [R][ldt] storage dtype: (dQ | dK | dV)^T, unscaled by 2/N
    int64_t ldt;                  // row stride of dyt (>= B*T)
    int batch, seq_len, n_heads, n_kv_heads, head_dim;
    // KL attention-map term (when qt != NULL): dS += kl_scale (P - P_t), P_t the teacher's map
    // from its projection (qt, kt: same layout and ldq as q, k) and base-2 log-sum-exp lse_t
    const void *qt, *kt;
    const float *lse_t;
    float kl_scale;
    // with the KL term: dS is multiplied by grad_scale (a power of two, 1 unless fp16 needs the
    // range), so the dQ and dK rows of dY^T hold grad_scale times the gradient
    float grad_scale;
    // optional (16-bit, head_dim 64 / 128): dS as the dK pass rounds it for its product, 2 KiB per
    // (sequence, query head, 32-query tile qt, 32-key tile kt <= qt) at tile index qt (qt + 1) / 2 +
    // kt (attn_bwd_ds_bytes); the dQ pass then reads it instead of recomputing S and dP
    void *ds;
};
// bytes of the stored dS of AttnBwdArgs::ds
inline size_t attn_bwd_ds_bytes(int batch, int n_heads, int seq_len) {
    const size_t nq = (size_t)(seq_len + 31) / 32;
    return (size_t)batch * n_heads * (nq * (nq + 1) / 2) * 2048;
}
hipError_t launch_attn_bwd(int dtype, const AttnBwdArgs &a, hipStream_t st);
// out[c][r] = in[r][c] for an rows x cols matrix of the storage dtype: transpose_ld(rows) columns
// (rows rounded up to 64; the padding columns written as 0) at row stride out_ld >= that.
// transpose_stride: the stride of the backward's transposed operands, one 128-byte line past the
// padded length, so that their rows (the weight-gradient GEMM's k-runs) do not sit a power of two
// apart in memory (at 32768 tokens they would be 64 KiB apart).
inline int64_t transpose_ld(int64_t rows) { return (rows + 63) / 64 * 64; }
inline int64_t transpose_stride(int64_t rows) { return transpose_ld(rows) + 64; }
hipError_t launch_transpose(int dtype, const void *in, void *out, int rows, int cols, int64_t out_ld, hipStream_t st);
// zero columns [c0, ld) of a rows x ld matrix of the storage dtype
hipError_t launch_zero_cols(int dtype, void *p, int rows, int ld, int c0, hipStream_t st);
// ds[r][j] = gamma_m * sum_{k in group j} dw[r][k] phi[r][k] (eq. lsq); rows with bits 0 get 0.
// dw2 (nullable): a second partial of dw, added into dw first (dw = dw + dw2); then the rows of
// W_Q and W_K are multiplied by qk_unscale (a power of two; 1 leaves them).
hipError_t launch_lsq_scale_grad(const QuantShape &sh, int dtype, const void *w, const float *scale,
                                 const uint8_t *zero, float *dw, const float *dw2, float qk_unscale,
                                 const float gamma[3], float *ds, hipStream_t st);

// Causal GQA flash attention over one batch of sequences.
//   q/k: element pointers with Q(b,t,h,c) = q[(b*T + t)*ld + h*dh + c] (k with the key/value
//   head index); v[i]: transposed values, V(b,t,g,c) = v[(g*dh + c)*ldv + b*Tp + vt_perm(t)]
//   with Tp = T rounded up to 32 (as written by launch_gemm_nt_vt); nv value tensors share
//   one score matrix.
//   mode: bit flags ATT_LOSS (read a_ref, write (sse, sum a_ref^2) per wave into
//   partials), ATT_STORE_O (store the output, fp32, into a_out), ATT_STORE_LSE (store
//   the base-2 log-sum-exp of the scaled scores, lse2, for the backward), ATT_STORE_G (with
//   ATT_LOSS, one value tensor: the backward seed g = dtype(a_hat - a_ref) into g_out and
//   D[b][h][t] = sum_c g a_hat into d_out)
enum { ATT_LOSS = 1, ATT_STORE_O = 2, ATT_STORE_LSE = 4, ATT_STORE_G = 8 };
struct AttnArgs {
    const void *q, *k, *v[4];
    int ld;                       // row stride of q and k in elements
    int64_t ldv;                  // row stride of the transposed values (>= batch * Tp)
    int batch, seq_len, n_heads, n_kv_heads, head_dim;
    int nv;                       // 1, 2 or 4 value tensors
    int mode;
    const float *a_ref;           // [B][T][Hq*dh]
    float *a_out;                 // [B][T][Hq*dh]
    float *lse2;                  // [B][Hq][T]
    void *g_out;                  // [B][T][Hq*dh] storage dtype
    float *d_out;                 // [B][Hq][T]
    double *partials[4];          // per value tensor: [B][Hq][ceil(T/32)][2]
};
int attn_partials_per_seq(int seq_len, int n_heads);   // (sse, sum a^2) pairs per sequence
int attn_max_nv(int dtype);   // value tensors one attention pass can share a score matrix with
hipError_t launch_attn_fwd(int dtype, const AttnArgs &a, hipStream_t st);

// KL attention-map term D_KL(P || Q) (eq. joint_loss) per query row, P from the teacher's
// projection qt and cached base-2 log-sum-exp lse_t, Q from the student's projection qs (both
// [B*T][ld] with the query heads first and the key heads at column Hq*dh).  partials
// [B][Hq][ceil(T/32)][2]: (sum of the rows' KL, sum of (sum_j P_ij - 1)) per 32-query tile.
struct KlArgs {
    const void *qs, *qt;
    int ld;
    const float *lse_t;           // [B][Hq][T]
    int batch, seq_len, n_heads, n_kv_heads, head_dim;
    double *partials;
};
hipError_t launch_attn_kl(int dtype, const KlArgs &a, hipStream_t st);

// Forward-mode derivative of causal GQA attention (eq. gn's J_A v and J_Q v) along the tangent of
// the projection: q, k, vt as AttnArgs (the float point's projection, transposed values), qd, kd,
// vdt the same layout for the tangent X v^T.  partials [B][Hq][ceil(T/32)][9]: per 32-query block
// the sums <aQ,aQ> <aK,aK> <aV,aV> <aQ,aK> <aQ,aV> <aK,aV> zQ.I.zQ zK.I.zK zQ.I.zK.
struct JvpArgs {
    const void *q, *k, *vt, *qd, *kd, *vdt;
    int ld;                       // row stride of q, k, qd, kd in elements
    int64_t ldv;                  // row stride of vt, vdt
    int batch, seq_len, n_heads, n_kv_heads, head_dim;
    double *partials;
};
// partials for any head_dim / dtype (at head_dim 128, and for fp32 from 64, the rows of the output
// tangents are covered in passes that each write their own set); *n_partials: the sets written
size_t jvp_partials_bytes(int batch, int seq_len, int n_heads);
hipError_t launch_attn_jvp(int dtype, const JvpArgs &a, hipStream_t st, int64_t *n_partials);
// fixed-order sum of the n partials into parts[9] (parts: curv_parts_bytes() of scratch), then
// out[7] = (t_Q, t_K, t_V, pooled, h_QQ, h_KK, h_VV) of H = 2 J_A^T J_A + lambda J_Q^T I(P) J_Q
size_t curv_parts_bytes();
hipError_t launch_curv_forms(const double *partials, int64_t n, double *parts, double lambda, double *out,
                             hipStream_t st);
// w_out = the int8 probe (+-1) in the storage dtype
hipError_t launch_probe_to_dtype(int dtype, const int8_t *probe, int64_t n, void *w_out, hipStream_t st);

// Deterministic reductions of the attention partials.
//   partials [n_sets][B][per_seq][2] -> seq_sums [n_sets][B][2] -> per set: loss, per-seq.
hipError_t launch_reduce_seq(const double *partials, int n_sets, int batch, int per_seq,
                             double *seq_sums, hipStream_t st);
// out layout per set s: out[s*stride + 0] = sse, +1 = sse * inv_n, +2 = sum a^2,
// +3+b = sse of sequence b (when per_seq_out is nonzero).
hipError_t launch_reduce_final(const double *seq_sums, int n_sets, int batch, double inv_n,
                               double *out, int stride, int with_stats, int per_seq_out,
                               hipStream_t st);
// Sweep layout: loss[s] = sse of set s, loss_per_seq[s][b] (may be null).
// sum of squares of a [R][d] fp32 matrix over the row ranges [r[u], r[u+1]), u < n_units (<= 3),
// in a fixed order: part holds unit_sumsq_part_bytes(n_units), out[u] the sums (fp64)
struct UnitRows {
    int64_t r[4];
};
size_t unit_sumsq_part_bytes(int n_units);
hipError_t launch_unit_sumsq(const float *a, int64_t d, const UnitRows &rows, int n_units, double *part,
                             double *out, hipStream_t st);
// ---- STE fine-tuning (ste.hip)
struct AdamStep {
    float rate;          // alpha * cosine factor; the kernel multiplies by the mean grid step
    float beta1, beta2, eps;
    float bc1, bc2;      // bias corrections 1 - beta^t
    float floor;         // lower bound after the step (0: none)
};
hipError_t launch_round_to_dtype(int dtype, const float *src, void *dst, int64_t n, hipStream_t st);
hipError_t launch_adam(int dtype, float *theta, const float *g, float *m, float *v, int64_t n, const AdamStep &a,
                       const double *sbar, void *copy, hipStream_t st);
hipError_t launch_mean_scale(const float *s, int64_t groups, const UnitRows &rows, int unit_mask, double *sbar,
                             hipStream_t st);
hipError_t launch_gate(const double *loss, double *stats, int step, int log_slot, int force, int *flag,
                       hipStream_t st);
hipError_t launch_copy_if(const int *flag, const float *src, float *dst, int64_t n, hipStream_t st);
// out = a + lam * b (b may be NULL: out = a), one double each
hipError_t launch_axpy_f64(const double *a, const double *b, double lam, double *out, hipStream_t st);
hipError_t launch_zero_f32(float *a, int64_t n, hipStream_t st);
size_t count_diff_part_bytes();
hipError_t launch_count_diff(const uint8_t *a, const uint8_t *b, int64_t d, const UnitRows &rows, int unit_mask,
                             long long *part, double *out, hipStream_t st);
// ---- rotary position embedding (rope.hip): table [T][dh/2] of (cos, sin); rows: the fp32
// projection src [M][lds] (`heads` heads of dh columns from column 0) turned and rounded to the
// dtype into dst [M][ldd] (dst == src allowed for fp32); cols: yt [heads*dh rows][ldt], ncols
// tokens (a multiple of 8), in place; inverse turns the other way (the transpose)
size_t rope_table_bytes(int T, int dh);
// tab_t (NULL to skip): the same values as [dh/4][T] float4, (cos, sin) of pairs 2q and 2q + 1
hipError_t launch_rope_table(int T, int dh, double theta, float2 *tab, float4 *tab_t, hipStream_t st);
hipError_t launch_rope_rows(int dtype, const float *src, int64_t lds, void *dst, int64_t ldd, int64_t M, int T,
                            int heads, int dh, const float2 *tab, hipStream_t st);
hipError_t launch_rope_cols(int dtype, void *yt, int64_t ldt, int64_t ncols, int T, int heads, int dh,
                            const float2 *tab, bool inverse, hipStream_t st);
hipError_t launch_reduce_sweep(const double *seq_sums, int n_sets, int batch, double *loss,
                               double *loss_per_seq, hipStream_t st);

}  // namespace jab
