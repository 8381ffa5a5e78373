// api.cpp -- the C ABI of libjab: argument validation, workspace layout and the
// launch sequence of each entry point.  Everything here is host code; every
// arithmetic step of the method runs in the kernels of the .hip files.
//
// Paper correspondence of the entry points:
//   jab_quant_init / jab_quantize  eq. quant (per-(output row, group) grid)
//   jab_attn_ref                   the teacher A(X) of eq. joint_loss
//   jab_loss_fwd                   eq. joint_loss, squared-error term
//   jab_loss_sweep                 the loss for every (b_Q, b_K, b_V) candidate of
//                                  the bit allocation (eq. mckp's choice set)
//   jab_loss_bwd                   eq. lsq (STE on weights, LSQ on scales)
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/jab.h"
#include "kernels.h"

namespace {

thread_local std::string g_err;

jab_status fail(jab_status st, const std::string &msg) {
    g_err = msg;
    return st;
}

#define JAB_CHECK(cond, status, msg)            \
    do {                                        \
        if (!(cond)) return fail(status, msg);  \
    } while (0)

size_t esize(int dtype) { return dtype == JAB_F32 ? 4 : 2; }
size_t align_up(size_t v) { return (v + 255) & ~(size_t)255; }

bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

struct Dims {
    int64_t B, T, d, Hq, Hkv, dh, g, R, M, ng;
};

Dims dims_of(const jab_problem &p) {
    Dims D;
    D.B = p.batch; D.T = p.seq_len; D.d = p.d_model; D.Hq = p.n_heads; D.Hkv = p.n_kv_heads;
    D.dh = p.head_dim; D.g = p.group_size;
    D.R = (D.Hq + 2 * D.Hkv) * D.dh;
    D.M = D.B * D.T;
    D.ng = D.g > 0 ? D.d / D.g : 0;
    return D;
}

jab_status check_problem(const jab_problem *p) {
    JAB_CHECK(p != nullptr, JAB_E_INVALID, "problem is NULL");
    JAB_CHECK(p->batch > 0 && p->seq_len > 0 && p->d_model > 0 && p->n_heads > 0 &&
                  p->n_kv_heads > 0 && p->head_dim > 0 && p->group_size > 0,
              JAB_E_INVALID, "all problem sizes must be positive");
    JAB_CHECK(p->n_heads % p->n_kv_heads == 0, JAB_E_INVALID, "n_heads must be a multiple of n_kv_heads");
    JAB_CHECK(p->d_model % p->group_size == 0, JAB_E_INVALID, "d_model must be a multiple of group_size");
    JAB_CHECK(p->scheme == JAB_ASYM || p->scheme == JAB_SYM, JAB_E_INVALID, "unknown quantization scheme");
    JAB_CHECK(std::isfinite(p->rope_theta) && p->rope_theta >= 0.f, JAB_E_INVALID,
              "rope_theta must be finite and >= 0");
    JAB_CHECK(p->dtype == JAB_F32 || p->dtype == JAB_F16 || p->dtype == JAB_BF16, JAB_E_UNSUPPORTED,
              "dtype must be JAB_F32, JAB_F16 or JAB_BF16");
    JAB_CHECK(p->head_dim == 16 || p->head_dim == 64 || p->head_dim == 128, JAB_E_UNSUPPORTED,
              "head_dim must be 16, 64 or 128");
    JAB_CHECK(p->group_size == 32 || p->group_size == 64 || p->group_size == 128, JAB_E_UNSUPPORTED,
              "group_size must be 32, 64 or 128");
    const int G = p->n_heads / p->n_kv_heads;
    JAB_CHECK(G == 1 || G == 2 || G % 4 == 0, JAB_E_UNSUPPORTED,
              "n_heads / n_kv_heads must be 1, 2 or a multiple of 4");
    const Dims D = dims_of(*p);
    JAB_CHECK(D.M <= INT32_MAX && D.R * D.d <= INT32_MAX && D.M * D.R <= ((int64_t)1 << 40),
              JAB_E_UNSUPPORTED, "problem too large for 32-bit row indices");
    return JAB_OK;
}

jab_status check_bits(int b) {
    JAB_CHECK(b == 0 || (b >= 2 && b <= 8), JAB_E_INVALID, "bit-widths must be 0 or 2..8");
    return JAB_OK;
}

jab_status check_quant(const jab_problem &p, const jab_quant *q) {
    JAB_CHECK(q != nullptr, JAB_E_INVALID, "quant is NULL");
    bool any = false;
    for (int m = 0; m < 3; ++m) {
        jab_status s = check_bits(q->bits[m]);
        if (s) return s;
        any |= q->bits[m] != 0;
    }
    if (any) {
        JAB_CHECK(q->scale != nullptr && aligned(q->scale, 4), JAB_E_INVALID, "scale is NULL or misaligned");
        if (p.scheme == JAB_ASYM)
            JAB_CHECK(q->zero != nullptr, JAB_E_INVALID, "zero-points are required for JAB_ASYM");
        else
            JAB_CHECK(q->zero == nullptr, JAB_E_INVALID, "zero-points must be NULL for JAB_SYM");
    }
    return JAB_OK;
}

jab::QuantShape quant_shape(const jab_problem &p, const int bits[3]) {
    const Dims D = dims_of(p);
    jab::QuantShape sh;
    sh.rows = (int)D.R; sh.cols = (int)D.d; sh.group = (int)D.g;
    sh.row_k = (int)(D.Hq * D.dh); sh.row_v = (int)((D.Hq + D.Hkv) * D.dh);
    for (int m = 0; m < 3; ++m) sh.bits[m] = bits[m];
    sh.scheme = p.scheme;
    return sh;
}

// ---------------------------------------------------------------- workspace
struct Carver {
    char *base;
    size_t off = 0;
    explicit Carver(void *b) : base(static_cast<char *>(b)) {}
    void *take(size_t bytes) {
        void *p = base ? base + off : nullptr;
        off += align_up(bytes);
        return p;
    }
};

// One projection set: [Q | K] row-major [B*T][(Hq+Hkv)*dh] and the transposed values
// [Hkv*dh][B*Tp] (Tp = T rounded up to 32, key order vt_perm inside blocks of 32).
struct Proj {
    void *qk, *vt;
};

struct FwdWs {
    void *w_op;
    Proj proj[8];                 // one per candidate bit-width (sweep), else proj[0]
    double *partials, *seq_sums;
};

// [Q|K] rows plus 32 rows of slack: the attention loads keys in blocks of 32 and reads up to
// 31 rows past the last token (keys the causal mask removes)
constexpr int64_t QK_SLACK_ROWS = 32;
size_t qk_main_bytes(const jab_problem &p) {
    const Dims D = dims_of(p);
    return (size_t)((D.M + QK_SLACK_ROWS) * (D.Hq + D.Hkv) * D.dh) * esize(p.dtype);
}
// 16-bit RoPE shapes whose [Q|K] GEMM cannot take the rotation in its epilogue project into an
// fp32 buffer first (the rotation acts on the projection before its rounding)
bool rope_needs_f32(const jab_problem &p) {
    const Dims D = dims_of(p);
    const int nqk = (int)((D.Hq + D.Hkv) * D.dh);
    return p.rope_theta > 0.f && p.dtype != JAB_F32 &&
           !jab::gemm_rope_fuses(p.dtype, (int)D.M, nqk, (int)D.d, nqk, p.head_dim);
}
size_t rope_f32_bytes(const jab_problem &p) {
    const Dims D = dims_of(p);
    return rope_needs_f32(p) ? (size_t)(D.M * (D.Hq + D.Hkv) * D.dh) * sizeof(float) : 0;
}
// the (cos, sin) table [T][dh/2] and its transposed copy (what the fused epilogue reads)
size_t rope_tab_bytes(const jab_problem &p) {
    return p.rope_theta > 0.f ? 2 * ((jab::rope_table_bytes(p.seq_len, p.head_dim) + 255) / 256 * 256) : 0;
}
// with RoPE the rotation table of the call (and the fp32 projection, where needed) follow the
// projection they rotate
size_t qk_bytes(const jab_problem &p) {
    return qk_main_bytes(p) + rope_tab_bytes(p) + rope_f32_bytes(p);
}
// transposed values: each sequence padded to a multiple of 32 tokens
int64_t vt_ld(const jab_problem &p) { return (int64_t)p.batch * ((p.seq_len + 31) / 32 * 32); }
size_t vt_bytes(const jab_problem &p) {
    const Dims D = dims_of(p);
    return (size_t)(D.Hkv * D.dh * vt_ld(p)) * esize(p.dtype);
}

int per_seq_waves(const jab_problem &p) { return jab::attn_partials_per_seq(p.seq_len, p.n_heads); }

FwdWs carve_fwd(const jab_problem &p, void *ws, size_t *bytes, int n_sets, int n_y) {
    const Dims D = dims_of(p);
    Carver c(ws);
    FwdWs w;
    w.w_op = c.take((size_t)(D.R * D.d) * esize(p.dtype));
    for (int i = 0; i < n_y; ++i) {
        w.proj[i].qk = c.take(qk_bytes(p));
        w.proj[i].vt = c.take(vt_bytes(p));
    }
    w.partials = static_cast<double *>(c.take((size_t)n_sets * D.B * per_seq_waves(p) * 2 * sizeof(double)));
    w.seq_sums = static_cast<double *>(c.take((size_t)n_sets * D.B * 2 * sizeof(double)));
    *bytes = c.off;
    return w;
}

// Curvature: the probe as a projection operand, the projection at the float point and its tangent,
// the tangent sums per (pass, sequence, head, 32-query block) and their total
struct CurvWs {
    void *w_op;
    Proj base, tan;
    double *partials, *parts;
};
CurvWs carve_curv(const jab_problem &p, void *ws, size_t *bytes) {
    const Dims D = dims_of(p);
    Carver c(ws);
    CurvWs r;
    r.w_op = c.take((size_t)(D.R * D.d) * esize(p.dtype));
    for (Proj *pr : {&r.base, &r.tan}) {
        pr->qk = c.take(qk_bytes(p));
        pr->vt = c.take(vt_bytes(p));
    }
    r.partials = static_cast<double *>(c.take(jab::jvp_partials_bytes(p.batch, p.seq_len, p.n_heads)));
    r.parts = static_cast<double *>(c.take(jab::curv_parts_bytes()));
    *bytes = c.off;
    return r;
}

struct BwdWs {
    FwdWs f;
    float *lse2, *D;
    void *g, *dyt, *xt, *vrow;
    float *dw2;                   // second half of a split weight-gradient product
    void *ds;                     // dS of the attention backward for its dQ pass (null: recomputed)
};

// The 16-bit backward at head_dim 64 / 128 keeps dS (2 bytes per causal (query, key, head) entry)
// between its dK and dQ passes, up to g_ds_limit bytes; past that the dQ pass recomputes it.
size_t g_ds_limit = (size_t)8 << 30;
size_t bwd_ds_bytes(const jab_problem &p) {
    if (p.dtype == JAB_F32 || (p.head_dim != 64 && p.head_dim != 128)) return 0;
    const size_t b = jab::attn_bwd_ds_bytes(p.batch, p.n_heads, p.seq_len);
    return b <= g_ds_limit ? b : 0;
}

BwdWs carve_bwd(const jab_problem &p, void *ws, size_t *bytes) {
    const Dims D = dims_of(p);
    size_t fwd_bytes = 0;
    BwdWs w;
    w.f = carve_fwd(p, ws, &fwd_bytes, 2, 1);     // loss partials, and the KL term's for jab_loss_bwd_kl
    Carver c(ws ? static_cast<char *>(ws) + fwd_bytes : nullptr);
    const size_t es = esize(p.dtype);
    const int64_t Ms = jab::transpose_stride(D.M);
    w.lse2 = static_cast<float *>(c.take((size_t)(D.B * D.Hq * D.T) * sizeof(float)));
    w.D = static_cast<float *>(c.take((size_t)(D.B * D.Hq * D.T) * sizeof(float)));
    w.g = c.take((size_t)(D.M * D.Hq * D.dh) * es);
    w.dyt = c.take((size_t)(D.R * Ms) * es);
    w.xt = c.take((size_t)(D.d * Ms) * es);
    w.vrow = c.take((size_t)(D.M * D.Hkv * D.dh) * es);
    w.dw2 = static_cast<float *>(c.take((size_t)(D.R * D.d) * sizeof(float)));
    const size_t dsb = bwd_ds_bytes(p);
    w.ds = dsb ? c.take(dsb) : nullptr;
    *bytes = fwd_bytes + c.off;
    return w;
}

// Fisher scores: the gradients jab_loss_bwd writes to caller buffers, and the partial sums
struct FisherWs {
    float *dw, *ds;
    double *part, *loss;
};
FisherWs carve_fisher(const jab_problem &p, Carver &c) {
    const Dims D = dims_of(p);
    FisherWs f;
    f.dw = static_cast<float *>(c.take((size_t)(D.R * D.d) * sizeof(float)));
    f.ds = static_cast<float *>(c.take((size_t)(D.R * (D.d / D.g)) * sizeof(float)));
    f.part = static_cast<double *>(c.take(jab::unit_sumsq_part_bytes(3)));
    f.loss = static_cast<double *>(c.take((size_t)2 * (3 + D.B) * sizeof(double)));
    return f;
}

// STE fine-tuning: Adam moments, the best checkpoint, the start's weights and codes, logs
struct SteWs {
    float *dw, *ds, *m_w, *v_w, *best_w, *m_s, *v_s, *best_s;
    void *w0;
    uint8_t *codes0, *codes1;
    double *train_out, *held_out, *sbar, *score;
    long long *part;
    int *flag;
};
SteWs carve_ste(const jab_problem &p, Carver &c) {
    const Dims D = dims_of(p);
    const size_t nw = (size_t)(D.R * D.d), ns = (size_t)(D.R * (D.d / D.g));
    SteWs t;
    t.dw = static_cast<float *>(c.take(nw * 4));
    t.m_w = static_cast<float *>(c.take(nw * 4));
    t.v_w = static_cast<float *>(c.take(nw * 4));
    t.best_w = static_cast<float *>(c.take(nw * 4));
    t.ds = static_cast<float *>(c.take(ns * 4));
    t.m_s = static_cast<float *>(c.take(ns * 4));
    t.v_s = static_cast<float *>(c.take(ns * 4));
    t.best_s = static_cast<float *>(c.take(ns * 4));
    t.w0 = c.take(nw * esize(p.dtype));
    t.codes0 = static_cast<uint8_t *>(c.take(nw));
    t.codes1 = static_cast<uint8_t *>(c.take(nw));
    t.train_out = static_cast<double *>(c.take((size_t)2 * (3 + D.B) * 8));
    t.held_out = static_cast<double *>(c.take((size_t)2 * (3 + D.B) * 8));
    t.sbar = static_cast<double *>(c.take(8));
    t.score = static_cast<double *>(c.take(8));
    t.part = static_cast<long long *>(c.take(jab::count_diff_part_bytes()));
    t.flag = static_cast<int *>(c.take(4));
    return t;
}

// ---------------------------------------------------------------- timing
struct TimedLaunch {
    int kind;
    hipEvent_t a, b;
};
struct TimingState {
    bool on = false;
    std::vector<TimedLaunch> pending;
    std::vector<hipEvent_t> pool;
    double ms[JAB_KT_COUNT] = {};
    int64_t n[JAB_KT_COUNT] = {};
};
thread_local TimingState g_timing;

hipEvent_t take_event() {
    if (!g_timing.pool.empty()) {
        hipEvent_t e = g_timing.pool.back();
        g_timing.pool.pop_back();
        return e;
    }
    // timing only: no system-scope fence (cache write-back and invalidation) when the event is
    // recorded, which otherwise opens a gap of about 10 us before the next kernel
    hipEvent_t e = nullptr;
    if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
    return e;
}

template <typename F>
jab_status launch(int kind, hipStream_t st, const char *what, F &&f) {
    hipEvent_t a = nullptr, b = nullptr;
    if (g_timing.on) {
        a = take_event();
        b = take_event();
        if (a) (void)hipEventRecord(a, st);
    }
    const hipError_t e = f();
    if (g_timing.on && a && b) {
        (void)hipEventRecord(b, st);
        g_timing.pending.push_back({kind, a, b});
    }
    if (e != hipSuccess)
        return fail(JAB_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
    return JAB_OK;
}

#define JAB_RUN(kind, st, what, expr)                                 \
    do {                                                              \
        jab_status s__ = launch(kind, st, what, [&]() { return (expr); }); \
        if (s__) return s__;                                          \
    } while (0)

// ---------------------------------------------------------------- shared sequences
jab_status run_project(const jab_problem &p, const void *x, const void *w_operand, void *y,
                       hipStream_t st) {
    const Dims D = dims_of(p);
    JAB_RUN(JAB_KT_GEMM, st, "projection GEMM",
            jab::launch_gemm_nt(p.dtype, x, w_operand, y, (int)D.M, (int)D.R, (int)D.d, (int)D.d,
                                (int)D.d, (int)D.R, st));
    return JAB_OK;
}

// [Q|K] = X W_QK^T and V^T = W_V X^T (same matrix-core kernel, operands swapped).
jab_status run_project_split(const jab_problem &p, const void *x, const void *w_operand, const Proj &pr,
                             hipStream_t st) {
    const Dims D = dims_of(p);
    const int nqk = (int)((D.Hq + D.Hkv) * D.dh);
    const void *w_v = static_cast<const char *>(w_operand) + (size_t)nqk * D.d * esize(p.dtype);
    if (p.rope_theta > 0.f) {
        // the rotary embedding turns the projection as accumulated (fp32) and rounds once: in the
        // [Q|K] GEMM's epilogue where the persistent kernel takes the shape, else as a pass over an
        // fp32 projection
        char *tail = static_cast<char *>(pr.qk) + qk_main_bytes(p);
        float2 *tab = reinterpret_cast<float2 *>(tail);
        float4 *tab_t = reinterpret_cast<float4 *>(tail + rope_tab_bytes(p) / 2);
        JAB_RUN(JAB_KT_MISC, st, "rotary table",
                jab::launch_rope_table(p.seq_len, p.head_dim, p.rope_theta, tab, tab_t, st));
        const int heads = p.n_heads + p.n_kv_heads;
        if (jab::gemm_rope_fuses(p.dtype, (int)D.M, nqk, (int)D.d, nqk, p.head_dim)) {
            JAB_RUN(JAB_KT_GEMM, st, "projection GEMM (Q, K) with the rotary embedding",
                    jab::launch_gemm_nt_rope(p.dtype, x, w_operand, pr.qk, (int)D.M, nqk, (int)D.d, (int)D.d,
                                             (int)D.d, nqk, p.head_dim, p.seq_len, tab_t, st));
        } else if (p.dtype == JAB_F32) {
            JAB_RUN(JAB_KT_GEMM, st, "projection GEMM (Q, K)",
                    jab::launch_gemm_nt(p.dtype, x, w_operand, pr.qk, (int)D.M, nqk, (int)D.d, (int)D.d, (int)D.d,
                                        nqk, st));
            JAB_RUN(JAB_KT_MISC, st, "rotary embedding",
                    jab::launch_rope_rows(p.dtype, static_cast<const float *>(pr.qk), nqk, pr.qk, nqk, D.M,
                                          p.seq_len, heads, p.head_dim, tab, st));
        } else {
            float *y32 = reinterpret_cast<float *>(tail + rope_tab_bytes(p));
            JAB_RUN(JAB_KT_GEMM, st, "projection GEMM (Q, K), fp32",
                    jab::launch_gemm_nt_f32out(p.dtype, x, w_operand, y32, (int)D.M, nqk, (int)D.d, (int)D.d,
                                               (int)D.d, nqk, 1.f, st, nullptr, nullptr));
            JAB_RUN(JAB_KT_MISC, st, "rotary embedding",
                    jab::launch_rope_rows(p.dtype, y32, nqk, pr.qk, nqk, D.M, p.seq_len, heads, p.head_dim, tab,
                                          st));
        }
    } else {
        JAB_RUN(JAB_KT_GEMM, st, "projection GEMM (Q, K)",
                jab::launch_gemm_nt(p.dtype, x, w_operand, pr.qk, (int)D.M, nqk, (int)D.d, (int)D.d, (int)D.d,
                                    nqk, st));
    }
    JAB_RUN(JAB_KT_GEMM_VT, st, "projection GEMM (V transposed)",
            jab::launch_gemm_nt_vt(p.dtype, w_v, x, pr.vt, (int)(D.Hkv * D.dh), (int)D.M, (int)D.d,
                                   (int)D.d, (int)D.d, (int)vt_ld(p), p.seq_len, st));
    JAB_RUN(JAB_KT_MISC, st, "value padding",
            jab::launch_zero_vt_pad(p.dtype, pr.vt, (int)(D.Hkv * D.dh), vt_ld(p), p.batch, p.seq_len, st));
    return JAB_OK;
}

// the KL attention-map term in the backward: the teacher's cache and lambda_KL
struct KlBwd {
    const void *qk_ref;
    const float *lse_ref;
    float lambda;
};

jab_status run_bwd(const jab_problem *p, const void *x, const void *w, const jab_quant *q, const float *a_ref,
                   const float *lsq_gscale, double *out, float *dw, float *dscale, const BwdWs &W, hipStream_t st,
                   bool transpose_x = true, const KlBwd *kl = nullptr);

jab::AttnArgs attn_args(const jab_problem &p, const Proj &pq, const Proj &pk, const Proj &pv) {
    const Dims D = dims_of(p);
    const size_t es = esize(p.dtype);
    jab::AttnArgs a;
    std::memset(&a, 0, sizeof(a));
    a.q = pq.qk;
    a.k = static_cast<const char *>(pk.qk) + (size_t)(D.Hq * D.dh) * es;
    a.v[0] = pv.vt;
    a.ld = (int)((D.Hq + D.Hkv) * D.dh);
    a.ldv = vt_ld(p);
    a.batch = p.batch; a.seq_len = p.seq_len; a.n_heads = p.n_heads; a.n_kv_heads = p.n_kv_heads;
    a.head_dim = p.head_dim;
    a.nv = 1;
    return a;
}

}  // namespace

namespace jab {
// the calling thread's error message (host routines in other translation units report here)
std::string &last_error_ref() { return g_err; }
}  // namespace jab

// =================================================================== ABI
extern "C" {

const char *jab_status_string(int32_t s) {
    switch (s) {
    case JAB_OK: return "JAB_OK";
    case JAB_E_INVALID: return "JAB_E_INVALID";
    case JAB_E_UNSUPPORTED: return "JAB_E_UNSUPPORTED";
    case JAB_E_WORKSPACE: return "JAB_E_WORKSPACE";
    case JAB_E_HIP: return "JAB_E_HIP";
    default: return "unknown jab_status";
    }
}

const char *jab_last_error(void) { return g_err.c_str(); }

size_t jab_workspace_size(const jab_problem *p, int32_t op, int32_t n_bits) {
    if (check_problem(p) != JAB_OK) return 0;
    size_t bytes = 0;
    const Dims D = dims_of(*p);
    switch (op) {
    case JAB_OP_FWD: carve_fwd(*p, nullptr, &bytes, 1, 1); return bytes;
    case JAB_OP_FWD_KL: carve_fwd(*p, nullptr, &bytes, 2, 1); return bytes;
    case JAB_OP_CURVATURE: carve_curv(*p, nullptr, &bytes); return bytes;
    case JAB_OP_STE: {
        carve_bwd(*p, nullptr, &bytes);
        Carver c(nullptr);
        carve_ste(*p, c);
        return bytes + c.off;
    }
    case JAB_OP_FISHER: {
        carve_bwd(*p, nullptr, &bytes);
        Carver c(nullptr);
        carve_fisher(*p, c);
        return bytes + c.off;
    }
    case JAB_OP_REF: {
        Carver c(nullptr);
        c.take(qk_bytes(*p));
        c.take(vt_bytes(*p));
        return c.off;
    }
    case JAB_OP_PROJECT: {
        Carver c(nullptr);
        c.take((size_t)(D.R * D.d) * esize(p->dtype));
        return c.off;
    }
    case JAB_OP_QUANTIZE: {
        Carver c(nullptr);
        const int nobits[3] = {0, 0, 0};
        c.take(jab::werr_scratch_doubles(quant_shape(*p, nobits)) * sizeof(double));
        return c.off;
    }
    case JAB_OP_BWD: carve_bwd(*p, nullptr, &bytes); return bytes;
    case JAB_OP_SWEEP: {
        if (n_bits <= 0 || n_bits > 7) return 0;
        carve_fwd(*p, nullptr, &bytes, n_bits * n_bits * n_bits, n_bits);
        return bytes;
    }
    default: return 0;
    }
}

jab_status jab_quant_init(const jab_problem *p, const void *w, const int32_t *bits, float *scale,
                          uint8_t *zero, void *stream) {
    jab_status s = check_problem(p);
    if (s) return s;
    JAB_CHECK(w && aligned(w, 16), JAB_E_INVALID, "w is NULL or not 16-byte aligned");
    JAB_CHECK(bits, JAB_E_INVALID, "bits is NULL");
    for (int m = 0; m < 3; ++m)
        if ((s = check_bits(bits[m]))) return s;
    JAB_CHECK(scale && aligned(scale, 4), JAB_E_INVALID, "scale is NULL or misaligned");
    if (p->scheme == JAB_ASYM)
        JAB_CHECK(zero, JAB_E_INVALID, "zero-points are required for JAB_ASYM");
    else
        JAB_CHECK(!zero, JAB_E_INVALID, "zero-points must be NULL for JAB_SYM");
    const int b3[3] = {bits[0], bits[1], bits[2]};
    const jab::QuantShape sh = quant_shape(*p, b3);
    hipStream_t st = static_cast<hipStream_t>(stream);
    JAB_RUN(JAB_KT_QUANT, st, "quant_init", jab::launch_quant_init(sh, p->dtype, w, scale, zero, st));
    return JAB_OK;
}

jab_status jab_quantize(const jab_problem *p, const void *w, const jab_quant *q, uint8_t *codes,
                        float *w_hat, double *werr, void *ws, size_t ws_bytes, void *stream) {
    jab_status s = check_problem(p);
    if (s) return s;
    if ((s = check_quant(*p, q))) return s;
    JAB_CHECK(w && aligned(w, 16), JAB_E_INVALID, "w is NULL or not 16-byte aligned");
    JAB_CHECK(!codes || aligned(codes, 16), JAB_E_INVALID, "codes not 16-byte aligned");
    JAB_CHECK(!w_hat || aligned(w_hat, 16), JAB_E_INVALID, "w_hat not 16-byte aligned");
    JAB_CHECK(!werr || aligned(werr, 8), JAB_E_INVALID, "werr not 8-byte aligned");
    const jab::QuantShape sh = quant_shape(*p, q->bits);
    double *part = nullptr;
    if (werr) {
        const size_t need = jab_workspace_size(p, JAB_OP_QUANTIZE, 0);
        JAB_CHECK(ws && aligned(ws, 256), JAB_E_INVALID, "workspace is NULL or not 256-byte aligned");
        JAB_CHECK(ws_bytes >= need, JAB_E_WORKSPACE, "workspace too small for jab_quantize");
        part = static_cast<double *>(ws);
    }
    hipStream_t st = static_cast<hipStream_t>(stream);
    JAB_RUN(JAB_KT_QUANT, st, "quantize",
            jab::launch_quantize(sh, p->dtype, w, q->scale, q->zero, codes, w_hat, nullptr, part, st));
    if (werr)
        JAB_RUN(JAB_KT_REDUCE, st, "werr reduce", jab::launch_werr_reduce(sh, part, werr, st));
    return JAB_OK;
}

jab_status jab_project(const jab_problem *p, const void *x, const void *w, const jab_quant *q,
                       void *y, void *ws, size_t ws_bytes, void *stream) {
    jab_status s = check_problem(p);
    if (s) return s;
    if (q && (s = check_quant(*p, q))) return s;
    JAB_CHECK(x && aligned(x, 16) && w && aligned(w, 16), JAB_E_INVALID, "x / w NULL or not 16-byte aligned");
    JAB_CHECK(y && aligned(y, 16), JAB_E_INVALID, "y NULL or not 16-byte aligned");
    hipStream_t st = static_cast<hipStream_t>(stream);
    const void *wop = w;
    if (q) {
        const size_t need = jab_workspace_size(p, JAB_OP_PROJECT, 0);
        JAB_CHECK(ws && aligned(ws, 256), JAB_E_INVALID, "workspace is NULL or not 256-byte aligned");
        JAB_CHECK(ws_bytes >= need, JAB_E_WORKSPACE, "workspace too small for jab_project");
        const jab::QuantShape sh = quant_shape(*p, q->bits);
        JAB_RUN(JAB_KT_QUANT, st, "quantize",
                jab::launch_quantize(sh, p->dtype, w, q->scale, q->zero, nullptr, nullptr, ws, nullptr, st));
        wop = ws;
    }
    return run_project(*p, x, wop, y, st);
}

jab_status jab_attn_ref(const jab_problem *p, const void *x, const void *w, float *a_ref, void *ws,
                        size_t ws_bytes, void *stream) {
    jab_status s = check_problem(p);
    if (s) return s;
    JAB_CHECK(x && aligned(x, 16) && w && aligned(w, 16), JAB_E_INVALID, "x / w NULL or not 16-byte aligned");
    JAB_CHECK(a_ref && aligned(a_ref, 16), JAB_E_INVALID, "a_ref NULL or not 16-byte aligned");
    JAB_CHECK(ws && aligned(ws, 256), JAB_E_INVALID, "workspace is NULL or not 256-byte aligned");
    JAB_CHECK(ws_bytes >= jab_workspace_size(p, JAB_OP_REF, 0), JAB_E_WORKSPACE,
              "workspace too small for jab_attn_ref");
    hipStream_t st = static_cast<hipStream_t>(stream);
    Carver c(ws);
    Proj pr;
    pr.qk = c.take(qk_bytes(*p));
    pr.vt = c.take(vt_bytes(*p));
    if ((s = run_project_split(*p, x, w, pr, st))) return s;
    jab::AttnArgs a = attn_args(*p, pr, pr, pr);
    a.mode = jab::ATT_STORE_O;
    a.a_out = a_ref;
    JAB_RUN(JAB_KT_ATTN, st, "attention", jab::launch_attn_fwd(p->dtype, a, st));
    return JAB_OK;
}

jab_status jab_loss_fwd(const jab_problem *p, const void *x, const void *w, const jab_quant *q,
                        const float *a_ref, double *out, void *ws, size_t ws_bytes, void *stream) {
    jab_status s = check_problem(p);
    if (s) return s;
    if ((s = check_quant(*p, q))) return s;
    JAB_CHECK(x && aligned(x, 16) && w && aligned(w, 16), JAB_E_INVALID, "x / w NULL or not 16-byte aligned");
    JAB_CHECK(a_ref && aligned(a_ref, 16), JAB_E_INVALID, "a_ref NULL or not 16-byte aligned");
    JAB_CHECK(out && aligned(out, 8), JAB_E_INVALID, "out NULL or not 8-byte aligned");
    JAB_CHECK(ws && aligned(ws, 256), JAB_E_INVALID, "workspace is NULL or not 256-byte aligned");
    size_t need = 0;
    const FwdWs W = carve_fwd(*p, ws, &need, 1, 1);
    JAB_CHECK(ws_bytes >= need, JAB_E_WORKSPACE, "workspace too small for jab_loss_fwd");
    const Dims D = dims_of(*p);
    hipStream_t st = static_cast<hipStream_t>(stream);
    const jab::QuantShape sh = quant_shape(*p, q->bits);
    JAB_RUN(JAB_KT_QUANT, st, "quantize",
            jab::launch_quantize(sh, p->dtype, w, q->scale, q->zero, nullptr, nullptr, W.w_op, nullptr, st));
    if ((s = run_project_split(*p, x, W.w_op, W.proj[0], st))) return s;
    jab::AttnArgs a = attn_args(*p, W.proj[0], W.proj[0], W.proj[0]);
    a.mode = jab::ATT_LOSS;
    a.a_ref = a_ref;
    a.partials[0] = W.partials;
    JAB_RUN(JAB_KT_ATTN, st, "attention", jab::launch_attn_fwd(p->dtype, a, st));
    JAB_RUN(JAB_KT_REDUCE, st, "reduce",
            jab::launch_reduce_seq(W.partials, 1, p->batch, per_seq_waves(*p), W.seq_sums, st));
    const double inv_n = 1.0 / ((double)D.M * (double)(D.Hq * D.dh));
    JAB_RUN(JAB_KT_REDUCE, st, "reduce",
            jab::launch_reduce_final(W.seq_sums, 1, p->batch, inv_n, out, 0, 1, 1, st));
    return JAB_OK;
}

jab_status jab_attn_ref_kl(const jab_problem *p, const void *x, const void *w, float *a_ref, void *qk_ref,
                           float *lse_ref, void *ws, size_t ws_bytes, void *stream) {
    jab_status s = check_problem(p);
    if (s) return s;
    JAB_CHECK(x && aligned(x, 16) && w && aligned(w, 16), JAB_E_INVALID, "x / w NULL or not 16-byte aligned");
    JAB_CHECK(a_ref && aligned(a_ref, 16), JAB_E_INVALID, "a_ref NULL or not 16-byte aligned");
    JAB_CHECK(qk_ref && aligned(qk_ref, 16), JAB_E_INVALID, "qk_ref NULL or not 16-byte aligned");
    JAB_CHECK(lse_ref && aligned(lse_ref, 4), JAB_E_INVALID, "lse_ref NULL or not 4-byte aligned");
    JAB_CHECK(ws && aligned(ws, 256), JAB_E_INVALID, "workspace is NULL or not 256-byte aligned");
    JAB_CHECK(ws_bytes >= jab_workspace_size(p, JAB_OP_REF, 0), JAB_E_WORKSPACE,
              "workspace too small for jab_attn_ref_kl");
    const Dims D = dims_of(*p);
    hipStream_t st = static_cast<hipStream_t>(stream);
    Carver c(ws);
    Proj pr;
    pr.qk = c.take(qk_bytes(*p));
    pr.vt = c.take(vt_bytes(*p));
    if ((s = run_project_split(*p, x, w, pr, st))) return s;
    jab::AttnArgs a = attn_args(*p, pr, pr, pr);
    a.mode = jab::ATT_STORE_O | jab::ATT_STORE_LSE;
    a.a_out = a_ref;
    a.lse2 = lse_ref;
    JAB_RUN(JAB_KT_ATTN, st, "attention", jab::launch_attn_fwd(p->dtype, a, st));
    // the projection without the slack rows the attention kernels read past the last token
    const size_t qk_keep = (size_t)(D.M * (D.Hq + D.Hkv) * D.dh) * esize(p->dtype);
    JAB_RUN(JAB_KT_MISC, st, "teacher projection copy",
            hipMemcpyAsync(qk_ref, pr.qk, qk_keep, hipMemcpyDeviceToDevice, st));
    return JAB_OK;
}

jab_status jab_loss_fwd_kl(const jab_problem *p, const void *x, const void *w, const jab_quant *q,
                           const float *a_ref, const void *qk_ref, const float *lse_ref, double *out, void *ws,
                           size_t ws_bytes, void *stream) {
    jab_status s = check_problem(p);
    if (s) return s;
    if ((s = check_quant(*p, q))) return s;
    JAB_CHECK(x && aligned(x, 16) && w && aligned(w, 16), JAB_E_INVALID, "x / w NULL or not 16-byte aligned");
    JAB_CHECK(a_ref && aligned(a_ref, 16), JAB_E_INVALID, "a_ref NULL or not 16-byte aligned");
    JAB_CHECK(qk_ref && aligned(qk_ref, 16), JAB_E_INVALID, "qk_ref NULL or not 16-byte aligned");
    JAB_CHECK(lse_ref && aligned(lse_ref, 4), JAB_E_INVALID, "lse_ref NULL or not 4-byte aligned");
    JAB_CHECK(out && aligned(out, 8), JAB_E_INVALID, "out NULL or not 8-byte aligned");
    JAB_CHECK(ws && aligned(ws, 256), JAB_E_INVALID, "workspace is NULL or not 256-byte aligned");
    size_t need = 0;
    const FwdWs W = carve_fwd(*p, ws, &need, 2, 1);
    JAB_CHECK(ws_bytes >= need, JAB_E_WORKSPACE, "workspace too small for jab_loss_fwd_kl");
    const Dims D = dims_of(*p);
    hipStream_t st = static_cast<hipStream_t>(stream);
    const jab::QuantShape sh = quant_shape(*p, q->bits);
    JAB_RUN(JAB_KT_QUANT, st, "quantize",
            jab::launch_quantize(sh, p->dtype, w, q->scale, q->zero, nullptr, nullptr, W.w_op, nullptr, st));
    if ((s = run_project_split(*p, x, W.w_op, W.proj[0], st))) return s;
    jab::AttnArgs a = attn_args(*p, W.proj[0], W.proj[0], W.proj[0]);
    a.mode = jab::ATT_LOSS;
    a.a_ref = a_ref;
    a.partials[0] = W.partials;
    JAB_RUN(JAB_KT_ATTN, st, "attention", jab::launch_attn_fwd(p->dtype, a, st));
    const int per_seq = per_seq_waves(*p);
    double *kl_partials = W.partials + (size_t)D.B * per_seq * 2;
    jab::KlArgs k;
    std::memset(&k, 0, sizeof(k));
    k.qs = W.proj[0].qk;
    k.qt = qk_ref;
    k.ld = (int)((D.Hq + D.Hkv) * D.dh);
    k.lse_t = lse_ref;
    k.batch = p->batch; k.seq_len = p->seq_len; k.n_heads = p->n_heads; k.n_kv_heads = p->n_kv_heads;
    k.head_dim = p->head_dim;
    k.partials = kl_partials;
    JAB_RUN(JAB_KT_KL, st, "KL attention-map term", jab::launch_attn_kl(p->dtype, k, st));
    JAB_RUN(JAB_KT_REDUCE, st, "reduce",
            jab::launch_reduce_seq(W.partials, 2, p->batch, per_seq, W.seq_sums, st));
    const double inv_n = 1.0 / ((double)D.M * (double)(D.Hq * D.dh));
    JAB_RUN(JAB_KT_REDUCE, st, "reduce",
            jab::launch_reduce_final(W.seq_sums, 1, p->batch, inv_n, out, 0, 1, 1, st));
    JAB_RUN(JAB_KT_REDUCE, st, "reduce",
            jab::launch_reduce_final(W.seq_sums + (size_t)D.B * 2, 1, p->batch, 1.0 / (double)D.B,
                                     out + 3 + D.B, 0, 1, 1, st));
    return JAB_OK;
}

jab_status jab_curvature(const jab_problem *p, const void *x, const void *w, float lambda_kl, int32_t n_probes,
                         const int8_t *probes, double *out, void *ws, size_t ws_bytes, void *stream) {
    jab_status s = check_problem(p);
    if (s) return s;
    JAB_CHECK(x && aligned(x, 16) && w && aligned(w, 16), JAB_E_INVALID, "x / w NULL or not 16-byte aligned");
    JAB_CHECK(std::isfinite(lambda_kl) && lambda_kl >= 0.f, JAB_E_INVALID, "lambda_kl must be finite and >= 0");
    JAB_CHECK(n_probes >= 1 && probes, JAB_E_INVALID, "need at least one probe");
    JAB_CHECK(out && aligned(out, 8), JAB_E_INVALID, "out NULL or not 8-byte aligned");
    JAB_CHECK(ws && aligned(ws, 256), JAB_E_INVALID, "workspace is NULL or not 256-byte aligned");
    size_t need = 0;
    const CurvWs W = carve_curv(*p, ws, &need);
    JAB_CHECK(ws_bytes >= need, JAB_E_WORKSPACE, "workspace too small for jab_curvature");
    const Dims D = dims_of(*p);
    const int64_t n = D.R * D.d;
    hipStream_t st = static_cast<hipStream_t>(stream);
    // the projection at the float point once; per probe its tangent X v^T (the projection of the
    // probe itself: the projection is linear), then one forward-mode pass through the attention
    if ((s = run_project_split(*p, x, w, W.base, st))) return s;
    jab::JvpArgs a;
    std::memset(&a, 0, sizeof(a));
    const size_t koff = (size_t)(D.Hq * D.dh) * esize(p->dtype);
    a.q = W.base.qk;
    a.k = static_cast<const char *>(W.base.qk) + koff;
    a.vt = W.base.vt;
    a.qd = W.tan.qk;
    a.kd = static_cast<const char *>(W.tan.qk) + koff;
    a.vdt = W.tan.vt;
    a.ld = (int)((D.Hq + D.Hkv) * D.dh);
    a.ldv = vt_ld(*p);
    a.batch = p->batch; a.seq_len = p->seq_len; a.n_heads = p->n_heads; a.n_kv_heads = p->n_kv_heads;
    a.head_dim = p->head_dim;
    a.partials = W.partials;
    for (int pr = 0; pr < n_probes; ++pr) {
        JAB_RUN(JAB_KT_QUANT, st, "probe operand",
                jab::launch_probe_to_dtype(p->dtype, probes + (size_t)pr * n, n, W.w_op, st));
        if ((s = run_project_split(*p, x, W.w_op, W.tan, st))) return s;
        int64_t n_part = 0;
        JAB_RUN(JAB_KT_ATTN, st, "attention tangent", jab::launch_attn_jvp(p->dtype, a, st, &n_part));
        JAB_RUN(JAB_KT_REDUCE, st, "curvature forms",
                jab::launch_curv_forms(W.partials, n_part, W.parts, (double)lambda_kl, out + 7 * (size_t)pr, st));
    }
    return JAB_OK;
}

jab_status jab_loss_bwd_kl(const jab_problem *p, const void *x, const void *w, const jab_quant *q,
                           const float *a_ref, const void *qk_ref, const float *lse_ref, const float *lsq_gscale,
                           float lambda_kl, double *out, float *dw, float *dscale, void *ws, size_t ws_bytes,
                           void *stream) {
    jab_status s = check_problem(p);
    if (s) return s;
    if ((s = check_quant(*p, q))) return s;
    JAB_CHECK(x && aligned(x, 16) && w && aligned(w, 16), JAB_E_INVALID, "x / w NULL or not 16-byte aligned");
    JAB_CHECK(a_ref && aligned(a_ref, 16), JAB_E_INVALID, "a_ref NULL or not 16-byte aligned");
    JAB_CHECK(qk_ref && aligned(qk_ref, 16), JAB_E_INVALID, "qk_ref NULL or not 16-byte aligned");
    JAB_CHECK(lse_ref && aligned(lse_ref, 4), JAB_E_INVALID, "lse_ref NULL or not 4-byte aligned");
    JAB_CHECK(std::isfinite(lambda_kl) && lambda_kl >= 0.f, JAB_E_INVALID, "lambda_kl must be finite and >= 0");
    JAB_CHECK(lsq_gscale, JAB_E_INVALID, "lsq_gscale is NULL");
    JAB_CHECK(out && aligned(out, 8), JAB_E_INVALID, "out NULL or not 8-byte aligned");
    JAB_CHECK(dw && aligned(dw, 16), JAB_E_INVALID, "dw NULL or not 16-byte aligned");
    JAB_CHECK(dscale && aligned(dscale, 4), JAB_E_INVALID, "dscale NULL or misaligned");
    JAB_CHECK(ws && aligned(ws, 256), JAB_E_INVALID, "workspace is NULL or not 256-byte aligned");
    size_t need = 0;
    const BwdWs W = carve_bwd(*p, ws, &need);
    JAB_CHECK(ws_bytes >= need, JAB_E_WORKSPACE, "workspace too small for jab_loss_bwd_kl");
    KlBwd kl{qk_ref, lse_ref, lambda_kl};
    return run_bwd(p, x, w, q, a_ref, lsq_gscale, out, dw, dscale, W, static_cast<hipStream_t>(stream), true, &kl);
}

jab_status jab_fisher(const jab_problem *p, const void *x, const void *w, const jab_quant *q, const float *a_ref,
                      const void *qk_ref, const float *lse_ref, float lambda_kl, double *out, void *ws,
                      size_t ws_bytes, void *stream) {
    jab_status s = check_problem(p);
    if (s) return s;
    if ((s = check_quant(*p, q))) return s;
    JAB_CHECK(x && aligned(x, 16) && w && aligned(w, 16), JAB_E_INVALID, "x / w NULL or not 16-byte aligned");
    JAB_CHECK(a_ref && aligned(a_ref, 16), JAB_E_INVALID, "a_ref NULL or not 16-byte aligned");
    JAB_CHECK(out && aligned(out, 8), JAB_E_INVALID, "out NULL or not 8-byte aligned");
    JAB_CHECK(ws && aligned(ws, 256), JAB_E_INVALID, "workspace is NULL or not 256-byte aligned");
    JAB_CHECK(ws_bytes >= jab_workspace_size(p, JAB_OP_FISHER, 0), JAB_E_WORKSPACE,
              "workspace too small for jab_fisher");
    JAB_CHECK(std::isfinite(lambda_kl) && lambda_kl >= 0.f, JAB_E_INVALID, "lambda_kl must be finite and >= 0");
    JAB_CHECK(lambda_kl == 0.f || (qk_ref && aligned(qk_ref, 16) && lse_ref && aligned(lse_ref, 4)), JAB_E_INVALID,
              "lambda_kl > 0 needs the teacher cache qk_ref / lse_ref");
    size_t bwd_bytes = 0;
    const BwdWs W = carve_bwd(*p, ws, &bwd_bytes);
    Carver c(static_cast<char *>(ws) + bwd_bytes);
    const FisherWs F = carve_fisher(*p, c);
    hipStream_t st = static_cast<hipStream_t>(stream);
    const float gamma[3] = {1.f, 1.f, 1.f};             // the scale gradient is not part of the score
    KlBwd kl{qk_ref, lse_ref, lambda_kl};
    if ((s = run_bwd(p, x, w, q, a_ref, gamma, F.loss, F.dw, F.ds, W, st, true, lambda_kl > 0.f ? &kl : nullptr)))
        return s;
    const Dims D = dims_of(*p);
    jab::UnitRows rows;
    rows.r[0] = 0; rows.r[1] = D.Hq * D.dh; rows.r[2] = (D.Hq + D.Hkv) * D.dh; rows.r[3] = D.R;
    JAB_RUN(JAB_KT_REDUCE, st, "gradient norms", jab::launch_unit_sumsq(F.dw, D.d, rows, 3, F.part, out, st));
    JAB_RUN(JAB_KT_MISC, st, "copy mse",
            hipMemcpyAsync(out + 3, F.loss + 1, sizeof(double), hipMemcpyDeviceToDevice, st));
    return JAB_OK;
}

int32_t jab_ste_stats_len(int32_t n_steps, int32_t eval_every) {
    if (n_steps < 0 || eval_every < 1) return 0;
    return 6 + n_steps + (n_steps + eval_every - 1) / eval_every;
}

jab_status jab_ste_finetune(const jab_problem *p, const jab_ste_config *cfg, const void *x, const float *a_ref,
                            int32_t held_batch, const void *x_held, const float *a_ref_held, const void *qk_ref,
                            const float *lse_ref, const void *qk_ref_held, const float *lse_ref_held, const int32_t *bits,
                            const float *lsq_gscale, float *w_master, void *w, float *scale, const uint8_t *zero,
                            double *stats, void *ws, size_t ws_bytes, void *stream) {
    jab_status s = check_problem(p);
    if (s) return s;
    JAB_CHECK(cfg && bits && lsq_gscale, JAB_E_INVALID, "cfg, bits or lsq_gscale is NULL");
    JAB_CHECK(cfg->n_steps >= 0 && cfg->eval_every >= 1, JAB_E_INVALID, "need n_steps >= 0 and eval_every >= 1");
    JAB_CHECK(std::isfinite(cfg->alpha_w) && std::isfinite(cfg->alpha_s) && cfg->alpha_w >= 0.f && cfg->alpha_s >= 0.f,
              JAB_E_INVALID, "alpha_w and alpha_s must be finite and non-negative");
    JAB_CHECK(cfg->beta1 >= 0.f && cfg->beta1 < 1.f && cfg->beta2 >= 0.f && cfg->beta2 < 1.f && cfg->adam_eps > 0.f &&
                  cfg->scale_floor >= 0.f,
              JAB_E_INVALID, "need 0 <= beta1, beta2 < 1, adam_eps > 0 and scale_floor >= 0");
    JAB_CHECK(held_batch >= 1 && held_batch <= p->batch, JAB_E_INVALID, "held_batch must be 1..batch");
    JAB_CHECK(std::isfinite(cfg->lambda_kl) && cfg->lambda_kl >= 0.f, JAB_E_INVALID,
              "lambda_kl must be finite and >= 0");
    const bool use_kl = cfg->lambda_kl > 0.f;
    JAB_CHECK(!use_kl || (qk_ref && aligned(qk_ref, 16) && lse_ref && aligned(lse_ref, 4) && qk_ref_held &&
                          aligned(qk_ref_held, 16) && lse_ref_held && aligned(lse_ref_held, 4)),
              JAB_E_INVALID, "lambda_kl > 0 needs the teacher caches qk_ref / lse_ref (training and held out)");
    jab_quant q;
    for (int m = 0; m < 3; ++m) q.bits[m] = bits[m];
    q.scale = scale;
    q.zero = zero;
    if ((s = check_quant(*p, &q))) return s;
    JAB_CHECK(x && aligned(x, 16) && x_held && aligned(x_held, 16), JAB_E_INVALID,
              "x / x_held NULL or not 16-byte aligned");
    JAB_CHECK(a_ref && aligned(a_ref, 16) && a_ref_held && aligned(a_ref_held, 16), JAB_E_INVALID,
              "a_ref / a_ref_held NULL or not 16-byte aligned");
    JAB_CHECK(w_master && aligned(w_master, 16) && w && aligned(w, 16), JAB_E_INVALID,
              "w_master / w NULL or not 16-byte aligned");
    JAB_CHECK(stats && aligned(stats, 8), JAB_E_INVALID, "stats NULL or not 8-byte aligned");
    JAB_CHECK(ws && aligned(ws, 256), JAB_E_INVALID, "workspace is NULL or not 256-byte aligned");
    JAB_CHECK(ws_bytes >= jab_workspace_size(p, JAB_OP_STE, 0), JAB_E_WORKSPACE,
              "workspace too small for jab_ste_finetune");
    size_t bwd_bytes = 0;
    const BwdWs W = carve_bwd(*p, ws, &bwd_bytes);
    Carver c(static_cast<char *>(ws) + bwd_bytes);
    const SteWs S = carve_ste(*p, c);
    hipStream_t st = static_cast<hipStream_t>(stream);
    const Dims D = dims_of(*p);
    const int64_t nw = D.R * D.d, groups = D.d / D.g, ns = D.R * groups;
    jab::UnitRows rows;
    rows.r[0] = 0; rows.r[1] = D.Hq * D.dh; rows.r[2] = (D.Hq + D.Hkv) * D.dh; rows.r[3] = D.R;
    const int mask = (bits[0] > 0) | (bits[1] > 0) << 1 | (bits[2] > 0) << 2;
    jab_problem held = *p;
    held.batch = held_batch;
    const int n_steps = cfg->n_steps, log0 = 6 + n_steps;
    const float gamma[3] = {lsq_gscale[0], lsq_gscale[1], lsq_gscale[2]};

    // start: the dtype operand and a copy of it, the mean grid step, zero moments, the held-out
    // loss of the start (the first best checkpoint)
    JAB_RUN(JAB_KT_MISC, st, "round", jab::launch_round_to_dtype(p->dtype, w_master, w, nw, st));
    JAB_RUN(JAB_KT_MISC, st, "round", jab::launch_round_to_dtype(p->dtype, w_master, S.w0, nw, st));
    JAB_RUN(JAB_KT_MISC, st, "mean grid step", jab::launch_mean_scale(scale, groups, rows, mask, S.sbar, st));
    for (float *a : {S.m_w, S.v_w}) JAB_RUN(JAB_KT_MISC, st, "zero", jab::launch_zero_f32(a, nw, st));
    for (float *a : {S.m_s, S.v_s}) JAB_RUN(JAB_KT_MISC, st, "zero", jab::launch_zero_f32(a, ns, st));
    // the held-out score: mse, plus lambda kl / B with the KL term
    auto score_held = [&]() -> jab_status {
        jab_status r = use_kl ? jab_loss_fwd_kl(&held, x_held, w, &q, a_ref_held, qk_ref_held, lse_ref_held,
                                                S.held_out, ws, bwd_bytes, stream)
                              : jab_loss_fwd(&held, x_held, w, &q, a_ref_held, S.held_out, ws, bwd_bytes, stream);
        if (r) return r;
        return launch(JAB_KT_MISC, st, "objective", [&]() {
            return jab::launch_axpy_f64(S.held_out + 1, use_kl ? S.held_out + 4 + held_batch : nullptr,
                                        cfg->lambda_kl, S.score, st);
        });
    };
    if ((s = score_held())) return s;
    JAB_RUN(JAB_KT_MISC, st, "gate", jab::launch_gate(S.score, stats, 0, -1, 1, S.flag, st));
    JAB_RUN(JAB_KT_MISC, st, "checkpoint", jab::launch_copy_if(nullptr, w_master, S.best_w, nw, st));
    JAB_RUN(JAB_KT_MISC, st, "checkpoint", jab::launch_copy_if(nullptr, scale, S.best_s, ns, st));

    int n_eval = 0;
    for (int t = 1; t <= n_steps; ++t) {
        // X^T survives the held-out scoring (its workspace lies below the transposed copy)
        KlBwd klb{qk_ref, lse_ref, cfg->lambda_kl};
        if ((s = run_bwd(p, x, w, &q, a_ref, gamma, S.train_out, S.dw, S.ds, W, st, t == 1, use_kl ? &klb : nullptr)))
            return s;
        JAB_RUN(JAB_KT_MISC, st, "log",
                jab::launch_axpy_f64(S.train_out + 1, use_kl ? S.train_out + 4 + D.B : nullptr, cfg->lambda_kl,
                                     stats + 6 + (t - 1), st));
        // cosine annealing over the run: the first step at the full rate
        const double cosf = 0.5 * (1.0 + std::cos(M_PI * (double)(t - 1) / (double)n_steps));
        jab::AdamStep a;
        a.beta1 = cfg->beta1; a.beta2 = cfg->beta2; a.eps = cfg->adam_eps;
        a.bc1 = (float)(1.0 - std::pow((double)cfg->beta1, t));
        a.bc2 = (float)(1.0 - std::pow((double)cfg->beta2, t));
        a.rate = (float)(cfg->alpha_w * cosf);
        a.floor = 0.f;
        JAB_RUN(JAB_KT_MISC, st, "adam (weights)",
                jab::launch_adam(p->dtype, w_master, S.dw, S.m_w, S.v_w, nw, a, S.sbar, w, st));
        a.rate = (float)(cfg->alpha_s * cosf);
        a.floor = cfg->scale_floor;
        JAB_RUN(JAB_KT_MISC, st, "adam (scales)",
                jab::launch_adam(JAB_F32, scale, S.ds, S.m_s, S.v_s, ns, a, S.sbar, nullptr, st));
        if (t % cfg->eval_every == 0 || t == n_steps) {
            if ((s = score_held())) return s;
            JAB_RUN(JAB_KT_MISC, st, "gate", jab::launch_gate(S.score, stats, t, log0 + n_eval, 0, S.flag, st));
            JAB_RUN(JAB_KT_MISC, st, "checkpoint", jab::launch_copy_if(S.flag, w_master, S.best_w, nw, st));
            JAB_RUN(JAB_KT_MISC, st, "checkpoint", jab::launch_copy_if(S.flag, scale, S.best_s, ns, st));
            ++n_eval;
        }
    }
    // write back the best checkpoint (the start unless an evaluation beat it)
    JAB_RUN(JAB_KT_MISC, st, "restore", jab::launch_copy_if(nullptr, S.best_w, w_master, nw, st));
    JAB_RUN(JAB_KT_MISC, st, "restore", jab::launch_copy_if(nullptr, S.best_s, scale, ns, st));
    JAB_RUN(JAB_KT_MISC, st, "round", jab::launch_round_to_dtype(p->dtype, w_master, w, nw, st));
    // flip rate (eq. flip): codes of the start and of the result, both on the returned grid
    const jab::QuantShape sh = quant_shape(*p, bits);
    JAB_RUN(JAB_KT_QUANT, st, "quantize",
            jab::launch_quantize(sh, p->dtype, S.w0, scale, zero, S.codes0, nullptr, nullptr, nullptr, st));
    JAB_RUN(JAB_KT_QUANT, st, "quantize",
            jab::launch_quantize(sh, p->dtype, w, scale, zero, S.codes1, nullptr, nullptr, nullptr, st));
    JAB_RUN(JAB_KT_REDUCE, st, "flip rate",
            jab::launch_count_diff(S.codes0, S.codes1, D.d, rows, mask, S.part, stats + 3, st));
    return JAB_OK;
}

jab_status jab_loss_sweep(const jab_problem *p, const void *x, const void *w, int32_t n_bits,
                          const int32_t *bits, const float *const *scale_by_bits,
                          const uint8_t *const *zero_by_bits, int32_t n_triples, const int32_t *triples,
                          const float *a_ref, double *loss, double *loss_per_seq, void *ws,
                          size_t ws_bytes, void *stream) {
    jab_status s = check_problem(p);
    if (s) return s;
    JAB_CHECK(n_bits >= 1 && n_bits <= 7 && bits && scale_by_bits, JAB_E_INVALID,
              "need 1..7 candidate bit-widths with scales");
    for (int i = 0; i < n_bits; ++i) {
        JAB_CHECK(bits[i] >= 2 && bits[i] <= 8, JAB_E_INVALID, "candidate bit-widths must be 2..8");
        for (int j = 0; j < i; ++j) JAB_CHECK(bits[i] != bits[j], JAB_E_INVALID, "candidate bit-widths must be distinct");
        JAB_CHECK(scale_by_bits[i] && aligned(scale_by_bits[i], 4), JAB_E_INVALID, "scale pointer NULL or misaligned");
        if (p->scheme == JAB_ASYM)
            JAB_CHECK(zero_by_bits && zero_by_bits[i], JAB_E_INVALID, "zero-points are required for JAB_ASYM");
        else
            JAB_CHECK(!zero_by_bits || !zero_by_bits[i], JAB_E_INVALID, "zero-points must be NULL for JAB_SYM");
    }
    JAB_CHECK(n_triples >= 1 && n_triples <= n_bits * n_bits * n_bits && triples, JAB_E_INVALID,
              "n_triples must be 1..n_bits^3");
    std::vector<int> tidx(3 * (size_t)n_triples);
    for (int t = 0; t < n_triples; ++t)
        for (int m = 0; m < 3; ++m) {
            int found = -1;
            for (int i = 0; i < n_bits; ++i)
                if (bits[i] == triples[3 * t + m]) found = i;
            JAB_CHECK(found >= 0, JAB_E_INVALID, "a triple uses a bit-width outside the candidate set");
            tidx[3 * t + m] = found;
        }
    JAB_CHECK(x && aligned(x, 16) && w && aligned(w, 16), JAB_E_INVALID, "x / w NULL or not 16-byte aligned");
    JAB_CHECK(a_ref && aligned(a_ref, 16), JAB_E_INVALID, "a_ref NULL or not 16-byte aligned");
    JAB_CHECK(loss && aligned(loss, 8), JAB_E_INVALID, "loss NULL or not 8-byte aligned");
    JAB_CHECK(!loss_per_seq || aligned(loss_per_seq, 8), JAB_E_INVALID, "loss_per_seq not 8-byte aligned");
    JAB_CHECK(ws && aligned(ws, 256), JAB_E_INVALID, "workspace is NULL or not 256-byte aligned");
    size_t need = 0;
    const FwdWs W = carve_fwd(*p, ws, &need, n_bits * n_bits * n_bits, n_bits);
    JAB_CHECK(ws_bytes >= need, JAB_E_WORKSPACE, "workspace too small for jab_loss_sweep");

    const Dims D = dims_of(*p);
    const int per_seq = per_seq_waves(*p);
    const size_t pstride = (size_t)D.B * per_seq * 2;
    hipStream_t st = static_cast<hipStream_t>(stream);
    // 1. one projection per candidate bit-width (each matrix at that width)
    for (int i = 0; i < n_bits; ++i) {
        const int b3[3] = {bits[i], bits[i], bits[i]};
        const jab::QuantShape sh = quant_shape(*p, b3);
        const uint8_t *z = zero_by_bits ? zero_by_bits[i] : nullptr;
        JAB_RUN(JAB_KT_QUANT, st, "quantize",
                jab::launch_quantize(sh, p->dtype, w, scale_by_bits[i], z, nullptr, nullptr, W.w_op, nullptr, st));
        if ((s = run_project_split(*p, x, W.w_op, W.proj[i], st))) return s;
    }
    // 2. one score matrix per (b_Q, b_K), applied to the value tensors of up to two triples
    std::vector<bool> done(n_triples, false);
    for (int t = 0; t < n_triples; ++t) {
        if (done[t]) continue;
        std::vector<int> group;
        for (int u = t; u < n_triples; ++u)
            if (!done[u] && tidx[3 * u] == tidx[3 * t] && tidx[3 * u + 1] == tidx[3 * t + 1]) group.push_back(u);
        for (size_t g0 = 0; g0 < group.size(); g0 += (size_t)jab::attn_max_nv(p->dtype)) {
            const int nv = (int)std::min(group.size() - g0, (size_t)jab::attn_max_nv(p->dtype));
            jab::AttnArgs a = attn_args(*p, W.proj[tidx[3 * t]], W.proj[tidx[3 * t + 1]], W.proj[0]);
            a.nv = nv;
            for (int v = 0; v < nv; ++v) {
                const int u = group[g0 + v];
                a.v[v] = W.proj[tidx[3 * u + 2]].vt;
                a.partials[v] = W.partials + (size_t)u * pstride;
                done[u] = true;
            }
            a.mode = jab::ATT_LOSS;
            a.a_ref = a_ref;
            JAB_RUN(JAB_KT_ATTN, st, "attention", jab::launch_attn_fwd(p->dtype, a, st));
        }
    }
    // 3. deterministic reductions
    JAB_RUN(JAB_KT_REDUCE, st, "reduce",
            jab::launch_reduce_seq(W.partials, n_triples, p->batch, per_seq, W.seq_sums, st));
    JAB_RUN(JAB_KT_REDUCE, st, "reduce",
            jab::launch_reduce_sweep(W.seq_sums, n_triples, p->batch, loss, loss_per_seq, st));
    return JAB_OK;
}

jab_status jab_loss_bwd(const jab_problem *p, const void *x, const void *w, const jab_quant *q,
                        const float *a_ref, const float *lsq_gscale, double *out, float *dw,
                        float *dscale, void *ws, size_t ws_bytes, void *stream) {
    jab_status s = check_problem(p);
    if (s) return s;
    if ((s = check_quant(*p, q))) return s;
    JAB_CHECK(x && aligned(x, 16) && w && aligned(w, 16), JAB_E_INVALID, "x / w NULL or not 16-byte aligned");
    JAB_CHECK(a_ref && aligned(a_ref, 16), JAB_E_INVALID, "a_ref NULL or not 16-byte aligned");
    JAB_CHECK(lsq_gscale, JAB_E_INVALID, "lsq_gscale is NULL");
    JAB_CHECK(out && aligned(out, 8), JAB_E_INVALID, "out NULL or not 8-byte aligned");
    JAB_CHECK(dw && aligned(dw, 16), JAB_E_INVALID, "dw NULL or not 16-byte aligned");
    JAB_CHECK(dscale && aligned(dscale, 4), JAB_E_INVALID, "dscale NULL or misaligned");
    JAB_CHECK(ws && aligned(ws, 256), JAB_E_INVALID, "workspace is NULL or not 256-byte aligned");
    size_t need = 0;
    const BwdWs W = carve_bwd(*p, ws, &need);
    JAB_CHECK(ws_bytes >= need, JAB_E_WORKSPACE, "workspace too small for jab_loss_bwd");
    return run_bwd(p, x, w, q, a_ref, lsq_gscale, out, dw, dscale, W, static_cast<hipStream_t>(stream));
}

}  // extern "C"

namespace {
// the loss and its straight-through / LSQ gradients (arguments already validated)
jab_status run_bwd(const jab_problem *p, const void *x, const void *w, const jab_quant *q, const float *a_ref,
                   const float *lsq_gscale, double *out, float *dw, float *dscale, const BwdWs &W, hipStream_t st,
                   bool transpose_x, const KlBwd *kl) {
    jab_status s = JAB_OK;
    const Dims D = dims_of(*p);
    const int64_t Mp = jab::transpose_ld(D.M);          // the contraction length of the weight gradient
    const int64_t Ms = jab::transpose_stride(D.M);      // the row stride of dY^T and X^T
    const jab::QuantShape sh = quant_shape(*p, q->bits);
    // forward: projection, attention storing the log-sum-exp and the backward seed (g, D), loss
    JAB_RUN(JAB_KT_QUANT, st, "quantize",
            jab::launch_quantize(sh, p->dtype, w, q->scale, q->zero, nullptr, nullptr, W.f.w_op, nullptr, st));
    if ((s = run_project_split(*p, x, W.f.w_op, W.f.proj[0], st))) return s;
    jab::AttnArgs a = attn_args(*p, W.f.proj[0], W.f.proj[0], W.f.proj[0]);
    a.mode = jab::ATT_LOSS | jab::ATT_STORE_G | jab::ATT_STORE_LSE;
    a.a_ref = a_ref;
    a.g_out = W.g;
    a.d_out = W.D;
    a.lse2 = W.lse2;
    a.partials[0] = W.f.partials;
    JAB_RUN(JAB_KT_ATTN, st, "attention", jab::launch_attn_fwd(p->dtype, a, st));
    const int per_seq = per_seq_waves(*p);
    if (kl) {   // the KL term's value, as jab_loss_fwd_kl reports it
        jab::KlArgs k;
        std::memset(&k, 0, sizeof(k));
        k.qs = W.f.proj[0].qk;
        k.qt = kl->qk_ref;
        k.ld = (int)((D.Hq + D.Hkv) * D.dh);
        k.lse_t = kl->lse_ref;
        k.batch = p->batch; k.seq_len = p->seq_len; k.n_heads = p->n_heads; k.n_kv_heads = p->n_kv_heads;
        k.head_dim = p->head_dim;
        k.partials = W.f.partials + (size_t)D.B * per_seq * 2;
        JAB_RUN(JAB_KT_KL, st, "KL attention-map term", jab::launch_attn_kl(p->dtype, k, st));
    }
    JAB_RUN(JAB_KT_REDUCE, st, "reduce",
            jab::launch_reduce_seq(W.f.partials, kl ? 2 : 1, p->batch, per_seq, W.f.seq_sums, st));
    const double n_out = (double)D.M * (double)(D.Hq * D.dh);
    JAB_RUN(JAB_KT_REDUCE, st, "reduce",
            jab::launch_reduce_final(W.f.seq_sums, 1, p->batch, 1.0 / n_out, out, 0, 1, 1, st));
    if (kl)
        JAB_RUN(JAB_KT_REDUCE, st, "reduce",
                jab::launch_reduce_final(W.f.seq_sums + (size_t)D.B * 2, 1, p->batch, 1.0 / (double)D.B,
                                         out + 3 + D.B, 0, 1, 1, st));
    // backward through attention (recomputed from the log-sum-exp) into dY^T
    JAB_RUN(JAB_KT_MISC, st, "zero padding",
            jab::launch_zero_cols(p->dtype, W.dyt, (int)D.R, (int)Ms, (int)D.M, st));
    jab::AttnBwdArgs ba;
    std::memset(&ba, 0, sizeof(ba));
    JAB_RUN(JAB_KT_MISC, st, "values to row-major",
            jab::launch_vt_to_v(p->dtype, W.f.proj[0].vt, W.vrow, (int)(D.Hkv * D.dh), vt_ld(*p), p->batch,
                                p->seq_len, (int)(D.Hkv * D.dh), st));
    ba.q = W.f.proj[0].qk;
    ba.k = static_cast<const char *>(W.f.proj[0].qk) + (size_t)(D.Hq * D.dh) * esize(p->dtype);
    ba.v = W.vrow;
    ba.ldq = (int)((D.Hq + D.Hkv) * D.dh);
    ba.ldv = (int)(D.Hkv * D.dh);
    ba.g = W.g; ba.lse2 = W.lse2; ba.D = W.D; ba.dyt = W.dyt; ba.ldt = Ms;
    ba.batch = p->batch; ba.seq_len = p->seq_len; ba.n_heads = p->n_heads; ba.n_kv_heads = p->n_kv_heads;
    ba.head_dim = p->head_dim;
    ba.grad_scale = 1.f;
    ba.ds = W.ds;
    if (kl) {
        // d(lambda KL / B) / d s_ij = (lambda / B) (Q_ij - P_ij) / sqrt(d_head) on the raw scores; dS is
        // kept unscaled by the 2 / N the weight-gradient GEMM applies, so the term enters as
        // (N / 2) (lambda / B) (Q - P)
        ba.qt = kl->qk_ref;
        ba.kt = static_cast<const char *>(kl->qk_ref) + (size_t)(D.Hq * D.dh) * esize(p->dtype);
        ba.lse_t = kl->lse_ref;
        ba.kl_scale = (float)(0.5 * n_out * (double)kl->lambda / (double)D.B);
        // fp16 ends at 65504 and kl_scale grows with seq_len * n_heads * head_dim: scale dS by a power
        // of two that brings the KL part of each dS entry (at most kl_scale) down to 64 or below; the
        // scale-gradient kernel divides it out of the W_Q and W_K rows of the weight gradient (exact:
        // powers of two)
        if (p->dtype == JAB_F16 && ba.kl_scale > 64.f) {
            int e = 0;
            (void)std::frexp((double)ba.kl_scale / 64.0, &e);      // kl_scale / 64 < 2^e
            ba.grad_scale = (float)std::ldexp(1.0, -e);
        }
    }
    JAB_RUN(JAB_KT_ATTN_BWD, st, "attention backward", jab::launch_attn_bwd(p->dtype, ba, st));
    // dW_hat = (2/N) dY^T X, contracted over tokens; dW = dW_hat (straight-through)
    if (p->rope_theta > 0.f) {   // through the rotation: its transpose on the rows of dQ and dK
        const float2 *tab =
            reinterpret_cast<const float2 *>(static_cast<const char *>(W.f.proj[0].qk) + qk_main_bytes(*p));
        JAB_RUN(JAB_KT_MISC, st, "rotary embedding (transpose)",
                jab::launch_rope_cols(p->dtype, W.dyt, Ms, Mp, p->seq_len, p->n_heads + p->n_kv_heads, p->head_dim,
                                      tab, true, st));
    }
    if (transpose_x)   // X^T stays in the workspace: a caller looping over one X transposes it once
        JAB_RUN(JAB_KT_MISC, st, "transpose", jab::launch_transpose(p->dtype, x, W.xt, (int)D.M, (int)D.d, Ms, st));
    int ksplit = 1;
    JAB_RUN(JAB_KT_DW_GEMM, st, "weight-gradient GEMM",
            jab::launch_gemm_nt_f32out(p->dtype, W.dyt, W.xt, dw, (int)D.R, (int)D.d, (int)Mp, (int)Ms,
                                       (int)Ms, (int)D.d, (float)(2.0 / n_out), st, W.dw2, &ksplit));
    // LSQ scale gradient (and the sum of the two halves of a split product)
    const float gamma[3] = {lsq_gscale[0], lsq_gscale[1], lsq_gscale[2]};
    JAB_RUN(JAB_KT_MISC, st, "scale gradient",
            jab::launch_lsq_scale_grad(sh, p->dtype, w, q->scale, q->zero, dw, ksplit == 2 ? W.dw2 : nullptr,
                                       1.f / ba.grad_scale, gamma, dscale, st));
    return JAB_OK;
}
}  // namespace

extern "C" {

jab_status jab_set_bwd_ds_limit(size_t max_bytes) {
    g_ds_limit = max_bytes;
    return JAB_OK;
}

jab_status jab_timing_enable(int32_t on) {
    g_timing.on = on != 0;
    return JAB_OK;
}

jab_status jab_timing_read(double *ms, int64_t *launches) {
    for (const TimedLaunch &t : g_timing.pending) {
        float v = 0.f;
        if (hipEventSynchronize(t.b) != hipSuccess || hipEventElapsedTime(&v, t.a, t.b) != hipSuccess)
            return fail(JAB_E_HIP, "event timing failed");
        g_timing.ms[t.kind] += v;
        g_timing.n[t.kind] += 1;
        g_timing.pool.push_back(t.a);
        g_timing.pool.push_back(t.b);
    }
    g_timing.pending.clear();
    for (int k = 0; k < JAB_KT_COUNT; ++k) {
        if (ms) ms[k] = g_timing.ms[k];
        if (launches) launches[k] = g_timing.n[k];
        g_timing.ms[k] = 0;
        g_timing.n[k] = 0;
    }
    return JAB_OK;
}

}  // extern "C"

// =================================================================== allocation-free forward loss
// jab_loss_fwd with its workspace in a file-scope device array instead of a caller's buffer, for
// callers that cannot allocate.  Each device holds its own copy of the array (placed there when the
// library's code object is loaded on that device); its device address is looked up once per device
// with hipGetSymbolAddress and only that address is handed to the kernels.  The forward loss
// writes every byte of its workspace that it reads (or reads bytes whose values cannot reach a
// result: key rows past a sequence, which the causal mask removes), so the array needs no clearing
// between calls.
namespace {
constexpr size_t kNoallocBytes = (size_t)JAB_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kNoallocBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// the current device's copy of `scratch` (looked up on the first call on that device)
jab_status noalloc_scratch(void **out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(JAB_E_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
    JAB_CHECK(dev >= 0 && dev < kMaxDevices, JAB_E_UNSUPPORTED, "device index beyond the scratch table");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[dev] == nullptr) {
        void *ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return fail(JAB_E_HIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
        JAB_CHECK(ptr != nullptr && aligned(ptr, 256), JAB_E_HIP, "scratch array has no aligned device address");
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return JAB_OK;
}
}  // namespace

extern "C" jab_status jab_loss_fwd_noalloc(const jab_problem *p, const void *x, const void *w, const jab_quant *q,
                                           const float *a_ref, double *out, void *stream) {
    jab_status s = check_problem(p);
    if (s) return s;
    if ((s = check_quant(*p, q))) return s;
    JAB_CHECK(x && aligned(x, 16) && w && aligned(w, 16), JAB_E_INVALID, "x / w NULL or not 16-byte aligned");
    JAB_CHECK(a_ref && aligned(a_ref, 16), JAB_E_INVALID, "a_ref NULL or not 16-byte aligned");
    JAB_CHECK(out && aligned(out, 8), JAB_E_INVALID, "out NULL or not 8-byte aligned");
    const size_t need = jab_workspace_size(p, JAB_OP_FWD, 0);
    JAB_CHECK(need > 0 && need <= kNoallocBytes, JAB_E_WORKSPACE,
              "problem needs " + std::to_string(need) + " bytes of scratch; jab_loss_fwd_noalloc holds " +
                  std::to_string(kNoallocBytes) + " (use jab_loss_fwd with a caller workspace)");
    void *ws = nullptr;
    if ((s = noalloc_scratch(&ws))) return s;
    const jab::GemmQueueNoAlloc no_queue_alloc;       // the GEMMs allocate no tile queue either
    return jab_loss_fwd(p, x, w, q, a_ref, out, ws, kNoallocBytes, stream);
}
