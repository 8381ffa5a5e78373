/*
 * jab_oracle.c -- plain fp64 CPU oracle for the JAB joint attention-block loss.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the tests, the smoke check and the benchmark's CPU
 * baseline leg do.  It shares no code, header, table or constant with the GPU
 * path.
 *
 * Every routine is the plain definition of one step of the method, written as
 * straight loops in double precision with no blocking, fusion or reordering:
 *
 *   - rounding to a storage format           (the precision contract)
 *   - quantizer scale / zero-point and codes  (Method, eq. quant; Appendix
 *                                              "Joint STE fine-tuning", (1))
 *   - QKV projection  y = x W^T               (Method, "Layer-wise PTQ")
 *   - causal softmax attention                (Method, "Layer-wise PTQ":
 *                                              A(X) = softmax(QK^T/sqrt(d_head)+M)V)
 *   - KL divergence of two attention maps      (Method, eq. joint_loss: D_KL(P || Q))
 *   - directional derivatives of attention     (Method, eq. gn: J_A v and J_Q v)
 *   - the attention backward                  (chain rule of the same formula)
 *   - the LSQ factor of the scale gradient    (eq. lsq)
 *   - dW_hat = dY^T X                         (chain rule of the projection)
 *
 * OpenMP splits only independent outer loops (rows, heads, output columns);
 * every sum runs in its natural index order, so results do not depend on the
 * thread count.
 *
 * Layouts (all row-major, double unless stated):
 *   x    [T][d]            one sequence of calibration activations
 *   w    [R][d]            fused weight, row = output channel (Q rows, K rows, V rows)
 *   y    [T][R]            projection; Q = y[:, 0:Hq*dh], K and V follow
 *   a    [T][Hq*dh]        merged attention output, head h in columns h*dh..h*dh+dh-1
 *   s, z [R][d/g]          per-(output row, group) scale and zero-point
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------- */
/* Rounding to a binary floating-point storage format, ties to even.          */
/* fmt: 0 = leave in float64, 1 = fp32, 2 = fp16, 3 = bf16.                   */
/* A format is (p significant bits, minimum normal exponent, largest finite).  */
/* ------------------------------------------------------------------------- */
static double round_to_format(double x, int fmt)
{
    int p, emin;
    double maxf;
    if (fmt == 0 || x == 0.0 || isnan(x) || isinf(x))
        return x;
    if (fmt == 1) {        /* IEEE binary32 */
        p = 24; emin = -126; maxf = ldexp(2.0 - ldexp(1.0, -23), 127);
    } else if (fmt == 2) { /* IEEE binary16 */
        p = 11; emin = -14;  maxf = 65504.0;
    } else {               /* bfloat16: binary32 exponent, 8 significant bits */
        p = 8;  emin = -126; maxf = ldexp(2.0 - ldexp(1.0, -7), 127);
    }
    int e2;
    frexp(x, &e2);                   /* |x| = m 2^e2, 0.5 <= m < 1 */
    int e = e2 - 1;                  /* 2^e <= |x| < 2^(e+1) */
    if (e < emin)
        e = emin;                    /* subnormal range: fixed quantum */
    double quantum = ldexp(1.0, e - (p - 1));
    double r = nearbyint(x / quantum) * quantum;   /* default mode: ties to even */
    if (fabs(r) > maxf)
        r = x > 0 ? INFINITY : -INFINITY;
    return r;
}

int orc_round(double *x, int64_t n, int fmt)
{
    if (fmt < 0 || fmt > 3)
        return -1;
    for (int64_t i = 0; i < n; ++i)
        x[i] = round_to_format(x[i], fmt);
    return 0;
}

static double rn32(double x) { return round_to_format(x, 1); }

/* ------------------------------------------------------------------------- */
/* Quantizer (eq. quant).                                                     */
/* scheme 0 = asymmetric (scale + integer zero-point, codes 0..2^b-1),        */
/*            min-max over the group with 0 included in the range;           */
/* scheme 1 = symmetric as printed: codes -q_max..q_max, q_max = 2^(b-1)-1,   */
/*            scale = max|w| / q_max.                                          */
/* Each fp32 quantity is rounded to fp32 after each operation, as an fp32     */
/* implementation of the quantizer computes it.                               */
/* ------------------------------------------------------------------------- */
int orc_quant_params(const double *w, int rows, int cols, int group, int bits, int scheme,
                     double *s, int32_t *z)
{
    if (group <= 0 || cols % group != 0 || bits < 2 || bits > 8 || (scheme != 0 && scheme != 1))
        return -1;
    const int ng = cols / group;
    const double levels = (double)((1 << bits) - 1);
    const double qmax = (double)((1 << (bits - 1)) - 1);
#pragma omp parallel for schedule(static)
    for (int r = 0; r < rows; ++r) {
        for (int j = 0; j < ng; ++j) {
            const double *g = w + (int64_t)r * cols + (int64_t)j * group;
            double sc, zp = 0.0;
            if (scheme == 0) {
                double lo = 0.0, hi = 0.0;
                for (int k = 0; k < group; ++k) {
                    if (g[k] < lo) lo = g[k];
                    if (g[k] > hi) hi = g[k];
                }
                sc = rn32(rn32(hi - lo) / levels);
                if (sc == 0.0)
                    sc = 1.0;
                zp = nearbyint(rn32(-lo / sc));
                if (zp < 0.0) zp = 0.0;
                if (zp > levels) zp = levels;
            } else {
                double amax = 0.0;
                for (int k = 0; k < group; ++k)
                    if (fabs(g[k]) > amax) amax = fabs(g[k]);
                sc = rn32(amax / qmax);
                if (sc == 0.0)
                    sc = 1.0;
            }
            s[(int64_t)r * ng + j] = sc;
            if (z)
                z[(int64_t)r * ng + j] = (int32_t)zp;
        }
    }
    return 0;
}

/*
 * Codes, fake-quantized weights and the LSQ factor of eq. lsq.
 *   v = w/s (fp32 quotient), u = round(v) ties to even;
 *   asymmetric: q = clip(u + z, 0, 2^b-1), w_hat = (q - z) s,
 *               phi = u - v      if -z <= v <= 2^b-1-z,
 *                     -z         if v < -z,
 *                     2^b-1-z    if v > 2^b-1-z;
 *   symmetric:  q = clip(u, -q_max, q_max), w_hat = q s, code = q + q_max,
 *               phi = q - v if |v| <= q_max, else sign(v) q_max.
 * w_hat is exact in double: an integer of at most 9 bits times an fp32 scale.
 * bits == 0 means "not quantized": w_hat = w, code 0, phi 0.
 * Any of codes / w_hat / phi may be NULL.
 */
int orc_fake_quant(const double *w, int rows, int cols, int group, int bits, int scheme,
                   const double *s, const int32_t *z, int32_t *codes, double *w_hat, double *phi)
{
    if (group <= 0 || cols % group != 0 || (bits != 0 && (bits < 2 || bits > 8)))
        return -1;
    const int ng = cols / group;
#pragma omp parallel for schedule(static)
    for (int r = 0; r < rows; ++r) {
        for (int k = 0; k < cols; ++k) {
            const int64_t i = (int64_t)r * cols + k;
            if (bits == 0) {
                if (codes) codes[i] = 0;
                if (w_hat) w_hat[i] = w[i];
                if (phi) phi[i] = 0.0;
                continue;
            }
            const int64_t gi = (int64_t)r * ng + k / group;
            const double sc = s[gi];
            const double v = rn32(w[i] / sc);
            const double u = nearbyint(v);
            double q, wh, ph;
            if (scheme == 0) {
                const double levels = (double)((1 << bits) - 1);
                const double zp = (double)z[gi];
                q = u + zp;
                if (q < 0.0) q = 0.0;
                if (q > levels) q = levels;
                wh = (q - zp) * sc;
                if (v < -zp)
                    ph = -zp;
                else if (v > levels - zp)
                    ph = levels - zp;
                else
                    ph = u - v;
                if (codes) codes[i] = (int32_t)q;
            } else {
                const double qmax = (double)((1 << (bits - 1)) - 1);
                q = u;
                if (q < -qmax) q = -qmax;
                if (q > qmax) q = qmax;
                wh = q * sc;
                if (fabs(v) <= qmax)
                    ph = q - v;
                else
                    ph = v > 0 ? qmax : -qmax;
                if (codes) codes[i] = (int32_t)(q + qmax);
            }
            if (w_hat) w_hat[i] = wh;
            if (phi) phi[i] = ph;
        }
    }
    return 0;
}

/* ------------------------------------------------------------------------- */
/* Projection y[t][n] = sum_k x[t][k] w[n][k]  (y = xW with W stored [R][d]). */
/* ------------------------------------------------------------------------- */
int orc_project(const double *x, int T, int d, const double *w, int R, double *y)
{
#pragma omp parallel for schedule(static)
    for (int t = 0; t < T; ++t) {
        const double *xr = x + (int64_t)t * d;
        for (int n = 0; n < R; ++n) {
            const double *wr = w + (int64_t)n * d;
            double acc = 0.0;
            for (int k = 0; k < d; ++k)
                acc += xr[k] * wr[k];
            y[(int64_t)t * R + n] = acc;
        }
    }
    return 0;
}

/* ------------------------------------------------------------------------- */
/* Causal grouped-query softmax attention on one sequence.                    */
/* Query head h reads key/value head floor(h * Hkv / Hq).  Query i attends to */
/* keys j <= i.  Softmax is max-subtracted.                                   */
/* a[t][h*dh + c]; lse[h][t] = log sum_j exp(S_ij) (NULL to skip);            */
/* *row_sum_dev = max_i |sum_j P_ij - 1| (NULL to skip).                      */
/* ------------------------------------------------------------------------- */
static int check_heads(int R, int Hq, int Hkv, int dh)
{
    if (Hq <= 0 || Hkv <= 0 || dh <= 0 || Hq % Hkv != 0 || R != (Hq + 2 * Hkv) * dh)
        return -1;
    return 0;
}

int orc_attention(const double *y, int T, int R, int Hq, int Hkv, int dh,
                  double *a, double *lse, double *row_sum_dev)
{
    if (check_heads(R, Hq, Hkv, dh))
        return -1;
    const int koff = Hq * dh, voff = (Hq + Hkv) * dh, ac = Hq * dh;
    const double inv_sqrt = 1.0 / sqrt((double)dh);
    double dev = 0.0;
#pragma omp parallel
    {
        double *p = (double *)malloc(sizeof(double) * (size_t)(T > 0 ? T : 1));
        double mydev = 0.0;
#pragma omp for schedule(dynamic, 4) collapse(2)
        for (int h = 0; h < Hq; ++h) {
            for (int i = 0; i < T; ++i) {
                const int kvh = (int)((int64_t)h * Hkv / Hq);
                const double *q = y + (int64_t)i * R + h * dh;
                double m = -INFINITY;
                for (int j = 0; j <= i; ++j) {
                    const double *k = y + (int64_t)j * R + koff + kvh * dh;
                    double dot = 0.0;
                    for (int c = 0; c < dh; ++c)
                        dot += q[c] * k[c];
                    p[j] = dot * inv_sqrt;
                    if (p[j] > m) m = p[j];
                }
                double l = 0.0;
                for (int j = 0; j <= i; ++j) {
                    p[j] = exp(p[j] - m);
                    l += p[j];
                }
                double psum = 0.0;
                for (int j = 0; j <= i; ++j) {
                    p[j] /= l;
                    psum += p[j];
                }
                if (fabs(psum - 1.0) > mydev) mydev = fabs(psum - 1.0);
                /* out[c] = sum_j p_j V_j[c], j ascending for every c */
                double *out = a + (int64_t)i * ac + h * dh;
                for (int c = 0; c < dh; ++c)
                    out[c] = 0.0;
                for (int j = 0; j <= i; ++j) {
                    const double *v = y + (int64_t)j * R + voff + kvh * dh;
                    for (int c = 0; c < dh; ++c)
                        out[c] += p[j] * v[c];
                }
                if (lse)
                    lse[(int64_t)h * T + i] = m + log(l);
            }
        }
#pragma omp critical
        if (mydev > dev) dev = mydev;
        free(p);
    }
    if (row_sum_dev)
        *row_sum_dev = dev;
    return 0;
}

/* ------------------------------------------------------------------------- */
/* KL divergence of attention maps, eq. joint_loss: D_KL(P || Q) with P the   */
/* causal softmax map of the teacher projection yt and Q that of the student  */
/* projection ys (both [T][R], the layout of orc_attention; only the query    */
/* and key columns are read).  Per head h and query i:                        */
/*   kl[h][i] = sum_{j <= i} P_ij (log P_ij - log Q_ij),                      */
/* log P_ij = St_ij - logsumexp_j St_ij, St = Qt Kt^T / sqrt(dh) (and Q from  */
/* the student's scores alike); a term with P_ij = 0 contributes 0.           */
/* *kl_sum = sum over h, i (h outer, i inner).  kl may be NULL.               */
/* ------------------------------------------------------------------------- */
int orc_attention_kl(const double *yt, const double *ys, int T, int R, int Hq, int Hkv, int dh,
                     double *kl, double *kl_sum)
{
    if (check_heads(R, Hq, Hkv, dh))
        return -1;
    const int koff = Hq * dh;
    const double inv_sqrt = 1.0 / sqrt((double)dh);
    double *rows = (double *)malloc(sizeof(double) * (size_t)(Hq > 0 && T > 0 ? Hq * T : 1));
    if (!rows)
        return -1;
#pragma omp parallel
    {
        double *st = (double *)malloc(sizeof(double) * (size_t)(T > 0 ? T : 1));
        double *ss = (double *)malloc(sizeof(double) * (size_t)(T > 0 ? T : 1));
#pragma omp for schedule(dynamic, 4) collapse(2)
        for (int h = 0; h < Hq; ++h) {
            for (int i = 0; i < T; ++i) {
                const int kvh = (int)((int64_t)h * Hkv / Hq);
                const double *qt = yt + (int64_t)i * R + h * dh;
                const double *qs = ys + (int64_t)i * R + h * dh;
                double mt = -INFINITY, ms = -INFINITY;
                for (int j = 0; j <= i; ++j) {
                    const double *kt = yt + (int64_t)j * R + koff + kvh * dh;
                    const double *ks = ys + (int64_t)j * R + koff + kvh * dh;
                    double dt = 0.0, ds = 0.0;
                    for (int c = 0; c < dh; ++c) {
                        dt += qt[c] * kt[c];
                        ds += qs[c] * ks[c];
                    }
                    st[j] = dt * inv_sqrt;
                    ss[j] = ds * inv_sqrt;
                    if (st[j] > mt) mt = st[j];
                    if (ss[j] > ms) ms = ss[j];
                }
                double lt = 0.0, ls = 0.0;
                for (int j = 0; j <= i; ++j) {
                    lt += exp(st[j] - mt);
                    ls += exp(ss[j] - ms);
                }
                const double lse_t = mt + log(lt), lse_s = ms + log(ls);
                double acc = 0.0;
                for (int j = 0; j <= i; ++j) {
                    const double logp = st[j] - lse_t, logq = ss[j] - lse_s;
                    const double pj = exp(logp);
                    if (pj > 0.0)
                        acc += pj * (logp - logq);
                }
                rows[(int64_t)h * T + i] = acc;
            }
        }
        free(st);
        free(ss);
    }
    double total = 0.0;
    for (int64_t r = 0; r < (int64_t)Hq * T; ++r)
        total += rows[r];
    if (kl)
        memcpy(kl, rows, sizeof(double) * (size_t)Hq * (size_t)T);
    *kl_sum = total;
    free(rows);
    return 0;
}

/* ------------------------------------------------------------------------- */
/* Directional derivatives of causal attention for the Gauss-Newton curvature */
/* of eq. gn, on one sequence.  y [T][R] is the projection at the float point */
/* and yd [T][R] its tangent X v^T for a probe v.  With z = Q K^T / sqrt(dh)  */
/* (masked), P = softmax(z) per row and A = P V, the tangent of the logits    */
/* splits by the weight matrix the probe moves:                               */
/*   zQ_ij = Qd_i . K_j / sqrt(dh)   (W_Q),   zK_ij = Q_i . Kd_j / sqrt(dh)   */
/* and the output tangent is the sum of the three unit parts                  */
/*   aQ_i = sum_j P_ij (zQ_ij - mQ_i) V_j,  mQ_i = sum_j P_ij zQ_ij (aK alike)*/
/*   aV_i = sum_j P_ij Vd_j                                                   */
/* (the derivative of softmax: dP_ij = P_ij (dz_ij - sum_k P_ik dz_ik)).      */
/* The Fisher information of a row's softmax in its logits is                 */
/* I(P) = diag(P) - P P^T, so for two logit tangents a, b:                    */
/*   a^T I(P) b = sum_j P_ij a_j b_j - (sum_j P_ij a_j)(sum_j P_ij b_j).      */
/* out[9] (accumulated over heads h outer, rows i inner):                     */
/*   0 <aQ,aQ>  1 <aK,aK>  2 <aV,aV>  3 <aQ,aK>  4 <aQ,aV>  5 <aK,aV>         */
/*   6 zQ^T I zQ  7 zK^T I zK  8 zQ^T I zK                                    */
/* (<.,.> summed over the head's output columns and every query row).         */
/* ------------------------------------------------------------------------- */
int orc_attention_jvp(const double *y, const double *yd, int T, int R, int Hq, int Hkv, int dh, double *out)
{
    if (check_heads(R, Hq, Hkv, dh))
        return -1;
    const int koff = Hq * dh, voff = (Hq + Hkv) * dh;
    const double inv_sqrt = 1.0 / sqrt((double)dh);
    double *rows = (double *)malloc(sizeof(double) * 9 * (size_t)(Hq > 0 && T > 0 ? Hq * T : 1));
    if (!rows)
        return -1;
#pragma omp parallel
    {
        const size_t n = (size_t)(T > 0 ? T : 1), m = (size_t)(dh > 0 ? dh : 1);
        double *z = (double *)malloc(sizeof(double) * n);
        double *zq = (double *)malloc(sizeof(double) * n);
        double *zk = (double *)malloc(sizeof(double) * n);
        double *aq = (double *)malloc(sizeof(double) * m);
        double *ak = (double *)malloc(sizeof(double) * m);
        double *av = (double *)malloc(sizeof(double) * m);
#pragma omp for schedule(dynamic, 4) collapse(2)
        for (int h = 0; h < Hq; ++h) {
            for (int i = 0; i < T; ++i) {
                const int kvh = (int)((int64_t)h * Hkv / Hq);
                const double *q = y + (int64_t)i * R + h * dh;
                const double *qd = yd + (int64_t)i * R + h * dh;
                double mx = -INFINITY;
                for (int j = 0; j <= i; ++j) {
                    const double *k = y + (int64_t)j * R + koff + kvh * dh;
                    const double *kd = yd + (int64_t)j * R + koff + kvh * dh;
                    double s = 0.0, sq = 0.0, sk = 0.0;
                    for (int c = 0; c < dh; ++c) {
                        s += q[c] * k[c];
                        sq += qd[c] * k[c];
                        sk += q[c] * kd[c];
                    }
                    z[j] = s * inv_sqrt;
                    zq[j] = sq * inv_sqrt;
                    zk[j] = sk * inv_sqrt;
                    if (z[j] > mx) mx = z[j];
                }
                double l = 0.0;
                for (int j = 0; j <= i; ++j) {
                    z[j] = exp(z[j] - mx);      /* z now holds the unnormalised probabilities */
                    l += z[j];
                }
                double mq = 0.0, mk = 0.0, cqq = 0.0, ckk = 0.0, cqk = 0.0;
                for (int j = 0; j <= i; ++j) {
                    const double pj = z[j] / l;
                    z[j] = pj;
                    mq += pj * zq[j];
                    mk += pj * zk[j];
                    cqq += pj * zq[j] * zq[j];
                    ckk += pj * zk[j] * zk[j];
                    cqk += pj * zq[j] * zk[j];
                }
                for (int c = 0; c < dh; ++c) {
                    aq[c] = 0.0;
                    ak[c] = 0.0;
                    av[c] = 0.0;
                }
                for (int j = 0; j <= i; ++j) {
                    const double *v = y + (int64_t)j * R + voff + kvh * dh;
                    const double *vd = yd + (int64_t)j * R + voff + kvh * dh;
                    const double wq = z[j] * (zq[j] - mq), wk = z[j] * (zk[j] - mk);
                    for (int c = 0; c < dh; ++c) {
                        aq[c] += wq * v[c];
                        ak[c] += wk * v[c];
                        av[c] += z[j] * vd[c];
                    }
                }
                double e[6] = {0, 0, 0, 0, 0, 0};
                for (int c = 0; c < dh; ++c) {
                    e[0] += aq[c] * aq[c];
                    e[1] += ak[c] * ak[c];
                    e[2] += av[c] * av[c];
                    e[3] += aq[c] * ak[c];
                    e[4] += aq[c] * av[c];
                    e[5] += ak[c] * av[c];
                }
                double *r = rows + 9 * ((int64_t)h * T + i);
                for (int t = 0; t < 6; ++t)
                    r[t] = e[t];
                r[6] = cqq - mq * mq;
                r[7] = ckk - mk * mk;
                r[8] = cqk - mq * mk;
            }
        }
        free(z); free(zq); free(zk); free(aq); free(ak); free(av);
    }
    for (int t = 0; t < 9; ++t)
        out[t] = 0.0;
    for (int64_t r = 0; r < (int64_t)Hq * T; ++r)
        for (int t = 0; t < 9; ++t)
            out[t] += rows[9 * r + t];
    free(rows);
    return 0;
}

/* ------------------------------------------------------------------------- */
/* Attention backward on one sequence, given g = dLoss/dA [T][Hq*dh].         */
/* With P the causal softmax of S = Q K^T / sqrt(dh):                         */
/*   dV_j  = sum_i P_ij g_i              (summed over the query heads of a    */
/*   dP_ij = g_i . V_j                    key/value group)                    */
/*   dS_ij = P_ij (dP_ij - sum_k P_ik dP_ik)                                  */
/*   dQ_i  = sum_j dS_ij K_j / sqrt(dh)                                       */
/*   dK_j  = sum_i dS_ij Q_i / sqrt(dh)                                       */
/* dy [T][R] receives [dQ | dK | dV] (overwritten).                           */
/* ------------------------------------------------------------------------- */
int orc_attention_bwd(const double *y, int T, int R, int Hq, int Hkv, int dh,
                      const double *g, double *dy)
{
    if (check_heads(R, Hq, Hkv, dh))
        return -1;
    const int koff = Hq * dh, voff = (Hq + Hkv) * dh, ac = Hq * dh;
    const int per = Hq / Hkv;
    const double inv_sqrt = 1.0 / sqrt((double)dh);
    memset(dy, 0, sizeof(double) * (size_t)T * (size_t)R);
    /* One key/value group per task: its query heads write only their own dQ
     * columns and the group's dK / dV columns, so tasks never overlap. */
#pragma omp parallel
    {
        double *P = (double *)malloc(sizeof(double) * (size_t)T * (size_t)T);
        double *dS = (double *)malloc(sizeof(double) * (size_t)T * (size_t)T);
        double *accv = (double *)malloc(sizeof(double) * (size_t)dh);
        double *acck = (double *)malloc(sizeof(double) * (size_t)dh);
#pragma omp for schedule(dynamic, 1)
        for (int kvh = 0; kvh < Hkv; ++kvh) {
            for (int hh = 0; hh < per; ++hh) {
                const int h = kvh * per + hh;
                /* recompute P */
                for (int i = 0; i < T; ++i) {
                    const double *q = y + (int64_t)i * R + h * dh;
                    double m = -INFINITY;
                    for (int j = 0; j <= i; ++j) {
                        const double *k = y + (int64_t)j * R + koff + kvh * dh;
                        double dot = 0.0;
                        for (int c = 0; c < dh; ++c)
                            dot += q[c] * k[c];
                        P[(int64_t)i * T + j] = dot * inv_sqrt;
                        if (P[(int64_t)i * T + j] > m) m = P[(int64_t)i * T + j];
                    }
                    double l = 0.0;
                    for (int j = 0; j <= i; ++j) {
                        P[(int64_t)i * T + j] = exp(P[(int64_t)i * T + j] - m);
                        l += P[(int64_t)i * T + j];
                    }
                    for (int j = 0; j <= i; ++j)
                        P[(int64_t)i * T + j] /= l;
                }
                /* dP, then dS */
                for (int i = 0; i < T; ++i) {
                    const double *gi = g + (int64_t)i * ac + h * dh;
                    double Di = 0.0;
                    for (int j = 0; j <= i; ++j) {
                        const double *vj = y + (int64_t)j * R + voff + kvh * dh;
                        double dp = 0.0;
                        for (int c = 0; c < dh; ++c)
                            dp += gi[c] * vj[c];
                        dS[(int64_t)i * T + j] = dp;
                        Di += P[(int64_t)i * T + j] * dp;
                    }
                    for (int j = 0; j <= i; ++j)
                        dS[(int64_t)i * T + j] = P[(int64_t)i * T + j] * (dS[(int64_t)i * T + j] - Di);
                }
                /* dV and dK (accumulated over the group's query heads);
                 * each sum runs over i = j..T-1 in ascending order */
                for (int j = 0; j < T; ++j) {
                    double *dv = dy + (int64_t)j * R + voff + kvh * dh;
                    double *dk = dy + (int64_t)j * R + koff + kvh * dh;
                    for (int c = 0; c < dh; ++c) {
                        accv[c] = 0.0;
                        acck[c] = 0.0;
                    }
                    for (int i = j; i < T; ++i) {
                        const double pij = P[(int64_t)i * T + j], dsij = dS[(int64_t)i * T + j];
                        const double *gi = g + (int64_t)i * ac + h * dh;
                        const double *qi = y + (int64_t)i * R + h * dh;
                        for (int c = 0; c < dh; ++c) {
                            accv[c] += pij * gi[c];
                            acck[c] += dsij * qi[c];
                        }
                    }
                    for (int c = 0; c < dh; ++c) {
                        dv[c] += accv[c];
                        dk[c] += acck[c] * inv_sqrt;
                    }
                }
                /* dQ: sum over j = 0..i in ascending order */
                for (int i = 0; i < T; ++i) {
                    double *dq = dy + (int64_t)i * R + h * dh;
                    for (int c = 0; c < dh; ++c)
                        accv[c] = 0.0;
                    for (int j = 0; j <= i; ++j) {
                        const double dsij = dS[(int64_t)i * T + j];
                        const double *kj = y + (int64_t)j * R + koff + kvh * dh;
                        for (int c = 0; c < dh; ++c)
                            accv[c] += dsij * kj[c];
                    }
                    for (int c = 0; c < dh; ++c)
                        dq[c] = accv[c] * inv_sqrt;
                }
            }
        }
        free(P);
        free(dS);
        free(accv);
        free(acck);
    }
    return 0;
}

/* ------------------------------------------------------------------------- */
/* dw_hat[n][k] += sum_t dy[t][n] x[t][k]  (chain rule of y = x W^T).         */
/* ------------------------------------------------------------------------- */
int orc_weight_grad(const double *dy, const double *x, int T, int d, int R, double *dw_hat)
{
#pragma omp parallel for schedule(static)
    for (int n = 0; n < R; ++n) {
        for (int k = 0; k < d; ++k) {
            double acc = 0.0;
            for (int t = 0; t < T; ++t)
                acc += dy[(int64_t)t * R + n] * x[(int64_t)t * d + k];
            dw_hat[(int64_t)n * d + k] += acc;
        }
    }
    return 0;
}

/* ------------------------------------------------------------------------- */
/* LSQ scale gradient: ds[r][j] = gamma * sum_{k in group j} dw_hat[r][k] phi[r][k]. */
/* ------------------------------------------------------------------------- */
int orc_scale_grad(const double *dw_hat, const double *phi, int rows, int cols, int group,
                   double gamma, double *ds)
{
    if (group <= 0 || cols % group != 0)
        return -1;
    const int ng = cols / group;
#pragma omp parallel for schedule(static)
    for (int r = 0; r < rows; ++r) {
        for (int j = 0; j < ng; ++j) {
            double acc = 0.0;
            for (int k = j * group; k < (j + 1) * group; ++k)
                acc += dw_hat[(int64_t)r * cols + k] * phi[(int64_t)r * cols + k];
            ds[(int64_t)r * ng + j] = gamma * acc;
        }
    }
    return 0;
}
