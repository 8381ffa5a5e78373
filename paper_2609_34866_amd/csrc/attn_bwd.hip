// attn_bwd.hip -- backward of the squared-error JAB loss through causal GQA
// attention, with the attention matrix recomputed from the forward's
// log-sum-exp; plus the LSQ scale gradient and a transpose helper.
//
// Paper: Method, "Joint fine-tuning through the quantizer" and the Appendix on
// its design decisions, (1) / eq. lsq: straight-through estimator on the weights,
// LSQ rule on the per-(row, group) scales, both applied to the gradient of the
// attention-output loss of eq. joint_loss.
//
// With G = a_hat - a_ref (the factor 2/N of d mse / d a_hat is applied once, in the
// weight-gradient GEMM, so 16-bit operands keep their range), P the causal softmax,
// D_i = sum_c G_ic a_hat_ic:
//   dV_j = sum_i P_ij G_i            (summed over the query heads of a kv group)
//   dP_ij = G_i . V_j,  dS_ij = P_ij (dP_ij - D_i)
//   dQ_i = sum_j dS_ij K_j / sqrt(dh),  dK_j = sum_i dS_ij Q_i / sqrt(dh)
//
// gfx950 design (no atomics, fixed summation order => deterministic):
//  * dK/dV kernel: a wave owns 32 keys of one kv head and keeps K and V for them in
//    registers as matrix-core B operands.  The workgroup walks the query tiles
//    (32 queries, staged row-major and transposed in LDS together with G) of every
//    query head of the group, so the GQA sum over heads stays in the accumulators.
//    S = Q K^T and dP = G V^T come out with one key per lane; P and dS then feed the
//    B operand of dV^T += G^T P and dK^T += Q^T dS directly from registers.
//  * dQ kernel: a wave owns 32 queries (Q and G in registers); 64-key tiles of K
//    (row-major and transposed) and V are staged in LDS; S^T and dP^T come out with
//    one query per lane, so lse and D are per-lane scalars, and dQ^T += K^T dS^T.
//  * Both write their results transposed, dY^T [R][tokens], the operand layout of
//    the weight-gradient GEMM, which contracts over tokens.
#include "device_common.h"
#include "kernels.h"

namespace jab {

// defined in attn_bwd_mfma.hip
template <int DT, int DH>
hipError_t run_bwd_dma(const AttnBwdArgs &a, hipStream_t st);

namespace {

template <int DT>
__device__ inline typename Mma<DT>::operand load_operand(const typename Mma<DT>::elem *p) {
    if constexpr (DT == F32)
        return *p;
    else
        return __builtin_bit_cast(typename Mma<DT>::operand, *reinterpret_cast<const u32x4 *>(p));
}

// B/A operand of a 16-bit MFMA from two 4-element runs (k-slots 0..3 and 4..7).
template <int DT>
__device__ inline typename Mma<DT>::operand load_operand_split(const typename Mma<DT>::elem *p0,
                                                               const typename Mma<DT>::elem *p1) {
    const u16x4 lo = *reinterpret_cast<const u16x4 *>(p0);
    const u16x4 hi = *reinterpret_cast<const u16x4 *>(p1);
    const u16x8 v = u16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return __builtin_bit_cast(typename Mma<DT>::operand, v);
}

template <int DT>
__device__ inline typename Mma<DT>::operand pack_operand(const f32x16 &v, int first) {
    if constexpr (DT == F32) {
        return v[first];
    } else {
        u16x8 b;
#pragma unroll
        for (int i = 0; i < 8; ++i) b[i] = from_f32<DT>(v[first + i]);
        return __builtin_bit_cast(typename Mma<DT>::operand, b);
    }
}

template <int DT, int DH>
struct BwdCfg {
    typedef typename Mma<DT>::elem elem;
    static constexpr int EPC = 16 / (int)sizeof(elem);
    static constexpr int NKC = DH / Mma<DT>::K;
    static constexpr int DHP = DH < 32 ? 32 : DH;
    static constexpr int NDB = DHP / 32;
    static constexpr int RST = DH + EPC;          // row-major tile stride (elements)
    // dK/dV kernel: Q, G row-major [32][RST] and transposed [DHP][QTS], then lse, D
    static constexpr int QTS = 32 + EPC;
    static constexpr size_t DKDV_ELEMS = 2 * 32 * RST + 2 * DHP * QTS;
    static constexpr size_t DKDV_LDS = (DKDV_ELEMS * sizeof(elem) + 15) / 16 * 16 + 2 * 32 * sizeof(float);
    // dQ kernel: K, V row-major [BNK][RST] and K transposed [DHP][KTS]
    static constexpr int BNK = 64;
    static constexpr int KTS = BNK + EPC;
    static constexpr size_t DQ_LDS = (2 * (size_t)BNK * RST + (size_t)DHP * KTS) * sizeof(elem);
};

// ------------------------------------------------------------------ dK / dV
template <int DT, int DH, bool KL>
__global__ __launch_bounds__(256, 1) void attn_bwd_dkdv_kernel(AttnBwdArgs a, float scale_log2,
                                                               float inv_sqrt, int nkb) {
    typedef BwdCfg<DT, DH> C;
    typedef typename C::elem elem;
    typedef Mma<DT> MM;
    constexpr int QTS = C::QTS;                       // transposed tile stride (elements)
    extern __shared__ __align__(16) unsigned char smem[];
    elem *Qs = reinterpret_cast<elem *>(smem);
    elem *Gs = Qs + 32 * C::RST;
    elem *Qt = Gs + 32 * C::RST;
    elem *Gt = Qt + C::DHP * QTS;
    float *lse_s = reinterpret_cast<float *>(smem + (C::DKDV_ELEMS * sizeof(elem) + 15) / 16 * 16);
    float *D_s = lse_s + 32;
    // KL term: the teacher's query tile and log-sum-exp after the regular layout
    elem *Qts = reinterpret_cast<elem *>(smem + C::DKDV_LDS);
    float *lset_s = reinterpret_cast<float *>(smem + C::DKDV_LDS + 32 * C::RST * sizeof(elem));

    const int T = a.seq_len, Hq = a.n_heads, Hkv = a.n_kv_heads;
    const int G = Hq / Hkv;

    const int nwg = gridDim.x;
    int lin = blockIdx.x;
    if ((nwg & 7) == 0) lin = (lin & 7) * (nwg >> 3) + (lin >> 3);
    const int kbi = lin % nkb;                         // ascending key block = heaviest first
    const int kvh = (lin / nkb) % Hkv;
    const int b = lin / (nkb * Hkv);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, half = lane >> 5;
    const int jw = kbi * 128 + wave * 32;              // first key of this wave
    const int key = jw + (lane & 31);
    const int64_t row0 = (int64_t)b * T;
    const elem *Qp = static_cast<const elem *>(a.q);
    const elem *Kp = static_cast<const elem *>(a.k);
    const elem *Vp = static_cast<const elem *>(a.v);
    const elem *Gg = static_cast<const elem *>(a.g);
    const int koff = Hq * DH, voff = (Hq + Hkv) * DH;     // row offsets of dK^T, dV^T in dY^T

    // K and V of this wave's keys as B operands (column = key, k = head dimension)
    typename MM::operand kf[C::NKC], vf[C::NKC], ktf[KL ? C::NKC : 1];
#pragma unroll
    for (int kc = 0; kc < C::NKC; ++kc) {
        const int c = kc * MM::K + half * MM::VEC;
        if (key < T) {
            kf[kc] = load_operand<DT>(Kp + (row0 + key) * a.ldq + kvh * DH + c);
            vf[kc] = load_operand<DT>(Vp + (row0 + key) * a.ldv + kvh * DH + c);
            if constexpr (KL)
                ktf[kc] = load_operand<DT>(static_cast<const elem *>(a.kt) + (row0 + key) * a.ldq + kvh * DH + c);
        } else {
            kf[kc] = pack_operand<DT>(f32x16{}, 0);
            vf[kc] = pack_operand<DT>(f32x16{}, 0);
            if constexpr (KL) ktf[kc] = pack_operand<DT>(f32x16{}, 0);
        }
    }
    f32x16 dvt[C::NDB], dkt[C::NDB];
#pragma unroll
    for (int d = 0; d < C::NDB; ++d)
#pragma unroll
        for (int e = 0; e < 16; ++e) { dvt[d][e] = 0.f; dkt[d][e] = 0.f; }

    if constexpr (DH < 32) {
        for (int i = tid; i < C::DHP * QTS; i += 256) { Qt[i] = from_f32<DT>(0.f); Gt[i] = from_f32<DT>(0.f); }
    }
    const int i_begin = kbi * 128;
    constexpr int CPR = DH / C::EPC;
    for (int hh = 0; hh < G; ++hh) {
        const int h = kvh * G + hh;
        for (int i0 = i_begin; i0 < T; i0 += 32) {
            __syncthreads();
            // ---- stage Q and G of queries i0..i0+31 (row-major and transposed), lse, D
            for (int idx = tid; idx < 32 * CPR; idx += 256) {
                const int r = idx / CPR, c = idx % CPR;
                const int q = i0 + r;
                u32x4 qv = u32x4{0u, 0u, 0u, 0u}, gv = u32x4{0u, 0u, 0u, 0u};
                if (q < T) {
                    qv = *reinterpret_cast<const u32x4 *>(Qp + (row0 + q) * a.ldq + h * DH + c * C::EPC);
                    gv = *reinterpret_cast<const u32x4 *>(Gg + ((row0 + q) * Hq + h) * DH + c * C::EPC);
                }
                *reinterpret_cast<u32x4 *>(Qs + r * C::RST + c * C::EPC) = qv;
                *reinterpret_cast<u32x4 *>(Gs + r * C::RST + c * C::EPC) = gv;
                if constexpr (KL) {
                    u32x4 tv = u32x4{0u, 0u, 0u, 0u};
                    if (q < T)
                        tv = *reinterpret_cast<const u32x4 *>(static_cast<const elem *>(a.qt) + (row0 + q) * a.ldq +
                                                              h * DH + c * C::EPC);
                    *reinterpret_cast<u32x4 *>(Qts + r * C::RST + c * C::EPC) = tv;
                }
                const elem *qe = reinterpret_cast<const elem *>(&qv);
                const elem *ge = reinterpret_cast<const elem *>(&gv);
#pragma unroll
                for (int i = 0; i < C::EPC; ++i) {
                    Qt[(c * C::EPC + i) * QTS + r] = qe[i];
                    Gt[(c * C::EPC + i) * QTS + r] = ge[i];
                }
            }
            if (tid < 32) {
                const int q = i0 + tid;
                lse_s[tid] = q < T ? a.lse2[((int64_t)b * Hq + h) * T + q] : INFINITY;
                D_s[tid] = q < T ? a.D[((int64_t)b * Hq + h) * T + q] : 0.f;
                if constexpr (KL) lset_s[tid] = q < T ? a.lse_t[((int64_t)b * Hq + h) * T + q] : INFINITY;
            }
            __syncthreads();
            if (jw >= T || i0 + 31 < jw) continue;     // no query of this tile sees these keys

            // ---- S = Q K^T and dP = G V^T: lane -> key, rows -> queries
            f32x16 s, dp;
#pragma unroll
            for (int e = 0; e < 16; ++e) { s[e] = 0.f; dp[e] = 0.f; }
#pragma unroll
            for (int kc = 0; kc < C::NKC; ++kc) {
                const int c = kc * MM::K + half * MM::VEC;
                s = MM::mma(load_operand<DT>(Qs + (lane & 31) * C::RST + c), kf[kc], s);
                dp = MM::mma(load_operand<DT>(Gs + (lane & 31) * C::RST + c), vf[kc], dp);
            }
            f32x16 st;                                   // teacher scores (KL term)
            if constexpr (KL) {
#pragma unroll
                for (int e = 0; e < 16; ++e) st[e] = 0.f;
#pragma unroll
                for (int kc = 0; kc < C::NKC; ++kc) {
                    const int c = kc * MM::K + half * MM::VEC;
                    st = MM::mma(load_operand<DT>(Qts + (lane & 31) * C::RST + c), ktf[kc], st);
                }
            }
            const bool diag = i0 < jw + 31;
#pragma unroll
            for (int e4 = 0; e4 < 4; ++e4) {
                const int r0 = 8 * e4 + 4 * half;
                const f32x4 ls = *reinterpret_cast<const f32x4 *>(lse_s + r0);
                const f32x4 dd = *reinterpret_cast<const f32x4 *>(D_s + r0);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int e = 4 * e4 + i;
                    float p = __builtin_amdgcn_exp2f(__builtin_fmaf(s[e], scale_log2, -ls[i]));
                    if (diag && i0 + r0 + i < key) p = 0.f;
                    s[e] = p;
                    dp[e] = p * (dp[e] - dd[i]);
                    if constexpr (KL) {
                        float pt = __builtin_amdgcn_exp2f(__builtin_fmaf(st[e], scale_log2, -lset_s[r0 + i]));
                        if (diag && i0 + r0 + i < key) pt = 0.f;
                        dp[e] = (dp[e] + a.kl_scale * (p - pt)) * a.grad_scale;
                    }
                }
            }
            // ---- dV^T += G^T P,  dK^T += Q^T dS  (k = the tile's 32 queries)
            if constexpr (DT == F32) {
#pragma unroll
                for (int kc2 = 0; kc2 < 16; ++kc2) {
                    const int q = 8 * (kc2 >> 2) + 4 * half + (kc2 & 3);
#pragma unroll
                    for (int d = 0; d < C::NDB; ++d) {
                        const int c = d * 32 + (lane & 31);
                        dvt[d] = MM::mma(Gt[c * QTS + q], s[kc2], dvt[d]);
                        dkt[d] = MM::mma(Qt[c * QTS + q], dp[kc2], dkt[d]);
                    }
                }
            } else {
#pragma unroll
                for (int kc2 = 0; kc2 < 2; ++kc2) {
                    const typename MM::operand pb = pack_operand<DT>(s, 8 * kc2);
                    const typename MM::operand sb = pack_operand<DT>(dp, 8 * kc2);
                    const int q0 = 16 * kc2 + 4 * half;
#pragma unroll
                    for (int d = 0; d < C::NDB; ++d) {
                        const int c = d * 32 + (lane & 31);
                        dvt[d] = MM::mma(load_operand_split<DT>(Gt + c * QTS + q0, Gt + c * QTS + q0 + 8), pb, dvt[d]);
                        dkt[d] = MM::mma(load_operand_split<DT>(Qt + c * QTS + q0, Qt + c * QTS + q0 + 8), sb, dkt[d]);
                    }
                }
            }
        }
    }
    // ---- write dK^T / dV^T: lane -> token (key), rows -> head-dimension index
    if (key < T) {
        elem *dyt = static_cast<elem *>(a.dyt);
        const int64_t m = row0 + key;
#pragma unroll
        for (int d = 0; d < C::NDB; ++d)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int c = d * 32 + 8 * (e >> 2) + 4 * half + (e & 3);
                if (DH < 32 && c >= DH) continue;
                dyt[(int64_t)(koff + kvh * DH + c) * a.ldt + m] = from_f32<DT>(dkt[d][e] * inv_sqrt);
                dyt[(int64_t)(voff + kvh * DH + c) * a.ldt + m] = from_f32<DT>(dvt[d][e]);
            }
    }
}

// ------------------------------------------------------------------ dQ
template <int DT, int DH, bool KL>
__global__ __launch_bounds__(256, 1) void attn_bwd_dq_kernel(AttnBwdArgs a, float scale_log2,
                                                             float inv_sqrt, int hpw, int nqt, int n_ht) {
    typedef BwdCfg<DT, DH> C;
    typedef typename C::elem elem;
    typedef Mma<DT> MM;
    constexpr int BNK = C::BNK;
    constexpr int KTS = C::KTS;
    extern __shared__ __align__(16) unsigned char smem[];
    elem *Ks = reinterpret_cast<elem *>(smem);
    elem *Vs = Ks + BNK * C::RST;
    elem *Kt = Vs + BNK * C::RST;
    elem *Kts = reinterpret_cast<elem *>(smem + C::DQ_LDS);   // KL term: the teacher's key tile

    const int T = a.seq_len, Hq = a.n_heads, Hkv = a.n_kv_heads;
    const int G = Hq / Hkv;
    const int QT = 128 / hpw;

    const int nwg = gridDim.x;
    int lin = blockIdx.x;
    if ((nwg & 7) == 0) lin = (lin & 7) * (nwg >> 3) + (lin >> 3);
    const int qt = nqt - 1 - lin % nqt;                // longest query tiles first
    const int ht = (lin / nqt) % n_ht;
    const int b = lin / (nqt * n_ht);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, half = lane >> 5;
    const int h = ht * hpw + wave % hpw;
    const int kvh = h / G;
    const int q0 = qt * QT + (wave / hpw) * 32;
    const int qrow = q0 + (lane & 31);
    const bool active = q0 < T;
    const int kend = min(T, qt * QT + QT);
    const int64_t row0 = (int64_t)b * T;
    const elem *Qp = static_cast<const elem *>(a.q);
    const elem *Kp = static_cast<const elem *>(a.k);
    const elem *Vp = static_cast<const elem *>(a.v);
    const elem *Gg = static_cast<const elem *>(a.g);

    typename MM::operand qf[C::NKC], gf[C::NKC], qtf[KL ? C::NKC : 1];
#pragma unroll
    for (int kc = 0; kc < C::NKC; ++kc) {
        const int c = kc * MM::K + half * MM::VEC;
        if (qrow < T) {
            qf[kc] = load_operand<DT>(Qp + (row0 + qrow) * a.ldq + h * DH + c);
            gf[kc] = load_operand<DT>(Gg + ((row0 + qrow) * Hq + h) * DH + c);
            if constexpr (KL)
                qtf[kc] = load_operand<DT>(static_cast<const elem *>(a.qt) + (row0 + qrow) * a.ldq + h * DH + c);
        } else {
            qf[kc] = pack_operand<DT>(f32x16{}, 0);
            gf[kc] = pack_operand<DT>(f32x16{}, 0);
            if constexpr (KL) qtf[kc] = pack_operand<DT>(f32x16{}, 0);
        }
    }
    const float lset = KL && qrow < T ? a.lse_t[((int64_t)b * Hq + h) * T + qrow] : INFINITY;
    const float lse = qrow < T ? a.lse2[((int64_t)b * Hq + h) * T + qrow] : INFINITY;
    const float Dq = qrow < T ? a.D[((int64_t)b * Hq + h) * T + qrow] : 0.f;
    f32x16 dqt[C::NDB];
#pragma unroll
    for (int d = 0; d < C::NDB; ++d)
#pragma unroll
        for (int e = 0; e < 16; ++e) dqt[d][e] = 0.f;
    if constexpr (DH < 32) {
        for (int i = tid; i < C::DHP * KTS; i += 256) Kt[i] = from_f32<DT>(0.f);
    }

    constexpr int CPR = DH / C::EPC;
    for (int kb = 0; kb < kend; kb += BNK) {
        __syncthreads();
        for (int idx = tid; idx < BNK * CPR; idx += 256) {
            const int r = idx / CPR, c = idx % CPR;
            const int k = kb + r;
            u32x4 kv = u32x4{0u, 0u, 0u, 0u}, vv = u32x4{0u, 0u, 0u, 0u};
            if (k < T) {
                kv = *reinterpret_cast<const u32x4 *>(Kp + (row0 + k) * a.ldq + kvh * DH + c * C::EPC);
                vv = *reinterpret_cast<const u32x4 *>(Vp + (row0 + k) * a.ldv + kvh * DH + c * C::EPC);
            }
            *reinterpret_cast<u32x4 *>(Ks + r * C::RST + c * C::EPC) = kv;
            *reinterpret_cast<u32x4 *>(Vs + r * C::RST + c * C::EPC) = vv;
            if constexpr (KL) {
                u32x4 tv = u32x4{0u, 0u, 0u, 0u};
                if (k < T)
                    tv = *reinterpret_cast<const u32x4 *>(static_cast<const elem *>(a.kt) + (row0 + k) * a.ldq +
                                                          kvh * DH + c * C::EPC);
                *reinterpret_cast<u32x4 *>(Kts + r * C::RST + c * C::EPC) = tv;
            }
            const elem *ke = reinterpret_cast<const elem *>(&kv);
#pragma unroll
            for (int i = 0; i < C::EPC; ++i) Kt[(c * C::EPC + i) * KTS + r] = ke[i];
        }
        __syncthreads();
        if (!active || kb > q0 + 31) continue;

        f32x16 s[2], dp[2];
#pragma unroll
        for (int sb = 0; sb < 2; ++sb) {
#pragma unroll
            for (int e = 0; e < 16; ++e) { s[sb][e] = 0.f; dp[sb][e] = 0.f; }
            const int krow = sb * 32 + (lane & 31);
#pragma unroll
            for (int kc = 0; kc < C::NKC; ++kc) {
                const int c = kc * MM::K + half * MM::VEC;
                s[sb] = MM::mma(load_operand<DT>(Ks + krow * C::RST + c), qf[kc], s[sb]);
                dp[sb] = MM::mma(load_operand<DT>(Vs + krow * C::RST + c), gf[kc], dp[sb]);
            }
        }
        f32x16 stt[KL ? 2 : 1];                          // teacher scores (KL term)
        if constexpr (KL) {
#pragma unroll
            for (int sb = 0; sb < 2; ++sb) {
#pragma unroll
                for (int e = 0; e < 16; ++e) stt[sb][e] = 0.f;
                const int krow = sb * 32 + (lane & 31);
#pragma unroll
                for (int kc = 0; kc < C::NKC; ++kc) {
                    const int c = kc * MM::K + half * MM::VEC;
                    stt[sb] = MM::mma(load_operand<DT>(Kts + krow * C::RST + c), qtf[kc], stt[sb]);
                }
            }
        }
        const bool diag = kb + BNK - 1 > q0;
#pragma unroll
        for (int sb = 0; sb < 2; ++sb)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int k = kb + sb * 32 + 8 * (e >> 2) + 4 * half + (e & 3);
                float p = __builtin_amdgcn_exp2f(__builtin_fmaf(s[sb][e], scale_log2, -lse));
                if (diag && k > qrow) p = 0.f;
                dp[sb][e] = p * (dp[sb][e] - Dq);
                if constexpr (KL) {
                    float pt = __builtin_amdgcn_exp2f(__builtin_fmaf(stt[sb][e], scale_log2, -lset));
                    if (diag && k > qrow) pt = 0.f;
                    dp[sb][e] = (dp[sb][e] + a.kl_scale * (p - pt)) * a.grad_scale;
                }
            }
        // ---- dQ^T += K^T dS^T (k = the tile's 64 keys)
        if constexpr (DT == F32) {
#pragma unroll
            for (int kc2 = 0; kc2 < 32; ++kc2) {
                const int sb = kc2 >> 4, e = kc2 & 15;
                const int k = sb * 32 + 8 * (e >> 2) + 4 * half + (e & 3);
#pragma unroll
                for (int d = 0; d < C::NDB; ++d)
                    dqt[d] = MM::mma(Kt[(d * 32 + (lane & 31)) * KTS + k], dp[sb][e], dqt[d]);
            }
        } else {
#pragma unroll
            for (int kc2 = 0; kc2 < 4; ++kc2) {
                const int sb = kc2 >> 1, hf = kc2 & 1;
                const typename MM::operand sbop = pack_operand<DT>(dp[sb], 8 * hf);
                const int k0 = sb * 32 + hf * 16 + 4 * half;
#pragma unroll
                for (int d = 0; d < C::NDB; ++d) {
                    const elem *rowp = Kt + (d * 32 + (lane & 31)) * KTS;
                    dqt[d] = MM::mma(load_operand_split<DT>(rowp + k0, rowp + k0 + 8), sbop, dqt[d]);
                }
            }
        }
    }
    if (active && qrow < T) {
        elem *dyt = static_cast<elem *>(a.dyt);
        const int64_t m = row0 + qrow;
#pragma unroll
        for (int d = 0; d < C::NDB; ++d)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int c = d * 32 + 8 * (e >> 2) + 4 * half + (e & 3);
                if (DH < 32 && c >= DH) continue;
                dyt[(int64_t)(h * DH + c) * a.ldt + m] = from_f32<DT>(dqt[d][e] * inv_sqrt);
            }
    }
}

// ------------------------------------------------------------------ transpose
template <typename E>
__global__ __launch_bounds__(256) void transpose_kernel(const E *__restrict__ in, E *__restrict__ out,
                                                        int rows, int cols, int kpad, int64_t out_ld) {
    __shared__ E tile[64][65];
    const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    for (int i = ty; i < 64; i += 4) {
        const int r = r0 + i, c = c0 + tx;
        tile[i][tx] = (r < rows && c < cols) ? in[(int64_t)r * cols + c] : E(0);
    }
    __syncthreads();
    for (int i = ty; i < 64; i += 4) {
        const int c = c0 + i, r = r0 + tx;        // out[c][r]
        if (c < cols && r < kpad) out[(int64_t)c * out_ld + r] = tile[tx][i];
    }
}

// The same for 2-byte elements with 16-byte global loads and stores (cols and out_ld multiples of 8,
// 16-byte aligned bases): a thread loads 8 consecutive elements of a row, the tile is turned in LDS
// (rows 33 words apart, so the eight rows a read instruction touches fall in distinct banks), and a
// thread stores 8 consecutive elements of an output row.
__global__ __launch_bounds__(256) void transpose16_kernel(const uint16_t *__restrict__ in, uint16_t *__restrict__ out,
                                                          int rows, int cols, int kpad, int64_t out_ld) {
    constexpr int LD = 66;                           // u16 per LDS row: 33 words
    __shared__ uint32_t tile[64 * LD / 2];
    const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
    const int t = threadIdx.x, cc = t & 7;
#pragma unroll
    for (int pass = 0; pass < 2; ++pass) {
        const int i = (t >> 3) + 32 * pass, r = r0 + i, c = c0 + 8 * cc;
        u32x4 v = u32x4{0u, 0u, 0u, 0u};
        if (r < rows && c < cols) v = *reinterpret_cast<const u32x4 *>(in + (int64_t)r * cols + c);
#pragma unroll
        for (int k = 0; k < 4; ++k) tile[(i * LD + 8 * cc) / 2 + k] = v[k];
    }
    __syncthreads();
    const uint16_t *t16 = reinterpret_cast<const uint16_t *>(tile);
#pragma unroll
    for (int pass = 0; pass < 2; ++pass) {
        const int j = (t >> 3) + 32 * pass, c = c0 + j;    // output row c, input rows 8 cc .. 8 cc + 7
        uint32_t w[4];
#pragma unroll
        for (int k = 0; k < 4; ++k)
            w[k] = (uint32_t)t16[(8 * cc + 2 * k) * LD + j] | ((uint32_t)t16[(8 * cc + 2 * k + 1) * LD + j] << 16);
        const int r = r0 + 8 * cc;
        if (c < cols && r < kpad) *reinterpret_cast<u32x4 *>(out + (int64_t)c * out_ld + r) = u32x4{w[0], w[1], w[2], w[3]};
    }
}

// zero columns [c0, ld) of a rows x ld matrix of 2- or 4-byte elements
template <typename E>
__global__ __launch_bounds__(256) void zero_cols_kernel(E *__restrict__ p, int rows, int ld, int c0) {
    const int w = ld - c0;
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < (int64_t)rows * w) p[(i / w) * ld + c0 + i % w] = E(0);
}

// ------------------------------------------------------------------ LSQ scale gradient
template <int DT>
__global__ __launch_bounds__(256) void lsq_kernel(QuantShape sh, const void *__restrict__ w,
                                                  const float *__restrict__ scale,
                                                  const uint8_t *__restrict__ zero,
                                                  float *__restrict__ dw, const float *__restrict__ dw2,
                                                  float qk_unscale, float g0, float g1, float g2,
                                                  float *__restrict__ ds) {
    typedef typename Mma<DT>::elem elem;
    const int64_t chunk = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t nchunks = (int64_t)sh.rows * sh.cols / 8;
    const int lpg = sh.group / 8;
    const bool live = chunk < nchunks;
    const int64_t e = live ? chunk * 8 : 0;
    const int r = (int)(e / sh.cols), col = (int)(e % sh.cols);
    const int m = r < sh.row_k ? 0 : (r < sh.row_v ? 1 : 2);
    const int bits = sh.bits[m];
    const int64_t gi = (int64_t)r * (sh.cols / sh.group) + col / sh.group;
    float acc = 0.f;
    f32x4 d0 = f32x4{0.f, 0.f, 0.f, 0.f}, d1 = d0;
    if (live) {
        f32x4 *dp = reinterpret_cast<f32x4 *>(dw + e);
        d0 = dp[0];
        d1 = dp[1];
        if (dw2 != nullptr) {                           // the second half of a split product
            const f32x4 *dq = reinterpret_cast<const f32x4 *>(dw2 + e);
            d0 += dq[0];
            d1 += dq[1];
        }
        // rows of W_Q and W_K: the backward kept their dS scaled by a power of two (qk_unscale is
        // its inverse, exact)
        const bool rescale = qk_unscale != 1.f && r < sh.row_v;
        if (rescale) {
            d0 *= qk_unscale;
            d1 *= qk_unscale;
        }
        if (dw2 != nullptr || rescale) {
            dp[0] = d0;
            dp[1] = d1;
        }
    }
    if (live && bits != 0) {
        const float s = scale[gi];
        const elem *wp = static_cast<const elem *>(w) + e;
        float lo, hi;
        if (sh.scheme == 0) {
            const float zf = (float)zero[gi];
            lo = -zf;
            hi = (float)((1 << bits) - 1) - zf;
        } else {
            hi = (float)((1 << (bits - 1)) - 1);
            lo = -hi;
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const float v = to_f32<DT>(wp[i]) / s;
            float phi;
            if (v < lo) phi = lo;
            else if (v > hi) phi = hi;
            else phi = rintf(v) - v;
            acc = __builtin_fmaf(i < 4 ? d0[i] : d1[i - 4], phi, acc);
        }
    }
    for (int off = lpg / 2; off >= 1; off >>= 1) acc += __shfl_xor(acc, off, 64);
    if (live && (threadIdx.x & (lpg - 1)) == 0) {
        const float gm = m == 0 ? g0 : (m == 1 ? g1 : g2);
        ds[gi] = bits != 0 ? gm * acc : 0.f;
    }
}

template <int DT, int DH, bool KL>
hipError_t run_bwd_kl(const AttnBwdArgs &a, hipStream_t st) {
    const float scale_log2 = 1.4426950408889634f / sqrtf((float)DH);
    const float inv_sqrt = 1.f / sqrtf((float)DH);
    typedef BwdCfg<DT, DH> C;
    typedef typename C::elem elem;
    // the KL term stages the teacher's query (dK/dV) or key (dQ) tile after the regular layout
    const size_t dkdv_lds = C::DKDV_LDS + (KL ? 32 * C::RST * sizeof(elem) + 32 * sizeof(float) : 0);
    const size_t dq_lds = C::DQ_LDS + (KL ? (size_t)C::BNK * C::RST * sizeof(elem) : 0);
    const int nkb = (a.seq_len + 127) / 128;
    hipError_t e = hipFuncSetAttribute((const void *)attn_bwd_dkdv_kernel<DT, DH, KL>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)dkdv_lds);
    if (e != hipSuccess) return e;
    e = hipFuncSetAttribute((const void *)attn_bwd_dq_kernel<DT, DH, KL>,
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)dq_lds);
    if (e != hipSuccess) return e;
    attn_bwd_dkdv_kernel<DT, DH, KL><<<dim3(nkb * a.n_kv_heads * a.batch), dim3(256), dkdv_lds, st>>>(
        a, scale_log2, inv_sqrt, nkb);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int G = a.n_heads / a.n_kv_heads;
    const int hpw = G % 4 == 0 ? 4 : G;
    const int QT = 128 / hpw;
    const int nqt = (a.seq_len + QT - 1) / QT;
    const int n_ht = a.n_heads / hpw;
    attn_bwd_dq_kernel<DT, DH, KL><<<dim3(nqt * n_ht * a.batch), dim3(256), dq_lds, st>>>(
        a, scale_log2, inv_sqrt, hpw, nqt, n_ht);
    return hipGetLastError();
}

template <int DT, int DH>
hipError_t run_bwd(const AttnBwdArgs &a, hipStream_t st) {
    if (a.qt) return run_bwd_kl<DT, DH, true>(a, st);
    return run_bwd_kl<DT, DH, false>(a, st);
}

template <int DT>
hipError_t bwd_dh(const AttnBwdArgs &a, hipStream_t st) {
    // the 16-bit dtypes at head_dim 64 / 128 take the DMA-pipelined kernels (with or without the
    // KL term)
    if constexpr (DT != F32) {
        if (a.head_dim == 64) return run_bwd_dma<DT, 64>(a, st);
        if (a.head_dim == 128) return run_bwd_dma<DT, 128>(a, st);
    }
    switch (a.head_dim) {
    case 16: return run_bwd<DT, 16>(a, st);
    case 64: return run_bwd<DT, 64>(a, st);
    default: return run_bwd<DT, 128>(a, st);
    }
}

}  // namespace

hipError_t launch_attn_bwd(int dtype, const AttnBwdArgs &a, hipStream_t st) {
    switch (dtype) {
    case F32: return bwd_dh<F32>(a, st);
    case F16: return bwd_dh<F16>(a, st);
    default: return bwd_dh<BF16>(a, st);
    }
}

hipError_t launch_transpose(int dtype, const void *in, void *out, int rows, int cols, int64_t out_ld,
                            hipStream_t st) {
    // columns [rows, kpad) of out are written as 0; [kpad, out_ld) are not touched
    const int kpad = (rows + 63) / 64 * 64;
    if (out_ld < kpad) return hipErrorInvalidValue;
    const dim3 grid((cols + 63) / 64, kpad / 64), block(256);
    if (dtype == F32)
        transpose_kernel<float><<<grid, block, 0, st>>>(static_cast<const float *>(in), static_cast<float *>(out), rows, cols, kpad, out_ld);
    else if (cols % 8 == 0 && out_ld % 8 == 0 && ((uintptr_t)in & 15) == 0 && ((uintptr_t)out & 15) == 0)
        transpose16_kernel<<<grid, block, 0, st>>>(static_cast<const uint16_t *>(in), static_cast<uint16_t *>(out), rows, cols, kpad, out_ld);
    else
        transpose_kernel<uint16_t><<<grid, block, 0, st>>>(static_cast<const uint16_t *>(in), static_cast<uint16_t *>(out), rows, cols, kpad, out_ld);
    return hipGetLastError();
}

hipError_t launch_zero_cols(int dtype, void *p, int rows, int ld, int c0, hipStream_t st) {
    if (c0 >= ld) return hipSuccess;
    const int64_t n = (int64_t)rows * (ld - c0);
    const dim3 grid((unsigned)((n + 255) / 256)), block(256);
    if (dtype == F32)
        zero_cols_kernel<float><<<grid, block, 0, st>>>(static_cast<float *>(p), rows, ld, c0);
    else
        zero_cols_kernel<uint16_t><<<grid, block, 0, st>>>(static_cast<uint16_t *>(p), rows, ld, c0);
    return hipGetLastError();
}

hipError_t launch_lsq_scale_grad(const QuantShape &sh, int dtype, const void *w, const float *scale,
                                 const uint8_t *zero, float *dw, const float *dw2, float qk_unscale,
                                 const float gamma[3], float *ds, hipStream_t st) {
    const int64_t nchunks = (int64_t)sh.rows * sh.cols / 8;
    const dim3 grid((unsigned)((nchunks + 255) / 256)), block(256);
    switch (dtype) {
    case F32: lsq_kernel<F32><<<grid, block, 0, st>>>(sh, w, scale, zero, dw, dw2, qk_unscale, gamma[0], gamma[1], gamma[2], ds); break;
    case F16: lsq_kernel<F16><<<grid, block, 0, st>>>(sh, w, scale, zero, dw, dw2, qk_unscale, gamma[0], gamma[1], gamma[2], ds); break;
    default: lsq_kernel<BF16><<<grid, block, 0, st>>>(sh, w, scale, zero, dw, dw2, qk_unscale, gamma[0], gamma[1], gamma[2], ds); break;
    }
    return hipGetLastError();
}

}  // namespace jab
