// attn_jvp.hip -- forward-mode derivative of causal grouped-query attention for the curvature
// scores of eq. gn: the exact Gauss-Newton quadratic forms at the float point.
//
// Paper: Method, "Sensitivity and allocation", eq. gn: at the float point the Hessian of the joint
// loss (eq. joint_loss) is H = 2 J_A^T J_A + lambda_KL J_Q^T I(P) J_Q, so each Hutchinson term needs
// the directional derivative of the attention output, J_A v, and of the attention logits, J_Q v,
// along a probe v.  The Appendix on per-unit traces partitions v^T H v over the units (W_Q, W_K,
// W_V): t_u = v_u^T (H v)_u.
//
// With the projection y = X W^T at the float point and its tangent yd = X v^T (the probe's W_Q rows
// move Q, its W_K rows K, its W_V rows V), per query row i of head h and logits z = q k^T / sqrt(dh):
//   zQ_ij = qd_i . k_j / sqrt(dh),  zK_ij = q_i . kd_j / sqrt(dh),  P = softmax_j(z),
//   aQ_i = sum_j P_ij (zQ_ij - mQ_i) v_j,  mQ_i = sum_j P_ij zQ_ij  (aK alike),  aV_i = sum_j P_ij vd_j,
// so J_A v = aQ + aK + aV and J_Q v = zQ + zK.  The kernel returns, per (sequence, head, 32-query
// block), the nine sums over rows of
//   <aQ,aQ> <aK,aK> <aV,aV> <aQ,aK> <aQ,aV> <aK,aV>  and  zQ.I.zQ  zK.I.zK  zQ.I.zK,
// a.I.b = sum_j P_ij a_j b_j - (sum_j P_ij a_j)(sum_j P_ij b_j) (the softmax's Fisher information),
// from which every form follows (curv_forms_kernel).
//
// gfx950 design
//  * One pass over the keys with an online softmax: per block of 32 keys, three score products on
//    the matrix cores (S^T = K Q^T, K Qd^T, Kd Q^T; lane = query, 16 keys per lane), one shared
//    reference maximum, and four value products O^T += V^T P^T, UQ^T += V^T (P zQ)^T,
//    UK^T += V^T (P zK)^T, W^T += Vd^T P^T.  The row sums l, sum P zQ, sum P zK, sum P zQ^2,
//    sum P zK^2, sum P zQ zK are lane-local fp32 sums (one half-wave exchange at the end); at the
//    end a_hat = O / l, aQ = UQ / l - (mQ / l) a_hat, ...
//  * Workgroups of 4 waves, one per SIMD (the four fp32 accumulator sets of 32 queries x head_dim
//    take 256 registers at head_dim 128); each wave owns 32 queries of one query head, and the
//    workgroup's waves share a key/value head, so one copy of the K, Kd, V^T, Vd^T tiles of a block
//    serves them all.  The tiles stream from global memory into an LDS ring by direct-to-LDS loads,
//    16-byte chunks XOR-swizzled per row (conflict-free fragment reads), one barrier per block.
//  * The reference maximum moves whenever a block's maximum exceeds it (probabilities at most 1,
//    so the tangent-weighted probabilities stay in fp16 range); a rescale multiplies every
//    accumulator and row sum by the same factor.  Deterministic: no atomics, fixed orders.
#include "attn_fwd_impl.h"

namespace jab {
namespace {

template <int DT, int DH>
struct JvpCfg {
    typedef typename Mma<DT>::elem elem;
    static constexpr int ES = (int)sizeof(elem);
    static constexpr int EPC = 16 / ES;                // elements per 16-byte chunk
    static constexpr int NKC = DH / Mma<DT>::K;        // k-steps of a score product
    static constexpr int DHP = DH < 32 ? 32 : DH;      // rows of the transposed accumulators
    static constexpr int NDB = DHP / 32;
    static constexpr int CK = DH * ES / 16;            // chunks per key row
    static constexpr int CV = 32 * ES / 16;            // chunks per transposed-value row (32 keys)
    static constexpr int KB = 32 * CK * 16;            // bytes of a key tile
    static constexpr int VB = DH * CV * 16;            // bytes of a transposed-value tile
    static constexpr int STAGE = 2 * KB + 2 * VB;      // K | Kd | V^T | Vd^T
    static constexpr int NS = 4 * STAGE <= 160 * 1024 ? 4 : (3 * STAGE <= 160 * 1024 ? 3 : 2);
    static constexpr int KI = KB / 1024, VI = VB / 1024;   // DMA instructions per tile
    static constexpr int NI = 2 * KI + 2 * VI;             // ... per block
    static constexpr int PW = NI / 4;                      // ... per wave
    static constexpr int KL = DT == F32 ? NKC / 4 : NKC;   // LDS reads of a key fragment set
    static constexpr int VG = DT == F32 ? 4 : 2;           // V^T reads per row block
    // 32-row blocks of the output tangents per pass: the four accumulator sets of a wave hold
    // NDBP x 64 registers; at head_dim 128 (and fp32 from 64) the rows are covered in several
    // passes, each recomputing the scores
    static constexpr int NDBP = (DT == F32 && DH >= 64) ? 1 : (DH == 128 ? 2 : NDB);
    static constexpr int NPASS = NDB / NDBP;
    static_assert(KB % 1024 == 0 && VB % 1024 == 0 && NI % 4 == 0, "whole DMA instructions per tile");
    static_assert(DT != F32 || NKC % 4 == 0, "fp32 key fragments are read 4 k-steps at a time");
};

constexpr int kJvpParts = 9;

template <int DT, int DH>
__global__ __launch_bounds__(256, 1) void attn_jvp_kernel(JvpArgs a, float scale_log2, float inv_sqrt, int hpw,
                                                          int nqt, int n_ht, int dpass) {
    typedef JvpCfg<DT, DH> C;
    typedef typename C::elem elem;
    typedef Mma<DT> MM;
    typedef typename MM::operand opnd;
    extern __shared__ __align__(16) unsigned char smem[];

    const int T = a.seq_len, Hq = a.n_heads;
    const int G = Hq / a.n_kv_heads;
    const int QT = 4 * 32 / hpw;                       // queries per workgroup tile
    const int Tp = vt_pad(T);

    // ---- workgroup -> (sequence, head tile, query tile): longest tiles first, and one XCD runs
    // all tiles of a (sequence, head tile)
    const int nwg = gridDim.x;
    int lin = blockIdx.x;
    if ((nwg & 7) == 0) lin = (lin & 7) * (nwg >> 3) + (lin >> 3);
    const int qt = nqt - 1 - lin % nqt;
    const int ht = (lin / nqt) % n_ht;
    const int b = lin / (nqt * n_ht);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, half = lane >> 5;
    const int h = ht * hpw + wave % hpw;
    const int kvh = h / G;
    const int q0 = qt * QT + (wave / hpw) * 32;        // first query of this wave
    const int qrow = q0 + (lane & 31);
    const int kend = min(T, qt * QT + QT);
    const int nblk = (kend + 31) / 32;                 // key blocks the workgroup loads
    const int jlast = q0 < T ? q0 / 32 : -1;           // the wave's diagonal block (-1: no queries)
    const int lim = min(qrow, T - 1);                  // last key this lane's query sees
    const int64_t row0 = (int64_t)b * T;

    // ---- the wave's queries and query tangents as B operands of the score products
    opnd qf[C::NKC], qdf[C::NKC];
    {
        const elem *qp = static_cast<const elem *>(a.q) + (row0 + min(qrow, T - 1)) * a.ld + h * DH;
        const elem *qdp = static_cast<const elem *>(a.qd) + (row0 + min(qrow, T - 1)) * a.ld + h * DH;
        if constexpr (DT == F32) {
#pragma unroll
            for (int i = 0; i < C::NKC / 4; ++i) {
                const f32x4 v = *reinterpret_cast<const f32x4 *>(qp + s_k<DT, DH>(4 * i, half));
                const f32x4 vd = *reinterpret_cast<const f32x4 *>(qdp + s_k<DT, DH>(4 * i, half));
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    qf[4 * i + t] = qrow < T ? v[t] : 0.f;
                    qdf[4 * i + t] = qrow < T ? vd[t] : 0.f;
                }
            }
        } else {
#pragma unroll
            for (int kc = 0; kc < C::NKC; ++kc) {
                u32x4 v = *reinterpret_cast<const u32x4 *>(qp + s_k<DT, DH>(kc, half));
                u32x4 vd = *reinterpret_cast<const u32x4 *>(qdp + s_k<DT, DH>(kc, half));
                if (qrow >= T) { v = u32x4{0u, 0u, 0u, 0u}; vd = v; }
                qf[kc] = __builtin_bit_cast(opnd, v);
                qdf[kc] = __builtin_bit_cast(opnd, vd);
            }
        }
    }

    // ---- DMA of key block j into ring slot j % NS: wave w issues instructions w, w + 4, ... of the
    // block's NI (K tile, Kd tile, V^T tile, Vd^T tile; 64 chunks = 1 KiB each).  Chunk P of a key
    // tile holds row P / CK, physical chunk P % CK = logical chunk ^ swz_key(row); transposed-value
    // tiles alike with CV.  Keys past the sequence read the rows that follow it (the next sequence,
    // or the slack rows after the last one) and the padded value columns (zero): the mask removes
    // them.
    // MUBUF form (buffer_load ... lds): a resource per tensor at this sequence and key/value head,
    // fixed per-lane byte offsets, the block's offset in a scalar register; the LDS counter stays
    // ordered, so each fragment read is waited for on its own
    const elem *kseq = static_cast<const elem *>(a.k) + row0 * a.ld + kvh * DH;
    const elem *kdseq = static_cast<const elem *>(a.kd) + row0 * a.ld + kvh * DH;
    const elem *vseq = static_cast<const elem *>(a.vt) + (int64_t)kvh * DH * a.ldv + (int64_t)b * Tp;
    const elem *vdseq = static_cast<const elem *>(a.vdt) + (int64_t)kvh * DH * a.ldv + (int64_t)b * Tp;
    const i32x4 rsrc[4] = {buffer_rsrc(kseq), buffer_rsrc(kdseq), buffer_rsrc(vseq), buffer_rsrc(vdseq)};
    const int wv_s = __builtin_amdgcn_readfirstlane(wave);
    uint32_t voff[C::PW];
    int tens[C::PW], dst[C::PW];
#pragma unroll
    for (int i = 0; i < C::PW; ++i) {
        const int idx = wave + 4 * i;
        if (idx < 2 * C::KI) {
            const int t = idx / C::KI, p = (idx % C::KI) * 64 + lane;
            const int r = p / C::CK, c = (p % C::CK) ^ swz_key<C::CK>(r);
            voff[i] = (uint32_t)((r * a.ld + c * C::EPC) * C::ES);
            tens[i] = t;
        } else {
            const int iv = idx - 2 * C::KI;
            const int t = iv / C::VI, p = (iv % C::VI) * 64 + lane;
            const int r = p / C::CV, c = (p % C::CV) ^ swz_key<C::CV>(r);
            voff[i] = (uint32_t)((r * (int)a.ldv + c * C::EPC) * C::ES);
            tens[i] = 2 + t;
        }
    }
    // destination of instruction i inside a slot (wave-uniform): the tile's offset plus its KiB
#pragma unroll
    for (int i = 0; i < C::PW; ++i) {
        const int idx = wv_s + 4 * i;
        dst[i] = idx < 2 * C::KI ? (idx / C::KI) * C::KB + (idx % C::KI) * 1024
                                 : 2 * C::KB + ((idx - 2 * C::KI) / C::VI) * C::VB + ((idx - 2 * C::KI) % C::VI) * 1024;
    }
    auto issue = [&](int j) {
        if (j >= nblk) return;
        unsigned char *st = smem + (j % C::NS) * C::STAGE;
        const int kofs = 32 * j * a.ld * C::ES, vofs = 32 * j * C::ES;
#pragma unroll
        for (int i = 0; i < C::PW; ++i) {
            // every instruction index of a wave has the same tensor in every lane: the tile order is
            // fixed per instruction slot, chosen by the wave-uniform index
            const int idx = wv_s + 4 * i;
            const int t = idx < 2 * C::KI ? idx / C::KI : 2 + (idx - 2 * C::KI) / C::VI;
            buffer_dma16(rsrc[t], voff[i], t < 2 ? kofs : vofs, st + dst[i]);
        }
    };

    // ---- LDS fragment reads (per-lane bases; swizzled chunks)
    const int kr = lane & 31;
    const int krow = kr * C::CK * 16, kkey = swz_key<C::CK>(kr) * 16;
    const int vrow = DH < 32 ? (lane & 31) % DH : (lane & 31);
    const int vbase = vrow * C::CV * 16, vkey = swz_key<C::CV>(vrow) * 16;   // equal for rows 32 apart
    // key fragments of read l (16-bit: k-step l; fp32: k-steps 4 l .. 4 l + 3)
    constexpr int KPL = C::NKC / C::KL;
    auto key_frag = [&](const unsigned char *tile, int l, opnd (&f)[KPL]) {
        const int cl = DT == F32 ? half * (DH / 8) + l : 2 * l + half;   // logical chunk
        const unsigned char *pk = tile + krow + ((cl * 16) ^ kkey);
        if constexpr (DT == F32) {
            const f32x4 v = *reinterpret_cast<const f32x4 *>(pk);
#pragma unroll
            for (int t = 0; t < 4; ++t) f[t] = v[t];
        } else {
            f[0] = __builtin_bit_cast(opnd, *reinterpret_cast<const u32x4 *>(pk));
        }
    };
    // V^T fragment g of row block d: 16-bit, the 8 keys of k-step g (logical chunk 2 g + half);
    // fp32, 4 keys in vt_perm order (logical chunk 4 (g / 2) + 2 half + g % 2)
    auto val_frag = [&](const unsigned char *tile, int d, int g) -> u32x4 {
        const int cl = DT == F32 ? 4 * (g >> 1) + 2 * half + (g & 1) : 2 * g + half;
        u32x4 x = *reinterpret_cast<const u32x4 *>(tile + vbase + d * 32 * C::CV * 16 + ((cl * 16) ^ vkey));
        if constexpr (DH < 32)
            if ((lane & 31) >= DH) x = u32x4{0u, 0u, 0u, 0u};
        return x;
    };

    // ---- running state
    f32x16 o[C::NDBP], uq[C::NDBP], uk[C::NDBP], wv[C::NDBP];
#pragma unroll
    for (int d = 0; d < C::NDBP; ++d)
#pragma unroll
        for (int e = 0; e < 16; ++e) { o[d][e] = 0.f; uq[d][e] = 0.f; uk[d][e] = 0.f; wv[d][e] = 0.f; }
    float m_run = -INFINITY;                           // reference maximum (log2 units)
    float l_run = 0.f, mq_run = 0.f, mk_run = 0.f, cqq = 0.f, ckk = 0.f, cqk = 0.f;

#pragma unroll
    for (int t = 0; t < C::NS - 1; ++t) issue(t);
    for (int j = 0; j < nblk; ++j) {
        // block j has landed for this wave (the blocks issued after it may be pending), then for every
        // wave; every wave is done with block j - 1, whose slot takes block j + NS - 1
        wait_lgkm0();
        wait_vm_groups<C::PW, C::NS - 2>(min(C::NS - 2, nblk - 1 - j));
        raw_barrier();
        issue(j + C::NS - 1);
        if (j > jlast) continue;                       // keys above every query of the wave
        const unsigned char *st = smem + (j % C::NS) * C::STAGE;
        const int kb = 32 * j;

        // scores: lane -> query, register e -> key kb + 8 (e / 4) + 4 half + e % 4
        f32x16 s, sq, sk;
#pragma unroll
        for (int e = 0; e < 16; ++e) { s[e] = 0.f; sq[e] = 0.f; sk[e] = 0.f; }
#pragma unroll
        for (int l = 0; l < C::KL; ++l) {
            opnd kf[KPL], kdf[KPL];
            key_frag(st, l, kf);
            key_frag(st + C::KB, l, kdf);
#pragma unroll
            for (int t = 0; t < KPL; ++t) {
                const int kc = l * KPL + t;
                s = MM::mma(kf[t], qf[kc], s);
                sq = MM::mma(kf[t], qdf[kc], sq);
                sk = MM::mma(kdf[t], qf[kc], sk);
            }
        }
        bool live[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) live[e] = j < jlast || kb + 8 * (e >> 2) + 4 * half + (e & 3) <= lim;
        float mb = -INFINITY;
#pragma unroll
        for (int e = 0; e < 16; ++e) mb = live[e] ? fmaxf(mb, s[e]) : mb;
        mb = halves_max(mb) * scale_log2;
        if (__any(mb > m_run)) {
            const float m_new = fmaxf(m_run, mb);
            const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);   // 0 on the first block
#pragma unroll
            for (int d = 0; d < C::NDBP; ++d)
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    o[d][e] *= alpha;
                    uq[d][e] *= alpha;
                    uk[d][e] *= alpha;
                    wv[d][e] *= alpha;
                }
            l_run *= alpha; mq_run *= alpha; mk_run *= alpha; cqq *= alpha; ckk *= alpha; cqk *= alpha;
            m_run = m_new;
        }
        float p[16], pq[16], pk[16];
        uint32_t bp2[8], bq2[8], bk2[8];                 // 16-bit: the same, rounded and packed in pairs
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const float tq = live[e] ? sq[e] * inv_sqrt : 0.f;      // logit tangents (natural units)
            const float tk = live[e] ? sk[e] * inv_sqrt : 0.f;
            p[e] = live[e] ? __builtin_amdgcn_exp2f(__builtin_fmaf(s[e], scale_log2, -m_run)) : 0.f;
            pq[e] = p[e] * tq;
            pk[e] = p[e] * tk;
            l_run += p[e];
            mq_run += pq[e];
            mk_run += pk[e];
            cqq += pq[e] * tq;
            ckk += pk[e] * tk;
            cqk += pq[e] * tk;
            if constexpr (DT != F32)
                if (e & 1) {
                    bp2[e >> 1] = pack2<DT>(p[e - 1], p[e]);
                    bq2[e >> 1] = pack2<DT>(pq[e - 1], pq[e]);
                    bk2[e >> 1] = pack2<DT>(pk[e - 1], pk[e]);
                }
        }
        // value products for this pass's row blocks: k = the block's 32 keys
        const unsigned char *sv = st + 2 * C::KB, *svd = sv + C::VB;
#pragma unroll
        for (int d = 0; d < C::NDBP; ++d) {
#pragma unroll
            for (int g = 0; g < C::VG; ++g) {
                const int db = dpass * C::NDBP + d;
                const u32x4 vf = val_frag(sv, db, g), vdf = val_frag(svd, db, g);
                if constexpr (DT == F32) {
#pragma unroll
                    for (int t = 0; t < 4; ++t) {
                        const int kk = 4 * g + t;
                        const uint32_t ve = vf[t], vde = vdf[t];
                        const float vv = __builtin_bit_cast(float, ve), vdv = __builtin_bit_cast(float, vde);
                        o[d] = MM::mma(vv, p[kk], o[d]);
                        uq[d] = MM::mma(vv, pq[kk], uq[d]);
                        uk[d] = MM::mma(vv, pk[kk], uk[d]);
                        wv[d] = MM::mma(vdv, p[kk], wv[d]);
                    }
                } else {
                    const opnd bp = __builtin_bit_cast(opnd, u32x4{bp2[4 * g], bp2[4 * g + 1], bp2[4 * g + 2], bp2[4 * g + 3]});
                    const opnd bq = __builtin_bit_cast(opnd, u32x4{bq2[4 * g], bq2[4 * g + 1], bq2[4 * g + 2], bq2[4 * g + 3]});
                    const opnd bk = __builtin_bit_cast(opnd, u32x4{bk2[4 * g], bk2[4 * g + 1], bk2[4 * g + 2], bk2[4 * g + 3]});
                    const opnd av = __builtin_bit_cast(opnd, vf), avd = __builtin_bit_cast(opnd, vdf);
                    o[d] = MM::mma(av, bp, o[d]);
                    uq[d] = MM::mma(av, bq, uq[d]);
                    uk[d] = MM::mma(av, bk, uk[d]);
                    wv[d] = MM::mma(avd, bp, wv[d]);
                }
            }
        }
    }
    wait_vmcnt<0>();

    // ---- epilogue: the unit tangents of the output and their dot products per query row
    l_run = halves_sum(l_run);
    mq_run = halves_sum(mq_run);
    mk_run = halves_sum(mk_run);
    cqq = halves_sum(cqq);
    ckk = halves_sum(ckk);
    cqk = halves_sum(cqk);
    if (q0 >= T) return;
    const bool valid = qrow < T;
    const float inv_l = valid ? 1.f / l_run : 0.f;
    const float mq = mq_run * inv_l, mk = mk_run * inv_l;
    float e6[6] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int d = 0; d < C::NDBP; ++d)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const float ah = o[d][e] * inv_l;
            const float aq = uq[d][e] * inv_l - mq * ah;
            const float ak = uk[d][e] * inv_l - mk * ah;
            const float av = wv[d][e] * inv_l;
            e6[0] = __builtin_fmaf(aq, aq, e6[0]);
            e6[1] = __builtin_fmaf(ak, ak, e6[1]);
            e6[2] = __builtin_fmaf(av, av, e6[2]);
            e6[3] = __builtin_fmaf(aq, ak, e6[3]);
            e6[4] = __builtin_fmaf(aq, av, e6[4]);
            e6[5] = __builtin_fmaf(ak, av, e6[5]);
        }
    double r[kJvpParts];
#pragma unroll
    for (int i = 0; i < 6; ++i) r[i] = valid ? (double)e6[i] : 0.0;   // each half holds half the columns
    // the Fisher-information terms are per row: counted once, on the lower half of the first pass
    const bool once = valid && half == 0 && dpass == 0;
    r[6] = once ? (double)(cqq * inv_l - mq * mq) : 0.0;
    r[7] = once ? (double)(ckk * inv_l - mk * mk) : 0.0;
    r[8] = once ? (double)(cqk * inv_l - mq * mk) : 0.0;
    const int nq32 = (T + 31) / 32;
    double *pp = a.partials + ((((int64_t)dpass * a.batch + b) * Hq + h) * nq32 + q0 / 32) * kJvpParts;
#pragma unroll
    for (int i = 0; i < kJvpParts; ++i) {
        const double t = wave_sum_f64(r[i]);
        if (lane == 0) pp[i] = t;
    }
}

// Sum of the [n][9] partials in a fixed order, in two stages: block c of stage 1 sums the
// contiguous chunk [c n / 256, (c + 1) n / 256) (thread t takes its entries t, t + 256, ... in
// ascending order, then a fixed tree over the threads) into chunk[c][9]; stage 2 sums the 256
// chunks the same way into parts[9].
constexpr int kJvpChunks = 256;
__global__ __launch_bounds__(256) void jvp_reduce_kernel(const double *__restrict__ partials, int64_t n,
                                                         double *__restrict__ out) {
    __shared__ double red[256][kJvpParts];
    const int t = threadIdx.x;
    const int64_t lo = (int64_t)blockIdx.x * n / gridDim.x, hi = (int64_t)(blockIdx.x + 1) * n / gridDim.x;
    double acc[kJvpParts];
#pragma unroll
    for (int i = 0; i < kJvpParts; ++i) acc[i] = 0.0;
    for (int64_t r = lo + t; r < hi; r += 256)
#pragma unroll
        for (int i = 0; i < kJvpParts; ++i) acc[i] += partials[r * kJvpParts + i];
#pragma unroll
    for (int i = 0; i < kJvpParts; ++i) red[t][i] = acc[i];
    __syncthreads();
    for (int s = 128; s >= 1; s >>= 1) {
        if (t < s)
#pragma unroll
            for (int i = 0; i < kJvpParts; ++i) red[t][i] += red[t + s][i];
        __syncthreads();
    }
    if (t < kJvpParts) out[(int64_t)blockIdx.x * kJvpParts + t] = red[0][t];
}

// The forms of eq. gn's H = 2 J_A^T J_A + lambda J_Q^T I(P) J_Q from the nine sums:
//   t_Q = 2 <aQ, aQ + aK + aV> + lambda (zQ.I.zQ + zQ.I.zK),  t_K alike,  t_V = 2 <aV, aQ + aK + aV>,
//   pooled = t_Q + t_K + t_V,  h_QQ = 2 <aQ,aQ> + lambda zQ.I.zQ,  h_KK alike,  h_VV = 2 <aV,aV>.
__global__ void curv_forms_kernel(const double *__restrict__ e, double lambda, double *__restrict__ out) {
    if (threadIdx.x != 0) return;
    const double qq = e[0], kk = e[1], vv = e[2], qk = e[3], qv = e[4], kv = e[5];
    const double fqq = e[6], fkk = e[7], fqk = e[8];
    const double tq = 2.0 * (qq + qk + qv) + lambda * (fqq + fqk);
    const double tk = 2.0 * (qk + kk + kv) + lambda * (fqk + fkk);
    const double tv = 2.0 * (qv + kv + vv);
    out[0] = tq;
    out[1] = tk;
    out[2] = tv;
    out[3] = tq + tk + tv;
    out[4] = 2.0 * qq + lambda * fqq;
    out[5] = 2.0 * kk + lambda * fkk;
    out[6] = 2.0 * vv;
}

template <int DT, int DH>
hipError_t run_jvp(const JvpArgs &a, hipStream_t st, int64_t *n_partials) {
    typedef JvpCfg<DT, DH> C;
    *n_partials = (int64_t)C::NPASS * a.batch * a.n_heads * ((a.seq_len + 31) / 32);
    // buffer offsets from a sequence's rows (keys) or a key/value head's rows (values) are 32-bit
    if ((int64_t)(a.seq_len + 32) * a.ld * C::ES >= (1ll << 31) || (int64_t)DH * a.ldv * C::ES >= (1ll << 31))
        return hipErrorInvalidValue;
    const int G = a.n_heads / a.n_kv_heads;
    const int hpw = G % 4 == 0 ? 4 : G;                // query heads per workgroup tile (1, 2 or 4)
    const int QT = 4 * 32 / hpw;
    const int nqt = (a.seq_len + QT - 1) / QT;
    const int n_ht = a.n_heads / hpw;
    const float scale_log2 = 1.4426950408889634f / sqrtf((float)DH);
    const float inv_sqrt = 1.f / sqrtf((float)DH);
    const size_t lds = (size_t)C::NS * C::STAGE;
    hipError_t e = hipFuncSetAttribute((const void *)attn_jvp_kernel<DT, DH>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    for (int pass = 0; pass < C::NPASS; ++pass) {
        attn_jvp_kernel<DT, DH><<<dim3(nqt * n_ht * a.batch), dim3(256), lds, st>>>(a, scale_log2, inv_sqrt, hpw,
                                                                                    nqt, n_ht, pass);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

template <int DT>
hipError_t jvp_dh(const JvpArgs &a, hipStream_t st, int64_t *n_partials) {
    switch (a.head_dim) {
    case 16: return run_jvp<DT, 16>(a, st, n_partials);
    case 64: return run_jvp<DT, 64>(a, st, n_partials);
    default: return run_jvp<DT, 128>(a, st, n_partials);
    }
}

// w_out[i] = dtype(probe[i]) (+-1, exact in every dtype): the probe as a projection operand
template <int DT>
__global__ __launch_bounds__(256) void probe_to_dtype_kernel(const int8_t *__restrict__ probe, int64_t n,
                                                             void *__restrict__ w_out) {
    typedef typename Mma<DT>::elem elem;
    elem *dst = static_cast<elem *>(w_out);
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        dst[i] = from_f32<DT>((float)probe[i]);
}

}  // namespace

// the largest pass count of any configuration (fp32 at head_dim 128)
constexpr int kMaxJvpPasses = JvpCfg<F32, 128>::NPASS;

size_t jvp_partials_bytes(int batch, int seq_len, int n_heads) {
    return (size_t)kMaxJvpPasses * batch * n_heads * ((seq_len + 31) / 32) * kJvpParts * sizeof(double);
}

hipError_t launch_attn_jvp(int dtype, const JvpArgs &a, hipStream_t st, int64_t *n_partials) {
    *n_partials = 0;
    if (a.batch <= 0 || a.seq_len <= 0) return hipSuccess;
    switch (dtype) {
    case F32: return jvp_dh<F32>(a, st, n_partials);
    case F16: return jvp_dh<F16>(a, st, n_partials);
    default: return jvp_dh<BF16>(a, st, n_partials);
    }
}

size_t curv_parts_bytes() { return (size_t)(kJvpChunks + 1) * kJvpParts * sizeof(double); }

hipError_t launch_curv_forms(const double *partials, int64_t n, double *parts, double lambda, double *out,
                             hipStream_t st) {
    double *chunks = parts + kJvpParts;
    jvp_reduce_kernel<<<kJvpChunks, 256, 0, st>>>(partials, n, chunks);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    jvp_reduce_kernel<<<1, 256, 0, st>>>(chunks, kJvpChunks, parts);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    curv_forms_kernel<<<1, 64, 0, st>>>(parts, lambda, out);
    return hipGetLastError();
}

hipError_t launch_probe_to_dtype(int dtype, const int8_t *probe, int64_t n, void *w_out, hipStream_t st) {
    const int blocks = (int)std::min<int64_t>((n + 255) / 256, 8192);
    switch (dtype) {
    case F32: probe_to_dtype_kernel<F32><<<blocks, 256, 0, st>>>(probe, n, w_out); break;
    case F16: probe_to_dtype_kernel<F16><<<blocks, 256, 0, st>>>(probe, n, w_out); break;
    default: probe_to_dtype_kernel<BF16><<<blocks, 256, 0, st>>>(probe, n, w_out); break;
    }
    return hipGetLastError();
}

}  // namespace jab
