// attn_kl.hip -- the KL attention-map term of the joint loss on the matrix cores.
//
// Paper: Method, eq. joint_loss: lambda_KL * D_KL(P || Q(w)), P the causal softmax map of the
// float block (the teacher), Q(w) that of the quantized block; the reduction is the Appendix's
// "batchmean" (summed over every map entry, divided by the batch size B; the division happens in
// the final reduction).
//
// Per query row i of a head:  D_KL(P_i || Q_i) = sum_j P_ij (log P_ij - log Q_ij).  With base-2
// log-sum-exps L_t (the teacher's, cached by its forward pass) and L_s (the student's, built in
// this pass), raw scores s = q . k and c = log2(e) / sqrt(d_head):
//   log P_ij = ln2 (c st_ij - L_t),  log Q_ij = ln2 (c ss_ij - L_s),  P_ij = 2^(c st_ij - L_t),
//   D_KL = ln2 [ c sum_j P_ij (st_ij - ss_ij) + (L_s - L_t) sum_j P_ij ],
// so one pass over the keys suffices: the running student maximum and row sum give L_s at the
// end, and the two P-weighted sums need only the cached L_t.  sum_j P_ij is 1 when L_t belongs
// to the cached teacher projection; its deviation is reported (second partial).
//
// Design: a wave owns one (sequence, query head, tile of 32 queries); the teacher's and the
// student's queries stay in registers as B operands of S^T = K Q^T (v_mfma_f32_32x32x16 for the
// 16-bit dtypes, 32x32x2 for fp32), so a lane holds 16 keys of one query.  Key fragments come
// straight from global memory (the waves of a workgroup are four heads of the same tile and
// mostly share a key/value head, so the L1 serves the repeats), double-buffered one key block
// ahead.  No LDS and no barriers: any GQA ratio, any dtype.  Per (sequence, head, query tile)
// the wave writes (sum of KL rows, sum of (sum_j P_ij - 1)) in fp64, the layout of the loss
// partials, for the same fixed-order reductions.
#include "attn_fwd_impl.h"                        // rescale_log2, sum16 (the attention kernels' rule)

namespace jab {
namespace {

// One key block of one query row (a lane's 16 keys, register e = key 8 (e / 4) + 4 half + e % 4 of
// the block, valid when that offset is <= lim; MASK false: every key valid).  The student's
// log-sum-exp follows the attention kernels' rule exactly: the reference starts at block 0's
// maximum and moves only when a block's maximum overshoots it by more than rescale_log2, each
// block adds the lane's 16 probabilities in the order of sum16, and the two lanes of a query add
// at the end.  A student equal to the teacher therefore reproduces the cached teacher value bit
// for bit, and its KL is exactly 0.  acc_d += sum P (st - ss), acc_p += sum P (teacher map).
template <int DT, bool MASK>
__device__ inline void kl_block(f32x16 &ss, const f32x16 &st, int lim, float scale_log2, float lse_t, float &m_s,
                                float &l_s, float &acc_d, float &acc_p) {
    float bm = -INFINITY;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
        if (MASK && 8 * (e >> 2) + (e & 3) > lim) ss[e] = -INFINITY;
        bm = fmaxf(bm, ss[e]);
    }
    const float ms = halves_max(bm) * scale_log2;
    if (ms > m_s + rescale_log2<DT>()) {               // per lane; both lanes of a query agree
        l_s *= __builtin_amdgcn_exp2f(m_s - ms);
        m_s = ms;
    }
    float p[16];
    float ad = 0.f, ap = 0.f;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
        p[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(ss[e], scale_log2, -m_s));
        const bool in = !MASK || 8 * (e >> 2) + (e & 3) <= lim;
        const float pt = in ? __builtin_amdgcn_exp2f(__builtin_fmaf(st[e], scale_log2, -lse_t)) : 0.f;
        ad = __builtin_fmaf(pt, in ? st[e] - ss[e] : 0.f, ad);
        ap += pt;
    }
    l_s += sum16(p);
    acc_d += ad;
    acc_p += ap;
}

// The end of a query row: the halves of its keys, L_s, the row's KL (nats), and the wave's
// partials (one lane per query; rows past the sequence excluded).
__device__ inline void kl_finish(float m_s, float l_s, float acc_d, float acc_p, float lse_t, float scale_log2,
                                 bool valid, double *pp) {
    l_s = halves_sum(l_s);
    acc_d = halves_sum(acc_d);
    acc_p = halves_sum(acc_p);
    const float lse_s = m_s + __builtin_amdgcn_logf(l_s);
    const bool mine = (threadIdx.x & 32) == 0 && valid;
    const float kl = 0.6931471805599453f * (scale_log2 * acc_d + (lse_s - lse_t) * acc_p);
    const double tkl = wave_sum_f64(mine ? (double)kl : 0.0);
    const double tdef = wave_sum_f64(mine ? (double)acc_p - 1.0 : 0.0);
    if ((threadIdx.x & 63) == 0) {
        pp[0] = tkl;
        pp[1] = tdef;
    }
}

template <int DT, int DH>
__global__ __launch_bounds__(256) void attn_kl_kernel(KlArgs a, float scale_log2, int nqt, int n_waves) {
    typedef Mma<DT> MM;
    typedef typename MM::operand opnd;
    typedef typename MM::elem elem;
    constexpr int VEC = MM::VEC;              // operand elements per lane
    constexpr int NK = DH / MM::K;            // MFMA k-steps of one 32 x 32 score tile
    static_assert(DH % MM::K == 0, "head_dim");

    const int lane = threadIdx.x & 63, half = lane >> 5, l32 = lane & 31;
    const int gw = blockIdx.x * 4 + (int)(threadIdx.x >> 6);
    if (gw >= n_waves) return;
    const int T = a.seq_len, Hq = a.n_heads;
    const int h = gw % Hq;
    const int qt = nqt - 1 - (gw / Hq) % nqt;          // longest tiles first
    const int b = gw / (Hq * nqt);
    const int kvh = h / (Hq / a.n_kv_heads);
    const int q0 = qt * 32, qrow = q0 + l32;
    const int64_t row0 = (int64_t)b * T;
    const elem *qs = static_cast<const elem *>(a.qs), *qt_ = static_cast<const elem *>(a.qt);

    auto load_op = [](const elem *p) -> opnd {
        if constexpr (VEC == 1) return *p;
        else return __builtin_bit_cast(opnd, *reinterpret_cast<const u32x4 *>(p));
    };

    // queries (clamped rows past the sequence are never counted).  Operand element order per
    // k-step: s_k, the attention kernels' (for fp32 the two half-waves take the two halves of
    // head_dim), so the scores here equal theirs bit for bit.
    opnd qfs[NK], qft[NK];
    {
        const int64_t r = (row0 + min(qrow, T - 1)) * a.ld + h * DH;
#pragma unroll
        for (int kc = 0; kc < NK; ++kc) {
            qfs[kc] = load_op(qs + r + s_k<DT, DH>(kc, half));
            qft[kc] = load_op(qt_ + r + s_k<DT, DH>(kc, half));
        }
    }
    const float lse_t = a.lse_t[((int64_t)b * Hq + h) * T + min(qrow, T - 1)];

    // key fragments of block kb: lane row l32 (key kb*32 + l32, clamped), elements s_k
    const int64_t kcol = (int64_t)Hq * DH + kvh * DH;
    auto load_keys = [&](int kb, opnd (&ks)[NK], opnd (&kt)[NK]) {
        const int64_t r = (row0 + min(kb * 32 + l32, T - 1)) * a.ld + kcol;
#pragma unroll
        for (int kc = 0; kc < NK; ++kc) {
            ks[kc] = load_op(qs + r + s_k<DT, DH>(kc, half));
            kt[kc] = load_op(qt_ + r + s_k<DT, DH>(kc, half));
        }
    };

    float m_s = -INFINITY, l_s = 0.f;                  // student: reference (log2 units), lane's sum
    float acc_d = 0.f, acc_p = 0.f;                    // lane's sum P (st - ss), sum P
    auto block = [&](int kb, const opnd (&ks)[NK], const opnd (&kt)[NK]) {
        f32x16 ss = {}, st = {};
#pragma unroll
        for (int kc = 0; kc < NK; ++kc) {
            ss = MM::mma(ks[kc], qfs[kc], ss);
            st = MM::mma(kt[kc], qft[kc], st);
        }
        kl_block<DT, true>(ss, st, qrow - kb * 32 - 4 * half, scale_log2, lse_t, m_s, l_s, acc_d, acc_p);
    };

    opnd ksa[NK], kta[NK], ksb[NK], ktb[NK];
    load_keys(0, ksa, kta);
    int kb = 0;
    for (; kb + 1 <= qt; kb += 2) {                    // blocks kb, kb + 1 (both <= qt)
        load_keys(kb + 1, ksb, ktb);
        block(kb, ksa, kta);
        if (kb + 2 <= qt) load_keys(kb + 2, ksa, kta);
        block(kb + 1, ksb, ktb);
    }
    if (kb == qt) block(kb, ksa, kta);

    kl_finish(m_s, l_s, acc_d, acc_p, lse_t, scale_log2, qrow < T, a.partials + (((int64_t)b * Hq + h) * nqt + qt) * 2);
}

// The common configuration (16-bit, head_dim 64 or 128, query heads per key/value head a multiple
// of 4, T a multiple of 32): a workgroup of 4 waves is 4 query heads of one key/value group over
// the same 32 queries, and the student's and the teacher's key blocks stream into a ring of four
// LDS slots (buffer_load ... lds, a block's loads shared by the four waves) three blocks ahead of
// use.  Block j: its 2 x NKC score MFMAs on fragments read during block j - 1; one barrier (block
// j + 1 has landed, and every wave has read block j's slot, which is then refilled with block
// j + 4); the fragment reads of block j + 1; then block j's vector work, under which those reads
// land.  Only the diagonal block is masked.  Same per-row arithmetic as attn_kl_kernel.
template <int DT, int DH>
__global__ __launch_bounds__(256, 2) void attn_kl_ring_kernel(KlArgs a, float scale_log2, int nqt, int n_ht) {
    typedef Mma<DT> MM;
    typedef typename MM::operand opnd;
    typedef typename MM::elem elem;
    static_assert(DT != F32 && (DH == 64 || DH == 128), "ring configuration");
    constexpr int NKC = DH / 16;                       // k-steps of a score tile
    constexpr int CK = DH * 2 / 16;                    // 16-byte chunks per key row
    constexpr int K_BYTES = 32 * CK * 16;              // one key block of one projection
    constexpr int BLK = 2 * K_BYTES;                   // student keys, then teacher keys
    constexpr int NS = 4;                              // ring slots
    constexpr int PK = K_BYTES / 1024 / 4;             // DMA instructions per wave per projection
    constexpr int PW = 2 * PK;
    extern __shared__ __align__(16) unsigned char smem[];

    const int T = a.seq_len, Hq = a.n_heads;
    const int nwg = gridDim.x;
    int lin = blockIdx.x;
    if ((nwg & 7) == 0) lin = (lin & 7) * (nwg >> 3) + (lin >> 3);
    const int qt = nqt - 1 - lin % nqt;                // longest tiles first
    const int ht = (lin / nqt) % n_ht;
    const int b = lin / (nqt * n_ht);
    const int lane = threadIdx.x & 63, half = lane >> 5, l32 = lane & 31;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int h = ht * 4 + wave;
    const int kvh = (ht * 4) / (Hq / a.n_kv_heads);
    const int q0 = qt * 32, qrow = q0 + l32;           // T is a multiple of 32: every query is valid
    const int jlast = qt;
    const int64_t row0 = (int64_t)b * T;
    const elem *qs = static_cast<const elem *>(a.qs), *qt_ = static_cast<const elem *>(a.qt);

    opnd qfs[NKC], qft[NKC];
    {
        const int64_t r = (row0 + qrow) * a.ld + h * DH;
#pragma unroll
        for (int kc = 0; kc < NKC; ++kc) {
            qfs[kc] = __builtin_bit_cast(opnd, *reinterpret_cast<const u32x4 *>(qs + r + s_k<DT, DH>(kc, half)));
            qft[kc] = __builtin_bit_cast(opnd, *reinterpret_cast<const u32x4 *>(qt_ + r + s_k<DT, DH>(kc, half)));
        }
    }
    const float lse_t = a.lse_t[((int64_t)b * Hq + h) * T + qrow];

    // DMA: load i < PK of this wave fills key-tile chunks 64 (wave + 4 i) + lane: key row p / CK,
    // physical chunk p % CK holding logical chunk (p % CK) ^ swz_key(row) (the attention kernels'
    // key tile); loads PK .. PW - 1 the teacher's tile likewise.  Blocks past the tile re-load its
    // last block into a slot that is never read.
    const int64_t kcol = (int64_t)Hq * DH + kvh * DH;
    const i32x4 rss = buffer_rsrc(qs + row0 * a.ld + kcol);
    const i32x4 rst = buffer_rsrc(qt_ + row0 * a.ld + kcol);
    uint32_t dvoff[PK];
#pragma unroll
    for (int i = 0; i < PK; ++i) {
        const int p = (wave + 4 * i) * 64 + lane, r = p / CK, c = (p % CK) ^ swz_key<CK>(r);
        dvoff[i] = (uint32_t)(r * a.ld * 2 + c * 16);
    }
    const int kstride = a.ld * 2 * 32;
    auto issue = [&](int j, unsigned char *slot) {
        const int jb = min(j, jlast);
#pragma unroll
        for (int i = 0; i < PK; ++i) {
            buffer_dma16(rss, dvoff[i], jb * kstride, slot + (wave + 4 * i) * 1024);
            buffer_dma16(rst, dvoff[i], jb * kstride, slot + K_BYTES + (wave + 4 * i) * 1024);
        }
    };
    uint32_t koff[NKC];
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc)
        koff[kc] = (uint32_t)(l32 * CK * 16 + (((2 * kc + half) ^ swz_key<CK>(l32)) * 16));
    opnd kfs[NKC], kft[NKC];
    auto rd = [&](const unsigned char *slot) {
#pragma unroll
        for (int kc = 0; kc < NKC; ++kc) {
            kfs[kc] = __builtin_bit_cast(opnd, *reinterpret_cast<const u32x4 *>(slot + koff[kc]));
            kft[kc] = __builtin_bit_cast(opnd, *reinterpret_cast<const u32x4 *>(slot + K_BYTES + koff[kc]));
        }
    };

    // prologue: blocks 0 .. 3 in flight, block 0 landed and read, its scores computed
#pragma unroll
    for (int t = 0; t < NS; ++t) issue(t, smem + t * BLK);
    wait_vmcnt<(NS - 1) * PW>();
    raw_barrier();
    rd(smem);
    f32x16 sA = {}, tA = {}, sB, tB;
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc) {
        sA = MM::mma(kfs[kc], qfs[kc], sA);
        tA = MM::mma(kft[kc], qft[kc], tA);
    }

    float m_s = -INFINITY, l_s = 0.f, acc_d = 0.f, acc_p = 0.f;
    // Block j (its scores in cs, ct): one barrier (block j + 1 landed; every wave has read block
    // j's slot, which is refilled with block j + NS), the fragment reads of block j + 1, then NKC
    // fenced slots, each one pair of block j + 1's score MFMAs (NEXT) with a share of block j's
    // vector work: slot 0 also takes the block maximum and the reference rule.  The arithmetic
    // per row is kl_block's, in the same order.
    auto step = [&](int j, f32x16 &cs, const f32x16 &ct, f32x16 &ns, f32x16 &nt, auto next_c, auto mask_c) {
        constexpr bool NEXT = decltype(next_c)::value;
        constexpr bool MASK = decltype(mask_c)::value;
        wait_lgkm0();
        wait_vmcnt<(NS - 2) * PW>();
        raw_barrier();
        issue(j + NS, smem + (j & (NS - 1)) * BLK);
        if constexpr (NEXT) rd(smem + ((j + 1) & (NS - 1)) * BLK);
        const int lim = qrow - j * 32 - 4 * half;
        float bm = -INFINITY;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            if (MASK && 8 * (e >> 2) + (e & 3) > lim) cs[e] = -INFINITY;
            bm = fmaxf(bm, cs[e]);
        }
        const float ms = halves_max(bm) * scale_log2;
        if (ms > m_s + rescale_log2<DT>()) {
            l_s *= __builtin_amdgcn_exp2f(m_s - ms);
            m_s = ms;
        }
        float p[16];
        float ad = 0.f, ap = 0.f;
        SCHED_FENCE();
#pragma unroll
        for (int i = 0; i < NKC; ++i) {
            if constexpr (NEXT) {
                ns = MM::mma(kfs[i], qfs[i], i == 0 ? f32x16{} : ns);
                nt = MM::mma(kft[i], qft[i], i == 0 ? f32x16{} : nt);
            }
#pragma unroll
            for (int e = i * 16 / NKC; e < (i + 1) * 16 / NKC; ++e) {
                p[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(cs[e], scale_log2, -m_s));
                const bool in = !MASK || 8 * (e >> 2) + (e & 3) <= lim;
                const float pt = in ? __builtin_amdgcn_exp2f(__builtin_fmaf(ct[e], scale_log2, -lse_t)) : 0.f;
                ad = __builtin_fmaf(pt, in ? ct[e] - cs[e] : 0.f, ad);
                ap += pt;
            }
            SCHED_FENCE();
        }
        l_s += sum16(p);
        acc_d += ad;
        acc_p += ap;
    };
    typedef std::integral_constant<bool, true> yes;
    typedef std::integral_constant<bool, false> no;
    int j = 0;
    for (; j + 2 <= jlast; j += 2) {                   // blocks j, j + 1 before the diagonal
        step(j, sA, tA, sB, tB, yes(), no());
        step(j + 1, sB, tB, sA, tA, yes(), no());
    }
    if (j < jlast) {                                   // block jlast - 1, then the diagonal
        step(j, sA, tA, sB, tB, yes(), no());
        step(j + 1, sB, tB, sA, tA, no(), yes());
    } else {
        step(j, sA, tA, sB, tB, no(), yes());
    }
    wait_vmcnt<0>();                                   // no DMA into LDS outlives the workgroup
    kl_finish(m_s, l_s, acc_d, acc_p, lse_t, scale_log2, true, a.partials + (((int64_t)b * Hq + h) * nqt + qt) * 2);
}

template <int DT, int DH>
hipError_t run_kl(const KlArgs &a, hipStream_t st) {
    const int nqt = (a.seq_len + 31) / 32;
    if constexpr (DT != F32 && (DH == 64 || DH == 128)) {
        if ((a.n_heads / a.n_kv_heads) % 4 == 0 && a.seq_len % 32 == 0) {
            constexpr int LDS = 4 * 2 * 32 * DH * 2;
            hipError_t e = hipFuncSetAttribute((const void *)attn_kl_ring_kernel<DT, DH>,
                                               hipFuncAttributeMaxDynamicSharedMemorySize, LDS);
            if (e != hipSuccess) return e;
            const int n_ht = a.n_heads / 4;
            attn_kl_ring_kernel<DT, DH><<<dim3(nqt * n_ht * a.batch), dim3(256), LDS, st>>>(
                a, 1.4426950408889634f / sqrtf((float)DH), nqt, n_ht);
            return hipGetLastError();
        }
    }
    const int64_t n_waves = (int64_t)a.batch * a.n_heads * nqt;
    const float scale_log2 = 1.4426950408889634f / sqrtf((float)DH);
    attn_kl_kernel<DT, DH><<<dim3((unsigned)((n_waves + 3) / 4)), dim3(256), 0, st>>>(a, scale_log2, nqt,
                                                                                     (int)n_waves);
    return hipGetLastError();
}

template <int DT>
hipError_t dispatch_kl(const KlArgs &a, hipStream_t st) {
    switch (a.head_dim) {
    case 16: return run_kl<DT, 16>(a, st);
    case 64: return run_kl<DT, 64>(a, st);
    case 128: return run_kl<DT, 128>(a, st);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_attn_kl(int dtype, const KlArgs &a, hipStream_t st) {
    if (a.batch <= 0 || a.seq_len <= 0) return hipSuccess;
    switch (dtype) {
    case F32: return dispatch_kl<F32>(a, st);
    case F16: return dispatch_kl<F16>(a, st);
    default: return dispatch_kl<BF16>(a, st);
    }
}

}  // namespace jab
