// attn_fwd_fast.h -- the causal GQA attention kernel for the common configuration: 16-bit
// dtype, head_dim 64 or 128, one value tensor, and a workgroup whose four waves are four query
// heads of one key/value group over the same 32 queries (included by attn_fwd.hip after
// attn_fwd_impl.h, whose helpers it uses).
//
// Paper: Method, "Layer-wise PTQ" (causal softmax attention) and eq. joint_loss (squared
// Frobenius distance to the teacher output); same arithmetic as attn_fwd_kernel.
//
// What differs from attn_fwd_kernel on this configuration:
//  * Key and transposed-value tiles arrive by buffer_load_dwordx4 ... lds: per-lane byte offsets
//    fixed for the whole kernel, the block's key offset in a scalar register, so a block's four
//    loads per wave cost no vector instructions, and the LDS counter stays ordered (each
//    fragment read is waited for individually).
//  * A ring of four key blocks, and the block loop runs in groups of four with the ring slot
//    of each block known at compile time: every LDS fragment read is a per-lane offset register
//    plus an immediate, and the two score buffers alternate without copies.  The blocks left
//    before the diagonal (at most three) and the two last blocks run one at a time with a
//    run-time slot.
//  * The row sums are fp32 sums of the probabilities (sum16, the same order as attn_fwd_kernel).
//  * With the loss epilogue, the refills of the last four key blocks of a tile (which would only
//    re-load the last block) bring the four waves' teacher tiles into the ring instead (one slot
//    per wave: 32 queries x head_dim fp32 is exactly one slot), so the epilogue reads the teacher
//    from LDS instead of waiting on memory at the end of the tile.
//  * A workgroup takes a pair of query tiles of one (sequence, head group): qt and nqt - 1 - qt,
//    nqt + 1 key blocks together for every pair, the longer first.  The second tile's queries and
//    first four key blocks are requested as soon as the first tile's epilogue has left the ring,
//    with no workgroup launch in between, and pairs of equal length keep the CUs' two workgroups
//    evenly loaded.  Pair ids are remapped so that one XCD (workgroup ids congruent mod 8) runs
//    all pairs of a (sequence, head group) and shares its keys and values through one L2.
//  * No per-block softmax bookkeeping: the reference maximum of a query is the exact maximum of its
//    first key block and stays there, so a block costs its exponentials and no maximum, no
//    compare and no branch (a branch on a vector compare waits for the wave's matrix-core work to
//    drain).  attn_fwd_kernel moves a query's reference when a block overshoots it by more than
//    R = rescale_log2 (2^64 for bf16, 2^15 for fp16); a query for which that never happens has
//    every probability at most 2^R, hence a row sum at most 2048 * 2^R.  After the pass, a query is
//    flagged when its row sum exceeds 2^R or an output is not finite: every unflagged query has
//    all probabilities at most 2^R and a finite result, exactly what the per-block rule gives it
//    without a move.  If a query of the workgroup is flagged, the workgroup repeats the tile
//    with the per-block rule for the flagged queries (threshold R) and none for the others, so
//    an unflagged query gets bitwise the same arithmetic in both passes: a query's result depends
//    only on its own scores, and equals attn_fwd_kernel's.
#pragma once

namespace jab {
namespace {

// S^T += K Q^T with the result in architectural registers, for the kernel whose output
// accumulators fill the 256 accumulation registers (the compiler would place this product's
// result in accumulation registers too and shuffle output blocks out and back every block).
// The compiler does not see the product inside the asm, so the hazards it would cover are covered
// here: two wait states before each product (a vector write of an operand), and 19 after the last
// product of a chain (LAST), inside the same asm, so that no instruction the compiler places after
// it (a copy of the result included) reads or writes the result too early.  Between the products
// of a chain the result passes from one asm to the next as a tied operand; the build checks the
// generated code for any other access within the window.
template <int DT>
__device__ inline f32x16 mma_v(typename Mma<DT>::operand a, typename Mma<DT>::operand b, f32x16 c, bool first,
                               bool last) {
    static_assert(DT == BF16 || DT == F16, "16-bit operands");
#define JAB_MMA_V(OP, C, TAIL, CON)                                                             \
    asm volatile("s_nop 1\n\t" OP " %0, %1, %2, " C TAIL : CON(d) : "v"(a), "v"(b))
#define JAB_DRAIN "\n\ts_nop 7\n\ts_nop 7\n\ts_nop 2"
#define JAB_MMA_V_ALL(OP)                                                                       \
    if (first && last) JAB_MMA_V(OP, "0", JAB_DRAIN, "=&v");                                    \
    else if (first) JAB_MMA_V(OP, "0", "", "=&v");                                              \
    else if (last) JAB_MMA_V(OP, "%0", JAB_DRAIN, "+v");                                        \
    else JAB_MMA_V(OP, "%0", "", "+v")
    f32x16 d = c;
    if constexpr (DT == BF16) {
        JAB_MMA_V_ALL("v_mfma_f32_32x32x16_bf16");
    } else {
        JAB_MMA_V_ALL("v_mfma_f32_32x32x16_f16");
    }
#undef JAB_MMA_V_ALL
#undef JAB_DRAIN
#undef JAB_MMA_V
    return d;
}

// NV value tensors share one score matrix (the sweep's triples that differ only in b_V): one value
// tensor, two workgroups per CU; two or four, one workgroup per CU (the output accumulators of a
// wave take NV * head_dim / 2 registers, and a ring slot holds the key tile and NV value tiles).
template <int DT, int DH, int NV = 1>
struct FastCfg {
    static constexpr int NKC = DH / 16;              // k-steps of S^T = K Q^T
    static constexpr int NDB = DH / 32;              // 32-row blocks of O^T
    static constexpr int CK = DH * 2 / 16;           // 16-byte chunks per key row
    static constexpr int K_BYTES = 32 * CK * 16;     // key tile of one block
    static constexpr int V_BYTES = DH * 4 * 16;      // transposed-value tile: DH rows of 32 keys
    static constexpr int BLK = K_BYTES + NV * V_BYTES;
    static constexpr int NS = 4;                     // ring slots
    static constexpr int KI = K_BYTES / 1024, VI = V_BYTES / 1024;   // DMA instructions per block and tile
    static constexpr int PK = KI / 4, PV = VI / 4;   // ... per wave
    static constexpr int PW = PK + NV * PV;
    static constexpr int NV_READ = NDB * 2;          // V^T fragment reads per value tensor and block
    static constexpr int MP1 = NDB * 2;              // MFMAs O^T += V^T P^T per value tensor
    static constexpr int MP = NV * MP1;              // MFMAs of phase O
    static constexpr int WPC = NV == 1 ? 2 : 1;      // workgroups per CU
    // Four value tensors at head_dim 128: their accumulators take the 256 accumulation registers,
    // so the V^T fragments are read as the products need them (VLEAD ahead) instead of all in
    // phase S, and a slot's key and value parts are refilled at different blocks (SV).
    static constexpr bool SV = NV == 4 && DH == 128;
    static constexpr int VLEAD = 4;
    // NV = 1: the pass flags follow the ring; NV > 1: they use slot 0, free when they are exchanged
    static constexpr size_t LDS_BYTES = (size_t)NS * BLK + (NV == 1 ? 16 : 0);
    static_assert(NV == 1 || NV == 2 || NV == 4, "one, two or four value tensors");
    static_assert(KI % 4 == 0 && VI % 4 == 0, "the four waves share a block's loads evenly");
    static_assert(NV > 1 || NS * BLK <= 65536, "immediate LDS offsets");
    static_assert(LDS_BYTES * WPC <= 160 * 1024, "LDS");
};

template <int DT, int DH, int NV>
__global__ __launch_bounds__(256, (FastCfg<DT, DH, NV>::WPC)) void attn_fast_kernel(AttnArgs a, float scale_log2,
                                                                                 int nqt, int n_ht) {
    typedef FastCfg<DT, DH, NV> C;
    typedef typename Mma<DT>::elem elem;
    typedef Mma<DT> MM;
    typedef typename MM::operand opnd;
    extern __shared__ __align__(16) unsigned char smem[];

    const int T = a.seq_len, Hq = a.n_heads;
    const int G = Hq / a.n_kv_heads;
    const int Tp = vt_pad(T);
    const int lane = threadIdx.x & 63, half = lane >> 5, l32 = lane & 31;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));

    // ---- the pair: pair p of group g = p / P (g = b n_ht + ht, P = ceil(nqt / 2)) holds query tiles
    // nqt - 1 - p % P (first) and p % P (second; none when they coincide, the middle tile of an odd
    // nqt).  With a grid that is a multiple of 8, XCD x (workgroup ids congruent to x mod 8) takes a
    // contiguous eighth of the pairs.
    const int nwg = gridDim.x;
    int pair = blockIdx.x;
    if ((nwg & 7) == 0) pair = (pair & 7) * (nwg >> 3) + (pair >> 3);
    const int P = (nqt + 1) >> 1;
    const int grp = pair / P, pp = pair - grp * P;
    const int n_tiles = pp == nqt - 1 - pp ? 1 : 2;

    // ---- DMA offsets (tile-invariant).  Load i < PK of this wave fills key-tile chunks 64 (wave +
    // 4 i) + lane: key row p / CK, physical chunk p % CK holding logical chunk (p % CK) ^
    // swz_key(row).  Load i >= PK fills transposed-value chunks the same way (DH rows of four
    // chunks).  Keys past the sequence read the rows that follow it (the next sequence, or the 32
    // rows of slack after the last): the causal mask removes them.  Blocks past the tile's range
    // re-load its last block into a slot that is never read.
    uint32_t dvoff[C::PK + C::PV];
#pragma unroll
    for (int i = 0; i < C::PK; ++i) {
        const int p = (wave + 4 * i) * 64 + lane, r = p / C::CK, c = (p % C::CK) ^ swz_key<C::CK>(r);
        dvoff[i] = (uint32_t)(r * a.ld * 2 + c * 16);
    }
#pragma unroll
    for (int i = 0; i < C::PV; ++i) {
        const int p = (wave + 4 * i) * 64 + lane, r = p / 4, c = (p % 4) ^ swz_key<4>(r);
        dvoff[C::PK + i] = (uint32_t)(r * (int)a.ldv * 2 + c * 16);
    }
    const int kstride = a.ld * 2 * 32;                 // bytes between key blocks of K

    // ---- a tile: its query tile, head group and sequence, and the buffer resources of its keys
    // and values (wave-uniform)
    struct Tile {
        int qt, ht, b;
        i32x4 rsk, rsv[NV];
    };
    auto make_tile = [&](int qt, int grp, Tile &t) {
        t.qt = qt;
        t.ht = grp % n_ht;
        t.b = grp / n_ht;
        const int kvh = (t.ht * 4) / G;                // G is a multiple of 4: one kv head per workgroup
        t.rsk = buffer_rsrc(static_cast<const elem *>(a.k) + (int64_t)t.b * T * a.ld + kvh * DH);
#pragma unroll
        for (int v = 0; v < NV; ++v)
            t.rsv[v] = buffer_rsrc(static_cast<const elem *>(a.v[v]) + (int64_t)kvh * DH * a.ldv + (int64_t)t.b * Tp);
    };
    // i-th of the wave's PW loads of block j of tile t (block index clamped to the tile's last)
    auto issue_t = [&](const Tile &t, int i, int j, unsigned char *slot) {
        const int jb = j < t.qt ? j : t.qt;
        if (i < C::PK) {
            buffer_dma16(t.rsk, dvoff[i], jb * kstride, slot + (wave + 4 * i) * 1024);
        } else {                                       // value tensor v, piece pc of its tile
            const int v = (i - C::PK) / C::PV, pc = (i - C::PK) % C::PV;
            buffer_dma16(t.rsv[v], dvoff[C::PK + pc], jb * 64, slot + C::K_BYTES + v * C::V_BYTES + (wave + 4 * pc) * 1024);
        }
    };
    auto issue_prologue = [&](const Tile &t) {        // the first NS blocks into slots 0 .. NS - 1
        if constexpr (C::SV) {
            // keys 0 and 1, values 0, then (keys u + 2, values u + 1) for u = 0, 1: the order in
            // which the block loop needs them (phase O of block m refills keys m + 4, values m + 3)
            auto kpart = [&](int u) {
#pragma unroll
                for (int i = 0; i < C::PK; ++i) issue_t(t, i, u, smem + u * C::BLK);
            };
            auto vpart = [&](int u) {
#pragma unroll
                for (int i = C::PK; i < C::PW; ++i) issue_t(t, i, u, smem + u * C::BLK);
            };
            kpart(0); kpart(1); vpart(0); kpart(2); vpart(1); kpart(3); vpart(2);
        } else {
#pragma unroll
            for (int u = 0; u < C::NS; ++u)
#pragma unroll
                for (int i = 0; i < C::PW; ++i) issue_t(t, i, u, smem + u * C::BLK);
        }
    };
    // this wave's queries of tile t as B operands of S^T = K Q^T
    opnd qf[C::NKC];
    auto load_q = [&](const Tile &t) {
        const int qrow = t.qt * 32 + l32;
        const elem *qp = static_cast<const elem *>(a.q) + ((int64_t)t.b * T + min(qrow, T - 1)) * a.ld +
                         (t.ht * 4 + wave) * DH;
#pragma unroll
        for (int kc = 0; kc < C::NKC; ++kc) {
            u32x4 v = *reinterpret_cast<const u32x4 *>(qp + kc * 16 + half * 8);
            if (qrow >= T) v = u32x4{0u, 0u, 0u, 0u};
            qf[kc] = __builtin_bit_cast(opnd, v);
        }
    };

    Tile cur;
    make_tile(nqt - 1 - pp, grp, cur);
    load_q(cur);
    issue_prologue(cur);
    constexpr int CR = DH / 4;                         // 16-byte chunks per teacher row
    const int ac = Hq * DH;
    const int nq32 = (T + 31) / 32;

  for (int n_tile = 0;; ++n_tile) {
    // ---- the current tile
    const int qt = cur.qt, ht = cur.ht, b = cur.b;
    const int h = ht * 4 + wave;
    const int q0 = qt * 32;
    const int jlast = qt;                              // blocks 0 .. qt; block qt is the diagonal
    const int64_t row0 = (int64_t)b * T;
    auto issue = [&](int i, int j, unsigned char *slot) { issue_t(cur, i, j, slot); };

    // ---- teacher prefetch (loss epilogue, tiles of at least four blocks).  Wave w's teacher tile is
    // 32 rows (queries) of CR 16-byte chunks; chunk c of row r sits at chunk c ^ (r & 15), so the
    // epilogue's reads (32 rows, one logical chunk) hit distinct banks.  Load i of a wave fills
    // chunks 64 (wave + 4 i) + lane of the slot; rows past the sequence read its last row.
    const bool pre_aref = NV == 1 && (a.mode & ATT_LOSS) && jlast >= 3;
    const i32x4 rsa = buffer_rsrc(a.a_ref + (row0 + q0) * ac + ht * 4 * DH);
    uint32_t aoff[NV == 1 ? C::PW : 1];
    if constexpr (NV == 1) {
#pragma unroll
        for (int i = 0; i < C::PW; ++i) {
            const int pch = (wave + 4 * i) * 64 + lane, r = pch / CR, c = (pch % CR) ^ (r & 15);
            aoff[i] = (uint32_t)(min(r, T - 1 - q0) * ac * 4 + c * 16);
        }
    }
    auto issue_aref = [&](int i, int wa, unsigned char *slot) {   // i-th load of wave wa's tile
        if constexpr (NV == 1) buffer_dma16(rsa, aoff[i], wa * DH * 4, slot + (wave + 4 * i) * 1024);
    };
    static_assert(NV > 1 || 32 * DH * 4 == C::BLK, "a teacher tile fills one slot");

    // ---- fragment reads: per-lane offsets, the slot added as an immediate
    uint32_t koff[C::NKC];                             // key fragment kc: row l32, chunk 2 kc + half
#pragma unroll
    for (int kc = 0; kc < C::NKC; ++kc)
        koff[kc] = (uint32_t)(l32 * C::CK * 16 + (((2 * kc + half) ^ swz_key<C::CK>(l32)) * 16));
    uint32_t voff[2];                                  // V^T fragment (d, g): row 32 d + l32, chunk 2 g + half
#pragma unroll
    for (int g = 0; g < 2; ++g)
        voff[g] = (uint32_t)(C::K_BYTES + l32 * 64 + (((2 * g + half) ^ swz_key<4>(l32)) * 16));
    opnd kf[C::NKC];
    // the V^T fragments of block j, every value tensor's, all read in phase S: the ring slot is
    // refilled during phase O, when another wave may already be issuing its share of the refill
    u32x4 vf[NV][C::NDB][2];
    auto rd_k = [&](const unsigned char *slot, int kc) {
        kf[kc] = __builtin_bit_cast(opnd, *reinterpret_cast<const u32x4 *>(slot + koff[kc]));
    };
    auto rd_v = [&](const unsigned char *slot, int t) {   // read t: value v = t / NV_READ, g, d of the rest
        const int v = t / C::NV_READ, r = t % C::NV_READ, g = r / C::NDB, d = r % C::NDB;
        vf[v][d][g] = *reinterpret_cast<const u32x4 *>(slot + voff[g] + v * C::V_BYTES + d * 32 * 64);
    };

    // ---- running state
    f32x16 o[NV][C::NDB];
    float l_run;                                       // the lane's partial row sum (its 16 keys of each block)
    float m_run;                                       // reference maximum (log2 units)
    float mx = 0.f;                                    // checked pass: maximum of the current block's raw scores
    f32x16 sa, sb;                                     // scores of two consecutive blocks
    uint32_t pk[8];                                    // probabilities of the current block, packed

    // score register e of a lane holds key kb + 8 (e / 4) + 4 half + e % 4 of query q0 + l32
    auto mask_el = [&](int kb, f32x16 &s, int e) {
        const int lim = q0 + l32 - kb - 4 * half;
        if (8 * (e >> 2) + (e & 3) > lim) s[e] = -INFINITY;
    };

    typedef std::integral_constant<bool, true> yes;
    typedef std::integral_constant<bool, false> no;
    typedef std::integral_constant<int, -1> dyn;

    // One pass over the tile's key blocks.  CHECKED: before each block's exponentials, move the
    // reference of the queries whose block maximum overshoots it by more than `thr` (rescale_log2
    // for flagged queries, infinity for the others).
    float thr = INFINITY;
    auto tile_pass = [&](auto checked_c, int pro) {
        constexpr bool CHECKED = decltype(checked_c)::value;
#pragma unroll
        for (int v = 0; v < NV; ++v)
#pragma unroll
            for (int d = 0; d < C::NDB; ++d)
#pragma unroll
                for (int e = 0; e < 16; ++e) o[v][d][e] = 0.f;
        l_run = 0.f;

        // prologue: the first NS blocks; blocks 0 and 1 landed for every wave.  pro 0: issue them
        // now; 1: issued last, after the query loads (stores in between only make the wait longer:
        // loads complete in order, so while a query load or block 0 or 1 is pending, so are the
        // last two blocks' loads)
        if (pro == 0) issue_prologue(cur);
        wait_vmcnt<(C::NS - 2) * C::PW>();
        raw_barrier();
#pragma unroll
        for (int kc = 0; kc < C::NKC; ++kc) rd_k(smem, kc);
#pragma unroll
        for (int kc = 0; kc < C::NKC; ++kc) sa = MM::mma(kf[kc], qf[kc], kc == 0 ? f32x16{} : sa);
        {
            if (jlast == 0)
#pragma unroll
                for (int e = 0; e < 16; ++e) mask_el(0, sa, e);
            float m = sa[0];
#pragma unroll
            for (int e = 1; e < 16; ++e) m = fmaxf(m, sa[e]);
            mx = halves_max(m);
            m_run = mx * scale_log2;                   // the reference: block 0's exact maximum
            if constexpr (!CHECKED) {
#pragma unroll
                for (int e = 0; e < 16; ++e) sa[e] = __builtin_fmaf(sa[e], scale_log2, -m_run);
            }
        }
#pragma unroll
        for (int kc = 0; kc < C::NKC; ++kc) rd_k(smem + C::BLK, kc);

        // ---- block j in two phases around one barrier; SLOT >= 0: ring slot j % NS known at
        // compile time.  Phase S (before the barrier): scores of block j + 1 (NEXT) on the matrix
        // cores, the exponentials of block j in their shadow, the V^T reads of block j.  Phase O
        // (after it): O^T += V^T P^T and the row sums for block j, the refill of block j's slot
        // with block j + NS, the mask (MASKN) of block j + 1 (and its maximum when CHECKED), the
        // key reads of block j + 2.
        auto fblock = [&](int j, auto slot_c, f32x16 &sc, f32x16 &sn, auto has_next, auto mask_next) {
            constexpr int SLOT = decltype(slot_c)::value;
            constexpr bool NEXT = decltype(has_next)::value;
            constexpr bool MASKN = decltype(mask_next)::value;
            const int s0 = SLOT >= 0 ? SLOT : (j & (C::NS - 1));
            unsigned char *st0 = smem + s0 * C::BLK;                                   // block j
            const unsigned char *st2 = smem + ((SLOT >= 0 ? SLOT + 2 : s0 + 2) & (C::NS - 1)) * C::BLK;   // j + 2

            if constexpr (CHECKED) {
                if (j > 0) {
                    const float ms = mx * scale_log2;
                    const bool move = ms > m_run + thr;
                    if (__any(move)) {
                        // only the lanes that overshoot move (the others multiply by exactly 1)
                        const float m_new = move ? ms : m_run;
                        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);

#pragma unroll
                        for (int v = 0; v < NV; ++v)
#pragma unroll
                            for (int d = 0; d < C::NDB; ++d)
#pragma unroll
                                for (int e = 0; e < 16; ++e) {
                                    if constexpr (C::SV) {
                                        // in place in the accumulation register (the compiler's
                                        // own form of this product stages the 256 accumulators
                                        // through the architectural registers and spills).  The
                                        // blocks are read in the order the products of the previous
                                        // phase O wrote them, in a basic block of their own: the
                                        // last write of block (v, d) is 27 - 8 v - d products and
                                        // 48 (4 v + d) instructions of this loop before its read
                                        float x = o[v][d][e], t;
                                        asm volatile("v_accvgpr_read_b32 %1, %0\n\tv_mul_f32 %1, %1, %2\n\tv_accvgpr_write_b32 %0, %1"
                                                     : "+a"(x), "=&v"(t) : "v"(alpha));
                                        o[v][d][e] = x;
                                    } else {
                                        o[v][d][e] *= alpha;
                                    }
                                }
                        l_run *= alpha;
                        m_run = m_new;
                    }
                }
            }
            const float nm = -m_run;
            constexpr int NSL = C::NKC;                // slots of phase S
            SCHED_FENCE();
#pragma unroll
            for (int i = 0; i < NSL; ++i) {
                if constexpr (NEXT) {
                    if constexpr (C::SV) sn = mma_v<DT>(kf[i], qf[i], sn, i == 0, i == NSL - 1);
                    else sn = MM::mma(kf[i], qf[i], i == 0 ? f32x16{} : sn);
                }
                if constexpr (C::SV) {
                    // the first VLEAD fragments of block j (its values landed at the previous barrier)
#pragma unroll
                    for (int t = 0; t < C::VLEAD; ++t)
                        if (t * NSL / C::VLEAD == i) rd_v(st0, t);
                } else {
#pragma unroll
                    for (int t = 0; t < NV * C::NV_READ; ++t)
                        if (t * NSL / (NV * C::NV_READ) == i) rd_v(st0, t);
                }
#pragma unroll
                for (int e = i * 16 / NSL; e < (i + 1) * 16 / NSL; ++e) {
                    // unchecked pass: the scores arrive already as s c - m (formed in the previous
                    // block's phase O)
                    sc[e] = __builtin_amdgcn_exp2f(CHECKED ? __builtin_fmaf(sc[e], scale_log2, nm) : sc[e]);
                    if (e & 1) pk[e >> 1] = pack2<DT>(sc[e - 1], sc[e]);
                }
                SCHED_FENCE();
            }
            // every wave has read block j's slot and block j + 1's keys; block j + 2 has landed (the
            // loads of block j + 3 may be in flight).  SV: every wave has read block j - 1's values
            // and block j + 1's keys; block j + 2's keys and block j + 1's values have landed
            wait_lgkm0();
            wait_vmcnt<(C::NS - 3) * C::PW>();
            raw_barrier();
            const int kbn = (j + 1) * 32;
            float m = -INFINITY;
            float ps[8];                               // the row sum's first level (sum16's order)
            static_assert(C::MP >= 4, "pair sums spread over the slots");
            SCHED_FENCE();
#pragma unroll
            for (int i = 0; i < C::MP; ++i) {
#pragma unroll
                for (int q = i * 8 / C::MP; q < (i + 1) * 8 / C::MP; ++q) ps[q] = sc[2 * q] + sc[2 * q + 1];
                if constexpr (C::SV)
                    if (i + C::VLEAD < C::MP) rd_v(st0, i + C::VLEAD);
                {
                    // MFMA i: value tensor v, k-step g, row block d (V^T fragment i)
                    const int v = i / C::MP1, ii = i % C::MP1, g = ii / C::NDB, d = ii % C::NDB;
                    const u32x4 pw = u32x4{pk[4 * g], pk[4 * g + 1], pk[4 * g + 2], pk[4 * g + 3]};
                    o[v][d] = MM::mma(__builtin_bit_cast(opnd, vf[v][d][g]), __builtin_bit_cast(opnd, pw), o[v][d]);
                }
#pragma unroll
                for (int k = 0; k < C::PW; ++k)
                    if (k * C::MP / C::PW == i) {
                        if constexpr (C::SV) {
                            // keys of block j + 4 into block j's slot (its keys were read two
                            // blocks ago), values of block j + 3 into block j - 1's slot
                            if (k < C::PK) issue(k, j + 4, st0);
                            else issue(k, j + 3, smem + ((SLOT >= 0 ? SLOT + 3 : s0 + 3) & (C::NS - 1)) * C::BLK);
                        } else if (SLOT < 0 && pre_aref && j + C::NS > jlast) {
                            // past the last block (only in the run-time-slot blocks): wave
                            // (j + NS - jlast - 1)'s teacher tile instead
                            issue_aref(k, j + C::NS - jlast - 1, st0);
                        } else {
                            issue(k, j + C::NS, st0);
                        }
                    }
                if constexpr (NEXT) {
#pragma unroll
                    for (int e = i * 16 / C::MP; e < (i + 1) * 16 / C::MP; ++e) {
                        if constexpr (MASKN) mask_el(kbn, sn, e);
                        if constexpr (CHECKED) m = fmaxf(m, sn[e]);
                        else sn[e] = __builtin_fmaf(sn[e], scale_log2, nm);
                    }
                }
#pragma unroll
                for (int kc = 0; kc < C::NKC; ++kc)
                    if (C::MP - C::NKC + kc == i) rd_k(st2, kc);
                SCHED_FENCE();
            }
            {
                const float b0 = ps[0] + ps[1], b1 = ps[2] + ps[3], b2 = ps[4] + ps[5], b3 = ps[6] + ps[7];
                l_run += (b0 + b1) + (b2 + b3);
            }
            if constexpr (NEXT && CHECKED) mx = halves_max(m);
        };

        int j = 0;
        // groups of four blocks whose refills are real blocks (j + 3 + NS <= jlast, so the next
        // block is unmasked too); the last NS blocks always run with a run-time slot
        for (; j + 3 + C::NS <= jlast; j += 4) {
            fblock(j, std::integral_constant<int, 0>(), sa, sb, yes(), no());
            fblock(j + 1, std::integral_constant<int, 1>(), sb, sa, yes(), no());
            fblock(j + 2, std::integral_constant<int, 2>(), sa, sb, yes(), no());
            fblock(j + 3, std::integral_constant<int, 3>(), sb, sa, yes(), no());
        }
        // the rest: unmasked blocks one at a time, the block before the diagonal, the diagonal
        for (; j + 1 < jlast; ++j) {
            fblock(j, dyn(), sa, sb, yes(), no());
            const f32x16 t = sa; sa = sb; sb = t;
        }
        if (j + 1 == jlast) {
            fblock(j, dyn(), sa, sb, yes(), yes());
            const f32x16 t = sa; sa = sb; sb = t;
            ++j;
        }
        fblock(j, dyn(), sa, sb, no(), no());
        wait_vmcnt<0>();
        l_run = halves_sum(l_run);                     // the query's row sum (both lanes)
    };

    tile_pass(no(), 1);                                // queries, then the first blocks, in flight
    {
        // a flagged query: row sum above 2^R (every probability is at most 2^R iff it is not, the
        // probabilities being non-negative), or an output that is not finite (0 * x is 0 for every
        // finite x and NaN otherwise); NaN sums are flagged too.  The workgroup's four waves decide
        // together (they share the key/value ring).
        float nonfin = 0.f;
#pragma unroll
        for (int v = 0; v < NV; ++v)
#pragma unroll
            for (int d = 0; d < C::NDB; ++d)
#pragma unroll
                for (int e = 0; e < 16; ++e) nonfin = __builtin_fmaf(o[v][d][e], 0.f, nonfin);
        const bool bad = !(l_run <= __builtin_exp2f(rescale_log2<DT>()) && nonfin == 0.f) && q0 + l32 < T;
        int *flags = reinterpret_cast<int *>(smem + (NV == 1 ? C::NS * C::BLK : 0));
        wait_lgkm0();
        raw_barrier();                                 // every wave is done with the ring
        const int any_bad = __any(bad) ? 1 : 0;         // with every lane active
        if (lane == 0) flags[wave] = any_bad;
        wait_lgkm0();
        raw_barrier();
        if (flags[0] | flags[1] | flags[2] | flags[3]) {
            raw_barrier();                             // every wave has read the flags
            thr = bad ? rescale_log2<DT>() : INFINITY;
            tile_pass(yes(), 0);
            // every wave's share of the teacher tiles has landed before any wave reads its own
            // (each wave waited for its own loads only)
            wait_lgkm0();
            raw_barrier();
        }
    }

    // ---- epilogue: partial sums per (query head, 32-query block).  The pair's second tile starts
    // loading its queries now (this tile's are no longer read), and its first key blocks once every
    // wave has read its teacher tile, so both are in flight during the rest of the epilogue.
    const float l_sum = l_run;
    const bool more = n_tile + 1 < n_tiles;
    Tile nxt;
    if (more) {
        make_tile(pp, grp, nxt);
        load_q(nxt);
    }
    // this wave's prefetched teacher tile: the slot of block jlast - 3 + wave
    const unsigned char *aslot = smem + ((jlast - 3 + wave) & (C::NS - 1)) * C::BLK + l32 * CR * 16;
    const int qrow = q0 + l32;
    float sse[NV], sa2 = 0.f, dpart = 0.f;
#pragma unroll
    for (int v = 0; v < NV; ++v) sse[v] = 0.f;
    if (qrow < T) {
        const float inv_l = 1.f / l_sum;
        const int64_t obase = (row0 + qrow) * ac + h * DH;
#pragma unroll
        for (int d = 0; d < C::NDB; ++d)
#pragma unroll
            for (int e4 = 0; e4 < 4; ++e4) {
                const int col = d * 32 + 8 * e4 + 4 * half;
                f32x4 val;
#pragma unroll
                for (int i = 0; i < 4; ++i) val[i] = o[0][d][4 * e4 + i] * inv_l;
                if (a.mode & ATT_LOSS) {
                    const f32x4 ref = pre_aref
                        ? *reinterpret_cast<const f32x4 *>(aslot + (((col / 4) ^ (l32 & 15)) * 16))
                        : *reinterpret_cast<const f32x4 *>(a.a_ref + obase + col);
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const float df = ref[i] - val[i];
                        sse[0] = __builtin_fmaf(df, df, sse[0]);
                        sa2 = __builtin_fmaf(ref[i], ref[i], sa2);
                    }
#pragma unroll
                    for (int v = 1; v < NV; ++v)
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            const float df = ref[i] - o[v][d][4 * e4 + i] * inv_l;
                            sse[v] = __builtin_fmaf(df, df, sse[v]);
                        }
                    if (NV == 1 && (a.mode & ATT_STORE_G)) {
                        // backward seed: g = dtype(a_hat - a_ref), D = sum g a_hat
                        elem gv[4];
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            gv[i] = from_f32<DT>(val[i] - ref[i]);
                            dpart = __builtin_fmaf(to_f32<DT>(gv[i]), val[i], dpart);
                        }
                        typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
                        *reinterpret_cast<u32x2 *>(static_cast<elem *>(a.g_out) + obase + col) =
                            u32x2{(uint32_t)gv[0] | ((uint32_t)gv[1] << 16), (uint32_t)gv[2] | ((uint32_t)gv[3] << 16)};
                    }
                }
                if (NV == 1 && (a.mode & ATT_STORE_O)) *reinterpret_cast<f32x4 *>(a.a_out + obase + col) = val;
            }
        if (NV == 1 && (a.mode & ATT_STORE_LSE) && half == 0)
            a.lse2[((int64_t)b * Hq + h) * T + qrow] = m_run + __builtin_amdgcn_logf(l_sum);
    }
    if (more) {                                        // every wave has left the ring
        wait_lgkm0();
        raw_barrier();
        issue_prologue(nxt);
    }
    if (NV == 1 && (a.mode & ATT_STORE_G)) {
        const float dsum = halves_sum(dpart);          // the query's two lanes
        if (qrow < T && half == 0) a.d_out[((int64_t)b * Hq + h) * T + qrow] = dsum;
    }
    if (a.mode & ATT_LOSS) {
        const double ta2 = wave_sum_f64((double)sa2);
#pragma unroll
        for (int v = 0; v < NV; ++v) {
            const double tse = wave_sum_f64((double)sse[v]);
            if (lane == 0) {
                double *ps = a.partials[v] + ((int64_t)b * Hq * nq32 + (int64_t)h * nq32 + qt) * 2;
                ps[0] = tse;
                ps[1] = ta2;
            }
        }
    }
    if (!more) break;
    cur = nxt;
  }
}

// NV > 1 takes the squared-error loss of NV value tensors (ATT_LOSS alone)
template <int DT, int DH, int NV = 1>
hipError_t launch_attn_fast(const AttnArgs &a, hipStream_t st) {
    typedef FastCfg<DT, DH, NV> C;
    if (NV > 1 && a.mode != ATT_LOSS) return hipErrorInvalidValue;
    const int nqt = (a.seq_len + 31) / 32;
    const int n_ht = a.n_heads / 4;
    const float scale_log2 = 1.4426950408889634f / sqrtf((float)DH);
    hipError_t e = hipFuncSetAttribute((const void *)attn_fast_kernel<DT, DH, NV>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)C::LDS_BYTES);
    if (e != hipSuccess) return e;
    const int n_pairs = (nqt + 1) / 2 * n_ht * a.batch;
    attn_fast_kernel<DT, DH, NV><<<dim3(n_pairs), dim3(256), C::LDS_BYTES, st>>>(a, scale_log2, nqt, n_ht);
    return hipGetLastError();
}

}  // namespace
}  // namespace jab
