// attn_fwd_impl.h -- causal grouped-query softmax attention with a fused
// squared-error epilogue (kernel template, included by the translation units that
// instantiate it).
//
// Paper: Method, "Layer-wise PTQ": A(X) = softmax(Q K^T / sqrt(d_head) + M) V with
// causal mask M; "The joint attention loss" (eq. joint_loss): the squared
// Frobenius distance between the teacher output A(X) and the student output.
// The merged output puts head h in columns h*d_head .. h*d_head + d_head - 1
// (Appendix "Evaluation metrics in full", M4: the merged pre-projection output).
//
// gfx950 design
//  * A workgroup is NW = 4 wavefronts; each wave owns 32 queries of one query head.  The
//    workgroup's waves share one key/value head: with n_heads/n_kv_heads a multiple of 4
//    they are 4 query heads of one group (every key/value tile read from memory serves all
//    of them).  For the 16-bit dtypes two workgroups share a CU (two waves per SIMD), so
//    one workgroup's start-up and teacher reads overlap the other's matrix work, and one
//    wave's vector work fills the other's matrix-core gaps.
//  * Scores are computed transposed, S^T = K Q^T, on 32x32 MFMAs: lane l owns query
//    (l % 32) and 16 of the 32 keys of a block, so a query's maximum is a lane-local pass
//    and one v_permlane32_swap exchange with lane l^32.
//  * O^T = V^T P^T: the probabilities go from the score registers straight into the
//    B operand.  V arrives already transposed, with keys permuted inside each block of
//    32 (vt_perm) so that the eight keys a lane contributes are one contiguous 16-byte
//    LDS read.  For the 16-bit dtypes the row sums come from the matrix cores too
//    (ONES P^T), so a lane ends up holding its query's full sum.
//  * The reference maximum of a query moves only when a block overshoots it by 2^64 for bf16,
//    2^15 for fp16, 2^8 for fp32 (rescale_log2), so the rescale of the output accumulators is
//    rare.
//  * K and V^T tiles of 32 keys stream from global memory straight into LDS
//    (global_load_lds_dwordx4) through a ring of stages of SB blocks, one barrier per
//    stage.  Tiles are dense with their 16-byte chunks XOR-swizzled per row (swz_key), so
//    the MFMA operand reads are free of bank conflicts.
//  * Each block runs in two phases: the MFMAs of the next block's scores interleaved with
//    this block's exponentials, then the PV MFMAs interleaved with the DMA refill and the
//    next block's mask and maximum.
//  * Query tiles are issued longest-first (causal work grows with the tile index), and
//    workgroup ids are remapped so one XCD processes all tiles of a (sequence, key/value
//    head) and reads its K/V through one L2.
//  * Epilogues: store the output (teacher, or the backward's forward), or read the
//    teacher tile and accumulate (a - a_hat)^2 and a^2 per wave (loss); the student
//    output never goes to memory in the loss.  All epilogues share one code path for the
//    output value, so a student equal to the teacher gives exactly 0.
#pragma once

#include <type_traits>

#include "device_common.h"
#include "kernels.h"
#include "lds_pipe.h"

namespace jab {
namespace {

// The running reference maximum of a query moves only when a block's maximum exceeds it
// by more than rescale_log2 binary orders of magnitude; in between, probabilities up to
// 2^rescale_log2 are accumulated against the old reference.  The output and the row sum
// always share one reference, so the normalised result does not depend on when the
// rescale happens; skipping most rescales saves the multiply of every accumulator.  The
// probabilities enter the value product rounded to the dtype: bf16 (and fp32) have the fp32
// exponent range, so bf16 lets them reach 2^64 (the output stays finite for values below
// 2^53), fp16 ends at 65504, so its probabilities stay at most 2^15.  attn_fast_kernel uses the
// same bound, so a query gets bitwise the same result from either kernel.
template <int DT> constexpr float rescale_log2() { return DT == F16 ? 15.f : DT == BF16 ? 64.f : 8.f; }

#ifndef ATT_LA
#define ATT_LA 2          // K fragment reads issued ahead of their MFMA
#endif
#ifndef ATT_LA_FAST
#define ATT_LA_FAST 8     // ... on the fast path
#endif
#ifndef ATT_FENCE
#define ATT_FENCE 1       // fence every MFMA slot so the interleave survives scheduling
#endif
#ifndef ATT_SB
#define ATT_SB 2          // key blocks of 32 per ring stage (one barrier per stage), 16-bit dtypes
#endif
#ifndef ATT_MINB
#define ATT_MINB 2        // workgroups per CU the 4-wave 16-bit single-value kernel is sized for
#endif
#ifndef ATT_KPRE
#define ATT_KPRE 0        // issue all of a block's K reads at the top of phase S
#endif
#ifndef ATT_VPRE
#define ATT_VPRE 0        // issue all of a block's V^T reads at the top of phase S
#endif

// Tile rows of C 16-byte chunks are stored with their chunks XOR-swizzled by a per-row key, so
// the 16 rows one LDS cycle serves (64 banks x 4 bytes) land on 16 distinct chunk slots when
// they read the same logical chunk: physical chunk = logical chunk ^ key(row).  Tiles stay
// dense (one DMA instruction fills 64 consecutive chunks), and a lane's reads within a row are
// its row base plus (logical chunk ^ key) * 16.
template <int C>
__host__ __device__ constexpr int swz_key(int r) {
    return C >= 16 ? (r & 15) : ((r / (16 / C)) & (C - 1));
}

// Sum of a lane's 16 probabilities of one key block in a fixed balanced order, shared by both
// attention kernels (so they add the same values in the same order).
__device__ inline float sum16(const float (&p)[16]) {
    float a[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) a[i] = p[2 * i] + p[2 * i + 1];
    const float b0 = a[0] + a[1], b1 = a[2] + a[3], b2 = a[4] + a[5], b3 = a[6] + a[7];
    return (b0 + b1) + (b2 + b3);
}

// workgroups per CU a configuration is built for: ATT_MINB for the 4-wave 16-bit single-value
// kernel (two rings fit in LDS), else one
template <int DT, int NV, int NW>
constexpr int att_wpc() { return NW == 4 && DT != F32 && NV == 1 ? ATT_MINB : 1; }

template <int DT, int DH, int NV, int QB, int NW>
struct AttnCfg {
    typedef typename Mma<DT>::elem elem;
    static constexpr int ES = (int)sizeof(elem);
    static constexpr int EPC = 16 / ES;                // elements per 16-byte chunk
    static constexpr int NKC = DH / Mma<DT>::K;        // k-steps of K Q^T
    static constexpr int DHP = DH < 32 ? 32 : DH;      // rows of O^T (padded to one MFMA block)
    static constexpr int NDB = DHP / 32;               // 32-row blocks of O^T
    static constexpr int CK = DH * ES / 16;            // chunks per K row (32 keys per block)
    static constexpr int CV = 32 * ES / 16;            // chunks per V^T row
    static constexpr int KCH = 32 * CK;                // DMA chunks of a K tile
    static constexpr int VCH = DH * CV;                // ... of one V^T tile (head_dim rows)
    static constexpr int K_BYTES = KCH * 16;
    static constexpr int V_BYTES = VCH * 16;
    static constexpr int VDS = 32 * CV * 16;           // bytes between 32-row blocks of V^T
    static constexpr int SUB = K_BYTES + NV * V_BYTES; // one block of 32 keys
    // blocks per ring stage (one barrier per stage): ATT_SB where three such stages fit in LDS
    static constexpr int SB = DT != F32 && 3 * ATT_SB * SUB * att_wpc<DT, NV, NW>() <= 160 * 1024 ? ATT_SB : 1;
    static constexpr int STAGE = SB * SUB;
    static constexpr int WPC = att_wpc<DT, NV, NW>();   // workgroups per CU
    static constexpr int NS_FIT = 160 * 1024 / WPC / STAGE;
    static constexpr int NS = NS_FIT < (SB == 1 ? 6 : 4) ? NS_FIT : (SB == 1 ? 6 : 4);   // stages in the ring
    static constexpr size_t LDS_BYTES = (size_t)NS * STAGE;
    static constexpr int KI = KCH / 64, VI = NV * VCH / 64;   // DMA instructions per block
    static constexpr int PWK = (KI + NW - 1) / NW, PWV = (VI + NW - 1) / NW, PW = PWK + PWV;   // per wave
    static constexpr int QW = 32 * QB;                 // queries per wave
    static constexpr int NE = 16 * QB;                 // score registers per lane and block
    static constexpr int MS = NKC * QB;                // MFMAs of S^T per block
    static constexpr int NPV = DT == F32 ? 16 : 2;     // k-steps of O^T += V^T P^T per block
    static constexpr int MP = NV * QB * NDB * NPV;     // MFMAs of phase O
    static constexpr int KL = DT == F32 ? NKC / 4 : NKC;      // LDS reads of a block's K fragments
    static constexpr int KPL = NKC / KL;                      // k-steps per read
    static constexpr int VG = DT == F32 ? 4 : 2;              // V^T reads per row block
    static constexpr int VL = NV * NDB * VG;                  // LDS reads of a block's V^T fragments
    static_assert(DT != F32 || NKC % 4 == 0, "fp32 K fragments are read 4 at a time");
    static_assert(KCH % 64 == 0 && VCH % 64 == 0, "a DMA instruction stays inside one tile");
    static_assert(LDS_BYTES * WPC <= 160 * 1024 && NS >= 3, "LDS ring");
};

// k index a lane supplies at k-step kc of S^T = K Q^T (any permutation shared by the K and
// Q operands gives the same product).  16-bit dtypes: 8 consecutive k per step, the
// native order.  fp32 (one k per lane and step): lanes of half h take the contiguous run
// h * DH/2 + kc, so their K row is read with 16-byte loads.
template <int DT, int DH>
__device__ inline int s_k(int kc, int half) {
    if constexpr (DT == F32) return half * (DH / 2) + kc;
    else return kc * Mma<DT>::K + half * Mma<DT>::VEC;
}

#if ATT_FENCE
#define SCHED_FENCE() __builtin_amdgcn_sched_barrier(0)
#else
#define SCHED_FENCE() do {} while (0)
#endif

// NW waves per workgroup; att_wpc workgroups per CU (two for the 16-bit single-value kernel:
// each wave gets half the register file).
//
// FAST: the workgroup's waves are NW query heads of one group over the same 32 queries (one
// query block per wave, one value tensor, one key block per ring stage).  Every wave then has
// the same blocks, so the block loop is peeled into a branch-free steady state (pairs of
// unmasked blocks) and a short tail; every stage is loaded (stages past the workgroup's range
// load its last block again into a slot that is never read), so each wait on the loads is a
// constant; ring slots advance by a running index instead of a division.
template <int DT, int DH, int NV, int QB, int NW, bool FAST>
__global__ __launch_bounds__(64 * NW, (att_wpc<DT, NV, NW>())) void attn_fwd_kernel(AttnArgs a, float scale_log2, int hpw,
                                                           int nqt, int n_ht) {
    typedef AttnCfg<DT, DH, NV, QB, NW> C;
    static_assert(!FAST || (QB == 1 && NV == 1 && C::SB == 1 && DT != F32), "single-block fast path");
    // K fragment reads in flight ahead of their MFMA: the fast path has the registers for all of a
    // block's (it has no per-wave branches to keep alive)
    constexpr int LA = FAST ? (C::KL < ATT_LA_FAST ? C::KL : ATT_LA_FAST) : (C::KL < ATT_LA ? C::KL : ATT_LA);
    typedef typename C::elem elem;
    typedef Mma<DT> MM;
    typedef typename MM::operand opnd;
    extern __shared__ __align__(16) unsigned char smem[];

    const int T = a.seq_len, Hq = a.n_heads;
    const int G = Hq / a.n_kv_heads;
    const int QT = NW * C::QW / hpw;                   // queries per workgroup tile
    const int Tp = vt_pad(T);

    // ---- workgroup -> (sequence, head tile, query tile)
    const int nwg = gridDim.x;
    int lin = blockIdx.x;
    if ((nwg & 7) == 0) lin = (lin & 7) * (nwg >> 3) + (lin >> 3);
    const int qt = nqt - 1 - lin % nqt;
    const int ht = (lin / nqt) % n_ht;
    const int b = lin / (nqt * n_ht);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, half = lane >> 5;
    const int h = ht * hpw + wave % hpw;
    const int kvh = h / G;
    // first query of this wave (a multiple of 32); with FAST all waves share it
    const int q0 = FAST ? qt * C::QW : qt * QT + (wave / hpw) * C::QW;
    const int q_last = q0 + C::QW - 1;
    const int kend = min(T, qt * QT + QT);
    const int nblk = (kend + 31) / 32;
    // last key block this wave computes (-1: no queries); blocks from jmask on hold keys
    // above some of the wave's queries and are masked
    const int jlast = q0 < T ? min(nblk - 1, q_last / 32) : -1;
    const int jmask = q0 / 32;
    const int64_t row0 = (int64_t)b * T;

    const elem *Qg = static_cast<const elem *>(a.q);

    // ---- this wave's queries as B operands of S^T = K Q^T
    opnd qf[QB][C::NKC];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        const int qrow = q0 + 32 * qb + (lane & 31);
        const elem *qp = Qg + (row0 + min(qrow, T - 1)) * a.ld + h * DH;
        if constexpr (DT == F32) {
#pragma unroll
            for (int i = 0; i < C::NKC / 4; ++i) {
                f32x4 v = *reinterpret_cast<const f32x4 *>(qp + s_k<DT, DH>(4 * i, half));
#pragma unroll
                for (int t = 0; t < 4; ++t) qf[qb][4 * i + t] = qrow < T ? v[t] : 0.f;
            }
        } else {
#pragma unroll
            for (int kc = 0; kc < C::NKC; ++kc) {
                u32x4 v = *reinterpret_cast<const u32x4 *>(qp + s_k<DT, DH>(kc, half));
                if (qrow >= T) v = u32x4{0u, 0u, 0u, 0u};
                qf[qb][kc] = __builtin_bit_cast(opnd, v);
            }
        }
    }

    // ---- DMA of key block j: each wave issues PWK of the block's KI K instructions and PWV
    // of its VI V^T instructions (64 chunks, one KiB of LDS each; a count not divisible by NW
    // repeats a load, which writes the same bytes).  Lane addresses are fixed per wave; a
    // block only adds its first key.  Keys past the sequence read the rows that follow it
    // (the next sequence, or the 32 rows of slack after the last one): the causal mask
    // removes them.  Blocks past the workgroup's range re-load its last block into a slot
    // that is never read again.  Pad positions load the tile's first chunk.
    int cur_j = 0, cur_s = 0;                          // FAST: block cur_j sits in ring slot cur_s
    auto blk = [&](int j) {
        if constexpr (FAST) {
            int s = cur_s + (j - cur_j);               // j - cur_j in [0, NS]
            s = s >= C::NS ? s - C::NS : s;
            return smem + s * C::STAGE;
        } else {
            return smem + ((j / C::SB) % C::NS) * C::STAGE + (j % C::SB) * C::SUB;
        }
    };
    const elem *kdma[C::PWK];
    int kdst[C::PWK];
#pragma unroll
    for (int i = 0; i < C::PWK; ++i) {
        const int idx = (wave + NW * i) % C::KI;
        const int p = idx * 64 + lane, r = p / C::CK, c = (p % C::CK) ^ swz_key<C::CK>(r);
        kdma[i] = static_cast<const elem *>(a.k) + (row0 + r) * a.ld + kvh * DH + c * C::EPC;
        kdst[i] = idx * 1024;
    }
    const elem *vdma[C::PWV];
    int vdst[C::PWV];
#pragma unroll
    for (int i = 0; i < C::PWV; ++i) {
        const int idx = (wave + NW * i) % C::VI;
        const int vb = idx * 64, v = vb / C::VCH, prb = vb % C::VCH;
        const int p = prb + lane, r = p / C::CV, c = (p % C::CV) ^ swz_key<C::CV>(r);
        const elem *vt = static_cast<const elem *>(NV > 1 && v ? a.v[1] : a.v[0]);
        vdma[i] = vt + (int64_t)(kvh * DH + r) * a.ldv + (int64_t)b * Tp + c * C::EPC;
        vdst[i] = C::K_BYTES + v * C::V_BYTES + prb * 16;
    }
    auto issue_dma = [&](int i, int j) {               // i-th of the wave's PW instructions for block j
        const int kb = (j < nblk ? j : nblk - 1) * 32;
        if (i < C::PWK) lds_dma16((const void *)(kdma[i] + (int64_t)kb * a.ld), blk(j) + kdst[i]);
        else lds_dma16((const void *)(vdma[i - C::PWK] + kb), blk(j) + vdst[i - C::PWK]);
    };
    // k-th of the wave's SB * PW instructions for ring stage t; only stages holding blocks of
    // this workgroup are loaded
    const int nst = (nblk + C::SB - 1) / C::SB;
    auto issue_stage_part = [&](int k, int t) {
        if (FAST || t < nst) issue_dma(k % C::PW, t * C::SB + k / C::PW);
    };

    // ---- LDS fragment reads: one per-lane base each, the rest immediate offsets
    const int kr = lane & 31;
    const int krow = kr * C::CK * 16, kkey = swz_key<C::CK>(kr) * 16;
    opnd kf[C::NKC];
    auto load_kl = [&](const unsigned char *st, int l) {   // read l of C::KL
        const int cl = DT == F32 ? half * (DH / 8) + l : 2 * l + half;   // logical chunk
        const unsigned char *pk = st + krow + ((cl * 16) ^ kkey);
        if constexpr (DT == F32) {
            const f32x4 v = *reinterpret_cast<const f32x4 *>(pk);
#pragma unroll
            for (int t = 0; t < 4; ++t) kf[4 * l + t] = v[t];
        } else {
            kf[l] = __builtin_bit_cast(opnd, *reinterpret_cast<const u32x4 *>(pk));
        }
    };
    // V^T fragments: 16-bit, [v][d][kc2] = the 8 keys of k-step kc2 for row d*32 + lane%32;
    // fp32, [v][d][g] = keys of register group g (4 consecutive positions in vt_perm order).
    // Read t covers (g, d, v) with g outermost, the order the MFMAs consume them.  Rows past
    // head_dim (head_dim < 32) read a real row and are zeroed.
    const int vrow = DH < 32 ? (lane & 31) % DH : (lane & 31);
    const int vbase = vrow * C::CV * 16, vkey = swz_key<C::CV>(vrow) * 16;   // key equal for rows 32 apart
    u32x4 vf[NV][C::NDB][C::VG];
    auto load_vl = [&](const unsigned char *st, int t) {
        const int v = t % NV, d = (t / NV) % C::NDB, g = t / (NV * C::NDB);
        // logical chunk of read g: 16-bit 2 g + half; fp32 4 (g / 2) + 2 half + g % 2
        const int cl = DT == F32 ? 4 * (g >> 1) + 2 * half + (g & 1) : 2 * g + half;
        u32x4 x = *reinterpret_cast<const u32x4 *>(st + C::K_BYTES + v * C::V_BYTES + vbase + d * C::VDS + ((cl * 16) ^ vkey));
        if constexpr (DH < 32)
            if ((lane & 31) >= DH) x = u32x4{0u, 0u, 0u, 0u};
        vf[v][d][g] = x;
    };

    // ---- running state
    f32x16 o[NV][QB][C::NDB];
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
#pragma unroll
            for (int d = 0; d < C::NDB; ++d)
#pragma unroll
                for (int e = 0; e < 16; ++e) o[v][qb][d][e] = 0.f;
    float m_run[QB], l_run[QB];                        // reference max (log2 units), lane's partial sum (fp32)
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) { m_run[qb] = -INFINITY; l_run[qb] = 0.f; }
    f32x16 sa[QB], sb[QB];                             // scores of two consecutive blocks (ping-pong)
    float mx[QB];                                      // maxima of the current block's scores (raw units)
    float p[QB][16];                                   // probabilities of the current block (fp32 dtype)
    uint32_t pk[QB][8];                                // ... packed pairwise (16-bit dtypes)

    // score register e of a lane holds key kb + 8 (e / 4) + 4 half + e % 4 of its query: it is
    // masked when 8 (e / 4) + e % 4 (a constant) exceeds query - kb - 4 half
    auto mask_el = [&](int kb, f32x16 (&s)[QB], int qb, int e) {
        const int lim = q0 + 32 * qb + (lane & 31) - kb - 4 * half;
        if (8 * (e >> 2) + (e & 3) > lim) s[qb][e] = -INFINITY;
    };

#pragma unroll
    for (int t = 0; t < C::NS; ++t)
#pragma unroll
        for (int k = 0; k < C::SB * C::PW; ++k) issue_stage_part(k, t);
    // stages 0 and 1 have landed (this wave's part): the stages issued after them may be pending
    if constexpr (FAST) wait_vmcnt<(C::NS - 2) * C::PW>();
    else wait_vm_groups<C::SB * C::PW, C::NS - 2>(min(C::NS, nst) - 2);
    __syncthreads();                                   // ... for every wave

    if (jlast >= 0) {
#pragma unroll
        for (int l = 0; l < C::KL; ++l) load_kl(smem, l);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
#pragma unroll
            for (int e = 0; e < 16; ++e) sa[qb][e] = 0.f;
#pragma unroll
        for (int kc = 0; kc < C::NKC; ++kc)
#pragma unroll
            for (int qb = 0; qb < QB; ++qb) sa[qb] = MM::mma(kf[kc], qf[qb][kc], sa[qb]);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
            if (jmask == 0)
#pragma unroll
                for (int e = 0; e < 16; ++e) mask_el(0, sa, qb, e);
            float m = sa[qb][0];
#pragma unroll
            for (int e = 1; e < 16; ++e) m = fmaxf(m, sa[qb][e]);
            mx[qb] = halves_max(m);
        }
        // first K reads of block 1 for the first pipelined step
#pragma unroll
        for (int l = 0; l < LA; ++l) load_kl(blk(1), l);
    }

    // ---- one block in two phases around the block's barrier.
    // Phase S (before): the scores of block j + 1 on the matrix cores, interleaved with the
    // exponentials of block j on the vector unit, and the reads of block j's V^T fragments.
    // Phase O (after): O^T += V^T P^T for block j on the matrix cores, interleaved with the DMA
    // of the stage block j ends (if it ends one), the mask and maxima of block j + 1, and the
    // first K reads of block j + 2.  Each slot below is fenced so the compiler keeps the
    // interleave (a matrix-core op every slot, vector work in its shadow).
    auto phase_s = [&](int j, auto has_next, f32x16 (&sc)[QB], f32x16 (&sn)[QB]) {
        constexpr bool NEXT = decltype(has_next)::value;
        // reference maxima: move them only where a block's maximum overshoots by 2^rescale_log2
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
            const float ms = mx[qb] * scale_log2;
            const bool move = ms > m_run[qb] + rescale_log2<DT>();
            if (__any(move)) {
                // only the lanes that overshoot move (the others multiply by exactly 1), so a
                // query's arithmetic never depends on the other queries of its wave
                const float m_new = move ? ms : m_run[qb];
                const float alpha = __builtin_amdgcn_exp2f(m_run[qb] - m_new);
#pragma unroll
                for (int v = 0; v < NV; ++v)
#pragma unroll
                    for (int d = 0; d < C::NDB; ++d)
#pragma unroll
                        for (int e = 0; e < 16; ++e) o[v][qb][d][e] *= alpha;
                l_run[qb] *= alpha;
                m_run[qb] = m_new;
            }
        }
        const unsigned char *stc = blk(j);
        const unsigned char *stn = blk(j + 1);
        float nm[QB];
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) nm[qb] = -m_run[qb];
        if constexpr (NEXT) {
#pragma unroll
            for (int qb = 0; qb < QB; ++qb)
#pragma unroll
                for (int e = 0; e < 16; ++e) sn[qb][e] = 0.f;
        }
        constexpr int NSL = NEXT ? C::MS : C::VL;      // slots
        if constexpr (NEXT && ATT_KPRE) {
#pragma unroll
            for (int l = LA; l < C::KL; ++l) load_kl(stn, l);
        }
        if constexpr (ATT_VPRE) {
#pragma unroll
            for (int t = 0; t < C::VL; ++t) load_vl(stc, t);
        }
        SCHED_FENCE();
#pragma unroll
        for (int i = 0; i < NSL; ++i) {
            if constexpr (NEXT) {
                const int kc = i / QB, qb = i % QB;
                if (!ATT_KPRE && qb == 0 && kc % C::KPL == 0 && kc / C::KPL + LA < C::KL)
                    load_kl(stn, kc / C::KPL + LA);
                sn[qb] = MM::mma(kf[kc], qf[qb][kc], sn[qb]);
            }
#pragma unroll
            for (int t = 0; t < C::VL; ++t)
                if (!ATT_VPRE && NSL / 2 + t * (NSL - NSL / 2) / C::VL == i) load_vl(stc, t);
#pragma unroll
            for (int el = i * C::NE / NSL; el < (i + 1) * C::NE / NSL; ++el) {
                const int qb = el / 16, e = el % 16;
                p[qb][e] = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[qb][e], scale_log2, nm[qb]));
                if constexpr (DT != F32)
                    if (e & 1) pk[qb][e >> 1] = pack2<DT>(p[qb][e - 1], p[qb][e]);
            }
            SCHED_FENCE();
        }
        // the lane's partial row sum (fp32 probabilities, the same order in both kernels)
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) l_run[qb] += sum16(p[qb]);
    };

    auto phase_o = [&](int j, auto has_next, auto mask_next, auto refill, f32x16 (&sn)[QB]) {
        constexpr bool NEXT = decltype(has_next)::value;
        constexpr bool MASKN = decltype(mask_next)::value;
        constexpr bool REFILL = decltype(refill)::value;   // block j ends its stage: refill the stage
        constexpr int ND = REFILL ? C::SB * C::PW : 0;
        constexpr int MO = NV * QB * C::NDB * C::NPV;       // PV MFMAs
        const unsigned char *st2 = blk(j + 2);
        const int kbn = (j + 1) * 32;
        float m[QB];
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) m[qb] = -INFINITY;
        SCHED_FENCE();
#pragma unroll
        for (int i = 0; i < C::MP; ++i) {
            if (i < MO) {
                // MFMA i: k-step g, row block d, value tensor v, query block qb (qb fastest)
                const int qb = i % QB, v = (i / QB) % NV, d = (i / (QB * NV)) % C::NDB, g = i / (QB * NV * C::NDB);
                if constexpr (DT == F32) {
                    // the element goes through a scalar: a bit_cast applied directly to a vector
                    // element picks the wrong element with this compiler
                    const uint32_t ve = vf[v][d][g >> 2][g & 3];
                    o[v][qb][d] = MM::mma(__builtin_bit_cast(float, ve), p[qb][g], o[v][qb][d]);
                } else {
                    const u32x4 pw = u32x4{pk[qb][4 * g], pk[qb][4 * g + 1], pk[qb][4 * g + 2], pk[qb][4 * g + 3]};
                    o[v][qb][d] = MM::mma(__builtin_bit_cast(opnd, vf[v][d][g]), __builtin_bit_cast(opnd, pw), o[v][qb][d]);
                }
            }
#pragma unroll
            for (int k = 0; k < ND; ++k)
                if (k * C::MP / ND == i) issue_stage_part(k, j / C::SB + C::NS);
            if constexpr (NEXT) {
#pragma unroll
                for (int el = i * C::NE / C::MP; el < (i + 1) * C::NE / C::MP; ++el) {
                    const int qe = el / 16, e = el % 16;
                    if constexpr (MASKN) mask_el(kbn, sn, qe, e);
                    m[qe] = fmaxf(m[qe], sn[qe][e]);
                }
            }
            if (i >= C::MP - LA) load_kl(st2, i - (C::MP - LA));
            SCHED_FENCE();
        }
        if constexpr (NEXT) {
#pragma unroll
            for (int qb = 0; qb < QB; ++qb) mx[qb] = halves_max(m[qb]);
        }
    };

    typedef std::integral_constant<bool, true> yes;
    typedef std::integral_constant<bool, false> no;
    // block j with scores in sc, the next block's scores produced into sn.  When block j is the
    // last of its stage (BAR), every wave syncs after its phase S: stage j / SB has then been read
    // by all of them and is refilled with stage j / SB + NS, and the stages holding blocks up to
    // j + SB + 1 (read before the next barrier) must have landed: stage j / SB + 2.
    auto block = [&](int j, f32x16 (&sc)[QB], f32x16 (&sn)[QB], auto bar) {
        constexpr bool BAR = decltype(bar)::value;
        if (j < jlast) phase_s(j, yes(), sc, sn);
        else if (j == jlast) phase_s(j, no(), sc, sn);
        if constexpr (BAR) {
            wait_lgkm0();
            // stage s + 2 (s = j / SB) has landed: the stages issued after it, up to s - 1 + NS
            // and within the workgroup's range, may be pending
            const int st = j / C::SB;
            wait_vm_groups<C::SB * C::PW, C::NS - 3>(min(st - 1 + C::NS, nst - 1) - (st + 2));
            raw_barrier();
        }
        if (j < jlast) {
            if (j + 1 >= jmask) phase_o(j, yes(), yes(), bar, sn);
            else phase_o(j, yes(), no(), bar, sn);
        } else if (j == jlast) {
            phase_o(j, no(), no(), bar, sn);
        } else if constexpr (BAR) {
#pragma unroll
            for (int k = 0; k < C::SB * C::PW; ++k) issue_stage_part(k, j / C::SB + C::NS);
        }
    };
    static_assert(C::SB == 1 || C::SB == 2, "the two-block unroll below places the barriers");
    typedef std::integral_constant<bool, C::SB == 1> even_bar;
    if constexpr (FAST) {
        // block j with its next block's scores (NEXT) and that block's mask (MASKN) known at
        // compile time; every block ends its stage
        auto fblock = [&](int j, f32x16 (&sc)[QB], f32x16 (&sn)[QB], auto has_next, auto mask_next) {
            phase_s(j, has_next, sc, sn);
            wait_lgkm0();
            wait_vmcnt<(C::NS - 3) * C::PW>();         // stage j + 2 has landed
            raw_barrier();
            phase_o(j, has_next, mask_next, yes(), sn);
            cur_j = j + 1;
            cur_s = cur_s + 1 == C::NS ? 0 : cur_s + 1;
        };
        // blocks whose next block is unmasked, the block before the diagonal, the diagonal block
        int j = 0;
        for (; j + 2 <= jlast; ++j) {
            fblock(j, sa, sb, yes(), no());
#pragma unroll
            for (int qb = 0; qb < QB; ++qb) { const f32x16 t = sa[qb]; sa[qb] = sb[qb]; sb[qb] = t; }
        }
        if (j + 1 == jlast) {
            fblock(j, sa, sb, yes(), yes());
#pragma unroll
            for (int qb = 0; qb < QB; ++qb) { const f32x16 t = sa[qb]; sa[qb] = sb[qb]; sb[qb] = t; }
            ++j;
        }
        fblock(j, sa, sb, no(), no());
    } else {
        for (int j = 0; j < nblk; j += 2) {
            block(j, sa, sb, even_bar());
            if (j + 1 < nblk) block(j + 1, sb, sa, yes());
        }
    }
    wait_vmcnt<0>();

    // ---- epilogue: partial sums per (query head, 32-query block), so their layout does not
    // depend on how many query blocks a wave owns
    const int nq32 = (T + 31) / 32;
    const int per_seq = Hq * nq32;
    const int ac = Hq * DH;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) l_run[qb] = halves_sum(l_run[qb]);
#pragma unroll
    for (int v = 0; v < NV; ++v) {
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
            const int qrow = q0 + 32 * qb + (lane & 31);
            float sse = 0.f, sa2 = 0.f, dpart = 0.f;
            if (qrow < T) {
                const float inv_l = 1.f / l_run[qb];
                const int64_t obase = (row0 + qrow) * ac + h * DH;
#pragma unroll
                for (int d = 0; d < C::NDB; ++d)
#pragma unroll
                    for (int e4 = 0; e4 < 4; ++e4) {
                        const int col = d * 32 + 8 * e4 + 4 * half;
                        if (DH < 32 && col >= DH) continue;
                        f32x4 val;
#pragma unroll
                        for (int i = 0; i < 4; ++i) val[i] = o[v][qb][d][4 * e4 + i] * inv_l;
                        if (a.mode & ATT_LOSS) {
                            const f32x4 ref = *reinterpret_cast<const f32x4 *>(a.a_ref + obase + col);
#pragma unroll
                            for (int i = 0; i < 4; ++i) {
                                const float df = ref[i] - val[i];
                                sse = __builtin_fmaf(df, df, sse);
                                sa2 = __builtin_fmaf(ref[i], ref[i], sa2);
                            }
                            if constexpr (NV == 1) {
                                if (a.mode & ATT_STORE_G) {
                                    // backward seed: g = dtype(a_hat - a_ref), D = sum g a_hat
                                    elem gv[4];
#pragma unroll
                                    for (int i = 0; i < 4; ++i) {
                                        gv[i] = from_f32<DT>(val[i] - ref[i]);
                                        dpart = __builtin_fmaf(to_f32<DT>(gv[i]), val[i], dpart);
                                    }
                                    elem *gp = static_cast<elem *>(a.g_out) + obase + col;
                                    if constexpr (DT == F32) {
                                        *reinterpret_cast<f32x4 *>(gp) = f32x4{gv[0], gv[1], gv[2], gv[3]};
                                    } else {
                                        typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
                                        *reinterpret_cast<u32x2 *>(gp) =
                                            u32x2{(uint32_t)gv[0] | ((uint32_t)gv[1] << 16),
                                                  (uint32_t)gv[2] | ((uint32_t)gv[3] << 16)};
                                    }
                                }
                            }
                        }
                        if (a.mode & ATT_STORE_O)
                            *reinterpret_cast<f32x4 *>(a.a_out + obase + col) = val;
                    }
                if (v == 0 && (a.mode & ATT_STORE_LSE) && half == 0)
                    a.lse2[((int64_t)b * Hq + h) * T + qrow] = m_run[qb] + __builtin_amdgcn_logf(l_run[qb]);
            }
            if constexpr (NV == 1) {                          // the backward runs one value tensor
                if (a.mode & ATT_STORE_G) {
                    const float dsum = halves_sum(dpart);      // the query's two lanes
                    if (qrow < T && half == 0) a.d_out[((int64_t)b * Hq + h) * T + qrow] = dsum;
                }
            }
            if ((a.mode & ATT_LOSS) && q0 + 32 * qb < T) {
                const double tse = wave_sum_f64((double)sse);
                const double ta2 = wave_sum_f64((double)sa2);
                if (lane == 0) {
                    double *pp = a.partials[v] + ((int64_t)b * per_seq + (int64_t)h * nq32 + (q0 / 32 + qb)) * 2;
                    pp[0] = tse;
                    pp[1] = ta2;
                }
            }
        }
    }
}

}  // namespace

template <int DT, int DH, int NV, int QB, int NW, bool FAST>
hipError_t launch_attn_kernel(const AttnArgs &a, int hpw, hipStream_t st) {
    typedef AttnCfg<DT, DH, NV, QB, NW> C;
    const int QT = NW * C::QW / hpw;
    const int nqt = (a.seq_len + QT - 1) / QT;
    const int n_ht = a.n_heads / hpw;
    const float scale_log2 = 1.4426950408889634f / sqrtf((float)DH);
    hipError_t e = hipFuncSetAttribute((const void *)attn_fwd_kernel<DT, DH, NV, QB, NW, FAST>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)C::LDS_BYTES);
    if (e != hipSuccess) return e;
    const int nwg = nqt * n_ht * a.batch;
    attn_fwd_kernel<DT, DH, NV, QB, NW, FAST><<<dim3(nwg), dim3(64 * NW), C::LDS_BYTES, st>>>(a, scale_log2, hpw, nqt, n_ht);
    return hipGetLastError();
}

template <int DT, int DH, int NV, int QB, int NW>
hipError_t run_attn_cfg(const AttnArgs &a, hipStream_t st) {
    typedef AttnCfg<DT, DH, NV, QB, NW> C;
    const int G = a.n_heads / a.n_kv_heads;
    const int hpw = G % 4 == 0 ? 4 : G;            // heads per workgroup tile (1, 2 or 4)
    if constexpr (QB == 1 && NV == 1 && C::SB == 1 && DT != F32) {
        if (hpw == NW) return launch_attn_kernel<DT, DH, NV, QB, NW, true>(a, hpw, st);
    }
    return launch_attn_kernel<DT, DH, NV, QB, NW, false>(a, hpw, st);
}

}  // namespace jab
