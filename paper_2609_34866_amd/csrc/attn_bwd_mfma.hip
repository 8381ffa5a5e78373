// attn_bwd_mfma.hip -- backward of the squared-error JAB loss through causal GQA attention
// for the 16-bit dtypes at head_dim 64 and 128: the dK/dV and dQ kernels with their
// operand tiles streamed into LDS by DMA.
//
// Paper: Method, "Joint fine-tuning through the quantizer" and the Appendix on its design
// decisions, (1) / eq. lsq: the gradient of the attention-output loss of eq. joint_loss
// reaches the weights through Q, K and V.  With G = a_hat - a_ref, P the causal softmax
// (recomputed from the forward's log-sum-exp), D_i = sum_c G_ic a_hat_ic:
//   dV_j = sum_i P_ij G_i   (summed over the query heads of a kv group)
//   dS_ij = P_ij (G_i . V_j - D_i)
//   dQ_i = sum_j dS_ij K_j / sqrt(dh),   dK_j = sum_i dS_ij Q_i / sqrt(dh)
//
// gfx950 design (no atomics, fixed summation order => deterministic)
//  * Operand tiles are 32 rows of Q, G (dK/dV) or K, V (dQ) in their row-major form, DMA'd
//    (global_load_lds_dwordx4) into a ring of LDS stages with one barrier per tile.  The
//    products that contract over tokens need the tiles transposed (G^T, Q^T, K^T): those
//    operands come from the same row-major tiles through transposed LDS reads
//    (ds_read_b64_tr_b16), so no transposed copy exists in memory or in LDS.
//  * Tiles are stored quad-major (TileLayout): 16-byte chunks in groups of four per row,
//    each group of 32 rows contiguous, the chunk inside a group rotated by row / 4.  Both
//    access patterns are then free of bank conflicts (16 rows reading one logical chunk;
//    4 consecutive rows reading 4 consecutive chunks), and every fragment of a wave is its
//    lane's base address plus a constant offset.
//  * dK/dV: a workgroup of NW waves owns 32 NW consecutive keys of one kv head, each wave
//    32 keys with K and V in registers as B operands.  It walks the 32-query tiles of the
//    group's query heads from the last tile down to its diagonal (workgroups of one kv head
//    that start together read the same tiles at the same time, through one L2), and takes
//    two key blocks, p and nkb - 1 - p, so every workgroup gets the same number of tiles.
//    S = Q K^T and dP = G V^T come out with one key per lane; P and dS go from registers
//    into the B operand of dV^T += G^T P and dK^T += Q^T dS.  With room for it in the
//    workspace, the dK pass also stores each 32 x 32 dS tile as that operand (2 KiB).
//  * dQ from the stored dS: a wave owns 32 queries of one query head; the workgroup's waves
//    share a kv head and walk its 32-key tiles, each wave's dS tiles riding the same LDS ring
//    and read transposed into the B operand of dQ^T += K^T dS^T (5 products in all).
//  * dQ recomputing dS (no stored dS): a wave owns 32 queries of one query head (Q and G in
//    registers as B operands); the workgroup's waves share a kv head and walk its 32-key
//    tiles.  S^T = K Q^T and dP^T = V G^T come out with one query per lane, so lse and D are
//    per-lane scalars, and dQ^T += K^T dS^T (7 products in all).
//  * Rows past the sequence are read at the sequence's last row (finite values) and
//    removed by the masks; the results are written transposed, dY^T [R][tokens], the
//    operand layout of the weight-gradient GEMM.
#include "device_common.h"
#include "kernels.h"
#include "lds_pipe.h"

namespace jab {
namespace {

// Quad-major tile layout: chunk c (16 bytes) of row r of a 32-row tile is stored at chunk slot
//   (c / 4) * 128 + 4 r + ((c % 4) ^ ((r / 4) % 4)).
// Row reads (16 rows, one logical chunk) land on 16 distinct 16-byte bank slots: 4 (r % 4) plus
// a rotation by r / 4.  Transposed reads (rows 4x .. 4x + 3, chunks 4m .. 4m + 3) use one row
// group per 64 bytes and one rotation: 16 distinct slots as well.
__host__ __device__ constexpr int quad_slot(int r, int c) { return (c >> 2) * 128 + 4 * r + ((c & 3) ^ ((r >> 2) & 3)); }

// MODE (the dK/dV kernel): 0 both products, 1 dV alone, 2 dK alone.  With the KL term the
// split pair (1 then 2) keeps two workgroups per CU where the kernel with both cannot.
template <int DT, int DH, int NW, bool KL = false, int MODE = 0>
struct BwdTiles {
    static constexpr int NKC = DH / 16;           // k-steps of 16 over the head dimension
    static constexpr int NDB = DH / 32;           // 32-row blocks of a transposed result
    static constexpr int CK = DH / 8;             // 16-byte chunks per row
    static constexpr int ROW = CK * 16;           // bytes per tile row
    static constexpr int TILE = 32 * ROW;         // one 32-row tile
    static constexpr int TI = TILE / 1024;        // DMA instructions per tile
    // dK/dV stage: Q tile | G tile (| teacher Q tile) | lse[32] | D[32] (| teacher lse[32] twice).
    // With the KL term the wave also keeps its keys' teacher K in registers: one wave per SIMD.
    static constexpr int NT_KV = KL ? 3 : 2;
    static constexpr int WPC_KV = (KL && MODE == 0) ? 1 : (NW == 4 ? 2 : 1);   // workgroups per CU
    static constexpr int NS_KV = (KL && MODE == 2) ? 3 : 4;                    // ring stages
    static constexpr int KV_STAGE = NT_KV * TILE + (KL ? 512 : 256);
    static constexpr int KV_PW = NT_KV * TI / NW + (KL ? 2 : 1);   // DMA instructions per wave and tile
    // dQ stage: K tile | V tile (| teacher K tile)
    static constexpr int NT_Q = KL ? 3 : 2;
    static constexpr int WPC_Q = NW == 4 ? 2 : 1;
    static constexpr int NS_Q = KL ? 3 : 4;
    static constexpr int Q_STAGE = NT_Q * TILE;
    static constexpr int Q_PW = NT_Q * TI / NW;
    static_assert(TI % NW == 0, "each tile splits evenly over the waves");
    static_assert((size_t)NS_KV * KV_STAGE * WPC_KV <= 160 * 1024, "LDS ring (dK/dV)");
    static_assert((size_t)NS_Q * Q_STAGE * WPC_Q <= 160 * 1024, "LDS ring (dQ)");
};

// per-lane byte offsets inside a tile: the row read of k-step kc (logical chunk 2 kc + half of
// row lane % 32) is at rd[kc % 2] + (kc / 2) * 2048; the transposed read of k-step ks, part p
// (rows 16 ks + 8 p + 4 half .. + 3) and row block db is at tr[p] + db * 2048 + ks * 1024.
struct TileLanes {
    int rd[2], tr[2];
    __device__ TileLanes(int lane) {
        const int r = lane & 31, half = lane >> 5;
#pragma unroll
        for (int k = 0; k < 2; ++k) rd[k] = 16 * quad_slot(r, 2 * k + half);
        const int j = lane & 15, ta = j & 3, ts = j >> 2, tg = lane >> 4;
#pragma unroll
        for (int p = 0; p < 2; ++p)
            tr[p] = 16 * quad_slot(8 * p + 4 * (tg >> 1) + ts, 2 * (tg & 1) + (ta >> 1)) + 8 * (ta & 1);
    }
};

// A operand of k-step kc from a row-major tile: row (lane % 32), logical chunk 2 kc + half
template <int DT>
__device__ inline typename Mma<DT>::operand row_frag(const lds_u8 *tile, const TileLanes &tl, int kc) {
    return __builtin_bit_cast(typename Mma<DT>::operand,
                              *reinterpret_cast<const __attribute__((address_space(3))) u32x4 *>(
                                  tile + tl.rd[kc & 1] + (kc >> 1) * 2048));
}
// A operand of a product contracting over the tile's rows: row (lane % 32) of the transposed
// row block db, k-slots = the 8 tile rows 16 ks + 4 half + {0..3, 8..11}
template <int DT>
__device__ inline typename Mma<DT>::operand tr_frag(const lds_u8 *tile, const TileLanes &tl, int ks, int db) {
    const s16x4 lo = lds_read_tr16(tile + tl.tr[0] + db * 2048 + ks * 1024);
    const s16x4 hi = lds_read_tr16(tile + tl.tr[1] + db * 2048 + ks * 1024);
    return __builtin_bit_cast(typename Mma<DT>::operand, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}
// global source chunk of DMA piece idx (1 KiB) of a tile for this lane: row and element column
__device__ inline void quad_source(int idx, int lane, int &row, int &col) {
    const int P = idx * 64 + lane, rem = P & 127, r = rem >> 2;
    row = r;
    col = (4 * (P >> 7) + ((rem & 3) ^ ((r >> 2) & 3))) * 8;
}
// B operand of k-step ks from an accumulator tile: values 8 ks .. 8 ks + 7 rounded and packed
template <int DT>
__device__ inline typename Mma<DT>::operand acc_operand(const f32x16 &v, int ks) {
    const u32x4 w = u32x4{pack2<DT>(v[8 * ks], v[8 * ks + 1]), pack2<DT>(v[8 * ks + 2], v[8 * ks + 3]),
                          pack2<DT>(v[8 * ks + 4], v[8 * ks + 5]), pack2<DT>(v[8 * ks + 6], v[8 * ks + 7])};
    return __builtin_bit_cast(typename Mma<DT>::operand, w);
}

__device__ inline int xcd_remap(int lin, int nwg) {
    return (nwg & 7) == 0 ? (lin & 7) * (nwg >> 3) + (lin >> 3) : lin;
}

// ------------------------------------------------------------------ dK / dV
// KL: the gradient of the KL attention-map term rides along (kl_scale (P - P_t) added to each dS
// entry, P_t the teacher's map rebuilt from its projection and log-sum-exp); dS is then multiplied
// by grad_scale (a power of two that keeps fp16 in range; the scale-gradient kernel divides it out
// of the W_Q and W_K rows of the weight gradient).
// DS: the dK pass stores dS (AttnBwdArgs::ds) for the dQ pass.
template <int DT, int DH, int NW, bool KL, int MODE = 0, bool DS = false>
__global__ __launch_bounds__(64 * NW, (BwdTiles<DT, DH, NW, KL, MODE>::WPC_KV)) void attn_bwd_dkdv_dma_kernel(
    AttnBwdArgs a, float scale_log2, float inv_sqrt, int nkb, int npair) {
    typedef BwdTiles<DT, DH, NW, KL, MODE> C;
    static_assert(MODE == 0 || MODE == 2 || !KL, "dV alone has no KL part");
    static_assert(!DS || MODE != 1, "dS comes from the dK pass");
    constexpr bool DO_DV = MODE != 2, DO_DK = MODE != 1;
    typedef Mma<DT> MM;
    typedef typename MM::operand opnd;
    typedef uint16_t elem;
    constexpr int BK = 32 * NW;                        // keys per block
    constexpr int NS = C::NS_KV;
    extern __shared__ __align__(16) unsigned char smem[];
    const lds_u8 *sm = (const lds_u8 *)smem;

    const int T = a.seq_len, Hq = a.n_heads, Hkv = a.n_kv_heads;
    const int G = Hq / Hkv;
    const int lin = xcd_remap(blockIdx.x, gridDim.x);
    const int pr = lin % npair;
    const int kvh = (lin / npair) % Hkv;
    const int b = lin / (npair * Hkv);
    const int kbA = pr, kbB = nkb - 1 - pr;            // equal for the middle block of an odd count
    const int nqA = (T - kbA * BK + 31) / 32, nqB = (T - kbB * BK + 31) / 32;
    const int nA = G * nqA;
    const int U = nA + (kbB != kbA ? G * nqB : 0);     // tiles of this workgroup

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, half = lane >> 5;
    const int64_t row0 = (int64_t)b * T;
    const elem *Qs = static_cast<const elem *>(a.q) + row0 * a.ldq;
    const elem *Gs = static_cast<const elem *>(a.g) + row0 * Hq * DH;
    const elem *Qts = KL ? static_cast<const elem *>(a.qt) + row0 * a.ldq : nullptr;
    const int64_t ld_base = (int64_t)b * Hq * T;       // lse2 / D of (b, h, t): ld_base + h T + t

    // tile u -> key block, query head, first query (tiles of a block: the group's heads for
    // the last query tile, then the tile below, down to the block's diagonal)
    auto tile_of = [&](int u, int &kb, int &h, int &q0) {
        const bool second = u >= nA;
        const int v = second ? u - nA : u;
        kb = second ? kbB : kbA;
        const int nq = second ? nqB : nqA;
        h = kvh * G + v % G;
        q0 = kb * BK + 32 * (nq - 1 - v / G);
    };

    // ---- DMA: instruction i of this wave loads 1 KiB piece wave + NW i of the stage's tiles
    // (pieces [0, TI): Q, [TI, 2 TI): G, [2 TI, 3 TI): the teacher's Q), then lse and D (one
    // 4-byte load per lane: lanes below 32 lse, the others D) and with the KL term the teacher's
    // lse (every lane; lanes 32..63 repeat lanes 0..31)
    constexpr int NP = C::NT_KV * C::TI / NW;
    auto stage_ptr = [&](int s) { return smem + s * C::KV_STAGE; };
    // piece wave + NW i lies in tile (NW i) / TI (TI is a multiple of NW); its LDS offset inside
    // that tile is wave KiB plus a constant
    const int wofs = __builtin_amdgcn_readfirstlane(wave * 1024);
    const float *ldp = (lane < 32 ? a.lse2 : a.D) + ld_base;
    auto issue = [&](int u) {
        if (u >= U) return;
        int kb, h, q0;
        tile_of(u, kb, h, q0);
        unsigned char *st = stage_ptr(u % NS) + wofs;
#pragma unroll
        for (int i = 0; i < NP; ++i) {
            const int tix = (NW * i) / C::TI;
            int drow, dcol;                            // formed per load: registers are scarce here
            quad_source((wave + NW * i) % C::TI, lane, drow, dcol);
            const int q = min(q0 + drow, T - 1);
            const elem *src = tix == 1 ? Gs + h * DH + (q * Hq * DH + dcol)
                                       : (tix == 0 ? Qs : Qts) + h * DH + (q * a.ldq + dcol);
            lds_dma16((const void *)src, st + tix * C::TILE + ((NW * i) % C::TI) * 1024);
        }
        const int q = min(q0 + (lane & 31), T - 1);
        lds_dma4((const void *)(ldp + (h * T + q)), stage_ptr(u % NS) + C::NT_KV * C::TILE);
        if constexpr (KL)
            lds_dma4((const void *)(a.lse_t + ld_base + (h * T + q)), stage_ptr(u % NS) + C::NT_KV * C::TILE + 256);
    };

    const TileLanes tl(lane);
    opnd kf[C::NKC], vf[C::NKC], ktf[KL ? C::NKC : 1];
    f32x16 dkt[C::NDB], dvt[C::NDB];
    auto begin_block = [&](int kb) {
        const int key = kb * BK + 32 * wave + (lane & 31);
        const int kr = min(key, T - 1);
        const elem *kp = static_cast<const elem *>(a.k) + (row0 + kr) * a.ldq + kvh * DH + half * 8;
        const elem *vp = static_cast<const elem *>(a.v) + (row0 + kr) * a.ldv + kvh * DH + half * 8;
#pragma unroll
        for (int kc = 0; kc < C::NKC; ++kc) {
            kf[kc] = __builtin_bit_cast(opnd, *reinterpret_cast<const u32x4 *>(kp + kc * 16));
            if constexpr (DO_DK) vf[kc] = __builtin_bit_cast(opnd, *reinterpret_cast<const u32x4 *>(vp + kc * 16));
        }
        if constexpr (KL) {
            const elem *ktp = static_cast<const elem *>(a.kt) + (row0 + kr) * a.ldq + kvh * DH + half * 8;
#pragma unroll
            for (int kc = 0; kc < C::NKC; ++kc)
                ktf[kc] = __builtin_bit_cast(opnd, *reinterpret_cast<const u32x4 *>(ktp + kc * 16));
        }
#pragma unroll
        for (int d = 0; d < C::NDB; ++d)
#pragma unroll
            for (int e = 0; e < 16; ++e) { dkt[d][e] = 0.f; dvt[d][e] = 0.f; }
    };
    // dK^T, dV^T: lane -> key (a token column of dY^T), registers -> head-dimension rows
    auto end_block = [&](int kb) {
        const int key = kb * BK + 32 * wave + (lane & 31);
        if (key >= T) return;
        elem *dyt = static_cast<elem *>(a.dyt) + row0 + key;
        const int koff = Hq * DH + kvh * DH, voff = (Hq + Hkv) * DH + kvh * DH;
#pragma unroll
        for (int d = 0; d < C::NDB; ++d)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int c = d * 32 + 8 * (e >> 2) + 4 * half + (e & 3);
                if constexpr (DO_DK) dyt[(int64_t)(koff + c) * a.ldt] = from_f32<DT>(dkt[d][e] * inv_sqrt);
                if constexpr (DO_DV) dyt[(int64_t)(voff + c) * a.ldt] = from_f32<DT>(dvt[d][e]);
            }
    };

    // tiles [u0, u1) of key block kb
    auto run_block = [&](int kb, int u0, int u1) {
        begin_block(kb);
        for (int u = u0; u < u1; ++u) {
            // this wave's part of tile u has landed (the tiles issued after it may be pending),
            // then every wave's part; every wave is also done reading tile u - 1, whose stage is
            // refilled
            wait_vm_groups<C::KV_PW, NS - 2>(min(NS - 2, U - 1 - u));
            raw_barrier();
            issue(u + NS - 1);
            int kbu, h, q0;
            tile_of(u, kbu, h, q0);
            const int kw = kb * BK + 32 * wave;        // first key of this wave
            if (q0 + 31 < kw || kw >= T) continue;     // no query of the tile sees these keys
            const lds_u8 *stq = sm + (u % NS) * C::KV_STAGE;
            const lds_u8 *stg = stq + C::TILE;
            const __attribute__((address_space(3))) float *lsd =
                (const __attribute__((address_space(3))) float *)(stq + C::NT_KV * C::TILE);

            // S = Q K^T, dP = G V^T (and the teacher's S_t = Q_t K_t^T): lane -> key, registers ->
            // queries 8 (e / 4) + 4 half + e % 4
            f32x16 s, dp, st;
#pragma unroll
            for (int e = 0; e < 16; ++e) { s[e] = 0.f; dp[e] = 0.f; st[e] = 0.f; }
#pragma unroll
            for (int kc = 0; kc < C::NKC; ++kc) {
                s = MM::mma(row_frag<DT>(stq, tl, kc), kf[kc], s);
                if constexpr (DO_DK) dp = MM::mma(row_frag<DT>(stg, tl, kc), vf[kc], dp);
                if constexpr (KL) st = MM::mma(row_frag<DT>(stq + 2 * C::TILE, tl, kc), ktf[kc], st);
            }
            const int key = kw + (lane & 31);
            const bool diag = q0 < kw + 31, tail = q0 + 31 >= T;
#pragma unroll
            for (int e4 = 0; e4 < 4; ++e4) {
                const int r0 = 8 * e4 + 4 * half;
                const f32x4 ls = *reinterpret_cast<const __attribute__((address_space(3))) f32x4 *>(lsd + r0);
                const f32x4 dd = *reinterpret_cast<const __attribute__((address_space(3))) f32x4 *>(lsd + 32 + r0);
                f32x4 lt;
                if constexpr (KL) lt = *reinterpret_cast<const __attribute__((address_space(3))) f32x4 *>(lsd + 64 + r0);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int e = 4 * e4 + i;
                    const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(s[e], scale_log2, -ls[i]));
                    float ds = p * (dp[e] - dd[i]);
                    if constexpr (KL) {
                        const float pt = __builtin_amdgcn_exp2f(__builtin_fmaf(st[e], scale_log2, -lt[i]));
                        ds = (ds + a.kl_scale * (p - pt)) * a.grad_scale;
                    }
                    s[e] = p;
                    dp[e] = ds;
                }
            }
            // the diagonal and sequence-tail tiles (wave-uniform): entries above the diagonal or
            // past the sequence are zero; the other tiles take no compare and no select
            if (diag || tail) {
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int q = q0 + 8 * (e >> 2) + 4 * half + (e & 3);
                    const bool off = q < key || q >= T;
                    s[e] = off ? 0.f : s[e];
                    dp[e] = off ? 0.f : dp[e];
                }
            }
            // dV^T += G^T P, dK^T += Q^T dS (k = the tile's 32 queries in two steps); with a dS store,
            // the operand of each step goes out before its products (2 KiB per tile: step ks, lane
            // at ks KiB + 16 lane), for the dQ pass.  The tile's address is wave-uniform (a buffer
            // resource in scalar registers); the store is non-temporal (read once, by the dQ pass),
            // so it does not push the Q and G tiles out of L2.
            i32x4 rds;
            if constexpr (DS) {
                const int qt = q0 / 32, kt = __builtin_amdgcn_readfirstlane(kw / 32), nq = (T + 31) / 32;
                rds = buffer_rsrc(static_cast<char *>(a.ds) +
                                  (((int64_t)b * Hq + h) * (nq * (nq + 1) / 2) + qt * (qt + 1) / 2 + kt) * 2048);
            }
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                const opnd pb = acc_operand<DT>(s, ks), sb = acc_operand<DT>(dp, ks);
                if constexpr (DS) buffer_store16_nt(rds, lane * 16, ks * 1024, __builtin_bit_cast(i32x4, sb));
#pragma unroll
                for (int d = 0; d < C::NDB; ++d) {
                    if constexpr (DO_DV) dvt[d] = MM::mma(tr_frag<DT>(stg, tl, ks, d), pb, dvt[d]);
                    if constexpr (DO_DK) dkt[d] = MM::mma(tr_frag<DT>(stq, tl, ks, d), sb, dkt[d]);
                }
            }
        }
        end_block(kb);
    };

#pragma unroll
    for (int t = 0; t < NS - 1; ++t) issue(t);
    run_block(kbA, 0, nA);
    if (U > nA) run_block(kbB, nA, U);
}

// ------------------------------------------------------------------ dQ
template <int DT, int DH, int NW, bool KL>
__global__ __launch_bounds__(64 * NW, (BwdTiles<DT, DH, NW, KL>::WPC_Q)) void attn_bwd_dq_dma_kernel(
    AttnBwdArgs a, float scale_log2, float inv_sqrt, int hpw, int nqt, int n_ht) {
    typedef BwdTiles<DT, DH, NW, KL> C;
    typedef Mma<DT> MM;
    typedef typename MM::operand opnd;
    typedef uint16_t elem;
    constexpr int NS = C::NS_Q;
    extern __shared__ __align__(16) unsigned char smem[];
    const lds_u8 *sm = (const lds_u8 *)smem;

    const int T = a.seq_len, Hq = a.n_heads;
    const int G = Hq / a.n_kv_heads;
    const int QT = 32 * NW / hpw;                      // queries per workgroup
    const int lin = xcd_remap(blockIdx.x, gridDim.x);
    const int qt = nqt - 1 - lin % nqt;                // longest query tiles first
    const int ht = (lin / nqt) % n_ht;
    const int b = lin / (nqt * n_ht);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, half = lane >> 5;
    const int h = ht * hpw + wave % hpw;
    const int kvh = h / G;
    const int q0 = qt * QT + (wave / hpw) * 32;        // first query of this wave
    const int qrow = q0 + (lane & 31);
    const int kend = min(T, qt * QT + QT);
    const int nblk = (kend + 31) / 32;
    const int jlast = q0 < T ? q0 / 32 : -1;           // the wave's diagonal block
    const int64_t row0 = (int64_t)b * T;
    const elem *Ks = static_cast<const elem *>(a.k) + row0 * a.ldq + kvh * DH;
    const elem *Vs = static_cast<const elem *>(a.v) + row0 * a.ldv + kvh * DH;
    const elem *Kts = KL ? static_cast<const elem *>(a.kt) + row0 * a.ldq + kvh * DH : nullptr;

    // this wave's queries as B operands of S^T = K Q^T and dP^T = V G^T (and of the teacher's
    // S_t^T = K_t Q_t^T)
    opnd qf[C::NKC], gf[C::NKC], qtf[KL ? C::NKC : 1];
    {
        const int qr = min(qrow, T - 1);
        const elem *qp = static_cast<const elem *>(a.q) + (row0 + qr) * a.ldq + h * DH + half * 8;
        const elem *gp = static_cast<const elem *>(a.g) + ((row0 + qr) * Hq + h) * DH + half * 8;
#pragma unroll
        for (int kc = 0; kc < C::NKC; ++kc) {
            u32x4 x = *reinterpret_cast<const u32x4 *>(qp + kc * 16);
            u32x4 y = *reinterpret_cast<const u32x4 *>(gp + kc * 16);
            if (qrow >= T) { x = u32x4{0u, 0u, 0u, 0u}; y = x; }
            qf[kc] = __builtin_bit_cast(opnd, x);
            gf[kc] = __builtin_bit_cast(opnd, y);
        }
        if constexpr (KL) {
            const elem *qtp = static_cast<const elem *>(a.qt) + (row0 + qr) * a.ldq + h * DH + half * 8;
#pragma unroll
            for (int kc = 0; kc < C::NKC; ++kc) {
                u32x4 x = *reinterpret_cast<const u32x4 *>(qtp + kc * 16);
                if (qrow >= T) x = u32x4{0u, 0u, 0u, 0u};
                qtf[kc] = __builtin_bit_cast(opnd, x);
            }
        }
    }
    const int64_t li = ((int64_t)b * Hq + h) * T + min(qrow, T - 1);
    const float lse = qrow < T ? a.lse2[li] : INFINITY;
    const float Dq = qrow < T ? a.D[li] : 0.f;
    const float lset = KL && qrow < T ? a.lse_t[li] : INFINITY;

    // ---- DMA: instruction i of this wave loads 1 KiB piece wave + NW i of the stage's K, V (and
    // teacher K) tiles (piece p lies in tile p / TI)
    constexpr int NP = C::Q_PW;
    int drow[NP], dcol[NP];
#pragma unroll
    for (int i = 0; i < NP; ++i) {
        quad_source((wave + NW * i) % C::TI, lane, drow[i], dcol[i]);
    }
    const int wofs = __builtin_amdgcn_readfirstlane(wave * 1024);
    auto issue = [&](int j) {
        if (j >= nblk) return;
        unsigned char *st = smem + (j % NS) * C::Q_STAGE + wofs;
#pragma unroll
        for (int i = 0; i < NP; ++i) {
            const int tix = (NW * i) / C::TI;
            const int k = min(32 * j + drow[i], T - 1);
            const elem *src = tix == 1 ? Vs + (k * a.ldv + dcol[i]) : (tix == 0 ? Ks : Kts) + (k * a.ldq + dcol[i]);
            lds_dma16((const void *)src, st + tix * C::TILE + ((NW * i) % C::TI) * 1024);
        }
    };

    const TileLanes tl(lane);
    f32x16 dqt[C::NDB];
#pragma unroll
    for (int d = 0; d < C::NDB; ++d)
#pragma unroll
        for (int e = 0; e < 16; ++e) dqt[d][e] = 0.f;

#pragma unroll
    for (int t = 0; t < NS - 1; ++t) issue(t);
    for (int j = 0; j < nblk; ++j) {
        wait_vm_groups<C::Q_PW, NS - 2>(min(NS - 2, nblk - 1 - j));
        raw_barrier();
        issue(j + NS - 1);
        if (j > jlast) continue;                       // keys above every query of the wave
        const lds_u8 *stk = sm + (j % NS) * C::Q_STAGE;
        const lds_u8 *stv = stk + C::TILE;
        // S^T = K Q^T, dP^T = V G^T: lane -> query, registers -> keys 8 (e / 4) + 4 half + e % 4
        f32x16 s, dp, st;
#pragma unroll
        for (int e = 0; e < 16; ++e) { s[e] = 0.f; dp[e] = 0.f; st[e] = 0.f; }
#pragma unroll
        for (int kc = 0; kc < C::NKC; ++kc) {
            s = MM::mma(row_frag<DT>(stk, tl, kc), qf[kc], s);
            dp = MM::mma(row_frag<DT>(stv, tl, kc), gf[kc], dp);
            if constexpr (KL) st = MM::mma(row_frag<DT>(stk + 2 * C::TILE, tl, kc), qtf[kc], st);
        }
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(s[e], scale_log2, -lse));
            float ds = p * (dp[e] - Dq);
            if constexpr (KL) {
                const float pt = __builtin_amdgcn_exp2f(__builtin_fmaf(st[e], scale_log2, -lset));
                ds = (ds + a.kl_scale * (p - pt)) * a.grad_scale;
            }
            dp[e] = ds;
        }
        if (j == jlast) {                              // the diagonal tile (wave-uniform) alone is masked
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int key = 32 * j + 8 * (e >> 2) + 4 * half + (e & 3);
                dp[e] = key > qrow ? 0.f : dp[e];
            }
        }
        // dQ^T += K^T dS^T (k = the tile's 32 keys in two steps)
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            const opnd sb = acc_operand<DT>(dp, ks);
#pragma unroll
            for (int d = 0; d < C::NDB; ++d) dqt[d] = MM::mma(tr_frag<DT>(stk, tl, ks, d), sb, dqt[d]);
        }
    }
    if (qrow < T) {
        elem *dyt = static_cast<elem *>(a.dyt) + row0 + qrow;
#pragma unroll
        for (int d = 0; d < C::NDB; ++d)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int c = d * 32 + 8 * (e >> 2) + 4 * half + (e & 3);
                dyt[(int64_t)(h * DH + c) * a.ldt] = from_f32<DT>(dqt[d][e] * inv_sqrt);
            }
    }
}

// ------------------------------------------------------------------ dQ from the stored dS
// dQ^T += K^T dS^T over the key tiles of the wave's queries, dS read back as the dK pass stored it
// (the operand of dK^T += Q^T dS: lane = key, eight queries per step).  The workgroup's waves share
// the kv head's key tiles (an LDS ring, as the recomputing kernel); each wave's dS tile rides the same
// stage and is read transposed (ds_read_b64_tr_b16) into the B operand of the dQ product: lane =
// query, keys 16 ks + 4 half + {0..3, 8..11}, the k-slots of tr_frag on the key tile.  The same
// product as the recomputing kernel, on the dK pass's dS.
template <int DT, int DH, int NW>
struct DqDsCfg {
    typedef BwdTiles<DT, DH, NW> B;
    static constexpr int NS = 3;                        // 48 KiB at head_dim 128: three workgroups per CU
    static constexpr int STAGE = B::TILE + NW * 2048;   // key tile | the waves' dS tiles
    static constexpr int PW = B::TI / NW + 2;            // DMA instructions per wave and stage
    static constexpr int WPC = NW == 4 ? 2 : 1;         // at least
    static_assert((size_t)NS * STAGE * WPC <= 160 * 1024, "LDS ring (dQ from dS)");
};

template <int DT, int DH, int NW>
__global__ __launch_bounds__(64 * NW, (DqDsCfg<DT, DH, NW>::WPC)) void attn_bwd_dq_ds_kernel(
    AttnBwdArgs a, float inv_sqrt, int hpw, int nqt, int n_ht) {
    typedef BwdTiles<DT, DH, NW> C;
    typedef DqDsCfg<DT, DH, NW> D;
    typedef Mma<DT> MM;
    typedef typename MM::operand opnd;
    typedef uint16_t elem;
    constexpr int NS = D::NS;
    extern __shared__ __align__(16) unsigned char smem[];
    const lds_u8 *sm = (const lds_u8 *)smem;

    const int T = a.seq_len, Hq = a.n_heads;
    const int G = Hq / a.n_kv_heads;
    const int QT = 32 * NW / hpw;                      // queries per workgroup
    const int lin = xcd_remap(blockIdx.x, gridDim.x);
    const int qt = nqt - 1 - lin % nqt;                // longest query tiles first
    const int ht = (lin / nqt) % n_ht;
    const int b = lin / (nqt * n_ht);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, half = lane >> 5;
    const int h = ht * hpw + wave % hpw;
    const int kvh = h / G;
    const int q0 = qt * QT + (wave / hpw) * 32;        // first query of this wave
    const int qrow = q0 + (lane & 31);
    const int kend = min(T, qt * QT + QT);
    const int nblk = (kend + 31) / 32;
    const int jlast = q0 < T ? q0 / 32 : -1;           // the wave's diagonal block
    const int64_t row0 = (int64_t)b * T;
    const elem *Ks = static_cast<const elem *>(a.k) + row0 * a.ldq + kvh * DH;
    const int nq = (T + 31) / 32;
    // the wave's dS tiles: (sequence b, head h, query tile q0 / 32, key tile j)
    const char *dsw = static_cast<const char *>(a.ds) +
                      (((int64_t)b * Hq + h) * (nq * (nq + 1) / 2) + (jlast >= 0 ? jlast * (jlast + 1) / 2 : 0)) * 2048;

    // ---- DMA: instruction i < TI / NW of this wave loads key-tile piece wave + NW i; the last two load
    // the wave's dS tile (blocks past its diagonal re-load the diagonal's, never read), its 16-byte
    // chunk c placed at chunk c ^ 8 (c >> 5 & 1) ^ 4 (c >> 6 & 1) of the wave's LDS area (an
    // involution) so the transposed reads below are free of bank conflicts
    constexpr int NK = C::TI / NW;
    int drow[NK], dcol[NK];
#pragma unroll
    for (int i = 0; i < NK; ++i) quad_source(wave + NW * i, lane, drow[i], dcol[i]);
    const int wofs = __builtin_amdgcn_readfirstlane(wave * 1024);
    const int dofs = __builtin_amdgcn_readfirstlane(C::TILE + wave * 2048);
    int dsrc[2];                                       // byte of the dS tile lane `lane` of piece i loads
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int pc = 64 * i + lane;
        dsrc[i] = (pc ^ (((pc >> 5) & 1) << 3) ^ (((pc >> 6) & 1) << 2)) * 16;
    }
    auto issue = [&](int j) {
        if (j >= nblk) return;
        unsigned char *st = smem + (j % NS) * D::STAGE;
#pragma unroll
        for (int i = 0; i < NK; ++i) {
            const int k = min(32 * j + drow[i], T - 1);
            lds_dma16((const void *)(Ks + (k * a.ldq + dcol[i])), st + wofs + NW * i * 1024);
        }
        // dS is read once: non-temporal, so it does not push the key tiles out of L2
        const char *src = dsw + (int64_t)min(j, max(jlast, 0)) * 2048;
#pragma unroll
        for (int i = 0; i < 2; ++i) lds_dma16_nt((const void *)(src + dsrc[i]), st + dofs + i * 1024);
    };

    // transposed reads of the dS tile: read rr of k-step ks, lane a + 4 s of its 16-lane group g:
    // key 16 ks + 4 (g / 2) + 8 rr + s, queries 16 (g % 2) + 4 a .. + 3, stored as chunk
    // c = 64 (g % 2) + 32 (a % 2) + key (16 bytes, the query pairs at 8 (a / 2) within it), which
    // the DMA placed at chunk c ^ 8 (a % 2) ^ 4 (g % 2)
    const int jg = lane & 15, ta = jg & 3, ts = jg >> 2, tg = lane >> 4;
    int dsoff[2];
#pragma unroll
    for (int rr = 0; rr < 2; ++rr)
        dsoff[rr] = (64 * (tg & 1) + 32 * (ta & 1) + 8 * ((ta & 1) ^ rr) + 4 * ((tg >> 1) ^ (tg & 1)) + ts) * 16 +
                    8 * (ta >> 1);
    const TileLanes tl(lane);
    f32x16 dqt[C::NDB];
#pragma unroll
    for (int d = 0; d < C::NDB; ++d)
#pragma unroll
        for (int e = 0; e < 16; ++e) dqt[d][e] = 0.f;

#pragma unroll
    for (int t = 0; t < NS - 1; ++t) issue(t);
    for (int j = 0; j < nblk; ++j) {
        wait_vm_groups<D::PW, NS - 2>(min(NS - 2, nblk - 1 - j));
        raw_barrier();
        issue(j + NS - 1);
        if (j > jlast) continue;                       // keys above every query of the wave
        const lds_u8 *stk = sm + (j % NS) * D::STAGE;
        const lds_u8 *std_ = stk + C::TILE + wave * 2048;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            const s16x4 lo = lds_read_tr16(std_ + dsoff[0] + ks * 256);
            const s16x4 hi = lds_read_tr16(std_ + dsoff[1] + ks * 256);
            const opnd sb = __builtin_bit_cast(opnd, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
            for (int d = 0; d < C::NDB; ++d) dqt[d] = MM::mma(tr_frag<DT>(stk, tl, ks, d), sb, dqt[d]);
        }
    }
    if (qrow < T) {
        elem *dyt = static_cast<elem *>(a.dyt) + row0 + qrow;
#pragma unroll
        for (int d = 0; d < C::NDB; ++d)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int c = d * 32 + 8 * (e >> 2) + 4 * half + (e & 3);
                dyt[(int64_t)(h * DH + c) * a.ldt] = from_f32<DT>(dqt[d][e] * inv_sqrt);
            }
    }
}

}  // namespace

// dK/dV and dQ for the 16-bit dtypes at head_dim 64 / 128 (KL: with the KL term's gradient)
template <int DT, int DH, bool KL>
hipError_t run_bwd_dma_kl(const AttnBwdArgs &a, hipStream_t st) {
    constexpr int NW = 4;
    typedef BwdTiles<DT, DH, NW, KL> C;
    const int T = a.seq_len;
    // per-sequence element offsets are 32-bit
    if ((int64_t)T * a.ldq >= (1ll << 31) || (int64_t)T * a.ldv >= (1ll << 31) ||
        (int64_t)T * a.n_heads * DH >= (1ll << 31))
        return hipErrorInvalidValue;
    const float scale_log2 = 1.4426950408889634f / sqrtf((float)DH);
    const float inv_sqrt = 1.f / sqrtf((float)DH);
    const size_t q_lds = (size_t)C::NS_Q * C::Q_STAGE;
    hipError_t e = hipFuncSetAttribute((const void *)attn_bwd_dq_dma_kernel<DT, DH, NW, KL>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)q_lds);
    if (e != hipSuccess) return e;
    const int nkb = (T + 32 * NW - 1) / (32 * NW);
    const int npair = (nkb + 1) / 2;
    const dim3 kv_grid(npair * a.n_kv_heads * a.batch);
    // dK and dV in one pass; with the KL term, dV alone (it does not see the map's KL part) and then
    // dK with the KL part, each at two workgroups per CU
    auto dkdv_ds = [&](auto kl_c, auto mode_c, auto ds_c) -> hipError_t {
        constexpr bool K2 = decltype(kl_c)::value;
        constexpr int MODE = decltype(mode_c)::value;
        constexpr bool DS = decltype(ds_c)::value;
        typedef BwdTiles<DT, DH, NW, K2, MODE> CM;
        const size_t lds = (size_t)CM::NS_KV * CM::KV_STAGE;
        hipError_t err = hipFuncSetAttribute((const void *)attn_bwd_dkdv_dma_kernel<DT, DH, NW, K2, MODE, DS>,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (err != hipSuccess) return err;
        attn_bwd_dkdv_dma_kernel<DT, DH, NW, K2, MODE, DS><<<kv_grid, dim3(64 * NW), lds, st>>>(
            a, scale_log2, inv_sqrt, nkb, npair);
        return hipGetLastError();
    };
    // the pass that computes dK stores dS when the caller gave it room
    auto dkdv = [&](auto kl_c, auto mode_c) -> hipError_t {
        if constexpr (decltype(mode_c)::value != 1)
            if (a.ds) return dkdv_ds(kl_c, mode_c, std::true_type());
        return dkdv_ds(kl_c, mode_c, std::false_type());
    };
    if constexpr (KL) {
        e = dkdv(std::false_type(), std::integral_constant<int, 1>());
        if (e == hipSuccess) e = dkdv(std::true_type(), std::integral_constant<int, 2>());
    } else {
        e = dkdv(std::false_type(), std::integral_constant<int, 0>());
    }
    if (e != hipSuccess) return e;
    const int G = a.n_heads / a.n_kv_heads;
    const int hpw = G % NW == 0 ? NW : G;              // query heads per workgroup
    const int QT = 32 * NW / hpw;
    const int nqt = (T + QT - 1) / QT;
    const int n_ht = a.n_heads / hpw;
    if (a.ds) {   // dQ from the dS the dK pass stored
        typedef DqDsCfg<DT, DH, NW> DC;
        const size_t lds = (size_t)DC::NS * DC::STAGE;
        e = hipFuncSetAttribute((const void *)attn_bwd_dq_ds_kernel<DT, DH, NW>,
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
        attn_bwd_dq_ds_kernel<DT, DH, NW><<<dim3(nqt * n_ht * a.batch), dim3(64 * NW), lds, st>>>(
            a, inv_sqrt, hpw, nqt, n_ht);
        return hipGetLastError();
    }
    attn_bwd_dq_dma_kernel<DT, DH, NW, KL><<<dim3(nqt * n_ht * a.batch), dim3(64 * NW), q_lds, st>>>(
        a, scale_log2, inv_sqrt, hpw, nqt, n_ht);
    return hipGetLastError();
}

template <int DT, int DH>
hipError_t run_bwd_dma(const AttnBwdArgs &a, hipStream_t st) {
    if (a.qt) return run_bwd_dma_kl<DT, DH, true>(a, st);
    return run_bwd_dma_kl<DT, DH, false>(a, st);
}

template hipError_t run_bwd_dma<F16, 64>(const AttnBwdArgs &, hipStream_t);
template hipError_t run_bwd_dma<F16, 128>(const AttnBwdArgs &, hipStream_t);
template hipError_t run_bwd_dma<BF16, 64>(const AttnBwdArgs &, hipStream_t);
template hipError_t run_bwd_dma<BF16, 128>(const AttnBwdArgs &, hipStream_t);

}  // namespace jab
