// gemm.hip -- projection GEMM of the fused QKV weight on the matrix cores.
//
// Paper: Method, "Layer-wise PTQ": y = x W with the QKV projection fused as
// W = [W_Q | W_K | W_V].  Here C[m][n] = sum_k A[m][k] B[n][k] with A = X
// [tokens][d_model] and B = W_hat [R][d_model] (one row per output channel), both
// k-contiguous, accumulated in fp32 and stored in the storage dtype.
//
// gfx950 design (16-bit dtypes, gemm_w4_kernel)
//  * 256 threads = 4 wavefronts in a 2 x 2 arrangement, one wave per SIMD; a workgroup
//    computes a 256 x 256 tile, each wave 128 x 128 as 4 x 4 blocks of
//    v_mfma_f32_32x32x16_{bf16,f16} (256 accumulator registers).  Per k-step a wave reads
//    4 + 4 operand fragments for 16 MFMAs, two thirds of the LDS traffic per flop of a
//    128 x 64 wave tile.
//  * k-tiles of 64 go straight from global memory into LDS (buffer_load_dwordx4 ... lds: a
//    scalar resource and k offset, one fixed per-lane offset per instruction, so no vector
//    address arithmetic) through two 64 KiB stages.  The MUBUF form keeps the LDS counter
//    ordered, so each MFMA waits only for its own fragments.
//  * One barrier per stage, before its last k-step.  The stage's refill is spread over that
//    k-step and the first k-step of the next stage (the other slot is being read then): the
//    vector-memory path cannot take all of a stage's loads in one k-step without stalling
//    the wave that issues them.
//  * Fragment reads for the next k-step are issued every other MFMA slot; 16-byte chunks
//    are XOR-swizzled per row so the 16 rows served per LDS cycle hit distinct banks.
//  * The MFMA operands are swapped (B first), so a lane's accumulators hold four
//    consecutive output columns of one row.  Storage-dtype outputs go through LDS (the ring
//    is free after the k loop) and leave as whole 512-byte rows; the transposed value
//    output and fp32 outputs are stored from registers, 8 and 16 bytes per lane.
//  * Workgroup ids are remapped so that each XCD (ids congruent mod 8 land on the same
//    XCD) walks a contiguous range of tiles, grouped 8 M-tiles at a time so that
//    concurrently running tiles share A and B panels in that XCD's L2.
//  * fp32 inputs use gemm_nt_kernel (4 waves, 128 x 128 tiles, v_mfma_f32_32x32x2_f32).
#include <map>
#include <mutex>
#include <utility>

#include "device_common.h"
#include "kernels.h"
#include "lds_pipe.h"


namespace jab {
namespace {

template <int DT, int BM, int BN, int NS, int CPR_ = 4, int NW_ = 4>
struct GemmCfg {
    typedef typename Mma<DT>::elem elem;
    static constexpr int EPC = 16 / (int)sizeof(elem);  // elements per 16-byte chunk
    static constexpr int CPR = CPR_;                    // chunks per k-tile row (4: 64 bytes, 8: 128 bytes)
    static constexpr int BK = CPR * EPC;                // k elements per stage
    static constexpr int NW = NW_;                      // waves per workgroup: a 2 x NW/2 grid
    static constexpr int WM = BM / 2, WN = BN / (NW / 2);
    static constexpr int FM = WM / 32, FN = WN / 32;
    static constexpr int KS = BK / Mma<DT>::K;          // MFMA k-steps per stage
    static constexpr int IA = BM * CPR / 64 / NW, IB = BN * CPR / 64 / NW;   // loads per wave per stage
    static constexpr int STAGE_BYTES = (BM + BN) * CPR * 16;
    static constexpr size_t LDS_BYTES = (size_t)NS * STAGE_BYTES;
};

// Physical 16-byte chunk of logical chunk c in row r of a k-tile row of CPR chunks.  A
// 16-byte-per-lane LDS read is served 16 lanes (256 bytes, the 64 banks) at a time; the
// 16 rows such a group touches would collide on a few bank positions, so the chunk index
// is rotated per row: by (r/4) mod 4 for 64-byte rows, by (r/2) mod 8 for 128-byte rows,
// which spreads each group over all 16 slots.
template <int CPR>
__device__ inline int swz(int r, int c) {
    if constexpr (CPR == 4) return c ^ ((r >> 2) & 3);
    else return c ^ ((r >> 1) & 7);
}

// Output modes:
//   OUT_DT : C[m][n] in the storage dtype
//   OUT_F32: C[m][n] = alpha * (A B^T) in fp32
//   OUT_VT : values transposed for the attention kernel, C[m][pos(n)] in the storage
//            dtype, where column n is the token index b*T + t of a batch of sequences of
//            length T; pos(n) = b*Tp + perm(t), Tp = T rounded up to 32, and perm swaps
//            bits 2 and 3 of t inside each block of 32 tokens (the key order in which an
//            MFMA lane consumes softmax probabilities, so each lane's eight keys are one
//            contiguous 16-byte read).
enum { OUT_DT = 0, OUT_F32 = 1, OUT_VT = 2 };

template <int DT, int BM, int BN, int NS, int MINB, int OUT, int CPR, int NW>
__global__ __launch_bounds__(64 * NW, MINB) void gemm_nt_kernel(const void *__restrict__ Ap,
                                                          const void *__restrict__ Bp,
                                                          void *__restrict__ Cp, int M, int N, int K,
                                                          int lda, int ldb, int ldc, int tiles_m,
                                                          int tiles_n, float alpha, int seq_T,
                                                          int seq_Tp, int ksplit, void *__restrict__ Cp2) {
    typedef GemmCfg<DT, BM, BN, NS, CPR, NW> G;
    typedef typename G::elem elem;
    typedef Mma<DT> MM;
    extern __shared__ __align__(16) unsigned char smem[];

    const elem *A = static_cast<const elem *>(Ap);
    const elem *B = static_cast<const elem *>(Bp);

    // ---- tile order: XCD-contiguous ranges, then groups of 8 M-tiles
    const int nwg = gridDim.x;
    int pid = blockIdx.x;
    if ((nwg & 7) == 0)
        pid = (pid & 7) * (nwg >> 3) + (pid >> 3);
    // split-K: workgroups past the tile count take the second half of k into the second output
    const int split = pid / (tiles_m * tiles_n);
    pid -= split * tiles_m * tiles_n;
    if (split) {
        Cp = Cp2;
        A += (int64_t)(K / ksplit);
        B += (int64_t)(K / ksplit);
    }
    const int group_tiles = 8 * tiles_n;
    const int first_m = (pid / group_tiles) * 8;
    const int gsz = min(tiles_m - first_m, 8);
    const int pm = first_m + (pid % group_tiles) % gsz;
    const int pn = (pid % group_tiles) / gsz;
    const int bm0 = pm * BM, bn0 = pn * BN;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm0 = (wave / (NW / 2)) * G::WM, wn0 = (wave % (NW / 2)) * G::WN;

    // ---- per-lane global source of each direct-to-LDS load.  A wave instruction fills
    // 64 consecutive chunks (1 KiB) of the stage; chunk p holds row p/4, physical chunk
    // p%4, i.e. logical chunk swz(row, p%4).  Rows past the matrix edge are clamped to
    // the last row: they only feed output rows / columns that are never stored.
    const elem *srcA[G::IA], *srcB[G::IB];
#pragma unroll
    for (int i = 0; i < G::IA; ++i) {
        const int p = (wave + NW * i) * 64 + lane, r = p / CPR;
        const int row = min(bm0 + r, M - 1);
        srcA[i] = A + (int64_t)row * lda + swz<CPR>(r, p % CPR) * G::EPC;
    }
#pragma unroll
    for (int i = 0; i < G::IB; ++i) {
        const int p = (wave + NW * i) * 64 + lane, r = p / CPR;
        const int row = min(bn0 + r, N - 1);
        srcB[i] = B + (int64_t)row * ldb + swz<CPR>(r, p % CPR) * G::EPC;
    }

    f32x16 acc[G::FM][G::FN];
#pragma unroll
    for (int i = 0; i < G::FM; ++i)
#pragma unroll
        for (int j = 0; j < G::FN; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

    // ---- operand fetch from LDS for k-step ks of a stage
    auto frag = [&](const unsigned char *S, int r, int ks) -> typename MM::operand {
        if constexpr (DT == F32) {
            const int k = ks * MM::K + (lane >> 5);          // one element per lane
            const float *p = reinterpret_cast<const float *>(S + (r * CPR + swz<CPR>(r, k >> 2)) * 16);
            return p[k & 3];
        } else {
            const int c = ks * 2 + (lane >> 5);               // eight elements per lane
            const u32x4 v = *reinterpret_cast<const u32x4 *>(S + (r * CPR + swz<CPR>(r, c)) * 16);
            return __builtin_bit_cast(typename MM::operand, v);
        }
    };

    const int nk = K / G::BK / ksplit;                       // K is a multiple of ksplit * BK
    // A stage is split into U units of KU k-steps (one unit = 16 MFMAs of 32x32 for the
    // 16-bit dtypes).  Unit fragments are double-buffered in registers.
    constexpr int KU0 = 16 / (G::FM * G::FN) > 0 ? 16 / (G::FM * G::FN) : 1;
    constexpr int KU = KU0 < G::KS / 2 ? KU0 : G::KS / 2;
    constexpr int U = G::KS / KU;
    static_assert(G::KS % KU == 0 && U >= 2 && U % 2 == 0, "a stage holds an even number of units");
    constexpr int PS = G::IA + G::IB;                        // load instructions per wave per stage
    constexpr int NREAD = KU * (G::FM + G::FN);              // fragment reads per unit
    constexpr int NMMA = KU * G::FM * G::FN;                 // MFMAs per unit
    constexpr int NSLOT = NMMA > NREAD ? (NMMA > PS ? NMMA : PS) : (NREAD > PS ? NREAD : PS);
    typename MM::operand fa[2][KU][G::FM], fb[2][KU][G::FN];
    // r-th fragment read of unit u of a stage, in the order the MFMAs consume them:
    // per k-step a[0], b[0..FN-1], a[1..FM-1].
    auto read_one = [&](const unsigned char *S, int u, int r, int buf) {
        const int k = r / (G::FM + G::FN), q = r % (G::FM + G::FN), ks = u * KU + k;
        if (q == 0)
            fa[buf][k][0] = frag(S, wm0 + (lane & 31), ks);
        else if (q <= G::FN)
            fb[buf][k][q - 1] = frag(S + BM * CPR * 16, wn0 + 32 * (q - 1) + (lane & 31), ks);
        else
            fa[buf][k][q - G::FN] = frag(S, wm0 + 32 * (q - G::FN) + (lane & 31), ks);
    };
    auto mma_one = [&](int m, int buf) {
        const int k = m / (G::FM * G::FN), i = (m / G::FN) % G::FM, j = m % G::FN;
        acc[i][j] = MM::mma(fa[buf][k][i], fb[buf][k][j], acc[i][j]);
    };
    // one direct-to-LDS load instruction of k-tile `ktile` into stage slot `slot`
    auto issue_one = [&](int idx, int ktile, int slot) {
        unsigned char *st = smem + (slot % NS) * G::STAGE_BYTES;
        const int k0 = (ktile < nk ? ktile : nk - 1) * G::BK;   // past K: harmless re-load
        if (idx < G::IA)
            lds_dma16((const void *)(srcA[idx] + k0), st + (wave + NW * idx) * 1024);
        else
            lds_dma16((const void *)(srcB[idx - G::IA] + k0), st + BM * CPR * 16 + (wave + NW * (idx - G::IA)) * 1024);
    };

    // Branch-free steady state with an explicit instruction order: each MFMA slot of a
    // unit carries at most one LDS fragment read (of the next unit) and one
    // global->LDS load, fenced by sched_barrier, so the matrix core never waits on a
    // block of memory instructions.  One barrier per stage, before its last unit: by then
    // every wave has read (and waited for) all fragments of the stage, so its slot is
    // refilled with k-tile kt+NS right away, and the next stage has landed.
#pragma unroll
    for (int s0 = 0; s0 < NS; ++s0)
#pragma unroll
        for (int i = 0; i < PS; ++i) issue_one(i, s0, s0);
    wait_vmcnt<(NS - 1) * PS>();
    raw_barrier();
#pragma unroll
    for (int r = 0; r < NREAD; ++r) read_one(smem, 0, r, 0);
    for (int kt = 0; kt < nk; ++kt) {
        const unsigned char *S = smem + (kt % NS) * G::STAGE_BYTES;
        const unsigned char *Sn = smem + ((kt + 1) % NS) * G::STAGE_BYTES;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int cur = u & 1;
            if (u == U - 1) {
                wait_lgkm0();                                 // this stage's reads are done
                wait_vmcnt<(NS - 2) * PS>();                  // k-tile kt+1 has landed
                raw_barrier();
            }
#pragma unroll
            for (int m = 0; m < NSLOT; ++m) {
                if (m < NMMA) mma_one(m, cur);
                if (m < NREAD) {
                    if (u < U - 1) read_one(S, u + 1, m, cur ^ 1);
                    else read_one(Sn, 0, m, cur ^ 1);
                }
                if (u == U - 1 && m < PS) issue_one(m, kt + NS, kt);   // refill this stage's slot
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    }
    wait_vmcnt<0>();

    // ---- epilogue: D layout -> C rows / columns
#pragma unroll
    for (int i = 0; i < G::FM; ++i) {
#pragma unroll
        for (int j = 0; j < G::FN; ++j) {
            const int col = bn0 + wn0 + 32 * j + (lane & 31);
            if (col >= N) continue;
            int64_t ccol = col;
            if constexpr (OUT == OUT_VT)
                ccol = (int64_t)(col / seq_T) * seq_Tp + vt_perm(col % seq_T);
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int row = bm0 + wm0 + 32 * i + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
                if (row < M) {
                    if constexpr (OUT == OUT_F32)
                        static_cast<float *>(Cp)[(int64_t)row * ldc + ccol] = alpha * acc[i][j][e];
                    else
                        static_cast<elem *>(Cp)[(int64_t)row * ldc + ccol] = from_f32<DT>(acc[i][j][e]);
                }
            }
        }
    }
}

// ---------------------------------------------------------------- 16-bit dtypes
// XOR key of LDS row r (16-byte chunks of a row of CPR chunks): rotates the chunk index so the
// 16 rows one LDS cycle serves land on 16 distinct chunk slots
template <int CPR>
__device__ inline int w4_key(int r) {
    if constexpr (CPR == 8) return (r >> 1) & 7;
    else return (r >> 2) & 3;
}

// C tile staged in LDS for the storage-dtype output: 256 rows of 512 bytes; the 16-byte chunk c
// of row m sits at chunk c ^ (m & 15) and its two 8-byte halves are exchanged when bit 4 of m is
// set, so the 32 rows written by one half-wave (same logical half-chunk) cover all 64 banks and
// a row read back by 32 lanes is conflict-free too.
__device__ inline int ctile_off(int m, int c, int h) {
    return m * 512 + ((c ^ (m & 15)) << 4) + ((h ^ ((m >> 4) & 1)) << 3);
}

template <int DT, int OUT, int CPR>
__global__ __launch_bounds__(256, 1) void gemm_w4_kernel(const void *__restrict__ Ap, const void *__restrict__ Bp,
                                                         void *__restrict__ Cp, int M, int N, int K, int lda,
                                                         int ldb, int ldc, int tiles_m, int tiles_n, float alpha,
                                                         int seq_T, int seq_Tp, int ksplit, void *__restrict__ Cp2) {
    typedef typename Mma<DT>::elem elem;
    typedef typename Mma<DT>::operand opnd;
    constexpr int BK = CPR * 8;               // k elements per stage
    constexpr int U = BK / 16;                // k-steps per stage
    constexpr int ROWB = CPR * 16;            // bytes per LDS row of a stage
    constexpr int HALF = 256 * ROWB;          // bytes of the A part of a stage (B follows)
    constexpr int STAGE = 2 * HALF;
    constexpr int NS = 2;                     // stages in the ring
    constexpr int DPW = 2 * 256 * CPR / 64 / 4;   // DMA instructions per wave per stage (A, then B)
    constexpr int DPA = DPW / 2;
    constexpr int RPI = 64 / CPR;             // rows per DMA instruction
    // k-steps over which a stage refill is spread: two when a stage has four (the second part then
    // still lands two k-steps before it is waited for), else one
    constexpr int SPR = U >= 4 ? 2 : 1;
    constexpr int PER = DPW / SPR;            // refill instructions per k-step
    static_assert(SPR <= U && 16 % PER == 0 && DPW % SPR == 0, "refill spread");
    extern __shared__ __align__(16) unsigned char smem[];

    // ---- tile order: XCD-contiguous ranges, then groups of 8 M-tiles; split-K halves
    const int nwg = gridDim.x;
    int pid = blockIdx.x;
    if ((nwg & 7) == 0) pid = (pid & 7) * (nwg >> 3) + (pid >> 3);
    const int split = pid / (tiles_m * tiles_n);
    pid -= split * tiles_m * tiles_n;
    const int k_begin = split * (K / ksplit);
    if (split) Cp = Cp2;
    const int group_tiles = 8 * tiles_n;
    const int first_m = (pid / group_tiles) * 8;
    const int gsz = min(tiles_m - first_m, 8);
    const int pm = first_m + (pid % group_tiles) % gsz;
    const int pn = (pid % group_tiles) / gsz;
    const int bm0 = pm * 256, bn0 = pn * 256;

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int wr = wave >> 1, wc = wave & 1;
    const int half = lane >> 5, l32 = lane & 31;

    // ---- DMA sources.  Instruction d < DPA of this wave fills rows RPI (wave + 4 d) .. + RPI - 1
    // of the A part (d >= DPA: of the B part); lane i writes row + i / CPR, physical chunk i % CPR,
    // which holds logical chunk (i % CPR) ^ key(row).  Rows past the matrix edge read the last
    // row: they only feed outputs that are never stored.
    const char *Ab = static_cast<const char *>(Ap) + ((int64_t)bm0 * lda + k_begin) * (int64_t)sizeof(elem);
    const char *Bb = static_cast<const char *>(Bp) + ((int64_t)bn0 * ldb + k_begin) * (int64_t)sizeof(elem);
    const i32x4 rsA = buffer_rsrc(Ab), rsB = buffer_rsrc(Bb);
    uint32_t voffA[DPA], voffB[DPA];
#pragma unroll
    for (int i = 0; i < DPA; ++i) {
        const int r = RPI * (wave + 4 * i) + lane / CPR, pc = lane % CPR;
        const int c = pc ^ w4_key<CPR>(r);
        const int ra = min(bm0 + r, M - 1) - bm0, rb = min(bn0 + r, N - 1) - bn0;
        voffA[i] = (uint32_t)(ra * lda * 2 + c * 16);
        voffB[i] = (uint32_t)(rb * ldb * 2 + c * 16);
    }
    const int nk = K / BK / ksplit;
    // d-th DMA instruction of this wave for k-tile `ktile` into ring slot `slot` (k-tiles past the
    // end re-load the last one into a slot that is never read)
    auto issue = [&](int d, int ktile, int slot) {
        const int kk = (ktile < nk ? ktile : nk - 1) * BK * 2;
        unsigned char *st = smem + slot * STAGE;
        if (d < DPA) buffer_dma16(rsA, voffA[d], kk, st + (wave + 4 * d) * 1024);
        else buffer_dma16(rsB, voffB[d - DPA], kk, st + HALF + (wave + 4 * (d - DPA)) * 1024);
    };

    // ---- fragment reads: lane row l32 of the wave's rows, logical chunk 2 ks + half.  The XOR key
    // of a row depends only on l32, so the four A (B) fragments of a k-step are one per-lane base
    // plus constant offsets.
    const int key = w4_key<CPR>(l32);
    uint32_t rda[U], rdb[U];
#pragma unroll
    for (int ks = 0; ks < U; ++ks) {
        const int pc = (2 * ks + half) ^ key;
        rda[ks] = (uint32_t)((wr * 128 + l32) * ROWB + pc * 16);
        rdb[ks] = (uint32_t)(HALF + (wc * 128 + l32) * ROWB + pc * 16);
    }
    opnd fa[2][4], fb[2][4];
    // r-th fragment read of a k-step, in the order the MFMAs consume them: a0, b0..b3, a1..a3
    auto rd = [&](int r, int slot, int ks, int buf) {
        const unsigned char *base = smem + slot * STAGE;
        if (r == 0) fa[buf][0] = __builtin_bit_cast(opnd, *(const u32x4 *)(base + rda[ks]));
        else if (r <= 4) fb[buf][r - 1] = __builtin_bit_cast(opnd, *(const u32x4 *)(base + rdb[ks] + (r - 1) * 32 * ROWB));
        else fa[buf][r - 4] = __builtin_bit_cast(opnd, *(const u32x4 *)(base + rda[ks] + (r - 4) * 32 * ROWB));
    };

    f32x16 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

#pragma unroll
    for (int s0 = 0; s0 < NS; ++s0)
#pragma unroll
        for (int d = 0; d < DPW; ++d) issue(d, s0, s0);
    wait_vmcnt<DPW>();
    raw_barrier();
#pragma unroll
    for (int r = 0; r < 8; ++r) rd(r, 0, 0, 0);

    // Steady state.  k-step u of stage kt: 16 MFMAs (acc[i][j] += B_j A_i, swapped so a lane's
    // accumulators run along output columns), a fragment read of the next k-step every other
    // MFMA slot, and refill loads.  Before the last k-step, one barrier: every wave has read
    // (and waited for) the stage's other fragments, and stage kt+1 has landed; the stage's slot
    // is refilled with k-tile kt+2 over that k-step and the first k-step of stage kt+1.
    int slot = 0;
    for (int kt = 0; kt < nk; ++kt) {
        const int nslot = slot ^ 1;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int cur = u & 1;
            if (u == U - 1) {
                wait_lgkm0();
                wait_vmcnt<0>();
                raw_barrier();
            }
#pragma unroll
            for (int m = 0; m < 16; ++m) {
                const int i = m >> 2, j = m & 3;
                acc[i][j] = Mma<DT>::mma(fb[cur][j], fa[cur][i], acc[i][j]);
                if ((m & 1) == 0) {
                    if (u < U - 1) rd(m >> 1, slot, u + 1, cur ^ 1);
                    else rd(m >> 1, nslot, 0, cur ^ 1);
                }
                constexpr int ST = 16 / PER;
                if (m % ST == 0) {
                    if (u == U - 1) issue(m / ST, kt + NS, slot);
                    else if (u + 1 < SPR && kt > 0) issue((u + 1) * PER + m / ST, kt - 1 + NS, nslot);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        slot = nslot;
    }
    wait_vmcnt<0>();

    // ---- epilogue.  acc[i][j][4 g + t] = C[row][col + t] with row = wr*128 + 32 i + l32 and
    // col = wc*128 + 32 j + 8 g + 4 half (tile coordinates).
    // Storage-dtype outputs go through LDS when every 32-token block of the transposed value output
    // lies inside one sequence (T a multiple of 32): the tile is written to LDS in destination
    // order and leaves as whole rows.
    if (OUT == OUT_DT || (OUT == OUT_VT && (seq_T & 31) == 0)) {
        // every wave's loads and fragment reads are done before the ring is reused
        wait_lgkm0();
        raw_barrier();
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int m = wr * 128 + 32 * i + l32;
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const uint32_t lo = pack2<DT>(acc[i][j][4 * g], acc[i][j][4 * g + 1]);
                    const uint32_t hi = pack2<DT>(acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]);
                    // tile column wc*128 + 32 j + 8 g + 4 half (+0..3); for the value output its
                    // position inside the 32-token block has bits 2 and 3 exchanged
                    const int c = OUT == OUT_DT ? 16 * wc + 4 * j + g : 16 * wc + 4 * j + 2 * (g >> 1) + half;
                    const int h = OUT == OUT_DT ? half : (g & 1);
                    *reinterpret_cast<uint2 *>(smem + ctile_off(m, c, h)) = make_uint2(lo, hi);
                }
        }
        wait_lgkm0();
        raw_barrier();
        // 32 rounds of 2 rows x 32 chunks: one store instruction writes two whole 512-byte rows.
        // A lane keeps its chunk c (8 columns) in every round.
        const int c = lane & 31;
        int64_t dcol;
        int ncol;                                  // valid columns of the chunk
        if constexpr (OUT == OUT_DT) {
            dcol = bn0 + 8 * c;
            ncol = min(8, N - (bn0 + 8 * c));
        } else {
            const int n = bn0 + 8 * c;             // tokens of this chunk's 32-block start at n & ~31
            const int sb = n / seq_T;
            dcol = (int64_t)sb * seq_Tp + (n - sb * seq_T);
            ncol = min(8, N - n);
        }
#pragma unroll 4
        for (int it = 0; it < 32; ++it) {
            const int m = it * 8 + wave * 2 + half;
            u32x4 v = *reinterpret_cast<const u32x4 *>(smem + ctile_off(m, c, 0) - ((((m >> 4) & 1)) << 3));
            if ((m >> 4) & 1) v = u32x4{v[2], v[3], v[0], v[1]};
            const int row = bm0 + m;
            if (row >= M || ncol <= 0) continue;
            elem *dst = static_cast<elem *>(Cp) + (int64_t)row * ldc + dcol;
            if (ncol == 8) {
                *reinterpret_cast<u32x4 *>(dst) = v;
            } else {
                for (int t = 0; t < ncol; ++t) dst[t] = (elem)(v[t >> 1] >> (16 * (t & 1)));
            }
        }
        return;
    }
    if constexpr (OUT == OUT_DT) {
        return;
    } else if constexpr (OUT == OUT_F32) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int row = bm0 + wr * 128 + 32 * i + l32;
            if (row >= M) continue;
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int col = bn0 + wc * 128 + 32 * j + 8 * g + 4 * half;   // columns col .. col + 3
                    if (col >= N) continue;
                    float *dst = static_cast<float *>(Cp) + (int64_t)row * ldc + col;
                    const f32x4 v = f32x4{alpha * acc[i][j][4 * g], alpha * acc[i][j][4 * g + 1],
                                          alpha * acc[i][j][4 * g + 2], alpha * acc[i][j][4 * g + 3]};
                    if (col + 4 <= N) {
                        *reinterpret_cast<f32x4 *>(dst) = v;
                    } else {
                        for (int t = 0; t < 4 && col + t < N; ++t) dst[t] = v[t];
                    }
                }
        }
    } else {
        // Column n = token b*T + t goes to b*Tp + perm(t).  With T a multiple of 4, four consecutive
        // tokens starting at a multiple of 4 stay in one sequence and in order (perm leaves bits 0
        // and 1 alone): one 8-byte store at the position of the first.
        const bool quad = (seq_T & 3) == 0;
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int col = bn0 + wc * 128 + 32 * j + 8 * g + 4 * half;
                if (col >= N) continue;
                const int sb = col / seq_T;
                const int dcol = sb * seq_Tp + vt_perm(col - sb * seq_T);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int row = bm0 + wr * 128 + 32 * i + l32;
                    if (row >= M) continue;
                    elem *base = static_cast<elem *>(Cp) + (int64_t)row * ldc;
                    if (quad && col + 4 <= N) {
                        const uint32_t lo = pack2<DT>(acc[i][j][4 * g], acc[i][j][4 * g + 1]);
                        const uint32_t hi = pack2<DT>(acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]);
                        *reinterpret_cast<uint2 *>(base + dcol) = make_uint2(lo, hi);
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const int n = col + e;
                            if (n < N) {
                                const int nb = n / seq_T;
                                base[nb * seq_Tp + vt_perm(n - nb * seq_T)] = from_f32<DT>(acc[i][j][4 * g + e]);
                            }
                        }
                    }
                }
            }
    }
}

// Persistent form of gemm_w4_kernel for the storage-dtype and transposed-value outputs: one
// workgroup per CU walks the tiles blockIdx.x, + gridDim.x, ... (in the same remapped order).  The
// operand that streams the tokens has an LDS ring of three k-tiles, the weights one of two (160 KiB
// at k-tiles of 64).  The rings run on across tiles: the refills of a tile's last stages bring the
// next tile's first two k-tiles, and the last stage's fragment reads already fetch its first k-step, so
// between two tiles only the epilogue remains; it stores from registers (16 bytes per lane) while
// the next tile's loads are in flight.  A tile is always whole: the last tile of a ragged M (N) is
// moved back to end at M (N), so the per-lane load offsets are the same for every tile (rows or
// columns it shares with its neighbour are written twice with the same values, the same products
// summed in the same order).  Needs M, N >= 256, at least three k-tiles, and for OUT_VT T a multiple
// of 32.
// RDH > 0 (storage-dtype output only): every output column belongs to a query or key head of
// RDH columns, rotated by the rotary embedding in the epilogue (see below).
// OUT_F32: alpha (A B^T) in fp32, K split in ksplit equal parts (work item w: tile w mod tiles,
// part w / tiles, written to Cp for part 0 and Cp2 for part 1).
// queue (grid a multiple of 8, at least six k-tiles per work item; else null and the static order
// above): the work items after the first are taken at run time, so that the XCDs that run faster
// take more of them.  XCD x (workgroups congruent to x mod 8) owns the items congruent to x mod 8
// (the static order's, so the L2 of an XCD still sees its own panels) and takes them in order
// through the counter queue[x]; once its own are gone it takes another XCD's (queue[(x + k) % 8],
// k = 1 .. 7).  Lane 0 of wave 0 takes the item that follows the current one at the start of the
// current one; it reaches the other waves through queue[16 + 2 b + parity] (workgroup b), stored
// after stage 0 and read after stage 1's barrier, long before stage nk - 2 needs it.
// queue[8] counts the workgroups that are done: the last one resets the counters, so each launch
// starts from zero.  No wait depends on another workgroup.  A work item is computed whole by one
// workgroup, so the output does not depend on the order.
template <int DT, int OUT, int CPR, int RDH = 0>
__global__ __launch_bounds__(256, 1) void gemm_w4p_kernel(const void *__restrict__ Ap, const void *__restrict__ Bp,
                                                          void *__restrict__ Cp, int M, int N, int K, int lda,
                                                          int ldb, int ldc, int tiles_m, int tiles_n, int seq_T,
                                                          int seq_Tp, int n_work, const float4 *__restrict__ rtab,
                                                          float alpha, int ksplit, void *__restrict__ Cp2,
                                                          int *__restrict__ queue) {
    static_assert(RDH == 0 || (OUT == OUT_DT && (RDH == 64 || RDH == 128)), "rotary epilogue");
    typedef typename Mma<DT>::elem elem;
    typedef typename Mma<DT>::operand opnd;
    constexpr int BK = CPR * 8;
    constexpr int U = BK / 16;
    constexpr int ROWB = CPR * 16;
    constexpr int HALF = 256 * ROWB;                  // one operand's k-tile
    constexpr int DPW = 2 * 256 * CPR / 64 / 4;
    constexpr int DPA = DPW / 2;
    constexpr int RPI = 64 / CPR;
    // The operand that streams the tokens (A = X for the row-major outputs, B = X for the transposed
    // value output) has a ring of three k-tiles, the other (the weights) one of two: LDS holds the
    // deep ring's slots 0..2, then the shallow ring's 0..1.
    constexpr bool DA = OUT != OUT_VT;
    constexpr int ABASE = DA ? 0 : 3 * HALF, BBASE = DA ? 3 * HALF : 0;
    static_assert(U >= 4 && DPW == 16, "refill schedule");
    extern __shared__ __align__(16) unsigned char smem[];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int wr = wave >> 1, wc = wave & 1;
    const int half = lane >> 5, l32 = lane & 31;
    const int nk = K / BK / ksplit;                   // k-tiles per work item

    // a work item: its tile's corner, its first k-tile, its output and the buffer resources of its
    // A and B panels (all wave-uniform)
    struct Tile {
        int bm0, bn0, k0, ks;
        void *out;
        i32x4 rsA, rsB;
    };
    auto decode = [&](int work, Tile &t) {
        int pid = work;
        if ((n_work & 7) == 0) pid = (pid & 7) * (n_work >> 3) + (pid >> 3);
        const int part = pid / (tiles_m * tiles_n);
        pid -= part * tiles_m * tiles_n;
        t.k0 = part * nk;
        t.out = part ? Cp2 : Cp;
        const int group_tiles = 8 * tiles_n;
        const int first_m = (pid / group_tiles) * 8;
        const int gsz = min(tiles_m - first_m, 8);
        const int pm = first_m + (pid % group_tiles) % gsz;
        const int pn = (pid % group_tiles) / gsz;
        // transposed value output: the k-loop of a tile starts at k-tile ks and wraps around, ks
        // different for the tiles of a set that share an A or a B panel (measured: 1.67 -> 1.62 ms
        // at 1024 x 262144 x 4096; no gain for the row-major output).  Only when every tile is
        // whole: a ragged last tile moved back over its neighbour must sum the shared elements in the
        // same order as the neighbour does (both write them).
        t.ks = OUT == OUT_VT && M % 256 == 0 && N % 256 == 0 ? ((pm & 7) + (pn & 3)) % nk : 0;
        t.bm0 = min(pm * 256, M - 256);
        t.bn0 = min(pn * 256, N - 256);
        t.rsA = buffer_rsrc(static_cast<const char *>(Ap) + (int64_t)t.bm0 * lda * (int64_t)sizeof(elem));
        t.rsB = buffer_rsrc(static_cast<const char *>(Bp) + (int64_t)t.bn0 * ldb * (int64_t)sizeof(elem));
    };
    // DMA instruction d < DPA fills rows RPI (wave + 4 d) .. + RPI - 1 of the A part (d >= DPA: of
    // the B part); lane i writes row + i / CPR, physical chunk i % CPR = logical chunk ^ key(row)
    uint32_t voffA[DPA], voffB[DPA];
#pragma unroll
    for (int i = 0; i < DPA; ++i) {
        const int r = RPI * (wave + 4 * i) + lane / CPR, pc = lane % CPR;
        const int c = pc ^ w4_key<CPR>(r);
        voffA[i] = (uint32_t)(r * lda * 2 + c * 16);
        voffB[i] = (uint32_t)(r * ldb * 2 + c * 16);
    }
    // DMA instruction d of k-tile ktile into the operand's ring slot `slot`
    auto issue = [&](const Tile &t, int d, int ktile, int slot) {
        int kx = ktile + t.ks;
        if (kx >= nk) kx -= nk;
        const int kk = (t.k0 + kx) * BK * 2;
        if (d < DPA) buffer_dma16(t.rsA, voffA[d], kk, smem + ABASE + slot * HALF + (wave + 4 * d) * 1024);
        else buffer_dma16(t.rsB, voffB[d - DPA], kk, smem + BBASE + slot * HALF + (wave + 4 * (d - DPA)) * 1024);
    };
    // the deep (D) and shallow (S) operands' instruction numbers
    auto dsn = [&](int i) { return DA ? i : DPA + i; };
    auto ssn = [&](int i) { return DA ? DPA + i : i; };

    const int key = w4_key<CPR>(l32);
    uint32_t rda[U], rdb[U];
#pragma unroll
    for (int ks = 0; ks < U; ++ks) {
        const int pc = (2 * ks + half) ^ key;
        rda[ks] = (uint32_t)((wr * 128 + l32) * ROWB + pc * 16);
        rdb[ks] = (uint32_t)((wc * 128 + l32) * ROWB + pc * 16);
    }
    opnd fa[2][4], fb[2][4];
    // fragment read r of k-step ks from the deep slot ds and the shallow slot ss
    auto rd = [&](int r, int ds, int ss, int ks, int buf) {
        const unsigned char *ab = smem + ABASE + (DA ? ds : ss) * HALF;
        const unsigned char *bb = smem + BBASE + (DA ? ss : ds) * HALF;
        if (r == 0) fa[buf][0] = __builtin_bit_cast(opnd, *(const u32x4 *)(ab + rda[ks]));
        else if (r <= 4) fb[buf][r - 1] = __builtin_bit_cast(opnd, *(const u32x4 *)(bb + rdb[ks] + (r - 1) * 32 * ROWB));
        else fa[buf][r - 4] = __builtin_bit_cast(opnd, *(const u32x4 *)(ab + rda[ks] + (r - 4) * 32 * ROWB));
    };

    const bool q0l0 = queue != nullptr && wave == 0 && lane == 0;
    // the next work item from the queue, or -1
    auto grab = [&]() -> int {
        const int x = blockIdx.x & 7, first = gridDim.x >> 3;   // first items of each XCD: static
        for (int k = 0; k < 8; ++k) {
            const int xx = (x + k) & 7;
            const int i = atomicAdd(queue + xx, 1) + first;
            if (i < ((n_work - xx + 7) >> 3)) return xx + 8 * i;
        }
        return -1;
    };
    auto finish = [&]() {
        if (q0l0 && atomicAdd(queue + 8, 1) == (int)gridDim.x - 1)
            for (int x = 0; x <= 8; ++x) atomicExch(queue + x, 0);
    };
    int work = blockIdx.x;
    if (work >= n_work) {
        finish();
        return;
    }
    Tile cur, nxt;
    decode(work, cur);
    bool has_next;
    if (queue) {                                      // resolved before stage 2
        has_next = false;
        nxt = cur;
    } else {
        has_next = work + (int)gridDim.x < n_work;
        // after the last tile the refills re-load its first k-tiles (in bounds, never read)
        if (has_next) decode(work + gridDim.x, nxt);
        else nxt = cur;
    }
    int par = 0;                                      // the queue's mailbox slot of this tile

    // prologue, as a previous tile's last stages leave the rings: k-tile 0 of both operands, k-tile
    // 1 of the deep one and the first half of the shallow one's (its second half goes out in the
    // first k-step of stage 0); then k-tile 0 has landed
#pragma unroll
    for (int d = 0; d < DPW; ++d) issue(cur, d, 0, 0);
#pragma unroll
    for (int i = 0; i < DPA; ++i) issue(cur, dsn(i), 1, 1);
#pragma unroll
    for (int i = 0; i < DPA / 2; ++i) issue(cur, ssn(i), 1, 1);
    wait_vmcnt<DPA + DPA / 2>();
    raw_barrier();
#pragma unroll
    for (int r = 0; r < 8; ++r) rd(r, 0, 0, 0, 0);

    f32x16 acc[4][4];
    int dslot = 0, sslot = 0;                         // the stage's deep and shallow ring slots
    for (;;) {
        // Stage kt of the current tile (FIRST: kt = 0, whose first k-step starts the accumulators
        // from zero).  The schedule is gemm_w4_kernel's; the refills past the tile's last k-tile
        // load the next tile's first ones.
        // Refills, one DMA instruction every fourth MFMA slot: k-step 0 sends the second half of
        // the shallow operand's k-tile kt + 1 (into the slot stage kt - 1 left), k-steps 1 and 2 the
        // deep operand's k-tile kt + 2 (into the deep slot stage kt - 1 left), the last k-step,
        // after the barrier, the first half of the shallow operand's k-tile kt + 2 (into this
        // stage's shallow slot).  The deep loads have about two stages to land, the shallow ones
        // one; the barrier's wait leaves the 8 deep loads of k-tile kt + 2 in flight.  (Measured at
        // [Q|K] 262144 x 5120 x 4096 on one box: two-stage rings with the refill spread over 2
        // k-steps 8.12 ms, this 7.93 ms.)
        auto stage = [&](int kt, auto first_c) {
            constexpr bool FIRST = decltype(first_c)::value;
            const int nd = dslot == 2 ? 0 : dslot + 1, ns = sslot ^ 1;
            const int rd_ = dslot == 0 ? 2 : dslot - 1;    // deep slot of k-tile kt + 2 (= kt - 1)
            const bool n2 = kt + 2 >= nk, n1 = kt + 1 >= nk;
            const Tile &t2 = n2 ? nxt : cur;
            const Tile &t1 = n1 ? nxt : cur;
            const int k2 = n2 ? kt + 2 - nk : kt + 2, k1 = n1 ? kt + 1 - nk : kt + 1;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int cb = u & 1;
                if (u == U - 1) {
                    wait_lgkm0();
                    wait_vmcnt<DPA>();
                    raw_barrier();
                }
#pragma unroll
                for (int m = 0; m < 16; ++m) {
                    const int i = m >> 2, j = m & 3;
                    if (FIRST && u == 0) acc[i][j] = Mma<DT>::mma(fb[cb][j], fa[cb][i], f32x16{});
                    else acc[i][j] = Mma<DT>::mma(fb[cb][j], fa[cb][i], acc[i][j]);
                    if ((m & 1) == 0) {
                        if (u < U - 1) rd(m >> 1, dslot, sslot, u + 1, cb ^ 1);
                        else rd(m >> 1, nd, ns, 0, cb ^ 1);
                    }
                    if ((m & 3) == 0) {
                        if (u == 0) issue(t1, ssn(DPA / 2 + (m >> 2)), k1, ns);
                        else if (u <= 2) issue(t2, dsn(4 * (u - 1) + (m >> 2)), k2, rd_);
                        else if (u == U - 1) issue(t2, ssn(m >> 2), k2, sslot);
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
            dslot = nd;
            sslot = ns;
        };
        // rotary epilogue: the table entries of row block i (this lane's position, its 32 head
        // columns: tb[4 (2 jp + pp) + k] holds the (cos, sin) of columns (32 jp for RDH 128) +
        // 16 pp + 8 (k / 2) + 4 half + 2 (k % 2) and + 1, from the transposed table rtab[q][t], so
        // a load's 32 positions are one contiguous run); block 0's are loaded before the tile's
        // last stage, block i + 1's while block i is rotated
        f32x4 tab[2][16];
        auto tload = [&](int i, f32x4 (&tb)[16]) {
            if constexpr (RDH > 0) {
                const int t = (cur.bm0 + wr * 128 + 32 * i + l32) % seq_T;
#pragma unroll
                for (int jp = 0; jp < 2; ++jp)
#pragma unroll
                    for (int pp = 0; pp < 2; ++pp)
#pragma unroll
                        for (int k = 0; k < 4; ++k) {
                            const int q = (RDH == 128 ? 16 * jp : 0) + 8 * pp + 4 * (k >> 1) + 2 * half + (k & 1);
                            tb[4 * (2 * jp + pp) + k] =
                                __builtin_bit_cast(f32x4, rtab[(int64_t)q * seq_T + t]);
                        }
            }
        };
        int taken = 0;
        if (q0l0) taken = grab();
        int *mbox = queue ? queue + 16 + 2 * blockIdx.x + par : nullptr;
        stage(0, std::integral_constant<bool, true>());
        // The grab's result has returned by stage 0's barrier wait (vector-memory operations
        // complete in issue order).  The store goes out before stage 1's refills, so the wait at
        // stage 1's barrier, which leaves only the last DPA of those in flight, has completed it.
        if (q0l0) __hip_atomic_store(mbox, taken, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        // after stage 1's barrier: the next work item (an agent-scope load, past the CU's cache)
        auto next_item = [&]() {
            const int w = __builtin_amdgcn_readfirstlane(__hip_atomic_load(mbox, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
            has_next = w >= 0;
            if (has_next) {
                work = w;
                decode(w, nxt);
            }
        };
        int kt = 1;                                   // nk >= 2
        if constexpr (RDH > 0) {
            while (kt < nk - 1) {
                if (queue && kt == 2) next_item();
                stage(kt++, std::integral_constant<bool, false>());
            }
            tload(0, tab[0]);
            stage(kt, std::integral_constant<bool, false>());
        } else {
            do {
                if (queue && kt == 2) next_item();
                stage(kt, std::integral_constant<bool, false>());
            } while (++kt < nk);
        }

        // ---- epilogue from registers.  acc[i][j][4 g + t] = C[row][col + t], row = wr*128 + 32 i +
        // l32, col = wc*128 + 32 j + 8 g + 4 half (tile coordinates).  Accumulators are read one
        // block at a time (explicit reads keep the compiler from copying all of them out at once).
        if constexpr (OUT == OUT_F32) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int row = cur.bm0 + wr * 128 + 32 * i + l32;
                float *crow = static_cast<float *>(cur.out) + (int64_t)row * ldc;
#pragma unroll
                for (int j = 0; j < 4; ++j)
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        float v[4];
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(v[e]) : "a"(acc[i][j][4 * g + e]));
                        const int col = cur.bn0 + wc * 128 + 32 * j + 8 * g + 4 * half;
                        *reinterpret_cast<f32x4 *>(crow + col) =
                            f32x4{alpha * v[0], alpha * v[1], alpha * v[2], alpha * v[3]};
                        __builtin_amdgcn_sched_barrier(0);
                    }
            }
        } else if constexpr (RDH > 0) {
            // Rotary embedding of the half-split pairs (column c of a head with c + RDH/2), token
            // row % seq_T.  A wave's 128 columns start on a head boundary (tiles start at multiples
            // of 256 or end at N, N a multiple of RDH), so a pair sits in one lane: blocks j and
            // j + 2 (RDH 128) or j and j + 1 (RDH 64), the same register.  The fp32 accumulators
            // turn by the fp32 (cos, sin) of the table (formed in fp64),
            // (a, b) -> (fma(a, cos, -b sin), fma(b, cos, a sin)), then round to the dtype once.
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                if (i + 1 < 4) tload(i + 1, tab[(i + 1) & 1]);
                const int row = cur.bm0 + wr * 128 + 32 * i + l32;
                elem *crow = static_cast<elem *>(Cp) + (int64_t)row * ldc;
#pragma unroll
                for (int jp = 0; jp < 2; ++jp) {
                    const int j1 = RDH == 128 ? jp : 2 * jp, j2 = RDH == 128 ? jp + 2 : 2 * jp + 1;
#pragma unroll
                    for (int pp = 0; pp < 2; ++pp) {
                        // elements 8 pp + e: head columns (32 jp for RDH 128) + 16 pp + 8 (e / 4) +
                        // 4 half + e % 4; tq[e / 2] holds the (cos, sin) of elements 2 (e / 2) and + 1
                        const f32x4 *tq = &tab[i & 1][4 * (2 * jp + pp)];
                        float v1[8], v2[8];
#pragma unroll
                        for (int e = 0; e < 8; ++e) {
                            asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(v1[e]) : "a"(acc[i][j1][8 * pp + e]));
                            asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(v2[e]) : "a"(acc[i][j2][8 * pp + e]));
                        }
                        uint32_t o1[4], o2[4];
#pragma unroll
                        for (int k = 0; k < 4; ++k) {
                            float y1[2], y2[2];
#pragma unroll
                            for (int h2 = 0; h2 < 2; ++h2) {
                                const int e = 2 * k + h2;
                                const f32x4 q = tq[e >> 1];
                                const float cs = q[2 * (e & 1)], sn = q[2 * (e & 1) + 1];
                                y1[h2] = __builtin_fmaf(v1[e], cs, -(v2[e] * sn));
                                y2[h2] = __builtin_fmaf(v2[e], cs, v1[e] * sn);
                            }
                            o1[k] = pack2<DT>(y1[0], y1[1]);
                            o2[k] = pack2<DT>(y2[0], y2[1]);
                        }
                        // as the plain epilogue: exchange halves so each lane stores 8 consecutive columns
                        asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1\n\tv_permlane32_swap_b32 %2, %3\n\ts_nop 1"
                                     : "+v"(o1[0]), "+v"(o1[2]), "+v"(o1[1]), "+v"(o1[3]));
                        asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1\n\tv_permlane32_swap_b32 %2, %3\n\ts_nop 1"
                                     : "+v"(o2[0]), "+v"(o2[2]), "+v"(o2[1]), "+v"(o2[3]));
                        const int cb1 = cur.bn0 + wc * 128 + 32 * j1, cb2 = cur.bn0 + wc * 128 + 32 * j2;
                        *reinterpret_cast<u32x4 *>(crow + cb1 + 16 * pp + 8 * half) = u32x4{o1[0], o1[1], o1[2], o1[3]};
                        *reinterpret_cast<u32x4 *>(crow + cb2 + 16 * pp + 8 * half) = u32x4{o2[0], o2[1], o2[2], o2[3]};
                        __builtin_amdgcn_sched_barrier(0);
                    }
                }
            }
        } else
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int row = cur.bm0 + wr * 128 + 32 * i + l32;
            elem *crow = static_cast<elem *>(Cp) + (int64_t)row * ldc;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int colb = cur.bn0 + wc * 128 + 32 * j;
#pragma unroll
                for (int pp = 0; pp < 2; ++pp) {
                    float v[8];
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(v[e]) : "a"(acc[i][j][8 * pp + e]));
                    uint32_t a0 = pack2<DT>(v[0], v[1]), a1 = pack2<DT>(v[2], v[3]);
                    uint32_t b0 = pack2<DT>(v[4], v[5]), b1 = pack2<DT>(v[6], v[7]);
                    int64_t dcol;
                    if constexpr (OUT == OUT_DT) {
                        // a lane holds columns 16 pp + 4 half + 0..3 (a) and 16 pp + 8 + 4 half + 0..3
                        // (b); exchanging a of the upper half-wave with b of the lower one leaves
                        // each lane eight consecutive columns, 16 pp + 8 half + 0..7
                        asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1\n\tv_permlane32_swap_b32 %2, %3\n\ts_nop 1"
                                     : "+v"(a0), "+v"(b0), "+v"(a1), "+v"(b1));
                        dcol = colb + 16 * pp + 8 * half;
                    } else {
                        // tokens 16 pp + 4 half + 0..3 and 16 pp + 8 + 4 half + 0..3 of the 32-token
                        // block colb: with bits 2 and 3 exchanged they are the eight consecutive
                        // positions 16 pp + 8 half + 0..7 (the block lies in one sequence)
                        const int sb = colb / seq_T;
                        dcol = (int64_t)sb * seq_Tp + (colb - sb * seq_T) + 16 * pp + 8 * half;
                    }
                    *reinterpret_cast<u32x4 *>(crow + dcol) = u32x4{a0, a1, b0, b1};
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
        }
        if (!has_next) break;
        cur = nxt;
        if (queue) {
            par ^= 1;
        } else {
            work += gridDim.x;
            has_next = work + (int)gridDim.x < n_work;
            if (has_next) decode(work + gridDim.x, nxt);
        }
    }
    wait_vmcnt<0>();
    finish();
}

}  // namespace

template <int DT, int BM, int BN, int NS, int MINB, int OUT, int CPR = 4, int NW = 4>
hipError_t run_gemm(const void *A, const void *B, void *C, int M, int N, int K, int lda, int ldb,
                    int ldc, float alpha, hipStream_t st, int seq_T = 1, int seq_Tp = 1,
                    void *C2 = nullptr, int *ksplit_used = nullptr) {
    typedef GemmCfg<DT, BM, BN, NS, CPR, NW> G;
    if (K % G::BK != 0) return hipErrorInvalidValue;
    const int tm = (M + BM - 1) / BM, tn = (N + BN - 1) / BN;
    // With a second output, split K in two when the tiles alone would leave a partial last round
    // of workgroups on the CUs and two halves fill the rounds better.
    int ksplit = 1;
    if (C2 != nullptr && (K / G::BK) % 2 == 0) {
        int dev = 0, ncu = 0;
        if (hipGetDevice(&dev) == hipSuccess &&
            hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && ncu > 0) {
            const int slots = ncu * MINB, t = tm * tn;
            const double e1 = (double)t / (((t + slots - 1) / slots) * slots);
            const double e2 = (double)(2 * t) / (((2 * t + slots - 1) / slots) * slots);
            if (e2 > e1 + 0.05) ksplit = 2;
        }
    }
    if (ksplit_used) *ksplit_used = ksplit;
    hipError_t e = hipFuncSetAttribute((const void *)gemm_nt_kernel<DT, BM, BN, NS, MINB, OUT, CPR, NW>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)G::LDS_BYTES);
    if (e != hipSuccess) return e;
    gemm_nt_kernel<DT, BM, BN, NS, MINB, OUT, CPR, NW><<<dim3(tm * tn * ksplit), dim3(64 * NW), G::LDS_BYTES, st>>>(
        A, B, C, M, N, K, lda, ldb, ldc, tm, tn, alpha, seq_T, seq_Tp, ksplit, C2);
    return hipGetLastError();
}

// Split K in two (second half into C2) when the tiles alone would leave a partial last round of
// workgroups on the CUs and two halves fill the rounds better.
inline int choose_ksplit(int tiles, int k_tiles, int slots_per_cu) {
    if (k_tiles % 2 != 0) return 1;
    int dev = 0, ncu = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || ncu <= 0)
        return 1;
    const int slots = ncu * slots_per_cu;
    const double e1 = (double)tiles / (((tiles + slots - 1) / slots) * slots);
    const double e2 = (double)(2 * tiles) / (((2 * tiles + slots - 1) / slots) * slots);
    return e2 > e1 + 0.05 ? 2 : 1;
}

template <int DT, int OUT, int CPR>
hipError_t run_gemm_w4(const void *A, const void *B, void *C, int M, int N, int K, int lda, int ldb, int ldc,
                       float alpha, hipStream_t st, int seq_T, int seq_Tp, void *C2, int *ksplit_used) {
    constexpr int BK = CPR * 8;
    // two ring stages; the storage-dtype output reuses LDS for a 256 x 256 C tile
    constexpr size_t RING = 2 * 2 * 256 * CPR * 16;
    constexpr size_t LDS = OUT == OUT_DT && RING < 256 * 512 ? 256 * 512 : RING;
    if (K % BK != 0) return hipErrorInvalidValue;
    const int tm = (M + 255) / 256, tn = (N + 255) / 256;
    const int ksplit = C2 != nullptr ? choose_ksplit(tm * tn, K / BK, 1) : 1;
    if (ksplit_used) *ksplit_used = ksplit;
    hipError_t e = hipFuncSetAttribute((const void *)gemm_w4_kernel<DT, OUT, CPR>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)LDS);
    if (e != hipSuccess) return e;
    gemm_w4_kernel<DT, OUT, CPR><<<dim3(tm * tn * ksplit), dim3(256), LDS, st>>>(
        A, B, C, M, N, K, lda, ldb, ldc, tm, tn, alpha, seq_T, seq_Tp, ksplit, C2);
    return hipGetLastError();
}

// the persistent GEMMs' tile queues: 4 KiB per (device, stream), allocated on the first launch on
// that stream and held until the process ends
constexpr size_t kQueueBytes = 4096;
std::mutex g_queue_mu;
std::map<std::pair<int, hipStream_t>, int *> g_queues;
thread_local int g_queue_noalloc = 0;

int *gemm_queue(int dev, hipStream_t st) {
    std::lock_guard<std::mutex> lock(g_queue_mu);
    const auto it = g_queues.find({dev, st});
    if (it != g_queues.end()) return it->second;
    if (g_queue_noalloc > 0) return nullptr;
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(st, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone) return nullptr;
    int *q = nullptr;
    if (hipMalloc(&q, kQueueBytes) != hipSuccess) {
        (void)hipGetLastError();
        return nullptr;
    }
    if (hipMemset(q, 0, kQueueBytes) != hipSuccess) {
        (void)hipGetLastError();
        (void)hipFree(q);
        return nullptr;
    }
    g_queues[{dev, st}] = q;
    return q;
}

template <int DT, int OUT, int CPR, int RDH = 0>
hipError_t run_gemm_w4p(const void *A, const void *B, void *C, int M, int N, int K, int lda, int ldb, int ldc,
                        hipStream_t st, int seq_T, int seq_Tp, const float4 *rtab = nullptr, float alpha = 1.f,
                        void *C2 = nullptr, int *ksplit_used = nullptr) {
    constexpr size_t LDS = 5 * 256 * CPR * 16;       // rings of three and two k-tiles
    int dev = 0, ncu = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    const int tm = (M + 255) / 256, tn = (N + 255) / 256;
    // with a second output: K in two parts when they fill the CUs' rounds better than the tiles alone
    // (each part keeps at least three k-tiles)
    int ksplit = 1;
    if (C2 != nullptr && (K / (CPR * 8)) % 2 == 0 && K / (CPR * 8) >= 6) {
        const int t = tm * tn;
        const double e1 = (double)t / (((t + ncu - 1) / ncu) * ncu);
        const double e2 = (double)(2 * t) / (((2 * t + ncu - 1) / ncu) * ncu);
        if (e2 > e1 + 0.05) ksplit = 2;
    }
    if (ksplit_used) *ksplit_used = ksplit;
    const int n_work = tm * tn * ksplit;
    e = hipFuncSetAttribute((const void *)gemm_w4p_kernel<DT, OUT, CPR, RDH>,
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)LDS);
    if (e != hipSuccess) return e;
    // the queue pays where a workgroup has many work items (measured: 80 per workgroup, the [Q|K]
    // projection of 128 x 2048 tokens at d 4096, 8.22 -> 8.00 ms; 10 and 2 per workgroup, the
    // projections of 16 x 2048 tokens, 1.8 and 8 % slower than the static order)
    const int grid = min(n_work, ncu);
    int *queue = grid % 8 == 0 && n_work >= 32 * grid && K / (CPR * 8) / ksplit >= 6 &&
                         (int)(kQueueBytes / 4) >= 16 + 2 * grid
                     ? gemm_queue(dev, st) : nullptr;
    gemm_w4p_kernel<DT, OUT, CPR, RDH><<<dim3(grid), dim3(256), LDS, st>>>(
        A, B, C, M, N, K, lda, ldb, ldc, tm, tn, seq_T, seq_Tp, n_work, rtab, alpha, ksplit, C2, queue);
    return hipGetLastError();
}

// The persistent kernel takes whole 256 x 256 tiles, 16-byte aligned output rows and at least three
// k-tiles; a split K (fp32 output with a second buffer) only where the tiles are whole in both
// directions (no tile moved back over its neighbour: the two parts are summed by the caller); for
// the transposed value output, 32-token blocks inside one sequence.
template <int OUT, int CPR>
bool persistent_fits(int M, int N, int K, int ldc, int seq_T, const void *C2) {
    if (C2 != nullptr && (OUT != OUT_F32 || M % 256 != 0 || N % 256 != 0)) return false;
    if (M < 256 || N < 256 || K % (CPR * 8) != 0 || K / (CPR * 8) < 3) return false;
    if (OUT == OUT_F32) return ldc % 4 == 0 && N % 4 == 0;
    if (ldc % 8 != 0) return false;
    if (OUT == OUT_DT) return N % 8 == 0;
    return seq_T % 32 == 0;
}

namespace {

template <int OUT>
hipError_t dispatch(int dtype, const void *A, const void *B, void *C, int M, int N, int K, int lda,
                    int ldb, int ldc, float alpha, hipStream_t st, int seq_T = 1, int seq_Tp = 1,
                    void *C2 = nullptr, int *ksplit_used = nullptr) {
    if (ksplit_used) *ksplit_used = 1;
    if (M <= 0 || N <= 0 || K <= 0) return hipSuccess;
    // 16-bit dtypes: 128-byte k-rows when K allows (each load covers whole cache lines), else 64-byte rows
    const bool wide = K % 64 == 0;
    switch (dtype) {
    case F32:
        return run_gemm<F32, 128, 128, 4, 1, OUT>(A, B, C, M, N, K, lda, ldb, ldc, alpha, st, seq_T, seq_Tp, C2, ksplit_used);
    case F16:
        if (wide && persistent_fits<OUT, 8>(M, N, K, ldc, seq_T, C2))
            return run_gemm_w4p<F16, OUT, 8>(A, B, C, M, N, K, lda, ldb, ldc, st, seq_T, seq_Tp, nullptr, alpha, C2,
                                             ksplit_used);
        return wide ? run_gemm_w4<F16, OUT, 8>(A, B, C, M, N, K, lda, ldb, ldc, alpha, st, seq_T, seq_Tp, C2, ksplit_used)
                    : run_gemm_w4<F16, OUT, 4>(A, B, C, M, N, K, lda, ldb, ldc, alpha, st, seq_T, seq_Tp, C2, ksplit_used);
    default:
        if (wide && persistent_fits<OUT, 8>(M, N, K, ldc, seq_T, C2))
            return run_gemm_w4p<BF16, OUT, 8>(A, B, C, M, N, K, lda, ldb, ldc, st, seq_T, seq_Tp, nullptr, alpha, C2,
                                              ksplit_used);
        return wide ? run_gemm_w4<BF16, OUT, 8>(A, B, C, M, N, K, lda, ldb, ldc, alpha, st, seq_T, seq_Tp, C2, ksplit_used)
                    : run_gemm_w4<BF16, OUT, 4>(A, B, C, M, N, K, lda, ldb, ldc, alpha, st, seq_T, seq_Tp, C2, ksplit_used);
    }
}

}  // namespace

GemmQueueNoAlloc::GemmQueueNoAlloc() { ++g_queue_noalloc; }
GemmQueueNoAlloc::~GemmQueueNoAlloc() { --g_queue_noalloc; }

hipError_t launch_gemm_nt(int dtype, const void *A, const void *B, void *C, int M, int N, int K,
                          int lda, int ldb, int ldc, hipStream_t st) {
    return dispatch<OUT_DT>(dtype, A, B, C, M, N, K, lda, ldb, ldc, 1.f, st);
}

hipError_t launch_gemm_nt_f32out(int dtype, const void *A, const void *B, float *C, int M, int N, int K,
                                 int lda, int ldb, int ldc, float alpha, hipStream_t st, float *C2,
                                 int *ksplit_used) {
    return dispatch<OUT_F32>(dtype, A, B, C, M, N, K, lda, ldb, ldc, alpha, st, 1, 1, C2, ksplit_used);
}

bool gemm_rope_fuses(int dtype, int M, int N, int K, int ldc, int head_dim) {
    return dtype != F32 && (head_dim == 64 || head_dim == 128) && N % head_dim == 0 && K % 64 == 0 &&
           persistent_fits<OUT_DT, 8>(M, N, K, ldc, 1, nullptr);
}

hipError_t launch_gemm_nt_rope(int dtype, const void *A, const void *B, void *C, int M, int N, int K, int lda,
                               int ldb, int ldc, int head_dim, int seq_T, const float4 *tab, hipStream_t st) {
    if (!gemm_rope_fuses(dtype, M, N, K, ldc, head_dim) || seq_T <= 0 || tab == nullptr) return hipErrorInvalidValue;
    if (dtype == F16)
        return head_dim == 64 ? run_gemm_w4p<F16, OUT_DT, 8, 64>(A, B, C, M, N, K, lda, ldb, ldc, st, seq_T, 1, tab)
                              : run_gemm_w4p<F16, OUT_DT, 8, 128>(A, B, C, M, N, K, lda, ldb, ldc, st, seq_T, 1, tab);
    return head_dim == 64 ? run_gemm_w4p<BF16, OUT_DT, 8, 64>(A, B, C, M, N, K, lda, ldb, ldc, st, seq_T, 1, tab)
                          : run_gemm_w4p<BF16, OUT_DT, 8, 128>(A, B, C, M, N, K, lda, ldb, ldc, st, seq_T, 1, tab);
}

hipError_t launch_gemm_nt_vt(int dtype, const void *A, const void *B, void *C, int M, int N, int K,
                             int lda, int ldb, int ldc, int seq_T, hipStream_t st) {
    return dispatch<OUT_VT>(dtype, A, B, C, M, N, K, lda, ldb, ldc, 1.f, st, seq_T, (seq_T + 31) / 32 * 32);
}

}  // namespace jab
