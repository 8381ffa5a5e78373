// gemm.hip -- projection GEMM of the fused QKV weight on the matrix cores.
//
// Paper: Method, "Layer-wise PTQ": y = x W with the QKV projection fused as
// W = [W_Q | W_K | W_V].  Here C[m][n] = sum_k A[m][k] B[n][k] with A = X
// [tokens][d_model] and B = W_hat [R][d_model] (one row per output channel), both
// k-contiguous, accumulated in fp32 and stored in the storage dtype.
//
// gfx950 design
//  * 256 threads = 4 wavefronts in a 2 x 2 arrangement; a workgroup computes a
//    BM x BN tile, each wave a (BM/2) x (BN/2) sub-tile of 32x32 MFMA blocks
//    (v_mfma_f32_32x32x16_{bf16,f16}; v_mfma_f32_32x32x2_f32 for fp32).
//  * k-tiles go straight from global memory into LDS (global_load_lds_dwordx4, no
//    register staging) through a ring of stages: two stages of 128-byte rows (each
//    load covers whole cache lines, 64 KiB per stage), or four of 64-byte rows when K
//    is not a multiple of 64 elements.  One barrier per stage, placed before its last
//    unit of MFMAs: the stage's slot is refilled immediately after it.
//  * Within a stage, operand fragments are double-buffered in registers and the
//    instruction order is fixed by hand: every MFMA slot carries at most one LDS
//    read (for the next unit) and one global->LDS load, so the matrix cores are not
//    starved while memory instructions issue.
//  * 16-byte chunks are stored rotated per row so that the 16 rows served together
//    by one LDS cycle (64 banks) land in distinct banks: conflict-free operand reads.
//  * Workgroup ids are remapped so that each XCD (ids congruent mod 8 land on the
//    same XCD) walks a contiguous range of tiles, grouped 8 M-tiles at a time so
//    that concurrently running tiles share A and B panels in that XCD's L2.
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

namespace {

template <int OUT>
hipError_t dispatch(int dtype, const void *A, const void *B, void *C, int M, int N, int K, int lda,
                    int ldb, int ldc, float alpha, hipStream_t st, int seq_T = 1, int seq_Tp = 1,
                    void *C2 = nullptr, int *ksplit_used = nullptr) {
    if (ksplit_used) *ksplit_used = 1;
    if (M <= 0 || N <= 0 || K <= 0) return hipSuccess;
    // 16-bit dtypes: 256x256 tiles; 128-byte k-rows (two 64 KiB stages) when K allows,
    // so each load covers whole 128-byte cache lines, else 64-byte rows in four stages.
    const bool wide = K % 64 == 0;
    switch (dtype) {
    case F32:
        return run_gemm<F32, 128, 128, 4, 1, OUT>(A, B, C, M, N, K, lda, ldb, ldc, alpha, st, seq_T, seq_Tp, C2, ksplit_used);
    case F16:
        return wide ? run_gemm<F16, 256, 256, 2, 1, OUT, 8, 8>(A, B, C, M, N, K, lda, ldb, ldc, alpha, st, seq_T, seq_Tp, C2, ksplit_used)
                    : run_gemm<F16, 256, 256, 4, 1, OUT, 4>(A, B, C, M, N, K, lda, ldb, ldc, alpha, st, seq_T, seq_Tp, C2, ksplit_used);
    default:
        return wide ? run_gemm<BF16, 256, 256, 2, 1, OUT, 8, 8>(A, B, C, M, N, K, lda, ldb, ldc, alpha, st, seq_T, seq_Tp, C2, ksplit_used)
                    : run_gemm<BF16, 256, 256, 4, 1, OUT, 4>(A, B, C, M, N, K, lda, ldb, ldc, alpha, st, seq_T, seq_Tp, C2, ksplit_used);
    }
}

}  // namespace

hipError_t launch_gemm_nt(int dtype, const void *A, const void *B, void *C, int M, int N, int K,
                          int lda, int ldb, int ldc, hipStream_t st) {
    return dispatch<OUT_DT>(dtype, A, B, C, M, N, K, lda, ldb, ldc, 1.f, st);
}

hipError_t launch_gemm_nt_f32out(int dtype, const void *A, const void *B, float *C, int M, int N, int K,
                                 int lda, int ldb, int ldc, float alpha, hipStream_t st, float *C2,
                                 int *ksplit_used) {
    return dispatch<OUT_F32>(dtype, A, B, C, M, N, K, lda, ldb, ldc, alpha, st, 1, 1, C2, ksplit_used);
}

hipError_t launch_gemm_nt_vt(int dtype, const void *A, const void *B, void *C, int M, int N, int K,
                             int lda, int ldb, int ldc, int seq_T, hipStream_t st) {
    return dispatch<OUT_VT>(dtype, A, B, C, M, N, K, lda, ldb, ldc, 1.f, st, seq_T, (seq_T + 31) / 32 * 32);
}

}  // namespace jab
