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
//  * k-tiles of 128 bytes per row are staged in LDS.  Row r stores its eight
//    16-byte chunks at chunk index (c ^ (r & 7)), so the 32 rows one MFMA operand
//    read touches spread over all banks.
//  * Two LDS stages: the next k-tile is fetched from global memory into
//    registers while the current one feeds the matrix cores, then written to the
//    other stage; one barrier per k-tile.
//  * Workgroup ids are remapped so that each XCD (ids congruent mod 8 land on the
//    same XCD) walks a contiguous range of tiles, grouped 8 M-tiles at a time so
//    that concurrently running tiles share A and B panels in that XCD's L2.
#include "device_common.h"
#include "kernels.h"

namespace jab {
namespace {

template <int DT, int BM, int BN>
struct GemmCfg {
    typedef typename Mma<DT>::elem elem;
    static constexpr int EPC = 16 / (int)sizeof(elem);  // elements per 16-byte chunk
    static constexpr int BK = 8 * EPC;                  // elements per 128-byte k-tile row
    static constexpr int WM = BM / 2, WN = BN / 2;
    static constexpr int FM = WM / 32, FN = WN / 32;
    static constexpr int LA = BM * 8 / 256, LB = BN * 8 / 256;   // chunk loads per thread
    static constexpr int STAGE_CHUNKS = (BM + BN) * 8;
    static constexpr size_t LDS_BYTES = 2 * (size_t)STAGE_CHUNKS * 16;
};

__device__ inline u32x4 zero4() { return u32x4{0u, 0u, 0u, 0u}; }

template <int DT, int BM, int BN>
__global__ __launch_bounds__(256, 1) void gemm_nt_kernel(const void *__restrict__ Ap,
                                                          const void *__restrict__ Bp,
                                                          void *__restrict__ Cp, int M, int N, int K,
                                                          int lda, int ldb, int ldc, int tiles_m,
                                                          int tiles_n) {
    typedef GemmCfg<DT, BM, BN> G;
    typedef typename G::elem elem;
    typedef Mma<DT> MM;
    extern __shared__ __align__(16) unsigned char smem[];
    u32x4 *lds = reinterpret_cast<u32x4 *>(smem);

    const elem *A = static_cast<const elem *>(Ap);
    const elem *B = static_cast<const elem *>(Bp);
    elem *C = static_cast<elem *>(Cp);

    // ---- tile order: XCD-contiguous ranges, then groups of 8 M-tiles
    const int nwg = gridDim.x;
    int pid = blockIdx.x;
    if ((nwg & 7) == 0)
        pid = (pid & 7) * (nwg >> 3) + (pid >> 3);
    const int group_tiles = 8 * tiles_n;
    const int first_m = (pid / group_tiles) * 8;
    const int gsz = min(tiles_m - first_m, 8);
    const int pm = first_m + (pid % group_tiles) % gsz;
    const int pn = (pid % group_tiles) / gsz;
    const int bm0 = pm * BM, bn0 = pn * BN;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm0 = (wave >> 1) * G::WM, wn0 = (wave & 1) * G::WN;

    // ---- global -> register fetch of one k-tile
    u32x4 ra[G::LA], rb[G::LB];
    auto fetch = [&](int k0) {
#pragma unroll
        for (int i = 0; i < G::LA; ++i) {
            const int idx = tid + 256 * i, r = idx >> 3, c = idx & 7;
            const int row = bm0 + r, col = k0 + c * G::EPC;
            ra[i] = (row < M && col < K)
                        ? *reinterpret_cast<const u32x4 *>(A + (int64_t)row * lda + col)
                        : zero4();
        }
#pragma unroll
        for (int i = 0; i < G::LB; ++i) {
            const int idx = tid + 256 * i, r = idx >> 3, c = idx & 7;
            const int row = bn0 + r, col = k0 + c * G::EPC;
            rb[i] = (row < N && col < K)
                        ? *reinterpret_cast<const u32x4 *>(B + (int64_t)row * ldb + col)
                        : zero4();
        }
    };
    auto stash = [&](int stage) {
        u32x4 *As = lds + stage * G::STAGE_CHUNKS;
        u32x4 *Bs = As + BM * 8;
#pragma unroll
        for (int i = 0; i < G::LA; ++i) {
            const int idx = tid + 256 * i, r = idx >> 3, c = idx & 7;
            As[r * 8 + (c ^ (r & 7))] = ra[i];
        }
#pragma unroll
        for (int i = 0; i < G::LB; ++i) {
            const int idx = tid + 256 * i, r = idx >> 3, c = idx & 7;
            Bs[r * 8 + (c ^ (r & 7))] = rb[i];
        }
    };

    f32x16 acc[G::FM][G::FN];
#pragma unroll
    for (int i = 0; i < G::FM; ++i)
#pragma unroll
        for (int j = 0; j < G::FN; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

    // ---- operand fetch from LDS for k-step ks of the tile
    auto frag = [&](const u32x4 *S, int r, int ks) -> typename MM::operand {
        if constexpr (DT == F32) {
            const int k = ks * MM::K + (lane >> 5);          // one element per lane
            const int c = k >> 2, sub = k & 3;
            const float *p = reinterpret_cast<const float *>(S + r * 8 + (c ^ (r & 7)));
            return p[sub];
        } else {
            const int c = ks * 2 + (lane >> 5);               // eight elements per lane
            const u32x4 v = S[r * 8 + (c ^ (r & 7))];
            return __builtin_bit_cast(typename MM::operand, v);
        }
    };

    const int nk = (K + G::BK - 1) / G::BK;
    fetch(0);
    stash(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int cur = kt & 1;
        if (kt + 1 < nk)
            fetch((kt + 1) * G::BK);
        const u32x4 *As = lds + cur * G::STAGE_CHUNKS;
        const u32x4 *Bs = As + BM * 8;
#pragma unroll
        for (int ks = 0; ks < G::BK / MM::K; ++ks) {
            typename MM::operand a[G::FM], b[G::FN];
#pragma unroll
            for (int i = 0; i < G::FM; ++i) a[i] = frag(As, wm0 + 32 * i + (lane & 31), ks);
#pragma unroll
            for (int j = 0; j < G::FN; ++j) b[j] = frag(Bs, wn0 + 32 * j + (lane & 31), ks);
#pragma unroll
            for (int i = 0; i < G::FM; ++i)
#pragma unroll
                for (int j = 0; j < G::FN; ++j) acc[i][j] = MM::mma(a[i], b[j], acc[i][j]);
        }
        if (kt + 1 < nk)
            stash(cur ^ 1);
        __syncthreads();
    }

    // ---- epilogue: D layout -> C rows / columns, converted to the storage dtype
#pragma unroll
    for (int i = 0; i < G::FM; ++i) {
#pragma unroll
        for (int j = 0; j < G::FN; ++j) {
            const int col = bn0 + wn0 + 32 * j + (lane & 31);
            if (col >= N) continue;
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int row = bm0 + wm0 + 32 * i + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
                if (row < M)
                    C[(int64_t)row * ldc + col] = from_f32<DT>(acc[i][j][e]);
            }
        }
    }
}

template <int DT, int BM, int BN>
hipError_t run_gemm(const void *A, const void *B, void *C, int M, int N, int K, int lda, int ldb,
                    int ldc, hipStream_t st) {
    typedef GemmCfg<DT, BM, BN> G;
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute((const void *)gemm_nt_kernel<DT, BM, BN>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize,
                                           (int)G::LDS_BYTES);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    const int tm = (M + BM - 1) / BM, tn = (N + BN - 1) / BN;
    gemm_nt_kernel<DT, BM, BN><<<dim3(tm * tn), dim3(256), G::LDS_BYTES, st>>>(A, B, C, M, N, K, lda,
                                                                              ldb, ldc, tm, tn);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_nt(int dtype, const void *A, const void *B, void *C, int M, int N, int K,
                          int lda, int ldb, int ldc, hipStream_t st) {
    if (M <= 0 || N <= 0 || K <= 0) return hipSuccess;
    switch (dtype) {
    case F32: return run_gemm<F32, 128, 128>(A, B, C, M, N, K, lda, ldb, ldc, st);
    case F16: return run_gemm<F16, 256, 256>(A, B, C, M, N, K, lda, ldb, ldc, st);
    default: return run_gemm<BF16, 256, 256>(A, B, C, M, N, K, lda, ldb, ldc, st);
    }
}

}  // namespace jab
