// rope.hip -- rotary position embedding on the query and key columns of the projection (the RoPE
// Mistral applies, half-split pairs: element j of a head with element j + d_head/2), and its
// transpose on the gradient rows dY^T of the backward.
//
// Position t turns pair j by t * theta^(-2j / d_head).  The angles and their cosines and sines
// are formed in fp64 once per call into a [T][d_head/2] table of fp32 pairs (angles reach 2^11
// radians at T = 2048, beyond what fp32 angle arithmetic resolves to the fp32 loss bar); the
// rotation itself runs in fp32 on the projection as accumulated (fp32) and rounds to the dtype
// once.  Each sequence starts at position 0.  Where the projection GEMM's epilogue does not take
// the rotation: one pass over the fp32 [Q|K] (HBM-bound).  The gradient's transposed turn runs on
// the dtype rows of dY^T.
#include "device_common.h"
#include "kernels.h"

namespace jab {
namespace {

// thread (t, q): pairs j = 2q, 2q + 1 of position t, into tab[t][j] and, when tab_t is given, the
// transposed copy tab_t[q][t] = (cos, sin of 2q, cos, sin of 2q + 1) that the projection GEMM's
// rotary epilogue reads (32 consecutive positions are one contiguous run of a load)
__global__ __launch_bounds__(256) void rope_table_kernel(int T, int dh, double theta, float2 *__restrict__ tab,
                                                         float4 *__restrict__ tab_t) {
    const int half = dh / 2, nq = half / 2;
    const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (i >= (int64_t)T * nq) return;
    const int t = (int)(i / nq), q = (int)(i % nq);
    float2 cs[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int j = 2 * q + u;
        const double ang = (double)t * pow(theta, -2.0 * (double)j / (double)dh);
        cs[u] = make_float2((float)cos(ang), (float)sin(ang));
        tab[(int64_t)t * half + j] = cs[u];
    }
    if (tab_t) tab_t[(int64_t)q * T + t] = make_float4(cs[0].x, cs[0].y, cs[1].x, cs[1].y);
}

// eight consecutive elements as one (16-bit) or two (fp32) 16-byte accesses
template <int DT>
__device__ inline void load8(const typename Mma<DT>::elem *p, float *v) {
    typedef typename Mma<DT>::elem elem;
    elem e[8];
    if constexpr (sizeof(elem) == 2) {
        *reinterpret_cast<uint4 *>(e) = *reinterpret_cast<const uint4 *>(p);
    } else {
        reinterpret_cast<float4 *>(e)[0] = reinterpret_cast<const float4 *>(p)[0];
        reinterpret_cast<float4 *>(e)[1] = reinterpret_cast<const float4 *>(p)[1];
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = to_f32<DT>(e[k]);
}

template <int DT>
__device__ inline void store8(typename Mma<DT>::elem *p, const float *v) {
    typedef typename Mma<DT>::elem elem;
    elem e[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) e[k] = from_f32<DT>(v[k]);
    if constexpr (sizeof(elem) == 2) {
        *reinterpret_cast<uint4 *>(p) = *reinterpret_cast<const uint4 *>(e);
    } else {
        reinterpret_cast<float4 *>(p)[0] = reinterpret_cast<const float4 *>(e)[0];
        reinterpret_cast<float4 *>(p)[1] = reinterpret_cast<const float4 *>(e)[1];
    }
}

// rows: the fp32 projection src[m][h * dh + j], src[m][h * dh + dh/2 + j] for token m (position
// m % T) turned and rounded once to the dtype into dst (the same rows and columns; dst may be src
// for fp32), 8 pairs per thread; (a, b) -> (fma(a, cos, -b sin), fma(b, cos, a sin)) as the
// projection GEMM's rotary epilogue forms them
template <int DT>
__global__ __launch_bounds__(256) void rope_rows_kernel(const float *src, int64_t lds, void *dst, int64_t ldd,
                                                        int64_t M, int T, int heads, int dh,
                                                        const float2 *__restrict__ tab) {
    typedef typename Mma<DT>::elem elem;
    const int half = dh / 2, per_head = half / 8;
    const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (i >= M * heads * per_head) return;
    const int j0 = (int)(i % per_head) * 8;
    const int64_t mh = i / per_head;
    const int h = (int)(mh % heads);
    const int64_t m = mh / heads;
    const int t = (int)(m % T);
    const float *a = src + m * lds + (int64_t)h * dh + j0;
    const float *b = a + half;
    elem *ao_p = static_cast<elem *>(dst) + m * ldd + (int64_t)h * dh + j0;
    const float4 *cs4 = reinterpret_cast<const float4 *>(tab + (int64_t)t * half + j0);
    float av[8], bv[8], c[8], s[8];
    load8<F32>(a, av);
    load8<F32>(b, bv);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const float4 q = cs4[k];
        c[2 * k] = q.x; s[2 * k] = q.y;
        c[2 * k + 1] = q.z; s[2 * k + 1] = q.w;
    }
    float ao[8], bo[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        ao[k] = __builtin_fmaf(av[k], c[k], -(bv[k] * s[k]));
        bo[k] = __builtin_fmaf(bv[k], c[k], av[k] * s[k]);
    }
    store8<DT>(ao_p, ao);
    store8<DT>(ao_p + half, bo);
}

// columns: dyt[h * dh + j][m], dyt[h * dh + dh/2 + j][m], 8 tokens per thread
template <int DT>
__global__ __launch_bounds__(256) void rope_cols_kernel(void *__restrict__ yt, int64_t ldt, int64_t ncols, int T,
                                                        int heads, int dh, const float2 *__restrict__ tab,
                                                        float sgn) {
    typedef typename Mma<DT>::elem elem;
    const int half = dh / 2;
    const int64_t per_row = ncols / 8;
    const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (i >= (int64_t)heads * half * per_row) return;
    const int64_t c0 = (i % per_row) * 8;
    const int64_t hj = i / per_row;
    const int h = (int)(hj / half), j = (int)(hj % half);
    elem *a = static_cast<elem *>(yt) + ((int64_t)h * dh + j) * ldt + c0;
    elem *b = a + (int64_t)half * ldt;
    float av[8], bv[8], ao[8], bo[8];
    load8<DT>(a, av);
    load8<DT>(b, bv);
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        const float2 cs = tab[(int64_t)((c0 + k) % T) * half + j];
        const float s = sgn * cs.y;
        ao[k] = av[k] * cs.x - bv[k] * s;
        bo[k] = bv[k] * cs.x + av[k] * s;
    }
    store8<DT>(a, ao);
    store8<DT>(b, bo);
}

inline unsigned blocks_of(int64_t n) { return (unsigned)((n + 255) / 256); }
}  // namespace

size_t rope_table_bytes(int T, int dh) { return (size_t)T * (dh / 2) * sizeof(float2); }

hipError_t launch_rope_table(int T, int dh, double theta, float2 *tab, float4 *tab_t, hipStream_t st) {
    if (dh % 4) return hipErrorInvalidValue;
    rope_table_kernel<<<blocks_of((int64_t)T * (dh / 4)), 256, 0, st>>>(T, dh, theta, tab, tab_t);
    return hipGetLastError();
}

hipError_t launch_rope_rows(int dtype, const float *src, int64_t lds, void *dst, int64_t ldd, int64_t M, int T,
                            int heads, int dh, const float2 *tab, hipStream_t st) {
    if (dh % 16 || M <= 0) return M <= 0 ? hipSuccess : hipErrorInvalidValue;
    const int64_t n = M * heads * (dh / 16);
    switch (dtype) {
    case F32: rope_rows_kernel<F32><<<blocks_of(n), 256, 0, st>>>(src, lds, dst, ldd, M, T, heads, dh, tab); break;
    case F16: rope_rows_kernel<F16><<<blocks_of(n), 256, 0, st>>>(src, lds, dst, ldd, M, T, heads, dh, tab); break;
    default: rope_rows_kernel<BF16><<<blocks_of(n), 256, 0, st>>>(src, lds, dst, ldd, M, T, heads, dh, tab); break;
    }
    return hipGetLastError();
}

hipError_t launch_rope_cols(int dtype, void *yt, int64_t ldt, int64_t ncols, int T, int heads, int dh,
                            const float2 *tab, bool inverse, hipStream_t st) {
    if (dh % 16 || ncols % 8 || ncols > ldt) return hipErrorInvalidValue;
    const int64_t n = (int64_t)heads * (dh / 2) * (ncols / 8);
    const float sgn = inverse ? -1.f : 1.f;
    switch (dtype) {
    case F32: rope_cols_kernel<F32><<<blocks_of(n), 256, 0, st>>>(yt, ldt, ncols, T, heads, dh, tab, sgn); break;
    case F16: rope_cols_kernel<F16><<<blocks_of(n), 256, 0, st>>>(yt, ldt, ncols, T, heads, dh, tab, sgn); break;
    default: rope_cols_kernel<BF16><<<blocks_of(n), 256, 0, st>>>(yt, ldt, ncols, T, heads, dh, tab, sgn); break;
    }
    return hipGetLastError();
}

}  // namespace jab
