// quant.hip -- per-(output row, group) quantizer of the fused QKV weight.
//
// Paper: Method, eq. quant (grid and clipping), Appendix "Joint STE fine-tuning"
// (1) (one scale per (output row, group)).  Asymmetric variant: scale and integer
// zero-point from the group's min-max range with 0 included.
//
// Work decomposition: one thread owns 8 consecutive weights of one row.  A group
// of g weights is g/8 consecutive lanes (g in {32, 64, 128} -> 4, 8, 16 lanes),
// so min/max reductions are lane shuffles inside one wavefront.  Loads and
// stores are 16-byte (32-byte for fp32) per thread and fully coalesced.  Every
// fp32 operation is IEEE-rounded (correctly rounded division, no contraction,
// no flush of denormals) so codes are bit-identical to an fp32 reference.
#include "device_common.h"
#include "kernels.h"

namespace jab {
namespace {

template <int DT> struct Chunk8;
template <> struct Chunk8<BF16> {
    u16x8 v;
    __device__ float get(int i) const { return bf16_bits_to_f32(v[i]); }
};
template <> struct Chunk8<F16> {
    u16x8 v;
    __device__ float get(int i) const { return f16_bits_to_f32(v[i]); }
};
template <> struct Chunk8<F32> {
    f32x4 a, b;
    __device__ float get(int i) const { return i < 4 ? a[i] : b[i - 4]; }
};

template <int DT>
__device__ inline void load8(const void *w, int64_t e, float out[8]) {
    if constexpr (DT == F32) {
        const f32x4 *p = reinterpret_cast<const f32x4 *>(static_cast<const float *>(w) + e);
        Chunk8<F32> c{p[0], p[1]};
#pragma unroll
        for (int i = 0; i < 8; ++i) out[i] = c.get(i);
    } else {
        Chunk8<DT> c{*reinterpret_cast<const u16x8 *>(static_cast<const uint16_t *>(w) + e)};
#pragma unroll
        for (int i = 0; i < 8; ++i) out[i] = c.get(i);
    }
}

template <int DT>
__device__ inline void store8(void *dst, int64_t e, const float v[8]) {
    if constexpr (DT == F32) {
        f32x4 *p = reinterpret_cast<f32x4 *>(static_cast<float *>(dst) + e);
        p[0] = f32x4{v[0], v[1], v[2], v[3]};
        p[1] = f32x4{v[4], v[5], v[6], v[7]};
    } else {
        u16x8 o;
#pragma unroll
        for (int i = 0; i < 8; ++i) o[i] = from_f32<DT>(v[i]);
        *reinterpret_cast<u16x8 *>(static_cast<uint16_t *>(dst) + e) = o;
    }
}

__device__ inline int matrix_of_row(int r, int row_k, int row_v) {
    return r < row_k ? 0 : (r < row_v ? 1 : 2);
}

// ------------------------------------------------------------------ quant-init
template <int DT>
__global__ __launch_bounds__(256) void quant_init_kernel(QuantShape sh, const void *__restrict__ w,
                                                         float *__restrict__ scale,
                                                         uint8_t *__restrict__ zero) {
    const int64_t chunk = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;   // 8 weights each
    const int64_t nchunks = (int64_t)sh.rows * sh.cols / 8;
    const int lpg = sh.group / 8;                     // lanes per group (power of two)
    // Threads past the end still take part in the shuffles (their lanes hold
    // neutral values); chunks never straddle groups since g is a multiple of 8.
    const bool live = chunk < nchunks;
    const int64_t e = live ? chunk * 8 : 0;
    const int r = (int)(e / sh.cols);
    const int col = (int)(e % sh.cols);
    const int m = matrix_of_row(r, sh.row_k, sh.row_v);
    const int bits = sh.bits[m];
    float v[8];
    load8<DT>(w, e, v);
    float lo = 0.f, hi = 0.f, amax = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        lo = fminf(lo, v[i]);
        hi = fmaxf(hi, v[i]);
        amax = fmaxf(amax, fabsf(v[i]));
    }
    for (int off = lpg / 2; off >= 1; off >>= 1) {
        lo = fminf(lo, __shfl_xor(lo, off, 64));
        hi = fmaxf(hi, __shfl_xor(hi, off, 64));
        amax = fmaxf(amax, __shfl_xor(amax, off, 64));
    }
    if (!live || (threadIdx.x & (lpg - 1)) != 0)
        return;
    const int64_t gi = (int64_t)r * (sh.cols / sh.group) + col / sh.group;
    float s = 1.f;
    int z = 0;
    if (bits != 0) {
        if (sh.scheme == 0) {
            const float levels = (float)((1 << bits) - 1);
            const float range = hi - lo;
            s = range / levels;
            if (s == 0.f) s = 1.f;
            float zf = rintf(-lo / s);
            zf = fminf(fmaxf(zf, 0.f), levels);
            z = (int)zf;
        } else {
            const float qmax = (float)((1 << (bits - 1)) - 1);
            s = amax / qmax;
            if (s == 0.f) s = 1.f;
        }
    }
    scale[gi] = s;
    if (zero) zero[gi] = (uint8_t)z;
}

// ------------------------------------------------------------------ fake quant
// Writes any of: codes (u8), w_hat (fp32), w_op (dtype; the projection operand),
// and per-block partial sums of (w_hat - w)^2 and w^2 for each matrix.  A thread takes
// QCPT chunks of 8 weights, 256 chunks apart (each of the block's QCPT passes reads 4 KiB
// (bf16) contiguously); all of its loads are issued before the arithmetic.
constexpr int QCPT = 4;

template <int DT>
__device__ inline void quant_chunk(const QuantShape &sh, int64_t e, const float v[8], const float *__restrict__ scale,
                                   const uint8_t *__restrict__ zero, uint8_t *__restrict__ codes,
                                   float *__restrict__ w_hat, void *__restrict__ w_op, bool want_err, double err[3],
                                   double nrm[3]) {
    // rows * cols fits 32 bits (problem validation) and the group size is a power of two
    const uint32_t eu = (uint32_t)e, cols = (uint32_t)sh.cols;
    const int r = (int)(eu / cols);
    const uint32_t col = eu - (uint32_t)r * cols;
    const int m = matrix_of_row(r, sh.row_k, sh.row_v);
    const int bits = sh.bits[m];
    float wh[8];
    uint8_t q8[8];
    if (bits == 0) {
#pragma unroll
        for (int i = 0; i < 8; ++i) { wh[i] = v[i]; q8[i] = 0; }
    } else {
        const int gsh = __builtin_ctz((unsigned)sh.group);
        const uint32_t gi = (uint32_t)r * (cols >> gsh) + (col >> gsh);
        const float s = scale[gi];
        float u[8];                                    // round half to even of fp32(v / s)
        if (s >= 0x1p-60f && s <= 0x1p60f) {
            // One correctly rounded reciprocal per chunk instead of eight divisions: with rs the
            // correctly rounded 1/s and q0 = fp32(v rs) (within one ulp of v / s), the remainder
            // v - q0 s is exact in one fma and q0 + rem rs, rounded once, is the correctly rounded
            // quotient (Markstein's theorem on division by a refined reciprocal, IBM J. Res. Dev.
            // 34(1), 1990).  The range of s keeps the remainder clear of underflow wherever the
            // quotient can round to a non-zero integer; an overflowing q0 is kept (infinite, as the
            // quotient is).
            const float rs = 1.f / s;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const float q0 = v[i] * rs;
                const float rem = __builtin_fmaf(-q0, s, v[i]);
                u[i] = rintf(__builtin_isinf(q0) ? q0 : __builtin_fmaf(rem, rs, q0));
            }
        } else {
#pragma unroll
            for (int i = 0; i < 8; ++i) u[i] = rintf(v[i] / s);
        }
        if (sh.scheme == 0) {
            const float levels = (float)((1 << bits) - 1);
            const float zf = (float)zero[gi];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const float q = fminf(fmaxf(u[i] + zf, 0.f), levels);
                q8[i] = (uint8_t)q;
                wh[i] = (q - zf) * s;
            }
        } else {
            const float qmax = (float)((1 << (bits - 1)) - 1);
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const float q = fminf(fmaxf(u[i], -qmax), qmax);
                q8[i] = (uint8_t)(int)(q + qmax);
                wh[i] = q * s;
            }
        }
    }
    if (codes) {
        uint32_t lo = q8[0] | (q8[1] << 8) | (q8[2] << 16) | ((uint32_t)q8[3] << 24);
        uint32_t hi = q8[4] | (q8[5] << 8) | (q8[6] << 16) | ((uint32_t)q8[7] << 24);
        *reinterpret_cast<uint2 *>(codes + e) = make_uint2(lo, hi);
    }
    if (w_hat) store8<F32>(w_hat, e, wh);
    if (w_op) store8<DT>(w_op, e, wh);
    if (want_err) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const double d = (double)wh[i] - (double)v[i];
            err[m] += d * d;
            nrm[m] += (double)v[i] * (double)v[i];
        }
    }
}

template <int DT>
__global__ __launch_bounds__(256) void quantize_kernel(QuantShape sh, const void *__restrict__ w,
                                                       const float *__restrict__ scale,
                                                       const uint8_t *__restrict__ zero,
                                                       uint8_t *__restrict__ codes,
                                                       float *__restrict__ w_hat,
                                                       void *__restrict__ w_op,
                                                       double *__restrict__ werr_part) {
    const int64_t nchunks = (int64_t)sh.rows * sh.cols / 8;
    const int64_t c0 = (int64_t)blockIdx.x * (256 * QCPT) + threadIdx.x;
    double err[3] = {0, 0, 0}, nrm[3] = {0, 0, 0};
    float v[QCPT][8];
#pragma unroll
    for (int i = 0; i < QCPT; ++i)
        if (c0 + i * 256 < nchunks) load8<DT>(w, (c0 + i * 256) * 8, v[i]);
#pragma unroll
    for (int i = 0; i < QCPT; ++i)
        if (c0 + i * 256 < nchunks)
            quant_chunk<DT>(sh, (c0 + i * 256) * 8, v[i], scale, zero, codes, w_hat, w_op, werr_part != nullptr, err,
                            nrm);
    if (!werr_part)
        return;
    // block reduction in a fixed order: wave sums, then the waves in order
    __shared__ double red[4][6];
    const int lane = lane_id(), wave = threadIdx.x >> 6;
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        const double a = wave_sum_f64(err[k]);
        const double b = wave_sum_f64(nrm[k]);
        if (lane == 0) { red[wave][2 * k] = a; red[wave][2 * k + 1] = b; }
    }
    __syncthreads();
    if (threadIdx.x < 6) {
        double t = 0;
        for (int i = 0; i < 4; ++i) t += red[i][threadIdx.x];
        werr_part[(int64_t)blockIdx.x * 6 + threadIdx.x] = t;
    }
}

// Sum of the per-block [6] partials in a fixed order, in two stages: workgroup g of
// kWerrGroups sums the blocks g L .. g L + L - 1 (thread t every 256th from t, then the waves
// in order) into stage[g][6]; one wavefront then sums the groups (lane l every 64th from l).
constexpr int kWerrGroups = 256;

__global__ __launch_bounds__(256) void werr_stage1_kernel(const double *__restrict__ part, int nblocks, int per,
                                                         double *__restrict__ stage) {
    const int g = blockIdx.x, lane = lane_id(), wave = threadIdx.x >> 6;
    const int b0 = g * per, b1 = min(nblocks, b0 + per);
    double acc[6] = {0, 0, 0, 0, 0, 0};
    for (int i = b0 + (int)threadIdx.x; i < b1; i += 256)
#pragma unroll
        for (int k = 0; k < 6; ++k) acc[k] += part[(int64_t)i * 6 + k];
    __shared__ double red[4][6];
#pragma unroll
    for (int k = 0; k < 6; ++k) {
        const double t = wave_sum_f64(acc[k]);
        if (lane == 0) red[wave][k] = t;
    }
    __syncthreads();
    if (threadIdx.x < 6) {
        double t = 0;
        for (int i = 0; i < 4; ++i) t += red[i][threadIdx.x];
        stage[g * 6 + threadIdx.x] = t;
    }
}

__global__ __launch_bounds__(64) void werr_reduce_kernel(const double *__restrict__ stage, int ngroups,
                                                         double *__restrict__ out) {
    const int lane = lane_id();
    double acc[6] = {0, 0, 0, 0, 0, 0};
    for (int i = lane; i < ngroups; i += 64)
#pragma unroll
        for (int k = 0; k < 6; ++k) acc[k] += stage[i * 6 + k];
#pragma unroll
    for (int k = 0; k < 6; ++k) {
        const double t = wave_sum_f64(acc[k]);
        if (lane == 0) out[k] = t;
    }
}

}  // namespace

static inline int blocks_for(const QuantShape &sh) {
    const int64_t nchunks = (int64_t)sh.rows * sh.cols / 8;
    return (int)((nchunks + 255) / 256);
}

int quant_blocks(const QuantShape &sh) {
    const int64_t nchunks = (int64_t)sh.rows * sh.cols / 8;
    return (int)((nchunks + 256 * QCPT - 1) / (256 * QCPT));
}

size_t werr_scratch_doubles(const QuantShape &sh) { return (size_t)(quant_blocks(sh) + kWerrGroups) * 6; }

hipError_t launch_quant_init(const QuantShape &sh, int dtype, const void *w, float *scale,
                             uint8_t *zero, hipStream_t st) {
    const dim3 grid(blocks_for(sh)), block(256);
    switch (dtype) {
    case F32: quant_init_kernel<F32><<<grid, block, 0, st>>>(sh, w, scale, zero); break;
    case F16: quant_init_kernel<F16><<<grid, block, 0, st>>>(sh, w, scale, zero); break;
    default: quant_init_kernel<BF16><<<grid, block, 0, st>>>(sh, w, scale, zero); break;
    }
    return hipGetLastError();
}

hipError_t launch_quantize(const QuantShape &sh, int dtype, const void *w, const float *scale,
                           const uint8_t *zero, uint8_t *codes, float *w_hat, void *w_op,
                           double *werr_part, hipStream_t st) {
    const dim3 grid(quant_blocks(sh)), block(256);
    switch (dtype) {
    case F32: quantize_kernel<F32><<<grid, block, 0, st>>>(sh, w, scale, zero, codes, w_hat, w_op, werr_part); break;
    case F16: quantize_kernel<F16><<<grid, block, 0, st>>>(sh, w, scale, zero, codes, w_hat, w_op, werr_part); break;
    default: quantize_kernel<BF16><<<grid, block, 0, st>>>(sh, w, scale, zero, codes, w_hat, w_op, werr_part); break;
    }
    return hipGetLastError();
}

hipError_t launch_werr_reduce(const QuantShape &sh, double *scratch, double *out, hipStream_t st) {
    const int nblocks = quant_blocks(sh);
    const int per = (nblocks + kWerrGroups - 1) / kWerrGroups;
    double *stage = scratch + (size_t)nblocks * 6;
    werr_stage1_kernel<<<kWerrGroups, 256, 0, st>>>(scratch, nblocks, per, stage);
    werr_reduce_kernel<<<1, 64, 0, st>>>(stage, kWerrGroups, out);
    return hipGetLastError();
}

}  // namespace jab
