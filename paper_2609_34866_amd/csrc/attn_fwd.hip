// attn_fwd.hip -- instantiations of the attention kernel with one value tensor per pass
// (the teacher, the loss, the backward's forward, the sweep's single passes) and the
// V^T helper kernels.  The sweep's two-value-tensor passes are instantiated in
// attn_fwd_nv2.hip.
#include "attn_fwd_impl.h"
#include "attn_fwd_fast.h"

#ifndef ATT_NW
#define ATT_NW 4          // waves per workgroup of the 16-bit single-value path
#endif

namespace jab {

// defined in attn_fwd_nv2.hip and attn_fwd_fast_multi.hip
template <int DT, int DH>
hipError_t run_attn_nv2(const AttnArgs &a, hipStream_t st);
template <int DT, int DH, int NV>
hipError_t run_attn_fast_multi(const AttnArgs &a, hipStream_t st);

namespace {

// 16-bit dtypes with one value tensor: 4-wave workgroups, two per CU (two waves per SIMD).  The
// passes with several value tensors (the sweep's triples sharing b_Q and b_K) and fp32 need more
// registers per wave: one workgroup per CU, one wave per SIMD.
// 16-bit, head_dim 64 or 128, query heads per key/value head a multiple of 4: attn_fast_kernel
// (workgroups of four query heads of one group over 32 queries), with four value tensors per pass,
// two or one for the rest of the set; each query gets bitwise the same result
// whichever pass takes its value tensor.  Elsewhere the generic kernel takes the value tensors in
// pairs.
template <int DT, int DH, int NV>
hipError_t run_attn(const AttnArgs &a, hipStream_t st) {
    if constexpr (NV == 2) {                           // a.nv = 2 .. 4 value tensors
        hipError_t e = hipSuccess;
        AttnArgs b = a;
        if constexpr (DT != F32 && (DH == 64 || DH == 128)) {
            if ((a.n_heads / a.n_kv_heads) % 4 == 0) {
                for (int v0 = 0; v0 < a.nv && e == hipSuccess; v0 += b.nv) {
                    const int left = a.nv - v0;
                    b.nv = left >= 4 ? 4 : (left >= 2 ? 2 : 1);
                    for (int v = 0; v < b.nv; ++v) {
                        b.v[v] = a.v[v0 + v];
                        b.partials[v] = a.partials[v0 + v];
                    }
                    if (b.nv == 4) e = run_attn_fast_multi<DT, DH, 4>(b, st);
                    else e = b.nv == 2 ? run_attn_fast_multi<DT, DH, 2>(b, st) : launch_attn_fast<DT, DH>(b, st);
                }
                return e;
            }
        }
        for (int v0 = 0; v0 < a.nv && e == hipSuccess; v0 += 2) {
            b.nv = min(2, a.nv - v0);
            for (int v = 0; v < b.nv; ++v) {
                b.v[v] = a.v[v0 + v];
                b.partials[v] = a.partials[v0 + v];
            }
            e = b.nv == 2 ? run_attn_nv2<DT, DH>(b, st) : run_attn_cfg<DT, DH, 1, 1, ATT_NW>(b, st);
        }
        return e;
    } else if constexpr (DT != F32) {
        if constexpr (DH == 64 || DH == 128)
            if ((a.n_heads / a.n_kv_heads) % 4 == 0) return launch_attn_fast<DT, DH>(a, st);
        return run_attn_cfg<DT, DH, 1, 1, ATT_NW>(a, st);
    } else {
        return run_attn_cfg<DT, DH, 1, 1, 4>(a, st);
    }
}

template <int DT, int NV>
hipError_t dispatch_dh(const AttnArgs &a, hipStream_t st) {
    switch (a.head_dim) {
    case 16: return run_attn<DT, 16, NV>(a, st);
    case 64: return run_attn<DT, 64, NV>(a, st);
    default: return run_attn<DT, 128, NV>(a, st);
    }
}

template <int DT>
hipError_t dispatch_nv(const AttnArgs &a, hipStream_t st) {
    if (a.nv >= 2) return dispatch_dh<DT, 2>(a, st);
    return dispatch_dh<DT, 1>(a, st);
}

template <>
hipError_t dispatch_nv<F32>(const AttnArgs &a, hipStream_t st) {
    // fp32 keeps one value tensor per pass (two would not fit the register file at d_head 128)
    return dispatch_dh<F32, 1>(a, st);
}

// zero the padding columns [T, Tp) of every sequence of a transposed value tensor
template <typename E>
__global__ __launch_bounds__(256) void zero_vt_pad_kernel(E *__restrict__ vt, int rows, int64_t ld, int batch,
                                                          int T, int Tp) {
    const int w = Tp - T;
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t n = (int64_t)rows * batch * w;
    if (i >= n) return;
    const int c = (int)(i % w);
    const int64_t rb = i / w;
    const int bb = (int)(rb % batch);
    const int64_t r = rb / batch;
    vt[r * ld + (int64_t)bb * Tp + vt_perm(T + c)] = E(0);
}

// V [B*T][ldv] (natural token order) from V^T [rows][B*Tp] (vt_perm order)
template <typename E>
__global__ __launch_bounds__(256) void vt_to_v_kernel(const E *__restrict__ vt, E *__restrict__ v, int rows,
                                                      int64_t ldt, int batch, int T, int Tp, int ldv) {
    __shared__ E tile[32][33];
    const int bb = blockIdx.z, t0 = blockIdx.x * 32, r0 = blockIdx.y * 32;
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;      // 32 x 8
    for (int i = ty; i < 32; i += 8) {
        const int r = r0 + i, t = t0 + tx;
        tile[i][tx] = (r < rows && t < T) ? vt[(int64_t)r * ldt + (int64_t)bb * Tp + vt_perm(t)] : E(0);
    }
    __syncthreads();
    for (int i = ty; i < 32; i += 8) {
        const int t = t0 + i, r = r0 + tx;
        if (t < T && r < rows) v[((int64_t)bb * T + t) * ldv + r] = tile[tx][i];
    }
}

// The same for 2-byte elements with 16-byte global loads and stores, on 64 x 64 tiles (rows and T
// multiples of 64, ldt, Tp and ldv multiples of 8): a thread loads eight consecutive positions of a
// V^T row, the tile is turned in LDS (rows 33 words apart), and a thread stores eight consecutive
// channels of the token whose position it reads (the permutation is its own inverse).
__global__ __launch_bounds__(256) void vt_to_v16_kernel(const uint16_t *__restrict__ vt, uint16_t *__restrict__ v,
                                                        int64_t ldt, int T, int Tp, int ldv) {
    constexpr int LD = 66;                           // u16 per LDS row: 33 words
    __shared__ uint32_t tile[64 * LD / 2];
    const int bb = blockIdx.z, t0 = blockIdx.x * 64, r0 = blockIdx.y * 64;
    const int t = threadIdx.x, cc = t & 7;
#pragma unroll
    for (int pass = 0; pass < 2; ++pass) {
        const int i = (t >> 3) + 32 * pass;          // channel r0 + i, positions t0 + 8 cc .. + 7
        const u32x4 x = *reinterpret_cast<const u32x4 *>(vt + (int64_t)(r0 + i) * ldt + (int64_t)bb * Tp + t0 + 8 * cc);
#pragma unroll
        for (int k = 0; k < 4; ++k) tile[(i * LD + 8 * cc) / 2 + k] = x[k];
    }
    __syncthreads();
    const uint16_t *t16 = reinterpret_cast<const uint16_t *>(tile);
#pragma unroll
    for (int pass = 0; pass < 2; ++pass) {
        const int j = (t >> 3) + 32 * pass, pos = vt_perm(j);   // token t0 + j sits at position t0 + pos
        uint32_t w[4];
#pragma unroll
        for (int k = 0; k < 4; ++k)
            w[k] = (uint32_t)t16[(8 * cc + 2 * k) * LD + pos] | ((uint32_t)t16[(8 * cc + 2 * k + 1) * LD + pos] << 16);
        *reinterpret_cast<u32x4 *>(v + ((int64_t)bb * T + t0 + j) * ldv + r0 + 8 * cc) = u32x4{w[0], w[1], w[2], w[3]};
    }
}

}  // namespace

int attn_max_nv(int dtype) { return dtype == F32 ? 1 : 4; }

int attn_partials_per_seq(int seq_len, int n_heads) { return n_heads * ((seq_len + 31) / 32); }

hipError_t launch_attn_fwd(int dtype, const AttnArgs &a, hipStream_t st) {
    if (a.batch <= 0 || a.seq_len <= 0) return hipSuccess;
    switch (dtype) {
    case F32: return dispatch_nv<F32>(a, st);
    case F16: return dispatch_nv<F16>(a, st);
    default: return dispatch_nv<BF16>(a, st);
    }
}

hipError_t launch_zero_vt_pad(int dtype, void *vt, int rows, int64_t ld, int batch, int T, hipStream_t st) {
    const int Tp = vt_pad(T);
    if (Tp == T) return hipSuccess;
    const int64_t n = (int64_t)rows * batch * (Tp - T);
    const dim3 grid((unsigned)((n + 255) / 256)), block(256);
    if (dtype == F32) zero_vt_pad_kernel<float><<<grid, block, 0, st>>>(static_cast<float *>(vt), rows, ld, batch, T, Tp);
    else zero_vt_pad_kernel<uint16_t><<<grid, block, 0, st>>>(static_cast<uint16_t *>(vt), rows, ld, batch, T, Tp);
    return hipGetLastError();
}

hipError_t launch_vt_to_v(int dtype, const void *vt, void *v, int rows, int64_t ldt, int batch, int T, int ldv,
                          hipStream_t st) {
    const int Tp = vt_pad(T);
    const dim3 grid((T + 31) / 32, (rows + 31) / 32, batch), block(256);
    if (dtype == F32)
        vt_to_v_kernel<float><<<grid, block, 0, st>>>(static_cast<const float *>(vt), static_cast<float *>(v), rows, ldt, batch, T, Tp, ldv);
    else if (rows % 64 == 0 && T % 64 == 0 && ldt % 8 == 0 && Tp % 8 == 0 && ldv % 8 == 0 &&
             ((uintptr_t)vt & 15) == 0 && ((uintptr_t)v & 15) == 0)
        vt_to_v16_kernel<<<dim3(T / 64, rows / 64, batch), block, 0, st>>>(static_cast<const uint16_t *>(vt),
                                                                          static_cast<uint16_t *>(v), ldt, T, Tp, ldv);
    else
        vt_to_v_kernel<uint16_t><<<grid, block, 0, st>>>(static_cast<const uint16_t *>(vt), static_cast<uint16_t *>(v), rows, ldt, batch, T, Tp, ldv);
    return hipGetLastError();
}

}  // namespace jab
