// ste.hip -- device steps of the joint STE fine-tuning loop (Appendix "Joint STE fine-tuning"):
// Adam on the fp32 latent weights and on the per-(row, group) scales with grid-relative rates
// (eq. lr), the held-out commit gate, and the flip-rate count (eq. flip).
//
// Every kernel reads its data-dependent scalars (the mean grid step, the held-out loss, the gate
// flag) from device memory, so the host loop issues a whole run without synchronising.
// Reductions are in a fixed order (fp64 sums, integer counts): runs are bitwise reproducible.
#include "device_common.h"
#include "kernels.h"

namespace jab {
namespace {

inline int grid_for(int64_t n) { return (int)(n + 255 < 256 * 8192LL ? (n + 255) / 256 : 8192); }

// dst = dtype(src)
template <int DT>
__global__ __launch_bounds__(256) void round_to_dtype_kernel(const float *__restrict__ src, void *__restrict__ dst,
                                                             int64_t n) {
    typedef typename Mma<DT>::elem elem;
    elem *d = static_cast<elem *>(dst);
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        d[i] = from_f32<DT>(src[i]);
}

// One Adam step (fp32): m, v moments; lr = rate * mean grid step; theta >= floor after the step;
// copy = dtype(theta) when requested.
template <int DT>
__global__ __launch_bounds__(256) void adam_kernel(float *__restrict__ theta, const float *__restrict__ g,
                                                   float *__restrict__ m, float *__restrict__ v, int64_t n, AdamStep a,
                                                   const double *__restrict__ sbar, void *__restrict__ copy) {
    typedef typename Mma<DT>::elem elem;
    const float lr = a.rate * (float)(*sbar);
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        const float gi = g[i];
        const float mi = a.beta1 * m[i] + (1.f - a.beta1) * gi;
        const float vi = a.beta2 * v[i] + (1.f - a.beta2) * (gi * gi);
        m[i] = mi;
        v[i] = vi;
        const float mh = mi / a.bc1, vh = vi / a.bc2;
        float t = theta[i] - lr * (mh / (sqrtf(vh) + a.eps));
        if (a.floor > 0.f && !(t >= a.floor)) t = a.floor;
        theta[i] = t;
        if (copy) static_cast<elem *>(copy)[i] = from_f32<DT>(t);
    }
}

// sbar = mean of the scales over the rows of the quantized units (fixed order), 0 if none
__global__ __launch_bounds__(256) void mean_scale_kernel(const float *__restrict__ s, int64_t groups, UnitRows rows,
                                                         int unit_mask, double *__restrict__ sbar) {
    const int tid = threadIdx.x;
    double acc = 0.0;
    int64_t count = 0;
    for (int u = 0; u < 3; ++u) {
        if (!((unit_mask >> u) & 1)) continue;
        const int64_t i0 = rows.r[u] * groups, i1 = rows.r[u + 1] * groups;
        for (int64_t i = i0 + tid; i < i1; i += 256) acc += (double)s[i];
        count += i1 - i0;
    }
    acc = wave_sum_f64(acc);
    __shared__ double wsum[4];
    if (lane_id() == 0) wsum[tid >> 6] = acc;
    __syncthreads();
    if (tid == 0) *sbar = count ? ((wsum[0] + wsum[1]) + (wsum[2] + wsum[3])) / (double)count : 0.0;
}

// the commit gate: take the evaluated loss as the new best if it is strictly lower (or when
// forced, at the start); record it in the evaluation log
__global__ void gate_kernel(const double *__restrict__ loss, double *__restrict__ stats, int step, int log_slot,
                            int force, int *__restrict__ flag) {
    if (threadIdx.x != 0) return;
    const double l = *loss;
    const int take = force || l < stats[1];
    if (take) {
        stats[1] = l;
        stats[2] = (double)step;
    }
    if (force) stats[0] = l;
    if (log_slot >= 0) stats[log_slot] = l;
    *flag = take;
}

__global__ __launch_bounds__(256) void copy_if_kernel(const int *__restrict__ flag, const float *__restrict__ src,
                                                      float *__restrict__ dst, int64_t n) {
    if (flag && !*flag) return;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        dst[i] = src[i];
}

__global__ void axpy_f64_kernel(const double *__restrict__ a, const double *__restrict__ b, double lam,
                                double *__restrict__ out) {
    if (threadIdx.x == 0) *out = b ? *a + lam * *b : *a;
}

constexpr int DIFF_BLOCKS = 256;   // partial counts per unit

// stage 1: block (b, u) counts the positions of its chunk of unit u where the codes differ
__global__ __launch_bounds__(256) void count_diff_kernel(const uint8_t *__restrict__ a, const uint8_t *__restrict__ b,
                                                         int64_t d, UnitRows rows, long long *__restrict__ part) {
    const int u = blockIdx.y, blk = blockIdx.x, tid = threadIdx.x;
    const int64_t base = rows.r[u] * d, n = (rows.r[u + 1] - rows.r[u]) * d;
    const int64_t chunk = (n + DIFF_BLOCKS - 1) / DIFF_BLOCKS;
    const int64_t i0 = (int64_t)blk * chunk, i1 = i0 + chunk < n ? i0 + chunk : n;
    long long c = 0;
    for (int64_t i = i0 + tid; i < i1; i += 256) c += a[base + i] != b[base + i];
    __shared__ long long cs[256];
    cs[tid] = c;
    __syncthreads();
    for (int off = 128; off > 0; off >>= 1) {
        if (tid < off) cs[tid] += cs[tid + off];
        __syncthreads();
    }
    if (tid == 0) part[u * DIFF_BLOCKS + blk] = cs[0];
}

// stage 2: out[u] = count / elements of unit u (0 for units outside the mask)
__global__ void count_diff_final_kernel(const long long *__restrict__ part, int64_t d, UnitRows rows, int unit_mask,
                                        double *__restrict__ out) {
    const int u = threadIdx.x;
    if (u >= 3) return;
    long long c = 0;
    for (int i = 0; i < DIFF_BLOCKS; ++i) c += part[u * DIFF_BLOCKS + i];
    const int64_t n = (rows.r[u + 1] - rows.r[u]) * d;
    out[u] = ((unit_mask >> u) & 1) && n ? (double)c / (double)n : 0.0;
}

}  // namespace

hipError_t launch_round_to_dtype(int dtype, const float *src, void *dst, int64_t n, hipStream_t st) {
    switch (dtype) {
    case F32: round_to_dtype_kernel<F32><<<grid_for(n), 256, 0, st>>>(src, dst, n); break;
    case F16: round_to_dtype_kernel<F16><<<grid_for(n), 256, 0, st>>>(src, dst, n); break;
    default: round_to_dtype_kernel<BF16><<<grid_for(n), 256, 0, st>>>(src, dst, n); break;
    }
    return hipGetLastError();
}

hipError_t launch_adam(int dtype, float *theta, const float *g, float *m, float *v, int64_t n, const AdamStep &a,
                       const double *sbar, void *copy, hipStream_t st) {
    switch (dtype) {
    case F32: adam_kernel<F32><<<grid_for(n), 256, 0, st>>>(theta, g, m, v, n, a, sbar, copy); break;
    case F16: adam_kernel<F16><<<grid_for(n), 256, 0, st>>>(theta, g, m, v, n, a, sbar, copy); break;
    default: adam_kernel<BF16><<<grid_for(n), 256, 0, st>>>(theta, g, m, v, n, a, sbar, copy); break;
    }
    return hipGetLastError();
}

hipError_t launch_mean_scale(const float *s, int64_t groups, const UnitRows &rows, int unit_mask, double *sbar,
                             hipStream_t st) {
    mean_scale_kernel<<<1, 256, 0, st>>>(s, groups, rows, unit_mask, sbar);
    return hipGetLastError();
}

hipError_t launch_gate(const double *loss, double *stats, int step, int log_slot, int force, int *flag,
                       hipStream_t st) {
    gate_kernel<<<1, 64, 0, st>>>(loss, stats, step, log_slot, force, flag);
    return hipGetLastError();
}

hipError_t launch_copy_if(const int *flag, const float *src, float *dst, int64_t n, hipStream_t st) {
    copy_if_kernel<<<grid_for(n), 256, 0, st>>>(flag, src, dst, n);
    return hipGetLastError();
}

hipError_t launch_axpy_f64(const double *a, const double *b, double lam, double *out, hipStream_t st) {
    axpy_f64_kernel<<<1, 64, 0, st>>>(a, b, lam, out);
    return hipGetLastError();
}

size_t count_diff_part_bytes() { return 3 * DIFF_BLOCKS * sizeof(long long); }

hipError_t launch_count_diff(const uint8_t *a, const uint8_t *b, int64_t d, const UnitRows &rows, int unit_mask,
                             long long *part, double *out, hipStream_t st) {
    count_diff_kernel<<<dim3(DIFF_BLOCKS, 3), 256, 0, st>>>(a, b, d, rows, part);
    count_diff_final_kernel<<<1, 64, 0, st>>>(part, d, rows, unit_mask, out);
    return hipGetLastError();
}

}  // namespace jab

namespace jab {
namespace {
__global__ __launch_bounds__(256) void zero_f32_kernel(float *__restrict__ a, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        a[i] = 0.f;
}
}  // namespace

hipError_t launch_zero_f32(float *a, int64_t n, hipStream_t st) {
    zero_f32_kernel<<<grid_for(n), 256, 0, st>>>(a, n);
    return hipGetLastError();
}
}  // namespace jab
