// reduce.hip -- deterministic reduction of the fused squared-error partials.
//
// Paper: eq. joint_loss (the Frobenius sum, reported as sse) and the Appendix on
// the effective weight of the KL term (the implementation's element-wise mean,
// reported as mse = sse / (B T n_heads d_head)); Appendix "Evaluation metrics in
// full", M4 (eps^A needs the teacher's sum of squares, reported alongside).
//
// Each attention wavefront leaves one (sse, sum a^2) pair in fp64.  One wavefront
// per (set, sequence) sums its pairs with a lane-strided loop and a butterfly in a
// fixed order, then one wavefront per set sums the sequences.  No atomics, so the
// result is bitwise reproducible.
#include "device_common.h"
#include "kernels.h"

namespace jab {
namespace {

__global__ __launch_bounds__(64) void reduce_seq_kernel(const double *__restrict__ part, int batch,
                                                        int per_seq, double *__restrict__ seq_sums) {
    const int b = blockIdx.x, set = blockIdx.y, lane = lane_id();
    const double *p = part + ((int64_t)set * batch + b) * per_seq * 2;
    double s0 = 0, s1 = 0;
    for (int i = lane; i < per_seq; i += 64) {
        s0 += p[2 * i];
        s1 += p[2 * i + 1];
    }
    s0 = wave_sum_f64(s0);
    s1 = wave_sum_f64(s1);
    if (lane == 0) {
        seq_sums[((int64_t)set * batch + b) * 2] = s0;
        seq_sums[((int64_t)set * batch + b) * 2 + 1] = s1;
    }
}

__global__ __launch_bounds__(64) void reduce_final_kernel(const double *__restrict__ seq_sums, int batch,
                                                          double inv_n, double *__restrict__ out,
                                                          int stride, int with_stats, int per_seq_out) {
    const int set = blockIdx.x, lane = lane_id();
    const double *p = seq_sums + (int64_t)set * batch * 2;
    double s0 = 0, s1 = 0;
    for (int i = lane; i < batch; i += 64) {
        s0 += p[2 * i];
        s1 += p[2 * i + 1];
    }
    s0 = wave_sum_f64(s0);
    s1 = wave_sum_f64(s1);
    double *o = out + (int64_t)set * stride;
    if (lane == 0) {
        o[0] = s0;
        if (with_stats) {
            o[1] = s0 * inv_n;
            o[2] = s1;
        }
    }
    if (per_seq_out) {
        const int base = with_stats ? 3 : 1;
        for (int i = lane; i < batch; i += 64) o[base + i] = p[2 * i];
    }
}

__global__ __launch_bounds__(64) void reduce_sweep_kernel(const double *__restrict__ seq_sums, int batch,
                                                          double *__restrict__ loss,
                                                          double *__restrict__ loss_per_seq) {
    const int set = blockIdx.x, lane = lane_id();
    const double *p = seq_sums + (int64_t)set * batch * 2;
    double s0 = 0;
    for (int i = lane; i < batch; i += 64) s0 += p[2 * i];
    s0 = wave_sum_f64(s0);
    if (lane == 0) loss[set] = s0;
    if (loss_per_seq)
        for (int i = lane; i < batch; i += 64) loss_per_seq[(int64_t)set * batch + i] = p[2 * i];
}

}  // namespace

hipError_t launch_reduce_seq(const double *partials, int n_sets, int batch, int per_seq,
                             double *seq_sums, hipStream_t st) {
    reduce_seq_kernel<<<dim3(batch, n_sets), dim3(64), 0, st>>>(partials, batch, per_seq, seq_sums);
    return hipGetLastError();
}

hipError_t launch_reduce_final(const double *seq_sums, int n_sets, int batch, double inv_n,
                               double *out, int stride, int with_stats, int per_seq_out,
                               hipStream_t st) {
    reduce_final_kernel<<<dim3(n_sets), dim3(64), 0, st>>>(seq_sums, batch, inv_n, out, stride,
                                                           with_stats, per_seq_out);
    return hipGetLastError();
}

namespace {
constexpr int SUMSQ_BLOCKS = 256;   // partial sums per unit

// stage 1: block (b, u) sums the squares of its contiguous chunk of unit u's elements
// (float4 loads, fp64 accumulation, fixed lane and wave order)
__global__ __launch_bounds__(256) void unit_sumsq_kernel(const float *__restrict__ a, int64_t d, UnitRows rows,
                                                         double *__restrict__ part) {
    const int u = blockIdx.y, b = blockIdx.x, tid = threadIdx.x;
    const int64_t n4 = (rows.r[u + 1] - rows.r[u]) * d / 4;
    const float4 *src = reinterpret_cast<const float4 *>(a + rows.r[u] * d);
    const int64_t chunk = (n4 + SUMSQ_BLOCKS - 1) / SUMSQ_BLOCKS;
    const int64_t i0 = (int64_t)b * chunk, i1 = i0 + chunk < n4 ? i0 + chunk : n4;
    double acc = 0.0;
    for (int64_t i = i0 + tid; i < i1; i += 256) {
        const float4 v = src[i];
        acc += (double)v.x * v.x + (double)v.y * v.y + (double)v.z * v.z + (double)v.w * v.w;
    }
    acc = wave_sum_f64(acc);
    __shared__ double wsum[4];
    if (lane_id() == 0) wsum[tid >> 6] = acc;
    __syncthreads();
    if (tid == 0) part[u * SUMSQ_BLOCKS + b] = (wsum[0] + wsum[1]) + (wsum[2] + wsum[3]);
}

// stage 2: one wavefront per unit sums its partials
__global__ __launch_bounds__(64) void unit_sumsq_final_kernel(const double *__restrict__ part,
                                                              double *__restrict__ out) {
    const int u = blockIdx.x, lane = lane_id();
    double acc = 0.0;
    for (int i = lane; i < SUMSQ_BLOCKS; i += 64) acc += part[u * SUMSQ_BLOCKS + i];
    acc = wave_sum_f64(acc);
    if (lane == 0) out[u] = acc;
}
}  // namespace

size_t unit_sumsq_part_bytes(int n_units) { return (size_t)n_units * SUMSQ_BLOCKS * sizeof(double); }

hipError_t launch_unit_sumsq(const float *a, int64_t d, const UnitRows &rows, int n_units, double *part,
                             double *out, hipStream_t st) {
    if (n_units < 1 || n_units > 3 || d % 4) return hipErrorInvalidValue;
    unit_sumsq_kernel<<<dim3(SUMSQ_BLOCKS, n_units), dim3(256), 0, st>>>(a, d, rows, part);
    unit_sumsq_final_kernel<<<dim3(n_units), dim3(64), 0, st>>>(part, out);
    return hipGetLastError();
}

hipError_t launch_reduce_sweep(const double *seq_sums, int n_sets, int batch, double *loss,
                               double *loss_per_seq, hipStream_t st) {
    reduce_sweep_kernel<<<dim3(n_sets), dim3(64), 0, st>>>(seq_sums, batch, loss, loss_per_seq);
    return hipGetLastError();
}

}  // namespace jab
