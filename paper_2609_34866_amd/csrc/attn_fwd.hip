// attn_fwd.hip -- causal grouped-query softmax attention with a fused
// squared-error epilogue.
//
// Paper: Method, "Layer-wise PTQ": A(X) = softmax(Q K^T / sqrt(d_head) + M) V with
// causal mask M; "The joint attention loss" (eq. joint_loss): the squared
// Frobenius distance between the teacher output A(X) and the student output.
// The merged output puts head h in columns h*d_head .. h*d_head + d_head - 1
// (Appendix "Evaluation metrics in full", M4: the merged pre-projection output).
//
// gfx950 design
//  * A workgroup is 4 wavefronts; each wave owns 32 queries of one query head.
//    The workgroup's waves share one key/value head: with n_heads/n_kv_heads a
//    multiple of 4 they are 4 query heads of one group at the same 32 queries
//    (so every key/value tile read from memory serves 4 heads); with ratio 2 or 1
//    they are 2 heads x 64 queries or 1 head x 128 queries.
//  * Per 64-key block, K is staged in LDS row-major and V transposed (V^T), both
//    with a 16-byte row pad against bank conflicts.
//  * Scores are computed transposed, S^T = K Q^T, on 32x32 MFMAs: lane l then
//    owns query (l % 32) and 16 keys of each 32-key block, so the running max and
//    sum of a query need only a lane-local pass and one exchange with lane l^32.
//  * O^T = V^T P^T: the probabilities go from the score registers straight into
//    the B operand (the pairing of keys between the two operands only has to be
//    consistent, not in order), V^T is read from LDS.  Each lane's accumulators
//    all belong to its own query, so the online-softmax rescale is a scalar.
//  * exp via exp2 with log2(e)/sqrt(d_head) folded into one FMA per score.
//  * Query tiles are issued longest-first (causal work grows with the tile
//    index), and workgroup ids are remapped so one XCD processes all tiles of a
//    (sequence, key/value head) and reads its K/V through one L2.
//  * Epilogues: store the output (teacher or backward), or read the teacher
//    tile and accumulate (a - a_hat)^2 and a^2 per wave (loss); the student
//    output never goes to memory in the loss.  Both epilogues share one code path
//    for the output value, so a student equal to the teacher gives exactly 0.
#include "device_common.h"
#include "kernels.h"

namespace jab {
namespace {

constexpr int BN = 64;   // keys per iteration

template <int DT, int DH, int NV>
struct AttnCfg {
    typedef typename Mma<DT>::elem elem;
    static constexpr int EPC = 16 / (int)sizeof(elem);
    static constexpr int KST = DH + EPC;          // K row stride (elements), 16-byte pad
    static constexpr int VST = BN + EPC;          // V^T row stride (elements)
    static constexpr int NKC = DH / Mma<DT>::K;   // k-steps of Q K^T
    static constexpr int DHP = DH < 32 ? 32 : DH; // rows of V^T (padded to one MFMA block)
    static constexpr int NDB = DHP / 32;          // 32-row blocks of O^T
    static constexpr int K_ELEMS = BN * KST;
    static constexpr int V_ELEMS = DHP * VST;
    static constexpr size_t LDS_BYTES = (size_t)(K_ELEMS + NV * V_ELEMS) * sizeof(elem);
};

template <int DT, int DH, int NV>
__global__ __launch_bounds__(256, 2) void attn_fwd_kernel(AttnArgs a, float scale_log2, int hpw,
                                                          int nqt, int n_ht) {
    typedef AttnCfg<DT, DH, NV> C;
    typedef typename C::elem elem;
    typedef Mma<DT> MM;
    extern __shared__ __align__(16) unsigned char smem[];
    elem *Ks = reinterpret_cast<elem *>(smem);
    elem *Vt = Ks + C::K_ELEMS;

    const int T = a.seq_len, Hq = a.n_heads;
    const int G = Hq / a.n_kv_heads;
    const int QT = 128 / hpw;                      // queries per workgroup tile

    // ---- workgroup -> (sequence, head tile, query tile)
    const int nwg = gridDim.x;
    int lin = blockIdx.x;
    if ((nwg & 7) == 0)
        lin = (lin & 7) * (nwg >> 3) + (lin >> 3);
    const int qt = nqt - 1 - lin % nqt;
    const int ht = (lin / nqt) % n_ht;
    const int b = lin / (nqt * n_ht);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int h = ht * hpw + wave % hpw;
    const int kvh = h / G;
    const int q0 = qt * QT + (wave / hpw) * 32;
    const int qrow = q0 + (lane & 31);             // this lane's query
    const int half = lane >> 5;
    const bool active = q0 < T;
    const int kend = min(T, qt * QT + QT);

    const elem *Qg = static_cast<const elem *>(a.q);
    const elem *Kg = static_cast<const elem *>(a.k);
    const int64_t seq_row0 = (int64_t)b * T;

    // ---- this wave's queries as B operands of S^T = K Q^T
    typename MM::operand qf[C::NKC];
#pragma unroll
    for (int kc = 0; kc < C::NKC; ++kc) {
        const int k = kc * MM::K + half * MM::VEC;
        if constexpr (DT == F32) {
            qf[kc] = (qrow < T) ? Qg[(seq_row0 + qrow) * a.ld + h * DH + k] : 0.f;
        } else {
            u32x4 v = u32x4{0u, 0u, 0u, 0u};
            if (qrow < T)
                v = *reinterpret_cast<const u32x4 *>(Qg + (seq_row0 + qrow) * a.ld + h * DH + k);
            qf[kc] = __builtin_bit_cast(typename MM::operand, v);
        }
    }

    f32x16 o[NV][C::NDB];
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int d = 0; d < C::NDB; ++d)
#pragma unroll
            for (int e = 0; e < 16; ++e) o[v][d][e] = 0.f;
    float m_run = -INFINITY, l_run = 0.f;
    if constexpr (DH < 32) {       // padding rows of V^T stay zero for the whole kernel
        for (int i = tid; i < NV * C::V_ELEMS; i += 256) Vt[i] = from_f32<DT>(0.f);
    }

    constexpr int CPR = DH / C::EPC;               // 16-byte chunks per K/V row
    for (int kb = 0; kb < kend; kb += BN) {
        // ---- stage K (row-major) and V (transposed) of keys kb..kb+63 in LDS
        __syncthreads();
        for (int idx = tid; idx < BN * CPR; idx += 256) {
            const int r = idx / CPR, c = idx % CPR;
            const int key = kb + r;
            u32x4 kv = u32x4{0u, 0u, 0u, 0u};
            if (key < T)
                kv = *reinterpret_cast<const u32x4 *>(Kg + (seq_row0 + key) * a.ld + kvh * DH + c * C::EPC);
            *reinterpret_cast<u32x4 *>(Ks + r * C::KST + c * C::EPC) = kv;
#pragma unroll
            for (int v = 0; v < NV; ++v) {
                const elem *Vg = static_cast<const elem *>(a.v[v]);
                u32x4 vv = u32x4{0u, 0u, 0u, 0u};
                if (key < T)
                    vv = *reinterpret_cast<const u32x4 *>(Vg + (seq_row0 + key) * a.ld + kvh * DH + c * C::EPC);
                const elem *ve = reinterpret_cast<const elem *>(&vv);
                elem *vt = Vt + v * C::V_ELEMS;
#pragma unroll
                for (int i = 0; i < C::EPC; ++i) vt[(c * C::EPC + i) * C::VST + r] = ve[i];
            }
        }
        __syncthreads();
        if (!active || kb > q0 + 31)
            continue;

        // ---- S^T for the two 32-key halves of the block
        f32x16 s[2];
#pragma unroll
        for (int sb = 0; sb < 2; ++sb) {
#pragma unroll
            for (int e = 0; e < 16; ++e) s[sb][e] = 0.f;
            const int krow = sb * 32 + (lane & 31);
#pragma unroll
            for (int kc = 0; kc < C::NKC; ++kc) {
                const int k = kc * MM::K + half * MM::VEC;
                typename MM::operand ka;
                if constexpr (DT == F32)
                    ka = Ks[krow * C::KST + k];
                else
                    ka = __builtin_bit_cast(typename MM::operand,
                                            *reinterpret_cast<const u32x4 *>(Ks + krow * C::KST + k));
                s[sb] = MM::mma(ka, qf[kc], s[sb]);
            }
        }
        // ---- causal mask (only blocks that reach past this wave's first query)
        if (kb + BN - 1 > q0) {
#pragma unroll
            for (int sb = 0; sb < 2; ++sb)
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int key = kb + sb * 32 + 8 * (e >> 2) + 4 * half + (e & 3);
                    if (key > qrow) s[sb][e] = -INFINITY;
                }
        }
        // ---- online softmax (base 2)
        float mx = -INFINITY;
#pragma unroll
        for (int sb = 0; sb < 2; ++sb)
#pragma unroll
            for (int e = 0; e < 16; ++e) mx = fmaxf(mx, s[sb][e]);
        mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
        const float m_new = fmaxf(m_run, mx * scale_log2);
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
        float rs = 0.f;
#pragma unroll
        for (int sb = 0; sb < 2; ++sb)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(s[sb][e], scale_log2, -m_new));
                s[sb][e] = p;
                rs += p;
            }
        rs += __shfl_xor(rs, 32, 64);
        l_run = l_run * alpha + rs;
        m_run = m_new;
#pragma unroll
        for (int v = 0; v < NV; ++v)
#pragma unroll
            for (int d = 0; d < C::NDB; ++d)
#pragma unroll
                for (int e = 0; e < 16; ++e) o[v][d][e] *= alpha;

        // ---- O^T += V^T P^T
        if constexpr (DT == F32) {
#pragma unroll
            for (int kc2 = 0; kc2 < BN / MM::K; ++kc2) {
                const int sb = kc2 >> 4, e = kc2 & 15;
                const int key = sb * 32 + 8 * (e >> 2) + 4 * half + (e & 3);
                const float pb = s[sb][e];
#pragma unroll
                for (int v = 0; v < NV; ++v)
#pragma unroll
                    for (int d = 0; d < C::NDB; ++d) {
                        const float va = Vt[v * C::V_ELEMS + (d * 32 + (lane & 31)) * C::VST + key];
                        o[v][d] = MM::mma(va, pb, o[v][d]);
                    }
            }
        } else {
#pragma unroll
            for (int kc2 = 0; kc2 < BN / MM::K; ++kc2) {
                const int sb = kc2 >> 1, hf = kc2 & 1;
                u16x8 pbits;
#pragma unroll
                for (int i = 0; i < 8; ++i) pbits[i] = from_f32<DT>(s[sb][hf * 8 + i]);
                const typename MM::operand pb = __builtin_bit_cast(typename MM::operand, pbits);
                const int key0 = sb * 32 + hf * 16 + 4 * half;
#pragma unroll
                for (int v = 0; v < NV; ++v)
#pragma unroll
                    for (int d = 0; d < C::NDB; ++d) {
                        const elem *row = Vt + v * C::V_ELEMS + (d * 32 + (lane & 31)) * C::VST;
                        const u16x4 lo = *reinterpret_cast<const u16x4 *>(row + key0);
                        const u16x4 hi = *reinterpret_cast<const u16x4 *>(row + key0 + 8);
                        const u16x8 vb = u16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
                        o[v][d] = MM::mma(__builtin_bit_cast(typename MM::operand, vb), pb, o[v][d]);
                    }
            }
        }
    }

    // ---- epilogue
    const int per_seq = n_ht * nqt * 4;
    const int widx = (ht * nqt + qt) * 4 + wave;
    const float inv_l = active ? 1.f / l_run : 0.f;
    const int ac = Hq * DH;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
        float sse = 0.f, sa2 = 0.f;
        if (active && qrow < T) {
            const int64_t obase = (seq_row0 + qrow) * ac + h * DH;
#pragma unroll
            for (int d = 0; d < C::NDB; ++d)
#pragma unroll
                for (int e4 = 0; e4 < 4; ++e4) {
                    const int col = d * 32 + 8 * e4 + 4 * half;
                    if (DH < 32 && col >= DH) continue;
                    f32x4 val;
#pragma unroll
                    for (int i = 0; i < 4; ++i) val[i] = o[v][d][4 * e4 + i] * inv_l;
                    if (a.mode & ATT_LOSS) {
                        const f32x4 ref = *reinterpret_cast<const f32x4 *>(a.a_ref + obase + col);
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            const float df = ref[i] - val[i];
                            sse = __builtin_fmaf(df, df, sse);
                            sa2 = __builtin_fmaf(ref[i], ref[i], sa2);
                        }
                    }
                    if (a.mode & ATT_STORE_O)
                        *reinterpret_cast<f32x4 *>(a.a_out + obase + col) = val;
                }
            if ((a.mode & ATT_STORE_LSE) && half == 0)
                a.lse2[((int64_t)b * Hq + h) * T + qrow] = m_run + __builtin_amdgcn_logf(l_run);
        }
        if (a.mode & ATT_LOSS) {
            const double tse = wave_sum_f64((double)sse);
            const double ta2 = wave_sum_f64((double)sa2);
            if (lane == 0) {
                double *p = a.partials[v] + ((int64_t)b * per_seq + widx) * 2;
                p[0] = tse;
                p[1] = ta2;
            }
        }
    }
}

template <int DT, int DH, int NV>
hipError_t run_attn(const AttnArgs &a, hipStream_t st) {
    typedef AttnCfg<DT, DH, NV> C;
    const int G = a.n_heads / a.n_kv_heads;
    const int hpw = G % 4 == 0 ? 4 : G;            // heads per workgroup tile (1, 2 or 4)
    const int QT = 128 / hpw;
    const int nqt = (a.seq_len + QT - 1) / QT;
    const int n_ht = a.n_heads / hpw;
    const float scale_log2 = 1.4426950408889634f / sqrtf((float)DH);
    hipError_t e = hipFuncSetAttribute((const void *)attn_fwd_kernel<DT, DH, NV>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)C::LDS_BYTES);
    if (e != hipSuccess) return e;
    const int nwg = nqt * n_ht * a.batch;
    attn_fwd_kernel<DT, DH, NV><<<dim3(nwg), dim3(256), C::LDS_BYTES, st>>>(a, scale_log2, hpw, nqt, n_ht);
    return hipGetLastError();
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
    if (a.nv == 2) return dispatch_dh<DT, 2>(a, st);
    return dispatch_dh<DT, 1>(a, st);
}

template <>
hipError_t dispatch_nv<F32>(const AttnArgs &a, hipStream_t st) {
    // fp32 keeps one value tensor per pass (two would not fit the register file at d_head 128)
    return dispatch_dh<F32, 1>(a, st);
}

}  // namespace

int attn_max_nv(int dtype) { return dtype == F32 ? 1 : 2; }

int attn_waves_per_seq(int seq_len, int n_heads, int n_kv_heads) {
    const int G = n_heads / n_kv_heads;
    const int hpw = G % 4 == 0 ? 4 : G;
    const int QT = 128 / hpw;
    return ((seq_len + QT - 1) / QT) * (n_heads / hpw) * 4;
}

hipError_t launch_attn_fwd(int dtype, const AttnArgs &a, hipStream_t st) {
    if (a.batch <= 0 || a.seq_len <= 0) return hipSuccess;
    switch (dtype) {
    case F32: return dispatch_nv<F32>(a, st);
    case F16: return dispatch_nv<F16>(a, st);
    default: return dispatch_nv<BF16>(a, st);
    }
}

}  // namespace jab
