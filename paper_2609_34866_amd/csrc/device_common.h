// device_common.h -- gfx950 building blocks shared by the kernels of libjab.
//
// Matrix-core conventions (CDNA3/CDNA4 MFMA, wave64) used throughout:
//   32x32xK products D[32][32] += A[32][K] * B[K][32].
//   A operand: lane l holds row (l % 32), VEC consecutive k values starting at
//              (l / 32) * VEC;  B operand: lane l holds column (l % 32) and the
//              same k values.  Any permutation of k applied identically to A and
//              B leaves the product unchanged, which the attention kernel uses
//              to feed a softmax tile straight from accumulator registers.
//   D (16 floats per lane): lane l holds column (l % 32) and rows
//              8 * (i / 4) + 4 * (l / 32) + (i % 4), i = 0..15.
#pragma once
#include <type_traits>

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace jab {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

enum Dtype { F32 = 0, F16 = 1, BF16 = 2 };

// Storage element and matrix-core operand for each dtype.
//   K    : reduction depth of one 32x32 MFMA
//   VEC  : k values one lane supplies per MFMA (= K / 2)
template <int DT> struct Mma;

template <> struct Mma<BF16> {
    typedef uint16_t elem;                   // raw bf16 bits in memory
    typedef bf16x8 operand;
    static constexpr int K = 16, VEC = 8;
    __device__ static inline f32x16 mma(operand a, operand b, f32x16 c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
    }
};

template <> struct Mma<F16> {
    typedef uint16_t elem;                   // raw fp16 bits in memory
    typedef f16x8 operand;
    static constexpr int K = 16, VEC = 8;
    __device__ static inline f32x16 mma(operand a, operand b, f32x16 c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
    }
};

template <> struct Mma<F32> {
    typedef float elem;
    typedef float operand;
    static constexpr int K = 2, VEC = 1;
    __device__ static inline f32x16 mma(operand a, operand b, f32x16 c) {
        return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
    }
};

// ---------------------------------------------------------------- conversions
// fp32 -> bf16 / fp16 with round-to-nearest-even (the hardware conversions
// v_cvt_pk_bf16_f32 / v_cvt_f16_f32 round to nearest even in the default mode).
__device__ inline uint16_t f32_to_bf16_bits(float x) {
    __bf16 h = (__bf16)x;
    return __builtin_bit_cast(uint16_t, h);
}
__device__ inline uint16_t f32_to_f16_bits(float x) {
    _Float16 h = (_Float16)x;
    return __builtin_bit_cast(uint16_t, h);
}
__device__ inline float bf16_bits_to_f32(uint16_t b) {
    return __builtin_bit_cast(float, (uint32_t)b << 16);
}
__device__ inline float f16_bits_to_f32(uint16_t b) {
    return (float)__builtin_bit_cast(_Float16, b);
}

template <int DT> __device__ inline float to_f32(typename Mma<DT>::elem v);
template <> __device__ inline float to_f32<BF16>(uint16_t v) { return bf16_bits_to_f32(v); }
template <> __device__ inline float to_f32<F16>(uint16_t v) { return f16_bits_to_f32(v); }
template <> __device__ inline float to_f32<F32>(float v) { return v; }

template <int DT> __device__ inline typename Mma<DT>::elem from_f32(float v);
template <> __device__ inline uint16_t from_f32<BF16>(float v) { return f32_to_bf16_bits(v); }
template <> __device__ inline uint16_t from_f32<F16>(float v) { return f32_to_f16_bits(v); }
template <> __device__ inline float from_f32<F32>(float v) { return v; }

// two fp32 values rounded to the 16-bit dtype (round to nearest even), packed
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
template <int DT>
__device__ inline uint32_t pack2(float x, float y) {
    if constexpr (DT == BF16) return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{x, y}, bf16x2_t));
    else return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{x, y}, f16x2_t));
}

// ---------------------------------------------------------------- wave reductions
// Sum over the 64 lanes of a wave, every lane receiving it: the butterfly v += v[lane ^ off] for
// off = 32, 16, 8, 4, 2, 1, all in VALU cross-lane moves (no LDS instruction, so it may run while
// the wave's direct-to-LDS loads are in flight).  The partner steps 32 and 16 use
// v_permlane32_swap / v_permlane16_swap (two copies of a value come back as the lower and the upper
// half, or row), the steps inside a row of 16 the DPP rotation row_ror:off, which pairs lane i with
// lane i ^ off wherever the values are already symmetric under the larger steps.  Each addition has
// the same two operands as in the plain butterfly (IEEE addition commutes), so the result is
// bitwise that of the shuffle version.
__device__ inline double wave_sum_f64(double v) {
    uint64_t u = __builtin_bit_cast(uint64_t, v);
    uint32_t a0 = (uint32_t)u, a1 = (uint32_t)(u >> 32), b0 = a0, b1 = a1;
    asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1\n\tv_permlane32_swap_b32 %2, %3\n\ts_nop 1"
                 : "+v"(a0), "+v"(b0), "+v"(a1), "+v"(b1));
    v = __builtin_bit_cast(double, ((uint64_t)a1 << 32) | a0) + __builtin_bit_cast(double, ((uint64_t)b1 << 32) | b0);
    u = __builtin_bit_cast(uint64_t, v);
    a0 = (uint32_t)u; a1 = (uint32_t)(u >> 32); b0 = a0; b1 = a1;
    asm volatile("s_nop 1\n\tv_permlane16_swap_b32 %0, %1\n\tv_permlane16_swap_b32 %2, %3\n\ts_nop 1"
                 : "+v"(a0), "+v"(b0), "+v"(a1), "+v"(b1));
    v = __builtin_bit_cast(double, ((uint64_t)a1 << 32) | a0) + __builtin_bit_cast(double, ((uint64_t)b1 << 32) | b0);
    auto ror = [](double x, auto ctrl_c) {
        constexpr int CTRL = decltype(ctrl_c)::value;
        const uint64_t w = __builtin_bit_cast(uint64_t, x);
        const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)w, CTRL, 0xF, 0xF, false);
        const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(w >> 32), CTRL, 0xF, 0xF, false);
        return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
    };
    v = v + ror(v, std::integral_constant<int, 0x128>());   // row_ror:8
    v = v + ror(v, std::integral_constant<int, 0x124>());   // row_ror:4
    v = v + ror(v, std::integral_constant<int, 0x122>());   // row_ror:2
    v = v + ror(v, std::integral_constant<int, 0x121>());   // row_ror:1
    return v;
}

__device__ inline int lane_id() { return (int)(threadIdx.x & 63); }

// Token order of the transposed value tensor inside each block of 32 keys: bits 2 and 3
// of the key index are swapped, which is the order in which one lane of a 32x32 MFMA
// consumes the softmax probabilities it holds (keys 8g + 4h + i for its half h), so the
// eight value entries a lane needs are contiguous.  The permutation is its own inverse.
__host__ __device__ inline int vt_perm(int t) {
    return (t & ~12) | ((t & 4) << 1) | ((t & 8) >> 1);
}
__host__ __device__ inline int vt_pad(int T) { return (T + 31) / 32 * 32; }

}  // namespace jab
