// lds_pipe.h -- building blocks of the global -> LDS pipelines of the matrix-core
// kernels (GEMM, attention forward and backward): direct-to-LDS loads, raw barriers,
// hand-placed waits on the vector-memory and LDS counters, transposed LDS reads, and
// the half-wave exchange of v_permlane32_swap.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace jab {
namespace {

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) unsigned char lds_u8;

// 16 bytes per lane from global memory straight into LDS: lane i of the wave writes
// bytes [16 i, 16 i + 16) after the wave-uniform LDS address `dst`.
__device__ inline void lds_dma16(const void *src, unsigned char *dst) {
    __builtin_amdgcn_global_load_lds(src, (lds_void *)dst, 16, 0, 0);
}
// the same with the non-temporal hint, for data read once
__device__ inline void lds_dma16_nt(const void *src, unsigned char *dst) {
    __builtin_amdgcn_global_load_lds(src, (lds_void *)dst, 16, 0, 2);
}
// 4 bytes per lane: lane i writes bytes [4 i, 4 i + 4) after `dst`.
__device__ inline void lds_dma4(const void *src, unsigned char *dst) {
    __builtin_amdgcn_global_load_lds(src, (lds_void *)dst, 4, 0, 0);
}

// The same transfer in the MUBUF form (buffer_load_dwordx4 ... lds): a wave-uniform buffer
// resource and byte offset (scalar registers) plus a per-lane byte offset.  Unlike the FLAT form
// above, it leaves the LDS counter ordered, so waits on fragment reads stay exact while such
// loads are in flight, and a k or key advance is one scalar add.
typedef int i32x4 __attribute__((ext_vector_type(4)));
__device__ void raw_buffer_load_lds(i32x4 rsrc, __attribute__((address_space(3))) uint32_t *lds, int size,
                                    int voffset, int soffset, int offset, int aux) __asm("llvm.amdgcn.raw.buffer.load.lds");
// resource of a raw byte range starting at `base` (wave-uniform): stride 0, 32-bit offsets, no
// range limit; the third word selects the plain buffer format
__device__ inline i32x4 buffer_rsrc(const void *base) {
    const uint64_t a = (uint64_t)base;
    i32x4 r;
    r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
    r[1] = __builtin_amdgcn_readfirstlane((int)(uint32_t)(a >> 32));
    r[2] = -1;
    r[3] = 0x00020000;
    return r;
}
// 16 bytes per lane from byte offset voff + soff of the resource: lane i writes bytes
// [16 i, 16 i + 16) after the wave-uniform LDS address dst
__device__ inline void buffer_dma16(i32x4 rsrc, uint32_t voff, int soff, unsigned char *dst) {
    raw_buffer_load_lds(rsrc, (__attribute__((address_space(3))) uint32_t *)dst, 16, (int)voff, soff, 0, 0);
}

// 16 bytes per lane to byte offset voff + soff of the resource (a vector-memory store: the data
// comes from the lane's registers, the address from the wave-uniform resource plus the lane's offset)
__device__ void raw_buffer_store_v4(i32x4 vdata, i32x4 rsrc, int voffset, int soffset, int aux) __asm("llvm.amdgcn.raw.buffer.store.v4i32");
__device__ inline void buffer_store16(i32x4 rsrc, uint32_t voff, int soff, i32x4 data) {
    raw_buffer_store_v4(data, rsrc, (int)voff, soff, 0);
}
// the same with the non-temporal hint (cache-policy bit 1), for data that is not read again soon
__device__ inline void buffer_store16_nt(i32x4 rsrc, uint32_t voff, int soff, i32x4 data) {
    raw_buffer_store_v4(data, rsrc, (int)voff, soff, 2);
}

__device__ inline void raw_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// vmcnt-only wait (expcnt and lgkmcnt left at their maxima): gfx9 s_waitcnt encoding
template <int N>
__device__ inline void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}
// wait until at most k groups of STEP vector-memory instructions are outstanding (k uniform,
// 0 <= k; values above MAXK wait for MAXK groups)
template <int STEP, int MAXK>
__device__ inline void wait_vm_groups(int k) {
    if constexpr (MAXK > 0) {
        if (k >= MAXK) { wait_vmcnt<MAXK * STEP>(); return; }
        wait_vm_groups<STEP, MAXK - 1>(k);
    } else {
        wait_vmcnt<0>();
    }
}
// lgkmcnt-only wait for all outstanding LDS operations (vmcnt, expcnt at their maxima)
__device__ inline void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14)); }

// Transposed LDS read of 16-bit elements (ds_read_b64_tr_b16).  Every lane names 8 bytes
// (4 elements); within each group of 16 lanes, lane i receives element i % 4 of the 8
// bytes named by lanes i / 4, i / 4 + 4, i / 4 + 8 and i / 4 + 12, in that order.  So if
// lane a + 4 s of a group names columns c0 + 4 a .. c0 + 4 a + 3 of row r0 + s of a
// row-major tile, lane i receives column c0 + i of rows r0 .. r0 + 3.
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
__device__ inline s16x4 lds_read_tr16(const lds_u8 *p) {
    typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)p);
}

// Every lane receives f(own value, value of lane l ^ 32): v_permlane32_swap exchanges
// the upper half of one register with the lower half of another, so two copies of v
// come back as (lower half, lower half) and (upper half, upper half).  Written as
// inline assembly because the compiler folds the builtin's two results into one when
// both inputs are the same value.
__device__ inline float halves_max(float v) {
    float a = v, b = v;
    asm("s_nop 1\n\tv_permlane32_swap_b32 %0, %1\n\ts_nop 1" : "+v"(a), "+v"(b));
    return fmaxf(a, b);
}
__device__ inline float halves_sum(float v) {
    float a = v, b = v;
    asm("s_nop 1\n\tv_permlane32_swap_b32 %0, %1\n\ts_nop 1" : "+v"(a), "+v"(b));
    return a + b;
}

}  // namespace
}  // namespace jab
