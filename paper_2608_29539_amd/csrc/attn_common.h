// attn_common.h -- device helpers shared by the attention kernels (forward
// and backward): vector types, lane-pair reductions, raw buffer descriptors,
// global -> LDS loads, the LDS transpose read and bf16 packing.  gfx950 only.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace logo {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

constexpr float kNegInf = -__builtin_inff();

// Value of the partner lane (l ^ 32) and own value, combined.
__device__ __forceinline__ float pair_max(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Wave-uniform value, made explicit so the compiler keeps it in SGPRs.
__device__ __forceinline__ int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }

// Buffer resource word 3 for raw (untyped, stride 0) buffer loads.
constexpr int kRawBufferFlags = 0x00020000;

// Raw buffer descriptor over nbytes (>= 0) bytes from p: loads at or past
// nbytes return zeros.  Words: base address (48 bits, stride 0), size, flags.
__device__ __forceinline__ u32x4 raw_rsrc(const void *p, int nbytes) {
    const uint64_t a = (uint64_t)p;
    u32x4 r;
    r[0] = __builtin_amdgcn_readfirstlane((uint32_t)a);
    r[1] = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32)) & 0xFFFFu;
    r[2] = __builtin_amdgcn_readfirstlane(nbytes);
    r[3] = kRawBufferFlags;
    return r;
}

// One 16-byte-per-lane global -> LDS load (buffer_load_dwordx4 ... lds: lane
// i writes the 16 bytes at lds + 16 i).  Issued as inline assembly so that
// the compiler does not make every later LDS read wait for it: the buffer it
// fills is only read after the wait + barrier that ends the pipeline step.
// M0 (the LDS base of the load) is saved and restored around it.
__device__ __forceinline__ void lds_load16(u32x4 r, const void *lds, int voffset) {
    const uint32_t lds_addr = __builtin_amdgcn_readfirstlane(
        (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)lds);
    uint32_t saved;
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %1\n\t"
        "s_nop 0\n\t"
        "buffer_load_dwordx4 %2, %3, 0 offen lds\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "s"(lds_addr), "v"(voffset), "s"(r)
        : "memory");
}

// s_waitcnt operand that waits for vmcnt = 0 only (lgkmcnt and expcnt at
// their maximum).  Issued through the builtin so the compiler knows that no
// vector-memory load is outstanding afterwards.
constexpr int kWaitVmcnt0 = 0x0F70;

// Completion of this wave's LDS-bound loads, then the workgroup barrier.
__device__ __forceinline__ void dma_wait_barrier() {
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    __syncthreads();
}

// gfx950 LDS transpose read of two 8-byte addresses (8 rows apart in the
// callers' layouts): within each 16-lane group, lane 4b+e receives element e
// of the 4-element rows addressed by lanes b, b+4, b+8, b+12.
__device__ __forceinline__ bf16x8 lds_tr_pair(const void *a0, const void *a1) {
    const s16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)a0);
    const s16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)a1);
    const s16x4 ab[2] = {a, b};
    return __builtin_bit_cast(bf16x8, ab);
}

// Two fp32 -> two bf16 (round to nearest even) in one v_cvt_pk_bf16_f32.
__device__ __forceinline__ bf16x2 cvt_bf16x2(float a, float b) {
    return __builtin_convertvector(f32x2{a, b}, bf16x2);
}
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
    return __builtin_bit_cast(uint32_t, cvt_bf16x2(a, b));
}

}  // namespace
}  // namespace logo
