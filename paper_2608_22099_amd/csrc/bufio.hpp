// Raw buffer loads/stores with the hardware range check of CDNA buffer
// resources: a load whose byte offset lies outside the buffer returns 0 and a
// store there is dropped.  Step loops use this instead of branching around
// memory operations, so they stay straight-line code and the compiler can keep
// a deep prefetch ring in flight (a memory operation under a branch makes it
// wait for every outstanding load at the join).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace bandlu {

// Offset that is outside every buffer this library builds (all are < 2 GiB).
constexpr uint32_t kOutside = 0x80000000u;
// Largest buffer, in bytes, for which kOutside is out of range.
constexpr int64_t kMaxBufferBytes = int64_t(0x7fffffff);

struct Buf {
    __amdgpu_buffer_rsrc_t r;
};

// word 3 of a gfx9-family raw buffer resource (dword access, no swizzle)
constexpr int kRsrcWord3 = 0x00020000;

__device__ __forceinline__ Buf make_buf(const void *base, uint32_t bytes) {
    return Buf{__builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes,
                                                 kRsrcWord3)};
}

__device__ __forceinline__ double buf_ld(Buf b, uint32_t byte_off) {
    return __builtin_bit_cast(double, __builtin_amdgcn_raw_buffer_load_b64(b.r, byte_off, 0, 0));
}

__device__ __forceinline__ void buf_st(Buf b, uint32_t byte_off, double v) {
    __builtin_amdgcn_raw_buffer_store_b64(
        __builtin_bit_cast(decltype(__builtin_amdgcn_raw_buffer_load_b64(b.r, 0, 0, 0)), v), b.r,
        byte_off, 0, 0);
}

// The same with a wave-uniform part of the offset in a scalar register.
__device__ __forceinline__ double buf_ld_so(Buf b, uint32_t voff, uint32_t soff) {
    return __builtin_bit_cast(double, __builtin_amdgcn_raw_buffer_load_b64(b.r, voff, soff, 0));
}

__device__ __forceinline__ void buf_st_so(Buf b, uint32_t voff, uint32_t soff, double v) {
    __builtin_amdgcn_raw_buffer_store_b64(
        __builtin_bit_cast(decltype(__builtin_amdgcn_raw_buffer_load_b64(b.r, 0, 0, 0)), v), b.r,
        voff, soff, 0);
}

__device__ __forceinline__ int buf_ld_i32(Buf b, uint32_t byte_off) {
    return (int)__builtin_amdgcn_raw_buffer_load_b32(b.r, byte_off, 0, 0);
}

__device__ __forceinline__ void buf_st_i32(Buf b, uint32_t byte_off, int v) {
    __builtin_amdgcn_raw_buffer_store_b32((unsigned)v, b.r, byte_off, 0, 0);
}

// A copy into a vector register of its own.  A value that moves from a
// prefetch register into a window slot is otherwise renamed, not copied: the
// ring's registers then rotate through the slots, and a loop's back edge
// needs copies of registers whose loads are still in flight (a wait for the
// newest load of the block).  It also keeps a wave-uniform value out of the
// scalar registers.
__device__ __forceinline__ double own_copy(double x) {
    double y;
    asm("v_mov_b64 %0, %1" : "=&v"(y) : "v"(x));
    return y;
}

__device__ __forceinline__ double readlane_d(double v, int lane) {
    const long long x = __double_as_longlong(v);
    const int lo = __builtin_amdgcn_readlane((int)(x & 0xffffffffll), lane);
    const int hi = __builtin_amdgcn_readlane((int)(x >> 32), lane);
    return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
}

}  // namespace bandlu
