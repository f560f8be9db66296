// Wavefront and workgroup primitives shared by the multi-wave LU kernels
// (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>

#include "bufio.hpp"

namespace bandlu {

// DPP lane move of a double: both 32-bit halves moved with the same control.
template <int CTRL>
__device__ __forceinline__ double dpp_d(double v) {
    const long long x = __double_as_longlong(v);
    const int lo = __builtin_amdgcn_mov_dpp((int)(x & 0xffffffffll), CTRL, 0xf, 0xf, false);
    const int hi = __builtin_amdgcn_mov_dpp((int)(x >> 32), CTRL, 0xf, 0xf, false);
    return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
}

// Maximum of a NaN-free double over the 64 lanes, returned uniform: DPP moves
// inside each row of 16 lanes, then the four row maxima read by readlane.
__device__ __forceinline__ double wave_max_d(double k) {
    k = fmax(k, dpp_d<0xB1>(k));   // quad_perm [1,0,3,2]
    k = fmax(k, dpp_d<0x4E>(k));   // quad_perm [2,3,0,1]
    k = fmax(k, dpp_d<0x141>(k));  // row_half_mirror
    k = fmax(k, dpp_d<0x140>(k));  // row_mirror
    return fmax(fmax(readlane_d(k, 0), readlane_d(k, 16)), fmax(readlane_d(k, 32), readlane_d(k, 48)));
}

// Minimum of an int over the 64 lanes, returned uniform.
__device__ __forceinline__ int wave_min_i32(int v) {
    v = min(v, __builtin_amdgcn_mov_dpp(v, 0xB1, 0xf, 0xf, false));
    v = min(v, __builtin_amdgcn_mov_dpp(v, 0x4E, 0xf, 0xf, false));
    v = min(v, __builtin_amdgcn_mov_dpp(v, 0x141, 0xf, 0xf, false));
    v = min(v, __builtin_amdgcn_mov_dpp(v, 0x140, 0xf, 0xf, false));
    return min(min(__builtin_amdgcn_readlane(v, 0), __builtin_amdgcn_readlane(v, 16)),
               min(__builtin_amdgcn_readlane(v, 32), __builtin_amdgcn_readlane(v, 48)));
}

// Pivot key of candidate t (t = 0 is the diagonal): |x|, with a NaN ranked
// above everything in position 0 and below every number elsewhere, so that the
// (largest key, smallest index) rule is the BLAS i_amax choice.
__device__ __forceinline__ double pivot_key(double x, int t) {
    return __builtin_isnan(x) ? (t == 0 ? __builtin_inf() : -1.0) : fabs(x);
}

__device__ __forceinline__ bool key_better(double ka, int ia, double kb, int ib) {
    return ka > kb || (ka == kb && ia < ib);
}

// Branch-free masked loads.  A load under a branch makes the compiler wait for
// every outstanding load at the join, and a row of selects keeps one SGPR
// mask pair per load alive until its data arrives (the compiler then runs out
// of SGPRs and waits for each load in turn).  Instead the address is clamped
// to p[0], which is always valid, the condition is kept as one bit of a VGPR
// bit field, and the loaded value is cleared afterwards with an integer AND.
__device__ __forceinline__ double ld_clamped(const double *p, int64_t idx, bool ok) {
    return p[ok ? idx : 0];
}

__device__ __forceinline__ double keep_if(double v, unsigned bits, int i) {
    const long long m = -(long long)((bits >> i) & 1u);
    return __longlong_as_double(__double_as_longlong(v) & m);
}

// Load p[idx] if ok, else 0 (for a load whose result is used at once).
__device__ __forceinline__ double ld_or_zero(const double *p, int64_t idx, bool ok) {
    return keep_if(ld_clamped(p, idx, ok), ok ? 1u : 0u, 0);
}

// Workgroup barrier that orders LDS only: outstanding global stores stay in
// flight (__syncthreads would wait for every one of them first).
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

}  // namespace bandlu
