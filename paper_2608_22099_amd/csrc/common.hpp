// Shared host/device helpers of libbandlu (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "bandlu.h"

namespace bandlu {

// Record a failure text for band_last_error() (thread-local).
void set_error(const char *fmt, ...);
// Record a HIP failure and return BANDLU_ERR_HIP.
int hip_fail(hipError_t e, const char *what);
// Forget the last error (called on entry of every API function).
void clear_error();

inline hipStream_t as_stream(void *s) { return reinterpret_cast<hipStream_t>(s); }

// Check the launch that was just enqueued.
#define BANDLU_CHECK_LAUNCH(what)                                        \
    do {                                                                 \
        hipError_t e_ = hipGetLastError();                               \
        if (e_ != hipSuccess) return ::bandlu::hip_fail(e_, what);       \
    } while (0)

#define BANDLU_ARG(cond, k, ...)                                         \
    do {                                                                 \
        if (!(cond)) {                                                   \
            ::bandlu::set_error(__VA_ARGS__);                            \
            return -(k);                                                 \
        }                                                                \
    } while (0)

constexpr int64_t kMaxN = (int64_t(1) << 31) - 1;

// Number of workgroups that keeps every CU busy with a few resident groups.
int device_cu_count();

// ---------------------------------------------------------------- device --
// Wave-wide max for 64-lane wavefronts (gfx9 wave64), uniform result: DPP
// moves inside rows of 16 lanes (no LDS round trips), then the four row maxima
// combined through scalar registers.
__device__ inline int wave_max_i32(int v) {
    v = max(v, __builtin_amdgcn_mov_dpp(v, 0xB1, 0xf, 0xf, false));   // quad_perm [1,0,3,2]
    v = max(v, __builtin_amdgcn_mov_dpp(v, 0x4E, 0xf, 0xf, false));   // quad_perm [2,3,0,1]
    v = max(v, __builtin_amdgcn_mov_dpp(v, 0x141, 0xf, 0xf, false));  // row_half_mirror
    v = max(v, __builtin_amdgcn_mov_dpp(v, 0x140, 0xf, 0xf, false));  // row_mirror
    const int a = max(__builtin_amdgcn_readlane(v, 0), __builtin_amdgcn_readlane(v, 16));
    const int b = max(__builtin_amdgcn_readlane(v, 32), __builtin_amdgcn_readlane(v, 48));
    return max(a, b);
}

}  // namespace bandlu
