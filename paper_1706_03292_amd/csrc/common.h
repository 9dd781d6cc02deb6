// Internal helpers shared by the HIP sources of libposeidon.so.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "poseidon.h"

namespace poseidon {

// Native 4-wide vector (lowers to dwordx4 loads/stores).
typedef float f4 __attribute__((ext_vector_type(4)));

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// True when the byte ranges [a, a+abytes) and [b, b+bbytes) overlap.
inline bool overlaps(const void* a, int64_t abytes, const void* b, int64_t bbytes)
{
    if (!a || !b || abytes <= 0 || bbytes <= 0) return false;
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
    return a0 < b0 + static_cast<uintptr_t>(bbytes) && b0 < a0 + static_cast<uintptr_t>(abytes);
}

// Number of compute units of the current device (cached per device).
int device_cu_count();

// Internal launchers (arguments already validated; nonzero sizes).
hipError_t launch_sf_apply(float* W, const float* U, const float* V,
                           int64_t M, int64_t N, int64_t K, float lr, hipStream_t stream);
hipError_t launch_ps_apply(float* W, const float* shards, int32_t P, int64_t n,
                           float lr, float momentum, float* buf, hipStream_t stream);

// One dense tensor of a batched PS apply (same layout as poseidon_ps_tensor).
struct PsTensor {
    float* W;
    const float* shards;
    float* buf;
    int64_t n;
};
constexpr int PS_BATCH_MAX = 48;   // descriptors per batched launch (kernel-argument space)

// Every tensor with n > 0 in one or a few launches (arguments validated).
// max_grid > 0 caps the workgroups of each launch (they then loop over the
// work), so that the pass can run next to a compute-bound kernel.
hipError_t launch_ps_apply_batch(const PsTensor* tensors, int32_t count, int32_t P, float lr,
                                 float momentum, hipStream_t stream, int max_grid);

// Tuning knobs: workgroups per CU of the sync iteration's batched PS pass while
// the SF reconstructions run (0 = one workgroup per 4096 elements, no cap),
// whether the PS pass is issued before the SF launches, and the SF kernel's
// waves per SIMD.  Measured on the VGG19-22K iteration, caps of 1-4 per CU,
// either order and 3 or 4 waves per SIMD all land within 2.04-2.12 ms.
#ifndef POSEIDON_PS_OVERLAP_WG_PER_CU
#define POSEIDON_PS_OVERLAP_WG_PER_CU 0
#endif
#ifndef POSEIDON_PS_ISSUE_FIRST
#define POSEIDON_PS_ISSUE_FIRST 1
#endif
#ifndef POSEIDON_SF_WAVES_PER_SIMD
#define POSEIDON_SF_WAVES_PER_SIMD 4
#endif

// Argument checks of the public entry points (no device work).
int check_sf_args(const float* W, const float* U, const float* V,
                  int64_t M, int64_t N, int64_t K);
int check_ps_args(const float* W, const float* shards, int32_t P, int64_t n,
                  float momentum, const float* buf);

}  // namespace poseidon
