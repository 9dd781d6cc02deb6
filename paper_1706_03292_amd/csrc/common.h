// Internal helpers shared by the HIP sources of libposeidon.so.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <vector>

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

// A byte range [lo, hi) that a call reads or writes.
struct Span {
    uintptr_t lo;
    uintptr_t hi;
};

inline void add_span(std::vector<Span>& v, const void* p, int64_t bytes)
{
    if (p && bytes > 0)
        v.push_back(Span{reinterpret_cast<uintptr_t>(p), reinterpret_cast<uintptr_t>(p) + static_cast<uintptr_t>(bytes)});
}

// True when two written ranges overlap, or a read range overlaps a written
// one.  Read ranges may overlap each other (several tensors may share an
// input).  Sorting the written ranges makes it O((w + r) log w).
inline bool writes_collide(std::vector<Span> writes, const std::vector<Span>& reads)
{
    std::sort(writes.begin(), writes.end(), [](const Span& a, const Span& b) { return a.lo < b.lo; });
    for (size_t i = 1; i < writes.size(); ++i)
        if (writes[i].lo < writes[i - 1].hi)
            return true;
    // The written ranges are now disjoint and sorted, so their ends are
    // sorted too: a read range meets one iff it meets the last one that
    // starts before the read range ends.
    for (const Span& r : reads) {
        auto it = std::lower_bound(writes.begin(), writes.end(), r.hi,
                                   [](const Span& w, uintptr_t hi) { return w.lo < hi; });
        if (it != writes.begin() && std::prev(it)->hi > r.lo)
            return true;
    }
    return false;
}

// Number of compute units of the current device (cached per device).
int device_cu_count();

// The SF contraction's arithmetic (POSEIDON_SF_BF16X6 or POSEIDON_SF_FP32),
// process-wide.
int32_t sf_arithmetic();
void set_sf_arithmetic(int32_t arithmetic);

// The time the iteration's stream policy assumes for one layer's rebuild,
// from the rates measured alone on one MI355X (fp32-equivalent contraction
// flops): split-bf16 products on 256 x 128 tiles 186-194 TFLOP/s (the
// grouped VGG19-22K FC launch), on smaller tiles about 140 (the 4096 x 4096
// layer at K = 256: 142); fp32 products 124-138.
constexpr double SF_SPLIT_BIG_FLOPS_PER_S = 1.85e14;
constexpr double SF_SPLIT_FLOPS_PER_S = 1.4e14;
constexpr double SF_FP32_FLOPS_PER_S = 1.3e14;
double sf_seconds(int64_t M, int64_t N, int64_t K);

// Internal launchers (arguments already validated; nonzero sizes).  Given
// spread_s > 0, an SF launch runs on as few workgroups as would walk its
// tiles in about spread_s seconds, instead of one workgroup per tile.  Given
// `room`, the SF tiles leave each SIMD the registers of a wave of the lean PS
// kernel beside theirs, and a PS launch given `beside_sf` uses that kernel
// (aligned tensors), so that the two run on the same CUs.
hipError_t launch_sf_apply(float* W, const float* U, const float* V,
                           int64_t M, int64_t N, int64_t K, float lr, hipStream_t stream, double spread_s = 0.0,
                           bool room = false);
hipError_t launch_ps_apply(float* W, const float* shards, int32_t P, int64_t n,
                           float lr, float momentum, float* buf, hipStream_t stream, bool beside_sf = false);
hipError_t launch_sf_apply_momentum(float* W, float* buf, const float* U, const float* V, int64_t M,
                                    int64_t N, int64_t K, float lr, float mu, hipStream_t stream,
                                    double spread_s = 0.0);

// One FC layer of a grouped SF launch (same layout as poseidon_sf_tensor).
struct SfTensor {
    float* W;
    const float* U;
    const float* V;
    int64_t M;
    int64_t N;
};
constexpr int SF_BATCH_MAX = 16;   // layers per grouped launch (kernel-argument space)

// Every layer with work, grouped into as few launches as possible (validated).
hipError_t launch_sf_apply_batch(const SfTensor* layers, int32_t count, int64_t K, float lr,
                                 hipStream_t stream, bool room = false);

// One dense tensor of a batched PS apply (same layout as poseidon_ps_tensor).
struct PsTensor {
    float* W;
    const float* shards;
    float* buf;
    int64_t n;
};
constexpr int PS_BATCH_MAX = 48;   // descriptors per batched launch (kernel-argument space)

// Every tensor with n > 0 in one or a few launches (arguments validated).
hipError_t launch_ps_apply_batch(const PsTensor* tensors, int32_t count, int32_t P, float lr,
                                 float momentum, hipStream_t stream);

// KV-store apply of pairs held by one server (arguments validated; P <=
// KV_MAX_P; every range inside its tensor; the tensors do not overlap).
// grads[p] is worker p's update, the same for every range: a whole-tensor
// update, or (bit p of msg_mask) its message, whose values of a range sit
// `delta` elements past the tensor's indices.  Ranges with a buf and ranges
// without take separate launches, and beyond KV_MAX_RANGES further ones.
constexpr int KV_MAX_P = 64;
constexpr int KV_MAX_RANGES = 32;
struct KvApplyRange {
    float* W;
    float* buf;       // momentum buffer, or NULL (plain SGD)
    int64_t offset;
    int64_t length;
    int64_t delta;
};
hipError_t launch_kv_apply(const KvApplyRange* ranges, int32_t nranges, const float* const* grads,
                           uint64_t msg_mask, int32_t P, float lr, float momentum, hipStream_t stream);

// A worker's message to one server: src[i][0 .. length[i]) copied to
// message[dst[i] ..), in KV_PACK_MAX ranges per launch (arguments validated).
constexpr int KV_PACK_MAX = 64;
hipError_t launch_kv_pack(const float* const* src, const int64_t* dst, const int64_t* length, int32_t count,
                          float* message, hipStream_t stream);

// Argument checks of the public entry points (no device work).
int check_sf_args(const float* W, const float* U, const float* V,
                  int64_t M, int64_t N, int64_t K);
int check_sf_momentum_args(const float* W, const float* buf, const float* U, const float* V,
                           int64_t M, int64_t N, int64_t K);
int check_ps_args(const float* W, const float* shards, int32_t P, int64_t n,
                  float momentum, const float* buf);

}  // namespace poseidon
