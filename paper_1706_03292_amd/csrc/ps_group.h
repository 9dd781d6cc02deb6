// The per-group update of the parameter-server apply (Sec. 2.1 "Parameter
// Server"; Sec. 4.1 "KV Store"), shared by every kernel that applies dense
// updates: the single-tensor, batched and KV-store launches.
//
//   s_i = sum_{p<P} G_p[i]   (p increasing, fp32)
//   buf_i = fma(mu, buf_i, s_i);  W_i = fma(-lr, buf_i, W_i)
//
// A thread owns one group of four consecutive elements and issues its shard
// loads (up to PS_CHUNK at a time) before the dependent adds; 16-byte
// accesses, aligned (AL) or at 4-byte alignment, all non-temporal (each array
// is touched once).
#pragma once

#include "common.h"

namespace poseidon {

// Shard loads in flight per step when P is a run-time value, and when a
// compile-time P is larger than this: with all 32 shard loads of P = 32 in
// flight a thread holds 128 VGPRs of them; eight at a time (behind a
// scheduling barrier, so that the compiler cannot hoist them all) the
// Inception-shaped step's batched pass runs at 5.60 instead of 5.47 TB/s and
// the P = 16 launches are unchanged (5.84 TB/s).
constexpr int PS_CHUNK = 8;

typedef float f4u __attribute__((ext_vector_type(4), aligned(4)));   // 16 bytes at a 4-byte boundary

__device__ inline f4 fma4(float a, f4 b, f4 c)
{
    return f4{fmaf(a, b.x, c.x), fmaf(a, b.y, c.y), fmaf(a, b.z, c.z), fmaf(a, b.w, c.w)};
}

template <bool AL>
__device__ inline f4 ld4(const float* p)
{
    if constexpr (AL)
        return __builtin_nontemporal_load(reinterpret_cast<const f4*>(p));
    else
        return __builtin_nontemporal_load(reinterpret_cast<const f4u*>(p));
}

template <bool AL>
__device__ inline void st4(float* p, f4 v)
{
    if constexpr (AL)
        __builtin_nontemporal_store(v, reinterpret_cast<f4*>(p));
    else
        __builtin_nontemporal_store(v, reinterpret_cast<f4u*>(p));
}

// Where worker p's values of a tensor start: P contiguous shards ...
struct Contiguous {
    const float* G;
    int64_t n;
    __device__ const float* operator()(int p) const { return G + static_cast<int64_t>(p) * n; }
};

// ... or one pointer per worker (the KV store): a whole-tensor update, or a
// message whose values for this range sit `delta` elements further on (bit p
// of msg_mask set).
struct PerWorker {
    const float* const* g;
    uint64_t msg_mask;
    int64_t delta;
    __device__ const float* operator()(int p) const { return g[p] + (((msg_mask >> p) & 1) ? delta : 0); }
};

// Sum of the P values of elements e .. e+3, in increasing p.
template <int PT, bool AL, class Src>
__device__ inline f4 sum4(const Src& src, int P, int64_t e)
{
    if constexpr (PT > PS_CHUNK) {
        f4 s = ld4<AL>(src(0) + e);
#pragma unroll
        for (int p0 = 1; p0 < PT; p0 += PS_CHUNK) {
            f4 g[PS_CHUNK];
#pragma unroll
            for (int c = 0; c < PS_CHUNK; ++c)
                if (p0 + c < PT)
                    g[c] = ld4<AL>(src(p0 + c) + e);
#pragma unroll
            for (int c = 0; c < PS_CHUNK; ++c)
                if (p0 + c < PT)
                    s += g[c];
            __builtin_amdgcn_sched_barrier(0);
        }
        return s;
    } else if constexpr (PT > 0) {
        f4 g[PT];
#pragma unroll
        for (int p = 0; p < PT; ++p)
            g[p] = ld4<AL>(src(p) + e);
        f4 s = g[0];
#pragma unroll
        for (int p = 1; p < PT; ++p)
            s += g[p];
        return s;
    } else {
        f4 s = ld4<AL>(src(0) + e);
        int p = 1;
        for (; p + PS_CHUNK <= P; p += PS_CHUNK) {
            f4 g[PS_CHUNK];
#pragma unroll
            for (int c = 0; c < PS_CHUNK; ++c)
                g[c] = ld4<AL>(src(p + c) + e);
#pragma unroll
            for (int c = 0; c < PS_CHUNK; ++c)
                s += g[c];
        }
        for (; p < P; ++p)
            s += ld4<AL>(src(p) + e);
        return s;
    }
}

// The update of elements e .. min(e + 4, end) - 1 of one tensor.
template <int PT, bool MOM, bool AL, class Src>
__device__ inline void apply_group(float* __restrict__ W, float* __restrict__ buf, const Src& src, int P, int64_t e,
                                   int64_t end, float lr, float mu)
{
    if (e + 3 < end) {
        const f4 s = sum4<PT, AL>(src, P, e);
        f4 w = ld4<AL>(W + e);
        if constexpr (MOM) {
            const f4 b = fma4(mu, ld4<AL>(buf + e), s);
            st4<AL>(buf + e, b);
            w = fma4(-lr, b, w);
        } else {
            w = fma4(-lr, s, w);
        }
        st4<AL>(W + e, w);
    } else {
        for (int64_t k = e; k < end; ++k) {
            float s = src(0)[k];
            for (int p = 1; p < (PT > 0 ? PT : P); ++p)
                s += src(p)[k];
            float w = W[k];
            if constexpr (MOM) {
                const float b = fmaf(mu, buf[k], s);
                buf[k] = b;
                w = fmaf(-lr, b, w);
            } else {
                w = fmaf(-lr, s, w);
            }
            W[k] = w;
        }
    }
}

// Two groups of one tensor, e and e + PS_PAIR_GAP (64 lanes' groups apart, so
// that a wave's two accesses to each array read 2 KB in a row instead of
// 1 KB; the single-tensor launch): when both are whole and P is a
// compile-time value, their loads are issued together, PS_PAIR_CHUNK shards
// at a time; otherwise the two groups are applied one after the other.  Per element the arithmetic and its order
// are apply_group's, so the results are the same, bitwise.  Single-tensor
// launches of 2,621,440 values at P = 32 ran at 5.97-6.03 TB/s against
// 5.49 with one group per thread, 4,194,304 values at P = 8 at 5.43-5.57
// against 4.85-4.90, and 2,359,296 values at P = 16 measured the same
// (5.45-5.54 against 5.46-5.62).
constexpr int64_t PS_PAIR_GAP = 256;
constexpr int PS_PAIR_CHUNK = 4;

template <int PT, bool MOM, bool AL, class Src>
__device__ inline void apply_pair(float* __restrict__ W, float* __restrict__ buf, const Src& src, int P, int64_t e,
                                  int64_t end, float lr, float mu)
{
    const int64_t e1 = e + PS_PAIR_GAP;
    if constexpr (PT > 0) {
        if (e1 + 3 < end) {
            f4 s0 = ld4<AL>(src(0) + e), s1 = ld4<AL>(src(0) + e1);
#pragma unroll
            for (int p0 = 1; p0 < PT; p0 += PS_PAIR_CHUNK) {
                f4 a[PS_PAIR_CHUNK], b[PS_PAIR_CHUNK];
#pragma unroll
                for (int c = 0; c < PS_PAIR_CHUNK; ++c)
                    if (p0 + c < PT) {
                        a[c] = ld4<AL>(src(p0 + c) + e);
                        b[c] = ld4<AL>(src(p0 + c) + e1);
                    }
#pragma unroll
                for (int c = 0; c < PS_PAIR_CHUNK; ++c)
                    if (p0 + c < PT) {
                        s0 += a[c];
                        s1 += b[c];
                    }
                // one chunk of both groups in registers at a time
                __builtin_amdgcn_sched_barrier(0);
            }
            f4 w0 = ld4<AL>(W + e), w1 = ld4<AL>(W + e1);
            if constexpr (MOM) {
                const f4 b0 = fma4(mu, ld4<AL>(buf + e), s0);
                const f4 b1 = fma4(mu, ld4<AL>(buf + e1), s1);
                st4<AL>(buf + e, b0);
                st4<AL>(buf + e1, b1);
                w0 = fma4(-lr, b0, w0);
                w1 = fma4(-lr, b1, w1);
            } else {
                w0 = fma4(-lr, s0, w0);
                w1 = fma4(-lr, s1, w1);
            }
            st4<AL>(W + e, w0);
            st4<AL>(W + e1, w1);
            return;
        }
    }
    apply_group<PT, MOM, AL>(W, buf, src, P, e, end, lr, mu);
    if (e1 < end)
        apply_group<PT, MOM, AL>(W, buf, src, P, e1, end, lr, mu);
}

}  // namespace poseidon
