// Parameter-server aggregation + momentum SGD apply (Sec. 2.1 "Parameter
// Server"; Sec. 4.1 "KV Store", "Managing Consistency").
//
//   s_i = sum_{p<P} G[p*n + i]   (p increasing, fp32)
//   buf_i = fma(mu, buf_i, s_i);  W_i = fma(-lr, buf_i, W_i)
//
// The kernel is bound by HBM bandwidth: per element it reads P shard values
// plus W and buf and writes W and buf (4P + 16 bytes), against ~P + 3 flops.
// Each thread owns one 16-byte group of four consecutive elements and issues
// all of its shard loads before the dependent adds (bytes in flight).  Every
// array is touched once per launch (shards read; W and buf read, then
// written), so all accesses are non-temporal (1-2% faster than cached W/buf
// accesses on 2.4M-16.8M elements).  One-wave workgroups, one
// group per thread, as many workgroups as groups: a launch-shape sweep over
// 37K-16.8M elements (block size 64-1024, one or two groups per thread,
// grid-stride loops capped at 4-16 workgroups per CU) found this within 3% of
// the best everywhere and 10% faster than a capped grid-stride loop on large
// tensors, whose last partial pass leaves the chip half idle.  A scalar
// variant covers sizes that are not a multiple of four or arrays that are not
// 16-byte aligned.
#include "common.h"

namespace poseidon {
namespace {

constexpr int PS_THREADS = 64;    // one wave per workgroup (single-tensor and batched launches)
constexpr int PS_THREADS_1 = PS_THREADS;
constexpr int PS_CHUNK = 8;       // shard loads in flight per step when P is a runtime value

__device__ inline f4 fma4(float a, f4 b, f4 c)
{
    return f4{fmaf(a, b.x, c.x), fmaf(a, b.y, c.y), fmaf(a, b.z, c.z), fmaf(a, b.w, c.w)};
}

// Sum of the P shard values at vector index i, in increasing p.
template <int PT>
__device__ inline f4 shard_sum4(const f4* __restrict__ G4, int P, int64_t n4, int64_t i)
{
    if constexpr (PT > 0) {
        f4 g[PT];
#pragma unroll
        for (int p = 0; p < PT; ++p)
            g[p] = __builtin_nontemporal_load(G4 + static_cast<int64_t>(p) * n4 + i);
        f4 s = g[0];
#pragma unroll
        for (int p = 1; p < PT; ++p)
            s += g[p];
        return s;
    } else {
        f4 s = __builtin_nontemporal_load(G4 + i);
        int p = 1;
        for (; p + PS_CHUNK <= P; p += PS_CHUNK) {
            f4 g[PS_CHUNK];
#pragma unroll
            for (int c = 0; c < PS_CHUNK; ++c)
                g[c] = __builtin_nontemporal_load(G4 + static_cast<int64_t>(p + c) * n4 + i);
#pragma unroll
            for (int c = 0; c < PS_CHUNK; ++c)
                s += g[c];
        }
        for (; p < P; ++p)
            s += __builtin_nontemporal_load(G4 + static_cast<int64_t>(p) * n4 + i);
        return s;
    }
}

template <int PT>
__device__ inline float shard_sum1(const float* __restrict__ G, int P, int64_t n, int64_t i)
{
    if constexpr (PT > 0) {
        float g[PT];
#pragma unroll
        for (int p = 0; p < PT; ++p)
            g[p] = __builtin_nontemporal_load(G + static_cast<int64_t>(p) * n + i);
        float s = g[0];
#pragma unroll
        for (int p = 1; p < PT; ++p)
            s += g[p];
        return s;
    } else {
        float s = __builtin_nontemporal_load(G + i);
        int p = 1;
        for (; p + PS_CHUNK <= P; p += PS_CHUNK) {
            float g[PS_CHUNK];
#pragma unroll
            for (int c = 0; c < PS_CHUNK; ++c)
                g[c] = __builtin_nontemporal_load(G + static_cast<int64_t>(p + c) * n + i);
#pragma unroll
            for (int c = 0; c < PS_CHUNK; ++c)
                s += g[c];
        }
        for (; p < P; ++p)
            s += __builtin_nontemporal_load(G + static_cast<int64_t>(p) * n + i);
        return s;
    }
}

template <int PT, bool MOM>
__global__ __launch_bounds__(PS_THREADS_1) void ps_apply_vec4(
    float* __restrict__ W, const float* __restrict__ G, int P, int64_t n4,
    float lr, float mu, float* __restrict__ buf)
{
    const f4* G4 = reinterpret_cast<const f4*>(G);
    f4* W4 = reinterpret_cast<f4*>(W);
    f4* B4 = reinterpret_cast<f4*>(buf);
    const int64_t stride = static_cast<int64_t>(gridDim.x) * PS_THREADS_1;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * PS_THREADS_1 + threadIdx.x; i < n4; i += stride) {
        const f4 s = shard_sum4<PT>(G4, P, n4, i);
        f4 w = __builtin_nontemporal_load(W4 + i);
        if constexpr (MOM) {
            const f4 b = fma4(mu, __builtin_nontemporal_load(B4 + i), s);
            __builtin_nontemporal_store(b, B4 + i);
            w = fma4(-lr, b, w);
        } else {
            w = fma4(-lr, s, w);
        }
        __builtin_nontemporal_store(w, W4 + i);
    }
}

template <int PT, bool MOM>
__global__ __launch_bounds__(PS_THREADS_1) void ps_apply_scalar(
    float* __restrict__ W, const float* __restrict__ G, int P, int64_t n,
    float lr, float mu, float* __restrict__ buf)
{
    const int64_t stride = static_cast<int64_t>(gridDim.x) * PS_THREADS_1;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * PS_THREADS_1 + threadIdx.x; i < n; i += stride) {
        const float s = shard_sum1<PT>(G, P, n, i);
        float w = W[i];
        if constexpr (MOM) {
            const float b = fmaf(mu, buf[i], s);
            buf[i] = b;
            w = fmaf(-lr, b, w);
        } else {
            w = fmaf(-lr, s, w);
        }
        W[i] = w;
    }
}

template <int PT, bool MOM>
hipError_t launch_pt(float* W, const float* G, int32_t P, int64_t n, float lr, float mu,
                     float* buf, bool vec, hipStream_t stream)
{
    const int64_t items = vec ? n / 4 : n;
    // One item per thread; the kernels' grid-stride loop only matters beyond
    // 2^30 workgroups.
    const int64_t want = (items + PS_THREADS_1 - 1) / PS_THREADS_1;
    const int64_t cap = int64_t{1} << 30;
    const int grid = static_cast<int>(want < cap ? want : cap);
    if (vec)
        ps_apply_vec4<PT, MOM><<<grid, PS_THREADS_1, 0, stream>>>(W, G, P, items, lr, mu, buf);
    else
        ps_apply_scalar<PT, MOM><<<grid, PS_THREADS_1, 0, stream>>>(W, G, P, items, lr, mu, buf);
    return hipGetLastError();
}

template <bool MOM>
hipError_t launch_mom(float* W, const float* G, int32_t P, int64_t n, float lr, float mu,
                      float* buf, bool vec, hipStream_t stream)
{
    switch (P) {
    case 1:  return launch_pt<1, MOM>(W, G, P, n, lr, mu, buf, vec, stream);
    case 2:  return launch_pt<2, MOM>(W, G, P, n, lr, mu, buf, vec, stream);
    case 4:  return launch_pt<4, MOM>(W, G, P, n, lr, mu, buf, vec, stream);
    case 8:  return launch_pt<8, MOM>(W, G, P, n, lr, mu, buf, vec, stream);
    case 16: return launch_pt<16, MOM>(W, G, P, n, lr, mu, buf, vec, stream);
    case 32: return launch_pt<32, MOM>(W, G, P, n, lr, mu, buf, vec, stream);
    default: return launch_pt<0, MOM>(W, G, P, n, lr, mu, buf, vec, stream);
    }
}

// ---------------------------------------------------------------------------
// Many tensors in one launch.  The descriptors travel by value in the kernel
// arguments; tensor t owns the workgroups [first_block[t], first_block[t+1]),
// each of which updates PS_BLOCK_ELEMS consecutive elements of it (16-byte
// groups when the tensor allows it, single elements otherwise).
// ---------------------------------------------------------------------------

constexpr int PS_BLOCK_ELEMS = 4 * PS_THREADS;  // elements per work block: one 16-byte group per thread
constexpr int PS_BATCH_MAX_GRID = 1 << 30;     // one workgroup per work block below this

struct PsBatchItem {
    float* W;
    const float* G;
    float* buf;
    int64_t n;
    int32_t first_block;
    int32_t vec;
};

struct PsBatchArgs {
    PsBatchItem item[PS_BATCH_MAX];
    int32_t count;
};

template <int PT, bool MOM>
__global__ __launch_bounds__(PS_THREADS) void ps_apply_batch_kernel(const PsBatchArgs args, int P, float lr,
                                                                    float mu, int total_blocks)
{
    // Workgroup g handles work blocks g, g + gridDim.x, ... (one pass when the
    // grid covers every block); the block's tensor is found by binary search
    // over the descriptors' first blocks (uniform, scalar loads).
    for (int b = blockIdx.x; b < total_blocks; b += gridDim.x) {
        int lo = 0, hi = args.count - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (args.item[mid].first_block <= b)
                lo = mid;
            else
                hi = mid - 1;
        }
        const int t = lo;
        float* __restrict__ W = args.item[t].W;
        const float* __restrict__ G = args.item[t].G;
        float* __restrict__ buf = args.item[t].buf;
        const int64_t n = args.item[t].n;
        const int64_t base = static_cast<int64_t>(b - args.item[t].first_block) * PS_BLOCK_ELEMS;
        if (args.item[t].vec) {
            const int64_t n4 = n >> 2;
            const f4* G4 = reinterpret_cast<const f4*>(G);
            f4* W4 = reinterpret_cast<f4*>(W);
            f4* B4 = reinterpret_cast<f4*>(buf);
#pragma unroll
            for (int u = 0; u < PS_BLOCK_ELEMS / 4 / PS_THREADS; ++u) {
                const int64_t i = (base >> 2) + u * PS_THREADS + threadIdx.x;
                if (i < n4) {
                    const f4 s = shard_sum4<PT>(G4, P, n4, i);
                    f4 w = __builtin_nontemporal_load(W4 + i);
                    if constexpr (MOM) {
                        const f4 bv = fma4(mu, __builtin_nontemporal_load(B4 + i), s);
                        __builtin_nontemporal_store(bv, B4 + i);
                        w = fma4(-lr, bv, w);
                    } else {
                        w = fma4(-lr, s, w);
                    }
                    __builtin_nontemporal_store(w, W4 + i);
                }
            }
        } else {
#pragma unroll 4
            for (int u = 0; u < PS_BLOCK_ELEMS / PS_THREADS; ++u) {
                const int64_t i = base + u * PS_THREADS + threadIdx.x;
                if (i < n) {
                    const float s = shard_sum1<PT>(G, P, n, i);
                    float w = W[i];
                    if constexpr (MOM) {
                        const float bv = fmaf(mu, buf[i], s);
                        buf[i] = bv;
                        w = fmaf(-lr, bv, w);
                    } else {
                        w = fmaf(-lr, s, w);
                    }
                    W[i] = w;
                }
            }
        }
    }
}

template <int PT, bool MOM>
void launch_batch_pt(const PsBatchArgs& a, int blocks, int grid, int32_t P, float lr, float mu, hipStream_t stream)
{
    ps_apply_batch_kernel<PT, MOM><<<grid, PS_THREADS, 0, stream>>>(a, P, lr, mu, blocks);
}

template <bool MOM>
void launch_batch_mom(const PsBatchArgs& a, int blocks, int grid, int32_t P, float lr, float mu,
                      hipStream_t stream)
{
    switch (P) {
    case 1:  launch_batch_pt<1, MOM>(a, blocks, grid, P, lr, mu, stream); break;
    case 2:  launch_batch_pt<2, MOM>(a, blocks, grid, P, lr, mu, stream); break;
    case 4:  launch_batch_pt<4, MOM>(a, blocks, grid, P, lr, mu, stream); break;
    case 8:  launch_batch_pt<8, MOM>(a, blocks, grid, P, lr, mu, stream); break;
    case 16: launch_batch_pt<16, MOM>(a, blocks, grid, P, lr, mu, stream); break;
    case 32: launch_batch_pt<32, MOM>(a, blocks, grid, P, lr, mu, stream); break;
    default: launch_batch_pt<0, MOM>(a, blocks, grid, P, lr, mu, stream); break;
    }
}

// ---------------------------------------------------------------------------
// KV-store apply: the pairs of one tensor that one server holds, with the P
// workers' updates at separate addresses (one pointer per worker, passed in
// worker order).  Range r covers tensor elements [offset, offset + length)
// and owns the workgroups [first_block[r], first_block[r+1]); each workgroup
// updates PS_BLOCK_ELEMS consecutive elements of its range, one group of four
// per thread (16-byte accesses when the whole launch allows them).
// ---------------------------------------------------------------------------

struct KvRange {
    int64_t offset;
    int64_t length;
    int32_t first_block;
    int32_t pad;
};

struct KvArgs {
    const float* g[KV_MAX_P];
    KvRange r[KV_MAX_RANGES];
    int32_t nranges;
};

// Sum of the P updates of the four elements at e, in increasing worker order.
template <int PT>
__device__ inline f4 kv_sum4(const KvArgs& a, int P, int64_t e)
{
    if constexpr (PT > 0) {
        f4 g[PT];
#pragma unroll
        for (int p = 0; p < PT; ++p)
            g[p] = __builtin_nontemporal_load(reinterpret_cast<const f4*>(a.g[p] + e));
        f4 s = g[0];
#pragma unroll
        for (int p = 1; p < PT; ++p)
            s += g[p];
        return s;
    } else {
        f4 s = __builtin_nontemporal_load(reinterpret_cast<const f4*>(a.g[0] + e));
        int p = 1;
        for (; p + PS_CHUNK <= P; p += PS_CHUNK) {
            f4 g[PS_CHUNK];
#pragma unroll
            for (int c = 0; c < PS_CHUNK; ++c)
                g[c] = __builtin_nontemporal_load(reinterpret_cast<const f4*>(a.g[p + c] + e));
#pragma unroll
            for (int c = 0; c < PS_CHUNK; ++c)
                s += g[c];
        }
        for (; p < P; ++p)
            s += __builtin_nontemporal_load(reinterpret_cast<const f4*>(a.g[p] + e));
        return s;
    }
}

template <int PT>
__device__ inline float kv_sum1(const KvArgs& a, int P, int64_t e)
{
    float s = a.g[0][e];
    for (int p = 1; p < (PT > 0 ? PT : P); ++p)
        s += a.g[p][e];
    return s;
}

template <int PT, bool MOM>
__global__ __launch_bounds__(PS_THREADS) void kv_apply_kernel(const KvArgs a, int P, float* __restrict__ W,
                                                               float* __restrict__ buf, float lr, float mu, int vec)
{
    const int b = blockIdx.x;
    int r = 0;
    while (r + 1 < a.nranges && a.r[r + 1].first_block <= b)
        ++r;
    const int64_t len = a.r[r].length;
    const int64_t j = static_cast<int64_t>(b - a.r[r].first_block) * PS_BLOCK_ELEMS + 4 * threadIdx.x;
    if (j >= len)
        return;
    const int64_t e = a.r[r].offset + j;
    if (vec && j + 3 < len) {
        const f4 s = kv_sum4<PT>(a, P, e);
        f4* W4 = reinterpret_cast<f4*>(W + e);
        f4 w = __builtin_nontemporal_load(W4);
        if constexpr (MOM) {
            f4* B4 = reinterpret_cast<f4*>(buf + e);
            const f4 bv = fma4(mu, __builtin_nontemporal_load(B4), s);
            __builtin_nontemporal_store(bv, B4);
            w = fma4(-lr, bv, w);
        } else {
            w = fma4(-lr, s, w);
        }
        __builtin_nontemporal_store(w, W4);
    } else {
        for (int q = 0; q < 4 && j + q < len; ++q) {
            const float s = kv_sum1<PT>(a, P, e + q);
            float w = W[e + q];
            if constexpr (MOM) {
                const float bv = fmaf(mu, buf[e + q], s);
                buf[e + q] = bv;
                w = fmaf(-lr, bv, w);
            } else {
                w = fmaf(-lr, s, w);
            }
            W[e + q] = w;
        }
    }
}

template <bool MOM>
void launch_kv_mom(const KvArgs& a, int grid, int32_t P, float* W, float* buf, float lr, float mu, int vec,
                   hipStream_t stream)
{
    switch (P) {
    case 4:  kv_apply_kernel<4, MOM><<<grid, PS_THREADS, 0, stream>>>(a, P, W, buf, lr, mu, vec); break;
    case 8:  kv_apply_kernel<8, MOM><<<grid, PS_THREADS, 0, stream>>>(a, P, W, buf, lr, mu, vec); break;
    case 16: kv_apply_kernel<16, MOM><<<grid, PS_THREADS, 0, stream>>>(a, P, W, buf, lr, mu, vec); break;
    case 32: kv_apply_kernel<32, MOM><<<grid, PS_THREADS, 0, stream>>>(a, P, W, buf, lr, mu, vec); break;
    default: kv_apply_kernel<0, MOM><<<grid, PS_THREADS, 0, stream>>>(a, P, W, buf, lr, mu, vec); break;
    }
}

}  // namespace

hipError_t launch_ps_apply(float* W, const float* shards, int32_t P, int64_t n,
                           float lr, float momentum, float* buf, hipStream_t stream)
{
    const bool vec = (n % 4 == 0) && aligned16(W) && aligned16(shards) && (!buf || aligned16(buf));
    if (buf)
        return launch_mom<true>(W, shards, P, n, lr, momentum, buf, vec, stream);
    return launch_mom<false>(W, shards, P, n, lr, 0.0f, nullptr, vec, stream);
}

hipError_t launch_ps_apply_batch(const PsTensor* t, int32_t count, int32_t P, float lr, float momentum,
                                 hipStream_t stream)
{
    // Tensors without a momentum buffer and tensors with one are launched
    // separately (the kernel is specialised on it); each launch carries up to
    // PS_BATCH_MAX descriptors.
    for (int pass = 0; pass < 2; ++pass) {
        const bool mom = pass == 1;
        PsBatchArgs a{};
        int64_t blocks = 0;
        auto flush = [&]() -> hipError_t {
            if (a.count == 0)
                return hipSuccess;
            const int nb = static_cast<int>(blocks);
            const int grid = nb < PS_BATCH_MAX_GRID ? nb : PS_BATCH_MAX_GRID;
            if (mom)
                launch_batch_mom<true>(a, nb, grid, P, lr, momentum, stream);
            else
                launch_batch_mom<false>(a, nb, grid, P, lr, 0.0f, stream);
            a = PsBatchArgs{};
            blocks = 0;
            return hipGetLastError();
        };
        for (int32_t i = 0; i < count; ++i) {
            if (t[i].n == 0 || (t[i].buf != nullptr) != mom)
                continue;
            const int64_t nb = (t[i].n + PS_BLOCK_ELEMS - 1) / PS_BLOCK_ELEMS;
            if (a.count == PS_BATCH_MAX || blocks + nb > INT32_MAX) {
                const hipError_t e = flush();
                if (e != hipSuccess)
                    return e;
            }
            PsBatchItem& it = a.item[a.count++];
            it.W = t[i].W;
            it.G = t[i].shards;
            it.buf = t[i].buf;
            it.n = t[i].n;
            it.first_block = static_cast<int32_t>(blocks);
            it.vec = (t[i].n % 4 == 0) && aligned16(t[i].W) && aligned16(t[i].shards) &&
                     (!t[i].buf || aligned16(t[i].buf));
            blocks += nb;
        }
        const hipError_t e = flush();
        if (e != hipSuccess)
            return e;
    }
    return hipSuccess;
}

hipError_t launch_kv_apply(float* W, float* buf, const float* const* grads, int32_t P, const int64_t* offsets,
                           const int64_t* lengths, int32_t nranges, float lr, float momentum, hipStream_t stream)
{
    bool vec = aligned16(W) && (!buf || aligned16(buf));
    for (int32_t p = 0; p < P; ++p)
        vec = vec && aligned16(grads[p]);
    for (int32_t i = 0; i < nranges; ++i)
        vec = vec && offsets[i] % 4 == 0;
    for (int32_t i0 = 0; i0 < nranges; i0 += KV_MAX_RANGES) {
        KvArgs a{};
        for (int32_t p = 0; p < P; ++p)
            a.g[p] = grads[p];
        int64_t blocks = 0;
        for (int32_t i = i0; i < nranges && i < i0 + KV_MAX_RANGES; ++i) {
            KvRange& r = a.r[a.nranges++];
            r.offset = offsets[i];
            r.length = lengths[i];
            r.first_block = static_cast<int32_t>(blocks);
            blocks += (lengths[i] + PS_BLOCK_ELEMS - 1) / PS_BLOCK_ELEMS;
            if (blocks > INT32_MAX)
                return hipErrorInvalidValue;
        }
        if (blocks == 0)
            continue;
        if (buf)
            launch_kv_mom<true>(a, static_cast<int>(blocks), P, W, buf, lr, momentum, vec ? 1 : 0, stream);
        else
            launch_kv_mom<false>(a, static_cast<int>(blocks), P, W, nullptr, lr, 0.0f, vec ? 1 : 0, stream);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess)
            return e;
    }
    return hipSuccess;
}

int check_ps_args(const float* W, const float* shards, int32_t P, int64_t n,
                  float momentum, const float* buf)
{
    if (P < 1 || n < 0)
        return POSEIDON_ERR_INVALID_ARG;
    if (n == 0)
        return POSEIDON_OK;
    if (!W || !shards || (!buf && momentum != 0.0f))
        return POSEIDON_ERR_INVALID_ARG;
    if (n > (INT64_MAX / 4) / P)
        return POSEIDON_ERR_INVALID_ARG;
    const int64_t wb = n * 4, gb = n * 4 * static_cast<int64_t>(P);
    if (overlaps(W, wb, shards, gb) || overlaps(buf, wb, shards, gb) || overlaps(W, wb, buf, wb))
        return POSEIDON_ERR_INVALID_ARG;
    return POSEIDON_OK;
}

}  // namespace poseidon

extern "C" int poseidon_ps_apply(float* W, const float* shards, int32_t P, int64_t n,
                                 float lr, float momentum, float* buf, hipStream_t stream)
{
    const int rc = poseidon::check_ps_args(W, shards, P, n, momentum, buf);
    if (rc != POSEIDON_OK || n == 0)
        return rc;
    return poseidon::launch_ps_apply(W, shards, P, n, lr, momentum, buf, stream) == hipSuccess
               ? POSEIDON_OK
               : POSEIDON_ERR_HIP;
}

extern "C" int poseidon_ps_apply_batch(const poseidon_ps_tensor* tensors, int32_t count, int32_t P,
                                       float lr, float momentum, hipStream_t stream)
{
    if (count < 0 || (count > 0 && !tensors) || P < 1)
        return POSEIDON_ERR_INVALID_ARG;
    for (int32_t i = 0; i < count; ++i) {
        const poseidon_ps_tensor& x = tensors[i];
        const int rc = poseidon::check_ps_args(x.W, x.shards, P, x.n, x.buf ? momentum : 0.0f, x.buf);
        if (rc != POSEIDON_OK)
            return rc;
    }
    static_assert(sizeof(poseidon_ps_tensor) == sizeof(poseidon::PsTensor), "descriptor layout");
    return poseidon::launch_ps_apply_batch(reinterpret_cast<const poseidon::PsTensor*>(tensors), count, P, lr,
                                           momentum, stream) == hipSuccess
               ? POSEIDON_OK
               : POSEIDON_ERR_HIP;
}
