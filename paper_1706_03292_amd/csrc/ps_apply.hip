// Parameter-server aggregation + momentum SGD apply (Sec. 2.1 "Parameter
// Server"; Sec. 4.1 "KV Store", "Managing Consistency").
//
//   s_i = sum_{p<P} G_p[i]   (p increasing, fp32)
//   buf_i = fma(mu, buf_i, s_i);  W_i = fma(-lr, buf_i, W_i)
//
// The kernels are bound by HBM bandwidth: per element they read P shard
// values plus W and buf and write W and buf (4P + 16 bytes), against ~P + 3
// flops.  Each thread owns a group of four consecutive elements -- two such
// groups, 256 elements apart, in the single-tensor launch (apply_pair: a
// wave's accesses to each array read 2 KB in a row) -- and issues its shard
// loads before the dependent adds (bytes in flight); the thread whose group
// runs past the end of the tensor finishes the last one to three elements
// one by one.  Every access is 16 bytes wide: aligned when all
// arrays are 16-byte aligned and the size is a multiple of four (so every
// shard row starts at a 16-byte boundary), otherwise at 4-byte alignment,
// which global loads and stores accept (a tensor of 2,786,166 values over 32
// shards: 5.0 TB/s this way against 3.9 TB/s with 4-byte accesses).  Every
// array is touched once per launch (shards read; W and buf read, then
// written), so all accesses are non-temporal (1-2% faster than cached W/buf
// accesses on 2.4M-16.8M elements).  As many workgroups as needed (one
// pass): a launch-shape sweep over 37K-16.8M elements (block size 64-1024,
// one or two adjacent groups per thread, grid-stride loops capped at 4-16
// workgroups per CU) found one group per thread within 3% of the best
// everywhere and 10% faster than a capped grid-stride loop on large tensors,
// whose last partial pass leaves the chip half idle; of the block sizes,
// 256 threads (PS_THREADS) is the best beside the SF rebuild.  Two groups
// 256 elements apart (rather than adjacent) then measured faster for single
// tensors at P = 8 and P = 32 and the same at P = 16 (ps_group.h).
//
// Three launch forms share the per-group update: one tensor with P
// contiguous shards, many such tensors in one launch, and the KV store's
// pairs (of one or several tensors) with the P workers' updates at separate
// addresses.
#include "common.h"
#include "ps_group.h"

namespace poseidon {
namespace {

// Four waves per workgroup: against one-wave workgroups, as fast on aligned
// tensors alone (5.86 vs 5.94 TB/s on 2,359,296 values at P = 16), faster on
// rows off 16-byte boundaries (6.0 vs 5.6 TB/s on 2,786,166 values at P =
// 32), and beside the SF rebuild a workgroup the size of a rebuild
// workgroup's slot gives that slot back whole (the Inception-shaped
// iteration 0.657 vs 0.681 ms; VGG19-22K 1.739 vs 1.745 ms).
constexpr int PS_THREADS = 256;
// Elements per work block of a single-tensor workgroup: two groups of four per
// thread (apply_pair), each wave covering 512 consecutive elements.  The
// batched pass keeps one group per thread (PS_BATCH_BLOCK_ELEMS): with two,
// its many mid-sized tensors ran slower (the Inception-shaped step's batched
// pass 0.445-0.447 against 0.428-0.430 ms in the iteration, and 0.449-0.453
// with 128- or 64-thread workgroups, which keep the workgroup count).
constexpr int PS_BLOCK_ELEMS = 8 * PS_THREADS;
constexpr int PS_BATCH_BLOCK_ELEMS = 4 * PS_THREADS;

// Offset of thread `tid`'s first element inside a work block.
__device__ inline int64_t pair_offset(int tid)
{
    return (tid >> 6) * (2 * PS_PAIR_GAP) + 4 * (tid & 63);
}
// The KV store's launches are small (one server's share of a tensor, a few
// hundred thousand elements): one-wave workgroups fill the chip better there
// (server 0's VGG19-22K applies at 5.5 vs 4.8 TB/s).
constexpr int KV_THREADS = 64;
constexpr int KV_BLOCK_ELEMS = 4 * KV_THREADS;
constexpr int64_t PS_MAX_GRID = int64_t{1} << 30;

// ---------------------------------------------------------------------------
// One tensor, P contiguous shards.
// ---------------------------------------------------------------------------
template <int PT, bool MOM, bool AL>
__global__ __launch_bounds__(PS_THREADS) void ps_apply_kernel(float* __restrict__ W, const float* __restrict__ G,
                                                              int P, int64_t n, float lr, float mu,
                                                              float* __restrict__ buf)
{
    const Contiguous src{G, n};
    const int64_t stride = static_cast<int64_t>(gridDim.x) * PS_BLOCK_ELEMS;
    for (int64_t e = static_cast<int64_t>(blockIdx.x) * PS_BLOCK_ELEMS + pair_offset(threadIdx.x); e < n; e += stride)
        apply_pair<PT, MOM, AL>(W, buf, src, P, e, n, lr, mu);
}

// ---------------------------------------------------------------------------
// One tensor beside the SF rebuild.  The rebuild's tiles, launched with room
// for it, take 118 VGPRs, so a SIMD's four SF waves leave it 32; a wave of
// this kernel takes 22: one VGPR offset shared by all of a thread's accesses
// (buffer loads, the shard stride in the scalar offset), the shard loads
// LEAN_CHUNK at a time.  It therefore runs on the CUs the rebuild keeps busy,
// streaming memory while the matrix cores work, instead of waiting for a
// rebuild workgroup's slot to free up (VGG19-22K iteration 1.702-1.710 ->
// 1.659-1.675 ms).  Its workgroups walk the tensor grid-stride: one per CU
// beside the fp32 rebuild, one per two CUs beside the split-bf16 one, whose
// matrix-core work the applies then slow less (VGG19-22K iteration
// 1.231-1.237 ms against 1.237-1.245 with one per CU and 1.242-1.250 with
// two; 3/8 and 5/8 of the CUs measured as one half).  The arithmetic and its
// order are apply_group's: the same results, bitwise.  Aligned tensors whose
// P*n*4 bytes fit 31-bit buffer offsets.
// ---------------------------------------------------------------------------
constexpr int LEAN_CHUNK = 4;
constexpr int BUF_DWORD = 0x00020000;   // buffer resource word 3: raw dword accesses
constexpr int NT_AUX = 2;               // non-temporal

typedef unsigned u4v __attribute__((ext_vector_type(4)));

__device__ inline f4 lean_ld(__amdgpu_buffer_rsrc_t r, int voff, int soff)
{
    return __builtin_bit_cast(f4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, NT_AUX));
}

__device__ inline void lean_st(__amdgpu_buffer_rsrc_t r, int voff, f4 v)
{
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u4v, v), r, voff, 0, NT_AUX);
}

template <int PT, bool MOM>
__global__ __launch_bounds__(PS_THREADS) void ps_apply_lean_kernel(float* __restrict__ W, const float* __restrict__ G,
                                                                   int P, int n, float lr, float mu,
                                                                   float* __restrict__ buf)
{
    const __amdgpu_buffer_rsrc_t gr =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(G), static_cast<short>(0), P * n * 4, BUF_DWORD);
    const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(W, static_cast<short>(0), n * 4, BUF_DWORD);
    const __amdgpu_buffer_rsrc_t br = __builtin_amdgcn_make_buffer_rsrc(buf, static_cast<short>(0), n * 4, BUF_DWORD);
    const int np = PT > 0 ? PT : P;
    const int groups = n / 4;
    for (int i = blockIdx.x * PS_THREADS + threadIdx.x; i < groups; i += gridDim.x * PS_THREADS) {
        const int vo = i * 16;
        f4 s = lean_ld(gr, vo, 0);
        for (int p = 1; p < np; p += LEAN_CHUNK) {
            f4 g[LEAN_CHUNK];
#pragma unroll
            for (int c = 0; c < LEAN_CHUNK; ++c)
                if (p + c < np)
                    g[c] = lean_ld(gr, vo, (p + c) * n * 4);
#pragma unroll
            for (int c = 0; c < LEAN_CHUNK; ++c)
                if (p + c < np)
                    s += g[c];
            // one chunk in registers at a time
            __builtin_amdgcn_sched_barrier(0);
        }
        f4 w = lean_ld(wr, vo, 0);
        if constexpr (MOM) {
            const f4 b = fma4(mu, lean_ld(br, vo, 0), s);
            lean_st(br, vo, b);
            w = fma4(-lr, b, w);
        } else {
            w = fma4(-lr, s, w);
        }
        lean_st(wr, vo, w);
    }
}

template <int PT, bool MOM>
hipError_t launch_pt(float* W, const float* G, int32_t P, int64_t n, float lr, float mu, float* buf, bool al,
                     bool beside_sf, hipStream_t stream)
{
    if (beside_sf && al && static_cast<int64_t>(P) * n * 4 <= 0x7fffffffLL) {
        const int64_t want = (n / 4 + PS_THREADS - 1) / PS_THREADS;
        const int64_t cus = device_cu_count();
        const int64_t grid = sf_arithmetic() == POSEIDON_SF_FP32 ? cus : (cus + 1) / 2;
        ps_apply_lean_kernel<PT, MOM><<<static_cast<int>(want < grid ? want : grid), PS_THREADS, 0, stream>>>(
            W, G, P, static_cast<int>(n), lr, mu, buf);
        return hipGetLastError();
    }
    // One work block per workgroup; the grid-stride loop only matters beyond 2^30 workgroups.
    const int64_t want = (n + PS_BLOCK_ELEMS - 1) / PS_BLOCK_ELEMS;
    const int grid = static_cast<int>(want < PS_MAX_GRID ? want : PS_MAX_GRID);
    if (al)
        ps_apply_kernel<PT, MOM, true><<<grid, PS_THREADS, 0, stream>>>(W, G, P, n, lr, mu, buf);
    else
        ps_apply_kernel<PT, MOM, false><<<grid, PS_THREADS, 0, stream>>>(W, G, P, n, lr, mu, buf);
    return hipGetLastError();
}

template <bool MOM>
hipError_t launch_mom(float* W, const float* G, int32_t P, int64_t n, float lr, float mu, float* buf, bool al,
                      bool beside_sf, hipStream_t stream)
{
    switch (P) {
    case 1:  return launch_pt<1, MOM>(W, G, P, n, lr, mu, buf, al, beside_sf, stream);
    case 2:  return launch_pt<2, MOM>(W, G, P, n, lr, mu, buf, al, beside_sf, stream);
    case 4:  return launch_pt<4, MOM>(W, G, P, n, lr, mu, buf, al, beside_sf, stream);
    case 8:  return launch_pt<8, MOM>(W, G, P, n, lr, mu, buf, al, beside_sf, stream);
    case 16: return launch_pt<16, MOM>(W, G, P, n, lr, mu, buf, al, beside_sf, stream);
    case 32: return launch_pt<32, MOM>(W, G, P, n, lr, mu, buf, al, beside_sf, stream);
    default: return launch_pt<0, MOM>(W, G, P, n, lr, mu, buf, al, beside_sf, stream);
    }
}

// ---------------------------------------------------------------------------
// Many tensors in one launch.  The descriptors travel by value in the kernel
// arguments; tensor t owns the workgroups [first_block[t], first_block[t+1]),
// each of which updates PS_BATCH_BLOCK_ELEMS consecutive elements of it, one
// group of four per thread.
// ---------------------------------------------------------------------------
struct PsBatchItem {
    float* W;
    const float* G;
    float* buf;
    int64_t n;
    int32_t first_block;
    int32_t aligned;
};

struct PsBatchArgs {
    int32_t first_block[PS_BATCH_MAX];   // item[t].first_block, contiguous: a few wide scalar loads
    PsBatchItem item[PS_BATCH_MAX];
    int32_t count;
};

template <int PT, bool MOM>
__global__ __launch_bounds__(PS_THREADS) void ps_apply_batch_kernel(const PsBatchArgs args, int P, float lr,
                                                                    float mu, int total_blocks)
{
    // Workgroup g handles work blocks g, g + gridDim.x, ... (one pass when the
    // grid covers every block).  The block's tensor is the number of later
    // descriptors whose first block it has reached: a fully unrolled count
    // over the contiguous first-block array, read with a few wide scalar
    // loads, so a wave waits for one load latency before it knows its tensor
    // (a binary search waits for one per step).
    for (int b = blockIdx.x; b < total_blocks; b += gridDim.x) {
        int t = 0;
#pragma unroll
        for (int k = 1; k < PS_BATCH_MAX; ++k)
            t += (k < args.count && args.first_block[k] <= b) ? 1 : 0;
        const PsBatchItem& it = args.item[t];
        const int64_t e = static_cast<int64_t>(b - it.first_block) * PS_BATCH_BLOCK_ELEMS + 4 * threadIdx.x;
        if (e < it.n) {
            const Contiguous src{it.G, it.n};
            if (it.aligned)
                apply_group<PT, MOM, true>(it.W, it.buf, src, P, e, it.n, lr, mu);
            else
                apply_group<PT, MOM, false>(it.W, it.buf, src, P, e, it.n, lr, mu);
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
// KV-store apply: pairs that one server holds, of one or several tensors,
// with the P workers' updates at separate addresses (one pointer per worker,
// passed in worker order, the same for every range of the launch).  Range r
// covers elements [offset, offset + length) of the tensor (W, buf) and owns
// the workgroups [first_block[r], first_block[r+1]); each workgroup updates
// KV_BLOCK_ELEMS consecutive elements of its range, with 16-byte accesses
// that are aligned when the range's arrays allow it.
// ---------------------------------------------------------------------------
struct KvRange {
    float* W;
    float* buf;          // NULL on a launch without momentum
    int64_t offset;
    int64_t length;
    int64_t delta;       // a message's values of element e are at message + delta + e
    int32_t first_block;
    int32_t aligned;
};

struct KvArgs {
    const float* g[KV_MAX_P];
    uint64_t msg_mask;                    // bit p: worker p's pointer is a message
    int32_t first_block[KV_MAX_RANGES];   // r[k].first_block, contiguous (as in the batched kernel)
    KvRange r[KV_MAX_RANGES];
    int32_t nranges;
};

template <int PT, bool MOM>
__global__ __launch_bounds__(KV_THREADS) void kv_apply_kernel(const KvArgs a, int P, float lr, float mu)
{
    const int b = blockIdx.x;
    int r = 0;                                  // as in the batched kernel: independent loads
#pragma unroll
    for (int k = 1; k < KV_MAX_RANGES; ++k)
        r += (k < a.nranges && a.first_block[k] <= b) ? 1 : 0;
    const KvRange& q = a.r[r];
    const int64_t j = static_cast<int64_t>(b - q.first_block) * KV_BLOCK_ELEMS + 4 * threadIdx.x;
    if (j >= q.length)
        return;
    const PerWorker src{a.g, a.msg_mask, q.delta};
    if (q.aligned)
        apply_group<PT, MOM, true>(q.W, q.buf, src, P, q.offset + j, q.offset + q.length, lr, mu);
    else
        apply_group<PT, MOM, false>(q.W, q.buf, src, P, q.offset + j, q.offset + q.length, lr, mu);
}

// ---------------------------------------------------------------------------
// KV-store message: the slices [src_k, src_k + length_k) of one worker's
// updates copied one after another into its message (range k starts at
// element dst_k).  Each workgroup copies PACK_BLOCK_ELEMS elements of
// one range: four 16-byte groups per thread, all loads issued before the
// stores (a copy moves few bytes per thread otherwise).
// ---------------------------------------------------------------------------
constexpr int PACK_UNROLL = 4;
constexpr int PACK_BLOCK_ELEMS = PACK_UNROLL * KV_BLOCK_ELEMS;

struct PackArgs {
    const float* src[KV_PACK_MAX];
    int64_t dst[KV_PACK_MAX];
    int64_t length[KV_PACK_MAX];
    int32_t first_block[KV_PACK_MAX];
    int32_t count;
};

__global__ __launch_bounds__(KV_THREADS) void kv_pack_kernel(const PackArgs a, float* __restrict__ message)
{
    const int b = blockIdx.x;
    int k = 0;
#pragma unroll
    for (int q = 1; q < KV_PACK_MAX; ++q)
        k += (q < a.count && a.first_block[q] <= b) ? 1 : 0;
    const int64_t j0 = static_cast<int64_t>(b - a.first_block[k]) * PACK_BLOCK_ELEMS + 4 * threadIdx.x;
    const int64_t len = a.length[k];
    const float* __restrict__ src = a.src[k];
    float* __restrict__ dst = message + a.dst[k];
    f4 v[PACK_UNROLL];
#pragma unroll
    for (int u = 0; u < PACK_UNROLL; ++u) {
        const int64_t j = j0 + u * KV_BLOCK_ELEMS;
        if (j + 3 < len)
            v[u] = ld4<false>(src + j);
    }
#pragma unroll
    for (int u = 0; u < PACK_UNROLL; ++u) {
        const int64_t j = j0 + u * KV_BLOCK_ELEMS;
        if (j + 3 < len) {
            st4<false>(dst + j, v[u]);
        } else {
            for (int64_t q = j; q < len; ++q)
                dst[q] = src[q];
        }
    }
}

template <bool MOM>
void launch_kv_mom(const KvArgs& a, int grid, int32_t P, float lr, float mu, hipStream_t stream)
{
    switch (P) {
    case 4:  kv_apply_kernel<4, MOM><<<grid, KV_THREADS, 0, stream>>>(a, P, lr, mu); break;
    case 8:  kv_apply_kernel<8, MOM><<<grid, KV_THREADS, 0, stream>>>(a, P, lr, mu); break;
    case 16: kv_apply_kernel<16, MOM><<<grid, KV_THREADS, 0, stream>>>(a, P, lr, mu); break;
    case 32: kv_apply_kernel<32, MOM><<<grid, KV_THREADS, 0, stream>>>(a, P, lr, mu); break;
    default: kv_apply_kernel<0, MOM><<<grid, KV_THREADS, 0, stream>>>(a, P, lr, mu); break;
    }
}

}  // namespace

hipError_t launch_ps_apply(float* W, const float* shards, int32_t P, int64_t n,
                           float lr, float momentum, float* buf, hipStream_t stream, bool beside_sf)
{
    const bool al = (n % 4 == 0) && aligned16(W) && aligned16(shards) && (!buf || aligned16(buf));
    if (buf)
        return launch_mom<true>(W, shards, P, n, lr, momentum, buf, al, beside_sf, stream);
    return launch_mom<false>(W, shards, P, n, lr, 0.0f, nullptr, al, beside_sf, stream);
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
            const int grid = nb < PS_MAX_GRID ? nb : static_cast<int>(PS_MAX_GRID);
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
            const int64_t nb = (t[i].n + PS_BATCH_BLOCK_ELEMS - 1) / PS_BATCH_BLOCK_ELEMS;
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
            a.first_block[a.count - 1] = it.first_block;
            it.aligned = (t[i].n % 4 == 0) && aligned16(t[i].W) && aligned16(t[i].shards) &&
                         (!t[i].buf || aligned16(t[i].buf));
            blocks += nb;
        }
        const hipError_t e = flush();
        if (e != hipSuccess)
            return e;
    }
    return hipSuccess;
}

hipError_t launch_kv_apply(const KvApplyRange* ranges, int32_t nranges, const float* const* grads,
                           uint64_t msg_mask, int32_t P, float lr, float momentum, hipStream_t stream)
{
    bool grads_al = true;
    for (int32_t p = 0; p < P; ++p)
        grads_al = grads_al && aligned16(grads[p]);
    // Ranges with a momentum buffer and ranges without take separate launches.
    for (int mom = 1; mom >= 0; --mom) {
        KvArgs a{};
        for (int32_t p = 0; p < P; ++p)
            a.g[p] = grads[p];
        a.msg_mask = msg_mask;
        int64_t blocks = 0;
        auto flush = [&]() -> hipError_t {
            if (blocks == 0)
                return hipSuccess;
            if (mom)
                launch_kv_mom<true>(a, static_cast<int>(blocks), P, lr, momentum, stream);
            else
                launch_kv_mom<false>(a, static_cast<int>(blocks), P, lr, 0.0f, stream);
            a.nranges = 0;
            blocks = 0;
            return hipGetLastError();
        };
        for (int32_t i = 0; i < nranges; ++i) {
            const KvApplyRange& x = ranges[i];
            if (x.length == 0 || (x.buf != nullptr) != (mom == 1))
                continue;
            const int64_t nb = (x.length + KV_BLOCK_ELEMS - 1) / KV_BLOCK_ELEMS;
            if (a.nranges == KV_MAX_RANGES || blocks + nb > INT32_MAX) {
                const hipError_t e = flush();
                if (e != hipSuccess)
                    return e;
            }
            KvRange& r = a.r[a.nranges];
            r.W = x.W;
            r.buf = x.buf;
            r.offset = x.offset;
            r.length = x.length;
            r.delta = x.delta;
            r.first_block = static_cast<int32_t>(blocks);
            r.aligned = grads_al && aligned16(x.W) && (!x.buf || aligned16(x.buf)) && x.offset % 4 == 0 &&
                        (msg_mask == 0 || x.delta % 4 == 0);
            a.first_block[a.nranges++] = r.first_block;
            blocks += nb;
        }
        const hipError_t e = flush();
        if (e != hipSuccess)
            return e;
    }
    return hipSuccess;
}

hipError_t launch_kv_pack(const float* const* src, const int64_t* dst, const int64_t* length, int32_t count,
                          float* message, hipStream_t stream)
{
    for (int32_t i0 = 0; i0 < count; i0 += KV_PACK_MAX) {
        PackArgs a{};
        int64_t blocks = 0;
        for (int32_t i = i0; i < count && i < i0 + KV_PACK_MAX; ++i) {
            const int32_t k = a.count++;
            a.src[k] = src[i];
            a.dst[k] = dst[i];
            a.length[k] = length[i];
            a.first_block[k] = static_cast<int32_t>(blocks);
            blocks += (length[i] + PACK_BLOCK_ELEMS - 1) / PACK_BLOCK_ELEMS;
            if (blocks > INT32_MAX)
                return hipErrorInvalidValue;
        }
        if (blocks == 0)
            continue;
        kv_pack_kernel<<<static_cast<int>(blocks), KV_THREADS, 0, stream>>>(a, message);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess)
            return e;
    }
    return hipSuccess;
}

}  // namespace poseidon
