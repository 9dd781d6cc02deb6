// One iteration's synchronisation of a network on a pool of HIP streams
// (Sec. 3 "wait-free backpropagation"; Sec. 4.1 "Client Library", "Managing
// Consistency"; Alg. 2).  The host walks the tensors in backpropagation
// order, asks Alg. 1 for each one's scheme, and enqueues the matching update
// on the caller's stream or a stream of the pool; a fork event and a join
// event per pool stream used make the whole iteration a single asynchronous
// operation on the caller's stream (the bulk-synchronous barrier).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <vector>

#include "common.h"

struct poseidon_stream_pool {
    int device = -1;
    std::vector<hipStream_t> streams;
    std::vector<hipEvent_t> joined;   // one per stream: its last update of the iteration
    hipEvent_t fork = nullptr;        // work enqueued on the caller's stream before the iteration
    bool timing = false;
    int32_t wfbp_policy = POSEIDON_WFBP_SERIAL;
    std::vector<hipEvent_t> t_start;  // per launch of the last timed iteration
    std::vector<hipEvent_t> t_stop;
    std::vector<poseidon_launch_record> t_rec;
    bool t_valid = false;             // a timed iteration has been enqueued
};

namespace poseidon {

int device_cu_count()
{
    static std::atomic<int> cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess)
        return 256;
    if (dev >= 0 && dev < 64) {
        const int c = cache[dev].load(std::memory_order_relaxed);
        if (c > 0)
            return c;
    }
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
        cus = 256;
    if (dev >= 0 && dev < 64)
        cache[dev].store(cus, std::memory_order_relaxed);
    return cus;
}

}  // namespace poseidon

namespace {

void destroy_pool(poseidon_stream_pool* pool)
{
    for (hipStream_t s : pool->streams)
        if (s) {
            (void)hipStreamSynchronize(s);
            (void)hipStreamDestroy(s);
        }
    for (hipEvent_t e : pool->joined)
        if (e)
            (void)hipEventDestroy(e);
    if (pool->fork)
        (void)hipEventDestroy(pool->fork);
    for (hipEvent_t e : pool->t_start)
        (void)hipEventDestroy(e);
    for (hipEvent_t e : pool->t_stop)
        (void)hipEventDestroy(e);
    delete pool;
}

// Make sure the pool holds timing events for `count` launches.
bool reserve_timing(poseidon_stream_pool* pool, int32_t count)
{
    while (static_cast<int32_t>(pool->t_start.size()) < count) {
        hipEvent_t a = nullptr, b = nullptr;
        if (hipEventCreate(&a) != hipSuccess)
            return false;
        if (hipEventCreate(&b) != hipSuccess) {
            (void)hipEventDestroy(a);
            return false;
        }
        pool->t_start.push_back(a);
        pool->t_stop.push_back(b);
    }
    pool->t_rec.clear();
    return true;
}

}  // namespace

extern "C" int poseidon_pool_create(int32_t num_streams, poseidon_stream_pool** out)
{
    if (!out || num_streams < 1 || num_streams > 64)
        return POSEIDON_ERR_INVALID_ARG;
    *out = nullptr;
    auto* pool = new poseidon_stream_pool;
    bool ok = hipGetDevice(&pool->device) == hipSuccess &&
              hipEventCreateWithFlags(&pool->fork, hipEventDisableTiming) == hipSuccess;
    for (int32_t i = 0; ok && i < num_streams; ++i) {
        hipStream_t s = nullptr;
        hipEvent_t e = nullptr;
        // Default priority on purpose: every stream of the library shares one.
        ok = hipStreamCreateWithFlags(&s, hipStreamNonBlocking) == hipSuccess;
        if (ok)
            pool->streams.push_back(s);
        ok = ok && hipEventCreateWithFlags(&e, hipEventDisableTiming) == hipSuccess;
        if (ok)
            pool->joined.push_back(e);
    }
    if (!ok) {
        destroy_pool(pool);
        return POSEIDON_ERR_HIP;
    }
    *out = pool;
    return POSEIDON_OK;
}

extern "C" int poseidon_pool_destroy(poseidon_stream_pool* pool)
{
    if (pool)
        destroy_pool(pool);
    return POSEIDON_OK;
}

namespace {

// PS tensors below SMALL_PS_ELEMS elements are launch-bound on their own (a
// launch costs a few microseconds; 2^17 elements at P = 32 move 19 MB, about
// 4 us of HBM time): the iteration gathers them into a batched pass.  When
// the PS applies are the iteration's critical path -- the SF rebuilds would
// take less time than them, judged by the kernels' rates on this GPU
// (sf_seconds; PS_BYTES_PER_S) -- every
// launch saved shortens the iteration, and tensors below PS_CRITICAL_ELEMS
// join the pass too (Inception-shaped workload, 95 tensors at P = 32:
// 0.69 vs 0.77 ms per iteration); when the SF chain is the critical path,
// large PS tensors keep launches of their own, which interleave with it
// (VGG19-22K: neutral to 0.8% slower with the larger threshold).
constexpr int64_t SMALL_PS_ELEMS = int64_t{1} << 17;
constexpr int64_t PS_CRITICAL_ELEMS = int64_t{1} << 21;
constexpr double PS_BYTES_PER_S = 5.0e12;   // the PS kernel's rate on this GPU (the SF one: sf_seconds)
// An iteration whose work would take less than this on one stream is bound
// by launch latency: the second stream's fork and join cost more than the
// overlap gains (a 1024 x 512 FC layer and a 1M-value PS layer at P = 4:
// 0.033 ms on one stream, 0.043-0.053 ms on two).
constexpr double ONE_STREAM_BELOW_S = 30e-6;
// Two streams pay when one kind of update is small next to the other: the
// small one's launches fill the gaps the large one leaves (its tile rounds'
// ends, the last partial round), and take little from it.  When the two are
// of comparable size neither has gaps to fill, and the co-running launches
// only delay each other: the 4096 x 4096 layer rebuilt at K = 256 (one round
// of tiles, 0.083 ms alone with fp32 products, 0.060 split) beside 805 MB of
// PS applies (0.139-0.152 ms alone) took 0.236 ms on two streams against
// 0.222 ms one after the other (split: 0.216 against 0.206).  Below this
// ratio of the smaller estimated time to the larger the iteration uses two
// streams (VGG19-22K: 0.27 split, 0.19 fp32, two streams 1.24 ms against
// 1.37 on one, split; the Inception-shaped workload: 0.05; that 4096 x 4096
// layer through both schemes: 0.38 split, 0.41 fp32).
constexpr double CORUN_MAX_RATIO = 0.35;
// When the PS applies are the longer kind on two streams, every SF launch is
// spread over few workgroups that walk its tiles, given this fraction of the
// applies' estimated time (each layer its share by flops): thin beside the
// HBM-bound applies the rebuilds take less from them than a short full-chip
// launch does (Inception-shaped iteration 0.651 -> 0.637 ms, its 1000 x 2048
// classifier on 64 workgroups for 0.52 ms instead of 512 for 0.08 ms; 48 or
// 56 workgroups, whose rebuild outlasts the applies, 0.67-0.69 ms; 72-96,
// 0.647 ms).
constexpr double SF_SPREAD_OF_PS = 0.9;
// When the SF rebuilds are the longer kind on two streams, the rebuilds
// leave each SIMD room for waves of the lean PS kernel and the large PS
// applies use it, so that they stream memory on the CUs the rebuilds keep
// busy -- provided the applies still end before the rebuilds: at the lean
// kernel's rate beside them they must take at most this fraction of the
// rebuilds' estimated time.  That rate is set by the lean kernel's grid
// (one workgroup on every second CU beside the split-bf16 rebuild: its
// 256 x 128 tiles' two waves of 228 VGPRs per SIMD; VGG19-22K's largest PS
// tensors, 189 MB, in 0.10 ms) and by the waves that fit beside the rebuild's
// (one workgroup per CU, one wave per SIMD beside the fp32 128 x 128 tiles'
// four of 120; 0.141 ms).
constexpr double LEAN_PS_BYTES_PER_S_SPLIT = 1.9e12;
constexpr double LEAN_PS_BYTES_PER_S_FP32 = 1.3e12;
constexpr double LEAN_OF_SF = 0.85;

// The iteration of poseidon_sync_iteration (ready == NULL: every update waits
// for the work enqueued on `stream` before the call) and of
// poseidon_sync_iteration_wfbp (tensor t's update waits for ready[t], or for
// every ready event, as the pool's schedule says).
int sync_impl(poseidon_stream_pool* pool, const poseidon_tensor* tensors, int32_t count, int64_t B, int32_t P,
              float lr, float momentum, const hipEvent_t* events, hipStream_t stream, int32_t* schemes)
{
    using namespace poseidon;
    if (!pool || count < 0 || (count > 0 && !tensors) || B < 0 || P < 1)
        return POSEIDON_ERR_INVALID_ARG;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess)
        return POSEIDON_ERR_HIP;
    if (dev != pool->device)
        return POSEIDON_ERR_INVALID_ARG;
    const int64_t K = B * static_cast<int64_t>(P);
    // Under POSEIDON_WFBP_SERIAL the caller's stream waits for every ready
    // event (below, once everything has been validated) and the iteration is
    // then poseidon_sync_iteration's on that stream: `ready` is what the
    // scheduling sees, `events` what the arguments hold.
    const bool serial = events && pool->wfbp_policy == POSEIDON_WFBP_SERIAL;
    const hipEvent_t* const ready = serial ? nullptr : events;

    // Validate everything and fix every scheme before enqueueing anything.
    std::vector<int32_t> plan(static_cast<size_t>(count));
    double sf_flops = 0.0, t_sf = 0.0, ps_bytes = 0.0;
    for (int32_t t = 0; t < count; ++t) {
        const poseidon_tensor& x = tensors[t];
        if ((x.kind != POSEIDON_KIND_FC && x.kind != POSEIDON_KIND_OTHER) || x.reserved != 0 ||
            x.M < 0 || x.N < 0 || (x.N > 0 && x.M > INT64_MAX / x.N))
            return POSEIDON_ERR_INVALID_ARG;
        int32_t scheme = POSEIDON_PS;
        if (x.kind == POSEIDON_KIND_FC) {
            scheme = poseidon_hybcomm_choose(x.M, x.N, B, P);
            if (scheme < 0)
                return POSEIDON_ERR_INVALID_ARG;
        }
        const int64_t n = x.M * x.N;
        int rc;
        if (scheme == POSEIDON_SFB) {
            if (n > 0 && K > 0 && (!x.U || !x.V))
                return POSEIDON_ERR_PAYLOAD;
            rc = x.buf ? check_sf_momentum_args(x.W, x.buf, x.U, x.V, x.M, x.N, K)
                       : check_sf_args(x.W, x.U, x.V, x.M, x.N, K);
            sf_flops += 2.0 * static_cast<double>(n) * static_cast<double>(K);
            if (rc == POSEIDON_OK && n > 0 && K > 0)
                t_sf += sf_seconds(x.M, x.N, K);
        } else {
            if (n > 0 && !x.shards)
                return POSEIDON_ERR_PAYLOAD;
            rc = check_ps_args(x.W, x.shards, P, n, x.buf ? momentum : 0.0f, x.buf);
            ps_bytes += static_cast<double>(n) * (4.0 * P + (x.buf ? 16.0 : 8.0));
        }
        if (rc != POSEIDON_OK)
            return rc;
        if (events && !events[t])
            return POSEIDON_ERR_INVALID_ARG;
        plan[static_cast<size_t>(t)] = scheme;
    }
    // Under POSEIDON_WFBP_ALL_LAST every update waits for every ready event
    // and the launches are the plain iteration's: `per` is what the per-tensor
    // scheduling sees.
    const bool all_last = ready && pool->wfbp_policy == POSEIDON_WFBP_ALL_LAST;
    const hipEvent_t* per = all_last ? nullptr : ready;
    // The tensors' updates run concurrently (two streams, batched and grouped
    // launches): no tensor may write where another one reads or writes.
    {
        std::vector<Span> writes, reads;
        for (int32_t t = 0; t < count; ++t) {
            const poseidon_tensor& x = tensors[t];
            const int64_t n = x.M * x.N;
            if (n == 0)
                continue;
            add_span(writes, x.W, n * 4);
            if (plan[static_cast<size_t>(t)] == POSEIDON_SFB) {
                if (x.buf)
                    add_span(writes, x.buf, n * 4);
                add_span(reads, x.U, K * x.M * 4);
                add_span(reads, x.V, K * x.N * 4);
            } else {
                if (x.buf)
                    add_span(writes, x.buf, n * 4);
                add_span(reads, x.shards, n * 4 * static_cast<int64_t>(P));
            }
        }
        if (writes_collide(std::move(writes), reads))
            return POSEIDON_ERR_INVALID_ARG;
    }
    if (schemes)
        for (int32_t t = 0; t < count; ++t)
            schemes[t] = plan[static_cast<size_t>(t)];
    // With ready events each large tensor keeps its own launch, so that it
    // starts as soon as its own backward pass has run.
    const double t_ps = ps_bytes / PS_BYTES_PER_S;
    const int64_t small_elems =
        (!per && t_sf < t_ps) ? PS_CRITICAL_ELEMS : SMALL_PS_ELEMS;
    int32_t active = 0;
    int32_t small_ps = 0;
    int32_t plain_sf = 0;     // SFB layers without a momentum buffer
    for (int32_t t = 0; t < count; ++t) {
        const poseidon_tensor& x = tensors[t];
        const int64_t n = x.M * x.N;
        if (n == 0)
            continue;
        if (plan[static_cast<size_t>(t)] == POSEIDON_SFB) {
            if (K > 0 || x.buf)
                ++active;
            if (K > 0 && !x.buf)
                ++plain_sf;
        } else if (n < small_elems) {
            ++small_ps;
        } else {
            ++active;
        }
    }
    // One launch per tensor with work, except: small PS tensors share one
    // batched pass after the other PS launches; and the SFB layers without a
    // momentum buffer share one grouped launch, at the place of the first of
    // them in backpropagation order, whose single tile list lets one layer's
    // last tiles (and a layer that is exactly one round of tiles, whose W
    // epilogues would otherwise all run at once) overlap the next layer's
    // (VGG19-22K iteration: 1.75 vs 1.78 ms, A/B in alternating processes).
    // With ready events that holds under the held schedules, where the SFB
    // rebuilds wait for the end of the caller's backward pass (on one GPU they
    // need the matrix cores its GEMMs use); under POSEIDON_WFBP_EACH every
    // SFB layer keeps its own launch, so that each starts as soon as its own
    // backward pass has run.
    const bool sfb_last = per && pool->wfbp_policy == POSEIDON_WFBP_SFB_LAST;
    const int32_t S = static_cast<int32_t>(pool->streams.size());
    const bool tiny = t_sf + t_ps < ONE_STREAM_BELOW_S;
    // With ready events the second stream also lets the updates start while
    // the caller's backward pass still runs, so it is kept.
    const bool balanced = !per && std::min(t_sf, t_ps) > CORUN_MAX_RATIO * std::max(t_sf, t_ps);
    // Spread SF launches (below) replace the grouped one; under the held
    // schedule the launches are the plain iteration's, spread included.
    const bool spread = (!ready || all_last) && S > 1 && !tiny && !balanced && t_ps > t_sf && sf_flops > 0.0;
    const bool group_sf = (!per || sfb_last) && plain_sf > 1 && !spread;
    std::vector<SfTensor> grouped;   // in backpropagation order
    if (group_sf)
        for (int32_t t = count - 1; t >= 0; --t) {
            const poseidon_tensor& x = tensors[t];
            if (plan[static_cast<size_t>(t)] == POSEIDON_SFB && x.M * x.N > 0 && K > 0 && !x.buf)
                grouped.push_back(SfTensor{x.W, x.U, x.V, x.M, x.N});
        }
    const int32_t launches = active - (group_sf ? plain_sf - 1 : 0) + (small_ps > 0 ? 1 : 0);
    if (pool->timing) {
        if (!reserve_timing(pool, launches))
            return POSEIDON_ERR_HIP;
        pool->t_valid = true;
    }
    if (launches == 0)
        return POSEIDON_OK;

    // Stream assignment: the compute-bound SF reconstructions and the
    // bandwidth-bound PS applies go to two streams (below: which), each kind
    // in backpropagation order, so that the two kinds overlap on the GPU
    // instead of queueing behind each other.  A one-stream pool, or an
    // iteration too small or too balanced to gain from the overlap,
    // serialises everything on one.
    const int32_t used = (S > 1 && launches > 1 && !tiny && !balanced) ? 2 : 1;
    hipEvent_t waited[2] = {nullptr, nullptr};   // last ready event each used stream waits on
    // An iteration issued on one stream that waits for nothing but the
    // caller's earlier work runs on the caller's stream itself: no fork and
    // join events (two fewer packets per iteration for latency-bound ones).
    const bool direct = !ready && used == 1;
    // Without ready events a two-stream iteration runs the kind with the
    // longer estimated time on the caller's stream itself and forks only the
    // other kind onto the pool's first stream, so that the iteration's
    // critical path crosses no queue boundary: with both kinds forked, the
    // join back to the caller's stream and the next iteration's fork left the
    // GPU idle for 24-29 us between iterations (VGG19-22K 1.745-1.754 ->
    // 1.725-1.747 ms, Inception-shaped 0.660 -> 0.650 ms).
    const bool split = !ready && used == 2;
    std::vector<hipStream_t> st(pool->streams.begin(), pool->streams.end());
    if (direct)
        st[0] = stream;
    int32_t forked = -1;   // split: the lane (0 SFB, 1 PS) on the pool stream
    // Seconds per flop given to the SF launches when they are spread.
    const double sf_spread = (spread && used == 2) ? SF_SPREAD_OF_PS * t_ps / sf_flops : 0.0;
    // The PS applies beside the rebuilds on the same CUs (see LEAN_OF_SF).
    const double lean_rate =
        sf_arithmetic() == POSEIDON_SF_FP32 ? LEAN_PS_BYTES_PER_S_FP32 : LEAN_PS_BYTES_PER_S_SPLIT;
    const bool room = (!ready || all_last) && used == 2 && t_sf >= t_ps && ps_bytes / lean_rate <= LEAN_OF_SF * t_sf;
    if (split) {
        const int32_t crit = t_sf >= t_ps ? 0 : 1;
        forked = 1 - crit;
        st[crit] = stream;
        st[forked] = pool->streams[0];
    }
    if (serial) {
        // The caller's stream itself waits: for events recorded on it these
        // waits are met in order, without a wake-up from another queue (the
        // waits gathered on a pool stream, and the caller's stream waiting for
        // that stream once, started the first update 81-84 us after the
        // backward pass's last kernel instead of 6-9).
        std::vector<hipEvent_t> seen;
        for (int32_t t = 0; t < count; ++t) {
            if (std::find(seen.begin(), seen.end(), events[t]) != seen.end())
                continue;
            seen.push_back(events[t]);
            if (hipStreamWaitEvent(stream, events[t], 0) != hipSuccess)
                return POSEIDON_ERR_HIP;
        }
    }
    if (split) {
        if (hipEventRecord(pool->fork, stream) != hipSuccess ||
            hipStreamWaitEvent(pool->streams[0], pool->fork, 0) != hipSuccess)
            return POSEIDON_ERR_HIP;
    } else if (!direct && !ready) {
        if (hipEventRecord(pool->fork, stream) != hipSuccess)
            return POSEIDON_ERR_HIP;
        for (int32_t s = 0; s < used; ++s)
            if (hipStreamWaitEvent(pool->streams[s], pool->fork, 0) != hipSuccess)
                return POSEIDON_ERR_HIP;
    } else if (all_last) {
        // The first stream waits for every distinct event, the second for
        // the first (one wait packet instead of one per event).
        std::vector<hipEvent_t> seen;
        for (int32_t t = 0; t < count; ++t)
            if (std::find(seen.begin(), seen.end(), ready[t]) == seen.end())
                seen.push_back(ready[t]);
        for (hipEvent_t e : seen)
            if (hipStreamWaitEvent(pool->streams[0], e, 0) != hipSuccess)
                return POSEIDON_ERR_HIP;
        if (used > 1 && (hipEventRecord(pool->fork, pool->streams[0]) != hipSuccess ||
                         hipStreamWaitEvent(pool->streams[1], pool->fork, 0) != hipSuccess))
            return POSEIDON_ERR_HIP;
    }

    // Tensor t's launch on pool stream si: with ready events it first waits
    // for ready[t] (once per run of equal events), then the timing events, if
    // on, bracket the launch alone.
    bool waited_all = false;         // sfb_last: stream 0 has waited for every ready event
    auto wait_all = [&](hipStream_t s) -> bool {
        std::vector<hipEvent_t> seen;
        for (int32_t t = 0; t < count; ++t) {
            if (std::find(seen.begin(), seen.end(), ready[t]) != seen.end())
                continue;
            seen.push_back(ready[t]);
            if (hipStreamWaitEvent(s, ready[t], 0) != hipSuccess)
                return false;
        }
        waited_all = true;
        return true;
    };
    auto timed = [&](hipStream_t s, int32_t scheme, int32_t tensor, int32_t si, auto&& launch) -> bool {
        if (sfb_last && scheme == POSEIDON_SFB) {
            if (!waited_all && !wait_all(s))
                return false;
        } else if (per && per[tensor] != waited[si]) {
            if (hipStreamWaitEvent(s, per[tensor], 0) != hipSuccess)
                return false;
            waited[si] = per[tensor];
        }
        const size_t r = pool->t_rec.size();
        if (pool->timing && hipEventRecord(pool->t_start[r], s) != hipSuccess)
            return false;
        if (launch() != hipSuccess)
            return false;
        if (pool->timing) {
            if (hipEventRecord(pool->t_stop[r], s) != hipSuccess)
                return false;
            pool->t_rec.push_back(poseidon_launch_record{scheme, tensor, si, 0.0f});
        }
        return true;
    };
    bool grouped_issued = false;
    std::vector<PsTensor> small;     // in backpropagation order
    std::vector<int32_t> small_idx;
    for (int32_t t = count - 1; t >= 0; --t) {
        const poseidon_tensor& x = tensors[t];
        const int64_t n = x.M * x.N;
        if (n == 0)
            continue;
        if (plan[static_cast<size_t>(t)] == POSEIDON_PS && n < small_elems) {
            small.push_back(PsTensor{x.W, x.shards, x.buf, n});
            small_idx.push_back(t);
            continue;
        }
        if (plan[static_cast<size_t>(t)] == POSEIDON_SFB) {
            if (K == 0 && !x.buf)
                continue;
            hipStream_t s = st[0];
            if (group_sf && !x.buf) {
                if (!grouped_issued) {
                    grouped_issued = true;
                    if (!timed(s, POSEIDON_SFB, -1, 0, [&] {
                            return launch_sf_apply_batch(grouped.data(), static_cast<int32_t>(grouped.size()), K,
                                                         lr, s, room);
                        }))
                        return POSEIDON_ERR_HIP;
                }
                continue;
            }
            if (!timed(s, POSEIDON_SFB, t, 0, [&] {
                    const double spread_s = sf_spread * 2.0 * static_cast<double>(n) * static_cast<double>(K);
                    return x.buf ? launch_sf_apply_momentum(x.W, x.buf, x.U, x.V, x.M, x.N, K, lr, momentum, s,
                                                            spread_s)
                                 : launch_sf_apply(x.W, x.U, x.V, x.M, x.N, K, lr, s, spread_s, room);
                }))
                return POSEIDON_ERR_HIP;
        } else {
            const int32_t si = used == 1 ? 0 : 1;
            hipStream_t s = st[si];
            if (!timed(s, POSEIDON_PS, t, si, [&] {
                    return launch_ps_apply(x.W, x.shards, P, n, lr, x.buf ? momentum : 0.0f, x.buf, s, room);
                }))
                return POSEIDON_ERR_HIP;
        }
    }

    if (!small.empty()) {
        // The batched pass waits for every ready event of its tensors.
        const int32_t si = used == 1 ? 0 : 1;
        hipStream_t s = st[si];
        if (per)
            for (int32_t t : small_idx)
                if (per[t] != waited[si]) {
                    if (hipStreamWaitEvent(s, per[t], 0) != hipSuccess)
                        return POSEIDON_ERR_HIP;
                    waited[si] = per[t];
                }
        const size_t r = pool->t_rec.size();
        if (pool->timing && hipEventRecord(pool->t_start[r], s) != hipSuccess)
            return POSEIDON_ERR_HIP;
        if (launch_ps_apply_batch(small.data(), static_cast<int32_t>(small.size()), P, lr, momentum, s) !=
            hipSuccess)
            return POSEIDON_ERR_HIP;
        if (pool->timing) {
            if (hipEventRecord(pool->t_stop[r], s) != hipSuccess)
                return POSEIDON_ERR_HIP;
            pool->t_rec.push_back(poseidon_launch_record{POSEIDON_PS, -1, si, 0.0f});
        }
    }

    if (split) {
        if (hipEventRecord(pool->joined[0], pool->streams[0]) != hipSuccess ||
            hipStreamWaitEvent(stream, pool->joined[0], 0) != hipSuccess)
            return POSEIDON_ERR_HIP;
        return POSEIDON_OK;
    }
    for (int32_t s = 0; s < used && !direct; ++s) {
        if (hipEventRecord(pool->joined[s], pool->streams[s]) != hipSuccess ||
            hipStreamWaitEvent(stream, pool->joined[s], 0) != hipSuccess)
            return POSEIDON_ERR_HIP;
    }
    return POSEIDON_OK;
}

}  // namespace

extern "C" int poseidon_sync_iteration(poseidon_stream_pool* pool,
                                       const poseidon_tensor* tensors, int32_t count,
                                       int64_t B, int32_t P, float lr, float momentum,
                                       hipStream_t stream, int32_t* schemes)
{
    return sync_impl(pool, tensors, count, B, P, lr, momentum, nullptr, stream, schemes);
}

extern "C" int poseidon_sync_iteration_wfbp(poseidon_stream_pool* pool,
                                            const poseidon_tensor* tensors, int32_t count,
                                            int64_t B, int32_t P, float lr, float momentum,
                                            const hipEvent_t* ready, hipStream_t stream, int32_t* schemes)
{
    if (count > 0 && !ready)
        return POSEIDON_ERR_INVALID_ARG;
    static const hipEvent_t none = nullptr;
    return sync_impl(pool, tensors, count, B, P, lr, momentum, count > 0 ? ready : &none, stream, schemes);
}

extern "C" int poseidon_pool_set_wfbp_policy(poseidon_stream_pool* pool, int32_t policy)
{
    if (!pool || (policy != POSEIDON_WFBP_EACH && policy != POSEIDON_WFBP_SFB_LAST && policy != POSEIDON_WFBP_ALL_LAST &&
                  policy != POSEIDON_WFBP_SERIAL))
        return POSEIDON_ERR_INVALID_ARG;
    pool->wfbp_policy = policy;
    return POSEIDON_OK;
}

extern "C" int poseidon_pool_set_timing(poseidon_stream_pool* pool, int32_t enable)
{
    if (!pool)
        return POSEIDON_ERR_INVALID_ARG;
    pool->timing = enable != 0;
    return POSEIDON_OK;
}

extern "C" int poseidon_pool_launch_times(poseidon_stream_pool* pool, poseidon_launch_record* records,
                                          int32_t capacity, int32_t* count)
{
    if (!pool || !count || capacity < 0 || (capacity > 0 && !records) || !pool->t_valid)
        return POSEIDON_ERR_INVALID_ARG;
    const int32_t n = static_cast<int32_t>(pool->t_rec.size());
    *count = n;
    if (capacity < n)
        return POSEIDON_ERR_INVALID_ARG;
    for (int32_t r = 0; r < n; ++r) {
        float ms = 0.0f;
        if (hipEventSynchronize(pool->t_stop[r]) != hipSuccess ||
            hipEventElapsedTime(&ms, pool->t_start[r], pool->t_stop[r]) != hipSuccess)
            return POSEIDON_ERR_HIP;
        records[r] = pool->t_rec[static_cast<size_t>(r)];
        records[r].ms = ms;
    }
    return POSEIDON_OK;
}

extern "C" int poseidon_abi_version(void) { return POSEIDON_ABI_VERSION; }
