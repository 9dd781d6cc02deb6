// The parameter server's KV store (Sec. 4.1 "Coordinator", "KV Store",
// "Managing Consistency"): the coordinator cuts the parameter-server tensors
// into fixed-size KV pairs hashed equally over the server nodes, and each
// server's store counts, per pair and iteration, the workers' updates that
// have arrived, applying a pair once every worker's update of it is there.
//
// The bookkeeping (layout, counts, the update pointers) is host state, as in
// the paper's KV store; the pairs of the tensors that one receive completes
// are applied by one kernel launch (per set of update pointers) on that
// receive's stream, summing the P workers' updates in worker order whatever
// the order they arrived in.  An
// update arrives either as a worker's whole tensor or inside the worker's
// message to this server (poseidon_kv_pack: its slices of this server's
// pairs, in pair order), and the apply reads each worker's values where they
// are.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <utility>
#include <vector>

#include "common.h"

struct poseidon_kv_store {
    int device = -1;
    int32_t P = 0;
    int32_t rank = 0;
    float lr = 0.f;
    float mu = 0.f;
    std::vector<poseidon_kv_tensor> tensors;
    std::vector<poseidon_kv_pair> pairs;           // the whole layout, all servers
    std::vector<std::vector<int32_t>> owned;        // per tensor: this server's pairs
    std::vector<int32_t> count;                     // per pair, this iteration
    std::vector<std::vector<const float*>> grads;   // per tensor: worker p's update (or NULL)
    std::vector<uint64_t> from_msg;                 // per tensor: bit p set when worker p's came in a message
    std::vector<int64_t> msg_off;                   // per pair held here: its first element in a message
    int64_t msg_len = 0;                            // elements of a message to this server
};

namespace {

// Number of pairs of the layout, or -1 when an argument is invalid or the
// count exceeds INT32_MAX.
int64_t count_pairs(const int64_t* sizes, int32_t count, int64_t pair_elems)
{
    int64_t total = 0;
    for (int32_t t = 0; t < count; ++t) {
        if (sizes[t] < 0)
            return -1;
        total += sizes[t] / pair_elems + (sizes[t] % pair_elems != 0);
        if (total > INT32_MAX)
            return -1;
    }
    return total;
}

// Enqueue the apply of the pairs held by the store of the tensors in `ts`
// (their counts have reached P): one launch for all the tensors whose P
// update pointers are the same (every update came in the same messages, the
// usual case), one more for each other set of pointers.
hipError_t apply_tensors(poseidon_kv_store* st, const std::vector<int32_t>& ts, hipStream_t stream)
{
    std::vector<bool> done(ts.size(), false);
    std::vector<poseidon::KvApplyRange> ranges;
    for (size_t a = 0; a < ts.size(); ++a) {
        if (done[a])
            continue;
        const size_t ta = static_cast<size_t>(ts[a]);
        ranges.clear();
        for (size_t b = a; b < ts.size(); ++b) {
            const size_t tb = static_cast<size_t>(ts[b]);
            if (done[b] || st->grads[tb] != st->grads[ta] || st->from_msg[tb] != st->from_msg[ta])
                continue;
            done[b] = true;
            const poseidon_kv_tensor& x = st->tensors[tb];
            for (int32_t j : st->owned[tb]) {
                const poseidon_kv_pair& q = st->pairs[static_cast<size_t>(j)];
                ranges.push_back(poseidon::KvApplyRange{x.W, x.buf, q.offset, q.length,
                                                         st->msg_off[static_cast<size_t>(j)] - q.offset});
            }
        }
        const hipError_t e = poseidon::launch_kv_apply(ranges.data(), static_cast<int32_t>(ranges.size()),
                                                       st->grads[ta].data(), st->from_msg[ta], st->P, st->lr,
                                                       st->mu, stream);
        if (e != hipSuccess)
            return e;
    }
    return hipSuccess;
}

void fill_layout(const int64_t* sizes, int32_t count, int64_t pair_elems, int32_t P, poseidon_kv_pair* out)
{
    int64_t j = 0;
    for (int32_t t = 0; t < count; ++t) {
        for (int64_t off = 0; off < sizes[t]; off += pair_elems, ++j) {
            poseidon_kv_pair& q = out[j];
            q.tensor = t;
            q.server = static_cast<int32_t>(j % P);
            q.offset = off;
            q.length = sizes[t] - off < pair_elems ? sizes[t] - off : pair_elems;
        }
    }
}

}  // namespace

extern "C" int poseidon_kv_layout(const int64_t* sizes, int32_t count, int64_t pair_elems, int32_t P,
                                  poseidon_kv_pair* pairs, int32_t capacity, int32_t* npairs)
{
    if (!npairs || count < 0 || (count > 0 && !sizes) || pair_elems < 1 || P < 1 || capacity < 0 ||
        (capacity > 0 && !pairs))
        return POSEIDON_ERR_INVALID_ARG;
    const int64_t total = count_pairs(sizes, count, pair_elems);
    if (total < 0)
        return POSEIDON_ERR_INVALID_ARG;
    *npairs = static_cast<int32_t>(total);
    if (capacity < total)
        return pairs == nullptr && capacity == 0 ? POSEIDON_OK : POSEIDON_ERR_INVALID_ARG;
    fill_layout(sizes, count, pair_elems, P, pairs);
    return POSEIDON_OK;
}

extern "C" int poseidon_kv_create(const poseidon_kv_tensor* tensors, int32_t count, int64_t pair_elems, int32_t P,
                                  int32_t rank, float lr, float momentum, poseidon_kv_store** out)
{
    using poseidon::overlaps;
    if (!out || count < 0 || (count > 0 && !tensors) || pair_elems < 1 || P < 1 || P > poseidon::KV_MAX_P ||
        rank < 0 || rank >= P)
        return POSEIDON_ERR_INVALID_ARG;
    *out = nullptr;
    std::vector<int64_t> sizes(static_cast<size_t>(count));
    for (int32_t t = 0; t < count; ++t) {
        const poseidon_kv_tensor& x = tensors[t];
        if (x.n < 0 || (x.n > 0 && !x.W) || x.n > INT64_MAX / 4)
            return POSEIDON_ERR_INVALID_ARG;
        if (overlaps(x.W, x.n * 4, x.buf, x.n * 4))
            return POSEIDON_ERR_INVALID_ARG;
        sizes[static_cast<size_t>(t)] = x.n;
    }
    // No two arrays of the store may overlap: one launch may apply pairs of
    // several tensors at once.
    std::vector<std::pair<uintptr_t, uintptr_t>> spans;
    for (int32_t t = 0; t < count; ++t) {
        const poseidon_kv_tensor& x = tensors[t];
        if (x.n == 0)
            continue;
        spans.emplace_back(reinterpret_cast<uintptr_t>(x.W), reinterpret_cast<uintptr_t>(x.W) + x.n * 4);
        if (x.buf)
            spans.emplace_back(reinterpret_cast<uintptr_t>(x.buf), reinterpret_cast<uintptr_t>(x.buf) + x.n * 4);
    }
    std::sort(spans.begin(), spans.end());
    for (size_t i = 1; i < spans.size(); ++i)
        if (spans[i].first < spans[i - 1].second)
            return POSEIDON_ERR_INVALID_ARG;
    const int64_t total = count_pairs(sizes.data(), count, pair_elems);
    if (total < 0)
        return POSEIDON_ERR_INVALID_ARG;
    auto* st = new poseidon_kv_store;
    if (hipGetDevice(&st->device) != hipSuccess) {
        delete st;
        return POSEIDON_ERR_HIP;
    }
    st->P = P;
    st->rank = rank;
    st->lr = lr;
    st->mu = momentum;
    st->tensors.assign(tensors, tensors + count);
    st->pairs.resize(static_cast<size_t>(total));
    fill_layout(sizes.data(), count, pair_elems, P, st->pairs.data());
    st->owned.resize(static_cast<size_t>(count));
    for (int32_t j = 0; j < static_cast<int32_t>(total); ++j)
        if (st->pairs[static_cast<size_t>(j)].server == rank)
            st->owned[static_cast<size_t>(st->pairs[static_cast<size_t>(j)].tensor)].push_back(j);
    st->count.assign(static_cast<size_t>(total), 0);
    st->grads.assign(static_cast<size_t>(count), std::vector<const float*>(static_cast<size_t>(P), nullptr));
    st->from_msg.assign(static_cast<size_t>(count), 0);
    st->msg_off.assign(static_cast<size_t>(total), 0);
    for (int32_t j = 0; j < static_cast<int32_t>(total); ++j)
        if (st->pairs[static_cast<size_t>(j)].server == rank) {
            st->msg_off[static_cast<size_t>(j)] = st->msg_len;
            st->msg_len += st->pairs[static_cast<size_t>(j)].length;
        }
    *out = st;
    return POSEIDON_OK;
}

extern "C" int poseidon_kv_destroy(poseidon_kv_store* store)
{
    delete store;
    return POSEIDON_OK;
}

extern "C" int poseidon_kv_begin(poseidon_kv_store* store)
{
    if (!store)
        return POSEIDON_ERR_INVALID_ARG;
    for (int32_t& c : store->count)
        c = 0;
    for (auto& g : store->grads)
        for (const float*& p : g)
            p = nullptr;
    for (uint64_t& m : store->from_msg)
        m = 0;
    return POSEIDON_OK;
}

extern "C" int poseidon_kv_receive(poseidon_kv_store* store, int32_t worker, int32_t tensor, const float* grad,
                                   hipStream_t stream)
{
    using poseidon::overlaps;
    if (!store || worker < 0 || worker >= store->P || tensor < 0 ||
        tensor >= static_cast<int32_t>(store->tensors.size()))
        return POSEIDON_ERR_INVALID_ARG;
    const poseidon_kv_tensor& x = store->tensors[static_cast<size_t>(tensor)];
    std::vector<const float*>& g = store->grads[static_cast<size_t>(tensor)];
    // An update is recorded as a non-NULL pointer; a zero-size tensor's
    // update may be NULL and is then recorded as its W (never read).
    const float* rec = x.n > 0 ? grad : reinterpret_cast<const float*>(&x);
    if ((x.n > 0 && !grad) || g[static_cast<size_t>(worker)] != nullptr ||
        overlaps(grad, x.n * 4, x.W, x.n * 4) || overlaps(grad, x.n * 4, x.buf, x.n * 4))
        return POSEIDON_ERR_INVALID_ARG;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess)
        return POSEIDON_ERR_HIP;
    if (dev != store->device)
        return POSEIDON_ERR_INVALID_ARG;
    g[static_cast<size_t>(worker)] = rec;
    const std::vector<int32_t>& mine = store->owned[static_cast<size_t>(tensor)];
    if (mine.empty())
        return 0;
    bool complete = true;
    for (int32_t j : mine)
        complete = ++store->count[static_cast<size_t>(j)] == store->P && complete;
    if (!complete)
        return 0;
    if (apply_tensors(store, std::vector<int32_t>{tensor}, stream) != hipSuccess)
        return POSEIDON_ERR_HIP;
    return static_cast<int32_t>(mine.size());
}

extern "C" int poseidon_kv_receive_message(poseidon_kv_store* store, int32_t worker, const float* message,
                                           hipStream_t stream)
{
    using poseidon::overlaps;
    if (!store || worker < 0 || worker >= store->P || (store->msg_len > 0 && !message))
        return POSEIDON_ERR_INVALID_ARG;
    const size_t T = store->tensors.size();
    for (size_t t = 0; t < T; ++t) {   // nothing of this worker's may have arrived yet this iteration
        const poseidon_kv_tensor& x = store->tensors[t];
        if (store->grads[t][static_cast<size_t>(worker)] != nullptr ||
            overlaps(message, store->msg_len * 4, x.W, x.n * 4) || overlaps(message, store->msg_len * 4, x.buf, x.n * 4))
            return POSEIDON_ERR_INVALID_ARG;
    }
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess)
        return POSEIDON_ERR_HIP;
    if (dev != store->device)
        return POSEIDON_ERR_INVALID_ARG;
    int32_t done = 0;
    std::vector<int32_t> complete_ts;   // applied together after the counts
    for (size_t t = 0; t < T; ++t) {
        const poseidon_kv_tensor& x = store->tensors[t];
        // The message stands for this worker's update of every tensor; a
        // tensor with no pair here is recorded with a marker (never read).
        const bool held = !store->owned[t].empty();
        store->grads[t][static_cast<size_t>(worker)] = held ? message : reinterpret_cast<const float*>(&x);
        if (!held)
            continue;
        store->from_msg[t] |= uint64_t{1} << worker;
        bool complete = true;
        for (int32_t j : store->owned[t])
            complete = ++store->count[static_cast<size_t>(j)] == store->P && complete;
        if (complete) {
            complete_ts.push_back(static_cast<int32_t>(t));
            done += static_cast<int32_t>(store->owned[t].size());
        }
    }
    if (!complete_ts.empty() && apply_tensors(store, complete_ts, stream) != hipSuccess)
        return POSEIDON_ERR_HIP;
    return done;
}

extern "C" int poseidon_kv_message_size(const poseidon_kv_store* store, int64_t* elems)
{
    if (!store || !elems)
        return POSEIDON_ERR_INVALID_ARG;
    *elems = store->msg_len;
    return POSEIDON_OK;
}

extern "C" int poseidon_kv_pack(const int64_t* sizes, const float* const* grads, int32_t count, int64_t pair_elems,
                                int32_t P, int32_t server, float* message, int64_t capacity, int64_t* length,
                                hipStream_t stream)
{
    using poseidon::overlaps;
    if (!length || count < 0 || (count > 0 && (!sizes || !grads)) || pair_elems < 1 || P < 1 || server < -1 ||
        server >= P || capacity < 0)
        return POSEIDON_ERR_INVALID_ARG;
    const int64_t total = count_pairs(sizes, count, pair_elems);
    if (total < 0)
        return POSEIDON_ERR_INVALID_ARG;
    std::vector<poseidon_kv_pair> pairs(static_cast<size_t>(total));
    fill_layout(sizes, count, pair_elems, P, pairs.data());
    std::vector<const float*> src;
    std::vector<int64_t> dst, len;
    int64_t n = 0;
    for (int32_t to = (server < 0 ? 0 : server); to <= (server < 0 ? P - 1 : server); ++to)
        for (const poseidon_kv_pair& q : pairs)
            if (q.server == to) {
                src.push_back(grads[q.tensor] + q.offset);
                dst.push_back(n);
                len.push_back(q.length);
                n += q.length;
            }
    *length = n;
    if (message == nullptr && capacity == 0)
        return POSEIDON_OK;                       // size query
    if (capacity < n || (n > 0 && !message))
        return POSEIDON_ERR_INVALID_ARG;
    for (int32_t t = 0; t < count; ++t)
        if (sizes[t] > 0 && (!grads[t] || overlaps(message, n * 4, grads[t], sizes[t] * 4)))
            return POSEIDON_ERR_INVALID_ARG;
    if (n == 0)
        return POSEIDON_OK;
    return poseidon::launch_kv_pack(src.data(), dst.data(), len.data(), static_cast<int32_t>(src.size()), message,
                                    stream) == hipSuccess
               ? POSEIDON_OK
               : POSEIDON_ERR_HIP;
}

extern "C" int poseidon_kv_pair_count(const poseidon_kv_store* store, int32_t pair, int32_t* count)
{
    if (!store || !count || pair < 0 || pair >= static_cast<int32_t>(store->pairs.size()))
        return POSEIDON_ERR_INVALID_ARG;
    *count = store->count[static_cast<size_t>(pair)];
    return POSEIDON_OK;
}
