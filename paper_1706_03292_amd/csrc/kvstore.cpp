// The parameter server's KV store (Sec. 4.1 "Coordinator", "KV Store",
// "Managing Consistency"): the coordinator cuts the parameter-server tensors
// into fixed-size KV pairs hashed equally over the server nodes, and each
// server's store counts, per pair and iteration, the workers' updates that
// have arrived, applying a pair once every worker's update of it is there.
//
// The bookkeeping (layout, counts, the update pointers) is host state, as in
// the paper's KV store; the apply of a completed tensor's pairs is one kernel
// launch on the stream of the receive that completed them, summing the P
// workers' updates in worker order whatever the order they arrived in.
#include <hip/hip_runtime.h>

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
    std::vector<int64_t> off, len;
    for (int32_t j : mine) {
        off.push_back(store->pairs[static_cast<size_t>(j)].offset);
        len.push_back(store->pairs[static_cast<size_t>(j)].length);
    }
    const hipError_t e = poseidon::launch_kv_apply(x.W, x.buf, g.data(), store->P, off.data(), len.data(),
                                                   static_cast<int32_t>(mine.size()), store->lr,
                                                   x.buf ? store->mu : 0.0f, stream);
    if (e != hipSuccess)
        return POSEIDON_ERR_HIP;
    return static_cast<int32_t>(mine.size());
}

extern "C" int poseidon_kv_pair_count(const poseidon_kv_store* store, int32_t pair, int32_t* count)
{
    if (!store || !count || pair < 0 || pair >= static_cast<int32_t>(store->pairs.size()))
        return POSEIDON_ERR_INVALID_ARG;
    *count = store->count[static_cast<size_t>(pair)];
    return POSEIDON_OK;
}
