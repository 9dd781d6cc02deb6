// The C entry points of the single-call updates (include/poseidon.h): the
// argument checks, then the launchers of sf_apply.hip and ps_apply.hip.  Host
// code only; every check runs before anything is enqueued.
#include "common.h"

namespace poseidon {

int check_sf_args(const float* W, const float* U, const float* V,
                  int64_t M, int64_t N, int64_t K)
{
    if (M < 0 || N < 0 || K < 0)
        return POSEIDON_ERR_INVALID_ARG;
    if (M == 0 || N == 0 || K == 0)
        return POSEIDON_OK;
    if (!W || !U || !V)
        return POSEIDON_ERR_INVALID_ARG;
    if (M > INT64_MAX / 4 / N || K > INT64_MAX / 4 / M || K > INT64_MAX / 4 / N)
        return POSEIDON_ERR_INVALID_ARG;
    const int64_t wb = M * N * 4;
    if (overlaps(W, wb, U, K * M * 4) || overlaps(W, wb, V, K * N * 4))
        return POSEIDON_ERR_INVALID_ARG;
    return POSEIDON_OK;
}

int check_sf_momentum_args(const float* W, const float* buf, const float* U, const float* V,
                           int64_t M, int64_t N, int64_t K)
{
    if (M < 0 || N < 0 || K < 0)
        return POSEIDON_ERR_INVALID_ARG;
    if (M == 0 || N == 0)
        return POSEIDON_OK;
    if (!W || !buf || (K > 0 && (!U || !V)))
        return POSEIDON_ERR_INVALID_ARG;
    if (M > INT64_MAX / 4 / N || K > INT64_MAX / 4 / M || K > INT64_MAX / 4 / N)
        return POSEIDON_ERR_INVALID_ARG;
    const int64_t wb = M * N * 4;
    if (overlaps(W, wb, buf, wb) || overlaps(W, wb, U, K * M * 4) || overlaps(W, wb, V, K * N * 4) ||
        overlaps(buf, wb, U, K * M * 4) || overlaps(buf, wb, V, K * N * 4))
        return POSEIDON_ERR_INVALID_ARG;
    return POSEIDON_OK;
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

// Every layer as for poseidon_sf_apply, and no layer's W overlapping another
// layer's W, U or V (the layers of one launch are updated in parallel).
int check_sf_batch(const poseidon_sf_tensor* layers, int32_t count, int64_t K)
{
    if (count < 0 || (count > 0 && !layers) || K < 0)
        return POSEIDON_ERR_INVALID_ARG;
    std::vector<Span> writes, reads;
    for (int32_t i = 0; i < count; ++i) {
        const poseidon_sf_tensor& x = layers[i];
        const int rc = check_sf_args(x.W, x.U, x.V, x.M, x.N, K);
        if (rc != POSEIDON_OK)
            return rc;
        if (x.M == 0 || x.N == 0 || K == 0)
            continue;
        add_span(writes, x.W, x.M * x.N * 4);
        add_span(reads, x.U, K * x.M * 4);
        add_span(reads, x.V, K * x.N * 4);
    }
    return writes_collide(std::move(writes), reads) ? POSEIDON_ERR_INVALID_ARG : POSEIDON_OK;
}

static_assert(sizeof(poseidon_sf_tensor) == sizeof(SfTensor), "descriptor layout");

}  // namespace poseidon

extern "C" int poseidon_sf_apply_momentum(float* W, float* buf, const float* U, const float* V, int64_t M,
                                          int64_t N, int64_t K, float lr, float momentum, hipStream_t stream)
{
    const int rc = poseidon::check_sf_momentum_args(W, buf, U, V, M, N, K);
    if (rc != POSEIDON_OK || M == 0 || N == 0)
        return rc;
    return poseidon::launch_sf_apply_momentum(W, buf, U, V, M, N, K, lr, momentum, stream) == hipSuccess
               ? POSEIDON_OK
               : POSEIDON_ERR_HIP;
}

extern "C" int poseidon_sf_apply(float* W, const float* U, const float* V,
                                 int64_t M, int64_t N, int64_t K, float lr, hipStream_t stream)
{
    const int rc = poseidon::check_sf_args(W, U, V, M, N, K);
    if (rc != POSEIDON_OK || M == 0 || N == 0 || K == 0)
        return rc;
    return poseidon::launch_sf_apply(W, U, V, M, N, K, lr, stream) == hipSuccess
               ? POSEIDON_OK
               : POSEIDON_ERR_HIP;
}

extern "C" int poseidon_sf_set_arithmetic(int32_t arithmetic)
{
    if (arithmetic != POSEIDON_SF_BF16X6 && arithmetic != POSEIDON_SF_FP32)
        return POSEIDON_ERR_INVALID_ARG;
    poseidon::set_sf_arithmetic(arithmetic);
    return POSEIDON_OK;
}

extern "C" int32_t poseidon_sf_arithmetic(void) { return poseidon::sf_arithmetic(); }

extern "C" int poseidon_sf_apply_batch(const poseidon_sf_tensor* layers, int32_t count, int64_t K, float lr,
                                       hipStream_t stream)
{
    const int rc = poseidon::check_sf_batch(layers, count, K);
    if (rc != POSEIDON_OK)
        return rc;
    return poseidon::launch_sf_apply_batch(reinterpret_cast<const poseidon::SfTensor*>(layers), count, K, lr,
                                           stream) == hipSuccess
               ? POSEIDON_OK
               : POSEIDON_ERR_HIP;
}

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
    // The tensors of one launch are applied in parallel: no tensor may write
    // where another one reads or writes.
    std::vector<poseidon::Span> writes, reads;
    for (int32_t i = 0; i < count; ++i) {
        const poseidon_ps_tensor& x = tensors[i];
        if (x.n == 0)
            continue;
        poseidon::add_span(writes, x.W, x.n * 4);
        poseidon::add_span(writes, x.buf, x.n * 4);
        poseidon::add_span(reads, x.shards, x.n * 4 * static_cast<int64_t>(P));
    }
    if (poseidon::writes_collide(std::move(writes), reads))
        return POSEIDON_ERR_INVALID_ARG;
    static_assert(sizeof(poseidon_ps_tensor) == sizeof(poseidon::PsTensor), "descriptor layout");
    return poseidon::launch_ps_apply_batch(reinterpret_cast<const poseidon::PsTensor*>(tensors), count, P, lr,
                                           momentum, stream) == hipSuccess
               ? POSEIDON_OK
               : POSEIDON_ERR_HIP;
}
