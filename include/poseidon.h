/*
 * poseidon.h -- C ABI of libposeidon.so: one node's per-layer gradient
 * synchronisation compute from Poseidon (Zhang et al., "Poseidon: An Efficient
 * Communication Architecture for Distributed Deep Learning on GPU Clusters",
 * arXiv 1706.03292), for AMD Instinct MI355X (gfx950).
 *
 * The paper synchronises each layer either through a parameter server (dense
 * gradients pushed to server shards, summed and applied there) or by
 * sufficient-factor broadcasting (the rank-1 factors u, v of each sample's
 * fully-connected gradient are broadcast and every node rebuilds the
 * gradient), choosing per layer by the bytes each scheme would move (hybrid
 * communication).  This library performs the node-local arithmetic of both
 * schemes on payloads that are already in device memory, and the choice.
 *
 * General conventions
 *  - All array arguments are device pointers to fp32 data owned by the caller.
 *    The library allocates no device memory and keeps no pointer past a call,
 *    except a KV store, which keeps its tensors' pointers for its lifetime and
 *    each received update's pointer until the work it triggers has been
 *    enqueued (and the caller keeps that memory valid until the work has run).
 *  - Work is enqueued asynchronously on `stream` (0 = the null stream).
 *    Argument errors are detected and reported synchronously, before anything
 *    is enqueued; a fault inside a kernel surfaces at the next synchronisation
 *    of the stream, as for any HIP kernel.
 *  - Empty work (a zero dimension) is a successful no-op.
 *  - Any 4-byte alignment is accepted; 16-byte aligned arrays whose row length
 *    is a multiple of 4 take the vectorised fast path.
 *  - Outputs must not overlap inputs (checked: overlapping ranges are an
 *    argument error).
 *  - The functions are thread-safe and keep no mutable global state, except the
 *    stream pool and KV store objects, which belong to their creator and must
 *    not be used by two threads at once.
 *  - Results are deterministic: the same inputs give bit-identical outputs.
 */
#ifndef POSEIDON_H
#define POSEIDON_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define POSEIDON_OK               0
#define POSEIDON_ERR_INVALID_ARG (-1)  /* bad size, NULL with nonzero size, P < 1, overlap */
#define POSEIDON_ERR_HIP         (-2)  /* a HIP runtime call or kernel launch failed */
#define POSEIDON_ERR_PAYLOAD     (-3)  /* the chosen scheme's payload was not supplied */

/* Synchronisation schemes (Alg. 1 returns one of these). */
#define POSEIDON_PS   0
#define POSEIDON_SFB  1
#define POSEIDON_ADAM 2   /* Adam's scheme (cost model only): SFs to one server, the matrix back */

/* Tensor kinds: only fully-connected weights can be synchronised by SFB;
 * convolution kernels, biases and normalisation vectors always use the
 * parameter server (Sec. 3.2, Alg. 1). */
#define POSEIDON_KIND_FC     0
#define POSEIDON_KIND_OTHER  1

/* Schedules of poseidon_sync_iteration_wfbp (poseidon_pool_set_wfbp_policy). */
#define POSEIDON_WFBP_ALL_LAST 0   /* every update after every ready event, on the pool's streams */
#define POSEIDON_WFBP_SFB_LAST 1   /* PS applies on their own events, SFB rebuilds after every event */
#define POSEIDON_WFBP_EACH     2   /* every update on its own ready event (Alg. 2) */
#define POSEIDON_WFBP_SERIAL   3   /* the caller's stream waits for every ready event, then the plain
                                      iteration on it: the serial order (default) */

/* Arithmetic of the SF reconstruction's contraction (poseidon_sf_set_arithmetic). */
#define POSEIDON_SF_BF16X6 0   /* split-bf16 products, fp32 accumulation (default) */
#define POSEIDON_SF_FP32   1   /* fp32 matrix-core products, fp32 accumulation */

/*
 * Sufficient-factor reconstruction fused with the SGD step (Sec. 2.1
 * "Sufficient Factor Broadcasting"; Eq. 2; Eq. 1), the work of a syncer's
 * Move(CPU2GPU) for an SFB layer (Sec. 4.1, Table 2):
 *
 *     W[m][n] <- W[m][n] - lr * sum_{k<K} U[k][m] * V[k][n]
 *
 * W : M x N row-major, updated in place (M = fan-out, the length of u;
 *     N = fan-in, the length of v).
 * U : K x M row-major; row k is the factor u_k.  V : K x N row-major; row k is
 *     v_k.  K = P * B is the number of factor pairs gathered from the P
 *     workers of per-worker batch B, this node's own included; the rows of
 *     worker p are contiguous.
 * The sum is accumulated in fp32 on the matrix cores and W is read and written
 * exactly once.  lr is applied as given (no 1/(P*B) scaling).  The products
 * are formed as poseidon_sf_set_arithmetic last chose: by default each fp32
 * operand is split exactly into three bf16 parts and six of their nine
 * products are accumulated (fp32-grade: the three left out are below 2^-23
 * of the product); POSEIDON_SF_FP32 uses the fp32 matrix-core product.
 * Operands whose byte offsets exceed 32 bits always take the fp32 product.
 * Returns POSEIDON_OK, POSEIDON_ERR_INVALID_ARG (negative size, NULL pointer
 * with nonzero size, W overlapping U or V) or POSEIDON_ERR_HIP.
 */
int poseidon_sf_apply(float* W, const float* U, const float* V,
                      int64_t M, int64_t N, int64_t K, float lr,
                      hipStream_t stream);

/*
 * The same reconstruction for an FC layer that keeps a heavy-ball momentum
 * buffer (the update rule of poseidon_ps_apply, with the reconstructed
 * gradient in place of the shard sum; Eq. 2 for the gradient):
 *
 *     buf[m][n] <- momentum * buf[m][n] + sum_{k<K} U[k][m] * V[k][n]
 *     W[m][n]   <- W[m][n] - lr * buf[m][n]
 *
 * buf: M x N row-major like W, caller-owned, updated in place; W and buf are
 * each read and written once (16 M N bytes).  K = 0 is a step on the buffer
 * alone (U and V may then be NULL).  Layouts and accumulation as for
 * poseidon_sf_apply.  Returns POSEIDON_OK, POSEIDON_ERR_INVALID_ARG (as
 * poseidon_sf_apply; also NULL buf with M*N > 0, or buf overlapping W, U or
 * V) or POSEIDON_ERR_HIP.
 */
int poseidon_sf_apply_momentum(float* W, float* buf, const float* U, const float* V,
                               int64_t M, int64_t N, int64_t K, float lr, float momentum,
                               hipStream_t stream);

/*
 * Chooses how every SF reconstruction enqueued after the call, from any
 * thread, forms its products (the sums, the update and the layouts are the
 * same): POSEIDON_SF_BF16X6 (the default) splits each fp32 operand x exactly
 * into bf16 parts h + m + l (h and m rounded to nearest, l the remainder,
 * which has at most 8 significant bits) and accumulates the six products
 * h*h, h*m, m*h, h*l, l*h and m*m in fp32 on the bf16 matrix cores (the six-
 * product split of Henry, Tang and Heinecke, ARITH 2019); POSEIDON_SF_FP32
 * accumulates the fp32 matrix-core products.  The two agree to fp32
 * rounding on finite operands below 3.39e38 in magnitude (the largest bf16);
 * an infinite or larger operand makes the outputs it reaches NaN with the
 * split products (inf or NaN with the fp32 ones).  The choice is process-wide
 * and does not change which scheme Alg. 1 picks.  Returns POSEIDON_OK or
 * POSEIDON_ERR_INVALID_ARG (an unknown value; the setting is unchanged).
 */
int poseidon_sf_set_arithmetic(int32_t arithmetic);

/* The current choice of poseidon_sf_set_arithmetic. */
int32_t poseidon_sf_arithmetic(void);

/* One fully-connected layer of a grouped SF reconstruction. */
typedef struct poseidon_sf_tensor {
    float*       W;   /* M x N row-major, updated in place */
    const float* U;   /* K x M row-major */
    const float* V;   /* K x N row-major */
    int64_t      M;
    int64_t      N;
} poseidon_sf_tensor;

/*
 * poseidon_sf_apply for several FC layers that share K (the same P workers and
 * batch B) in one pass: each layer is updated exactly as by
 * poseidon_sf_apply(W, U, V, M, N, K, lr).  Their tiles form one work list
 * (in the order given), so the GPU is never left half idle between layers;
 * layers whose rows are too long for the grouped kernel, and groups too small
 * to fill the GPU, are launched one by one instead.  The W arrays must not
 * overlap each other or any U, V.  All layers are validated before anything
 * is enqueued.  Returns POSEIDON_OK, POSEIDON_ERR_INVALID_ARG (as for
 * poseidon_sf_apply, for any layer; count < 0; NULL layers with count > 0;
 * overlapping W) or POSEIDON_ERR_HIP.
 */
int poseidon_sf_apply_batch(const poseidon_sf_tensor* layers, int32_t count, int64_t K, float lr,
                            hipStream_t stream);

/*
 * Parameter-server aggregation and apply: the KV store's Receive of all P
 * workers' updates followed by their application (Sec. 2.1 "Parameter
 * Server"; Sec. 4.1 "KV Store", "Managing Consistency"), with heavy-ball
 * momentum:
 *
 *     s_i   = sum_{p<P} shards[p*n + i]          (p in increasing order)
 *     buf_i <- momentum * buf_i + s_i
 *     W_i   <- W_i - lr * buf_i
 *
 * shards : P x n, shard p at offset p*n.  W, buf : n values, updated in place.
 * buf == NULL is allowed only with momentum == 0 and gives W_i -= lr * s_i.
 * Returns POSEIDON_OK, POSEIDON_ERR_INVALID_ARG (P < 1, n < 0, NULL pointer
 * with n > 0, momentum != 0 without buf, overlapping arrays) or
 * POSEIDON_ERR_HIP.
 */
int poseidon_ps_apply(float* W, const float* shards, int32_t P, int64_t n,
                      float lr, float momentum, float* buf,
                      hipStream_t stream);

/* One dense tensor of a batched parameter-server apply. */
typedef struct poseidon_ps_tensor {
    float*       W;       /* n values, updated in place */
    const float* shards;  /* P x n, shard p at offset p*n */
    float*       buf;     /* momentum buffer (n values) or NULL for plain SGD */
    int64_t      n;
} poseidon_ps_tensor;

/*
 * poseidon_ps_apply for many tensors at once: a KV store applying every pair
 * it received in one pass (Sec. 4.1 "KV Store").  Each tensor is updated
 * exactly as by poseidon_ps_apply(W, shards, P, n, lr, buf ? momentum : 0,
 * buf); tensors with n = 0 are skipped.  The work is issued as one launch per
 * group of up to 48 tensors of the same kind (with / without buffer), so that
 * small tensors do not each pay a kernel launch.  All tensors are validated
 * before anything is enqueued; the tensors are applied in parallel, so no
 * tensor's W or buf may overlap another tensor's W, buf or shards (tensors may
 * share shards).  Returns POSEIDON_OK, POSEIDON_ERR_INVALID_ARG (as for
 * poseidon_ps_apply, for any tensor; count < 0; NULL tensors with count > 0;
 * a W or buf overlapping another tensor's arrays) or POSEIDON_ERR_HIP.
 */
int poseidon_ps_apply_batch(const poseidon_ps_tensor* tensors, int32_t count, int32_t P,
                            float lr, float momentum, hipStream_t stream);

/*
 * KV store (Sec. 4.1 "Coordinator", "KV Store", "Managing Consistency").
 *
 * The parameter-server tensors are cut into KV pairs of a fixed small size
 * (2 MB in the paper) that the coordinator hashes equally over the P server
 * nodes, so that every server carries the same share of the traffic instead
 * of one server per tensor (Sec. 5.2).  Each server's KV store counts, per
 * pair and per iteration, the workers' updates that have arrived, and applies
 * a pair -- the sum of the P updates, then the momentum SGD step of
 * poseidon_ps_apply -- once its count equals the number of workers, after
 * which the pair is ready to be sent back.  On one GPU a store is one node's
 * server role: it updates only the pairs hashed to its rank, in place in the
 * caller's full parameter tensors.
 */

/* One KV pair. */
typedef struct poseidon_kv_pair {
    int32_t tensor;   /* index into the tensor list */
    int32_t server;   /* rank of the KV store that holds the pair */
    int64_t offset;   /* first element of the pair in its tensor */
    int64_t length;   /* elements: pair_elems, or fewer for a tensor's last pair */
} poseidon_kv_pair;

/*
 * The coordinator's partition of `count` tensors of sizes[t] elements: each
 * tensor, in order, is cut into consecutive pairs of pair_elems elements (the
 * last pair of a tensor may be shorter; a pair never spans two tensors, as
 * every layer has a syncer of its own), and the j-th pair overall goes to
 * server j mod P (pair counts per server differ by at most one; the pieces of
 * a big tensor land on consecutive servers).  Writes the pairs in order to
 * pairs[0 .. *npairs) when capacity suffices (pairs may be NULL with capacity
 * 0 to query *npairs).  Host-only.  Returns POSEIDON_OK or
 * POSEIDON_ERR_INVALID_ARG (count < 0, a negative size, pair_elems < 1,
 * P < 1, NULL sizes or npairs, more than 2^31 - 1 pairs, capacity too small
 * -- *npairs is still set).
 */
int poseidon_kv_layout(const int64_t* sizes, int32_t count, int64_t pair_elems, int32_t P,
                       poseidon_kv_pair* pairs, int32_t capacity, int32_t* npairs);

/* One parameter-server tensor of a KV store: W (n values) and its momentum
 * buffer (n values, or NULL for plain SGD), caller-owned device memory that
 * must stay valid for the store's lifetime. */
typedef struct poseidon_kv_tensor {
    float*  W;
    float*  buf;
    int64_t n;
} poseidon_kv_tensor;

typedef struct poseidon_kv_store poseidon_kv_store;

/*
 * Create the KV store of server `rank` (0 .. P-1) over the given tensors,
 * laid out as by poseidon_kv_layout(sizes, count, pair_elems, P), with the
 * step's lr and momentum (used only for tensors that have a buf).  The store
 * keeps the tensor list, the layout, one count per pair and one update
 * pointer per (tensor, worker); it allocates no device memory.  All counts
 * start at 0 (as after poseidon_kv_begin).  P <= 64.  No two of the
 * tensors' W and buf arrays may overlap (one launch may apply pairs of several
 * tensors).  Returns POSEIDON_OK, POSEIDON_ERR_INVALID_ARG (bad sizes, NULL W
 * with n > 0, overlapping arrays, rank outside 0..P-1, P outside 1..64,
 * count < 0, NULL out) or POSEIDON_ERR_HIP.
 */
int poseidon_kv_create(const poseidon_kv_tensor* tensors, int32_t count, int64_t pair_elems, int32_t P,
                       int32_t rank, float lr, float momentum, poseidon_kv_store** out);

/* Destroy a store (no device work is pending on its behalf once the streams
 * its receives used have drained).  NULL is a no-op. */
int poseidon_kv_destroy(poseidon_kv_store* store);

/* Start of an iteration: every pair's count back to 0, every recorded update
 * forgotten.  Returns POSEIDON_OK or POSEIDON_ERR_INVALID_ARG. */
int poseidon_kv_begin(poseidon_kv_store* store);

/*
 * Worker `worker`'s update of tensor `tensor` has arrived: grad holds the
 * tensor's n gradient values (device memory, caller-owned, not modified; only
 * the slices of this store's pairs are read).  The count of every pair of the
 * tensor that this store holds goes up by one.  When those counts reach P,
 * the pairs are applied on `stream`: for every element i of them
 *
 *     s_i = sum_{p<P} grad_p[i]  (p in increasing worker order, whatever the
 *                                 order of arrival; fp32)
 *     buf_i <- momentum * buf_i + s_i ;  W_i <- W_i - lr * buf_i
 *
 * (without buf: W_i <- W_i - lr * s_i), the arithmetic of poseidon_ps_apply.
 * The P update pointers of the tensor must stay valid, and their data
 * complete in the order of `stream`, until that work has run.  Returns the
 * number of pairs this call completed (their counts reached P), or
 * POSEIDON_ERR_INVALID_ARG (NULL store; worker or tensor out of range; NULL
 * grad with n > 0; grad overlapping W or buf; this worker's update of the
 * tensor already received in this iteration -- nothing changes then) or
 * POSEIDON_ERR_HIP.
 */
int poseidon_kv_receive(poseidon_kv_store* store, int32_t worker, int32_t tensor, const float* grad,
                        hipStream_t stream);

/*
 * Worker `worker`'s message to this store has arrived: its slices of every
 * pair this store holds, in pair order, concatenated (as poseidon_kv_pack
 * makes it; poseidon_kv_message_size elements of device memory, caller-owned,
 * not modified).  It stands for that worker's update of every tensor, as if
 * poseidon_kv_receive had been called for each: every count of this store's
 * pairs goes up by one, and the tensors whose pairs reach P are applied on
 * `stream` (together: one launch for the tensors whose P updates all arrived
 * the same way), reading every worker's values where they arrived (a message
 * or a whole-tensor update), summed in worker order.  The message must stay valid,
 * and its data complete in the order of `stream`, until that work has run.
 * Returns the number of pairs completed, or POSEIDON_ERR_INVALID_ARG (NULL
 * store; worker out of range; NULL message when this store holds pairs; a
 * message overlapping a W or buf; any update of this worker already received
 * in this iteration -- nothing changes then) or POSEIDON_ERR_HIP.
 */
int poseidon_kv_receive_message(poseidon_kv_store* store, int32_t worker, const float* message,
                                hipStream_t stream);

/* The number of values in a message to this store (the total length of the
 * pairs it holds).  Returns POSEIDON_OK or POSEIDON_ERR_INVALID_ARG. */
int poseidon_kv_message_size(const poseidon_kv_store* store, int64_t* elems);

/*
 * The worker side of a push (Sec. 4.1 "KV Store"): one worker's updates of
 * the `count` tensors (grads[t], sizes[t] values each, device memory), cut as
 * poseidon_kv_layout(sizes, count, pair_elems, P) cuts them, and the slices of
 * the pairs held by `server` copied one after another, in pair order, into
 * `message` (device memory, capacity values) on `stream` -- the message that
 * worker sends to that server.  server == -1 writes every server's message,
 * one after another in server order, in one pass.  *length receives the
 * length written; message == NULL with capacity 0 only queries it.  Returns
 * POSEIDON_OK or POSEIDON_ERR_INVALID_ARG (bad layout arguments, server
 * outside -1..P-1, NULL
 * grads[t] with sizes[t] > 0, capacity too small, message overlapping an
 * update) or POSEIDON_ERR_HIP.
 */
int poseidon_kv_pack(const int64_t* sizes, const float* const* grads, int32_t count, int64_t pair_elems, int32_t P,
                     int32_t server, float* message, int64_t capacity, int64_t* length, hipStream_t stream);

/* The store's count of pair `pair` (an index into its layout) in the current
 * iteration: the number of workers whose update of it has arrived, or 0 for
 * a pair held by another server.  A pair whose count equals P has been
 * applied (enqueued) and may be sent.  Returns POSEIDON_OK or
 * POSEIDON_ERR_INVALID_ARG. */
int poseidon_kv_pair_count(const poseidon_kv_store* store, int32_t pair, int32_t* count);

/*
 * Coordinator.BestScheme for a fully-connected M x N layer (Alg. 1; Table 1)
 * on a cluster of P nodes that are each both worker and server (P1 = P2 = P),
 * per-worker batch B:
 *
 *     SFB  iff  2 B (P-1) (M+N)  <=  2 M N (P1 + P2 - 2) / P2
 *
 * evaluated exactly in integers (both sides multiplied by P2).  A tie goes to
 * SFB; P = 1 is a tie (nothing is sent either way).  Host-only; no device work.
 * Returns POSEIDON_SFB, POSEIDON_PS, or POSEIDON_ERR_INVALID_ARG (negative
 * M, N or B; P < 1; any argument above 2^31 - 1).
 */
int poseidon_hybcomm_choose(int64_t M, int64_t N, int64_t B, int64_t P);

/*
 * Table 1's per-node traffic of one synchronisation of an M x N FC layer, in
 * values (not bytes), multiplied by P2 so that it stays an integer:
 *   *ps_x_p2  = 2 M N (P1 + P2 - 2)   (a node that is both server and worker)
 *   *sfb_x_p2 = 2 B (P1 - 1) (M + N) P2
 * Host-only.  Returns POSEIDON_OK or POSEIDON_ERR_INVALID_ARG (negative
 * sizes, P1 or P2 < 1, arguments above 2^31 - 1, NULL outputs, or a result
 * that does not fit in int64).
 */
int poseidon_hybcomm_cost(int64_t M, int64_t N, int64_t B, int64_t P1, int64_t P2,
                          int64_t* ps_x_p2, int64_t* sfb_x_p2);

/*
 * Table 1's Adam row (Sec. 3.2): workers send their B factor pairs to the
 * one server holding the layer, which sends the whole rebuilt M x N matrix
 * back to every worker.  Per-node traffic in values, multiplied by P2 like
 * poseidon_hybcomm_cost:
 *   *server_x_p2 = (P1 M N + P1 B (M + N)) P2    (the holder, not a worker)
 *   *worker_x_p2 = (B (M + N) + M N) P2          (a worker, not the holder)
 *   *both_x_p2   = (P1 - 1)(M N + B (M + N)) P2  (the holder that is also a worker)
 * Host-only.  Returns POSEIDON_OK or POSEIDON_ERR_INVALID_ARG (as
 * poseidon_hybcomm_cost).
 */
int poseidon_hybcomm_cost_adam(int64_t M, int64_t N, int64_t B, int64_t P1, int64_t P2,
                               int64_t* server_x_p2, int64_t* worker_x_p2, int64_t* both_x_p2);

/*
 * The three-way choice between PS, SFB and Adam's scheme for an M x N FC
 * layer on P nodes that are each worker and server (Table 1; Sec. 5.3 ranks
 * the schemes by the load of the busiest node, which for Adam is the node
 * holding the layer): the scheme whose busiest node moves the fewest values,
 *   PS   2 M N (2P - 2) / P,   SFB   2 B (P - 1)(M + N),
 *   Adam (P - 1)(M N + B (M + N)),
 * compared exactly in integers; a tie prefers SFB, then PS.  With P1 = P2
 * Adam never moves strictly less than both others, so the result always
 * equals poseidon_hybcomm_choose.  Host-only.  Returns POSEIDON_PS,
 * POSEIDON_SFB, POSEIDON_ADAM or POSEIDON_ERR_INVALID_ARG (as
 * poseidon_hybcomm_choose).
 */
int poseidon_hybcomm_choose3(int64_t M, int64_t N, int64_t B, int64_t P);

/*
 * One parameter tensor of a network, as handed to poseidon_sync_iteration.
 * W has M*N values (kind FC: M x N row-major; other kinds: any shape
 * flattened, M*N = n).  U/V are the SF payload (K x M and K x N, K = P*B) and
 * shards the dense payload (P x M*N); a tensor carries the payload of the
 * scheme it will use and may set the other to NULL.  buf is the momentum
 * buffer (M*N values) used by either scheme's update, or NULL for plain SGD.
 */
typedef struct poseidon_tensor {
    int32_t      kind;     /* POSEIDON_KIND_FC or POSEIDON_KIND_OTHER */
    int32_t      reserved; /* must be 0 */
    float*       W;
    int64_t      M;
    int64_t      N;
    const float* U;
    const float* V;
    const float* shards;
    float*       buf;
} poseidon_tensor;

/* The client library's GPU stream pool (Sec. 4.1 "Client Library"): a fixed
 * set of non-blocking, default-priority HIP streams on the current device plus
 * the events that fork them from and join them back to a caller stream. */
typedef struct poseidon_stream_pool poseidon_stream_pool;

/* Create a pool of num_streams (1..64) streams on the current device.  An
 * iteration uses at most two of them.  HIP runs a process's streams on at most
 * GPU_MAX_HW_QUEUES hardware queues (4 by default), and streams that share a
 * queue run in order: for the two kinds of updates to overlap each other and
 * the caller's work, keep the streams in use (these two and the caller's)
 * within that number -- a two-stream pool is enough.
 * Returns POSEIDON_OK, POSEIDON_ERR_INVALID_ARG or POSEIDON_ERR_HIP. */
int poseidon_pool_create(int32_t num_streams, poseidon_stream_pool** pool);

/* Destroy a pool (waits for its streams to drain).  NULL is a no-op. */
int poseidon_pool_destroy(poseidon_stream_pool* pool);

/*
 * One iteration's synchronisation of a whole network (Sec. 3 "wait-free
 * backpropagation"; Alg. 2 TRAIN/sync): tensors[] is given in forward order
 * and issued from the last to the first (backpropagation order).  For each
 * tensor the scheme is Alg. 1's (FC: poseidon_hybcomm_choose(M, N, B, P);
 * other kinds: PS).  Every tensor with work is one launch, in
 * backpropagation order: the SFB updates (bound by the matrix cores) and the
 * PS updates (bound by memory bandwidth) on two streams, so that the two
 * kinds overlap -- the kind with the longer estimated time (at the rates
 * below) on the caller's `stream` itself, the other on the pool's first
 * stream, forked from and joined back to `stream`; a one-stream pool, an iteration
 * whose work would take under 30 us at the kernels' rates (130 TFLOP/s for
 * SFB, 5 TB/s for PS), or one whose two kinds would take comparable times at
 * those rates (the smaller above 0.35 of the larger: neither leaves gaps the
 * other could fill, so co-running only delays both) runs everything in order
 * on one stream (without ready events the caller's `stream` itself, with no
 * fork and join events).  Two kinds of tensors share launches instead (with
 * the kernels and arithmetic of the single-tensor calls, so the same
 * results): PS tensors of
 * fewer than 2^17 values, which a launch of their own would leave
 * latency-bound, are applied together, in backpropagation order, by one
 * batched pass (poseidon_ps_apply_batch) after the other PS launches -- and
 * when the PS applies are the iteration's critical path (the SFB rebuilds
 * come to fewer than 26 flops per PS byte, 2*M*N*P*B flops against
 * n*(4P+16) bytes, or 4P+8 without a buffer), so do PS tensors of fewer than
 * 2^21 values; and the SFB tensors without a momentum buffer, when there are
 * several, are rebuilt by one grouped launch (poseidon_sf_apply_batch) at the
 * place of the first of them, so that the layers' tiles share one work list
 * -- except in a two-stream iteration whose PS applies are the longer kind:
 * there every SFB launch runs on few workgroups that each walk several of
 * its tiles, sized to take about 90% of the applies' estimated time, so that
 * the rebuilds run thin beside the applies.  Conversely, when the SFB
 * rebuilds are the longer kind (and the applies would still end first at
 * the rate they get beside them: 1.9 TB/s beside the split-bf16 rebuild,
 * 1.3 beside the fp32 one), the rebuilds leave each SIMD the registers of
 * more waves and the PS applies of aligned tensors use a low-register kernel
 * that runs in them, on the CUs the rebuilds keep busy.  Every variant
 * computes the same results, bitwise.
 * SFB tensors take poseidon_sf_apply(W, U, V, M, N, P*B, lr), or
 * poseidon_sf_apply_momentum(W, buf, U, V, M, N, P*B, lr, momentum) when
 * buf != NULL; PS tensors take poseidon_ps_apply(W, shards, P, M*N, lr,
 * momentum, buf) (momentum is used only when buf != NULL).  The pool
 * stream used first waits for the work already
 * enqueued on `stream`, and `stream` then waits for every tensor's update, so
 * the call behaves like one asynchronous operation on `stream` (the
 * bulk-synchronous barrier of Sec. 4.1 "Managing Consistency").
 * schemes (optional, count entries) receives each tensor's scheme.
 * All arguments are validated before anything is enqueued.  The updates run
 * concurrently, so no tensor may write (W; buf when it has one) where another
 * tensor reads or writes (W, buf, and the payload of its chosen scheme: U and
 * V, or shards); tensors may share a payload.  Returns POSEIDON_OK,
 * POSEIDON_ERR_INVALID_ARG (also for such an overlap), POSEIDON_ERR_PAYLOAD
 * (the chosen scheme's payload is NULL) or POSEIDON_ERR_HIP.
 * The call may be captured into a HIP graph (stream capture on `stream`, with
 * launch timing off): it enqueues only kernel launches and event records and
 * waits that fork from `stream` and join back to it.  A replay repeats the
 * launches chosen at capture (for the shapes, the pool and the arithmetic
 * setting of that time) on the same arrays.
 */
int poseidon_sync_iteration(poseidon_stream_pool* pool,
                            const poseidon_tensor* tensors, int32_t count,
                            int64_t B, int32_t P, float lr, float momentum,
                            hipStream_t stream, int32_t* schemes);

/*
 * The same iteration with wait-free backpropagation (Sec. 3.1; Alg. 2: the
 * sync of layer l is scheduled as soon as BackwardThrough(l) has run): tensor
 * t's update starts once the caller's event ready[t] has completed, not after
 * everything enqueued on `stream`, so the updates of the upper layers run
 * while the backward pass of the lower layers is still computing.  ready[t]
 * marks the point after which W_t may change: the caller records it (with
 * hipEventRecord, on any stream of the current device, BEFORE this call --
 * an event never recorded counts as complete) after the last kernel that
 * reads W_t or writes t's payload (U/V rows or shards) in this iteration;
 * tensors of one layer may share an event.  Issue order, schemes, payload
 * rules and results are those of poseidon_sync_iteration (bitwise: the same
 * kernels).  The pool's schedule (poseidon_pool_set_wfbp_policy) decides
 * what the updates wait for.  By default (POSEIDON_WFBP_SERIAL) `stream`
 * waits for every ready event and the call then is poseidon_sync_iteration
 * on `stream`: the updates also wait for whatever was enqueued on `stream`
 * before the call (the serial order; on one GPU the cheapest, see
 * poseidon_pool_set_wfbp_policy).  Under the other schedules every update
 * runs on the pool's streams (the SFB updates on its first, the PS updates on
 * its second, or all on the first in a one-stream iteration), none on
 * `stream`, so that later work on `stream` can run beside them; only PS
 * tensors of fewer than 2^17 values share the batched pass, so that each
 * other PS update starts after its own event; under POSEIDON_WFBP_SFB_LAST
 * the SFB tensors wait for every ready event and share one grouped launch;
 * under POSEIDON_WFBP_ALL_LAST every update waits for every ready event and
 * the launches are poseidon_sync_iteration's; under POSEIDON_WFBP_EACH every
 * SFB tensor keeps a launch of its own that starts after its own event.
 * `stream` waits for every update at the end.
 * ready: count non-NULL events, caller-owned, not retained after the call.
 * Returns POSEIDON_OK, POSEIDON_ERR_INVALID_ARG (also for NULL ready or a NULL
 * entry), POSEIDON_ERR_PAYLOAD or POSEIDON_ERR_HIP.
 */
int poseidon_sync_iteration_wfbp(poseidon_stream_pool* pool,
                                 const poseidon_tensor* tensors, int32_t count,
                                 int64_t B, int32_t P, float lr, float momentum,
                                 const hipEvent_t* ready, hipStream_t stream, int32_t* schemes);

/*
 * Launch timing (the per-layer synchronisation times the paper's evaluation
 * reasons about, Sec. 5).  While enabled (default: off), every launch that
 * poseidon_sync_iteration or poseidon_sync_iteration_wfbp enqueues is
 * bracketed by two timing events on the stream it runs on (after any wait on a
 * ready event).  Returns POSEIDON_OK or POSEIDON_ERR_INVALID_ARG.
 */
int poseidon_pool_set_timing(poseidon_stream_pool* pool, int32_t enable);

/*
 * The schedule poseidon_sync_iteration_wfbp uses on this pool.
 * POSEIDON_WFBP_EACH is Alg. 2's: every tensor's update starts on its own
 * ready event.  POSEIDON_WFBP_SFB_LAST starts the PS applies on their own
 * events but holds the SFB rebuilds until every tensor's event has completed
 * and runs them as one grouped launch.  POSEIDON_WFBP_ALL_LAST holds every
 * update until every tensor's event has completed and then issues
 * poseidon_sync_iteration's launches on the pool's streams.
 * POSEIDON_WFBP_SERIAL (the default) makes the caller's stream wait for every
 * event and runs poseidon_sync_iteration on it.  On one GPU the updates are
 * local computation that competes with the caller's backward pass -- the
 * rebuilds for the matrix cores its GEMMs use, the applies for the memory
 * bandwidth and CU slots of its elementwise steps -- so nothing is hidden,
 * and the serial order on the caller's stream is the cheapest: the first
 * update starts 10-12 us after the backward pass's last kernel (7 us without
 * events), against 72-84 us for the other held schedules, whose updates wait
 * on another queue.  What the events themselves cost the backward pass that
 * records them (19 per-layer events in a 34.5 ms synthetic VGG19-22K
 * backward pass: 0.06-0.11 ms) is the caller's.  What Alg. 2 hides is time
 * the GPU would otherwise spend waiting for the network; EACH is for callers
 * that have such time.  Results are the same under every schedule
 * (bit-identical kernels).
 * Returns POSEIDON_OK or POSEIDON_ERR_INVALID_ARG (NULL pool, unknown policy).
 */
int poseidon_pool_set_wfbp_policy(poseidon_stream_pool* pool, int32_t policy);

/* One launch of the last iteration run with timing enabled. */
typedef struct poseidon_launch_record {
    int32_t scheme;   /* POSEIDON_SFB or POSEIDON_PS */
    int32_t tensor;   /* index into that call's tensors[], or -1 for a shared launch (scheme
                         POSEIDON_PS: the batched pass of the small PS tensors; POSEIDON_SFB:
                         the grouped launch of the SFB tensors without a buffer) */
    int32_t stream;   /* 0: the SFB updates' stream, 1: the PS updates' (one-stream
                         iterations: 0); see poseidon_sync_iteration for which
                         stream each is */
    float   ms;       /* time between the events around the launch */
} poseidon_launch_record;

/*
 * Copies the launch records of the last timed iteration, in issue order, into
 * records[0 .. *count), waiting for those launches to finish.  *count is set
 * even when capacity is too small (then POSEIDON_ERR_INVALID_ARG).  Returns
 * POSEIDON_OK, POSEIDON_ERR_INVALID_ARG (no timed iteration yet, capacity too
 * small, NULL pointers) or POSEIDON_ERR_HIP.
 */
int poseidon_pool_launch_times(poseidon_stream_pool* pool, poseidon_launch_record* records,
                               int32_t capacity, int32_t* count);

/* Library version, for the binding's load check: returns POSEIDON_ABI_VERSION. */
#define POSEIDON_ABI_VERSION 3
int poseidon_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* POSEIDON_H */
