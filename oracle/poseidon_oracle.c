/*
 * Plain, slow, obviously-correct CPU oracle for one node's per-layer
 * gradient synchronisation in Poseidon (Zhang et al., "Poseidon: An
 * Efficient Communication Architecture for Distributed Deep Learning on GPU
 * Clusters", arXiv 1706.03292).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header, table or helper with the HIP library it checks.
 *
 * Floating point: inputs and stored outputs are fp32 (the storage type of the
 * layers); every sum is taken in fp64 and rounded to fp32 only where a value is
 * stored.  Sums follow the order stated at each function.  No fast-math.
 *
 * Readings of the paper used here (each is listed with its reason in the
 * design notes of the repository):
 *  - The update equations (Eq. 1, Eq. 2) write theta + eps * grad with the
 *    gradient taken as the descent direction; this oracle applies
 *    W <- W - lr * g with g = dL/dW.
 *  - Gradients are SUMMED over samples and workers (Eq. 2, and the additivity
 *    remark after Eq. 1); no 1/(P*B) factor.  Callers fold any normalisation
 *    into lr or into the factors.
 *  - Momentum is not in the paper; the parameter-server apply uses the common
 *    heavy-ball form buf <- mu*buf + g, W <- W - lr*buf (no dampening, no
 *    Nesterov, no weight decay).  mu == 0 with buf == NULL is plain SGD.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <omp.h>

/* ------------------------------------------------------------------------ */
/* Sufficient-factor reconstruction (Sec. 2.1, "Sufficient Factor            */
/* Broadcasting"; Fig. 2b): the gradient of a fully-connected layer over one */
/* sample is the rank-1 matrix u v^T, and over a batch gathered from P        */
/* workers it is the sum of those outer products (Eq. 2).                    */
/*                                                                          */
/* Layout: W is M x N row-major (M = length of u = fan-out, N = length of v = */
/* fan-in).  U is K x M row-major (row k is u_k), V is K x N row-major (row k */
/* is v_k); K = P * B factor pairs.                                          */
/* ------------------------------------------------------------------------ */

/* dW[m][n] = sum over k = 0..K-1, in increasing k, of (double)U[k][m] * (double)V[k][n]. */
void oracle_sf_delta(double *dW, const float *U, const float *V,
                     int64_t M, int64_t N, int64_t K)
{
    #pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; ++m) {
        double *row = dW + m * N;
        for (int64_t n = 0; n < N; ++n)
            row[n] = 0.0;
        for (int64_t k = 0; k < K; ++k) {
            const double u = (double)U[k * M + m];
            const float *vk = V + k * N;
            for (int64_t n = 0; n < N; ++n)
                row[n] += u * (double)vk[n];
        }
    }
}

/* SGD step (Eq. 1) with the reconstructed gradient, rows m0 <= m < m1 only:
 *   W[m][n] <- (float)((double)W[m][n] - (double)lr * dW[m][n]).
 * lr is the fp32 value the caller passes (0.01f is not 0.01). */
void oracle_sf_apply_rows(float *W, const float *U, const float *V,
                          int64_t M, int64_t N, int64_t K, float lr,
                          int64_t m0, int64_t m1)
{
    if (m0 < 0) m0 = 0;
    if (m1 > M) m1 = M;
    #pragma omp parallel
    {
        double *acc = (double *)malloc((size_t)(N > 0 ? N : 1) * sizeof(double));
        #pragma omp for schedule(static)
        for (int64_t m = m0; m < m1; ++m) {
            for (int64_t n = 0; n < N; ++n)
                acc[n] = 0.0;
            for (int64_t k = 0; k < K; ++k) {
                const double u = (double)U[k * M + m];
                const float *vk = V + k * N;
                for (int64_t n = 0; n < N; ++n)
                    acc[n] += u * (double)vk[n];
            }
            float *w = W + m * N;
            for (int64_t n = 0; n < N; ++n)
                w[n] = (float)((double)w[n] - (double)lr * acc[n]);
        }
        free(acc);
    }
}

void oracle_sf_apply(float *W, const float *U, const float *V,
                     int64_t M, int64_t N, int64_t K, float lr)
{
    oracle_sf_apply_rows(W, U, V, M, N, K, lr, 0, M);
}

/* The same update at cnt chosen points (rows[i], cols[i]) of a W that is not
 * modified; out[i] receives the updated value.  Used to check layers too large
 * for the full oracle. */
void oracle_sf_apply_points(const float *W, const float *U, const float *V,
                            int64_t M, int64_t N, int64_t K, float lr,
                            const int64_t *rows, const int64_t *cols,
                            int64_t cnt, float *out)
{
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < cnt; ++i) {
        const int64_t m = rows[i], n = cols[i];
        double acc = 0.0;
        for (int64_t k = 0; k < K; ++k)
            acc += (double)U[k * M + m] * (double)V[k * N + n];
        out[i] = (float)((double)W[m * N + n] - (double)lr * acc);
    }
}

/* An SFB layer that keeps a momentum buffer: the same heavy-ball rule as the
 * parameter-server apply below, with the reconstructed gradient in place of
 * the shard sum (the paper's solver settings use momentum for every layer;
 * Eq. 1 itself is plain SGD):
 *   b = (double)mu * buf[m][n] + dW[m][n];  buf' = (float)b;
 *   W'  = (float)((double)W[m][n] - (double)lr * (double)buf').
 * Rows m0 <= m < m1 only. */
void oracle_sf_apply_momentum_rows(float *W, float *buf, const float *U, const float *V,
                                   int64_t M, int64_t N, int64_t K, float lr, float mu,
                                   int64_t m0, int64_t m1)
{
    if (m0 < 0) m0 = 0;
    if (m1 > M) m1 = M;
    #pragma omp parallel
    {
        double *acc = (double *)malloc((size_t)(N > 0 ? N : 1) * sizeof(double));
        #pragma omp for schedule(static)
        for (int64_t m = m0; m < m1; ++m) {
            for (int64_t n = 0; n < N; ++n)
                acc[n] = 0.0;
            for (int64_t k = 0; k < K; ++k) {
                const double u = (double)U[k * M + m];
                const float *vk = V + k * N;
                for (int64_t n = 0; n < N; ++n)
                    acc[n] += u * (double)vk[n];
            }
            float *w = W + m * N, *b = buf + m * N;
            for (int64_t n = 0; n < N; ++n) {
                const float nb = (float)((double)mu * (double)b[n] + acc[n]);
                b[n] = nb;
                w[n] = (float)((double)w[n] - (double)lr * (double)nb);
            }
        }
        free(acc);
    }
}

/* The same at cnt chosen points of W and buf (not modified); w_out[i] and
 * b_out[i] receive the updated values. */
void oracle_sf_apply_momentum_points(const float *W, const float *buf, const float *U, const float *V,
                                     int64_t M, int64_t N, int64_t K, float lr, float mu,
                                     const int64_t *rows, const int64_t *cols, int64_t cnt,
                                     float *w_out, float *b_out)
{
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < cnt; ++i) {
        const int64_t m = rows[i], n = cols[i];
        double acc = 0.0;
        for (int64_t k = 0; k < K; ++k)
            acc += (double)U[k * M + m] * (double)V[k * N + n];
        const float nb = (float)((double)mu * (double)buf[m * N + n] + acc);
        b_out[i] = nb;
        w_out[i] = (float)((double)W[m * N + n] - (double)lr * (double)nb);
    }
}

/* ------------------------------------------------------------------------ */
/* Parameter-server aggregation and apply (Sec. 2.1, "Parameter Server",     */
/* steps (1)-(2); Sec. 4.1, "KV Store" and "Managing Consistency"): the       */
/* server applies the sum of all P workers' gradients once every worker's     */
/* update has arrived.  Because the update must not depend on the order in    */
/* which the P updates arrive, the oracle sums the P values of each element   */
/* in a canonical order (ascending value) so that its result is exactly       */
/* invariant to any permutation of the shards.                                */
/*                                                                          */
/* Layout: shard p occupies shards[p*n .. p*n + n).                          */
/* ------------------------------------------------------------------------ */

static int cmp_float_asc(const void *a, const void *b)
{
    const float x = *(const float *)a, y = *(const float *)b;
    return (x > y) - (x < y);
}

/* Canonical-order fp64 sum of the P values G[p][i]; tmp holds P floats. */
static double canonical_sum(const float *shards, int32_t P, int64_t n,
                            int64_t i, float *tmp)
{
    for (int32_t p = 0; p < P; ++p)
        tmp[p] = shards[(int64_t)p * n + i];
    qsort(tmp, (size_t)P, sizeof(float), cmp_float_asc);
    double s = 0.0;
    for (int32_t p = 0; p < P; ++p)
        s += (double)tmp[p];
    return s;
}

/* One element of the apply:
 *   s = canonical sum of G[.][i]
 *   with buf:    b = (double)mu * buf[i] + s;  buf[i] = (float)b;
 *                W[i] = (float)((double)W[i] - (double)lr * (double)buf[i])
 *   without buf: W[i] = (float)((double)W[i] - (double)lr * s)               */
static void ps_element(float *w, float *b, double s, float lr, float mu)
{
    if (b) {
        const float nb = (float)((double)mu * (double)(*b) + s);
        *b = nb;
        *w = (float)((double)(*w) - (double)lr * (double)nb);
    } else {
        *w = (float)((double)(*w) - (double)lr * s);
    }
}

/* Elements i0 <= i < i1.  buf may be NULL only when mu == 0.  Returns 0, or -1
 * for invalid arguments. */
int oracle_ps_apply_range(float *W, const float *shards, int32_t P, int64_t n,
                          float lr, float mu, float *buf, int64_t i0, int64_t i1)
{
    if (P < 1 || n < 0 || (buf == NULL && mu != 0.0f))
        return -1;
    if (i0 < 0) i0 = 0;
    if (i1 > n) i1 = n;
    int bad = 0;
    #pragma omp parallel
    {
        float *tmp = (float *)malloc((size_t)P * sizeof(float));
        if (!tmp) {
            #pragma omp atomic write
            bad = 1;
        } else {
            #pragma omp for schedule(static)
            for (int64_t i = i0; i < i1; ++i) {
                const double s = canonical_sum(shards, P, n, i, tmp);
                ps_element(W + i, buf ? buf + i : NULL, s, lr, mu);
            }
            free(tmp);
        }
    }
    return bad ? -1 : 0;
}

int oracle_ps_apply(float *W, const float *shards, int32_t P, int64_t n,
                    float lr, float mu, float *buf)
{
    return oracle_ps_apply_range(W, shards, P, n, lr, mu, buf, 0, n);
}

/* The same apply at cnt chosen element indices of W/buf that are not modified;
 * w_out[i] (and b_out[i] when buf != NULL) receive the updated values. */
int oracle_ps_apply_points(const float *W, const float *shards, int32_t P,
                           int64_t n, float lr, float mu, const float *buf,
                           const int64_t *idx, int64_t cnt,
                           float *w_out, float *b_out)
{
    if (P < 1 || n < 0 || (buf == NULL && mu != 0.0f))
        return -1;
    float *tmp = (float *)malloc((size_t)P * sizeof(float));
    if (!tmp)
        return -1;
    for (int64_t j = 0; j < cnt; ++j) {
        const int64_t i = idx[j];
        float w = W[i];
        float b = buf ? buf[i] : 0.0f;
        const double s = canonical_sum(shards, P, n, i, tmp);
        ps_element(&w, buf ? &b : NULL, s, lr, mu);
        w_out[j] = w;
        if (buf && b_out)
            b_out[j] = b;
    }
    free(tmp);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Hybrid communication by exhaustive message counting (Sec. 3.2, Table 1,   */
/* Alg. 1).  One synchronisation of one M x N fully-connected layer is        */
/* enumerated message by message on a cluster whose node j has role          */
/* roles[j] (bit 0: worker, bit 1: server).  Messages between two roles on    */
/* the same node do not cross the network and are not counted; every other    */
/* message is counted at both of its endpoints.                              */
/*                                                                          */
/*  PS   : the parameters are split equally over the P2 servers, so every     */
/*         worker sends MN/P2 gradient values to each server and receives     */
/*         MN/P2 fresh parameters back from each server.                      */
/*  SFB  : every worker sends its B sufficient-factor pairs, B*(M+N) values,  */
/*         to every other worker (peer-to-peer broadcast).                    */
/*  Adam : every worker sends its B(M+N) factor values to the one server that */
/*         holds the layer (the first server node), which sends the whole    */
/*         rebuilt MN matrix back to every worker.                           */
/*                                                                          */
/* Counts are in units of 1/P2 of a value so that MN/P2 stays an integer:    */
/* per_node[j] = P2 * (values node j sends or receives over the network).    */
/* Returns 0, or -1 on invalid input or int64 overflow.                      */
/* ------------------------------------------------------------------------ */

enum { ORACLE_PS = 0, ORACLE_SFB = 1, ORACLE_ADAM = 2 };
enum { ROLE_WORKER = 1, ROLE_SERVER = 2 };

static int add_msg(int64_t *per_node, int32_t src, int32_t dst, int64_t units)
{
    if (src == dst)
        return 0;                         /* same machine: no network traffic */
    if (__builtin_add_overflow(per_node[src], units, &per_node[src]))
        return -1;
    if (__builtin_add_overflow(per_node[dst], units, &per_node[dst]))
        return -1;
    return 0;
}

int oracle_hybcomm_traffic(int64_t M, int64_t N, int64_t B,
                           const int32_t *roles, int32_t nodes, int32_t scheme,
                           int64_t *per_node)
{
    if (M < 0 || N < 0 || B < 0 || nodes < 1 || !roles || !per_node)
        return -1;
    int64_t P2 = 0;
    int32_t first_server = -1;
    for (int32_t j = 0; j < nodes; ++j) {
        per_node[j] = 0;
        if (roles[j] & ROLE_SERVER) {
            if (first_server < 0)
                first_server = j;
            ++P2;
        }
    }
    if (P2 < 1)
        return -1;

    int64_t mn, mpn, bmn, sf_units, ps_units, full_units;
    if (__builtin_mul_overflow(M, N, &mn)) return -1;
    if (__builtin_add_overflow(M, N, &mpn)) return -1;
    if (__builtin_mul_overflow(B, mpn, &bmn)) return -1;
    if (__builtin_mul_overflow(bmn, P2, &sf_units)) return -1;   /* B(M+N) values */
    ps_units = mn;                                               /* MN/P2 values  */
    if (__builtin_mul_overflow(mn, P2, &full_units)) return -1;  /* MN values     */

    for (int32_t w = 0; w < nodes; ++w) {
        if (!(roles[w] & ROLE_WORKER))
            continue;
        if (scheme == ORACLE_PS) {
            for (int32_t s = 0; s < nodes; ++s) {
                if (!(roles[s] & ROLE_SERVER))
                    continue;
                if (add_msg(per_node, w, s, ps_units)) return -1;  /* push */
                if (add_msg(per_node, s, w, ps_units)) return -1;  /* pull */
            }
        } else if (scheme == ORACLE_SFB) {
            for (int32_t q = 0; q < nodes; ++q) {
                if (q == w || !(roles[q] & ROLE_WORKER))
                    continue;
                if (add_msg(per_node, w, q, sf_units)) return -1;  /* broadcast */
            }
        } else if (scheme == ORACLE_ADAM) {
            if (add_msg(per_node, w, first_server, sf_units)) return -1;
            if (add_msg(per_node, first_server, w, full_units)) return -1;
        } else {
            return -1;
        }
    }
    return 0;
}

/* Alg. 1 as a comparison of enumerated traffic on the cluster the boundary
 * assumes: P nodes, each both worker and server (P1 = P2 = P), which is the
 * setting of the worked example in Sec. 3.2.  Returns 1 (SFB) when the total
 * network traffic of SFB does not exceed that of PS (the comparison in Alg. 1
 * is "<=", so a tie goes to SFB), 0 (PS) otherwise, -1 on invalid input. */
int oracle_hybcomm_choose(int64_t M, int64_t N, int64_t B, int64_t P)
{
    if (P < 1 || P > 1 << 16 || M < 0 || N < 0 || B < 0)
        return -1;
    const int32_t nodes = (int32_t)P;
    int32_t *roles = (int32_t *)malloc((size_t)nodes * sizeof(int32_t));
    int64_t *ps = (int64_t *)malloc((size_t)nodes * sizeof(int64_t));
    int64_t *sfb = (int64_t *)malloc((size_t)nodes * sizeof(int64_t));
    int rc = -1;
    if (roles && ps && sfb) {
        for (int32_t j = 0; j < nodes; ++j)
            roles[j] = ROLE_WORKER | ROLE_SERVER;
        if (oracle_hybcomm_traffic(M, N, B, roles, nodes, ORACLE_PS, ps) == 0 &&
            oracle_hybcomm_traffic(M, N, B, roles, nodes, ORACLE_SFB, sfb) == 0) {
            int64_t tps = 0, tsfb = 0;
            int ovf = 0;
            for (int32_t j = 0; j < nodes; ++j) {
                ovf |= __builtin_add_overflow(tps, ps[j], &tps);
                ovf |= __builtin_add_overflow(tsfb, sfb[j], &tsfb);
            }
            if (!ovf)
                rc = (tsfb <= tps) ? 1 : 0;
        }
    }
    free(roles);
    free(ps);
    free(sfb);
    return rc;
}

/* The three-way choice with Adam's scheme added (Table 1's Adam row; Sec.
 * 5.3 compares the three by the load on the busiest node, Adam's row being
 * that maximum).  On P nodes that are each worker and server, every scheme's
 * traffic is enumerated as above and the one whose busiest node moves the
 * fewest values wins; on a tie SFB is preferred (Alg. 1's "<="), then PS,
 * then Adam.  Returns 0 (PS), 1 (SFB), 2 (Adam) or -1 on invalid input. */
int oracle_hybcomm_choose3(int64_t M, int64_t N, int64_t B, int64_t P)
{
    if (P < 1 || P > 1 << 16 || M < 0 || N < 0 || B < 0)
        return -1;
    const int32_t nodes = (int32_t)P;
    int32_t *roles = (int32_t *)malloc((size_t)nodes * sizeof(int32_t));
    int64_t *t = (int64_t *)malloc((size_t)nodes * sizeof(int64_t));
    int64_t busiest[3] = {0, 0, 0};
    int rc = -1;
    if (roles && t) {
        for (int32_t j = 0; j < nodes; ++j)
            roles[j] = ROLE_WORKER | ROLE_SERVER;
        rc = 0;
        for (int32_t scheme = 0; scheme < 3 && rc == 0; ++scheme) {
            if (oracle_hybcomm_traffic(M, N, B, roles, nodes, scheme, t) != 0) {
                rc = -1;
                break;
            }
            for (int32_t j = 0; j < nodes; ++j)
                if (t[j] > busiest[scheme])
                    busiest[scheme] = t[j];
        }
        if (rc == 0) {
            const int order[3] = {ORACLE_SFB, ORACLE_PS, ORACLE_ADAM};   /* tie preference */
            int best = order[0];
            for (int i = 1; i < 3; ++i)
                if (busiest[order[i]] < busiest[best])
                    best = order[i];
            rc = best;
        }
    }
    free(roles);
    free(t);
    return rc;
}

/* Threads the parallel loops above use (for reporting the CPU baseline). */
int oracle_num_threads(void)
{
    return omp_get_max_threads();
}
