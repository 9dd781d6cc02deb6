/*
 * A plain C program using libposeidon.so through include/poseidon.h alone --
 * no Python, no PyTorch: device memory from the HIP runtime, every result
 * compared with the CPU oracle (liboracle.so, test infrastructure).  Built by
 * tests/build_c_consumer.py, run by tests/test_gpu_c_abi.py; prints one line
 * per check and exits 0 only if all pass.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "poseidon.h"

/* The oracle's entry points used here (oracle/poseidon_oracle.c). */
void oracle_sf_apply(float *W, const float *U, const float *V, int64_t M, int64_t N, int64_t K, float lr);
int oracle_ps_apply(float *W, const float *shards, int32_t P, int64_t n, float lr, float mu, float *buf);
int oracle_hybcomm_choose(int64_t M, int64_t N, int64_t B, int64_t P);

static int failures = 0;

#define HIP_OK(x)                                                                      \
    do {                                                                               \
        hipError_t e_ = (x);                                                           \
        if (e_ != hipSuccess) {                                                        \
            fprintf(stderr, "HIP error %d at line %d\n", (int)e_, __LINE__);           \
            exit(2);                                                                   \
        }                                                                              \
    } while (0)

/* Seeded inputs: a 64-bit LCG mapped to (-scale, scale). */
static void fill(float *x, int64_t n, uint64_t seed, float scale)
{
    uint64_t s = seed * 6364136223846793005ULL + 1442695040888963407ULL;
    for (int64_t i = 0; i < n; ++i) {
        s = s * 6364136223846793005ULL + 1442695040888963407ULL;
        x[i] = scale * ((float)((s >> 40) & 0xFFFFFF) / 8388608.0f - 1.0f);
    }
}

static void check(const char *what, const float *got, const float *ref, int64_t n, double tol)
{
    double err = 0.0, scale = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        const double d = fabs((double)got[i] - (double)ref[i]);
        if (d > err || d != d)
            err = d;
        if (fabs((double)ref[i]) > scale)
            scale = fabs((double)ref[i]);
    }
    const double rel = scale > 0 ? err / scale : err;
    const int ok = rel <= tol;
    printf("%-44s max|err|/max|ref| = %.3e (tol %.0e) %s\n", what, rel, tol, ok ? "ok" : "FAIL");
    failures += !ok;
}

static float *dev_copy(const float *h, int64_t n)
{
    float *d = NULL;
    HIP_OK(hipMalloc((void **)&d, (size_t)(n > 0 ? n : 1) * sizeof(float)));
    if (n > 0)
        HIP_OK(hipMemcpy(d, h, (size_t)n * sizeof(float), hipMemcpyHostToDevice));
    return d;
}

static void to_host(float *h, const float *d, int64_t n)
{
    HIP_OK(hipMemcpy(h, d, (size_t)n * sizeof(float), hipMemcpyDeviceToHost));
}

int main(void)
{
    HIP_OK(hipSetDevice(0));
    printf("poseidon ABI version %d\n", poseidon_abi_version());

    /* SF reconstruction + SGD, ragged shape, with each arithmetic of the
     * products (the default split-bf16 and the fp32 matrix-core products). */
    if (poseidon_sf_arithmetic() != POSEIDON_SF_BF16X6 || poseidon_sf_set_arithmetic(5) != POSEIDON_ERR_INVALID_ARG) {
        printf("poseidon_sf_arithmetic default / bad value FAIL\n");
        ++failures;
    }
    for (int a = 0; a < 2; ++a) {
        const int32_t arith = a == 0 ? POSEIDON_SF_BF16X6 : POSEIDON_SF_FP32;
        const int64_t M = 300, N = 200, K = 37;
        float *W = malloc(M * N * 4), *U = malloc(K * M * 4), *V = malloc(K * N * 4), *got = malloc(M * N * 4);
        fill(W, M * N, 1, 0.01f);
        fill(U, K * M, 2, 1.0f);
        fill(V, K * N, 3, 1.0f);
        float *dW = dev_copy(W, M * N), *dU = dev_copy(U, K * M), *dV = dev_copy(V, K * N);
        const int rs = poseidon_sf_set_arithmetic(arith);
        const int rc = poseidon_sf_apply(dW, dU, dV, M, N, K, 0.01f, 0);
        HIP_OK(hipDeviceSynchronize());
        poseidon_sf_set_arithmetic(POSEIDON_SF_BF16X6);
        to_host(got, dW, M * N);
        oracle_sf_apply(W, U, V, M, N, K, 0.01f);
        if (rc != POSEIDON_OK || rs != POSEIDON_OK) {
            printf("poseidon_sf_apply returned %d (arithmetic %d: %d) FAIL\n", rc, (int)arith, rs);
            ++failures;
        }
        check(a == 0 ? "poseidon_sf_apply 300x200 K=37 (split-bf16 products)"
                     : "poseidon_sf_apply 300x200 K=37 (fp32 products)", got, W, M * N, 1e-4);
        HIP_OK(hipFree(dW));
        HIP_OK(hipFree(dU));
        HIP_OK(hipFree(dV));
        free(W), free(U), free(V), free(got);
    }

    /* PS aggregation + momentum SGD, ragged size, run-time P. */
    {
        const int32_t P = 5;
        const int64_t n = 1001;
        float *W = malloc(n * 4), *G = malloc(P * n * 4), *B = malloc(n * 4), *got = malloc(n * 4),
              *gotb = malloc(n * 4);
        fill(W, n, 4, 0.01f);
        fill(G, P * n, 5, 1e-3f);
        fill(B, n, 6, 1e-3f);
        float *dW = dev_copy(W, n), *dG = dev_copy(G, P * n), *dB = dev_copy(B, n);
        const int rc = poseidon_ps_apply(dW, dG, P, n, 0.01f, 0.9f, dB, 0);
        HIP_OK(hipDeviceSynchronize());
        to_host(got, dW, n);
        to_host(gotb, dB, n);
        oracle_ps_apply(W, G, P, n, 0.01f, 0.9f, B);
        if (rc != POSEIDON_OK) {
            printf("poseidon_ps_apply returned %d FAIL\n", rc);
            ++failures;
        }
        check("poseidon_ps_apply P=5 n=1001 (W)", got, W, n, 1e-4);
        check("poseidon_ps_apply P=5 n=1001 (buf)", gotb, B, n, 1e-5);
        HIP_OK(hipFree(dW));
        HIP_OK(hipFree(dG));
        HIP_OK(hipFree(dB));
        free(W), free(G), free(B), free(got), free(gotb);
    }

    /* HybComm decision on a grid, bit-exact. */
    {
        int bad = 0, cases = 0;
        for (int64_t M = 1; M <= 40; M += 3)
            for (int64_t N = 1; N <= 40; N += 5)
                for (int64_t B = 1; B <= 9; B += 4)
                    for (int64_t P = 1; P <= 17; P += 2) {
                        bad += poseidon_hybcomm_choose(M, N, B, P) != oracle_hybcomm_choose(M, N, B, P);
                        ++cases;
                    }
        printf("%-44s %d of %d cases differ %s\n", "poseidon_hybcomm_choose", bad, cases, bad ? "FAIL" : "ok");
        failures += bad != 0;
    }

    /* One iteration on a stream pool: an FC layer (SFB) and a dense tensor (PS). */
    {
        const int64_t M = 256, N = 384, Bsz = 4, n = 5000;
        const int32_t P = 4;
        const int64_t K = P * Bsz;
        float *W1 = malloc(M * N * 4), *U = malloc(K * M * 4), *V = malloc(K * N * 4), *g1 = malloc(M * N * 4);
        float *W2 = malloc(n * 4), *G = malloc(P * n * 4), *B2 = malloc(n * 4), *g2 = malloc(n * 4);
        fill(W1, M * N, 7, 0.01f);
        fill(U, K * M, 8, 1.0f);
        fill(V, K * N, 9, 1.0f);
        fill(W2, n, 10, 0.01f);
        fill(G, P * n, 11, 1e-3f);
        memset(B2, 0, n * 4);
        float *dW1 = dev_copy(W1, M * N), *dU = dev_copy(U, K * M), *dV = dev_copy(V, K * N);
        float *dW2 = dev_copy(W2, n), *dG = dev_copy(G, P * n), *dB2 = dev_copy(B2, n);
        /* the same start for the wait-free iterations below, one copy per schedule */
        float *eW1[3], *eW2[3], *eB2[3];
        for (int c = 0; c < 3; ++c)
            eW1[c] = dev_copy(W1, M * N), eW2[c] = dev_copy(W2, n), eB2[c] = dev_copy(B2, n);
        poseidon_stream_pool *pool = NULL;
        int rc = poseidon_pool_create(2, &pool);
        poseidon_tensor t[2];
        memset(t, 0, sizeof t);
        t[0].kind = POSEIDON_KIND_FC;
        t[0].W = dW1, t[0].M = M, t[0].N = N, t[0].U = dU, t[0].V = dV;
        t[1].kind = POSEIDON_KIND_OTHER;
        t[1].W = dW2, t[1].M = n, t[1].N = 1, t[1].shards = dG, t[1].buf = dB2;
        int32_t schemes[2] = {-9, -9};
        if (rc == POSEIDON_OK)
            rc = poseidon_sync_iteration(pool, t, 2, Bsz, P, 0.01f, 0.9f, 0, schemes);
        HIP_OK(hipDeviceSynchronize());
        to_host(g1, dW1, M * N);
        to_host(g2, dW2, n);
        /* The wait-free iteration under Alg. 2's schedule, under
         * POSEIDON_WFBP_ALL_LAST (every update after every event) and under
         * POSEIDON_WFBP_SERIAL (the caller's stream waits, then the plain
         * iteration): the same results. */
        {
            hipEvent_t ev;
            HIP_OK(hipEventCreate(&ev));
            HIP_OK(hipEventRecord(ev, 0));
            const hipEvent_t ready[2] = {ev, ev};
            const int32_t pol[3] = {POSEIDON_WFBP_EACH, POSEIDON_WFBP_ALL_LAST, POSEIDON_WFBP_SERIAL};
            int same = 1, wrc = POSEIDON_OK;
            float *h1 = malloc(M * N * 4), *h2 = malloc(n * 4);
            for (int c = 0; c < 3 && wrc == POSEIDON_OK; ++c) {
                poseidon_tensor u[2];
                memcpy(u, t, sizeof u);
                u[0].W = eW1[c], u[1].W = eW2[c], u[1].buf = eB2[c];
                wrc = poseidon_pool_set_wfbp_policy(pool, pol[c]);
                if (wrc == POSEIDON_OK)
                    wrc = poseidon_sync_iteration_wfbp(pool, u, 2, Bsz, P, 0.01f, 0.9f, ready, 0, NULL);
                HIP_OK(hipDeviceSynchronize());
                to_host(h1, eW1[c], M * N);
                to_host(h2, eW2[c], n);
                same &= memcmp(h1, g1, M * N * 4) == 0 && memcmp(h2, g2, n * 4) == 0;
            }
            const int bad_policy = poseidon_pool_set_wfbp_policy(pool, 17) == POSEIDON_ERR_INVALID_ARG;
            printf("%-44s rc %d %s\n", "poseidon_sync_iteration_wfbp (3 schedules)", wrc,
                   wrc == POSEIDON_OK && same && bad_policy ? "ok" : "FAIL");
            failures += !(wrc == POSEIDON_OK && same && bad_policy);
            free(h1), free(h2);
            HIP_OK(hipEventDestroy(ev));
            for (int c = 0; c < 3; ++c) {
                HIP_OK(hipFree(eW1[c]));
                HIP_OK(hipFree(eW2[c]));
                HIP_OK(hipFree(eB2[c]));
            }
        }
        poseidon_pool_destroy(pool);
        const int want0 = oracle_hybcomm_choose(M, N, Bsz, P);
        if (want0 == 1)
            oracle_sf_apply(W1, U, V, M, N, K, 0.01f);
        oracle_ps_apply(W2, G, P, n, 0.01f, 0.9f, B2);
        const int ok = rc == POSEIDON_OK && schemes[0] == want0 && schemes[1] == POSEIDON_PS;
        printf("%-44s rc %d, schemes %d %d %s\n", "poseidon_sync_iteration", rc, schemes[0], schemes[1],
               ok ? "ok" : "FAIL");
        failures += !ok;
        check("poseidon_sync_iteration (FC layer)", g1, W1, M * N, 1e-4);
        check("poseidon_sync_iteration (dense tensor)", g2, W2, n, 1e-4);
        HIP_OK(hipFree(dW1));
        HIP_OK(hipFree(dU));
        HIP_OK(hipFree(dV));
        HIP_OK(hipFree(dW2));
        HIP_OK(hipFree(dG));
        HIP_OK(hipFree(dB2));
        free(W1), free(U), free(V), free(g1), free(W2), free(G), free(B2), free(g2);
    }

    /* Two-stream iterations on a caller's stream of its own, each followed on
     * that stream by a copy of the weights taken with no synchronisation in
     * between (the iteration is one operation on the caller's stream):
     * (a) the PS apply the longer kind (8M values at P = 4 beside a
     *     1000 x 2048 layer at K = 32: the rebuild spread thin beside it);
     * (b) the SF rebuild the longer kind (4096 x 4096 at K = 128 beside a
     *     1M-value tensor at P = 4: the rebuild on the caller's stream). */
    for (int c = 0; c < 2; ++c) {
        const int64_t M = c == 0 ? 1000 : 4096, N = c == 0 ? 2048 : 4096;
        const int64_t n = c == 0 ? (int64_t)8 << 20 : (int64_t)1 << 20;
        const int64_t Bsz = c == 0 ? 8 : 32;
        const int32_t P = 4;
        const int64_t K = P * Bsz;
        float *W1 = malloc(M * N * 4), *U = malloc(K * M * 4), *V = malloc(K * N * 4), *g1 = malloc(M * N * 4);
        float *W2 = malloc(n * 4), *G = malloc(P * n * 4), *B2 = malloc(n * 4), *g2 = malloc(n * 4);
        fill(W1, M * N, 20 + c, 0.01f);
        fill(U, K * M, 22 + c, 0.1f);
        fill(V, K * N, 24 + c, 0.1f);
        fill(W2, n, 26 + c, 0.01f);
        fill(G, P * n, 28 + c, 1e-3f);
        fill(B2, n, 30 + c, 1e-3f);
        float *dW1 = dev_copy(W1, M * N), *dU = dev_copy(U, K * M), *dV = dev_copy(V, K * N);
        float *dW2 = dev_copy(W2, n), *dG = dev_copy(G, P * n), *dB2 = dev_copy(B2, n);
        float *cW1 = NULL, *cW2 = NULL;
        HIP_OK(hipMalloc((void **)&cW1, (size_t)(M * N) * 4));
        HIP_OK(hipMalloc((void **)&cW2, (size_t)n * 4));
        hipStream_t cs;
        HIP_OK(hipStreamCreateWithFlags(&cs, hipStreamNonBlocking));
        poseidon_stream_pool *pool = NULL;
        int rc = poseidon_pool_create(2, &pool);
        poseidon_tensor t[2];
        memset(t, 0, sizeof t);
        t[0].kind = POSEIDON_KIND_FC;
        t[0].W = dW1, t[0].M = M, t[0].N = N, t[0].U = dU, t[0].V = dV;
        t[1].kind = POSEIDON_KIND_OTHER;
        t[1].W = dW2, t[1].M = n, t[1].N = 1, t[1].shards = dG, t[1].buf = dB2;
        int32_t schemes[2] = {-9, -9};
        if (rc == POSEIDON_OK)
            rc = poseidon_sync_iteration(pool, t, 2, Bsz, P, 0.01f, 0.9f, cs, schemes);
        HIP_OK(hipMemcpyAsync(cW1, dW1, (size_t)(M * N) * 4, hipMemcpyDeviceToDevice, cs));
        HIP_OK(hipMemcpyAsync(cW2, dW2, (size_t)n * 4, hipMemcpyDeviceToDevice, cs));
        HIP_OK(hipStreamSynchronize(cs));
        to_host(g1, cW1, M * N);
        to_host(g2, cW2, n);
        poseidon_pool_destroy(pool);
        HIP_OK(hipStreamDestroy(cs));
        oracle_sf_apply(W1, U, V, M, N, K, 0.01f);
        oracle_ps_apply(W2, G, P, n, 0.01f, 0.9f, B2);
        const int ok = rc == POSEIDON_OK && schemes[0] == POSEIDON_SFB && schemes[1] == POSEIDON_PS;
        printf("%-44s rc %d, schemes %d %d %s\n", c == 0 ? "two streams, PS longer: rc" : "two streams, SF longer: rc",
               rc, schemes[0], schemes[1], ok ? "ok" : "FAIL");
        failures += !ok;
        check(c == 0 ? "two streams, PS longer (FC layer, spread)" : "two streams, SF longer (FC layer)", g1, W1, M * N,
              1e-4);
        check(c == 0 ? "two streams, PS longer (dense tensor)" : "two streams, SF longer (dense tensor)", g2, W2, n,
              1e-4);
        HIP_OK(hipFree(dW1));
        HIP_OK(hipFree(dU));
        HIP_OK(hipFree(dV));
        HIP_OK(hipFree(dW2));
        HIP_OK(hipFree(dG));
        HIP_OK(hipFree(dB2));
        HIP_OK(hipFree(cW1));
        HIP_OK(hipFree(cW2));
        free(W1), free(U), free(V), free(g1), free(W2), free(G), free(B2), free(g2);
    }

    /* The KV store: every server of P = 3 applies its pairs from the workers'
     * messages; together they equal the plain PS apply of the whole tensor. */
    {
        const int32_t P = 3;
        const int64_t n = 2500, pair = 256;
        float *W = malloc(n * 4), *G = malloc(P * n * 4), *got = malloc(n * 4);
        fill(W, n, 12, 0.01f);
        fill(G, P * n, 13, 1e-3f);
        float *dW = dev_copy(W, n), *dG = dev_copy(G, P * n);
        int rc = POSEIDON_OK;
        for (int32_t r = 0; r < P && rc >= 0; ++r) {
            poseidon_kv_tensor kt = {dW, NULL, n};
            poseidon_kv_store *st = NULL;
            rc = poseidon_kv_create(&kt, 1, pair, P, r, 0.01f, 0.0f, &st);
            int64_t len = 0;
            if (rc == POSEIDON_OK)
                rc = poseidon_kv_message_size(st, &len);
            /* one message per worker: the store reads all P when the last arrives */
            float *msg[3] = {NULL, NULL, NULL};
            for (int32_t p = 0; p < P; ++p)
                HIP_OK(hipMalloc((void **)&msg[p], (size_t)(len > 0 ? len : 1) * 4));
            for (int32_t p = 0; p < P && rc >= 0; ++p) {
                const float *gp = dG + (int64_t)p * n;
                int64_t wrote = 0;
                rc = poseidon_kv_pack(&n, &gp, 1, pair, P, r, msg[p], len, &wrote, 0);
                if (rc == POSEIDON_OK)
                    rc = poseidon_kv_receive_message(st, p, msg[p], 0);
            }
            HIP_OK(hipDeviceSynchronize());
            for (int32_t p = 0; p < P; ++p)
                HIP_OK(hipFree(msg[p]));
            poseidon_kv_destroy(st);
        }
        to_host(got, dW, n);
        oracle_ps_apply(W, G, P, n, 0.01f, 0.0f, NULL);
        printf("%-44s rc %d %s\n", "poseidon_kv_* (3 servers, messages)", rc, rc >= 0 ? "ok" : "FAIL");
        failures += rc < 0;
        check("poseidon_kv_* union of the servers", got, W, n, 1e-4);
        HIP_OK(hipFree(dW));
        HIP_OK(hipFree(dG));
        free(W), free(G), free(got);
    }

    printf("%s: %d failure(s)\n", failures ? "FAILED" : "PASSED", failures);
    return failures ? 1 : 0;
}
