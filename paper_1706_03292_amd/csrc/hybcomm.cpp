// Hybrid communication: the coordinator's BestScheme (Sec. 3.2, Table 1,
// Alg. 1), evaluated exactly in 128-bit integers.  Host-only.
#include <stdint.h>

#include "poseidon.h"

namespace {

constexpr int64_t kMaxArg = INT32_MAX;   // every argument fits in 31 bits

inline bool in_range(int64_t x, int64_t lo) { return x >= lo && x <= kMaxArg; }

// Table 1, multiplied through by P2 so that PS's MN/P2 partition stays exact.
//   PS, node that is both server and worker:  2 M N (P1 + P2 - 2) / P2
//   SFB, worker:                              2 B (P1 - 1) (M + N)
inline __int128 ps_cost_x_p2(int64_t M, int64_t N, int64_t P1, int64_t P2)
{
    return static_cast<__int128>(2) * M * N * (P1 + P2 - 2);
}

inline __int128 sfb_cost_x_p2(int64_t M, int64_t N, int64_t B, int64_t P1, int64_t P2)
{
    return static_cast<__int128>(2) * B * (P1 - 1) * (M + N) * P2;
}

// Table 1, Adam row (x P2): the holder of the layer, a plain worker, and a
// holder that is also a worker.
inline __int128 adam_server_x_p2(int64_t M, int64_t N, int64_t B, int64_t P1, int64_t P2)
{
    return (static_cast<__int128>(P1) * M * N + static_cast<__int128>(P1) * B * (M + N)) * P2;
}

inline __int128 adam_worker_x_p2(int64_t M, int64_t N, int64_t B, int64_t P2)
{
    return (static_cast<__int128>(B) * (M + N) + static_cast<__int128>(M) * N) * P2;
}

inline __int128 adam_both_x_p2(int64_t M, int64_t N, int64_t B, int64_t P1, int64_t P2)
{
    return static_cast<__int128>(P1 - 1) * (static_cast<__int128>(M) * N + static_cast<__int128>(B) * (M + N)) *
           P2;
}

}  // namespace

extern "C" int poseidon_hybcomm_cost(int64_t M, int64_t N, int64_t B, int64_t P1, int64_t P2,
                                     int64_t* ps_x_p2, int64_t* sfb_x_p2)
{
    if (!in_range(M, 0) || !in_range(N, 0) || !in_range(B, 0) || !in_range(P1, 1) ||
        !in_range(P2, 1) || !ps_x_p2 || !sfb_x_p2)
        return POSEIDON_ERR_INVALID_ARG;
    const __int128 ps = ps_cost_x_p2(M, N, P1, P2);
    const __int128 sfb = sfb_cost_x_p2(M, N, B, P1, P2);
    if (ps > INT64_MAX || sfb > INT64_MAX)
        return POSEIDON_ERR_INVALID_ARG;
    *ps_x_p2 = static_cast<int64_t>(ps);
    *sfb_x_p2 = static_cast<int64_t>(sfb);
    return POSEIDON_OK;
}

extern "C" int poseidon_hybcomm_choose(int64_t M, int64_t N, int64_t B, int64_t P)
{
    if (!in_range(M, 0) || !in_range(N, 0) || !in_range(B, 0) || !in_range(P, 1))
        return POSEIDON_ERR_INVALID_ARG;
    // Alg. 1 with P1 = P2 = P; "<=" sends a tie to SFB.  The 31-bit bounds keep
    // every product below 2^127.
    return sfb_cost_x_p2(M, N, B, P, P) <= ps_cost_x_p2(M, N, P, P) ? POSEIDON_SFB : POSEIDON_PS;
}

extern "C" int poseidon_hybcomm_cost_adam(int64_t M, int64_t N, int64_t B, int64_t P1, int64_t P2,
                                          int64_t* server_x_p2, int64_t* worker_x_p2, int64_t* both_x_p2)
{
    if (!in_range(M, 0) || !in_range(N, 0) || !in_range(B, 0) || !in_range(P1, 1) ||
        !in_range(P2, 1) || !server_x_p2 || !worker_x_p2 || !both_x_p2)
        return POSEIDON_ERR_INVALID_ARG;
    const __int128 s = adam_server_x_p2(M, N, B, P1, P2);
    const __int128 w = adam_worker_x_p2(M, N, B, P2);
    const __int128 b = adam_both_x_p2(M, N, B, P1, P2);
    if (s > INT64_MAX || w > INT64_MAX || b > INT64_MAX)
        return POSEIDON_ERR_INVALID_ARG;
    *server_x_p2 = static_cast<int64_t>(s);
    *worker_x_p2 = static_cast<int64_t>(w);
    *both_x_p2 = static_cast<int64_t>(b);
    return POSEIDON_OK;
}

extern "C" int poseidon_hybcomm_choose3(int64_t M, int64_t N, int64_t B, int64_t P)
{
    if (!in_range(M, 0) || !in_range(N, 0) || !in_range(B, 0) || !in_range(P, 1))
        return POSEIDON_ERR_INVALID_ARG;
    // Busiest node of each scheme, x P (P1 = P2 = P): every node for PS and
    // SFB; for Adam the holder, which moves at least what any other node does.
    const __int128 ps = ps_cost_x_p2(M, N, P, P);
    const __int128 sfb = sfb_cost_x_p2(M, N, B, P, P);
    const __int128 adam = adam_both_x_p2(M, N, B, P, P);
    if (sfb <= ps && sfb <= adam)
        return POSEIDON_SFB;
    return ps <= adam ? POSEIDON_PS : POSEIDON_ADAM;
}
