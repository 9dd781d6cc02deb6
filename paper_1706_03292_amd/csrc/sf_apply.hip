// Sufficient-factor reconstruction fused with the SGD step (Sec. 2.1
// "Sufficient Factor Broadcasting"; Eq. 1, Eq. 2):
//
//   W[m][n] <- W[m][n] - lr * sum_{k<K} U[k][m] * V[k][n]
//
// A dense contraction of depth K = P*B with both operands stored K-major
// (row k of U is u_k, row k of V is v_k).  It runs on the fp32 matrix cores
// (v_mfma_f32_32x32x2_f32: a 32x32 output block from a 32x2 and a 2x32
// operand, 64 lanes, 16 accumulator registers per lane).
//
// Tiling: a workgroup owns a BM x BN block of W and loops over K in steps of
// BK.  U[k0:k0+BK, m0:m0+BM] and V[k0:k0+BK, n0:n0+BN] are staged through LDS,
// double-buffered, with the next step's global loads in flight while the
// matrix cores work on the current one.  Each wave owns a WM x WN sub-block
// (WM/32 x WN/32 MFMA blocks).  The SGD update is the epilogue: W is read
// once and written once, straight from the accumulators, so the kernel never
// materialises the gradient.
#include "common.h"

namespace poseidon {
namespace {

typedef float f16v __attribute__((ext_vector_type(16)));

constexpr int LDS_PAD = 4;   // floats of padding per LDS row (keeps 16-byte alignment)

template <int BM, int BN, int BK, int WM, int WN>
struct SfTile {
    static constexpr int NWM = BM / WM;
    static constexpr int NWN = BN / WN;
    static constexpr int THREADS = NWM * NWN * 64;
    static constexpr int TM = WM / 32;
    static constexpr int TN = WN / 32;
    static constexpr int LDA = BM + LDS_PAD;
    static constexpr int LDB = BN + LDS_PAD;
    static constexpr int A_V4 = BK * BM / 4 / THREADS;   // 16-byte groups per thread per step
    static constexpr int B_V4 = BK * BN / 4 / THREADS;
    static_assert(BM % WM == 0 && BN % WN == 0 && WM % 32 == 0 && WN % 32 == 0, "tile");
    static_assert(BK % 2 == 0, "MFMA depth is 2");
    static_assert(A_V4 * THREADS * 4 == BK * BM && B_V4 * THREADS * 4 == BK * BN, "staging");
};

// Load one BK x (4*cols4) panel slice of a K-major operand X (row stride ld)
// into registers: group j of this thread covers row r = g / cols4, columns
// 4*(g % cols4) .. +3 with g = tid + j*THREADS.  Out-of-range rows/columns
// read as 0, which adds nothing to the sum.
template <int NV4, int COLS4, int THREADS, bool VEC>
__device__ inline void load_panel(f4 (&r)[NV4], const float* __restrict__ X, int64_t ld,
                                  int64_t rows, int64_t k0, int64_t c0, int tid)
{
#pragma unroll
    for (int j = 0; j < NV4; ++j) {
        const int g = tid + j * THREADS;
        const int64_t k = k0 + g / COLS4;
        const int64_t c = c0 + 4 * (g % COLS4);
        const float* src = X + k * ld + c;
        if constexpr (VEC) {
            // ld % 4 == 0 and X 16-byte aligned: a group is wholly in or out.
            r[j] = (k < rows && c < ld) ? *reinterpret_cast<const f4*>(src) : f4{0.f, 0.f, 0.f, 0.f};
        } else {
            const bool kin = k < rows;
            r[j].x = (kin && c + 0 < ld) ? src[0] : 0.f;
            r[j].y = (kin && c + 1 < ld) ? src[1] : 0.f;
            r[j].z = (kin && c + 2 < ld) ? src[2] : 0.f;
            r[j].w = (kin && c + 3 < ld) ? src[3] : 0.f;
        }
    }
}

template <int NV4, int COLS4, int THREADS, int LD>
__device__ inline void store_panel(float* lds, const f4 (&r)[NV4], int tid)
{
#pragma unroll
    for (int j = 0; j < NV4; ++j) {
        const int g = tid + j * THREADS;
        *reinterpret_cast<f4*>(lds + (g / COLS4) * LD + 4 * (g % COLS4)) = r[j];
    }
}

template <int BM, int BN, int BK, int WM, int WN, bool VEC>
__global__ __launch_bounds__((BM / WM) * (BN / WN) * 64) void sf_apply_kernel(
    float* __restrict__ W, const float* __restrict__ U, const float* __restrict__ V,
    int64_t M, int64_t N, int64_t K, float lr, int tiles_n)
{
    using T = SfTile<BM, BN, BK, WM, WN>;
    __shared__ float As[2][BK * T::LDA];
    __shared__ float Bs[2][BK * T::LDB];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int64_t m0 = static_cast<int64_t>(blockIdx.x / tiles_n) * BM;
    const int64_t n0 = static_cast<int64_t>(blockIdx.x % tiles_n) * BN;
    const int wm = (wave / T::NWN) * WM;
    const int wn = (wave % T::NWN) * WN;
    const int lrow = lane >> 5;        // which of the two k of an MFMA step this lane supplies
    const int lcol = lane & 31;

    f16v acc[T::TM][T::TN];
#pragma unroll
    for (int i = 0; i < T::TM; ++i)
#pragma unroll
        for (int j = 0; j < T::TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                acc[i][j][r] = 0.f;

    f4 ra[T::A_V4], rb[T::B_V4];
    const int64_t nkt = (K + BK - 1) / BK;

    load_panel<T::A_V4, BM / 4, T::THREADS, VEC>(ra, U, M, K, 0, m0, tid);
    load_panel<T::B_V4, BN / 4, T::THREADS, VEC>(rb, V, N, K, 0, n0, tid);
    store_panel<T::A_V4, BM / 4, T::THREADS, T::LDA>(As[0], ra, tid);
    store_panel<T::B_V4, BN / 4, T::THREADS, T::LDB>(Bs[0], rb, tid);
    __syncthreads();

    for (int64_t kt = 0; kt < nkt; ++kt) {
        const int cur = static_cast<int>(kt & 1);
        const bool more = kt + 1 < nkt;
        if (more) {
            load_panel<T::A_V4, BM / 4, T::THREADS, VEC>(ra, U, M, K, (kt + 1) * BK, m0, tid);
            load_panel<T::B_V4, BN / 4, T::THREADS, VEC>(rb, V, N, K, (kt + 1) * BK, n0, tid);
        }
        const float* a_s = As[cur];
        const float* b_s = Bs[cur];
#pragma unroll
        for (int kk = 0; kk < BK; kk += 2) {
            float a[T::TM], b[T::TN];
#pragma unroll
            for (int i = 0; i < T::TM; ++i)
                a[i] = a_s[(kk + lrow) * T::LDA + wm + 32 * i + lcol];
#pragma unroll
            for (int j = 0; j < T::TN; ++j)
                b[j] = b_s[(kk + lrow) * T::LDB + wn + 32 * j + lcol];
#pragma unroll
            for (int i = 0; i < T::TM; ++i)
#pragma unroll
                for (int j = 0; j < T::TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i], b[j], acc[i][j], 0, 0, 0);
        }
        if (more) {
            store_panel<T::A_V4, BM / 4, T::THREADS, T::LDA>(As[cur ^ 1], ra, tid);
            store_panel<T::B_V4, BN / 4, T::THREADS, T::LDB>(Bs[cur ^ 1], rb, tid);
        }
        __syncthreads();
    }

    // Epilogue: accumulator register r of lane l holds block row
    // 8*(r/4) + 4*(l/32) + r%4, block column l%32.
#pragma unroll
    for (int i = 0; i < T::TM; ++i) {
#pragma unroll
        for (int j = 0; j < T::TN; ++j) {
            const int64_t col = n0 + wn + 32 * j + lcol;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int64_t row = m0 + wm + 32 * i + 8 * (r >> 2) + 4 * lrow + (r & 3);
                if (row < M && col < N) {
                    float* w = W + row * N + col;
                    *w = fmaf(-lr, acc[i][j][r], *w);
                }
            }
        }
    }
}

template <int BM, int BN, int BK, int WM, int WN>
hipError_t launch_cfg(float* W, const float* U, const float* V, int64_t M, int64_t N, int64_t K,
                      float lr, bool vec, hipStream_t stream)
{
    using T = SfTile<BM, BN, BK, WM, WN>;
    const int64_t tiles_m = (M + BM - 1) / BM;
    const int64_t tiles_n = (N + BN - 1) / BN;
    const int64_t tiles = tiles_m * tiles_n;
    if (tiles > INT32_MAX || tiles_n > INT32_MAX)
        return hipErrorInvalidValue;
    if (vec)
        sf_apply_kernel<BM, BN, BK, WM, WN, true><<<static_cast<int>(tiles), T::THREADS, 0, stream>>>(
            W, U, V, M, N, K, lr, static_cast<int>(tiles_n));
    else
        sf_apply_kernel<BM, BN, BK, WM, WN, false><<<static_cast<int>(tiles), T::THREADS, 0, stream>>>(
            W, U, V, M, N, K, lr, static_cast<int>(tiles_n));
    return hipGetLastError();
}

}  // namespace

hipError_t launch_sf_apply(float* W, const float* U, const float* V,
                           int64_t M, int64_t N, int64_t K, float lr, hipStream_t stream)
{
    const bool vec = (M % 4 == 0) && (N % 4 == 0) && aligned16(U) && aligned16(V);
    return launch_cfg<128, 128, 16, 64, 64>(W, U, V, M, N, K, lr, vec, stream);
}

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

}  // namespace poseidon

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
