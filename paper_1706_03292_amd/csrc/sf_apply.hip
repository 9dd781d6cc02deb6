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
// matrix cores work on the current one, and each wave reads the operand
// fragments of the next MFMA step while the current one runs.  Each wave owns a
// WM x WN sub-block (WM/32 x WN/32 MFMA blocks).
//
// The SGD update is the epilogue: W is read once and written once, straight
// from the accumulators, so the gradient is never materialised.  On tiles that
// lie wholly inside W the epilogue's loads are issued before the last K step
// (their latency hides behind its MFMAs) and carry no per-element branch.
//
// Tile order: the hardware hands consecutive workgroups to the 8 XCDs in turn,
// and each XCD has its own L2.  Workgroup ids are remapped so that every XCD
// owns one contiguous run of tiles, walked a group of tile rows at a time, so
// the tiles an XCD runs at the same time share U and V panels in its L2.
#include <vector>

#include "common.h"

namespace poseidon {
namespace {

typedef float f16v __attribute__((ext_vector_type(16)));
typedef float f4u __attribute__((ext_vector_type(4), aligned(4)));   // 16 bytes, 4-byte aligned

constexpr int LDS_PAD = 4;    // floats of padding per LDS row (keeps 16-byte alignment)
constexpr int NUM_XCD = 8;    // MI355X: 8 accelerator complex dies, one L2 each

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

// Load one BK x (4*COLS4) slice of a K-major operand X (row length ld = its
// number of columns) into registers: group j of this thread covers row
// g / COLS4 and columns 4*(g % COLS4) .. +3 with g = tid + j*THREADS.
// Out-of-range rows/columns read as 0, which adds nothing to the sum.  Every
// group is one 16-byte load: with VEC (ld % 4 == 0, X 16-byte aligned) a group
// is wholly in or out; otherwise rows start at any 4-byte boundary (global
// loads of several dwords need only 4-byte alignment) and only a group that
// runs past the end of its row is read element by element.
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
        const bool kin = k < rows;
        if constexpr (VEC) {
            r[j] = (kin && c < ld) ? *reinterpret_cast<const f4*>(src) : f4{0.f, 0.f, 0.f, 0.f};
        } else if (kin && c + 3 < ld) {
            r[j] = *reinterpret_cast<const f4u*>(src);
        } else {
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

// Workgroup id -> (tile row, tile column): contiguous runs per XCD, GM tile
// rows at a time inside a run (GM = 0: plain row-major order, no remap).
template <int GM>
__device__ inline void tile_coords(int bid, int tiles, int tiles_m, int tiles_n, int& tm, int& tn)
{
    if constexpr (GM == 0) {
        tm = bid / tiles_n;
        tn = bid % tiles_n;
    } else {
        const int q = tiles / NUM_XCD, r = tiles % NUM_XCD;
        const int x = bid % NUM_XCD, j = bid / NUM_XCD;
        const int t = x * q + (x < r ? x : r) + j;
        const int per_group = GM * tiles_n;
        const int g = t / per_group;
        const int first_m = g * GM;
        const int rows = (tiles_m - first_m) < GM ? (tiles_m - first_m) : GM;
        const int in = t - g * per_group;
        tm = first_m + in % rows;
        tn = in / rows;
    }
}

// One BK-deep step of the contraction out of LDS: each wave reads its U and V
// fragments for MFMA step kk+2 while the matrix cores work on step kk (the
// compiler interleaves the reads with the MFMAs; pinning other orders with
// scheduling barriers or priorities measured no faster).
template <int BK, int LDA, int LDB, int TM, int TN>
__device__ inline void mma_step(f16v (&acc)[TM][TN], const float* a_s, const float* b_s)
{
    float a[2][TM], b[2][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
        a[0][i] = a_s[32 * i];
#pragma unroll
    for (int j = 0; j < TN; ++j)
        b[0][j] = b_s[32 * j];
#pragma unroll
    for (int kk = 0; kk < BK; kk += 2) {
        const int c = (kk >> 1) & 1;
        if (kk + 2 < BK) {
#pragma unroll
            for (int i = 0; i < TM; ++i)
                a[c ^ 1][i] = a_s[(kk + 2) * LDA + 32 * i];
#pragma unroll
            for (int j = 0; j < TN; ++j)
                b[c ^ 1][j] = b_s[(kk + 2) * LDB + 32 * j];
        }
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[c][i], b[c][j], acc[i][j], 0, 0, 0);
    }
}

// Buffer resource word 3 for raw (untyped) dword accesses on CDNA.  The raw
// buffer builtins move 32-bit integers: values are bit-cast, never converted.
constexpr int BUF_RSRC_WORD3 = 0x00020000;

// One BM x BN tile of W: the whole K loop and the fused update.  EPI: MFMA
// blocks of W (16 values per lane each) read per epilogue chunk.  The
// double-buffered K slices live in the caller's LDS arrays (As: 2 x BK*LDA
// floats, Bs: 2 x BK*LDB; buffer b starts at b*BK*LD), so that several
// inlined variants share one allocation.  Always inlined: as a called function it would keep both the
// 16-byte and the scalar operand loads and pay the call convention.
//
// MOM: the layer keeps a momentum buffer (same shape as W): the epilogue
// updates buf <- mu*buf + dW and W <- W - lr*buf, and K may be 0 (a step on
// the buffer alone).
template <int BM, int BN, int BK, int WM, int WN, bool VEC_A, bool VEC_B, bool PREFETCH_W, int EPI, bool HUGE_N,
          bool MOM = false>
__device__ __forceinline__ void sf_tile(
    float* As, float* Bs, float* __restrict__ W, const float* __restrict__ U, const float* __restrict__ V,
    int64_t M, int64_t N, int64_t K, float lr, int tm, int tn, float* __restrict__ buf = nullptr, float mu = 0.f)
{
    using T = SfTile<BM, BN, BK, WM, WN>;
    constexpr int SA = BK * T::LDA, SB = BK * T::LDB;   // floats per LDS buffer

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int64_t m0 = static_cast<int64_t>(tm) * BM;
    const int64_t n0 = static_cast<int64_t>(tn) * BN;
    const int wm = (wave / T::NWN) * WM;
    const int wn = (wave % T::NWN) * WN;
    const int lrow = lane >> 5;        // which of the two k of an MFMA step this lane supplies
    const int lcol = lane & 31;
    const bool interior = (m0 + BM <= M) && (n0 + BN <= N);

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

    load_panel<T::A_V4, BM / 4, T::THREADS, VEC_A>(ra, U, M, K, 0, m0, tid);
    load_panel<T::B_V4, BN / 4, T::THREADS, VEC_B>(rb, V, N, K, 0, n0, tid);
    store_panel<T::A_V4, BM / 4, T::THREADS, T::LDA>(As, ra, tid);
    store_panel<T::B_V4, BN / 4, T::THREADS, T::LDB>(Bs, rb, tid);
    __syncthreads();

    const int a_off = lrow * T::LDA + wm + lcol;
    const int b_off = lrow * T::LDB + wn + lcol;
    for (int64_t kt = 0; kt + 1 < nkt; ++kt) {
        const int cur = static_cast<int>(kt & 1);
        load_panel<T::A_V4, BM / 4, T::THREADS, VEC_A>(ra, U, M, K, (kt + 1) * BK, m0, tid);
        load_panel<T::B_V4, BN / 4, T::THREADS, VEC_B>(rb, V, N, K, (kt + 1) * BK, n0, tid);
        mma_step<BK, T::LDA, T::LDB, T::TM, T::TN>(acc, As + cur * SA + a_off, Bs + cur * SB + b_off);
        store_panel<T::A_V4, BM / 4, T::THREADS, T::LDA>(As + (cur ^ 1) * SA, ra, tid);
        store_panel<T::B_V4, BN / 4, T::THREADS, T::LDB>(Bs + (cur ^ 1) * SB, rb, tid);
        __syncthreads();
    }
    const int last = static_cast<int>((nkt - 1) & 1);

    // Epilogue: accumulator register r of lane l holds block row
    // 8*(r/4) + 4*(l/32) + r%4, block column l%32.
    if constexpr (MOM) {
        if (nkt > 0)
            mma_step<BK, T::LDA, T::LDB, T::TM, T::TN>(acc, As + last * SA + a_off, Bs + last * SB + b_off);
        const int rows_left = static_cast<int>(M - m0 < BM ? M - m0 : BM);
        const int cols_left = static_cast<int>(N - n0 < BN ? N - n0 : BN);
        if constexpr (!HUGE_N) {
            // Half an MFMA block (8 values per lane) at a time: W and buf
            // loads in flight together, then both stores.  Elements outside
            // W read the tile origin (inside W) and are not stored.
            const int64_t first = m0 * N + n0;
            const int64_t avail = (M * N - first) * 4;
            const int nrec = static_cast<int>(avail < 0x7fffffff ? avail : 0x7fffffff);
            const __amdgpu_buffer_rsrc_t wr =
                __builtin_amdgcn_make_buffer_rsrc(W + first, static_cast<short>(0), nrec, BUF_RSRC_WORD3);
            const __amdgpu_buffer_rsrc_t br =
                __builtin_amdgcn_make_buffer_rsrc(buf + first, static_cast<short>(0), nrec, BUF_RSRC_WORD3);
            const int ni = static_cast<int>(N);
#pragma unroll
            for (int i = 0; i < T::TM; ++i) {
#pragma unroll
                for (int j = 0; j < T::TN; ++j) {
                    const int col = wn + 32 * j + lcol;
#pragma unroll
                    for (int h = 0; h < 16; h += 8) {
                        float wv[8], bv[8];
                        int off[8];
#pragma unroll
                        for (int q = 0; q < 8; ++q) {
                            const int r = h + q;
                            const int row = wm + 32 * i + 8 * (r >> 2) + 4 * lrow + (r & 3);
                            off[q] = (row < rows_left && col < cols_left) ? (row * ni + col) * 4 : 0;
                            wv[q] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(wr, off[q], 0, 0));
                            bv[q] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(br, off[q], 0, 0));
                        }
#pragma unroll
                        for (int q = 0; q < 8; ++q) {
                            const int r = h + q;
                            const int row = wm + 32 * i + 8 * (r >> 2) + 4 * lrow + (r & 3);
                            if (row < rows_left && col < cols_left) {
                                const float nb = fmaf(mu, bv[q], acc[i][j][r]);
                                __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, nb), br, off[q], 0, 0);
                                __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, fmaf(-lr, nb, wv[q])), wr,
                                                                      off[q], 0, 0);
                            }
                        }
                        __builtin_amdgcn_sched_barrier(0);
                    }
                }
            }
        } else {
#pragma unroll
            for (int i = 0; i < T::TM; ++i) {
#pragma unroll
                for (int j = 0; j < T::TN; ++j) {
                    const int col = wn + 32 * j + lcol;
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int row = wm + 32 * i + 8 * (r >> 2) + 4 * lrow + (r & 3);
                        if (row < rows_left && col < cols_left) {
                            const int64_t e = (m0 + row) * N + n0 + col;
                            const float nb = fmaf(mu, buf[e], acc[i][j][r]);
                            buf[e] = nb;
                            W[e] = fmaf(-lr, nb, W[e]);
                        }
                    }
                }
            }
        }
        return;
    }
    if constexpr (!HUGE_N) {
        // Buffer-addressed epilogue: byte offsets from the tile's first
        // element fit in 31 bits (the host picks HUGE_N otherwise).
        const int64_t first = m0 * N + n0;
        const int64_t avail = (M * N - first) * 4;
        const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
            W + first, static_cast<short>(0), static_cast<int>(avail < 0x7fffffff ? avail : 0x7fffffff),
            BUF_RSRC_WORD3);
        const int ni = static_cast<int>(N);
        const int voff = ((wm + 4 * lrow) * ni + wn + lcol) * 4;
        const int n4 = ni * 4;
        constexpr int NB = T::TM * T::TN;
        constexpr int CH = NB < EPI ? NB : EPI;
        static_assert(NB % CH == 0, "epilogue chunking");
        // W is read in chunks of up to EPI MFMA blocks (16 values per block
        // and lane, all loads of a chunk in flight together).  Interior tiles
        // use one shared lane offset and uniform row offsets; with PREFETCH_W
        // their first chunk is loaded before the last step's MFMAs so that the
        // latency hides behind them.
        float wv[CH][16];
        if (PREFETCH_W && interior) {
#pragma unroll
            for (int c = 0; c < CH; ++c) {
                const int i = c / T::TN, j = c % T::TN;
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    wv[c][r] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                        wr, voff + 128 * j, (32 * i + 8 * (r >> 2) + (r & 3)) * n4, 0));
            }
        }
        mma_step<BK, T::LDA, T::LDB, T::TM, T::TN>(acc, As + last * SA + a_off, Bs + last * SB + b_off);
        if (interior) {
#pragma unroll
            for (int c0 = 0; c0 < NB; c0 += CH) {
                if (c0 > 0 || !PREFETCH_W) {
#pragma unroll
                    for (int c = 0; c < CH; ++c) {
                        const int i = (c0 + c) / T::TN, j = (c0 + c) % T::TN;
#pragma unroll
                        for (int r = 0; r < 16; ++r)
                            wv[c][r] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                wr, voff + 128 * j, (32 * i + 8 * (r >> 2) + (r & 3)) * n4, 0));
                    }
                }
#pragma unroll
                for (int c = 0; c < CH; ++c) {
                    const int i = (c0 + c) / T::TN, j = (c0 + c) % T::TN;
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        __builtin_amdgcn_raw_buffer_store_b32(
                            __builtin_bit_cast(unsigned, fmaf(-lr, acc[i][j][r], wv[c][r])), wr, voff + 128 * j,
                            (32 * i + 8 * (r >> 2) + (r & 3)) * n4, 0);
                }
            }
        } else {
            // Ragged edge tile: every element gets its own lane offset; an
            // element outside W loads the tile's first element instead (always
            // inside W, value unused) and is not stored.
            const int rows_left = static_cast<int>(M - m0 < BM ? M - m0 : BM);
            const int cols_left = static_cast<int>(N - n0 < BN ? N - n0 : BN);
#pragma unroll
            for (int i = 0; i < T::TM; ++i) {
#pragma unroll
                for (int j = 0; j < T::TN; ++j) {
                    const int col = wn + 32 * j + lcol;
                    float ev[16];
                    int off[16];
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int row = wm + 32 * i + 8 * (r >> 2) + 4 * lrow + (r & 3);
                        off[r] = (row < rows_left && col < cols_left) ? (row * ni + col) * 4 : 0;
                        ev[r] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(wr, off[r], 0, 0));
                    }
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int row = wm + 32 * i + 8 * (r >> 2) + 4 * lrow + (r & 3);
                        if (row < rows_left && col < cols_left)
                            __builtin_amdgcn_raw_buffer_store_b32(
                                __builtin_bit_cast(unsigned, fmaf(-lr, acc[i][j][r], ev[r])), wr, off[r], 0, 0);
                    }
                    // One MFMA block at a time: keeps the scheduler from
                    // hoisting every block's loads and offsets together.
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
        }
    } else {
        // Rows so long that tile offsets need 64 bits: plain guarded accesses.
        mma_step<BK, T::LDA, T::LDB, T::TM, T::TN>(acc, As + last * SA + a_off, Bs + last * SB + b_off);
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
}

template <int BM, int BN, int BK, int WM, int WN, bool VEC_A, bool VEC_B, bool PREFETCH_W, int OCC, int EPI,
          int GM, bool HUGE_N>
__global__ __launch_bounds__((BM / WM) * (BN / WN) * 64)
__attribute__((amdgpu_waves_per_eu(OCC, OCC))) void sf_apply_kernel(
    float* __restrict__ W, const float* __restrict__ U, const float* __restrict__ V,
    int64_t M, int64_t N, int64_t K, float lr, int tiles_m, int tiles_n)
{
    using T = SfTile<BM, BN, BK, WM, WN>;
    __shared__ float As[2 * BK * T::LDA];
    __shared__ float Bs[2 * BK * T::LDB];
    int tm, tn;
    tile_coords<GM>(blockIdx.x, tiles_m * tiles_n, tiles_m, tiles_n, tm, tn);
    sf_tile<BM, BN, BK, WM, WN, VEC_A, VEC_B, PREFETCH_W, EPI, HUGE_N>(As, Bs, W, U, V, M, N, K, lr, tm, tn);
}

// The layer keeps a momentum buffer (poseidon_sf_apply_momentum).
template <int BM, int BN, int BK, int WM, int WN, bool VEC_A, bool VEC_B, int OCC, bool HUGE_N>
__global__ __launch_bounds__((BM / WM) * (BN / WN) * 64)
__attribute__((amdgpu_waves_per_eu(OCC, OCC))) void sf_apply_mom_kernel(
    float* __restrict__ W, float* __restrict__ buf, const float* __restrict__ U, const float* __restrict__ V,
    int64_t M, int64_t N, int64_t K, float lr, float mu, int tiles_m, int tiles_n)
{
    using T = SfTile<BM, BN, BK, WM, WN>;
    __shared__ float As[2 * BK * T::LDA];
    __shared__ float Bs[2 * BK * T::LDB];
    int tm, tn;
    tile_coords<8>(blockIdx.x, tiles_m * tiles_n, tiles_m, tiles_n, tm, tn);
    sf_tile<BM, BN, BK, WM, WN, VEC_A, VEC_B, false, 1, HUGE_N, true>(As, Bs, W, U, V, M, N, K, lr, tm, tn, buf, mu);
}

// ---------------------------------------------------------------------------
// Several layers in one launch (same K): one tile list, so the chip is filled
// by the tiles of the next layer while the last ones of a layer finish,
// instead of every layer ending in a partly idle round.  Layer descriptors
// travel by value in the kernel arguments; the XCD-aware order runs over the
// combined list (layer by layer, in the order given), and inside a layer tile
// rows are walked 8 at a time.
// ---------------------------------------------------------------------------
struct SfBatchItem {
    float* W;
    const float* U;
    const float* V;
    int64_t M;
    int64_t N;
    int32_t first_tile;
    int32_t tiles_m;
    int32_t tiles_n;
    int32_t vec;   // bit 0: U rows 16-byte loadable, bit 1: V rows
};

struct SfBatchArgs {
    SfBatchItem item[SF_BATCH_MAX];
    int32_t count;
    int32_t total_tiles;
};

template <int BM, int BN, int BK, int WM, int WN, bool PREFETCH_W, int OCC, int EPI>
__global__ __launch_bounds__((BM / WM) * (BN / WN) * 64)
__attribute__((amdgpu_waves_per_eu(OCC, OCC))) void sf_apply_batch_kernel(const SfBatchArgs args, int64_t K,
                                                                           float lr)
{
    const int tiles = args.total_tiles;
    const int q = tiles / NUM_XCD, r = tiles % NUM_XCD;
    const int x = blockIdx.x % NUM_XCD, j = blockIdx.x / NUM_XCD;
    const int t = x * q + (x < r ? x : r) + j;
    int l = 0;
    while (l + 1 < args.count && t >= args.item[l + 1].first_tile)
        ++l;
    const int local = t - args.item[l].first_tile;
    const int tiles_m = args.item[l].tiles_m, tiles_n = args.item[l].tiles_n;
    constexpr int G = 8;
    const int per_group = G * tiles_n;
    const int g = local / per_group;
    const int first_m = g * G;
    const int rows = (tiles_m - first_m) < G ? (tiles_m - first_m) : G;
    const int in = local - g * per_group;
    using T = SfTile<BM, BN, BK, WM, WN>;
    __shared__ float As[2 * BK * T::LDA];
    __shared__ float Bs[2 * BK * T::LDB];
    const SfBatchItem& it = args.item[l];
    const int tm = first_m + in % rows, tn = in / rows;
    // The operand-load variant is uniform per layer: four inlined copies.
    switch (it.vec & 3) {
    case 3:
        sf_tile<BM, BN, BK, WM, WN, true, true, PREFETCH_W, EPI, false>(As, Bs, it.W, it.U, it.V, it.M, it.N, K, lr,
                                                                        tm, tn);
        break;
    case 2:
        sf_tile<BM, BN, BK, WM, WN, false, true, PREFETCH_W, EPI, false>(As, Bs, it.W, it.U, it.V, it.M, it.N, K, lr,
                                                                         tm, tn);
        break;
    case 1:
        sf_tile<BM, BN, BK, WM, WN, true, false, PREFETCH_W, EPI, false>(As, Bs, it.W, it.U, it.V, it.M, it.N, K, lr,
                                                                         tm, tn);
        break;
    default:
        sf_tile<BM, BN, BK, WM, WN, false, false, PREFETCH_W, EPI, false>(As, Bs, it.W, it.U, it.V, it.M, it.N, K,
                                                                          lr, tm, tn);
        break;
    }
}

template <int BM, int BN, int BK, int WM, int WN, bool PREF, int OCC, int EPI, int GM, bool VA, bool VB>
void launch_kernel(int tiles, int tiles_m, int tiles_n, float* W, const float* U, const float* V,
                   int64_t M, int64_t N, int64_t K, float lr, hipStream_t stream)
{
    // The buffer-addressed epilogue needs every byte offset inside a tile,
    // ((BM-1)*N + BN) * 4, to fit in a signed 32-bit offset.
    constexpr int NT = SfTile<BM, BN, BK, WM, WN>::THREADS;
    if ((static_cast<int64_t>(BM) * N + BN) * 4 < 0x7fffffffLL)
        sf_apply_kernel<BM, BN, BK, WM, WN, VA, VB, PREF, OCC, EPI, GM, false><<<tiles, NT, 0, stream>>>(
            W, U, V, M, N, K, lr, tiles_m, tiles_n);
    else
        sf_apply_kernel<BM, BN, BK, WM, WN, VA, VB, PREF, OCC, EPI, GM, true><<<tiles, NT, 0, stream>>>(
            W, U, V, M, N, K, lr, tiles_m, tiles_n);
}

template <int BM, int BN, int BK, int WM, int WN, bool PREF, int OCC, int EPI = 4, int GM = 8>
hipError_t launch_cfg(float* W, const float* U, const float* V, int64_t M, int64_t N, int64_t K,
                      float lr, hipStream_t stream)
{
    const int64_t tiles_m = (M + BM - 1) / BM;
    const int64_t tiles_n = (N + BN - 1) / BN;
    const int64_t tiles = tiles_m * tiles_n;
    if (tiles > INT32_MAX)
        return hipErrorInvalidValue;
    const bool va = (M % 4 == 0) && aligned16(U);
    const bool vb = (N % 4 == 0) && aligned16(V);
    const int t = static_cast<int>(tiles), tmi = static_cast<int>(tiles_m), tni = static_cast<int>(tiles_n);
    if (va && vb)
        launch_kernel<BM, BN, BK, WM, WN, PREF, OCC, EPI, GM, true, true>(t, tmi, tni, W, U, V, M, N, K, lr, stream);
    else if (va)
        launch_kernel<BM, BN, BK, WM, WN, PREF, OCC, EPI, GM, true, false>(t, tmi, tni, W, U, V, M, N, K, lr, stream);
    else if (vb)
        launch_kernel<BM, BN, BK, WM, WN, PREF, OCC, EPI, GM, false, true>(t, tmi, tni, W, U, V, M, N, K, lr, stream);
    else
        launch_kernel<BM, BN, BK, WM, WN, PREF, OCC, EPI, GM, false, false>(t, tmi, tni, W, U, V, M, N, K, lr, stream);
    return hipGetLastError();
}

}  // namespace

// Tile choice: 128 x 128 workgroup tiles (64 x 64 per wave, W prefetched,
// 4 waves per SIMD) when the layer has at least two such tiles per CU;
// otherwise 64 x 64 tiles so that small layers still fill the chip.
hipError_t launch_sf_apply(float* W, const float* U, const float* V,
                           int64_t M, int64_t N, int64_t K, float lr, hipStream_t stream)
{
    const int64_t big_tiles = ((M + 127) / 128) * ((N + 127) / 128);
    if (big_tiles >= 2 * static_cast<int64_t>(device_cu_count()))
        return launch_cfg<128, 128, 16, 64, 64, true, 4, 1, 8>(W, U, V, M, N, K, lr, stream);
    return launch_cfg<64, 64, 32, 32, 32, true, 4, 1, 8>(W, U, V, M, N, K, lr, stream);
}

namespace {

template <int BM, int BN, int BK, int WM, int WN, bool VA, bool VB>
void launch_mom(float* W, float* buf, const float* U, const float* V, int64_t M, int64_t N, int64_t K, float lr,
                float mu, int tiles, int tiles_m, int tiles_n, hipStream_t stream)
{
    constexpr int NT = SfTile<BM, BN, BK, WM, WN>::THREADS;
    if ((static_cast<int64_t>(BM) * N + BN) * 4 < 0x7fffffffLL)
        sf_apply_mom_kernel<BM, BN, BK, WM, WN, VA, VB, 4, false><<<tiles, NT, 0, stream>>>(
            W, buf, U, V, M, N, K, lr, mu, tiles_m, tiles_n);
    else
        sf_apply_mom_kernel<BM, BN, BK, WM, WN, VA, VB, 4, true><<<tiles, NT, 0, stream>>>(
            W, buf, U, V, M, N, K, lr, mu, tiles_m, tiles_n);
}

template <int BM, int BN, int BK, int WM, int WN>
hipError_t launch_mom_cfg(float* W, float* buf, const float* U, const float* V, int64_t M, int64_t N, int64_t K,
                          float lr, float mu, hipStream_t stream)
{
    const int64_t tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
    if (tiles_m * tiles_n > INT32_MAX)
        return hipErrorInvalidValue;
    const int t = static_cast<int>(tiles_m * tiles_n), tmi = static_cast<int>(tiles_m),
              tni = static_cast<int>(tiles_n);
    const bool va = (M % 4 == 0) && aligned16(U), vb = (N % 4 == 0) && aligned16(V);
    if (va && vb)
        launch_mom<BM, BN, BK, WM, WN, true, true>(W, buf, U, V, M, N, K, lr, mu, t, tmi, tni, stream);
    else if (va)
        launch_mom<BM, BN, BK, WM, WN, true, false>(W, buf, U, V, M, N, K, lr, mu, t, tmi, tni, stream);
    else if (vb)
        launch_mom<BM, BN, BK, WM, WN, false, true>(W, buf, U, V, M, N, K, lr, mu, t, tmi, tni, stream);
    else
        launch_mom<BM, BN, BK, WM, WN, false, false>(W, buf, U, V, M, N, K, lr, mu, t, tmi, tni, stream);
    return hipGetLastError();
}

}  // namespace

// The same tile choice as launch_sf_apply.
hipError_t launch_sf_apply_momentum(float* W, float* buf, const float* U, const float* V, int64_t M, int64_t N,
                                    int64_t K, float lr, float mu, hipStream_t stream)
{
    const int64_t big_tiles = ((M + 127) / 128) * ((N + 127) / 128);
    if (big_tiles >= 2 * static_cast<int64_t>(device_cu_count()))
        return launch_mom_cfg<128, 128, 16, 64, 64>(W, buf, U, V, M, N, K, lr, mu, stream);
    return launch_mom_cfg<64, 64, 32, 32, 32>(W, buf, U, V, M, N, K, lr, mu, stream);
}

// Grouped launch: every layer whose tile offsets fit 32 bits joins one tile
// list (128 x 128 tiles) when the group has at least two tiles per CU; the
// others, and groups too small to fill the chip, take per-layer launches.
hipError_t launch_sf_apply_batch(const SfTensor* t, int32_t count, int64_t K, float lr, hipStream_t stream)
{
    constexpr int BM = 128, BN = 128;
    std::vector<int32_t> grouped;
    int64_t tiles = 0;
    for (int32_t i = 0; i < count; ++i) {
        if (t[i].M == 0 || t[i].N == 0 || K == 0)
            continue;
        const int64_t tl = ((t[i].M + BM - 1) / BM) * ((t[i].N + BN - 1) / BN);
        if ((static_cast<int64_t>(BM) * t[i].N + BN) * 4 < 0x7fffffffLL && tiles + tl <= INT32_MAX) {
            grouped.push_back(i);
            tiles += tl;
        } else {
            const hipError_t e = launch_sf_apply(t[i].W, t[i].U, t[i].V, t[i].M, t[i].N, K, lr, stream);
            if (e != hipSuccess)
                return e;
        }
    }
    if (tiles < 2 * static_cast<int64_t>(device_cu_count())) {
        for (int32_t i : grouped) {
            const hipError_t e = launch_sf_apply(t[i].W, t[i].U, t[i].V, t[i].M, t[i].N, K, lr, stream);
            if (e != hipSuccess)
                return e;
        }
        return hipSuccess;
    }
    for (size_t g0 = 0; g0 < grouped.size(); g0 += SF_BATCH_MAX) {
        SfBatchArgs a{};
        int32_t first = 0;
        for (size_t g = g0; g < grouped.size() && g < g0 + SF_BATCH_MAX; ++g) {
            const SfTensor& x = t[grouped[g]];
            SfBatchItem& it = a.item[a.count++];
            it.W = x.W;
            it.U = x.U;
            it.V = x.V;
            it.M = x.M;
            it.N = x.N;
            it.tiles_m = static_cast<int32_t>((x.M + BM - 1) / BM);
            it.tiles_n = static_cast<int32_t>((x.N + BN - 1) / BN);
            it.first_tile = first;
            it.vec = ((x.M % 4 == 0) && aligned16(x.U) ? 1 : 0) | ((x.N % 4 == 0) && aligned16(x.V) ? 2 : 0);
            first += it.tiles_m * it.tiles_n;
        }
        a.total_tiles = first;
        sf_apply_batch_kernel<BM, BN, 16, 64, 64, true, 4, 1><<<first, 256, 0, stream>>>(a, K, lr);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess)
            return e;
    }
    return hipSuccess;
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

extern "C" int poseidon_sf_apply_batch(const poseidon_sf_tensor* layers, int32_t count, int64_t K, float lr,
                                       hipStream_t stream)
{
    if (count < 0 || (count > 0 && !layers) || K < 0)
        return POSEIDON_ERR_INVALID_ARG;
    for (int32_t i = 0; i < count; ++i) {
        const poseidon_sf_tensor& x = layers[i];
        const int rc = poseidon::check_sf_args(x.W, x.U, x.V, x.M, x.N, K);
        if (rc != POSEIDON_OK)
            return rc;
        for (int32_t j = 0; j < count; ++j) {   // no W may overlap another layer's W, U or V
            if (j == i)
                continue;
            const poseidon_sf_tensor& y = layers[j];
            const int64_t wb = x.M * x.N * 4;
            if (poseidon::overlaps(x.W, wb, y.W, y.M * y.N * 4) || poseidon::overlaps(x.W, wb, y.U, K * y.M * 4) ||
                poseidon::overlaps(x.W, wb, y.V, K * y.N * 4))
                return POSEIDON_ERR_INVALID_ARG;
        }
    }
    static_assert(sizeof(poseidon_sf_tensor) == sizeof(poseidon::SfTensor), "descriptor layout");
    return poseidon::launch_sf_apply_batch(reinterpret_cast<const poseidon::SfTensor*>(layers), count, K, lr,
                                           stream) == hipSuccess
               ? POSEIDON_OK
               : POSEIDON_ERR_HIP;
}
