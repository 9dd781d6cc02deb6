// Sufficient-factor reconstruction fused with the SGD step (Sec. 2.1
// "Sufficient Factor Broadcasting"; Eq. 1, Eq. 2):
//
//   W[m][n] <- W[m][n] - lr * sum_{k<K} U[k][m] * V[k][n]
//
// A dense contraction of depth K = P*B with both operands stored K-major
// (row k of U is u_k, row k of V is v_k), on the matrix cores in 32x32 output
// blocks (64 lanes, 16 fp32 accumulator registers per lane).  By default the
// fp32 products are formed on the bf16 matrix cores (v_mfma_f32_32x32x16_bf16)
// from an exact three-part bf16 split of each operand, six part products per
// fp32 product (see "Split-bf16 products" below); the fp32 matrix cores
// (v_mfma_f32_32x32x2_f32) are the alternative the caller can choose, and the
// register-staged variant for very large operands always uses them.
//
// Tiling: a workgroup owns a BM x BN block of W and loops over K in steps of
// BK; each wave owns a WM x WN sub-block (WM/32 x WN/32 MFMA blocks): 256 x
// 128 tiles of 128 x 64 sub-blocks for large layers with the split products,
// else 128 x 128 tiles of 64 x 64, or 64 x 64 tiles of 32 x 32 for small ones.  The
// K-slices U[k0:k0+BK, m0:m0+BM] and V[k0:k0+BK, n0:n0+BN] go straight from
// global memory into LDS with the gfx950 LDS-direct buffer loads (each lane
// moves 16 bytes, a wave instruction fills 1 KB of LDS), two slices in
// flight: the next slice streams in while the matrix cores work on the
// current one, with no register staging and no LDS store instructions.
// Out-of-range operand reads are handled by the buffer resource's range
// check (they read 0), so the K tail needs no branch; reads past the end of a
// row in the last tile column fetch the next row's values, which only feed
// outputs outside W that are never stored.  Inside a slice, 16-byte chunks of
// odd rows are stored with their chunk index XOR 8, so the two half-waves of
// an MFMA operand read (rows k and k+1) hit disjoint LDS banks.
//
// The SGD update is the epilogue: W is read once and written once, straight
// from the accumulators, so the gradient is never materialised, with
// non-temporal accesses that leave the L2 to the operand panels.  On tiles
// that lie wholly inside W the first block of W is loaded before the last K
// step (its latency hides behind that step's MFMAs) and no access carries a
// per-element branch.
//
// Tile order: the hardware hands consecutive workgroups to the 8 XCDs in turn,
// and each XCD has its own L2.  Workgroup ids are remapped so that every XCD
// owns one contiguous run of tiles, walked a group of tile rows at a time, so
// the tiles an XCD runs at the same time share U and V panels in its L2.
//
// Operands whose byte offsets do not fit the 32-bit buffer offsets (K*M or
// K*N of 2^29 elements and more, or rows over 4,194,303 elements) take a
// register-staged variant of the same tile with 64-bit addressing.
//
// Launch forms: one workgroup per tile (a layer, or several layers of one K
// as one grouped tile list), or a spread launch whose few workgroups each
// walk several tiles, for running the rebuild thin beside longer PS work.
#include <atomic>
#include <vector>

#include "common.h"

namespace poseidon {
namespace {

typedef float f16v __attribute__((ext_vector_type(16)));
typedef float f4u __attribute__((ext_vector_type(4), aligned(4)));   // 16 bytes, 4-byte aligned
typedef __attribute__((address_space(3))) void lds_void;

constexpr int NUM_XCD = 8;    // MI355X: 8 accelerator complex dies, one L2 each

// Buffer resource word 3 for raw (untyped) dword accesses on CDNA.  The raw
// buffer builtins move 32-bit integers: values are bit-cast, never converted.
constexpr int BUF_RSRC_WORD3 = 0x00020000;

template <int BM, int BN, int BK, int WM, int WN>
struct SfTile {
    static constexpr int NWM = BM / WM;
    static constexpr int NWN = BN / WN;
    static constexpr int THREADS = NWM * NWN * 64;
    static constexpr int TM = WM / 32;
    static constexpr int TN = WN / 32;
    static_assert(BM % WM == 0 && BN % WN == 0 && WM % 32 == 0 && WN % 32 == 0, "tile");
    static_assert(BK % 2 == 0, "MFMA depth is 2");
};

// Waves per SIMD a tile shape is compiled for: 4 (at most 128 VGPRs a wave)
// for wave sub-blocks up to 64 x 64, else 2 (256 VGPRs: the accumulators of a
// 128 x 64 sub-block alone take 128).
template <int WM, int WN>
struct SfOcc {
    static constexpr int W = WM * WN > 64 * 64 ? 2 : 4;
};

// Tile shapes (workgroup BM x BN, K-slices of BK, wave sub-block WM x WN).
// Split-bf16 layers with at least four 256 x 128 tiles per CU take that tile
// (two waves per SIMD, each on a 128 x 64 sub-block: 48 MFMAs per 48 split
// operand values instead of 24 per 32); otherwise, and for fp32 MFMA layers,
// 128 x 128 tiles when there are at least two per CU, else 64 x 64.
struct Big {
    static constexpr int BM = 256, BN = 128, BK = 16, WM = 128, WN = 64;
};
struct Mid {
    static constexpr int BM = 128, BN = 128, BK = 16, WM = 64, WN = 64;
};
struct Small {
    static constexpr int BM = 64, BN = 64, BK = 32, WM = 32, WN = 32;
};
constexpr int64_t BIG_TILES_PER_CU = 4, MID_TILES_PER_CU = 2;

// Tile rows an XCD's run walks at a time: 8 of 128 rows (the 128 workgroups
// an XCD runs together then read 8 U and 16 V panels, the fewest for 128 such
// tiles), 4 of 256 rows (its 64 workgroups of 256 x 128 read 4 U and 16 V
// panels: the VGG19-22K grouped launch fetched 1.50 GB from memory against
// 1.81 GB with 8 rows, 1.85 with 2 and 2.57 with 16, in equal time).
template <int BM>
struct TileRows {
    static constexpr int G = BM >= 256 ? 4 : 8;
};

// Workgroup id -> (tile row, tile column): contiguous runs per XCD, GM tile
// rows at a time inside a run.
template <int GM>
__device__ inline void tile_coords(int bid, int tiles, int tiles_m, int tiles_n, int& tm, int& tn)
{
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

template <int TM, int TN>
__device__ __forceinline__ void zero_acc(f16v (&acc)[TM][TN])
{
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                acc[i][j][r] = 0.f;
}

// ---------------------------------------------------------------------------
// Epilogues.  Accumulator register r of lane l holds block row
// 8*(r/4) + 4*(l/32) + r%4, block column l%32.  `wr` (and `br`) address W
// (buf) from the tile's first element; the byte offsets of a tile fit in 31
// bits (the host checks).
// ---------------------------------------------------------------------------

// Row offset (bytes / n4) of accumulator register r in block row i.
__device__ __forceinline__ constexpr int acc_row(int i, int r) { return 32 * i + 8 * (r >> 2) + (r & 3); }

// Values of W's first MFMA block that an interior tile loads ahead of the last
// K step (as many as the register budget holds without spilling).  Launches
// that leave room for PS waves beside the rebuild load none ahead: 118
// instead of 127 VGPRs, so that a SIMD's four SF waves leave it 32.
constexpr int W_PRE = 10;

// Cache policy of the epilogue's W and buf accesses: non-temporal (the
// buffer instructions' nt bit).  Each value is read and written once, and
// without the hint the 128 KB of W a tile moves through the XCD's L2 evicts
// the U and V panel slices the tiles running beside it still read: the
// VGG19-22K grouped launch fetched 1975 MB from memory with it off and
// 1453 MB with it on (algorithmic 966 MB), and the iteration ran 1.2% faster.
constexpr int W_AUX = 2;

__device__ __forceinline__ void load_w_block(float (&wv)[16], __amdgpu_buffer_rsrc_t wr, int voff, int n4, int r0,
                                             int r1)
{
#pragma unroll
    for (int r = r0; r < r1; ++r)
        wv[r] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(wr, voff, acc_row(0, r) * n4, W_AUX));
}

// Interior tile: one shared lane offset (voff) and uniform row offsets, one
// MFMA block at a time; the first W_PRE values of block 0 are already in wv.
template <int TM, int TN, int PRE>
__device__ __forceinline__ void epi_interior(const f16v (&acc)[TM][TN], float (&wv)[16], __amdgpu_buffer_rsrc_t wr,
                                             int voff, int n4, float lr)
{
#pragma unroll
    for (int c = 0; c < TM * TN; ++c) {
        const int i = c / TN, j = c % TN;
#pragma unroll
        for (int r = (c == 0 ? PRE : 0); r < 16; ++r)
            wv[r] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                wr, voff + 128 * j, acc_row(i, r) * n4, W_AUX));
#pragma unroll
        for (int r = 0; r < 16; ++r)
            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, fmaf(-lr, acc[i][j][r], wv[r])), wr,
                                                  voff + 128 * j, acc_row(i, r) * n4, W_AUX);
    }
}

// Ragged edge tile: every element gets its own lane offset; an element outside
// W loads the tile's first element instead (always inside W, value unused) and
// is not stored.
template <int TM, int TN>
__device__ __forceinline__ void epi_edge(const f16v (&acc)[TM][TN], __amdgpu_buffer_rsrc_t wr, int ni, int wm, int wn,
                                         int lrow, int lcol, int rows_left, int cols_left, float lr)
{
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int col = wn + 32 * j + lcol;
            float ev[16];
            int off[16];
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row = wm + 32 * i + 8 * (r >> 2) + 4 * lrow + (r & 3);
                off[r] = (row < rows_left && col < cols_left) ? (row * ni + col) * 4 : 0;
                ev[r] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(wr, off[r], 0, W_AUX));
            }
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row = wm + 32 * i + 8 * (r >> 2) + 4 * lrow + (r & 3);
                if (row < rows_left && col < cols_left)
                    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, fmaf(-lr, acc[i][j][r], ev[r])),
                                                          wr, off[r], 0, W_AUX);
            }
            // One MFMA block at a time: keeps the scheduler from hoisting
            // every block's loads and offsets together.
            __builtin_amdgcn_sched_barrier(0);
        }
    }
}

// Momentum on an edge tile: buf <- mu*buf + dW, W <- W - lr*buf, half an MFMA
// block (8 values per lane) at a time, W and buf loads in flight together,
// then both stores; elements outside W as in epi_edge.
template <int TM, int TN>
__device__ __forceinline__ void epi_momentum(const f16v (&acc)[TM][TN], __amdgpu_buffer_rsrc_t wr,
                                             __amdgpu_buffer_rsrc_t br, int ni, int wm, int wn, int lrow, int lcol,
                                             int rows_left, int cols_left, float lr, float mu)
{
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
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
                    wv[q] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(wr, off[q], 0, W_AUX));
                    bv[q] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(br, off[q], 0, W_AUX));
                }
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    const int r = h + q;
                    const int row = wm + 32 * i + 8 * (r >> 2) + 4 * lrow + (r & 3);
                    if (row < rows_left && col < cols_left) {
                        const float nb = fmaf(mu, bv[q], acc[i][j][r]);
                        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, nb), br, off[q], 0, W_AUX);
                        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, fmaf(-lr, nb, wv[q])), wr,
                                                              off[q], 0, W_AUX);
                    }
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    }
}

// Momentum on an interior tile: one shared lane offset and uniform row offsets
// for both W and buf, half an MFMA block at a time.
template <int TM, int TN>
__device__ __forceinline__ void epi_momentum_interior(const f16v (&acc)[TM][TN], __amdgpu_buffer_rsrc_t wr,
                                                      __amdgpu_buffer_rsrc_t br, int voff, int n4, float lr, float mu)
{
#pragma unroll
    for (int c = 0; c < TM * TN; ++c) {
        const int i = c / TN, j = c % TN;
#pragma unroll
        for (int h = 0; h < 16; h += 8) {
            float wv[8], bv[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                wv[q] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                    wr, voff + 128 * j, acc_row(i, h + q) * n4, W_AUX));
                bv[q] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                    br, voff + 128 * j, acc_row(i, h + q) * n4, W_AUX));
            }
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const float nb = fmaf(mu, bv[q], acc[i][j][h + q]);
                __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, nb), br, voff + 128 * j,
                                                      acc_row(i, h + q) * n4, W_AUX);
                __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, fmaf(-lr, nb, wv[q])), wr,
                                                      voff + 128 * j, acc_row(i, h + q) * n4, W_AUX);
            }
        }
    }
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(float* base, int64_t M, int64_t N, int64_t first)
{
    const int64_t avail = (M * N - first) * 4;
    return __builtin_amdgcn_make_buffer_rsrc(base + first, static_cast<short>(0),
                                             static_cast<int>(avail < 0x7fffffff ? avail : 0x7fffffff),
                                             BUF_RSRC_WORD3);
}

// The epilogue of one tile for offsets that fit 31 bits.  On an interior
// tile the caller has loaded the first PRE values of block 0 into wv.
template <int TM, int TN, bool MOM, int PRE = W_PRE>
__device__ __forceinline__ void epilogue(const f16v (&acc)[TM][TN], float (&wv)[16], __amdgpu_buffer_rsrc_t wr,
                                         float* __restrict__ buf, int64_t M, int64_t N, int64_t m0, int64_t n0,
                                         int BM, int BN, int wm, int wn, int lrow, int lcol, bool interior,
                                         float lr, float mu)
{
    const int ni = static_cast<int>(N);
    const int rows_left = static_cast<int>(M - m0 < BM ? M - m0 : BM);
    const int cols_left = static_cast<int>(N - n0 < BN ? N - n0 : BN);
    if constexpr (MOM) {
        const __amdgpu_buffer_rsrc_t br = tile_rsrc(buf, M, N, m0 * N + n0);
        if (interior)
            epi_momentum_interior<TM, TN>(acc, wr, br, ((wm + 4 * lrow) * ni + wn + lcol) * 4, ni * 4, lr, mu);
        else
            epi_momentum<TM, TN>(acc, wr, br, ni, wm, wn, lrow, lcol, rows_left, cols_left, lr, mu);
    } else if (interior) {
        epi_interior<TM, TN, PRE>(acc, wv, wr, ((wm + 4 * lrow) * ni + wn + lcol) * 4, ni * 4, lr);
    } else {
        epi_edge<TM, TN>(acc, wr, ni, wm, wn, lrow, lcol, rows_left, cols_left, lr);
    }
}

// ---------------------------------------------------------------------------
// LDS-direct tile (the main path).
// ---------------------------------------------------------------------------

// Each pipeline stage is an LDS object of its own: the compiler can then tell
// that the in-flight LDS-direct loads into one stage do not alias the LDS
// reads of the other, and does not wait for them before reading.
template <int SIZE, int S, int WHICH>
struct LdsStage {
    static __device__ __forceinline__ float* ptr()
    {
        __shared__ float a[SIZE];
        return a;
    }
};

// ---------------------------------------------------------------------------
// Split-bf16 products (the default arithmetic).  An fp32 value x is the exact
// sum of three bf16 values: h = bf16(x) and m = bf16(x - h), each rounded to
// nearest, and l = x - h - m, which has at most 8 significant bits (bf16
// keeps 8 of fp32's 24 and the same exponent range).  A product x*y is the
// sum of the nine products of the parts; the six kept here (h*h, h*m, m*h,
// h*l, l*h, m*m) are each exact in fp32 and formed on the bf16 matrix cores
// with fp32 accumulation.  The three dropped (m*l, l*m, l*l) are below 2^-23
// of |x*y| together and of either sign.  This is the six-product split of
// Henry, Tang and Heinecke, "Leveraging the bfloat16 Artificial Intelligence
// Datatype For Higher-Precision Computations" (ARITH 2019).
// ---------------------------------------------------------------------------
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf2 __attribute__((ext_vector_type(2)));
typedef float fl2 __attribute__((ext_vector_type(2)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

struct Split3 {
    bf8 h, m, l;
};

// Two values rounded to bf16 and packed (the first in the low half).
__device__ __forceinline__ unsigned pack_bf16(float a, float b)
{
    return __builtin_bit_cast(unsigned, __builtin_convertvector((fl2){a, b}, bf2));
}

// The top halves of two fp32 values packed (a's in the low half): exact for
// values of at most 8 significant bits.
__device__ __forceinline__ unsigned pack_top(float a, float b)
{
    return __builtin_amdgcn_perm(__builtin_bit_cast(unsigned, b), __builtin_bit_cast(unsigned, a), 0x07060302u);
}

// x minus half HI of the packed pair p (a bf16's fp32 value is its bits in
// the top half of the word).
template <int HI>
__device__ __forceinline__ float minus_half(float x, unsigned p)
{
    return x - __builtin_bit_cast(float, HI ? (p & 0xffff0000u) : (p << 16));
}

// The parts of x[0..7], two values per conversion.
__device__ __forceinline__ Split3 split3(const float (&x)[8])
{
    u32x4 h, m, l;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const unsigned hp = pack_bf16(x[2 * q], x[2 * q + 1]);
        const float r0 = minus_half<0>(x[2 * q], hp);
        const float r1 = minus_half<1>(x[2 * q + 1], hp);
        const unsigned mp = pack_bf16(r0, r1);
        h[q] = hp;
        m[q] = mp;
        l[q] = pack_top(minus_half<0>(r0, mp), minus_half<1>(r1, mp));
    }
    return {__builtin_bit_cast(bf8, h), __builtin_bit_cast(bf8, m), __builtin_bit_cast(bf8, l)};
}

// acc[j] += A * B_j over 16 values of K: the six products, the small ones
// first, each over every block of the row before the next.
template <int TN>
__device__ __forceinline__ void split_products(f16v (&acc)[TN], const Split3& a, const Split3 (&b)[TN])
{
    auto each = [&](auto pick_a, auto pick_b) {
#pragma unroll
        for (int j = 0; j < TN; ++j)
            acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pick_a(a), pick_b(b[j]), acc[j], 0, 0, 0);
    };
    auto H = [](const Split3& x) { return x.h; };
    auto Mi = [](const Split3& x) { return x.m; };
    auto L = [](const Split3& x) { return x.l; };
    each(Mi, Mi);
    each(H, L);
    each(L, H);
    each(H, Mi);
    each(Mi, H);
    each(H, H);
}

// Chunk (16 bytes) c of slice row k is stored at chunk position c ^ swz(k).
__device__ __forceinline__ constexpr int swz(int k) { return (k & 1) << 3; }

// Wait for every outstanding vector-memory load of this wave (the LDS-direct
// loads included); the workgroup barrier that follows makes every wave's
// loads of the slice visible.
__device__ __forceinline__ void wait_loads() { __builtin_amdgcn_s_waitcnt(0x0F70); }   // vmcnt(0)

template <int BM, int BN, int BK, int WM, int WN, bool SPLIT>
struct Direct {
    using T = SfTile<BM, BN, BK, WM, WN>;
    static constexpr int NT = T::THREADS;
    template <int S> static __device__ __forceinline__ float* A() { return LdsStage<BK * BM, S, 0>::ptr(); }
    template <int S> static __device__ __forceinline__ float* B() { return LdsStage<BK * BN, S, 1>::ptr(); }

    // One BK x BX slice of a K-major operand into an LDS stage.  Wave
    // instruction q fills LDS chunks 64q .. 64q+63 (row-major, BX/4 chunks a
    // row); its lane l loads global chunk (row g / (BX/4), column chunk
    // (g % (BX/4)) ^ swz(row)) with g = 64q + l.  `rs` addresses the operand
    // from the tile's first column; voffsets are bytes from there, and the
    // resource's size makes every read at or past row K return 0.
    template <int BX>
    static __device__ __forceinline__ void issue_panel(__amdgpu_buffer_rsrc_t rs, float* stage, int ld_bytes, int k0,
                                                       int tid)
    {
        constexpr int CPR = BX / 4;
        constexpr int PER = BK * CPR / NT;
        static_assert(PER * NT == BK * CPR, "slice");
        const int wave = tid >> 6, lane = tid & 63;
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            const int g0 = (wave + j * (NT / 64)) * 64;
            const int g = g0 + lane;
            const int k = g / CPR;
            const int c = (g % CPR) ^ swz(k);
            const int voff = (k0 + k) * ld_bytes + c * 16;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void*)(stage + g0 * 4), 16, voff, 0, 0, 0);
        }
    }

    template <int S>
    static __device__ __forceinline__ void issue(__amdgpu_buffer_rsrc_t ur, __amdgpu_buffer_rsrc_t vr, int ldu,
                                                 int ldv, int kt, int tid)
    {
        issue_panel<BM>(ur, A<S>(), ldu, kt * BK, tid);
        issue_panel<BN>(vr, B<S>(), ldv, kt * BK, tid);
    }

    // One BK-deep step of the contraction out of LDS stage S.
    template <int S>
    static __device__ __forceinline__ void mma(f16v (&acc)[T::TM][T::TN], int wm, int wn, int lane)
    {
        if constexpr (SPLIT)
            mma_split<S>(acc, wm, wn, lane);
        else
            mma_f32<S>(acc, wm, wn, lane);
    }

    // Split-bf16 step: 16 values of K per MFMA.  Lane l of an operand holds
    // slot q = 0..7 of its row (column) as K index 2q + l/32, the LDS reads
    // of the fp32 step below, eight at a time; A and B use the same slots.
    template <int S>
    static __device__ __forceinline__ void mma_split(f16v (&acc)[T::TM][T::TN], int wm, int wn, int lane)
    {
        static_assert(BK % 16 == 0, "bf16 MFMA depth is 16");
        const float* a_s = A<S>();
        const float* b_s = B<S>();
        const int lrow = lane >> 5, lcol = lane & 31;
        auto at = [&](const float* s, int ld, int kk, int x) {
            const int k = kk + lrow;
            return s[k * ld + ((((x >> 2) ^ swz(k)) << 2) | (x & 3))];
        };
#pragma unroll
        for (int kk = 0; kk < BK; kk += 16) {
            Split3 b[T::TN];
#pragma unroll
            for (int j = 0; j < T::TN; ++j) {
                float x[8];
#pragma unroll
                for (int q = 0; q < 8; ++q)
                    x[q] = at(b_s, BN, kk + 2 * q, wn + 32 * j + lcol);
                b[j] = split3(x);
            }
            // One A block row at a time (its parts and B's stay in registers).
#pragma unroll
            for (int i = 0; i < T::TM; ++i) {
                float x[8];
#pragma unroll
                for (int q = 0; q < 8; ++q)
                    x[q] = at(a_s, BM, kk + 2 * q, wm + 32 * i + lcol);
                split_products<T::TN>(acc[i], split3(x), b);
            }
        }
    }

    // fp32 step: the MFMA operands of step kk+2 are read while the matrix
    // cores work on step kk.
    template <int S>
    static __device__ __forceinline__ void mma_f32(f16v (&acc)[T::TM][T::TN], int wm, int wn, int lane)
    {
        const float* a_s = A<S>();
        const float* b_s = B<S>();
        const int lrow = lane >> 5, lcol = lane & 31;
        auto at = [&](const float* s, int ld, int kk, int x) {
            const int k = kk + lrow;
            return s[k * ld + ((((x >> 2) ^ swz(k)) << 2) | (x & 3))];
        };
        float a[2][T::TM], b[2][T::TN];
#pragma unroll
        for (int i = 0; i < T::TM; ++i)
            a[0][i] = at(a_s, BM, 0, wm + 32 * i + lcol);
#pragma unroll
        for (int j = 0; j < T::TN; ++j)
            b[0][j] = at(b_s, BN, 0, wn + 32 * j + lcol);
#pragma unroll
        for (int kk = 0; kk < BK; kk += 2) {
            const int c = (kk >> 1) & 1;
            if (kk + 2 < BK) {
#pragma unroll
                for (int i = 0; i < T::TM; ++i)
                    a[c ^ 1][i] = at(a_s, BM, kk + 2, wm + 32 * i + lcol);
#pragma unroll
                for (int j = 0; j < T::TN; ++j)
                    b[c ^ 1][j] = at(b_s, BN, kk + 2, wn + 32 * j + lcol);
            }
#pragma unroll
            for (int i = 0; i < T::TM; ++i)
#pragma unroll
                for (int j = 0; j < T::TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[c][i], b[c][j], acc[i][j], 0, 0, 0);
        }
    }

    // Slice kt (not the last) in stage S: wait until it has landed, then
    // start slice kt+1 into the other stage (free: every wave has passed the
    // barrier after reading it) and multiply.
    template <int S>
    static __device__ __forceinline__ void step(f16v (&acc)[T::TM][T::TN], __amdgpu_buffer_rsrc_t ur,
                                                __amdgpu_buffer_rsrc_t vr, int ldu, int ldv, int kt, int wm, int wn,
                                                int lane, int tid)
    {
        wait_loads();
        __syncthreads();
        issue<S ^ 1>(ur, vr, ldu, ldv, kt + 1, tid);
        // Keep the loads ahead of the multiply: left to itself the scheduler
        // sinks them (they have no register results) to the end of the slice,
        // just before the next step waits for them, and their latency is then
        // hidden only by the other workgroups on the CU.
        __builtin_amdgcn_sched_barrier(0);
        mma<S>(acc, wm, wn, lane);
    }
};

// One BM x BN tile of W: the whole K loop and the fused update.  Slice kt
// lives in stage (nkt-1-kt) & 1, so the last slice is always in stage 0 and
// the loop body and the final step are each emitted once.  An interior tile
// loads PRE values of W ahead of the last K step.
template <int BM, int BN, int BK, int WM, int WN, bool SPLIT, bool MOM, int PRE = W_PRE>
__device__ __forceinline__ void sf_tile_direct(float* __restrict__ W, const float* __restrict__ U,
                                               const float* __restrict__ V, int64_t M, int64_t N, int64_t K,
                                               float lr, int tm, int tn, float* __restrict__ buf, float mu)
{
    using D = Direct<BM, BN, BK, WM, WN, SPLIT>;
    using T = SfTile<BM, BN, BK, WM, WN>;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int64_t m0 = static_cast<int64_t>(tm) * BM;
    const int64_t n0 = static_cast<int64_t>(tn) * BN;
    const int wm = (wave / T::NWN) * WM;
    const int wn = (wave % T::NWN) * WN;
    const int lrow = lane >> 5, lcol = lane & 31;
    const bool interior = (m0 + BM <= M) && (n0 + BN <= N);

    f16v acc[T::TM][T::TN];
    zero_acc(acc);
    const int64_t first = m0 * N + n0;
    const __amdgpu_buffer_rsrc_t wr = tile_rsrc(W, M, N, first);
    const int ni = static_cast<int>(N);
    const int voff = ((wm + 4 * lrow) * ni + wn + lcol) * 4;
    float wv[16];

    const int nkt = static_cast<int>((K + BK - 1) / BK);
    if (nkt > 0) {
        const __amdgpu_buffer_rsrc_t ur = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<float*>(U) + m0, static_cast<short>(0), static_cast<int>((K * M - m0) * 4), BUF_RSRC_WORD3);
        const __amdgpu_buffer_rsrc_t vr = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<float*>(V) + n0, static_cast<short>(0), static_cast<int>((K * N - n0) * 4), BUF_RSRC_WORD3);
        const int ldu = static_cast<int>(M) * 4, ldv = static_cast<int>(N) * 4;
        int kt = 0;
        if ((nkt & 1) == 0) {
            D::template issue<1>(ur, vr, ldu, ldv, 0, tid);
            D::template step<1>(acc, ur, vr, ldu, ldv, 0, wm, wn, lane, tid);
            kt = 1;
        } else {
            D::template issue<0>(ur, vr, ldu, ldv, 0, tid);
        }
        for (; kt < nkt - 1; kt += 2) {
            D::template step<0>(acc, ur, vr, ldu, ldv, kt, wm, wn, lane, tid);
            D::template step<1>(acc, ur, vr, ldu, ldv, kt + 1, wm, wn, lane, tid);
        }
        wait_loads();
        __syncthreads();
        if (!MOM && interior)
            load_w_block(wv, wr, voff, ni * 4, 0, PRE);
        D::template mma<0>(acc, wm, wn, lane);
    }
    epilogue<T::TM, T::TN, MOM, PRE>(acc, wv, wr, buf, M, N, m0, n0, BM, BN, wm, wn, lrow, lcol, interior, lr, mu);
}

// ---------------------------------------------------------------------------
// Register-staged tile for operands beyond 32-bit offsets: K-slices go global
// -> registers -> LDS (row-padded by 4 floats), double-buffered; 64-bit
// addressing throughout, and W rows too long for 32-bit tile offsets
// (WIDE) take guarded 64-bit accesses in the epilogue.
// ---------------------------------------------------------------------------
constexpr int LDS_PAD = 4;

// Load one BK x (4*COLS4) slice of a K-major operand X (row length ld) into
// registers: group j of this thread covers row g / COLS4 and columns
// 4*(g % COLS4) .. +3 with g = tid + j*THREADS.  Out-of-range rows/columns
// read as 0.  Global loads of several dwords need only 4-byte alignment;
// only a group that runs past the end of its row is read element by element.
template <int NV4, int COLS4, int THREADS>
__device__ inline void load_panel(f4 (&r)[NV4], const float* __restrict__ X, int64_t ld, int64_t rows, int64_t k0,
                                  int64_t c0, int tid)
{
#pragma unroll
    for (int j = 0; j < NV4; ++j) {
        const int g = tid + j * THREADS;
        const int64_t k = k0 + g / COLS4;
        const int64_t c = c0 + 4 * (g % COLS4);
        const float* src = X + k * ld + c;
        const bool kin = k < rows;
        if (kin && c + 3 < ld) {
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

template <int BK, int LDA, int LDB, int TM, int TN>
__device__ inline void mma_staged(f16v (&acc)[TM][TN], const float* a_s, const float* b_s)
{
#pragma unroll
    for (int kk = 0; kk < BK; kk += 2) {
        float a[TM], b[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i)
            a[i] = a_s[kk * LDA + 32 * i];
#pragma unroll
        for (int j = 0; j < TN; ++j)
            b[j] = b_s[kk * LDB + 32 * j];
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i], b[j], acc[i][j], 0, 0, 0);
    }
}

template <int BM, int BN, int BK, int WM, int WN, bool WIDE, bool MOM>
__device__ __forceinline__ void sf_tile_staged(float* As, float* Bs, float* __restrict__ W,
                                               const float* __restrict__ U, const float* __restrict__ V, int64_t M,
                                               int64_t N, int64_t K, float lr, int tm, int tn,
                                               float* __restrict__ buf, float mu)
{
    using T = SfTile<BM, BN, BK, WM, WN>;
    constexpr int LDA = BM + LDS_PAD, LDB = BN + LDS_PAD;
    constexpr int SA = BK * LDA, SB = BK * LDB;
    constexpr int A_V4 = BK * BM / 4 / T::THREADS, B_V4 = BK * BN / 4 / T::THREADS;
    static_assert(A_V4 * T::THREADS * 4 == BK * BM && B_V4 * T::THREADS * 4 == BK * BN, "staging");

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int64_t m0 = static_cast<int64_t>(tm) * BM;
    const int64_t n0 = static_cast<int64_t>(tn) * BN;
    const int wm = (wave / T::NWN) * WM;
    const int wn = (wave % T::NWN) * WN;
    const int lrow = lane >> 5, lcol = lane & 31;

    f16v acc[T::TM][T::TN];
    zero_acc(acc);
    f4 ra[A_V4], rb[B_V4];
    const int64_t nkt = (K + BK - 1) / BK;
    if (nkt > 0) {
        load_panel<A_V4, BM / 4, T::THREADS>(ra, U, M, K, 0, m0, tid);
        load_panel<B_V4, BN / 4, T::THREADS>(rb, V, N, K, 0, n0, tid);
        store_panel<A_V4, BM / 4, T::THREADS, LDA>(As, ra, tid);
        store_panel<B_V4, BN / 4, T::THREADS, LDB>(Bs, rb, tid);
        __syncthreads();
        const int a_off = lrow * LDA + wm + lcol;
        const int b_off = lrow * LDB + wn + lcol;
        for (int64_t kt = 0; kt < nkt; ++kt) {
            const int cur = static_cast<int>(kt & 1);
            if (kt + 1 < nkt) {
                load_panel<A_V4, BM / 4, T::THREADS>(ra, U, M, K, (kt + 1) * BK, m0, tid);
                load_panel<B_V4, BN / 4, T::THREADS>(rb, V, N, K, (kt + 1) * BK, n0, tid);
            }
            mma_staged<BK, LDA, LDB, T::TM, T::TN>(acc, As + cur * SA + a_off, Bs + cur * SB + b_off);
            if (kt + 1 < nkt) {
                store_panel<A_V4, BM / 4, T::THREADS, LDA>(As + (cur ^ 1) * SA, ra, tid);
                store_panel<B_V4, BN / 4, T::THREADS, LDB>(Bs + (cur ^ 1) * SB, rb, tid);
            }
            __syncthreads();
        }
    }
    if constexpr (!WIDE) {
        const bool interior = (m0 + BM <= M) && (n0 + BN <= N);
        const __amdgpu_buffer_rsrc_t wr = tile_rsrc(W, M, N, m0 * N + n0);
        float wv[16];
        if (!MOM && interior)
            load_w_block(wv, wr, ((wm + 4 * lrow) * static_cast<int>(N) + wn + lcol) * 4, static_cast<int>(N) * 4, 0,
                         W_PRE);
        epilogue<T::TM, T::TN, MOM>(acc, wv, wr, buf, M, N, m0, n0, BM, BN, wm, wn, lrow, lcol, interior, lr, mu);
    } else {
#pragma unroll
        for (int i = 0; i < T::TM; ++i) {
#pragma unroll
            for (int j = 0; j < T::TN; ++j) {
                const int64_t col = n0 + wn + 32 * j + lcol;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int64_t row = m0 + wm + 32 * i + 8 * (r >> 2) + 4 * lrow + (r & 3);
                    if (row < M && col < N) {
                        const int64_t e = row * N + col;
                        if constexpr (MOM) {
                            const float nb = fmaf(mu, buf[e], acc[i][j][r]);
                            buf[e] = nb;
                            W[e] = fmaf(-lr, nb, W[e]);
                        } else {
                            W[e] = fmaf(-lr, acc[i][j][r], W[e]);
                        }
                    }
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Kernels, compiled for the waves per SIMD of their tile shape (SfOcc: 4, at
// most 128 VGPRs a wave, or 2 for the 128 x 64 sub-blocks).
// ---------------------------------------------------------------------------
template <int BM, int BN, int BK, int WM, int WN, bool SPLIT, bool MOM, int PRE = W_PRE>
__global__ __launch_bounds__((BM / WM) * (BN / WN) * 64)
__attribute__((amdgpu_waves_per_eu(SfOcc<WM, WN>::W, SfOcc<WM, WN>::W))) void sf_apply_kernel(
    float* __restrict__ W, const float* __restrict__ U, const float* __restrict__ V, int64_t M, int64_t N, int64_t K,
    float lr, int tiles_m, int tiles_n, float* __restrict__ buf, float mu)
{
    int tm, tn;
    tile_coords<TileRows<BM>::G>(blockIdx.x, tiles_m * tiles_n, tiles_m, tiles_n, tm, tn);
    sf_tile_direct<BM, BN, BK, WM, WN, SPLIT, MOM, PRE>(W, U, V, M, N, K, lr, tm, tn, buf, mu);
}

// The spread launch: fewer workgroups than tiles (a multiple of 8, so that
// tile t stays on the XCD of workgroup t % 8), each walking the tiles
// grid-stride.  A kernel of its own: the loop makes the compiler keep more
// values live (the 128 x 128 tile spilled 61 VGPRs at the one-tile kernel's
// 128), and a spread launch has few workgroups resident, so it is compiled
// for 2 waves per SIMD (two workgroups per CU).  The barrier keeps a wave's first loads of the next
// tile out of the LDS stage the others may still read.
template <int BM, int BN, int BK, int WM, int WN, bool SPLIT, bool MOM>
__global__ __launch_bounds__((BM / WM) * (BN / WN) * 64)
__attribute__((amdgpu_waves_per_eu(2, 2))) void sf_apply_walk_kernel(
    float* __restrict__ W, const float* __restrict__ U, const float* __restrict__ V, int64_t M, int64_t N, int64_t K,
    float lr, int tiles_m, int tiles_n, float* __restrict__ buf, float mu)
{
    const int tiles = tiles_m * tiles_n;
    for (int t = blockIdx.x; t < tiles; t += gridDim.x) {
        if (t != static_cast<int>(blockIdx.x))
            __syncthreads();
        int tm, tn;
        tile_coords<8>(t, tiles, tiles_m, tiles_n, tm, tn);
        sf_tile_direct<BM, BN, BK, WM, WN, SPLIT, MOM>(W, U, V, M, N, K, lr, tm, tn, buf, mu);
    }
}

template <int BM, int BN, int BK, int WM, int WN, bool WIDE, bool MOM>
__global__ __launch_bounds__((BM / WM) * (BN / WN) * 64)
__attribute__((amdgpu_waves_per_eu(SfOcc<WM, WN>::W, SfOcc<WM, WN>::W))) void sf_apply_staged_kernel(
    float* __restrict__ W, const float* __restrict__ U, const float* __restrict__ V, int64_t M, int64_t N, int64_t K,
    float lr, int tiles_m, int tiles_n, float* __restrict__ buf, float mu)
{
    __shared__ float As[2 * BK * (BM + LDS_PAD)];
    __shared__ float Bs[2 * BK * (BN + LDS_PAD)];
    int tm, tn;
    tile_coords<8>(blockIdx.x, tiles_m * tiles_n, tiles_m, tiles_n, tm, tn);
    sf_tile_staged<BM, BN, BK, WM, WN, WIDE, MOM>(As, Bs, W, U, V, M, N, K, lr, tm, tn, buf, mu);
}

// ---------------------------------------------------------------------------
// Several layers in one launch (same K): one tile list, so the chip is filled
// by the tiles of the next layer while the last ones of a layer finish,
// instead of every layer ending in a partly idle round.  Layer descriptors
// travel by value in the kernel arguments; the XCD-aware order runs over the
// combined list (layer by layer, in the order given), and inside a layer tile
// rows are walked a group (TileRows) at a time.
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
    int32_t pad;
};

struct SfBatchArgs {
    SfBatchItem item[SF_BATCH_MAX];
    int32_t count;
    int32_t total_tiles;
};

// Tile t of the combined list (layer by layer; inside a layer tile rows
// walked a group (TileRows) at a time).
template <int BM, int BN, int BK, int WM, int WN, bool SPLIT, int PRE = W_PRE>
__device__ __forceinline__ void batch_tile(const SfBatchArgs& args, int t, int64_t K, float lr)
{
    int l = 0;
    while (l + 1 < args.count && t >= args.item[l + 1].first_tile)
        ++l;
    const int local = t - args.item[l].first_tile;
    const int tiles_m = args.item[l].tiles_m, tiles_n = args.item[l].tiles_n;
    constexpr int G = TileRows<BM>::G;
    const int per_group = G * tiles_n;
    const int g = local / per_group;
    const int first_m = g * G;
    const int rows = (tiles_m - first_m) < G ? (tiles_m - first_m) : G;
    const int in = local - g * per_group;
    const SfBatchItem& it = args.item[l];
    sf_tile_direct<BM, BN, BK, WM, WN, SPLIT, false, PRE>(it.W, it.U, it.V, it.M, it.N, K, lr, first_m + in % rows,
                                                   in / rows, nullptr, 0.f);
}

template <int BM, int BN, int BK, int WM, int WN, bool SPLIT, int PRE = W_PRE>
__global__ __launch_bounds__((BM / WM) * (BN / WN) * 64)
__attribute__((amdgpu_waves_per_eu(SfOcc<WM, WN>::W, SfOcc<WM, WN>::W))) void sf_apply_batch_kernel(const SfBatchArgs args, int64_t K, float lr)
{
    const int tiles = args.total_tiles;
    const int q = tiles / NUM_XCD, r = tiles % NUM_XCD;
    const int x = blockIdx.x % NUM_XCD, j = blockIdx.x / NUM_XCD;
    batch_tile<BM, BN, BK, WM, WN, SPLIT, PRE>(args, x * q + (x < r ? x : r) + j, K, lr);
}

// True when the LDS-direct tile's 32-bit buffer offsets cover the layer: the
// operand reads (K + BK rows, so the last slice's rows past K still have
// representable offsets) and the W offsets inside one BM-row tile.
bool direct_fits(int64_t M, int64_t N, int64_t K, int BM, int BN, int BK)
{
    constexpr int64_t LIM = 0x7fffffffLL;
    return (K + BK) * M * 4 < LIM && (K + BK) * N * 4 < LIM && (static_cast<int64_t>(BM) * N + BN) * 4 < LIM;
}

// Workgroups of the spread kernel that one CU holds at once (its register
// and LDS needs; cached per instantiation).
template <int BM, int BN, int BK, int WM, int WN, bool SPLIT, bool MOM>
int64_t walk_groups_per_cu()
{
    static std::atomic<int> cached{0};
    int n = cached.load(std::memory_order_relaxed);
    if (n > 0)
        return n;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, sf_apply_walk_kernel<BM, BN, BK, WM, WN, SPLIT, MOM>,
                                                     SfTile<BM, BN, BK, WM, WN>::THREADS, 0) != hipSuccess ||
        n < 1)
        n = 1;
    cached.store(n, std::memory_order_relaxed);
    return n;
}

// A workgroup's rate when few of them walk a layer's tiles beside the PS
// applies (the 1000 x 2048 classifier at K = 1024: 8 tiles of 64 x 64 each
// on 64 workgroups in 0.52 ms, 1.29e11 flop/s), a little under.
constexpr double SPREAD_WG_FLOPS_PER_S = 1.2e11;

template <class TL, bool SPLIT, bool MOM>
hipError_t launch_tiles(float* W, float* buf, const float* U, const float* V, int64_t M, int64_t N, int64_t K,
                        float lr, float mu, double spread_s, bool room, hipStream_t stream)
{
    constexpr int BM = TL::BM, BN = TL::BN, BK = TL::BK, WM = TL::WM, WN = TL::WN;
    constexpr int NT = SfTile<BM, BN, BK, WM, WN>::THREADS;
    const int64_t tiles_m = (M + BM - 1) / BM;
    const int64_t tiles_n = (N + BN - 1) / BN;
    if (tiles_m * tiles_n > INT32_MAX)
        return hipErrorInvalidValue;
    const int t = static_cast<int>(tiles_m * tiles_n), tmi = static_cast<int>(tiles_m),
              tni = static_cast<int>(tiles_n);
    // The large tile is only chosen where it fits the LDS-direct path, and
    // never spread: the staged and spread kernels come in the other shapes.
    constexpr bool LARGE = WM * WN > 64 * 64;
    if (LARGE || direct_fits(M, N, K, BM, BN, BK)) {
        // Spread: as few workgroups (a multiple of 8) as walk the tiles
        // within spread_s at SPREAD_WG_FLOPS_PER_S each -- provided the chip
        // holds them all at once (otherwise the later ones would wait for
        // the first to finish all their tiles).
        int grid = t;
        if constexpr (!LARGE) {
            if (spread_s > 0.0) {
                const double per = spread_s * SPREAD_WG_FLOPS_PER_S / (2.0 * BM * BN * static_cast<double>(K));
                if (per >= 2.0) {
                    const int64_t p = per < t ? static_cast<int64_t>(per) : t;
                    const int64_t g = ((t + p - 1) / p + NUM_XCD - 1) / NUM_XCD * NUM_XCD;
                    const int64_t resident =
                        walk_groups_per_cu<BM, BN, BK, WM, WN, SPLIT, MOM>() * device_cu_count();
                    if (g < t && g <= resident)
                        grid = static_cast<int>(g);
                }
            }
        }
        // (The momentum epilogue loads no W ahead anyway.)
        constexpr bool can_drop_pre = !MOM;
        if constexpr (!LARGE) {
            if (grid < t) {
                sf_apply_walk_kernel<BM, BN, BK, WM, WN, SPLIT, MOM><<<grid, NT, 0, stream>>>(W, U, V, M, N, K, lr,
                                                                                             tmi, tni, buf, mu);
                return hipGetLastError();
            }
        }
        if (room && can_drop_pre)
            sf_apply_kernel<BM, BN, BK, WM, WN, SPLIT, MOM, can_drop_pre ? 0 : W_PRE><<<t, NT, 0, stream>>>(
                W, U, V, M, N, K, lr, tmi, tni, buf, mu);
        else
            sf_apply_kernel<BM, BN, BK, WM, WN, SPLIT, MOM><<<t, NT, 0, stream>>>(W, U, V, M, N, K, lr, tmi, tni,
                                                                                 buf, mu);
    }
    else if constexpr (!LARGE) {
        if ((static_cast<int64_t>(BM) * N + BN) * 4 < 0x7fffffffLL)
            sf_apply_staged_kernel<BM, BN, BK, WM, WN, false, MOM><<<t, NT, 0, stream>>>(W, U, V, M, N, K, lr, tmi,
                                                                                         tni, buf, mu);
        else
            sf_apply_staged_kernel<BM, BN, BK, WM, WN, true, MOM><<<t, NT, 0, stream>>>(W, U, V, M, N, K, lr, tmi,
                                                                                        tni, buf, mu);
    }
    return hipGetLastError();
}

template <class TL>
int64_t tiles_of(int64_t M, int64_t N)
{
    return ((M + TL::BM - 1) / TL::BM) * ((N + TL::BN - 1) / TL::BN);
}

// Tile choice (see Big, Mid, Small).  A spread launch takes the 128 x 128 or
// 64 x 64 tile: its few workgroups walk the tiles at two per CU.
template <bool SPLIT, bool MOM>
hipError_t launch_sf(float* W, float* buf, const float* U, const float* V, int64_t M, int64_t N, int64_t K, float lr,
                     float mu, double spread_s, bool room, hipStream_t stream)
{
    const int64_t cus = device_cu_count();
    if constexpr (SPLIT) {
        if (spread_s <= 0.0 && tiles_of<Big>(M, N) >= BIG_TILES_PER_CU * cus &&
            direct_fits(M, N, K, Big::BM, Big::BN, Big::BK))
            return launch_tiles<Big, SPLIT, MOM>(W, buf, U, V, M, N, K, lr, mu, 0.0, room, stream);
    }
    if (tiles_of<Mid>(M, N) >= MID_TILES_PER_CU * cus)
        return launch_tiles<Mid, SPLIT, MOM>(W, buf, U, V, M, N, K, lr, mu, spread_s, room, stream);
    return launch_tiles<Small, SPLIT, MOM>(W, buf, U, V, M, N, K, lr, mu, spread_s, room, stream);
}

template <bool MOM>
hipError_t launch_sf_arith(float* W, float* buf, const float* U, const float* V, int64_t M, int64_t N, int64_t K,
                           float lr, float mu, double spread_s, bool room, hipStream_t stream)
{
    if (sf_arithmetic() == POSEIDON_SF_FP32)
        return launch_sf<false, MOM>(W, buf, U, V, M, N, K, lr, mu, spread_s, room, stream);
    return launch_sf<true, MOM>(W, buf, U, V, M, N, K, lr, mu, spread_s, room, stream);
}

// One grouped launch per SF_BATCH_MAX layers of `grouped` (every one covered
// by the LDS-direct tile TL).
template <class TL, bool SPLIT>
hipError_t launch_grouped(const SfTensor* t, const std::vector<int32_t>& grouped, int64_t K, float lr, bool room,
                          hipStream_t stream)
{
    constexpr int BM = TL::BM, BN = TL::BN, BK = TL::BK;
    constexpr int NT = SfTile<BM, BN, BK, TL::WM, TL::WN>::THREADS;
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
            first += it.tiles_m * it.tiles_n;
        }
        a.total_tiles = first;
        if (room)
            sf_apply_batch_kernel<BM, BN, BK, TL::WM, TL::WN, SPLIT, 0><<<first, NT, 0, stream>>>(a, K, lr);
        else
            sf_apply_batch_kernel<BM, BN, BK, TL::WM, TL::WN, SPLIT><<<first, NT, 0, stream>>>(a, K, lr);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess)
            return e;
    }
    return hipSuccess;
}

// Grouped launch: every layer the LDS-direct tile covers joins one tile list
// -- of 256 x 128 tiles (split-bf16) when the group has at least four per CU,
// else of 128 x 128 tiles when it has at least two per CU; the others, and
// groups too small to fill the chip, take per-layer launches.
template <bool SPLIT>
hipError_t launch_batch(const SfTensor* t, int32_t count, int64_t K, float lr, hipStream_t stream, bool room)
{
    std::vector<int32_t> grouped;
    int64_t big = 0, mid = 0;
    for (int32_t i = 0; i < count; ++i) {
        if (t[i].M == 0 || t[i].N == 0 || K == 0)
            continue;
        // A layer joins the list when the 32-bit offsets of the 256-row
        // tile cover it (then those of the 128-row tile do too), so that
        // either shape can run the list; the 128 x 128 tiles are the more
        // numerous, so their count bounds both.
        const int64_t tm = tiles_of<Mid>(t[i].M, t[i].N);
        if (direct_fits(t[i].M, t[i].N, K, Big::BM, Mid::BN, Mid::BK) && mid + tm <= INT32_MAX) {
            grouped.push_back(i);
            mid += tm;
            big += tiles_of<Big>(t[i].M, t[i].N);
        } else {
            const hipError_t e =
                launch_sf<SPLIT, false>(t[i].W, nullptr, t[i].U, t[i].V, t[i].M, t[i].N, K, lr, 0.f, 0.0, room,
                                        stream);
            if (e != hipSuccess)
                return e;
        }
    }
    const int64_t cus = device_cu_count();
    if constexpr (SPLIT) {
        if (big >= BIG_TILES_PER_CU * cus)
            return launch_grouped<Big, SPLIT>(t, grouped, K, lr, room, stream);
    }
    if (mid >= MID_TILES_PER_CU * cus)
        return launch_grouped<Mid, SPLIT>(t, grouped, K, lr, room, stream);
    for (int32_t i : grouped) {
        const hipError_t e =
            launch_sf<SPLIT, false>(t[i].W, nullptr, t[i].U, t[i].V, t[i].M, t[i].N, K, lr, 0.f, 0.0, room, stream);
        if (e != hipSuccess)
            return e;
    }
    return hipSuccess;
}

std::atomic<int32_t> g_arithmetic{POSEIDON_SF_BF16X6};

}  // namespace

int32_t sf_arithmetic() { return g_arithmetic.load(std::memory_order_relaxed); }

void set_sf_arithmetic(int32_t a) { g_arithmetic.store(a, std::memory_order_relaxed); }

double sf_seconds(int64_t M, int64_t N, int64_t K)
{
    const double flops = 2.0 * static_cast<double>(M) * static_cast<double>(N) * static_cast<double>(K);
    if (sf_arithmetic() == POSEIDON_SF_FP32)
        return flops / SF_FP32_FLOPS_PER_S;
    const bool big = tiles_of<Big>(M, N) >= BIG_TILES_PER_CU * device_cu_count() &&
                     direct_fits(M, N, K, Big::BM, Big::BN, Big::BK);
    return flops / (big ? SF_SPLIT_BIG_FLOPS_PER_S : SF_SPLIT_FLOPS_PER_S);
}

hipError_t launch_sf_apply(float* W, const float* U, const float* V, int64_t M, int64_t N, int64_t K, float lr,
                           hipStream_t stream, double spread_s, bool room)
{
    return launch_sf_arith<false>(W, nullptr, U, V, M, N, K, lr, 0.f, spread_s, room, stream);
}

hipError_t launch_sf_apply_momentum(float* W, float* buf, const float* U, const float* V, int64_t M, int64_t N,
                                    int64_t K, float lr, float mu, hipStream_t stream, double spread_s)
{
    return launch_sf_arith<true>(W, buf, U, V, M, N, K, lr, mu, spread_s, false, stream);
}

hipError_t launch_sf_apply_batch(const SfTensor* t, int32_t count, int64_t K, float lr, hipStream_t stream, bool room)
{
    if (sf_arithmetic() == POSEIDON_SF_FP32)
        return launch_batch<false>(t, count, K, lr, stream, room);
    return launch_batch<true>(t, count, K, lr, stream, room);
}

}  // namespace poseidon
