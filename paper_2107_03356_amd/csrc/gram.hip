// Gram matrices K = G G^T on the matrix cores (Section 3.2 initial setup:
// "evaluating G G^T in a straightforward fashion", O(d m^2); Section 3.1
// block-wise precompute, one m x m Gram per block).
//
// Tiling: one work-group (8 waves) per 128 x 128 lower-triangular output tile;
// each wave owns a 32 x 64 piece as 2 x 4 MFMA 16x16x4 tiles. Operands are
// staged through double-buffered LDS in 128 x 32 fp32 panels (row pitch 36
// floats: the 16-row x 4-k read pattern of one MFMA operand is conflict-free).
//
// Window Gram: fp64 MFMA (v_mfma_f64_16x16x4f64) on the fp32 window values
// (exact products, fp64 sums, as in the passes that keep K up to date). The
// column range of the window is split over work-groups and the split
// partials are summed in fp64, in a fixed order, by k_gram_reduce.
// Static blocks: fp64 MFMA (v_mfma_f64_16x16x4f64) over the block's columns
// in 128 x 128 tiles, written straight into the block's padded fp64 matrix
// with m*lambda added on the diagonal, because the keep-mask is decided in fp64.
// When a batch has too few tiles to fill the chip (few, wide blocks; B = d is
// the full-d precompute of Section 3.1) the block's columns are also split
// over work-groups and the fp64 partial tiles are summed in split order by
// k_gram_blocks_reduce.
// The fast static mode's k_gram_blocks32 runs the block Gram on fp32 MFMA in
// 256 x 256 tiles (see there).
#include "internal.h"
#include "tile_util.h"

namespace mfac {
namespace {

constexpr int KB = 32;     // columns per LDS stage
constexpr int PITCH = 36;  // LDS row pitch (floats)

__device__ __forceinline__ void tile_of(int idx, int& ti, int& tj) {
    int t = (int)((sqrtf(8.0f * (float)idx + 1.0f) - 1.0f) * 0.5f);
    while ((t + 1) * (t + 2) / 2 <= idx) ++t;
    while (t * (t + 1) / 2 > idx) --t;
    ti = t;
    tj = idx - t * (t + 1) / 2;
}

// Window Gram partials. Grid (ntiles, nsplit): work-group (t, s) computes the
// 128 x 128 lower tile t of K over slabs [s*sps, min(nslab, (s+1)*sps)). Eight
// waves, each owning a 32 x 64 piece as 2 x 4 fp64 MFMA tiles (two waves per
// SIMD hide each other's LDS and memory waits), operands converted from fp32
// as they are read from LDS. The slab's rows stream through double-buffered
// LDS in 32-column chunks (128 x 32 fp32 per operand), the next chunk's global
// loads in flight during the MFMAs. Rows past m load clamped, in-bounds data;
// only rows and columns below m of the partial are ever summed into K.
constexpr int WT = 128;  // window Gram tile

// Two work-groups per CU (4 waves per SIMD).
__global__ __launch_bounds__(512, 4) void k_gram_window(const float* __restrict__ G, int m, int64_t nslab,
                                                     int64_t sps, double* __restrict__ part, int ntiles) {
    __shared__ float As[2][WT][PITCH];
    __shared__ float Bs[2][WT][PITCH];
    int ti, tj;
    tile_of(blockIdx.x, ti, tj);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wr = wave >> 1, wc = wave & 1;  // rows wr*32, columns wc*64
    const int rl = lane & 15, kl = lane >> 4;
    // in a diagonal tile, waves whose piece lies wholly above the diagonal only
    // stage operands (the reduction reads the lower triangle of such tiles)
    const bool upper_wave = ti == tj && wr * 32 + 31 < wc * 64;
    const int64_t s0 = (int64_t)blockIdx.y * sps;
    const int64_t s1 = min(s0 + sps, nslab);

    // staging: 128 rows x 32 columns per operand, 8 floats per thread and operand
    const int sr = tid >> 2, sc = (tid & 3) * 8;
    const int64_t offa = (int64_t)min(ti * WT + sr, m - 1) * SLAB + sc;
    const int64_t offb = (int64_t)min(tj * WT + sr, m - 1) * SLAB + sc;
    // staged chunk: two float4 per operand, kept in named registers
    float4 pa0, pa1, pb0, pb1;
#define MFAC_GW_LOAD(S_, K0_)                                            \
    {                                                                    \
        const float* base_ = G + (S_) * (int64_t)m * SLAB + (K0_);       \
        const float4* a_ = reinterpret_cast<const float4*>(base_ + offa); \
        const float4* b_ = reinterpret_cast<const float4*>(base_ + offb); \
        pa0 = a_[0];                                                     \
        pa1 = a_[1];                                                     \
        pb0 = b_[0];                                                     \
        pb1 = b_[1];                                                     \
    }
#define MFAC_GW_STORE(BUF_)                                              \
    {                                                                    \
        float4* a_ = reinterpret_cast<float4*>(&As[BUF_][sr][sc]);       \
        float4* b_ = reinterpret_cast<float4*>(&Bs[BUF_][sr][sc]);       \
        a_[0] = pa0;                                                     \
        a_[1] = pa1;                                                     \
        b_[0] = pb0;                                                     \
        b_[1] = pb1;                                                     \
    }

    v4d accd[2][4];
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y) accd[x][y] = v4d{0.0, 0.0, 0.0, 0.0};
    constexpr int NCH = SLAB / KB;  // chunks per slab
    if (s0 < s1) {
        MFAC_GW_LOAD(s0, 0)
        MFAC_GW_STORE(0)
        __syncthreads();
    }
    int buf = 0;
    for (int64_t s = s0; s < s1; ++s) {
        for (int c = 0; c < NCH; ++c) {
            // next chunk: the following columns of this slab, or the next slab's first
            const bool more = c + 1 < NCH || s + 1 < s1;
            const int64_t sn = c + 1 < NCH ? s : s + 1;
            const int kn = c + 1 < NCH ? (c + 1) * KB : 0;
            if (more) MFAC_GW_LOAD(sn, kn)
            float (*Ab)[PITCH] = As[buf];
            float (*Bb)[PITCH] = Bs[buf];
            if (!upper_wave) {
#pragma unroll
                for (int kk = 0; kk < KB / 4; ++kk) {
                    double av[2], bv[4];
#pragma unroll
                    for (int x = 0; x < 2; ++x) av[x] = (double)Ab[wr * 32 + x * 16 + rl][kk * 4 + kl];
#pragma unroll
                    for (int y = 0; y < 4; ++y) bv[y] = (double)Bb[wc * 64 + y * 16 + rl][kk * 4 + kl];
#pragma unroll
                    for (int x = 0; x < 2; ++x)
#pragma unroll
                        for (int y = 0; y < 4; ++y)
                            accd[x][y] = __builtin_amdgcn_mfma_f64_16x16x4f64(av[x], bv[y], accd[x][y], 0, 0, 0);
                }
            }
            if (more) MFAC_GW_STORE(buf ^ 1)
            __syncthreads();
            buf ^= 1;
        }
    }

    if (upper_wave) return;
    double* out = part + ((int64_t)blockIdx.y * ntiles + blockIdx.x) * (WT * WT);
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                // fp64 MFMA result: lane l register r is row (l/16) + 4r
                const int row = wr * 32 + x * 16 + kl + 4 * r;
                const int col = wc * 64 + y * 16 + rl;
                out[row * WT + col] = accd[x][y][r];
            }
}

#undef MFAC_GW_LOAD
#undef MFAC_GW_STORE

// K[row][col] (both triangles) = sum over splits of the tile partials, in split
// order; a diagonal tile contributes its lower triangle (mirrored).
__global__ __launch_bounds__(256) void k_gram_reduce(const double* __restrict__ part, int nsplit,
                                                     int ntiles, int m, double* __restrict__ K) {
    int ti, tj;
    tile_of(blockIdx.x, ti, tj);
    for (int e = threadIdx.x; e < WT * WT; e += 256) {
        const int rr = e / WT, cc = e % WT;
        const int row = ti * WT + rr, col = tj * WT + cc;
        if (row >= m || col >= m || (ti == tj && rr < cc)) continue;  // diagonal tiles: lower triangle
        double s = 0.0;
        for (int k = 0; k < nsplit; ++k) s += part[((int64_t)k * ntiles + blockIdx.x) * (WT * WT) + e];
        K[(int64_t)row * m + col] = s;
        K[(int64_t)col * m + row] = s;
    }
}

// Static blocks, fp64 MFMA. One work-group per 128 x 128 lower-triangular tile
// of one block's Gram matrix and column split (flattened over blocks, splits
// and tiles, XCD-remapped so the tiles of one block and split share an L2);
// the split's columns stream through double-buffered LDS in 32-column chunks,
// the next chunk's loads in flight during the MFMAs.
constexpr int GT = 128;

// Eight waves per 128 x 128 tile, each owning 32 x 64 as 2 x 4 MFMA tiles, and
// two work-groups per CU (4 waves per SIMD hide each other's LDS and memory
// waits). Staged chunk values live in named registers. nsplit == 1: the tile
// goes straight into A (plus mu on the diagonal; with accum, added to what A
// holds instead, no mu); otherwise split s of the block's columns
// [s*kcols, min(B, (s+1)*kcols)) writes its fp64 partial tile to
// part[(block*nsplit + s)*ntiles + tile].
__global__ __launch_bounds__(512, 4) void k_gram_blocks(const float* __restrict__ G, int m, int64_t d, int B,
                                                        int b0, int ntiles, int nsplit, int kcols, double mu,
                                                        int accum, double* __restrict__ A, int mp,
                                                        double* __restrict__ part) {
    __shared__ float As[2][GT][PITCH];
    __shared__ float Bs[2][GT][PITCH];
    const int lid = xcd_remap(blockIdx.x, gridDim.x);
    const int per_block = ntiles * nsplit;
    const int bl = lid / per_block;
    const int rem = lid - bl * per_block;
    const int sp = rem / ntiles;
    const int tile = rem - sp * ntiles;
    int ti, tj;
    tile_of(tile, ti, tj);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wr = wave >> 1, wc = wave & 1;  // rows wr*32, columns wc*64
    const int rl = lane & 15, kl = lane >> 4;
    const bool diag_tile = ti == tj;
    // in a diagonal tile the part above the diagonal is never read (the
    // factorization uses the lower triangle): waves wholly above it only stage
    const bool upper_wave = diag_tile && wr * 32 + 31 < wc * 64;
    const int cbeg = sp * kcols;
    const int ncols = (B - cbeg) < kcols ? (B - cbeg) : kcols;
    const float* base = G + (int64_t)(b0 + bl) * B + cbeg;
    const int ra0 = ti * GT, rb0 = tj * GT;
    // staging: 128 rows x 32 columns per operand, 8 floats per thread and operand
    const int sr = tid >> 2, sc = (tid & 3) * 8;
    const bool oka = ra0 + sr < m, okb = rb0 + sr < m;
    // loads from clamped, in-bounds addresses (ncols is a positive multiple of
    // 4), the values outside the tile replaced by zeros in registers
    const float* rowa = base + (int64_t)min(ra0 + sr, m - 1) * d;
    const float* rowb = base + (int64_t)min(rb0 + sr, m - 1) * d;
    float4 pa0, pa1, pb0, pb1;
#define MFAC_GB_LOAD(K0_)                                                          \
    {                                                                                    \
        const int c_ = (K0_) + sc;                                                       \
        const int ca_ = min(c_, ncols - 4), cb_ = min(c_ + 4, ncols - 4);                \
        pa0 = *reinterpret_cast<const float4*>(rowa + ca_);                              \
        pa1 = *reinterpret_cast<const float4*>(rowa + cb_);                              \
        if (!diag_tile) {                                                                \
            pb0 = *reinterpret_cast<const float4*>(rowb + ca_);                          \
            pb1 = *reinterpret_cast<const float4*>(rowb + cb_);                          \
        }                                                                                \
    }
#define MFAC_GB_STORE(BUF_, K0_)                                                   \
    {                                                                                    \
        const int c_ = (K0_) + sc;                                                       \
        float4* a_ = reinterpret_cast<float4*>(&As[BUF_][sr][sc]);                       \
        a_[0] = keep4(oka && c_ < ncols, pa0);                                           \
        a_[1] = keep4(oka && c_ + 4 < ncols, pa1);                                       \
        if (!diag_tile) {                                                                \
            float4* b_ = reinterpret_cast<float4*>(&Bs[BUF_][sr][sc]);                   \
            b_[0] = keep4(okb && c_ < ncols, pb0);                                       \
            b_[1] = keep4(okb && c_ + 4 < ncols, pb1);                                   \
        }                                                                                \
    }

    v4d acc[2][4];
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y) acc[x][y] = v4d{0.0, 0.0, 0.0, 0.0};
    const int nchunk = (ncols + KB - 1) / KB;
    MFAC_GB_LOAD(0)
    MFAC_GB_STORE(0, 0)
    __syncthreads();
    for (int c = 0; c < nchunk; ++c) {
        const int buf = c & 1;
        if (c + 1 < nchunk) MFAC_GB_LOAD((c + 1) * KB)
        float (*Ab)[PITCH] = As[buf];
        float (*Bb)[PITCH] = diag_tile ? As[buf] : Bs[buf];
        if (!upper_wave) {
#pragma unroll
            for (int kk = 0; kk < KB / 4; ++kk) {
                double av[2], bv[4];
#pragma unroll
                for (int x = 0; x < 2; ++x) av[x] = (double)Ab[wr * 32 + x * 16 + rl][kk * 4 + kl];
#pragma unroll
                for (int y = 0; y < 4; ++y) bv[y] = (double)Bb[wc * 64 + y * 16 + rl][kk * 4 + kl];
#pragma unroll
                for (int x = 0; x < 2; ++x)
#pragma unroll
                    for (int y = 0; y < 4; ++y)
                        acc[x][y] = __builtin_amdgcn_mfma_f64_16x16x4f64(av[x], bv[y], acc[x][y], 0, 0, 0);
            }
        }
        if (c + 1 < nchunk) MFAC_GB_STORE(buf ^ 1, (c + 1) * KB)
        __syncthreads();
    }
#undef MFAC_GB_LOAD
#undef MFAC_GB_STORE
    if (upper_wave) return;
    if (nsplit > 1) {
        double* out = part + ((int64_t)bl * nsplit + sp) * ntiles * (GT * GT) + (int64_t)tile * (GT * GT);
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
            for (int y = 0; y < 4; ++y)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    out[(wr * 32 + x * 16 + kl + 4 * r) * GT + wc * 64 + y * 16 + rl] = acc[x][y][r];
        return;
    }
    double* Ab = A + (int64_t)bl * mp * mp;
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                // fp64 MFMA result: lane l register r is row (l/16) + 4r
                const int row = ra0 + wr * 32 + x * 16 + kl + 4 * r;
                const int col = rb0 + wc * 64 + y * 16 + rl;
                if (row < mp && col < mp) {
                    double v = acc[x][y][r];
                    if (accum)
                        v += Ab[(int64_t)row * mp + col];
                    else if (row == col)
                        v += (row < m) ? mu : 1.0;
                    Ab[(int64_t)row * mp + col] = v;
                }
            }
}

// A_b (lower triangle of every tile the factorization reads) = sum over the
// column splits of the partial tiles (TS x TS), in split order, plus mu on the diagonal
// (identity on the padding rows); with accum, the sum is added to A_b instead.
// Grid (ntiles, nb).
template <typename OT, int TS>
__global__ __launch_bounds__(256) void k_gram_blocks_reduce(const double* __restrict__ part, int nsplit, int ntiles,
                                                            int m, double mu, int accum, OT* __restrict__ A,
                                                            int mp) {
    const int tile = blockIdx.x, bl = blockIdx.y;
    int ti, tj;
    tile_of(tile, ti, tj);
    const double* src = part + (int64_t)bl * nsplit * ntiles * (TS * TS) + (int64_t)tile * (TS * TS);
    const int64_t sstride = (int64_t)ntiles * (TS * TS);
    OT* Ab = A + (int64_t)bl * mp * mp;
    for (int e = threadIdx.x; e < TS * TS; e += 256) {
        const int rr = e / TS, cc = e % TS;
        const int row = ti * TS + rr, col = tj * TS + cc;
        if (row >= mp || col >= mp || (ti == tj && rr < cc)) continue;
        double v = 0.0;
        for (int s = 0; s < nsplit; ++s) v += src[s * sstride + e];
        if (accum)
            v += (double)Ab[(int64_t)row * mp + col];
        else if (row == col)
            v += (row < m) ? mu : 1.0;
        Ab[(int64_t)row * mp + col] = (OT)v;
    }
}

// Static blocks on fp32 MFMA (v_mfma_f32_16x16x4f32), for the fast mode. At
// twice the fp64 rate the 128 x 128 tiles of k_gram_blocks are bound by
// their operand traffic out of L2, so this kernel takes 256 x 256 lower
// tiles: one work-group of 16 waves per tile and column split, each wave
// owning 64 x 64 as 4 x 4 MFMA tiles (two MFMAs per LDS read instead of
// 1.33, half the operand bytes per flop), 32-column chunks double-buffered
// in LDS (256 rows x 36 floats per operand: the 16-row x 4-k read of one
// MFMA operand on distinct banks), the next chunk's loads in flight during
// the MFMAs. Products accumulate in fp32 over at most SPLIT32 columns; wider
// blocks are split and the splits summed in fp64 (k_gram_blocks_reduce).
// In diagonal tiles the waves wholly above the diagonal only stage operands.
constexpr int GT32 = 256;
constexpr int KB32 = 32;
constexpr int PITCH32 = KB32 + 4;
constexpr int SPLIT32 = 2048;

__global__ __launch_bounds__(1024) void k_gram_blocks32(const float* __restrict__ G, int m, int64_t d, int B, int b0,
                                                        int ntiles, int nsplit, int kcols, double mu,
                                                        float* __restrict__ A, int mp, double* __restrict__ part) {
    __shared__ float As[2][GT32][PITCH32];
    __shared__ float Bs[2][GT32][PITCH32];
    const int lid = xcd_remap(blockIdx.x, gridDim.x);
    const int per_block = ntiles * nsplit;
    const int bl = lid / per_block;
    const int rem = lid - bl * per_block;
    const int sp = rem / ntiles;
    const int tile = rem - sp * ntiles;
    int ti, tj;
    tile_of(tile, ti, tj);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // wave -> 64 x 64 piece (rows wr*64, columns wc*64): a permutation under
    // which the ten pieces on or below the diagonal of a diagonal tile fall
    // 3, 2, 3, 2 on the four SIMDs whether waves go round-robin (wave & 3) or
    // in runs of four (wave >> 2), so such a tile costs three waves per SIMD
    const int code = (int)((0xbfed76ca98354021ull >> (4 * wave)) & 15u);
    const int wr = code >> 2, wc = code & 3;
    const int rl = lane & 15, kl = lane >> 4;
    const bool diag_tile = ti == tj;
    const bool upper_wave = diag_tile && wr < wc;
    const int cbeg = sp * kcols;
    const int ncols = (B - cbeg) < kcols ? (B - cbeg) : kcols;
    const float* base = G + (int64_t)(b0 + bl) * B + cbeg;
    const int ra0 = ti * GT32, rb0 = tj * GT32;
    // staging: 256 rows x 32 columns per operand, 8 floats per thread and operand
    const int sr = tid >> 2, sc = (tid & 3) * 8;
    const bool oka = ra0 + sr < m, okb = rb0 + sr < m;
    // loads from clamped, in-bounds addresses (ncols is a positive multiple of
    // 4), the values outside the tile replaced by zeros in registers
    const float* rowa = base + (int64_t)min(ra0 + sr, m - 1) * d;
    const float* rowb = base + (int64_t)min(rb0 + sr, m - 1) * d;
    float4 pa0, pa1, pb0, pb1;
#define MFAC_G32_LOAD(K0_)                                                          \
    {                                                                                    \
        const int c_ = (K0_) + sc;                                                       \
        const int ca_ = min(c_, ncols - 4), cb_ = min(c_ + 4, ncols - 4);                \
        pa0 = *reinterpret_cast<const float4*>(rowa + ca_);                              \
        pa1 = *reinterpret_cast<const float4*>(rowa + cb_);                              \
        if (!diag_tile) {                                                                \
            pb0 = *reinterpret_cast<const float4*>(rowb + ca_);                          \
            pb1 = *reinterpret_cast<const float4*>(rowb + cb_);                          \
        }                                                                                \
    }
#define MFAC_G32_STORE(BUF_, K0_)                                                   \
    {                                                                                    \
        const int c_ = (K0_) + sc;                                                       \
        float4* a_ = reinterpret_cast<float4*>(&As[BUF_][sr][sc]);                       \
        a_[0] = keep4(oka && c_ < ncols, pa0);                                           \
        a_[1] = keep4(oka && c_ + 4 < ncols, pa1);                                       \
        if (!diag_tile) {                                                                \
            float4* b_ = reinterpret_cast<float4*>(&Bs[BUF_][sr][sc]);                   \
            b_[0] = keep4(okb && c_ < ncols, pb0);                                       \
            b_[1] = keep4(okb && c_ + 4 < ncols, pb1);                                   \
        }                                                                                \
    }

    v4f acc[4][4];
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y) acc[x][y] = v4f{0.f, 0.f, 0.f, 0.f};
    const int nchunk = (ncols + KB32 - 1) / KB32;
    MFAC_G32_LOAD(0)
    MFAC_G32_STORE(0, 0)
    __syncthreads();
    for (int c = 0; c < nchunk; ++c) {
        const int buf = c & 1;
        if (c + 1 < nchunk) MFAC_G32_LOAD((c + 1) * KB32)
        float (*Ab)[PITCH32] = As[buf];
        float (*Bb)[PITCH32] = diag_tile ? As[buf] : Bs[buf];
        if (!upper_wave) {
#pragma unroll
            for (int kk = 0; kk < KB32 / 4; ++kk) {
                float av[4], bv[4];
#pragma unroll
                for (int x = 0; x < 4; ++x) av[x] = Ab[wr * 64 + x * 16 + rl][kk * 4 + kl];
#pragma unroll
                for (int y = 0; y < 4; ++y) bv[y] = Bb[wc * 64 + y * 16 + rl][kk * 4 + kl];
#pragma unroll
                for (int x = 0; x < 4; ++x)
#pragma unroll
                    for (int y = 0; y < 4; ++y)
                        acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[x], bv[y], acc[x][y], 0, 0, 0);
            }
        }
        if (c + 1 < nchunk) MFAC_G32_STORE(buf ^ 1, (c + 1) * KB32)
        __syncthreads();
    }
#undef MFAC_G32_LOAD
#undef MFAC_G32_STORE
    if (upper_wave) return;
    if (nsplit > 1) {
        double* out = part + ((int64_t)bl * nsplit + sp) * ntiles * (GT32 * GT32) + (int64_t)tile * (GT32 * GT32);
#pragma unroll
        for (int x = 0; x < 4; ++x)
#pragma unroll
            for (int y = 0; y < 4; ++y)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    out[(wr * 64 + x * 16 + mfma32_row(lane, r)) * GT32 + wc * 64 + y * 16 + rl] = acc[x][y][r];
        return;
    }
    float* Ab = A + (int64_t)bl * mp * mp;
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = ra0 + wr * 64 + x * 16 + mfma32_row(lane, r);
                const int col = rb0 + wc * 64 + y * 16 + rl;
                if (row < mp && col < mp) {
                    double v = (double)acc[x][y][r];
                    if (row == col) v += (row < m) ? mu : 1.0;
                    Ab[(int64_t)row * mp + col] = (float)v;
                }
            }
}

}  // namespace

namespace {
// splits of the slab range: enough work-groups for ~8 per CU
int64_t gram_window_splits(int m, int64_t nslab, int& ntiles) {
    const int T = (int)ceil_div(m, WT);
    ntiles = T * (T + 1) / 2;
    int64_t nsplit = ceil_div(2048, ntiles);
    if (nsplit > nslab) nsplit = nslab;
    if (nsplit < 1) nsplit = 1;
    const int64_t sps = ceil_div(nslab, nsplit);
    return ceil_div(nslab, sps);
}
}  // namespace

int64_t gram_window_part_doubles(int m, int64_t nslab) {
    int ntiles;
    const int64_t nsplit = gram_window_splits(m, nslab, ntiles);
    return nsplit * ntiles * (int64_t)(WT * WT);
}

hipError_t launch_gram_window(const float* G, int m, int64_t nslab, double* part, double* K,
                              hipStream_t st) {
    int ntiles;
    const int64_t nsplit = gram_window_splits(m, nslab, ntiles);
    const int64_t sps = ceil_div(nslab, nsplit);
    hipLaunchKernelGGL(k_gram_window, dim3(ntiles, (unsigned)nsplit), dim3(512), 0, st, G, m, nslab,
                       sps, part, ntiles);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_gram_reduce, dim3(ntiles), dim3(256), 0, st, part, (int)nsplit, ntiles, m, K);
    return hipGetLastError();
}

namespace {
// Column splits of a batch of nb blocks: none when the batch has >= 1024
// tiles; otherwise up to 2048 work-groups (four rounds of the 512 that are
// resident at once, two per CU, without a nearly empty fifth), each split
// >= 2048 columns (its fp64 partial tile stays small next to the operand
// reads). kcols is a multiple of the 32-column stage, so every split starts
// 16-byte aligned.
int gram_blocks_splits(int nb, int mp, int B, int& ntiles, int& kcols) {
    const int T = (int)ceil_div(mp, GT);
    ntiles = T * (T + 1) / 2;
    const int64_t wgs = (int64_t)nb * ntiles;
    int64_t ns = 1;
    if (wgs < 1024) {
        ns = 2048 / wgs;
        const int64_t maxs = B / 2048;
        if (ns > maxs) ns = maxs;
        if (ns < 1) ns = 1;
    }
    kcols = (int)round_up(ceil_div(B, ns), KB);
    return (int)ceil_div(B, kcols);
}

// Column splits of the fp32 kernel: at most SPLIT32 columns each (fp32 sums
// stay short), and more when a batch has fewer tiles than CUs (splits of at
// least SPLIT32 columns, up to ~1024 work-groups).
int gram32_splits(int nb, int mp, int B, int& ntiles, int& kcols) {
    const int T = (int)ceil_div(mp, GT32);
    ntiles = T * (T + 1) / 2;
    const int64_t wgs = (int64_t)nb * ntiles;
    int64_t ns = ceil_div(B, SPLIT32);
    if (wgs < 256) {
        int64_t fill = 1024 / wgs;
        if (fill > B / SPLIT32) fill = B / SPLIT32;
        if (fill > ns) ns = fill;
    }
    if (ns < 1) ns = 1;
    kcols = (int)round_up(ceil_div(B, ns), KB32);
    return (int)ceil_div(B, kcols);
}
}  // namespace

int64_t gram_blocks32_part_doubles(int nb, int mp, int B) {
    int ntiles, kcols;
    const int ns = gram32_splits(nb, mp, B, ntiles, kcols);
    return ns > 1 ? (int64_t)nb * ns * ntiles * (GT32 * GT32) : 0;
}

int64_t gram_blocks_part_doubles(int nb, int mp, int B) {
    int ntiles, kcols;
    const int ns = gram_blocks_splits(nb, mp, B, ntiles, kcols);
    return ns > 1 ? (int64_t)nb * ns * ntiles * (GT * GT) : 0;
}

hipError_t launch_gram_blocks32(const float* G, int m, int64_t d, int B, int b0, int nb, double mu, float* A,
                                int mp, double* part, hipStream_t st) {
    int ntiles, kcols;
    const int ns = gram32_splits(nb, mp, B, ntiles, kcols);
    hipLaunchKernelGGL(k_gram_blocks32, dim3((unsigned)(ntiles * ns * nb)), dim3(1024), 0, st, G, m, d, B, b0, ntiles,
                       ns, kcols, mu, A, mp, part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || ns == 1) return e;
    hipLaunchKernelGGL((k_gram_blocks_reduce<float, GT32>), dim3((unsigned)ntiles, (unsigned)nb), dim3(256), 0, st,
                       part, ns, ntiles, m, mu, 0, A, mp);
    return hipGetLastError();
}

hipError_t launch_gram_blocks(const float* G, int m, int64_t d, int B, int b0, int nb, double mu,
                              double* A, int mp, double* part, hipStream_t st, bool accumulate) {
    int ntiles, kcols;
    const int ns = gram_blocks_splits(nb, mp, B, ntiles, kcols);
    const int acc = accumulate ? 1 : 0;
    hipLaunchKernelGGL(k_gram_blocks, dim3((unsigned)(ntiles * ns * nb)), dim3(512), 0, st, G, m, d, B, b0, ntiles,
                       ns, kcols, mu, acc, A, mp, part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || ns == 1) return e;
    hipLaunchKernelGGL((k_gram_blocks_reduce<double, GT>), dim3((unsigned)ntiles, (unsigned)nb), dim3(256), 0, st,
                       part, ns, ntiles, m, mu, acc, A, mp);
    return hipGetLastError();
}

}  // namespace mfac
