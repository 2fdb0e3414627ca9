// Gram matrices K = G G^T on the matrix cores (Section 3.2 initial setup:
// "evaluating G G^T in a straightforward fashion", O(d m^2); Section 3.1
// block-wise precompute, one m x m Gram per block).
//
// Tiling: one work-group (4 waves) per 64 x 64 lower-triangular output tile;
// each wave owns a 32 x 32 quadrant as 2 x 2 MFMA 16x16x4 tiles. Operands are
// staged through LDS in 64 x 32 fp32 panels (row pitch 36 floats: the 16-row x
// 4-k read pattern of one MFMA operand then hits every bank at most twice).
//
// Window Gram: fp32 MFMA (v_mfma_f32_16x16x4f32). The column range of the
// window is split over work-groups; each work-group flushes its fp32 MFMA
// accumulators into fp64 registers after every 2048-column slab, and the
// split partials are summed in fp64, in a fixed order, by k_gram_reduce.
// Static blocks: fp64 MFMA (v_mfma_f64_16x16x4f64) over the block's columns
// in 128 x 128 tiles, written straight into the block's padded fp64 matrix
// with m*lambda added on the diagonal, because the keep-mask is decided in fp64.
#include "internal.h"
#include "tile_util.h"

namespace mfac {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));
constexpr int KB = 32;     // columns per LDS stage
constexpr int PITCH = 36;  // LDS row pitch (floats)

__device__ __forceinline__ void tile_of(int idx, int& ti, int& tj) {
    int t = (int)((sqrtf(8.0f * (float)idx + 1.0f) - 1.0f) * 0.5f);
    while ((t + 1) * (t + 2) / 2 <= idx) ++t;
    while (t * (t + 1) / 2 > idx) --t;
    ti = t;
    tj = idx - t * (t + 1) / 2;
}

// Stage rows [r0, r0+64) x columns [k0, k0+KB) of a segment into LDS.
__device__ __forceinline__ void stage(float (*S)[PITCH], const float* __restrict__ base, int64_t ld,
                                      int r0, int m, int k0, int w) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int q = threadIdx.x + 256 * h;
        const int row = q >> 3;
        const int c4 = (q & 7) * 4;
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (r0 + row < m && k0 + c4 < w)
            v = *reinterpret_cast<const float4*>(base + (int64_t)(r0 + row) * ld + k0 + c4);
        *reinterpret_cast<float4*>(&S[row][c4]) = v;
    }
}

// One KB-column stage of MFMA work for this wave's 2x2 sub-tiles.
template <typename Acc, bool F64>
__device__ __forceinline__ void mfma_stage(float (*As)[PITCH], float (*Bs)[PITCH], int wr, int wc,
                                           int lane, Acc (&acc)[2][2]) {
    const int rl = lane & 15;
    const int kl = lane >> 4;
#pragma unroll
    for (int kk = 0; kk < KB / 4; ++kk) {
        float a[2], b[2];
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            a[s] = As[wr * 32 + s * 16 + rl][kk * 4 + kl];
            b[s] = Bs[wc * 32 + s * 16 + rl][kk * 4 + kl];
        }
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
            for (int y = 0; y < 2; ++y) {
                if constexpr (F64)
                    acc[x][y] = __builtin_amdgcn_mfma_f64_16x16x4f64((double)a[x], (double)b[y], acc[x][y], 0, 0, 0);
                else
                    acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[x], b[y], acc[x][y], 0, 0, 0);
            }
    }
}

// Window Gram partials: grid (ntiles, nsplit); split s sums slabs [s*sps, min(nslab, (s+1)*sps)).
__global__ __launch_bounds__(256) void k_gram_window(const float* __restrict__ G, int m, int64_t nslab,
                                                     int64_t sps, double* __restrict__ part, int ntiles) {
    __shared__ float As[64][PITCH];
    __shared__ float Bs[64][PITCH];
    int ti, tj;
    tile_of(blockIdx.x, ti, tj);
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int wr = wave >> 1, wc = wave & 1;
    const int64_t s0 = (int64_t)blockIdx.y * sps;
    int64_t s1 = s0 + sps;
    if (s1 > nslab) s1 = nslab;

    v4d accd[2][2];
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y) accd[x][y] = v4d{0.0, 0.0, 0.0, 0.0};

    for (int64_t s = s0; s < s1; ++s) {
        const float* base = G + s * (int64_t)m * SLAB;
        v4f acc[2][2];
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
            for (int y = 0; y < 2; ++y) acc[x][y] = v4f{0.f, 0.f, 0.f, 0.f};
        for (int k0 = 0; k0 < SLAB; k0 += KB) {
            stage(As, base, SLAB, ti * 64, m, k0, SLAB);
            if (ti != tj) stage(Bs, base, SLAB, tj * 64, m, k0, SLAB);
            __syncthreads();
            if (ti != tj)
                mfma_stage<v4f, false>(As, Bs, wr, wc, lane, acc);
            else
                mfma_stage<v4f, false>(As, As, wr, wc, lane, acc);
            __syncthreads();
        }
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
            for (int y = 0; y < 2; ++y)
#pragma unroll
                for (int r = 0; r < 4; ++r) accd[x][y][r] += (double)acc[x][y][r];
    }

    double* out = part + ((int64_t)blockIdx.y * ntiles + blockIdx.x) * (64 * 64);
    const int rl = lane & 15, kl = lane >> 4;
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                // fp32 MFMA result: lane l register r is row 4(l/16) + r
                const int row = wr * 32 + x * 16 + kl * 4 + r;
                const int col = wc * 32 + y * 16 + rl;
                out[row * 64 + col] = accd[x][y][r];
            }
}

// K[row][col] (both triangles) = sum over splits of the tile partials.
__global__ __launch_bounds__(256) void k_gram_reduce(const double* __restrict__ part, int nsplit,
                                                     int ntiles, int m, double* __restrict__ K) {
    int ti, tj;
    tile_of(blockIdx.x, ti, tj);
    for (int e = threadIdx.x; e < 64 * 64; e += 256) {
        const int rr = e >> 6, cc = e & 63;
        const int row = ti * 64 + rr, col = tj * 64 + cc;
        if (row >= m || col >= m) continue;
        double s = 0.0;
        for (int k = 0; k < nsplit; ++k) s += part[((int64_t)k * ntiles + blockIdx.x) * 4096 + e];
        K[(int64_t)row * m + col] = s;
        K[(int64_t)col * m + row] = s;
    }
}

// Static blocks, fp64 MFMA. One work-group per 128 x 128 lower-triangular tile
// of one block's Gram matrix (flattened over blocks, XCD-remapped so the tiles
// of a block share an L2); the block's columns stream through double-buffered
// LDS in 32-column chunks, the next chunk's loads in flight during the MFMAs.
constexpr int GT = 128;

__global__ __launch_bounds__(256) void k_gram_blocks(const float* __restrict__ G, int m, int64_t d, int B, int b0,
                                                     int ntiles, double mu, double* __restrict__ A, int mp) {
    __shared__ float As[2][GT][PITCH];
    __shared__ float Bs[2][GT][PITCH];
    const int lid = xcd_remap(blockIdx.x, gridDim.x);
    const int bl = lid / ntiles;
    int ti, tj;
    tile_of(lid - bl * ntiles, ti, tj);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wr = wave >> 1, wc = wave & 1;
    const int rl = lane & 15, kl = lane >> 4;
    const bool diag_tile = ti == tj;
    const float* base = G + (int64_t)(b0 + bl) * B;
    const int ra0 = ti * GT, rb0 = tj * GT;
    // staging: 128 rows x 32 columns per operand, 16 floats per thread
    const int sr = tid >> 1, sc = (tid & 1) * 16;
    float4 pa[4], pb[4];
    auto load_chunk = [&](int k0) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int col = k0 + sc + 4 * q;
            const bool okc = col < B;
            pa[q] = (ra0 + sr < m && okc) ? *reinterpret_cast<const float4*>(base + (int64_t)(ra0 + sr) * d + col)
                                          : make_float4(0.f, 0.f, 0.f, 0.f);
            if (!diag_tile)
                pb[q] = (rb0 + sr < m && okc) ? *reinterpret_cast<const float4*>(base + (int64_t)(rb0 + sr) * d + col)
                                              : make_float4(0.f, 0.f, 0.f, 0.f);
        }
    };
    auto store_chunk = [&](int buf) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            *reinterpret_cast<float4*>(&As[buf][sr][sc + 4 * q]) = pa[q];
            if (!diag_tile) *reinterpret_cast<float4*>(&Bs[buf][sr][sc + 4 * q]) = pb[q];
        }
    };

    v4d acc[4][4];
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y) acc[x][y] = v4d{0.0, 0.0, 0.0, 0.0};
    const int nchunk = (B + KB - 1) / KB;
    load_chunk(0);
    store_chunk(0);
    __syncthreads();
    for (int c = 0; c < nchunk; ++c) {
        const int buf = c & 1;
        if (c + 1 < nchunk) load_chunk((c + 1) * KB);
        float (*Ab)[PITCH] = As[buf];
        float (*Bb)[PITCH] = diag_tile ? As[buf] : Bs[buf];
#pragma unroll
        for (int kk = 0; kk < KB / 4; ++kk) {
            double av[4], bv[4];
#pragma unroll
            for (int x = 0; x < 4; ++x) av[x] = (double)Ab[wr * 64 + x * 16 + rl][kk * 4 + kl];
#pragma unroll
            for (int y = 0; y < 4; ++y) bv[y] = (double)Bb[wc * 64 + y * 16 + rl][kk * 4 + kl];
#pragma unroll
            for (int x = 0; x < 4; ++x)
#pragma unroll
                for (int y = 0; y < 4; ++y)
                    acc[x][y] = __builtin_amdgcn_mfma_f64_16x16x4f64(av[x], bv[y], acc[x][y], 0, 0, 0);
        }
        if (c + 1 < nchunk) store_chunk(buf ^ 1);
        __syncthreads();
    }
    double* Ab = A + (int64_t)bl * mp * mp;
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                // fp64 MFMA result: lane l register r is row (l/16) + 4r
                const int row = ra0 + wr * 64 + x * 16 + kl + 4 * r;
                const int col = rb0 + wc * 64 + y * 16 + rl;
                if (row < mp && col < mp) {
                    double v = acc[x][y][r];
                    if (row == col) v += (row < m) ? mu : 1.0;
                    Ab[(int64_t)row * mp + col] = v;
                }
            }
}

}  // namespace

int64_t gram_window_part_doubles(int m, int64_t nslab) {
    const int T = (int)ceil_div(m, 64);
    const int ntiles = T * (T + 1) / 2;
    int64_t nsplit = ceil_div(2048, ntiles);
    if (nsplit > nslab) nsplit = nslab;
    if (nsplit < 1) nsplit = 1;
    return nsplit * ntiles * 4096;
}

hipError_t launch_gram_window(const float* G, int m, int64_t nslab, double* part, double* K,
                              hipStream_t st) {
    const int T = (int)ceil_div(m, 64);
    const int ntiles = T * (T + 1) / 2;
    int64_t nsplit = ceil_div(2048, ntiles);
    if (nsplit > nslab) nsplit = nslab;
    if (nsplit < 1) nsplit = 1;
    const int64_t sps = ceil_div(nslab, nsplit);
    nsplit = ceil_div(nslab, sps);
    hipLaunchKernelGGL(k_gram_window, dim3(ntiles, (unsigned)nsplit), dim3(256), 0, st, G, m, nslab,
                       sps, part, ntiles);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_gram_reduce, dim3(ntiles), dim3(256), 0, st, part, (int)nsplit, ntiles, m, K);
    return hipGetLastError();
}

hipError_t launch_gram_blocks(const float* G, int m, int64_t d, int B, int b0, int nb, double mu,
                              double* A, int mp, hipStream_t st) {
    const int T = (int)ceil_div(mp, GT);
    const int ntiles = T * (T + 1) / 2;
    hipLaunchKernelGGL(k_gram_blocks, dim3((unsigned)(ntiles * nb)), dim3(256), 0, st, G, m, d, B, b0, ntiles, mu, A,
                       mp);
    return hipGetLastError();
}

}  // namespace mfac
