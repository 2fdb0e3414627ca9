// Static block-wise path: the inverse diagonal and the OBD keep-mask.
//
// Per block b (Section 3.1, block-wise paragraph): with L_b the Cholesky
// factor of G_b G_b^T + m*lambda*I, W_b = L_b^-1 G_b plays the role of the
// paper's V (Algorithm 3 writes V over G; here V_i = sqrt(q_i/lambda) W_i) and
// diag(F_b^-1) = (1 - sum_i W_b[i,:]^2) / lambda (Appendix C, diagonal
// extraction). k_trmm_diag forms W_b = Linv_b G_b tile by tile on fp64 MFMA,
// writes it over G in fp32 and accumulates the column sums of squares from the
// unrounded fp64 tiles. A work-group owns one 128-column slice of one block and
// walks the 128-row tiles from the bottom up, so every tile of G it still
// needs is untouched when it overwrites a finished one. Each tile's k-loop runs
// in 16-deep chunks through double-buffered LDS, the next chunk's global loads
// in flight during the current chunk's MFMAs.
//
// Keep-mask (Section 4.1, OBD saliency, global over all blocks): fp64 scores,
// then an 8-pass radix selection of the keep-th largest key (8-bit digits of
// the IEEE bit pattern, which orders non-negative doubles), then a mask pass
// that ranks exact ties by index with a deterministic chunked scan.
#include "internal.h"
#include "tile_util.h"

namespace mfac {
namespace {

constexpr int TM = 128, TN = 128, TK = 16;  // W tile rows x columns, k-chunk
constexpr int PA = TK + 2;                  // LDS pitch of the L^-1 chunk, [row][k] (doubles)
constexpr int PB = TN + 16;                 // LDS pitch of the G chunk, [k][col] (doubles)

// grid: nslice * nb work-groups (flattened, remapped); slice = TN columns of a
// block. Each work-group walks the 128-row tiles of its slice from the bottom
// up; tile r needs L^-1 columns [0, (r+1)*128) and the same rows of G, so G
// rows that tile r overwrites are never read again. Eight waves, each owning
// 32 x 64 of the tile as 2 x 4 MFMA tiles, and two work-groups per CU.
//
// Operand values that are never used load clamped, in-bounds addresses:
// L^-1 rows past mp, G rows past m (their L^-1 coefficients are the exact
// zeros above the diagonal; the K range stays inside the diagonal 128-block,
// whose upper part is zero) and columns past the slice. W rows past m (zero
// padding or clamped rows) are neither stored nor summed.
__global__ __launch_bounds__(512, 4) void k_trmm_diag(const double* __restrict__ Linv, int mp, int64_t bstride,
                                                      float* __restrict__ G, int m, int64_t d, int B, int b0,
                                                      int nslice, double inv_lam, double* __restrict__ diag) {
    __shared__ double As[2][TM][PA];
    __shared__ double Bs[2][TK][PB];
    __shared__ double red[4][TN];
    const int lid = xcd_remap(blockIdx.x, gridDim.x);
    const int bl = lid / nslice, sl = lid - (lid / nslice) * nslice;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wr = wave >> 1, wc = wave & 1;  // rows wr*32, columns wc*64
    const int rl = lane & 15, kl = lane >> 4;
    const int b = b0 + bl;
    const int c0 = sl * TN;
    const int ncol = (B - c0) < TN ? (B - c0) : TN;
    const double* __restrict__ Lb = Linv + (int64_t)bl * bstride;
    float* __restrict__ Gb = G + (int64_t)b * B + c0;
    const int T = (mp + TM - 1) / TM;

    // staging of one k-chunk: L^-1 rows [r0, r0+128) x cols [k0, k0+16), 4
    // doubles per thread (row tid/4, cols (tid%4)*4..+3); G rows [k0, k0+16) x
    // 128 columns, 4 floats per thread (row tid/32, cols (tid%32)*4..+3)
    const int ar = tid >> 2, ac = (tid & 3) * 4;
    const int br = tid >> 5, bc = (tid & 31) * 4;
    const int bcc = min(bc, ncol - 4);
    double2 ra0, ra1;
    float4 rb;
#define MFAC_TR_LOAD(R0_, K0_)                                                                  \
    {                                                                                          \
        const double* src_ = Lb + (int64_t)min((R0_) + ar, mp - 1) * mp + (K0_) + ac;          \
        ra0 = *reinterpret_cast<const double2*>(src_);                                         \
        ra1 = *reinterpret_cast<const double2*>(src_ + 2);                                     \
        rb = *reinterpret_cast<const float4*>(Gb + (int64_t)min((K0_) + br, m - 1) * d + bcc); \
    }
#define MFAC_TR_STORE(BUF_)                                                                     \
    {                                                                                          \
        double* ad_ = &As[BUF_][ar][ac];                                                       \
        ad_[0] = ra0.x;                                                                        \
        ad_[1] = ra0.y;                                                                        \
        ad_[2] = ra1.x;                                                                        \
        ad_[3] = ra1.y;                                                                        \
        double* bd_ = &Bs[BUF_][br][bc];                                                       \
        bd_[0] = rb.x;                                                                         \
        bd_[1] = rb.y;                                                                         \
        bd_[2] = rb.z;                                                                         \
        bd_[3] = rb.w;                                                                         \
    }

    double sq[4] = {0.0, 0.0, 0.0, 0.0};
    for (int r = T - 1; r >= 0; --r) {
        v4d acc[2][4];
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
            for (int y = 0; y < 4; ++y) acc[x][y] = v4d{0.0, 0.0, 0.0, 0.0};
        const int khi = min((r + 1) * TM, mp);
        const int nchunk = khi / TK;
        MFAC_TR_LOAD(r * TM, 0)
        MFAC_TR_STORE(0)
        __syncthreads();
        for (int c = 0; c < nchunk; ++c) {
            const int buf = c & 1;
            if (c + 1 < nchunk) MFAC_TR_LOAD(r * TM, (c + 1) * TK)
#pragma unroll
            for (int kk = 0; kk < TK / 4; ++kk) {
                double av[2], bv[4];
#pragma unroll
                for (int x = 0; x < 2; ++x) av[x] = As[buf][wr * 32 + x * 16 + rl][kk * 4 + kl];
#pragma unroll
                for (int y = 0; y < 4; ++y) bv[y] = Bs[buf][kk * 4 + kl][wc * 64 + y * 16 + rl];
#pragma unroll
                for (int x = 0; x < 2; ++x)
#pragma unroll
                    for (int y = 0; y < 4; ++y)
                        acc[x][y] = __builtin_amdgcn_mfma_f64_16x16x4f64(av[x], bv[y], acc[x][y], 0, 0, 0);
            }
            if (c + 1 < nchunk) MFAC_TR_STORE(buf ^ 1)
            __syncthreads();
        }
        // W tile r: write over G (fp32) and accumulate squares from the fp64 values
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
            for (int y = 0; y < 4; ++y)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int row = r * TM + wr * 32 + x * 16 + kl + 4 * q;  // fp64 MFMA: row (l/16) + 4q
                    const int col = wc * 64 + y * 16 + rl;
                    const double w = acc[x][y][q];
                    if (row < m) {
                        sq[y] += w * w;
                        if (col < ncol) Gb[(int64_t)row * d + col] = (float)w;
                    }
                }
    }
#undef MFAC_TR_LOAD
#undef MFAC_TR_STORE
    // column sums of squares: over kl (lanes +16, +32), then over the four wr
#pragma unroll
    for (int y = 0; y < 4; ++y) {
        sq[y] += __shfl_xor(sq[y], 16, 64);
        sq[y] += __shfl_xor(sq[y], 32, 64);
    }
    if (kl == 0) {
#pragma unroll
        for (int y = 0; y < 4; ++y) red[wr][wc * 64 + y * 16 + rl] = sq[y];
    }
    __syncthreads();
    if (tid < ncol)
        diag[(int64_t)b * B + c0 + tid] = (1.0 - ((red[0][tid] + red[1][tid]) + (red[2][tid] + red[3][tid]))) * inv_lam;
}

// fp32 MFMA variant (v_mfma_f32_16x16x4f32) for the fast static mode: the
// same walk as k_trmm_diag, 32-deep k-chunks of fp32 operands in LDS ([row][k]
// for L^-1 with a 36-float pitch, [k][column] for G with a 144-float pitch:
// the 16-row x 4-k and 4-k x 16-column read patterns of one MFMA operand hit
// distinct banks), L^-1 the fp32 factor's output. G is only read. W is
// stored (fp32, row stride d) when Wout is set; the column sums of squares of
// the fp32 W values are summed in fp64 and give the diagonal when diag is set.
constexpr int TK32 = 32;
constexpr int PA32 = TK32 + 4;   // [row][k] pitch (floats)
constexpr int PB32 = TN + 16;    // [k][column] pitch (floats)

__global__ __launch_bounds__(512, 2) void k_trmm32(const float* __restrict__ Linv, int mp, int64_t lstride,
                                                   const float* __restrict__ G, int m, int64_t d, int B, int b0,
                                                   int nslice, double inv_lam, double* __restrict__ diag,
                                                   float* __restrict__ Wout) {
    __shared__ float As[2][TM][PA32];
    __shared__ float Bs[2][TK32][PB32];
    __shared__ double red[4][TN];
    const int lid = xcd_remap(blockIdx.x, gridDim.x);
    const int bl = lid / nslice, sl = lid - (lid / nslice) * nslice;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // wave -> 32 x 64 piece (rows wr*32, columns wc*64). Waves w and w+4 share
    // a SIMD (round-robin placement); pairing row pieces {0, 3} and {1, 2}
    // there balances the chunks skipped in the diagonal 128-block below.
    const int wr = (wave & 2) ? ((wave & 4) ? 2 : 1) : ((wave & 4) ? 3 : 0);
    const int wc = wave & 1;
    const int rl = lane & 15, kl = lane >> 4;
    const int b = b0 + bl;
    const int c0 = sl * TN;
    const int ncol = (B - c0) < TN ? (B - c0) : TN;
    const float* __restrict__ Lb = Linv + (int64_t)bl * lstride;
    const float* __restrict__ Gb = G + (int64_t)b * B + c0;
    const int T = (mp + TM - 1) / TM;

    // staging of one k-chunk: L^-1 rows [r0, r0+128) x k [k0, k0+32), 8 per
    // thread (row tid/4, k (tid%4)*8 .. +7); G rows [k0, k0+32) x 128 columns,
    // 8 per thread (row tid/16, columns (tid%16)*8 .. +7)
    const int ar = tid >> 2, ac = (tid & 3) * 8;
    const int br = tid >> 4, bc = (tid & 15) * 8;
    // each float4 clamped on its own (ncol is a multiple of 4): the quads
    // inside the slice load their own columns, the others in-bounds data that
    // lands in columns nothing reads
    const int bc0 = min(bc, ncol - 4), bc1 = min(bc + 4, ncol - 4);
    float4 ra0, ra1, rb0, rb1;
    auto load = [&](int r0, int k0) {
        const int64_t arow = (int64_t)min(r0 + ar, mp - 1) * mp + k0 + ac;
        const float4* p = reinterpret_cast<const float4*>(Lb + arow);
        ra0 = p[0];
        ra1 = p[1];
        const float* gp = Gb + (int64_t)min(k0 + br, m - 1) * d;
        rb0 = *reinterpret_cast<const float4*>(gp + bc0);
        rb1 = *reinterpret_cast<const float4*>(gp + bc1);
    };
    auto store = [&](int buf) {
        float4* a = reinterpret_cast<float4*>(&As[buf][ar][ac]);
        a[0] = ra0;
        a[1] = ra1;
        float4* q = reinterpret_cast<float4*>(&Bs[buf][br][bc]);
        q[0] = rb0;
        q[1] = rb1;
    };

    double sq[4] = {0.0, 0.0, 0.0, 0.0};
    for (int r = T - 1; r >= 0; --r) {
        v4f acc[2][4];
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
            for (int y = 0; y < 4; ++y) acc[x][y] = v4f{0.f, 0.f, 0.f, 0.f};
        const int khi = min((r + 1) * TM, mp);
        const int nchunk = khi / TK32;
        load(r * TM, 0);
        store(0);
        __syncthreads();
        for (int c = 0; c < nchunk; ++c) {
            const int buf = c & 1;
            if (c + 1 < nchunk) load(r * TM, (c + 1) * TK32);
            // L^-1 is zero right of this wave's rows: chunks wholly there add nothing
            if (c * TK32 < r * TM + wr * 32 + 32) {
#pragma unroll
                for (int kk = 0; kk < TK32 / 4; ++kk) {
                    float av[2], bv[4];
#pragma unroll
                    for (int x = 0; x < 2; ++x) av[x] = As[buf][wr * 32 + x * 16 + rl][kk * 4 + kl];
#pragma unroll
                    for (int y = 0; y < 4; ++y) bv[y] = Bs[buf][kk * 4 + kl][wc * 64 + y * 16 + rl];
#pragma unroll
                    for (int x = 0; x < 2; ++x)
#pragma unroll
                        for (int y = 0; y < 4; ++y)
                            acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[x], bv[y], acc[x][y], 0, 0, 0);
                }
            }
            if (c + 1 < nchunk) store(buf ^ 1);
            __syncthreads();
        }
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
            for (int y = 0; y < 4; ++y)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int row = r * TM + wr * 32 + x * 16 + mfma32_row(lane, q);
                    const int col = wc * 64 + y * 16 + rl;
                    const float w = acc[x][y][q];
                    if (row < m) {
                        sq[y] += (double)w * (double)w;
                        if (Wout && col < ncol) Wout[(int64_t)row * d + (int64_t)b * B + c0 + col] = w;
                    }
                }
    }
    if (!diag) return;
    // column sums of squares: over the lanes of one column (+16, +32), then over the four wr
#pragma unroll
    for (int y = 0; y < 4; ++y) {
        sq[y] += __shfl_xor(sq[y], 16, 64);
        sq[y] += __shfl_xor(sq[y], 32, 64);
    }
    if (kl == 0) {
#pragma unroll
        for (int y = 0; y < 4; ++y) red[wr][wc * 64 + y * 16 + rl] = sq[y];
    }
    __syncthreads();
    if (tid < ncol)
        diag[(int64_t)b * B + c0 + tid] = (1.0 - ((red[0][tid] + red[1][tid]) + (red[2][tid] + red[3][tid]))) * inv_lam;
}

__global__ void k_diag_to_f32(const double* __restrict__ dg, int64_t d, float* __restrict__ out) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < d) out[i] = (float)dg[i];
}

__global__ void k_scores(const float* __restrict__ theta, const double* __restrict__ dg, int64_t d,
                         double* __restrict__ s, int* __restrict__ err) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= d) return;
    const double t = (double)theta[i];
    const double g = dg[i];
    if (!(g > 0.0) || !isfinite(g) || !isfinite(t)) atomicOr(err, 8);
    s[i] = t * t / (2.0 * g);
}

__device__ __forceinline__ unsigned long long key_of(double x) {
    return (unsigned long long)__double_as_longlong(x);
}

// state: [0] prefix, [1] mask, [2] remaining rank (1-based) among keys matching the prefix
__global__ void k_select_init(unsigned long long* state, unsigned int* hist, int64_t keep) {
    if (threadIdx.x == 0) {
        state[0] = 0ull;
        state[1] = 0ull;
        state[2] = (unsigned long long)keep;
    }
    hist[threadIdx.x] = 0u;
}

__global__ __launch_bounds__(256) void k_select_hist(const double* __restrict__ s, int64_t d,
                                                     const unsigned long long* __restrict__ state, int shift,
                                                     unsigned int* __restrict__ hist) {
    __shared__ unsigned int h[256];
    h[threadIdx.x] = 0u;
    __syncthreads();
    const unsigned long long prefix = state[0], mask = state[1];
    int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * 256;
    for (; i < d; i += stride) {
        const unsigned long long k = key_of(s[i]);
        if ((k & mask) == prefix) atomicAdd(&h[(unsigned)((k >> shift) & 255ull)], 1u);
    }
    __syncthreads();
    const unsigned int c = h[threadIdx.x];
    if (c) atomicAdd(&hist[threadIdx.x], c);
}

// Pick the digit holding the remaining rank, counting from the top digit down.
__global__ void k_select_pick(unsigned long long* state, unsigned int* hist, int shift) {
    __shared__ unsigned int h[256];
    h[threadIdx.x] = hist[threadIdx.x];
    __syncthreads();
    hist[threadIdx.x] = 0u;  // ready for the next pass
    if (threadIdx.x == 0) {
        unsigned long long rem = state[2];
        unsigned long long above = 0;
        int dsel = 0;
        for (int dg = 255; dg >= 0; --dg) {
            if (above + h[dg] >= rem) {
                dsel = dg;
                break;
            }
            above += h[dg];
        }
        state[0] |= ((unsigned long long)dsel) << shift;
        state[1] |= 255ull << shift;
        state[2] = rem - above;
    }
}

constexpr int CHUNK = 1024;  // elements per mask chunk (256 threads x 4)

__global__ __launch_bounds__(256) void k_tie_count(const double* __restrict__ s, int64_t d,
                                                   const unsigned long long* __restrict__ state,
                                                   unsigned int* __restrict__ cnt) {
    __shared__ unsigned int red[256];
    const unsigned long long T = state[0];
    const int64_t base = (int64_t)blockIdx.x * CHUNK + threadIdx.x * 4;
    unsigned int c = 0;
    for (int q = 0; q < 4; ++q)
        if (base + q < d && key_of(s[base + q]) == T) ++c;
    red[threadIdx.x] = c;
    __syncthreads();
    for (int o = 128; o > 0; o >>= 1) {
        if (threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
        __syncthreads();
    }
    if (threadIdx.x == 0) cnt[blockIdx.x] = red[0];
}

// exclusive scan of the per-chunk tie counts, in place (one work-group)
__global__ __launch_bounds__(256) void k_tie_scan(unsigned int* __restrict__ cnt, int n) {
    __shared__ unsigned int tot[256];
    const int per = (n + 255) / 256;
    const int lo = threadIdx.x * per;
    unsigned int s = 0;
    for (int i = lo; i < lo + per && i < n; ++i) s += cnt[i];
    tot[threadIdx.x] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned int run = 0;
        for (int k = 0; k < 256; ++k) {
            const unsigned int v = tot[k];
            tot[k] = run;
            run += v;
        }
    }
    __syncthreads();
    unsigned int run = tot[threadIdx.x];
    for (int i = lo; i < lo + per && i < n; ++i) {
        const unsigned int v = cnt[i];
        cnt[i] = run;
        run += v;
    }
}

__global__ __launch_bounds__(256) void k_mask(const double* __restrict__ s, int64_t d,
                                              const unsigned long long* __restrict__ state,
                                              const unsigned int* __restrict__ chunk_prefix,
                                              uint8_t* __restrict__ mask) {
    __shared__ unsigned int pre[256];
    const unsigned long long T = state[0];
    const unsigned long long need = state[2];  // ties kept, in index order
    const int64_t base = (int64_t)blockIdx.x * CHUNK + threadIdx.x * 4;
    unsigned long long k[4];
    unsigned int c = 0;
    for (int q = 0; q < 4; ++q) {
        k[q] = (base + q < d) ? key_of(s[base + q]) : 0ull;
        if (base + q < d && k[q] == T) ++c;
    }
    pre[threadIdx.x] = c;
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned int run = 0;
        for (int t = 0; t < 256; ++t) {
            const unsigned int v = pre[t];
            pre[t] = run;
            run += v;
        }
    }
    __syncthreads();
    unsigned long long rank = (unsigned long long)chunk_prefix[blockIdx.x] + pre[threadIdx.x];
    for (int q = 0; q < 4; ++q) {
        if (base + q >= d) break;
        uint8_t out;
        if (k[q] > T) {
            out = 1;
        } else if (k[q] == T) {
            out = rank < need ? 1 : 0;
            ++rank;
        } else {
            out = 0;
        }
        mask[base + q] = out;
    }
}

// ------------------------------------------------------------------ band of the fast mode
// The fast mode's diagonal carries the fp32 path's rounding. Its scores are
// exact enough to decide every coordinate whose score lies outside
// [t(1 - tau), t(1 + tau)], t the keep-th largest score, as long as the
// relative score error stays below tau / (1 + tau): such a coordinate is on
// the same side of the fp64 cut. The coordinates inside that band get their
// diagonal recomputed exactly in fp64 (k_band_refine), then the selection
// runs again.
__global__ __launch_bounds__(256) void k_band_collect(const double* __restrict__ s, int64_t d,
                                                      const unsigned long long* __restrict__ state, double tau,
                                                      unsigned int* __restrict__ count, unsigned int* __restrict__ list) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= d) return;
    const double t = __longlong_as_double((long long)state[0]);
    const double v = s[i];
    // zero scores (theta_j = 0) are exact in either precision
    if (v != 0.0 && fabs(v - t) <= tau * t) {
        const unsigned int k = atomicAdd(count, 1u);
        list[k] = (unsigned int)i;
    }
}

__device__ __forceinline__ double wave_sum_dbl(double x) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
    return x;
}

constexpr int BAND_THREADS = 512;
constexpr int BAND_WAVES = BAND_THREADS / 64;
constexpr int BAND_COLS = BAND_WAVES * 128;  // block columns per chunk of the matrix-free product
constexpr int BAND_MAXIT = 12;

// Work-group reductions (every thread gets the result); sh: BAND_WAVES doubles.
__device__ __forceinline__ double block_sum_band(double x, double* sh) {
    x = wave_sum_dbl(x);
    __syncthreads();
    if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = x;
    __syncthreads();
    double r = 0.0;
#pragma unroll
    for (int w = 0; w < BAND_WAVES; ++w) r += sh[w];
    return r;
}

__device__ __forceinline__ double block_max_band(double x, double* sh) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x = fmax(x, __shfl_xor(x, o, 64));
    __syncthreads();
    if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = x;
    __syncthreads();
    double r = 0.0;
#pragma unroll
    for (int w = 0; w < BAND_WAVES; ++w) r = fmax(r, sh[w]);
    return r;
}

// ------------------------------------------------------------------ band refinement, wide
// The refinement of k_band_refine for up to BR_SLOTS band coordinates at once,
// each of its steps a launch over the whole grid, so that every slot's passes
// over G_b and L^-1 run on many work-groups at the HBM rate (one work-group
// per coordinate streams a block at a small fraction of it). Slot c works on
// list[c]; BR_ITERS steps are launched, and k_band_refine finishes a slot
// that has not converged by then (from its x) and the coordinates past the
// slots. Every sum has a fixed order.
constexpr int BR_SLOTS = 64;
constexpr int BR_ITERS = 6;
constexpr int BR_CH = 4096;  // u columns staged in LDS by the residual pass

struct BandWork {
    double *x, *r, *z, *u;            // x, r, z: BR_SLOTS x mq; u: BR_SLOTS x B
    unsigned long long *wmax, *xmax;  // BR_ITERS x BR_SLOTS: max |update|, max |x| (non-negative doubles' bits)
    int mq;
};

__device__ __forceinline__ bool band_slot(const unsigned int* __restrict__ count,
                                          const unsigned int* __restrict__ list, int c, int B, int64_t& j,
                                          int64_t& b, int64_t& jj) {
    if ((unsigned int)c >= *count) return false;
    j = list[c];
    b = j / B;
    jj = j - b * B;
    return true;
}

// Whether slot c met k_band_refine's stopping test at a step before `it`.
__device__ __forceinline__ bool band_converged(const BandWork& w, int c, int it) {
    for (int t = 1; t < it; ++t) {
        const double wt = __longlong_as_double((long long)w.wmax[t * BR_SLOTS + c]);
        const double wp = __longlong_as_double((long long)w.wmax[(t - 1) * BR_SLOTS + c]);
        const double xt = __longlong_as_double((long long)w.xmax[t * BR_SLOTS + c]);
        if (wt * (wt / wp) <= 1e-13 * xt) return true;
    }
    return false;
}

// x = r = 0 for every slot (r's padding must read as zeros), statistics cleared
__global__ void k_br_init(BandWork w) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i < BR_SLOTS * w.mq) {
        w.x[i] = 0.0;
        w.r[i] = 0.0;
    }
    if (i < BR_ITERS * BR_SLOTS) {
        w.wmax[i] = 0ull;
        w.xmax[i] = 0ull;
    }
}

// u = G_b^T x. Grid (ceil(B / 256), BR_SLOTS), 16 waves: each lane four
// columns, each wave a sixteenth of the rows; the waves' sums added in order.
__global__ __launch_bounds__(1024) void k_br_u(const float* __restrict__ G, int m, int64_t d, int B,
                                               const unsigned int* __restrict__ count,
                                               const unsigned int* __restrict__ list, BandWork w, int it) {
    const int c = blockIdx.y;
    int64_t j, b, jj;
    if (!band_slot(count, list, c, B, j, b, jj) || band_converged(w, c, it)) return;
    __shared__ double xs[4096];
    __shared__ double red[16][256];
    const double* __restrict__ x = w.x + (int64_t)c * w.mq;
    for (int i = threadIdx.x; i < m; i += 1024) xs[i] = x[i];
    __syncthreads();
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int col = blockIdx.x * 256 + lane * 4;
    const bool ok = col < B;  // B is a multiple of 4: the quad is whole
    const int per = (m + 15) / 16;
    const int i0 = min(m, wave * per), i1 = min(m, i0 + per);
    const float* __restrict__ gp = G + b * B + (ok ? col : 0);
    double a0 = 0.0, a1 = 0.0, a2 = 0.0, a3 = 0.0;
    int i = i0;
    for (; i + 8 <= i1; i += 8) {
        float4 q[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) q[t] = *reinterpret_cast<const float4*>(gp + (int64_t)(i + t) * d);
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const double xv = xs[i + t];
            a0 += (double)q[t].x * xv;
            a1 += (double)q[t].y * xv;
            a2 += (double)q[t].z * xv;
            a3 += (double)q[t].w * xv;
        }
    }
    for (; i < i1; ++i) {
        const float4 q = *reinterpret_cast<const float4*>(gp + (int64_t)i * d);
        const double xv = xs[i];
        a0 += (double)q.x * xv;
        a1 += (double)q.y * xv;
        a2 += (double)q.z * xv;
        a3 += (double)q.w * xv;
    }
    red[wave][lane * 4 + 0] = a0;
    red[wave][lane * 4 + 1] = a1;
    red[wave][lane * 4 + 2] = a2;
    red[wave][lane * 4 + 3] = a3;
    __syncthreads();
    if (threadIdx.x < 256) {
        const int cc = blockIdx.x * 256 + threadIdx.x;
        if (cc < B) {
            double sum = 0.0;
#pragma unroll
            for (int v = 0; v < 16; ++v) sum += red[v][threadIdx.x];
            w.u[(int64_t)c * B + cc] = sum;
        }
    }
}

// r = g - G_b u - mu x (r = g at the first step, x = 0). Grid (ceil(m / 16),
// BR_SLOTS): four rows per wave, u staged through LDS in column chunks.
__global__ __launch_bounds__(256) void k_br_r(const float* __restrict__ G, int m, int64_t d, int B,
                                              const unsigned int* __restrict__ count,
                                              const unsigned int* __restrict__ list, BandWork w, double mu, int it) {
    const int c = blockIdx.y;
    int64_t j, b, jj;
    if (!band_slot(count, list, c, B, j, b, jj) || band_converged(w, c, it)) return;
    __shared__ double us[BR_CH];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int rb = blockIdx.x * 16 + wave * 4;
    const float* __restrict__ Gb = G + b * B;
    double a[4] = {0.0, 0.0, 0.0, 0.0};
    if (it > 0) {
        const double* __restrict__ u = w.u + (int64_t)c * B;
        for (int c0 = 0; c0 < B; c0 += BR_CH) {
            const int nc = min(BR_CH, B - c0);
            __syncthreads();
            for (int t = threadIdx.x; t < nc; t += 256) us[t] = u[c0 + t];
            __syncthreads();
            for (int cc = lane * 4; cc < nc; cc += 256) {
                float4 q[4];
#pragma unroll
                for (int t = 0; t < 4; ++t)
                    q[t] = keep4(rb + t < m,
                                 *reinterpret_cast<const float4*>(Gb + (int64_t)min(rb + t, m - 1) * d + c0 + cc));
#pragma unroll
                for (int t = 0; t < 4; ++t)
                    a[t] += (double)q[t].x * us[cc] + (double)q[t].y * us[cc + 1] + (double)q[t].z * us[cc + 2] +
                            (double)q[t].w * us[cc + 3];
            }
        }
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) a[t] = wave_sum_dbl(a[t]);
    if (lane == 0) {
        const double* __restrict__ x = w.x + (int64_t)c * w.mq;
        double* __restrict__ r = w.r + (int64_t)c * w.mq;
#pragma unroll
        for (int t = 0; t < 4; ++t)
            if (rb + t < m) r[rb + t] = (double)Gb[(int64_t)(rb + t) * d + jj] - a[t] - mu * x[rb + t];
    }
}

// z = L^-1 r. Grid (ceil(m / 16), BR_SLOTS): four rows per wave; row i reads
// its whole quads up to (i + 4) & ~3 (zeros past i inside its diagonal tile).
__global__ __launch_bounds__(256) void k_br_z(int m, int B, const float* __restrict__ L32, int mp, int64_t lstride,
                                              const unsigned int* __restrict__ count,
                                              const unsigned int* __restrict__ list, BandWork w, int it) {
    const int c = blockIdx.y;
    int64_t j, b, jj;
    if (!band_slot(count, list, c, B, j, b, jj) || band_converged(w, c, it)) return;
    __shared__ double rs[4096];
    const double* __restrict__ r = w.r + (int64_t)c * w.mq;
    for (int i = threadIdx.x; i < w.mq; i += 256) rs[i] = r[i];
    __syncthreads();
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int i0 = blockIdx.x * 16 + wave * 4;
    if (i0 >= m) return;
    const float* __restrict__ L = L32 + b * lstride;
    double a[4] = {0.0, 0.0, 0.0, 0.0};
    const int kend = (min(i0 + 3, m - 1) + 4) & ~3;
    for (int k = lane * 4; k < kend; k += 256) {
        float4 q[4];
#pragma unroll
        for (int t = 0; t < 4; ++t)
            q[t] = keep4(i0 + t < m && k < ((i0 + t + 4) & ~3),
                         *reinterpret_cast<const float4*>(L + (int64_t)min(i0 + t, m - 1) * mp + k));
#pragma unroll
        for (int t = 0; t < 4; ++t)
            a[t] += (double)q[t].x * rs[k] + (double)q[t].y * rs[k + 1] + (double)q[t].z * rs[k + 2] +
                    (double)q[t].w * rs[k + 3];
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) a[t] = wave_sum_dbl(a[t]);
    if (lane == 0) {
        double* __restrict__ z = w.z + (int64_t)c * w.mq;
#pragma unroll
        for (int t = 0; t < 4; ++t)
            if (i0 + t < m) z[i0 + t] = a[t];
    }
}

// x += L^-T z and the step's statistics. Grid (ceil(m / 64), BR_SLOTS): lane
// k of the 64 columns, each wave a quarter of the rows from the tile's first
// column down (entries above the diagonal masked), summed in wave order.
__global__ __launch_bounds__(256) void k_br_x(int m, int B, const float* __restrict__ L32, int mp, int64_t lstride,
                                              const unsigned int* __restrict__ count,
                                              const unsigned int* __restrict__ list, BandWork w, int it) {
    const int c = blockIdx.y;
    int64_t j, b, jj;
    if (!band_slot(count, list, c, B, j, b, jj) || band_converged(w, c, it)) return;
    __shared__ double zs[4096];
    __shared__ double part[4][64];
    const double* __restrict__ z = w.z + (int64_t)c * w.mq;
    for (int i = threadIdx.x; i < m; i += 256) zs[i] = z[i];
    __syncthreads();
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int k0 = blockIdx.x * 64, k = k0 + lane;
    const bool okk = k < m;
    const int per = (m - k0 + 3) / 4;
    const int i0 = min(m, k0 + wave * per), i1 = min(m, i0 + per);
    const float* __restrict__ lp = L32 + b * lstride + (okk ? k : 0);
    double a[8] = {0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0};
    int i = i0;
    for (; i + 16 <= i1; i += 16) {
        float q[16];
#pragma unroll
        for (int t = 0; t < 16; ++t) q[t] = lp[(int64_t)(i + t) * mp];
#pragma unroll
        for (int t = 0; t < 16; ++t) a[t & 7] += (i + t >= k) ? (double)q[t] * zs[i + t] : 0.0;
    }
    for (; i < i1; ++i) {
        const float q = lp[(int64_t)i * mp];
        a[0] += (i >= k) ? (double)q * zs[i] : 0.0;
    }
    part[wave][lane] = ((a[0] + a[1]) + (a[2] + a[3])) + ((a[4] + a[5]) + (a[6] + a[7]));
    __syncthreads();
    if (wave == 0) {
        double wmax = 0.0, xmax = 0.0;
        if (okk) {
            const double upd = ((part[0][lane] + part[1][lane]) + (part[2][lane] + part[3][lane]));
            double* __restrict__ x = w.x + (int64_t)c * w.mq;
            const double xn = x[k] + upd;
            x[k] = xn;
            wmax = fabs(upd);
            xmax = fabs(xn);
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
            wmax = fmax(wmax, __shfl_xor(wmax, o, 64));
            xmax = fmax(xmax, __shfl_xor(xmax, o, 64));
        }
        if (lane == 0) {
            atomicMax(&w.wmax[it * BR_SLOTS + c], (unsigned long long)__double_as_longlong(wmax));
            atomicMax(&w.xmax[it * BR_SLOTS + c], (unsigned long long)__double_as_longlong(xmax));
        }
    }
}

// The diagonal entry and score of every slot that converged within the
// launched steps (k_band_refine finishes the others). Grid BR_SLOTS.
__global__ __launch_bounds__(256) void k_br_final(const float* __restrict__ G, int m, int64_t d, int B,
                                                  const unsigned int* __restrict__ count,
                                                  const unsigned int* __restrict__ list, BandWork w, double lam,
                                                  double tau, const float* __restrict__ theta,
                                                  double* __restrict__ diag, double* __restrict__ scores,
                                                  int* __restrict__ err) {
    const int c = blockIdx.x;
    int64_t j, b, jj;
    if (!band_slot(count, list, c, B, j, b, jj) || !band_converged(w, c, BR_ITERS)) return;
    __shared__ double red[4];
    const double* __restrict__ x = w.x + (int64_t)c * w.mq;
    const float* __restrict__ Gb = G + b * B;
    double a = 0.0;
    for (int i = threadIdx.x; i < m; i += 256) a += (double)Gb[(int64_t)i * d + jj] * x[i];
    a = wave_sum_dbl(a);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = a;
    __syncthreads();
    if (threadIdx.x == 0) {
        const double S = (red[0] + red[1]) + (red[2] + red[3]);
        const double dg = (1.0 - S) / lam;
        diag[j] = dg;
        const double th = (double)theta[j];
        const double s_new = th * th / (2.0 * dg);
        if (!(fabs(scores[j] - s_new) <= 0.25 * tau * s_new)) atomicOr(err, 64);
        scores[j] = s_new;
        if (!(dg > 0.0) || !isfinite(dg)) atomicOr(err, 8);
    }
}

// The exact diagonal entry of one band coordinate j (block b, column g = G_b[:, j]):
// x = A^-1 g for A = G_b G_b^T + m*lambda*I by iterative refinement in fp64,
// x <- x + M (g - A x), where A x is applied matrix-free from the fp32 G
// (exact products, fp64 sums) and M = L^-T L^-1 is the fp32 copy of the
// block's inverse factor (the factor of the fp32-path Gram, a close
// preconditioner: each step multiplies the error by the contraction rho, of
// the order of that factor's relative error). It stops once the estimated
// remaining error, rho |w| with rho = |w_k| / |w_(k-1)| (w the last update),
// is below 1e-15 |x|; err |= 32 if that takes more than BAND_MAXIT steps.
// Then [F_b^-1]_jj = (1 - g.x) / lambda and its score. One work-group of 8
// waves per band coordinate, persistent over the band list; every sum has a
// fixed order, so the results do not depend on the schedule. LDS: x, r, z (m
// doubles each) and a chunk of G_b^T x. Entries below BR_SLOTS were refined
// by the wide kernels: the converged ones are skipped, the others resume from
// their x.
__global__ __launch_bounds__(BAND_THREADS) void k_band_refine(const float* __restrict__ G, int m, int64_t d, int B,
                                                              const float* __restrict__ L32, int mp, int64_t lstride,
                                                              const unsigned int* __restrict__ count,
                                                              const unsigned int* __restrict__ list, BandWork bw,
                                                              double lam, double tau, const float* __restrict__ theta,
                                                              double* __restrict__ diag, double* __restrict__ scores,
                                                              int* __restrict__ err) {
    extern __shared__ double sh[];
    const int mq = (m + 3) & ~3;  // vectors padded to whole quads (r's padding stays 0)
    double* x = sh;
    double* r = x + mq;
    double* z = r + mq;
    double* u = z + mq;
    __shared__ double red[BAND_WAVES];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const unsigned int n = *count;
    const double mu = (double)m * lam;
    for (unsigned int c = blockIdx.x; c < n; c += gridDim.x) {
        const bool resume = c < (unsigned int)BR_SLOTS;
        if (resume && band_converged(bw, (int)c, BR_ITERS)) continue;
        const int64_t j = list[c];
        const int64_t b = j / B;
        const int64_t jj = j - b * B;
        const float* __restrict__ Gb = G + b * B;
        const float* __restrict__ L = L32 + b * lstride;
        for (int i = tid; i < m; i += BAND_THREADS) x[i] = resume ? bw.x[(int64_t)c * bw.mq + i] : 0.0;
        double wprev = 0.0;
        bool conv = false;
        for (int it = 0; it < BAND_MAXIT && !conv; ++it) {
            __syncthreads();
            for (int i = tid; i < mq; i += BAND_THREADS) r[i] = 0.0;
            __syncthreads();
            // r = G_b (G_b^T x), column chunk by column chunk (x = 0 at a fresh first step)
            for (int c0 = 0; (it > 0 || resume) && c0 < B; c0 += BAND_COLS) {
                const int nc = min(BAND_COLS, B - c0);
                // u = G_b[:, chunk]^T x: wave w owns columns [128w, 128w + 128)
                // of the chunk, two per lane; sixteen rows of loads in flight
                // (rows are d floats apart: each load is its own translation)
                {
                    const int col = wave * 128 + lane * 2;
                    const bool ok = col < nc;  // nc is a multiple of 4: the pair is whole
                    const float* gp = Gb + c0 + (ok ? col : 0);
                    double a0 = 0.0, a1 = 0.0;
                    int i = 0;
                    for (; i + 16 <= m; i += 16) {
                        float2 q[16];
#pragma unroll
                        for (int t = 0; t < 16; ++t) q[t] = *reinterpret_cast<const float2*>(gp + (int64_t)(i + t) * d);
#pragma unroll
                        for (int t = 0; t < 16; ++t) {
                            a0 += (double)q[t].x * x[i + t];
                            a1 += (double)q[t].y * x[i + t];
                        }
                    }
                    for (; i < m; ++i) {
                        const float2 q = *reinterpret_cast<const float2*>(gp + (int64_t)i * d);
                        a0 += (double)q.x * x[i];
                        a1 += (double)q.y * x[i];
                    }
                    if (ok) {
                        u[col] = a0;
                        u[col + 1] = a1;
                    }
                }
                __syncthreads();
                // r_i += G_b[i, chunk] . u: four rows per wave at a time (their
                // loads in flight together), float4 per lane
                for (int i0 = wave * 4; i0 < m; i0 += BAND_WAVES * 4) {
                    double a[4] = {0.0, 0.0, 0.0, 0.0};
                    for (int cc = lane * 4; cc < nc; cc += 256) {
                        float4 q[4];
#pragma unroll
                        for (int t = 0; t < 4; ++t)
                            q[t] = (i0 + t < m) ? *reinterpret_cast<const float4*>(Gb + (int64_t)(i0 + t) * d + c0 + cc)
                                                : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
                        for (int t = 0; t < 4; ++t)
                            a[t] += (double)q[t].x * u[cc] + (double)q[t].y * u[cc + 1] +
                                    (double)q[t].z * u[cc + 2] + (double)q[t].w * u[cc + 3];
                    }
#pragma unroll
                    for (int t = 0; t < 4; ++t) a[t] = wave_sum_dbl(a[t]);
                    if (lane == 0)
#pragma unroll
                        for (int t = 0; t < 4; ++t)
                            if (i0 + t < m) r[i0 + t] += a[t];
                }
                __syncthreads();
            }
            // residual of the block system
            for (int i = tid; i < m; i += BAND_THREADS) r[i] = (double)Gb[(int64_t)i * d + jj] - r[i] - mu * x[i];
            __syncthreads();
            // z = L^-1 r: wave per row i, entries k <= i (the stored row is zero
            // from i + 1 to the end of its diagonal 128-block, so whole quads are read)
            for (int i0 = wave * 4; i0 < m; i0 += BAND_WAVES * 4) {
                // four rows at a time; row i reads its quads below (i + 4) & ~3
                double a[4] = {0.0, 0.0, 0.0, 0.0};
                const int kend = (min(i0 + 3, m - 1) + 4) & ~3;
                for (int k = lane * 4; k < kend; k += 256) {
                    float4 q[4];
#pragma unroll
                    for (int t = 0; t < 4; ++t)
                        q[t] = (i0 + t < m && k < ((i0 + t + 4) & ~3))
                                   ? *reinterpret_cast<const float4*>(L + (int64_t)(i0 + t) * mp + k)
                                   : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
                    for (int t = 0; t < 4; ++t)
                        a[t] += (double)q[t].x * r[k] + (double)q[t].y * r[k + 1] + (double)q[t].z * r[k + 2] +
                                (double)q[t].w * r[k + 3];
                }
#pragma unroll
                for (int t = 0; t < 4; ++t) a[t] = wave_sum_dbl(a[t]);
                if (lane == 0)
#pragma unroll
                    for (int t = 0; t < 4; ++t)
                        if (i0 + t < m) z[i0 + t] = a[t];
            }
            __syncthreads();
            // x += L^-T z: thread k sums column k over rows i >= k, sixteen
            // rows of loads in flight (coalesced across the wave)
            double wmax = 0.0, xmax = 0.0;
            for (int k = tid; k < m; k += BAND_THREADS) {
                const float* lp = L + k;
                double a[8] = {0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0};
                int i = k;
                for (; i + 16 <= m; i += 16) {
                    float q[16];
#pragma unroll
                    for (int t = 0; t < 16; ++t) q[t] = lp[(int64_t)(i + t) * mp];
#pragma unroll
                    for (int t = 0; t < 16; ++t) a[t & 7] += (double)q[t] * z[i + t];
                }
                for (; i < m; ++i) a[0] += (double)lp[(int64_t)i * mp] * z[i];
                const double w = ((a[0] + a[1]) + (a[2] + a[3])) + ((a[4] + a[5]) + (a[6] + a[7]));
                const double xn = x[k] + w;
                x[k] = xn;
                wmax = fmax(wmax, fabs(w));
                xmax = fmax(xmax, fabs(xn));
            }
            wmax = block_max_band(wmax, red);
            xmax = block_max_band(xmax, red);
            // estimated remaining error: the next update, rho |w| with the
            // contraction rho measured on the last two updates; 1e-13 of x is
            // the level at which two fp64 evaluations (this one, a Cholesky
            // solve) differ anyway
            conv = it > 0 && wmax * (wmax / wprev) <= 1e-13 * xmax;
            wprev = wmax;
        }
        if (!conv && tid == 0) atomicOr(err, 32);
        double a = 0.0;
        for (int i = tid; i < m; i += BAND_THREADS) a += (double)Gb[(int64_t)i * d + jj] * x[i];
        const double S = block_sum_band(a, red);
        if (tid == 0) {
            const double dg = (1.0 - S) / lam;
            diag[j] = dg;
            const double th = (double)theta[j];
            const double s_new = th * th / (2.0 * dg);
            // the fp32 path's error, measured at the cut: the band's width is
            // only safe while it stays well below tau
            if (!(fabs(scores[j] - s_new) <= 0.25 * tau * s_new)) atomicOr(err, 64);
            scores[j] = s_new;
            if (!(dg > 0.0) || !isfinite(dg)) atomicOr(err, 8);
        }
        __syncthreads();
    }
}

__global__ void k_fill_u32(unsigned int* __restrict__ p, int n, unsigned int v) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i < n) p[i] = v;
}

__global__ void k_fill_u8(uint8_t* __restrict__ p, int64_t n, uint8_t v) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n) p[i] = v;
}

}  // namespace

hipError_t launch_trmm_diag(const double* Linv, int mp, int64_t bstride, float* G, int m, int64_t d, int B,
                            int b0, int nb, double lam, double* diag, hipStream_t st) {
    const int nslice = (int)ceil_div(B, TN);
    hipLaunchKernelGGL(k_trmm_diag, dim3((unsigned)(nslice * nb)), dim3(512), 0, st, Linv, mp, bstride, G, m, d, B,
                       b0, nslice, 1.0 / lam, diag);
    return hipGetLastError();
}

hipError_t launch_trmm32(const float* Linv, int mp, int64_t lstride, const float* G, int m, int64_t d, int B, int b0,
                         int nb, double lam, double* diag, float* Wout, hipStream_t st) {
    const int nslice = (int)ceil_div(B, TN);
    hipLaunchKernelGGL(k_trmm32, dim3((unsigned)(nslice * nb)), dim3(512), 0, st, Linv, mp, lstride, G, m, d, B, b0,
                       nslice, 1.0 / lam, diag, Wout);
    return hipGetLastError();
}

hipError_t launch_diag_to_f32(const double* diag, int64_t d, float* out, hipStream_t st) {
    hipLaunchKernelGGL(k_diag_to_f32, dim3((unsigned)ceil_div(d, 256)), dim3(256), 0, st, diag, d, out);
    return hipGetLastError();
}

hipError_t launch_scores(const float* theta, const double* diag, int64_t d, double* scores, int* err,
                         hipStream_t st) {
    hipLaunchKernelGGL(k_scores, dim3((unsigned)ceil_div(d, 256)), dim3(256), 0, st, theta, diag, d, scores, err);
    return hipGetLastError();
}

int64_t select_scratch_bytes(int64_t d) {
    const int64_t nchunk = ceil_div(d, CHUNK);
    return 256 * 4 + 4 * 8 + round_up(nchunk * 4, 256) + 256;
}

SelectScratch select_scratch_carve(void* base, int64_t d) {
    SelectScratch s;
    char* p = (char*)base;
    s.hist = (unsigned int*)p;
    s.state = (unsigned long long*)(p + 1024);
    s.chunk_cnt = (unsigned int*)(p + 1024 + 256);
    s.nchunk = (int)ceil_div(d, CHUNK);
    return s;
}

namespace {
// The keep-th largest key into sc.state (8 radix passes); 0 < keep < d.
hipError_t select_kth(const double* scores, int64_t d, int64_t keep, SelectScratch sc, hipStream_t st) {
    hipLaunchKernelGGL(k_select_init, dim3(1), dim3(256), 0, st, sc.state, sc.hist, keep);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    int64_t hgrid = ceil_div(d, 256 * 16);
    if (hgrid > 2048) hgrid = 2048;
    for (int pass = 0; pass < 8; ++pass) {
        const int shift = 56 - 8 * pass;
        hipLaunchKernelGGL(k_select_hist, dim3((unsigned)hgrid), dim3(256), 0, st, scores, d, sc.state, shift,
                           sc.hist);
        hipLaunchKernelGGL(k_select_pick, dim3(1), dim3(256), 0, st, sc.state, sc.hist, shift);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}
}  // namespace

int64_t band_work_doubles(int m, int B) {
    const int64_t mq = (m + 3) & ~3;
    return (int64_t)BR_SLOTS * (3 * mq + B) + 2 * BR_ITERS * BR_SLOTS;
}

hipError_t launch_band_refine(const double* scores_in, int64_t d, int64_t keep, SelectScratch sc, double tau,
                              unsigned int* count, unsigned int* list, double* work, const float* G, int m, int B,
                              const float* L32, int mp, int64_t lstride, double lam, const float* theta,
                              double* diag, double* scores, int* err, hipStream_t st) {
    if (d <= 0 || keep <= 0 || keep >= d) return hipSuccess;  // the mask needs no cut
    hipError_t e = select_kth(scores_in, d, keep, sc, st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_fill_u32, dim3(1), dim3(256), 0, st, count, 1, 0u);
    hipLaunchKernelGGL(k_band_collect, dim3((unsigned)ceil_div(d, 256)), dim3(256), 0, st, scores_in, d, sc.state,
                       tau, count, list);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    BandWork w;
    w.mq = (m + 3) & ~3;
    w.x = work;
    w.r = w.x + (int64_t)BR_SLOTS * w.mq;
    w.z = w.r + (int64_t)BR_SLOTS * w.mq;
    w.u = w.z + (int64_t)BR_SLOTS * w.mq;
    w.wmax = reinterpret_cast<unsigned long long*>(w.u + (int64_t)BR_SLOTS * B);
    w.xmax = w.wmax + BR_ITERS * BR_SLOTS;
    const double mu = (double)m * lam;
    const unsigned rows16 = (unsigned)ceil_div(m, 16);
    const int64_t ninit = (int64_t)BR_SLOTS * w.mq > BR_ITERS * BR_SLOTS ? (int64_t)BR_SLOTS * w.mq : BR_ITERS * BR_SLOTS;
    hipLaunchKernelGGL(k_br_init, dim3((unsigned)ceil_div(ninit, 256)), dim3(256), 0, st, w);
    for (int it = 0; it < BR_ITERS; ++it) {
        if (it > 0)
            hipLaunchKernelGGL(k_br_u, dim3((unsigned)ceil_div(B, 256), BR_SLOTS), dim3(1024), 0, st, G, m, d, B,
                               count, list, w, it);
        hipLaunchKernelGGL(k_br_r, dim3(rows16, BR_SLOTS), dim3(256), 0, st, G, m, d, B, count, list, w, mu, it);
        hipLaunchKernelGGL(k_br_z, dim3(rows16, BR_SLOTS), dim3(256), 0, st, m, B, L32, mp, lstride, count, list, w,
                           it);
        hipLaunchKernelGGL(k_br_x, dim3((unsigned)ceil_div(m, 64), BR_SLOTS), dim3(256), 0, st, m, B, L32, mp,
                           lstride, count, list, w, it);
    }
    hipLaunchKernelGGL(k_br_final, dim3(BR_SLOTS), dim3(256), 0, st, G, m, d, B, count, list, w, lam, tau, theta,
                       diag, scores, err);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const size_t lds = (size_t)(3 * ((m + 3) & ~3) + BAND_COLS) * sizeof(double);
    if (lds > 65536) {
        e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_band_refine),
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(k_band_refine, dim3(256), dim3(BAND_THREADS), lds, st, G, m, d, B, L32, mp, lstride, count,
                       list, w, lam, tau, theta, diag, scores, err);
    return hipGetLastError();
}

hipError_t launch_topk_mask(const double* scores, int64_t d, int64_t keep, SelectScratch sc, uint8_t* mask,
                            hipStream_t st) {
    if (d <= 0) return hipSuccess;
    if (keep <= 0 || keep >= d) {
        hipLaunchKernelGGL(k_fill_u8, dim3((unsigned)ceil_div(d, 256)), dim3(256), 0, st, mask, d,
                           (uint8_t)(keep <= 0 ? 0 : 1));
        return hipGetLastError();
    }
    hipError_t e = select_kth(scores, d, keep, sc, st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_tie_count, dim3(sc.nchunk), dim3(256), 0, st, scores, d, sc.state, sc.chunk_cnt);
    hipLaunchKernelGGL(k_tie_scan, dim3(1), dim3(256), 0, st, sc.chunk_cnt, sc.nchunk);
    hipLaunchKernelGGL(k_mask, dim3(sc.nchunk), dim3(256), 0, st, scores, d, sc.state, sc.chunk_cnt, mask);
    return hipGetLastError();
}

}  // namespace mfac
