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

hipError_t launch_topk_mask(const double* scores, int64_t d, int64_t keep, SelectScratch sc, uint8_t* mask,
                            hipStream_t st) {
    if (d <= 0) return hipSuccess;
    if (keep <= 0 || keep >= d) {
        hipLaunchKernelGGL(k_fill_u8, dim3((unsigned)ceil_div(d, 256)), dim3(256), 0, st, mask, d,
                           (uint8_t)(keep <= 0 ? 0 : 1));
        return hipGetLastError();
    }
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
    hipLaunchKernelGGL(k_tie_count, dim3(sc.nchunk), dim3(256), 0, st, scores, d, sc.state, sc.chunk_cnt);
    hipLaunchKernelGGL(k_tie_scan, dim3(1), dim3(256), 0, st, sc.chunk_cnt, sc.nchunk);
    hipLaunchKernelGGL(k_mask, dim3(sc.nchunk), dim3(256), 0, st, scores, d, sc.state, sc.chunk_cnt, mask);
    return hipGetLastError();
}

}  // namespace mfac
