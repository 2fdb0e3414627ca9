// Queries of the static block-wise path over W (W_b = R_b^-1 G_b, written over
// G by the precompute; row-major m x d).
//
// IHVP (Appendix C eq. 9 with W for V and q): F_b^-1 x_b = (x_b - W_b^T W_b x_b)/lambda,
// in two passes over W like the dynamic path: pass 1 forms p_b = W_b x_b per
// column chunk (partial dots per chunk, reduced per block in fp64), pass 2
// forms alpha x - W_b^T c_b with c_b = scale * p_b. The OBS correction of
// Section 4.1 is the IHVP of x_j = theta_j / [F^-1]_jj on removed coordinates,
// negated. Element queries (eq. 5) are O(m) gathers of two W columns.
#include "device_util.h"
#include "internal.h"

namespace mfac {
namespace {

// pass-1 partials for up to 4 vectors at the narrowest chunk width (1024)
int64_t static_query_main_doubles(int64_t d, int B, int m) { return (d / B) * ceil_div(B, 1024) * (int64_t)m * 4; }

// Pass 1: column chunks of width 256*U inside the blocks, taken by a
// persistent grid (chunk c by work-group c mod gridDim.x).
// part[c][i*NV + v] = sum_{j in chunk c} W[i, j] x_v[j]: exact products of the
// fp32 values summed in fp64; each (row, vector) sum of the chunk comes from
// one wave and is stored directly.
template <int NV, int U>
__global__ __launch_bounds__(256) void k_sq_pass1(const float* __restrict__ W, int m, int64_t d, int B, int cpb,
                                                  int nchunk, const float* __restrict__ X, double* __restrict__ part) {
    constexpr int CW = 256 * U;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int mnv = m * NV;
    for (int c = blockIdx.x; c < nchunk; c += gridDim.x) {
        const int b = c / cpb, cb = c - (c / cpb) * cpb;
        const int64_t j0 = (int64_t)b * B + (int64_t)cb * CW;
        int64_t jend = (int64_t)(b + 1) * B;
        if (jend > j0 + CW) jend = j0 + CW;
        double* out = part + (int64_t)c * mnv;

        float4 vr[NV][U];
#pragma unroll
        for (int v = 0; v < NV; ++v)
#pragma unroll
            for (int u = 0; u < U; ++u) vr[v][u] = ld4(X + (int64_t)v * d, j0 + u * 256 + lane * 4, jend, 1);

        for (int i = wave; i < m; i += 8) {
            const bool has2 = i + 4 < m;
            const int i2 = has2 ? i + 4 : i;
            float4 ga[U], gb[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t j = j0 + u * 256 + lane * 4;
                ga[u] = (j < jend) ? ld_stream(W + (int64_t)i * d + j) : make_float4(0.f, 0.f, 0.f, 0.f);
                gb[u] = (j < jend) ? ld_stream(W + (int64_t)i2 * d + j) : make_float4(0.f, 0.f, 0.f, 0.f);
            }
            double sv[2 * NV];
#pragma unroll
            for (int v = 0; v < NV; ++v) {
                double a = 0.0, bb = 0.0;
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    a = dot4d(ga[u], vr[v][u], a);
                    bb = dot4d(gb[u], vr[v][u], bb);
                }
                sv[v] = a;
                sv[NV + v] = bb;
            }
            int idx;
            bool writer;
            const double tot = wave_reduce_many<2 * NV>(sv, lane, idx, writer);
            if (writer) {
                if (idx < NV)
                    out[i * NV + idx] = tot;
                else if (has2)
                    out[i2 * NV + (idx - NV)] = tot;
            }
        }
    }
}

// coef[b][t] = scale * sum_{cb < cpb} part[b*cpb + cb][t]   (fixed order, fp64)
__global__ __launch_bounds__(256) void k_sq_reduce(const double* __restrict__ part, int cpb, int mnv, double scale,
                                                   double* __restrict__ coef) {
    const int b = blockIdx.y;
    const int t = blockIdx.x * 256 + threadIdx.x;
    if (t >= mnv) return;
    double s = 0.0;
    for (int cb = 0; cb < cpb; ++cb) s += part[((int64_t)b * cpb + cb) * mnv + t];
    coef[(int64_t)b * mnv + t] = scale * s;
}

// Wide blocks (many chunks per block): first sum segments of SEG chunks in
// parallel, part2[(b*nseg + s)*mnv + t] = sum over chunks [s*SEG, (s+1)*SEG)
// (fixed order); k_sq_reduce then sums the nseg segments of each block.
constexpr int SEG = 64;
__global__ __launch_bounds__(256) void k_sq_reduce_seg(const double* __restrict__ part, int cpb, int nseg, int mnv,
                                                       double* __restrict__ part2) {
    const int bs = blockIdx.y;  // block * nseg + segment
    const int b = bs / nseg, sg = bs - (bs / nseg) * nseg;
    const int t = blockIdx.x * 256 + threadIdx.x;
    if (t >= mnv) return;
    const int c0 = sg * SEG, c1 = (c0 + SEG) < cpb ? (c0 + SEG) : cpb;
    double s = 0.0;
    for (int cb = c0; cb < c1; ++cb) s += part[((int64_t)b * cpb + cb) * mnv + t];
    part2[(int64_t)bs * mnv + t] = s;
}

// Pass 2: one wave per 256*U-column chunk of one block:
// y_v[j] = alpha * x_v[j] - sum_i coef[b][i*NV + v] W[i, j], summed in fp64
// (fp64 coefficients times fp32 W) and rounded to fp32 once. Rows go in
// batches of RB, all RB*U loads issued before the batch's first FMA.
template <int NV, int U, int RB>
__global__ __launch_bounds__(256) void k_sq_pass2(const float* __restrict__ W, int m, int64_t d, int B, int cpb2,
                                                  int64_t nwchunk, const double* __restrict__ coef,
                                                  const float* __restrict__ X, float alpha, float* __restrict__ Y) {
    constexpr int WCW = 256 * U;
    const int lane = threadIdx.x & 63;
    const int64_t c = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (c >= nwchunk) return;
    const int b = (int)(c / cpb2), cb = (int)(c - (c / cpb2) * cpb2);
    const int64_t j0 = (int64_t)b * B + (int64_t)cb * WCW;
    int64_t jend = (int64_t)(b + 1) * B;
    if (jend > j0 + WCW) jend = j0 + WCW;
    const double* cf = coef + (int64_t)b * m * NV;

    double acc[NV][U][4];
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int k = 0; k < 4; ++k) acc[v][u][k] = 0.0;
    auto fold = [&](const float4 (&g)[U], int i) {
#pragma unroll
        for (int v = 0; v < NV; ++v) {
            const double cv = cf[i * NV + v];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                acc[v][u][0] = fma(cv, (double)g[u].x, acc[v][u][0]);
                acc[v][u][1] = fma(cv, (double)g[u].y, acc[v][u][1]);
                acc[v][u][2] = fma(cv, (double)g[u].z, acc[v][u][2]);
                acc[v][u][3] = fma(cv, (double)g[u].w, acc[v][u][3]);
            }
        }
    };
    auto load = [&](float4 (&g)[U], int i) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t j = j0 + u * 256 + lane * 4;
            g[u] = (j < jend) ? ld_stream(W + (int64_t)i * d + j) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
    };
    int i = 0;
    for (; i + RB <= m; i += RB) {
        float4 g[RB][U];
#pragma unroll
        for (int r = 0; r < RB; ++r) load(g[r], i + r);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int r = 0; r < RB; ++r) fold(g[r], i + r);
    }
    for (; i < m; ++i) {
        float4 g[U];
        load(g, i);
        fold(g, i);
    }
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t j = j0 + u * 256 + lane * 4;
            if (j < jend) {
                const float4 x = *reinterpret_cast<const float4*>(X + (int64_t)v * d + j);
                float4 y;
                const double a = alpha;
                y.x = (float)(a * x.x - acc[v][u][0]);
                y.y = (float)(a * x.y - acc[v][u][1]);
                y.z = (float)(a * x.z - acc[v][u][2]);
                y.w = (float)(a * x.w - acc[v][u][3]);
                st_stream(Y + (int64_t)v * d + j, y);
            }
        }
}

// x_j = theta_j / [F^-1]_jj where keep_mask_j == 0, else 0
__global__ void k_obs_x(const float* __restrict__ theta, const uint8_t* __restrict__ keep,
                        const double* __restrict__ diag, int64_t d, float* __restrict__ x) {
    const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (j < d) x[j] = keep[j] ? 0.f : (float)((double)theta[j] / diag[j]);
}

// One wave per query: (delta_ij - sum_k W[k,i] W[k,j]) / lambda within a block.
__global__ __launch_bounds__(256) void k_static_element(const float* __restrict__ W, int m, int64_t d, int B,
                                                        int64_t nq, const int64_t* __restrict__ ij, double inv_lam,
                                                        double* __restrict__ out, int* __restrict__ err) {
    const int lane = threadIdx.x & 63;
    // one wave per query, grid-strided (the grid is capped)
    for (int64_t q = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); q < nq; q += (int64_t)gridDim.x * 4) {
        const int64_t i = ij[2 * q], j = ij[2 * q + 1];
        if (i < 0 || i >= d || j < 0 || j >= d) {
            if (lane == 0) {
                out[q] = __longlong_as_double(0x7ff8000000000000ll);
                atomicOr(err, 32);
            }
            continue;
        }
        if (i / B != j / B) {
            if (lane == 0) out[q] = 0.0;
            continue;
        }
        double s = 0.0;
        for (int k = lane; k < m; k += 64) s += (double)W[(int64_t)k * d + i] * (double)W[(int64_t)k * d + j];
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
        if (lane == 0) out[q] = ((i == j ? 1.0 : 0.0) - s) * inv_lam;
    }
}

template <int NV>
struct SqCfg {
    // Measured on the 17 GB W of the 2048-block workload (m = 1024) over chunk
    // widths, grids and rows in flight. Pass 1: 2048-column chunks up to 3
    // vectors (1024 for 4, which would spill at 2048) on a persistent grid of
    // GRID1 work-groups (0: one per chunk); pass 2: 512-column wave chunks
    // with RB2 rows of loads in flight.
    static constexpr int U = NV <= 3 ? 8 : 4;
    static constexpr int GRID1 = NV == 1 ? 256 : NV <= 3 ? 512 : 0;
    static constexpr int U2 = 2;
    static constexpr int RB2 = NV == 2 ? 8 : 4;
};

template <int NV>
hipError_t sq_ihvp_nv(const float* W, int m, int64_t d, int B, const float* X, float alpha, double pscale, float* Y,
                      double* part, double* coef, hipStream_t st) {
    constexpr int U = SqCfg<NV>::U, U2 = SqCfg<NV>::U2, RB2 = SqCfg<NV>::RB2;
    static_assert(256 * U >= 1024, "partials are sized for chunks of at least 1024 columns");
    const int nblocks = (int)(d / B);
    const int cpb = (int)ceil_div(B, 256 * U);
    const int nchunk = nblocks * cpb;
    constexpr int target = SqCfg<NV>::GRID1;
    const int grid = (target == 0 || nchunk < target) ? nchunk : target;
    hipLaunchKernelGGL((k_sq_pass1<NV, U>), dim3((unsigned)grid), dim3(256), 0, st, W, m, d, B, cpb, nchunk, X,
                       part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (cpb > SEG) {
        // part2 follows the pass-1 partials (static_query_part_doubles holds both)
        double* part2 = part + static_query_main_doubles(d, B, m);
        const int nseg = (int)ceil_div(cpb, SEG);
        hipLaunchKernelGGL(k_sq_reduce_seg, dim3((unsigned)ceil_div(m * NV, 256), (unsigned)(nblocks * nseg)),
                           dim3(256), 0, st, part, cpb, nseg, m * NV, part2);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(k_sq_reduce, dim3((unsigned)ceil_div(m * NV, 256), nblocks), dim3(256), 0, st, part2,
                           nseg, m * NV, pscale, coef);
    } else {
        hipLaunchKernelGGL(k_sq_reduce, dim3((unsigned)ceil_div(m * NV, 256), nblocks), dim3(256), 0, st, part,
                           cpb, m * NV, pscale, coef);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int cpb2 = (int)ceil_div(B, 256 * U2);
    const int64_t nw = (int64_t)nblocks * cpb2;
    hipLaunchKernelGGL((k_sq_pass2<NV, U2, RB2>), dim3((unsigned)ceil_div(nw, 4)), dim3(256), 0, st, W, m, d, B, cpb2, nw,
                       coef, X, alpha, Y);
    return hipGetLastError();
}

}  // namespace

int64_t static_query_part_doubles(int64_t d, int B, int m) {
    // pass-1 partials, then the per-segment sums of wide blocks
    return static_query_main_doubles(d, B, m) + (d / B) * ceil_div(ceil_div(B, 1024), SEG) * (int64_t)m * 4;
}

hipError_t launch_static_ihvp(const float* W, int m, int64_t d, int B, int n, const float* X, float alpha,
                              double pscale, float* Y, double* part, double* coef, hipStream_t st) {
    switch (n) {
        case 1: return sq_ihvp_nv<1>(W, m, d, B, X, alpha, pscale, Y, part, coef, st);
        case 2: return sq_ihvp_nv<2>(W, m, d, B, X, alpha, pscale, Y, part, coef, st);
        case 3: return sq_ihvp_nv<3>(W, m, d, B, X, alpha, pscale, Y, part, coef, st);
        case 4: return sq_ihvp_nv<4>(W, m, d, B, X, alpha, pscale, Y, part, coef, st);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_obs_x(const float* theta, const uint8_t* keep, const double* diag, int64_t d, float* x,
                        hipStream_t st) {
    hipLaunchKernelGGL(k_obs_x, dim3((unsigned)ceil_div(d, 256)), dim3(256), 0, st, theta, keep, diag, d, x);
    return hipGetLastError();
}

hipError_t launch_static_element(const float* W, int m, int64_t d, int B, int64_t nq, const int64_t* ij, double lam,
                                 double* out, int* err, hipStream_t st) {
    if (nq <= 0) return hipSuccess;
    int64_t grid = ceil_div(nq, 4);
    if (grid > 65536) grid = 65536;
    hipLaunchKernelGGL(k_static_element, dim3((unsigned)grid), dim3(256), 0, st, W, m, d, B, nq, ij,
                       1.0 / lam, out, err);
    return hipGetLastError();
}

}  // namespace mfac
