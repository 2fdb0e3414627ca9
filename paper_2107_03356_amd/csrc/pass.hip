// Streaming passes over the window (the two O(dm) matrix-vector products of
// the dynamic algorithm, Section 3.2 complexity analysis; Appendix B: the
// update reuses p = G g for both the Gram row and the IHVP).
//
// Both passes are HBM-bound (0.5 flop per byte). The window is stored as
// column slabs (internal.h), so every wave reads rows of 8 KB contiguous and
// all rows of a slab lie in one contiguous m*8 KB region.
//
// A replace first writes the new gradient into its slot (k_write_row, 2 d
// floats of traffic), so both passes below are pure read streams: interleaving
// that write with pass 1's reads cost ~8% of pass 1's bandwidth on gfx950.
//
// Pass 1: every work-group owns a set of column chunks (and, when m * NV is
// large, one group of rows) and keeps per-row running sums in LDS. A wave
// takes R rows at a time, loads U float4 per lane and row (128-bit coalesced
// loads), multiplies with the register-resident vector chunks and reduces the
// R x NV sums across the wave with lane shuffles. Work-group partials go to a
// fp64 buffer, summed in a fixed order by the reduce kernel (deterministic,
// no float atomics).
//
// Pass 2, one vector (m <= 4096): each work-group owns whole slabs; its four
// waves take interleaved rows across the full slab width, so the work-group
// streams 32 KB-contiguous blocks as pass 1 does, and the four fp64 column
// partials of a slab are summed through LDS. Pass 2, several vectors: each
// wave owns one column chunk of the output and walks all m rows, accumulating
// coef[i] * G[i, chunk] in registers (coefficients staged in LDS); no
// cross-lane traffic.
#include <type_traits>

#include "device_util.h"
#include "internal.h"

namespace mfac {
namespace {

__global__ void k_fill_zero(float* __restrict__ p, int64_t n) {
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (; i < n; i += stride) p[i] = 0.f;
}

__global__ __launch_bounds__(256) void k_set_rows(float* __restrict__ G, int m, int64_t d,
                                                  int64_t ncolpad, int first,
                                                  const float* __restrict__ rows, int64_t ld,
                                                  int aligned) {
    const int64_t j = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
    if (j >= ncolpad) return;
    const int r = blockIdx.y;
    const float4 v = ld4(rows + (int64_t)r * ld, j, d, aligned);
    const int64_t slab = j / SLAB;
    const int64_t off = j - slab * SLAB;
    *reinterpret_cast<float4*>(G + slab * (int64_t)m * SLAB + (int64_t)(first + r) * SLAB + off) = v;
}

__global__ __launch_bounds__(256) void k_get_rows(const float* __restrict__ G, int m, int64_t d,
                                                  int first, float* __restrict__ rows, int64_t ld,
                                                  int aligned) {
    const int64_t j = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
    if (j >= d) return;
    const int r = blockIdx.y;
    const int64_t slab = j / SLAB;
    const int64_t off = j - slab * SLAB;
    const float4 v =
        *reinterpret_cast<const float4*>(G + slab * (int64_t)m * SLAB + (int64_t)(first + r) * SLAB + off);
    st4(rows + (int64_t)r * ld, j, d, aligned, v);
}

// Accumulation precision of the passes: fp64 (exact products, fp64 sums) for
// up to 4 fused vectors, fp32 per lane for wider fusions; the sums across
// lanes, chunks and work-groups are fp64 either way.
template <int NV>
struct AccType {
    static constexpr bool f64 = NV <= 4;
    using T = typename std::conditional<f64, double, float>::type;
};

// Work-group (x, y) takes chunks x, x + gridDim.x, ... of rows
// [y * mg, min(m, (y + 1) * mg)) and writes its row sums to
// part[(y * gridDim.x + x) * mg * NV + (row - y * mg) * NV + v].
template <int NV, int U, int R>
__global__ __launch_bounds__(256) void k_pass1(const float* __restrict__ G, int m, int mg, int64_t d,
                                               int64_t nchunk, VecIn vin, int aligned,
                                               double* __restrict__ part) {
    extern __shared__ double acc[];  // mg * NV running sums (fp64)
    constexpr int CW = 256 * U;     // chunk width (floats): 64 lanes x float4 x U
    constexpr int CPS = SLAB / CW;  // chunks per slab
    static_assert(SLAB % CW == 0, "chunk must tile the slab");
    static_assert(R * NV <= 64, "one wave reduces at most 64 sums at a time");
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int r0 = blockIdx.y * mg;
    const int r1 = r0 + mg < m ? r0 + mg : m;
    const int nv_rows = (r1 - r0) * NV;
    for (int t = threadIdx.x; t < nv_rows; t += 256) acc[t] = 0.0;
    __syncthreads();

    for (int64_t c = blockIdx.x; c < nchunk; c += gridDim.x) {
        const int64_t slab = c / CPS;
        const int off = (int)(c - slab * CPS) * CW;
        const int64_t j0 = slab * SLAB + off;
        const float* Gs = G + slab * (int64_t)m * SLAB + off + lane * 4;

        float4 vr[NV][U];
#pragma unroll
        for (int v = 0; v < NV; ++v)
#pragma unroll
            for (int u = 0; u < U; ++u) vr[v][u] = ld4(vin.v[v], j0 + u * 256 + lane * 4, d, aligned);

        // R rows per iteration: rows i, i + 4, ..., i + 4(R-1) of this wave; a
        // missing row re-reads row i and its sums are dropped (no branch around loads)
        for (int i = r0 + wave; i < r1; i += 4 * R) {
            int row[R];
#pragma unroll
            for (int r = 0; r < R; ++r) row[r] = i + 4 * r < r1 ? i + 4 * r : i;
            float4 g[R][U];
#pragma unroll
            for (int r = 0; r < R; ++r)
#pragma unroll
                for (int u = 0; u < U; ++u) g[r][u] = ld_stream(Gs + (int64_t)row[r] * SLAB + u * 256);
            // keep all R*U loads in flight before the first use (the scheduler
            // otherwise recycles a few load registers and waits on each load)
            __builtin_amdgcn_sched_barrier(0);
            // per-lane partial dots (value r*NV + v is row r's dot with vector
            // v): in fp64, exact products of the fp32 values, for up to 4
            // vectors; in fp32 for wider fusions, which would otherwise be
            // bound by the fp64 conversions and FMAs
            using T = typename AccType<NV>::T;
            T sv[R * NV];
#pragma unroll
            for (int v = 0; v < NV; ++v)
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    T a = 0;
#pragma unroll
                    for (int u = 0; u < U; ++u) {
                        if constexpr (AccType<NV>::f64)
                            a = dot4d(g[r][u], vr[v][u], a);
                        else
                            a = dot4(g[r][u], vr[v][u], a);
                    }
                    sv[r * NV + v] = a;
                }
            int idx;
            bool writer;
            const double tot = (double)wave_reduce_many<R * NV>(sv, lane, idx, writer);
            if (writer) {
                const int r = idx / NV, v = idx - (idx / NV) * NV;
                if (i + 4 * r < r1) acc[(i + 4 * r - r0) * NV + v] += tot;
            }
        }
    }
    __syncthreads();
    double* out = part + ((int64_t)blockIdx.y * gridDim.x + blockIdx.x) * mg * NV;
    for (int t = threadIdx.x; t < nv_rows; t += 256) out[t] = acc[t];
}

// p[row * nv + v] = sum over the gx work-groups of the row's group of their
// partials (layout of k_pass1), in a fixed order.
__global__ __launch_bounds__(256) void k_reduce_partials(const double* __restrict__ part, Pass1Grid pg, int nv,
                                                         int mnv, double* __restrict__ p) {
    __shared__ double red[16][17];
    const int to = threadIdx.x & 15;
    const int bg = threadIdx.x >> 4;
    const int t = blockIdx.x * 16 + to;
    double s = 0.0;
    if (t < mnv) {
        const int row = t / nv, v = t - (t / nv) * nv;
        const int g = row / pg.mg;
        const int64_t stride = (int64_t)pg.mg * nv;
        const double* src = part + (int64_t)g * pg.gx * stride + (int64_t)(row - g * pg.mg) * nv + v;
        // eight loads in flight, added in the order of b
        for (int b = bg; b < pg.gx; b += 16 * 8) {
            double q[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) q[u] = b + 16 * u < pg.gx ? src[(int64_t)(b + 16 * u) * stride] : 0.0;
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if (b + 16 * u < pg.gx) s += q[u];
        }
    }
    red[bg][to] = s;
    __syncthreads();
    if (bg == 0 && t < mnv) {
        double r = 0.0;
        for (int k = 0; k < 16; ++k) r += red[k][to];
        p[t] = r;
    }
}

// Row stride of the coefficients staged in LDS (in the accumulation type).
// fp32 rows from 3 vectors on are padded to quads and read as 16-byte words
// (+3% at 9 vectors over scalar reads); at most m * (NV + 3) * 4 <= 105 KB
// under m * NV <= 16384. fp64 rows stay unpadded (2 and 4 vectors are still
// read as pairs): m * NV * 8 <= 128 KB, where padding 3 vectors to 4 would
// pass the 160 KB of LDS above m = 5120.
template <int NV>
struct CoefStride {
    static constexpr int P = AccType<NV>::f64 ? NV : NV >= 3 ? (NV + 3) / 4 * 4 : NV;
};

template <int NV, int NP, typename T>
__device__ __forceinline__ void coef_row(const T* __restrict__ row, T (&cv)[NP]) {
    constexpr int W = 16 / sizeof(T);
    if constexpr (NP % W == 0) {
#pragma unroll
        for (int q = 0; q < NP / W; ++q) {
            if constexpr (W == 2) {
                const double2 t = *reinterpret_cast<const double2*>(row + 2 * q);
                cv[2 * q] = t.x;
                cv[2 * q + 1] = t.y;
            } else {
                const float4 t = *reinterpret_cast<const float4*>(row + 4 * q);
                cv[4 * q] = t.x;
                cv[4 * q + 1] = t.y;
                cv[4 * q + 2] = t.z;
                cv[4 * q + 3] = t.w;
            }
        }
    } else {
#pragma unroll
        for (int v = 0; v < NV; ++v) cv[v] = row[v];
    }
}

// Pass 2: y_v = alpha_v x_v - sum_i coef[i][v] G[i, :], the coefficients and
// sums in the accumulation type of AccType (fp64: each window value converted
// once per row), rounded to fp32 on the store. Each wave owns a 256*U-column
// chunk and walks all m rows with RB rows of loads in flight.
template <int NV, int U, int RB>
__global__ __launch_bounds__(256) void k_pass2(const float* __restrict__ G, int m, int64_t d,
                                               int64_t nwchunk, const double* __restrict__ coef,
                                               VecOut vout, int aligned) {
    using T = typename AccType<NV>::T;
    constexpr int NP = CoefStride<NV>::P;
    extern __shared__ __align__(16) unsigned char cl_raw[];
    T* cl = reinterpret_cast<T*>(cl_raw);  // m rows of NP coefficients (NV used)
    constexpr int WCW = 256 * U;    // wave chunk width (floats)
    constexpr int CPS = SLAB / WCW;
    static_assert(SLAB % WCW == 0, "chunk must tile the slab");
    for (int t = threadIdx.x; t < m * NP; t += 256) {
        const int i = t / NP, v = t - (t / NP) * NP;
        cl[t] = v < NV ? (T)coef[i * NV + v] : T(0);
    }
    __syncthreads();
    const int lane = threadIdx.x & 63;
    const int64_t c = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (c >= nwchunk) return;
    const int64_t slab = c / CPS;
    const int off = (int)(c - slab * CPS) * WCW;
    const int64_t j0 = slab * SLAB + off;
    const float* Gs = G + slab * (int64_t)m * SLAB + off + lane * 4;

    T acc[NV][U][4];
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int u = 0; u < U; ++u) acc[v][u][0] = acc[v][u][1] = acc[v][u][2] = acc[v][u][3] = T(0);

    // RB rows per batch: all RB*U loads are issued before the first FMA
    auto fold = [&](const float4 (&g)[U], const T* crow) {
        T cv[NP];
        coef_row<NV, NP>(crow, cv);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const T gx = g[u].x, gy = g[u].y, gz = g[u].z, gw = g[u].w;
#pragma unroll
            for (int v = 0; v < NV; ++v) {
                acc[v][u][0] = fma(cv[v], gx, acc[v][u][0]);
                acc[v][u][1] = fma(cv[v], gy, acc[v][u][1]);
                acc[v][u][2] = fma(cv[v], gz, acc[v][u][2]);
                acc[v][u][3] = fma(cv[v], gw, acc[v][u][3]);
            }
        }
    };
    int i = 0;
    for (; i + RB <= m; i += RB) {
        float4 g[RB][U];
#pragma unroll
        for (int r = 0; r < RB; ++r)
#pragma unroll
            for (int u = 0; u < U; ++u) g[r][u] = ld_stream(Gs + (int64_t)(i + r) * SLAB + u * 256);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int r = 0; r < RB; ++r) fold(g[r], cl + (i + r) * NP);
    }
    for (; i < m; ++i) {
        float4 g[U];
#pragma unroll
        for (int u = 0; u < U; ++u) g[u] = ld_stream(Gs + (int64_t)i * SLAB + u * 256);
        fold(g, cl + i * NP);
    }

#pragma unroll
    for (int v = 0; v < NV; ++v) {
        const float a = vout.alpha[v];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t j = j0 + u * 256 + lane * 4;
            float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
            if (a != 0.f) x = ld4(vout.x[v], j, d, aligned);
            float4 y;
            y.x = (float)((T)a * (T)x.x - acc[v][u][0]);
            y.y = (float)((T)a * (T)x.y - acc[v][u][1]);
            y.z = (float)((T)a * (T)x.z - acc[v][u][2]);
            y.w = (float)((T)a * (T)x.w - acc[v][u][3]);
            st4_stream(vout.y[v], j, d, aligned, y);
        }
    }
}

// Pass 2 for one vector, y = alpha x - G^T coef, m <= 4096. Work-group b
// takes slabs b, b + gridDim.x, ...; wave w folds rows w, w + 4, ... over the
// full slab width (8 float4 per lane), issuing the next row's loads as soon
// as a row is folded and the next slab's first row before the slab's
// reduction. The four fp64 column partials of a slab go through LDS (two
// buffers, so one LDS barrier per slab) and are summed in a fixed order.
__device__ __forceinline__ void load_slab_row(float4 (&g)[8], const float* __restrict__ G, int m, int64_t s, int i,
                                              int lane) {
    const float* p = G + (s * m + i) * (int64_t)SLAB + lane * 4;
#pragma unroll
    for (int u = 0; u < 8; ++u) g[u] = ld_stream(p + u * 256);
}

// Waits for this wave's LDS operations, then for every wave of the
// work-group; outstanding global loads stay in flight.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

constexpr int PASS2_ROWS_MAX_M = 4096;  // m coefficients + 2 x 4 x SLAB partials = 160 KB of LDS
constexpr int PASS2_ROWS_GRID = 256;    // one work-group per CU (the LDS holds one)

__global__ __launch_bounds__(256) void k_pass2_rows(const float* __restrict__ G, int m, int64_t d, int64_t nslab,
                                                    const double* __restrict__ coef, VecOut vout, int aligned) {
    extern __shared__ __align__(16) double sh[];
    const int mpad = (m + 1) & ~1;  // keeps the partials 16-byte aligned
    double* cl = sh;
    double* red = sh + mpad;  // [2][4][SLAB]
    for (int t = threadIdx.x; t < m; t += 256) cl[t] = coef[t];
    __syncthreads();
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const float alpha = vout.alpha[0];
    const float* __restrict__ x = vout.x[0];
    float* __restrict__ y = vout.y[0];
    float4 g[8];
    int64_t s = blockIdx.x;
    if (s < nslab && wave < m) load_slab_row(g, G, m, s, wave, lane);
    for (int t = 0; s < nslab; s += gridDim.x, ++t) {
        double acc[8][4];
#pragma unroll
        for (int u = 0; u < 8; ++u) acc[u][0] = acc[u][1] = acc[u][2] = acc[u][3] = 0.0;
        for (int i = wave; i < m; i += 4) {
            const double cv = cl[i];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                acc[u][0] = fma(cv, (double)g[u].x, acc[u][0]);
                acc[u][1] = fma(cv, (double)g[u].y, acc[u][1]);
                acc[u][2] = fma(cv, (double)g[u].z, acc[u][2]);
                acc[u][3] = fma(cv, (double)g[u].w, acc[u][3]);
            }
            if (i + 4 < m)
                load_slab_row(g, G, m, s, i + 4, lane);
            else if (s + gridDim.x < nslab)
                load_slab_row(g, G, m, s + gridDim.x, wave, lane);
        }
        double* rb = red + (t & 1) * 4 * SLAB;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            double* q = rb + wave * SLAB + u * 256 + lane * 4;
            *reinterpret_cast<double2*>(q) = make_double2(acc[u][0], acc[u][1]);
            *reinterpret_cast<double2*>(q + 2) = make_double2(acc[u][2], acc[u][3]);
        }
        lds_barrier();
        // wave w writes columns [512 w, 512 w + 512) of the slab
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int col = wave * 512 + h * 256 + lane * 4;
            const int64_t j = s * SLAB + col;
            double sum[4];
#pragma unroll
            for (int k = 0; k < 4; ++k)
                sum[k] = rb[col + k] + rb[SLAB + col + k] + rb[2 * SLAB + col + k] + rb[3 * SLAB + col + k];
            float4 xv = make_float4(0.f, 0.f, 0.f, 0.f);
            if (alpha != 0.f) xv = ld4(x, j, d, aligned);
            const double a = alpha;
            float4 o;
            o.x = (float)(a * xv.x - sum[0]);
            o.y = (float)(a * xv.y - sum[1]);
            o.z = (float)(a * xv.z - sum[2]);
            o.w = (float)(a * xv.w - sum[3]);
            st4_stream(y, j, d, aligned, o);
        }
    }
}

// Pass 2 of one step fused with pass 1 of the next, for a sequence of
// gradients that are all known in advance (m <= PASS21_MAX_M). In the one
// read of the window it forms y = -G^T coef exactly as k_pass2_rows does
// (same order of every sum, so y is bitwise the same for the same
// coefficients) and the dots of every row with the next gradient gn. Row
// knext, the slot gn will take after this pass, gets gn . gn instead of its
// current row's dot, which makes the dots those of the window after the
// insertion. The dots follow the precision of k_pass1 for one vector (exact
// fp32 products summed in fp64): each wave reduces the per-lane sums of RB
// of its rows at a time across its lanes, and the work-group keeps fp64 row
// sums in LDS, written out in the partial layout of k_pass1 (one row group).
constexpr int PASS21_RB = 8;

__global__ __launch_bounds__(256) void k_pass2_next(const float* __restrict__ G, int m, int64_t d, int64_t nslab,
                                                    const double* __restrict__ coef, float* __restrict__ y,
                                                    const float* __restrict__ gn, int knext, int aligned,
                                                    double* __restrict__ part) {
    extern __shared__ __align__(16) double sh[];
    const int mpad = (m + 1) & ~1;  // keeps the partials 16-byte aligned
    double* cl = sh;
    double* rs = sh + mpad;    // row sums of this work-group's slabs
    double* red = rs + mpad;   // [2][4][SLAB]
    for (int t = threadIdx.x; t < m; t += 256) {
        cl[t] = coef[t];
        rs[t] = 0.0;
    }
    __syncthreads();
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    float4 g[8], gv[8];
    int64_t s = blockIdx.x;
    if (s < nslab && wave < m) load_slab_row(g, G, m, s, wave, lane);
    for (int t = 0; s < nslab; s += gridDim.x, ++t) {
#pragma unroll
        for (int u = 0; u < 8; ++u) gv[u] = ld4(gn, s * SLAB + u * 256 + lane * 4, d, aligned);
        double acc[8][4];
#pragma unroll
        for (int u = 0; u < 8; ++u) acc[u][0] = acc[u][1] = acc[u][2] = acc[u][3] = 0.0;
        for (int i0 = wave; i0 < m; i0 += 4 * PASS21_RB) {
            double sv[PASS21_RB];
#pragma unroll
            for (int r = 0; r < PASS21_RB; ++r) {
                const int i = i0 + 4 * r;
                double dv = 0.0;
                if (i < m) {
                    const double cv = cl[i];
#pragma unroll
                    for (int u = 0; u < 8; ++u) {
                        acc[u][0] = fma(cv, (double)g[u].x, acc[u][0]);
                        acc[u][1] = fma(cv, (double)g[u].y, acc[u][1]);
                        acc[u][2] = fma(cv, (double)g[u].z, acc[u][2]);
                        acc[u][3] = fma(cv, (double)g[u].w, acc[u][3]);
                    }
                    if (i == knext) {
#pragma unroll
                        for (int u = 0; u < 8; ++u) dv = dot4d(gv[u], gv[u], dv);
                    } else {
#pragma unroll
                        for (int u = 0; u < 8; ++u) dv = dot4d(g[u], gv[u], dv);
                    }
                    if (i + 4 < m)
                        load_slab_row(g, G, m, s, i + 4, lane);
                    else if (s + gridDim.x < nslab)
                        load_slab_row(g, G, m, s + gridDim.x, wave, lane);
                }
                sv[r] = dv;
            }
            int idx;
            bool writer;
            const double tot = wave_reduce_many<PASS21_RB>(sv, lane, idx, writer);
            if (writer && i0 + 4 * idx < m) rs[i0 + 4 * idx] += tot;
        }
        double* rb = red + (t & 1) * 4 * SLAB;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            double* q = rb + wave * SLAB + u * 256 + lane * 4;
            *reinterpret_cast<double2*>(q) = make_double2(acc[u][0], acc[u][1]);
            *reinterpret_cast<double2*>(q + 2) = make_double2(acc[u][2], acc[u][3]);
        }
        lds_barrier();
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int col = wave * 512 + h * 256 + lane * 4;
            const int64_t j = s * SLAB + col;
            double sum[4];
#pragma unroll
            for (int k = 0; k < 4; ++k)
                sum[k] = rb[col + k] + rb[SLAB + col + k] + rb[2 * SLAB + col + k] + rb[3 * SLAB + col + k];
            // y = 0 - sum (not -sum: an exact zero sum stores +0, as in k_pass2_rows)
            float4 o;
            o.x = (float)(0.0 - sum[0]);
            o.y = (float)(0.0 - sum[1]);
            o.z = (float)(0.0 - sum[2]);
            o.w = (float)(0.0 - sum[3]);
            st4_stream(y, j, d, aligned, o);
        }
    }
    __syncthreads();
    double* out = part + (int64_t)blockIdx.x * m;
    for (int t = threadIdx.x; t < m; t += 256) out[t] = rs[t];
}

// The new gradient into row k of the window (padding past d stays zero).
__global__ __launch_bounds__(256) void k_write_row(float* __restrict__ G, int m, int64_t d, int64_t ncolpad,
                                                   int k, const float* __restrict__ g, int aligned) {
    const int64_t j = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
    if (j >= ncolpad) return;
    const float4 v = ld4(g, j, d, aligned);
    const int64_t slab = j / SLAB;
    *reinterpret_cast<float4*>(G + slab * (int64_t)m * SLAB + (int64_t)k * SLAB + (j - slab * SLAB)) = v;
}

template <int NV>
struct PassCfg {
    // Pass 1: U float4 per lane and row (the vector chunks stay in registers),
    // R rows per wave iteration, GRID work-groups. Measured on the 105 GB
    // window (m = 1024) over U in {1, 2, 4, 8}, R in {1, ..., 8} and grids of
    // 256 / 384 / 512: one or two vectors stream best from one work-group per
    // CU (7.4 TB/s against 6.95 at two per CU); wider fusions need two.
    // A later re-sweep of R at 8-10 vectors gave R = 4 for 9 and 10 vectors
    // (6.75 and 6.67 TB/s against 6.66 and 6.36 with R = 3) and kept 3 for 8.
    // Above 10 vectors the rows split into two groups of 256 work-groups.
    static constexpr int U = NV <= 4 ? 4 : 2;
    static constexpr int R = NV <= 2 ? 2 : NV <= 4 ? 1 : NV <= 7 ? 2 : NV == 8 ? 3 : NV <= 16 ? 4 : 3;
    static constexpr int GRID = NV <= 2 ? 256 : 512;
    // Pass 2 (the per-wave column chunk kernel): U2 float4 per lane (chunks of
    // 256 * U2 columns), RB2 rows of loads in flight per wave; measured over
    // U2 in {1, 2, 4} and RB2 in {2, ..., 16}.
    static constexpr int U2 = NV == 2 ? 4 : NV <= 5 ? 2 : 1;
    static constexpr int RB2 = NV == 1 ? 8 : NV == 2 ? 4 : NV <= 4 ? 2 : NV == 5 ? 4 : 8;
};

// Pass-1 rows per work-group: the fp64 row sums of a work-group stay within
// 80 KB of LDS (two work-groups per CU); larger m * NV splits the rows into
// groups, each re-reading the vector chunks (NV * 4 bytes per column per extra
// group, under 2% of the pass).
constexpr int64_t ROWSUM_LDS = 80 * 1024;
inline Pass1Grid pass1_grid(int m, int nv, int64_t nchunk, int target) {
    const int64_t bytes = (int64_t)m * nv * 8;
    const int ng = (int)((bytes + ROWSUM_LDS - 1) / ROWSUM_LDS);
    Pass1Grid pg;
    pg.mg = (m + ng - 1) / ng;
    pg.ng = (m + pg.mg - 1) / pg.mg;
    int64_t gx = target / pg.ng;
    if (gx > nchunk) gx = nchunk;
    if (gx < 1) gx = 1;
    pg.gx = (int)gx;
    return pg;
}

template <int NV>
hipError_t pass1_nv(const float* G, int m, int64_t d, int64_t nslab, const VecIn& vin, bool aligned,
                    double* part, Pass1Grid* grid_out, hipStream_t st) {
    constexpr int U = PassCfg<NV>::U, R = PassCfg<NV>::R;
    static_assert(PassCfg<NV>::GRID <= PASS1_MAX_GRID, "partials sized for PASS1_MAX_GRID work-groups");
    const int64_t nchunk = nslab * (SLAB / (256 * U));
    const Pass1Grid pg = pass1_grid(m, NV, nchunk, PassCfg<NV>::GRID);
    const size_t lds = (size_t)pg.mg * NV * sizeof(double);
    if (lds > 65536) {
        // fp64 row sums of a row group: just above 80 KB at most. Set on every
        // such launch: the attribute is per device, and the call is cheap next
        // to a pass over the window.
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_pass1<NV, U, R>),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL((k_pass1<NV, U, R>), dim3(pg.gx, pg.ng), dim3(256), lds, st, G, m, pg.mg, d, nchunk, vin,
                       aligned ? 1 : 0, part);
    *grid_out = pg;
    return hipGetLastError();
}

template <int NV>
hipError_t pass2_nv(const float* G, int m, int64_t d, int64_t nslab, const double* coef,
                    const VecOut& vout, bool aligned, hipStream_t st) {
    if constexpr (NV == 1) {
        if (m <= PASS2_ROWS_MAX_M) {
            const size_t lds = (size_t)(((m + 1) & ~1) + 8 * SLAB) * sizeof(double);
            hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_pass2_rows),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
            if (e != hipSuccess) return e;
            const int64_t grid = nslab < PASS2_ROWS_GRID ? nslab : PASS2_ROWS_GRID;
            hipLaunchKernelGGL(k_pass2_rows, dim3((unsigned)grid), dim3(256), lds, st, G, m, d, nslab, coef, vout,
                               aligned ? 1 : 0);
            return hipGetLastError();
        }
    }
    constexpr int U = PassCfg<NV>::U2, RB = PassCfg<NV>::RB2;
    const int64_t nwchunk = nslab * (SLAB / (256 * U));
    const int64_t grid = ceil_div(nwchunk, 4);
    const size_t lds = (size_t)m * CoefStride<NV>::P * sizeof(typename AccType<NV>::T);
    if (lds > 65536) {
        // set on every such launch (per device; cheap next to the pass)
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_pass2<NV, U, RB>),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL((k_pass2<NV, U, RB>), dim3((unsigned)grid), dim3(256), lds, st, G, m, d, nwchunk, coef, vout,
                       aligned ? 1 : 0);
    return hipGetLastError();
}


}  // namespace

hipError_t launch_fill_zero(float* p, int64_t n, hipStream_t st) {
    int64_t blocks = ceil_div(n, 256);
    if (blocks > 65536) blocks = 65536;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(k_fill_zero, dim3((unsigned)blocks), dim3(256), 0, st, p, n);
    return hipGetLastError();
}

hipError_t launch_set_rows(float* G, int m, int64_t d, int64_t nslab, int first, int count,
                           const float* rows, int64_t ld, hipStream_t st) {
    if (count <= 0) return hipSuccess;
    const int64_t ncolpad = nslab * SLAB;
    const bool aligned = ((uintptr_t)rows % 16 == 0) && (ld % 4 == 0);
    dim3 grid((unsigned)ceil_div(ncolpad / 4, 256), (unsigned)count);
    hipLaunchKernelGGL(k_set_rows, grid, dim3(256), 0, st, G, m, d, ncolpad, first, rows, ld,
                       aligned ? 1 : 0);
    return hipGetLastError();
}

hipError_t launch_get_rows(const float* G, int m, int64_t d, int first, int count, float* rows,
                           int64_t ld, hipStream_t st) {
    if (count <= 0) return hipSuccess;
    const bool aligned = ((uintptr_t)rows % 16 == 0) && (ld % 4 == 0);
    dim3 grid((unsigned)ceil_div(ceil_div(d, 4), 256), (unsigned)count);
    hipLaunchKernelGGL(k_get_rows, grid, dim3(256), 0, st, G, m, d, first, rows, ld, aligned ? 1 : 0);
    return hipGetLastError();
}

#define MFAC_NV_CASES(X) \
    X(1) X(2) X(3) X(4) X(5) X(6) X(7) X(8) X(9) X(10) X(11) X(12) X(13) X(14) X(15) X(16) X(17)

hipError_t launch_write_row(float* G, int m, int64_t d, int64_t nslab, int k, const float* g, hipStream_t st) {
    const int64_t ncolpad = nslab * SLAB;
    const bool aligned = ((uintptr_t)g % 16) == 0;
    hipLaunchKernelGGL(k_write_row, dim3((unsigned)ceil_div(ncolpad / 4, 256)), dim3(256), 0, st, G, m, d, ncolpad,
                       k, g, aligned ? 1 : 0);
    return hipGetLastError();
}

hipError_t launch_pass1(const float* G, int m, int64_t d, int64_t nslab, int nv, const VecIn& vin,
                        bool aligned, double* part, Pass1Grid* grid_out, hipStream_t st) {
    switch (nv) {
#define CASE(N) \
    case N: return pass1_nv<N>(G, m, d, nslab, vin, aligned, part, grid_out, st);
        MFAC_NV_CASES(CASE)
#undef CASE
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_pass2_next(const float* G, int m, int64_t d, int64_t nslab, const double* coef, float* y,
                             const float* gn, int knext, bool aligned, double* part, Pass1Grid* grid_out,
                             hipStream_t st) {
    if (m > PASS21_MAX_M) return hipErrorInvalidValue;
    const size_t lds = (size_t)(2 * ((m + 1) & ~1) + 8 * SLAB) * sizeof(double);
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_pass2_next),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e != hipSuccess) return e;
    const int64_t grid = nslab < PASS2_ROWS_GRID ? nslab : PASS2_ROWS_GRID;
    hipLaunchKernelGGL(k_pass2_next, dim3((unsigned)grid), dim3(256), lds, st, G, m, d, nslab, coef, y, gn, knext,
                       aligned ? 1 : 0, part);
    grid_out->gx = (int)grid;
    grid_out->ng = 1;
    grid_out->mg = m;
    return hipGetLastError();
}

hipError_t launch_reduce_partials(const double* part, const Pass1Grid& pg, int m, int nv, double* p,
                                  hipStream_t st) {
    const int mnv = m * nv;
    hipLaunchKernelGGL(k_reduce_partials, dim3((unsigned)ceil_div(mnv, 16)), dim3(256), 0, st, part, pg, nv,
                       mnv, p);
    return hipGetLastError();
}

hipError_t launch_pass2(const float* G, int m, int64_t d, int64_t nslab, int nv, const double* coef,
                        const VecOut& vout, bool aligned, hipStream_t st) {
    switch (nv) {
#define CASE(N) \
    case N: return pass2_nv<N>(G, m, d, nslab, coef, vout, aligned, st);
        MFAC_NV_CASES(CASE)
#undef CASE
        default: return hipErrorInvalidValue;
    }
}

}  // namespace mfac
