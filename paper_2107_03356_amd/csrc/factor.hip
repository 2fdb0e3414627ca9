// Recursive blocked Cholesky factor and triangular inverse of a batch of
// padded SPD matrices A = G G^T + m*lambda*I (the coefficient matrices of
// both the dynamic and the static path): L L^T = A, and L^-1.
//
// A node of size n splits at h (a multiple of 64):
//   [A11  .  ]   L11 L11^T = A11                      (recursion)
//   [A21 A22 ]   L21 = A21 L11^-T                      (GEMM, L11^-T upper)
//                A22 <- A22 - L21 L21^T                (GEMM, lower tiles)
//                L22 L22^T = A22                      (recursion)
//                L^-1 21 = -L22^-1 (L21 L11^-1)        (two GEMMs, triangular)
// Nodes of 64 or 128 are factored and inverted whole in one launch
// (k_factor_node, in LDS). L itself is not kept: L21 lives in the (unused)
// upper block A12 while the node needs it,
// and L21 L11^-1 goes into A21, whose input values are consumed by then.
// Every GEMM is batched over the matrices and skips the K-range its
// triangular operand makes zero, so the flops are m^3/3 for the factor and
// m^3/3 for the inverse, nearly all of it in large MFMA tiles.
#include "internal.h"
#include "tile_util.h"

namespace mfac {

// defined in chol.hip
template <typename T>
hipError_t launch_zero_superdiag(T* M, int mp, int nbatch, int64_t bstride, hipStream_t st);
template <typename T>
hipError_t launch_factor_node(T* A, T* Linv, int mp, int nbatch, int64_t bstride, int o, int n, int* err,
                              hipStream_t st);

namespace {

constexpr int TILE = 128;  // the large GEMM tile (k_bgemm's BT; small products take 64)

// Per element type: the MFMA (16x16x4: fp64, or fp32 on twice the rate), its
// accumulator, the row of an accumulator register, the k-chunk depth (16 for
// both: 32-deep fp32 chunks measured slower) and the LDS pitches: [row][k] chunks (the 16-row x 4-k read of one MFMA operand
// on distinct banks) and [k][n] chunks (rows k .. k+3 on disjoint banks).
template <typename T>
struct Mf;
template <>
struct Mf<double> {
    typedef v4d acc;
    typedef double2 pair;
    static constexpr int BK = 16;
    static constexpr int PA = BK + 2;
    static __device__ __forceinline__ acc mfma(double a, double b, acc c) {
        return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
    }
    static __device__ __forceinline__ int row(int lane, int r) { return mfma64_row(lane, r); }
};
template <>
struct Mf<float> {
    typedef v4f acc;
    typedef float2 pair;
    static constexpr int BK = 16;
    static constexpr int PA = BK + 4;
    static __device__ __forceinline__ acc mfma(float a, float b, acc c) {
        return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
    }
    static __device__ __forceinline__ int row(int lane, int r) { return mfma32_row(lane, r); }
};

enum : int {
    KHI_ROW = 1,   // A lower triangular: k < (I+1)*BT for output row tile I
    KHI_COL = 2,   // op(B) upper triangular: k < (J+1)*BT for output column tile J
    KLO_COL = 4,   // op(B) lower triangular: k >= J*BT
    LOWER_ONLY = 8 // only output tiles with I >= J
};

template <typename T>
struct GemmArgs {
    const T* A;
    const T* B;
    T* C;
    int ld;
    int64_t bstride;
    int a0r, a0c;  // stored A origin (row, col)
    int b0r, b0c;  // stored B origin
    int cm0, cn0;  // C origin
    int M, N, K;
    double alpha, beta;
    int flags;
    int tiles_m, tiles_n;
    int mode;   // task layout, see task_tiles
    int ntask;  // tasks per batch item
    // split K: nsplit > 1 gives each task nsplit work-groups, work-group s
    // summing segment s of each tile's K range into part (unscaled, one
    // BT x BT tile per segment, batch item and tile); k_bgemm_reduce then
    // forms C from the segments
    int nsplit, nbatch;
    T* part;
};

enum : int {
    TASK_PLAIN = 0,      // one tile per task
    TASK_LOWER = 1,      // lower-triangle tiles only (I >= J), compact
    TASK_PAIR_ROWS = 2,  // tiles (i, J) and (T-1-i, J): equal total K range under KHI_ROW
    TASK_PAIR_COLS = 3   // tiles (I, j) and (I, T-1-j): equal total K range under KLO_COL / KHI_COL
};

// Output tiles of one task (I1 < 0: a single tile).
template <typename T>
__device__ __forceinline__ void task_tiles(const GemmArgs<T>& g, int t, int& I0, int& J0, int& I1, int& J1) {
    I1 = J1 = -1;
    if (g.mode == TASK_LOWER) {
        int i = (int)((sqrtf(8.0f * (float)t + 1.0f) - 1.0f) * 0.5f);
        while ((i + 1) * (i + 2) / 2 <= t) ++i;
        while (i * (i + 1) / 2 > t) --i;
        I0 = i;
        J0 = t - i * (i + 1) / 2;
    } else if (g.mode == TASK_PAIR_ROWS) {
        const int i = t / g.tiles_n;
        J0 = J1 = t - i * g.tiles_n;
        I0 = i;
        if (g.tiles_m - 1 - i != i) I1 = g.tiles_m - 1 - i;
        else J1 = -1;
    } else if (g.mode == TASK_PAIR_COLS) {
        const int half = (g.tiles_n + 1) / 2;
        const int j = t % half;
        I0 = I1 = t / half;
        J0 = j;
        if (g.tiles_n - 1 - j != j) J1 = g.tiles_n - 1 - j;
        else I1 = -1;
    } else {
        I0 = t / g.tiles_n;
        J0 = t - I0 * g.tiles_n;
    }
}

// C = alpha * op(A) op(B) + beta * C on sub-matrices of every batch item:
//   op(A)[m][k] = TA ? A[a0r+k][a0c+m] : A[a0r+m][a0c+k]
//   op(B)[k][n] = TB ? B[b0r+n][b0c+k] : B[b0r+k][b0c+n]
// One work-group per task of one or two BT x BT output tiles (a long and a
// short tile of a triangular product together, so tasks take equal time;
// lower-triangle products launch only their lower tiles), 16-deep k-chunks
// through double-buffered LDS with the next chunk's loads in flight. BT / 16
// waves per work-group, each owning 32 x BT/2 of a tile as 2 x BT/32 MFMA
// tiles: BT = 128 (eight waves, two work-groups per CU) or 64 (four waves,
// four per CU). Rows/columns past M/N (a half tile when M or N is an odd
// multiple of 64) load clamped, in-bounds data and are never stored. The elements C
// writes are disjoint from the ones A and B read (they may share a buffer).
template <typename T, bool TA, bool TB, int BT>
__global__ __launch_bounds__(4 * BT, 4) void k_bgemm(GemmArgs<T> g) {
    using M = Mf<T>;
    using T2 = typename M::pair;
    constexpr int NT = 4 * BT;       // threads: BT / 16 waves of 32 x BT/2
    constexpr int HW = BT / 2;       // a wave's column extent
    constexpr int NY = BT / 32;      // its 16-column MFMA tiles
    constexpr int PA = M::PA, PBN = BT + 16, BK = M::BK;
    constexpr int NP = BT * BK / (NT * 2);  // operand pairs per thread and chunk
    // [m][k] chunks for a non-transposed A / transposed B, [k][m] otherwise
    __shared__ T As[2][TA ? BK : BT][TA ? PBN : PA];
    __shared__ T Bs[2][TB ? BT : BK][TB ? PA : PBN];
    const int lid0 = xcd_remap(blockIdx.x, gridDim.x);
    const int seg = lid0 % g.nsplit;
    const int lid = lid0 / g.nsplit;
    const int bt = lid / g.ntask;
    int I0, J0, I1, J1;
    task_tiles(g, lid - bt * g.ntask, I0, J0, I1, J1);
    const T* __restrict__ A = g.A + (int64_t)bt * g.bstride;
    const T* __restrict__ B = g.B + (int64_t)bt * g.bstride;
    T* __restrict__ C = g.C + (int64_t)bt * g.bstride;
    const int ld = g.ld;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wr = wave >> 1, wc = wave & 1;  // rows wr*32, columns wc*HW
    const int rl = lane & 15, kl = lane >> 4;
    auto tile = [&](int I, int J) {
        int klo = 0, khi = g.K;
        if (g.flags & KHI_ROW) khi = min(khi, (I + 1) * BT);
        if (g.flags & KHI_COL) khi = min(khi, (J + 1) * BT);
        if (g.flags & KLO_COL) klo = J * BT;
        if (g.nsplit > 1) {
            // this work-group's segment of the tile's K range (whole chunks; may be empty)
            const int kc = ((khi - klo + g.nsplit - 1) / g.nsplit + BK - 1) / BK * BK;
            const int a = min(khi, klo + seg * kc), b = min(khi, a + kc);
            klo = a;
            khi = b;
        }
        const int mrow0 = I * BT, ncol0 = J * BT;

        // staging of BT x BK elements per operand and chunk, NP pairs per
        // thread, kept in registers:
        //   [row][k] layout: row tid/4, k (tid%4)*(BK/4) .. +BK/4-1 (row pieces)
        //   [k][row] layout: k tid/HW + 8q, row 2*(tid%HW) .. +1 (HW threads per k)
        const int sr = tid >> 2, sk = (tid & 3) * (BK / 4);
        const int tk = tid / HW, tn = (tid % HW) * 2;
        // clamped source rows / columns (M, N are even, so a clamped pair stays
        // inside the operand)
        const int am = min(mrow0 + (TA ? tn : sr), g.M - (TA ? 2 : 1));
        const int bn = min(ncol0 + (TB ? sr : tn), g.N - (TB ? 1 : 2));
        const T* __restrict__ ap =
            TA ? A + (int64_t)g.a0r * ld + g.a0c + am : A + (int64_t)(g.a0r + am) * ld + g.a0c + sk;
        const T* __restrict__ bp =
            TB ? B + (int64_t)(g.b0r + bn) * ld + g.b0c + sk : B + (int64_t)g.b0r * ld + g.b0c + bn;
        T2 pa[NP], pb[NP];
        auto load_chunk = [&](int k0) {
#pragma unroll
            for (int q = 0; q < NP; ++q) {
                pa[q] = TA ? *reinterpret_cast<const T2*>(ap + (int64_t)(k0 + tk + 8 * q) * ld)
                           : *reinterpret_cast<const T2*>(ap + k0 + 2 * q);
                pb[q] = TB ? *reinterpret_cast<const T2*>(bp + k0 + 2 * q)
                           : *reinterpret_cast<const T2*>(bp + (int64_t)(k0 + tk + 8 * q) * ld);
            }
        };
        auto put = [](T* dst, T2 v) {
            dst[0] = v.x;
            dst[1] = v.y;
        };
        auto store_chunk = [&](int buf) {
#pragma unroll
            for (int q = 0; q < NP; ++q) {
                if constexpr (TA)
                    put(&As[buf][tk + 8 * q][tn], pa[q]);
                else
                    put(&As[buf][sr][sk + 2 * q], pa[q]);
                if constexpr (TB)
                    put(&Bs[buf][sr][sk + 2 * q], pb[q]);
                else
                    put(&Bs[buf][tk + 8 * q][tn], pb[q]);
            }
        };

        // C tile coordinates of accumulator (x, y, r): the MFMA result's row
        // of register r of this lane, column lane % 16
        auto crow = [&](int x, int r) { return mrow0 + wr * 32 + x * 16 + M::row(lane, r); };
        auto ccol = [&](int y) { return ncol0 + wc * HW + y * 16 + rl; };
        const int nchunk = (khi - klo) / BK;
        // This wave's own K range: a triangular operand is zero outside it, so
        // the wave skips the MFMAs of chunks that lie wholly outside (the
        // trimmed K range above is per tile; this is per 32 rows / HW
        // columns). A wave whose rows or columns all lie past M / N, or that
        // sits above the diagonal of a diagonal tile of a lower-triangle
        // product, computes and stores nothing.
        int wkhi = khi, wklo = klo;
        if (g.flags & KHI_ROW) wkhi = min(wkhi, mrow0 + wr * 32 + 32);
        if (g.flags & KLO_COL) wklo = max(wklo, ncol0 + wc * HW);
        const bool idle = mrow0 + wr * 32 >= g.M || ncol0 + wc * HW >= g.N ||
                          ((g.flags & LOWER_ONLY) && I == J && wr * 32 + 31 < wc * HW);
        if (nchunk > 0) load_chunk(klo);
        // beta C enters as the accumulator's start value (scaled by 1/alpha), so
        // its loads issue together with the first chunk's
        // (the test is uniform and outside the loops, so all 32 loads issue
        // before the first wait)
        typename M::acc acc[2][NY];
        const T cs = (T)(g.beta / g.alpha);
        if (g.beta != 0.0 && !idle && g.nsplit == 1) {
    #pragma unroll
            for (int x = 0; x < 2; ++x)
    #pragma unroll
                for (int y = 0; y < NY; ++y)
    #pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int row = min(crow(x, r), g.M - 1), col = min(ccol(y), g.N - 1);
                        acc[x][y][r] = C[(int64_t)(g.cm0 + row) * ld + g.cn0 + col];
                    }
    #pragma unroll
            for (int x = 0; x < 2; ++x)
    #pragma unroll
                for (int y = 0; y < NY; ++y) acc[x][y] *= cs;
        } else {
    #pragma unroll
            for (int x = 0; x < 2; ++x)
    #pragma unroll
                for (int y = 0; y < NY; ++y) acc[x][y] = typename M::acc{0, 0, 0, 0};
        }
        if (nchunk > 0) {
            store_chunk(0);
            __syncthreads();
        }
        for (int c = 0; c < nchunk; ++c) {
            const int buf = c & 1;
            if (c + 1 < nchunk) load_chunk(klo + (c + 1) * BK);
            const int k0 = klo + c * BK;
            if (!idle && k0 + BK > wklo && k0 < wkhi) {
    #pragma unroll
            for (int kk = 0; kk < BK / 4; ++kk) {
                T av[2], bv[NY];
    #pragma unroll
                for (int x = 0; x < 2; ++x)
                    av[x] = TA ? As[buf][kk * 4 + kl][wr * 32 + x * 16 + rl] : As[buf][wr * 32 + x * 16 + rl][kk * 4 + kl];
    #pragma unroll
                for (int y = 0; y < NY; ++y)
                    bv[y] = TB ? Bs[buf][wc * HW + y * 16 + rl][kk * 4 + kl] : Bs[buf][kk * 4 + kl][wc * HW + y * 16 + rl];
    #pragma unroll
                for (int x = 0; x < 2; ++x)
    #pragma unroll
                    for (int y = 0; y < NY; ++y)
                        acc[x][y] = M::mfma(av[x], bv[y], acc[x][y]);
            }
            }
            if (c + 1 < nchunk) store_chunk(buf ^ 1);
            __syncthreads();
        }
        if (idle) return;
        if (g.nsplit > 1) {
            T* P = g.part + ((((int64_t)seg * g.nbatch + bt) * g.tiles_m + I) * g.tiles_n + J) * (BT * BT);
    #pragma unroll
            for (int x = 0; x < 2; ++x)
    #pragma unroll
                for (int y = 0; y < NY; ++y)
    #pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int row = crow(x, r), col = ccol(y);
                        if (row < g.M && col < g.N) P[(row - mrow0) * BT + (col - ncol0)] = acc[x][y][r];
                    }
            return;
        }
    #pragma unroll
        for (int x = 0; x < 2; ++x)
    #pragma unroll
            for (int y = 0; y < NY; ++y)
    #pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int row = crow(x, r), col = ccol(y);
                    if (row < g.M && col < g.N) C[(int64_t)(g.cm0 + row) * ld + g.cn0 + col] = (T)g.alpha * acc[x][y][r];
                }
    };
    tile(I0, J0);
    if (I1 >= 0) {
        __syncthreads();
        tile(I1, J1);
    }
}

// C = alpha * (sum of the K segments, in segment order) + beta * C over the
// elements k_bgemm would write (inside M x N, not in the idle upper pieces of
// a lower-triangle product's diagonal tiles). One work-group per 1024-element
// chunk of each task's tiles, four adjacent columns a thread, every segment
// loaded before the sum so that the loads overlap.
template <typename T, int BT>
__global__ __launch_bounds__(256) void k_bgemm_reduce(GemmArgs<T> g) {
    typedef T v4 __attribute__((ext_vector_type(4)));
    constexpr int CH = BT * BT / 1024;
    const int ch = blockIdx.x % CH, q = (blockIdx.x / CH) & 1, lid = blockIdx.x / (2 * CH);
    const int bt = lid / g.ntask;
    int I0, J0, I1, J1;
    task_tiles(g, lid - bt * g.ntask, I0, J0, I1, J1);
    const int I = q == 0 ? I0 : I1, J = q == 0 ? J0 : J1;
    if (I < 0) return;
    const int e = ch * 1024 + threadIdx.x * 4;
    const int r = e / BT, c = e - r * BT;
    const int row = I * BT + r, col = J * BT + c;
    if (row >= g.M || col >= g.N) return;
    if ((g.flags & LOWER_ONLY) && I == J && (r / 32) * 32 + 31 < (c / (BT / 2)) * (BT / 2)) return;
    const int64_t sstride = (int64_t)g.nbatch * g.tiles_m * g.tiles_n * (BT * BT);
    const T* P = g.part + (((int64_t)bt * g.tiles_m + I) * g.tiles_n + J) * (BT * BT) + e;
    v4 s[8];
#pragma unroll
    for (int sg = 0; sg < 8; ++sg)
        if (sg < g.nsplit) s[sg] = *reinterpret_cast<const v4*>(P + sg * sstride);
    v4 v = s[0];
#pragma unroll
    for (int sg = 1; sg < 8; ++sg)
        if (sg < g.nsplit) v += s[sg];
    T* dst = g.C + (int64_t)bt * g.bstride + (int64_t)(g.cm0 + row) * g.ld + g.cn0 + col;
#pragma unroll
    for (int k = 0; k < 4; ++k)
        if (col + k < g.N) dst[k] = g.beta != 0.0 ? (T)g.alpha * v[k] + (T)g.beta * dst[k] : (T)g.alpha * v[k];
}

template <typename T, int BT>
void launch_bgemm(bool ta, bool tb, int64_t grid, const GemmArgs<T>& g, hipStream_t st) {
    if (!ta && !tb) hipLaunchKernelGGL((k_bgemm<T, false, false, BT>), dim3((unsigned)grid), dim3(4 * BT), 0, st, g);
    if (!ta && tb) hipLaunchKernelGGL((k_bgemm<T, false, true, BT>), dim3((unsigned)grid), dim3(4 * BT), 0, st, g);
    if (ta && !tb) hipLaunchKernelGGL((k_bgemm<T, true, false, BT>), dim3((unsigned)grid), dim3(4 * BT), 0, st, g);
    if (ta && tb) hipLaunchKernelGGL((k_bgemm<T, true, true, BT>), dim3((unsigned)grid), dim3(4 * BT), 0, st, g);
}

template <typename T>
hipError_t gemm(bool ta, bool tb, const T* A, int a0r, int a0c, const T* B, int b0r, int b0c, T* C, int cm0, int cn0,
                int M, int N, int K, double alpha, double beta, int flags, int mp, int nbatch, int64_t bstride,
                T* part, int64_t part_elems, hipStream_t st) {
    GemmArgs<T> g;
    g.A = A;
    g.B = B;
    g.C = C;
    g.ld = mp;
    g.bstride = bstride;
    g.a0r = a0r;
    g.a0c = a0c;
    g.b0r = b0r;
    g.b0c = b0c;
    g.cm0 = cm0;
    g.cn0 = cn0;
    g.M = M;
    g.N = N;
    g.K = K;
    g.alpha = alpha;
    g.beta = beta;
    g.flags = flags;
    // 64 x 64 tiles (four waves, four work-groups per CU) for products of at
    // most 256 x 256, the recursion's short levels, where 128 x 128 tiles
    // leave one or four tiles per matrix: 7-8% off the 256 x 256 level in
    // fp64 and off a single-matrix factor; no change at 128 x 128
    const int bt = (M <= 256 && N <= 256) ? 64 : 128;
    g.tiles_m = (int)ceil_div(M, bt);
    g.tiles_n = (int)ceil_div(N, bt);
    if (flags & LOWER_ONLY) {
        g.mode = TASK_LOWER;  // square: tiles_m == tiles_n
        g.ntask = g.tiles_m * (g.tiles_m + 1) / 2;
    } else if (flags & KHI_ROW) {
        g.mode = TASK_PAIR_ROWS;
        g.ntask = (g.tiles_m + 1) / 2 * g.tiles_n;
    } else if (flags & (KLO_COL | KHI_COL)) {
        g.mode = TASK_PAIR_COLS;
        g.ntask = g.tiles_m * ((g.tiles_n + 1) / 2);
    } else {
        g.mode = TASK_PLAIN;
        g.ntask = g.tiles_m * g.tiles_n;
    }
    // Few tasks (one matrix, or a handful) leave most CUs idle and make each
    // work-group walk its whole K range chunk after chunk: split K over up to
    // 8 work-groups per task, as far as part holds the segments.
    const int64_t tasks = (int64_t)g.ntask * nbatch;
    g.nsplit = 1;
    g.nbatch = nbatch;
    g.part = part;
    if (part && tasks < 256 && K >= 4 * Mf<T>::BK) {
        int ns = (int)(256 / tasks < 8 ? 256 / tasks : 8);
        if (ns > K / (2 * Mf<T>::BK)) ns = K / (2 * Mf<T>::BK);
        while (ns > 1 && (int64_t)ns * nbatch * g.tiles_m * g.tiles_n * (bt * bt) > part_elems) --ns;
        g.nsplit = ns < 1 ? 1 : ns;
    }
    const int64_t grid = tasks * g.nsplit;
    if (bt == 64)
        launch_bgemm<T, 64>(ta, tb, grid, g, st);
    else
        launch_bgemm<T, 128>(ta, tb, grid, g, st);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || g.nsplit == 1) return e;
    if (bt == 64)
        hipLaunchKernelGGL((k_bgemm_reduce<T, 64>), dim3((unsigned)(tasks * 2 * (64 * 64 / 1024))), dim3(256), 0, st, g);
    else
        hipLaunchKernelGGL((k_bgemm_reduce<T, 128>), dim3((unsigned)(tasks * 2 * (128 * 128 / 1024))), dim3(256), 0,
                           st, g);
    return hipGetLastError();
}

// Factor and invert the diagonal block [o, o+n) of every batch item (n a
// multiple of 64). U = L21^T (h x n2) is kept in the upper block A12.
template <typename T>
hipError_t factor_node(T* A, T* Linv, int o, int n, int mp, int nbatch, int64_t bstride, int* err, T* part,
                       int64_t part_elems, hipStream_t st) {
    if (n <= 128) return launch_factor_node(A, Linv, mp, nbatch, bstride, o, n, err, st);
    const int h = (n / 128) * 64;  // split at a multiple of 64; n2 >= h
    const int n2 = n - h;
    const int p = o + h;
    hipError_t e = factor_node(A, Linv, o, h, mp, nbatch, bstride, err, part, part_elems, st);
    if (e != hipSuccess) return e;
    // U = Linv11 A21^T (h x n2) -> A12; Linv11 lower: k < (I+1) BT
    e = gemm(false, true, Linv, o, o, A, p, o, A, o, p, h, n2, h, 1.0, 0.0, KHI_ROW, mp, nbatch, bstride, part,
             part_elems, st);
    if (e != hipSuccess) return e;
    // A22 -= U^T U (lower tiles)
    e = gemm(true, false, A, o, p, A, o, p, A, p, p, n2, n2, h, -1.0, 1.0, LOWER_ONLY, mp, nbatch, bstride, part,
             part_elems, st);
    if (e != hipSuccess) return e;
    e = factor_node(A, Linv, p, n2, mp, nbatch, bstride, err, part, part_elems, st);
    if (e != hipSuccess) return e;
    // T = U^T Linv11 (n2 x h) -> A21; Linv11 lower: op(B)[k][j] = 0 for k < j
    e = gemm(true, false, A, o, p, Linv, o, o, A, p, o, n2, h, h, 1.0, 0.0, KLO_COL, mp, nbatch, bstride, part,
             part_elems, st);
    if (e != hipSuccess) return e;
    // Linv21 = -Linv22 T; Linv22 lower
    return gemm(false, false, Linv, p, p, A, p, o, Linv, p, o, n2, h, n2, -1.0, 0.0, KHI_ROW, mp, nbatch, bstride,
                part, part_elems, st);
}

}  // namespace

template <typename T>
hipError_t factor_invert(T* A, T* Linv, int mp, int nbatch, int64_t bstride, int* err, T* part, int64_t part_elems,
                         hipStream_t st) {
    // The trimmed K ranges read Linv only in the lower triangle and in the
    // first superdiagonal of 64 x 64 tiles (upper halves of 128-wide diagonal
    // blocks at 64-aligned origins); the leaves write zeros above their own
    // diagonals, so only that superdiagonal needs clearing.
    hipError_t e = launch_zero_superdiag(Linv, mp, nbatch, bstride, st);
    if (e != hipSuccess) return e;
    return factor_node(A, Linv, 0, mp, mp, nbatch, bstride, err, part, part_elems, st);
}

int64_t splitk_part_doubles(int mp) {
    if (mp <= 128) return 0;  // a single node: no GEMMs
    // segments x tiles <= 8 x (all 128 x 128 tiles of the largest product) and
    // <= 512 tiles (split only below 256 tasks, at most two tiles a task); 64 x
    // 64 tiles cover the same area, and 512 of them a quarter of it
    const int64_t t = ceil_div(mp, TILE) * ceil_div(mp, TILE);
    const int64_t tiles = 8 * t < 512 ? 8 * t : 512;
    return tiles * (TILE * TILE);
}

hipError_t launch_factor_invert(double* A, double* Linv, int mp, int nbatch, int64_t bstride, int* err,
                                hipStream_t st, double* part, int64_t part_elems) {
    return factor_invert<double>(A, Linv, mp, nbatch, bstride, err, part, part_elems, st);
}

hipError_t launch_factor_invert32(float* A, float* Linv, int mp, int nbatch, int64_t bstride, int* err,
                                  hipStream_t st) {
    return factor_invert<float>(A, Linv, mp, nbatch, bstride, err, nullptr, 0, st);
}

}  // namespace mfac
