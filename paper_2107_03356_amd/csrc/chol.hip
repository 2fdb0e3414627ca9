// The m x m coefficient phase, in fp64.
//
// The paper's D (Section 3.2) is the upper LU factor, without pivoting, of
// K/lambda + m I minus m I (Appendix B); equivalently D and B come from the
// Cholesky factor R of A = K + m*lambda*I: A = lambda * Ru Ru^T with
// D = diag(Ru) Ru^T - m I and B = lambda^-1 (Ru diag(Ru)^-1)^-1. The
// coefficients of Theorem 1 are then c = lambda^-1 A^-1 G x. The library
// keeps the explicit inverse A^-1 (the paper's remark that a modified
// Cholesky kernel would beat its LU): factor.hip computes L and L^-1 with a
// recursive blocked algorithm whose diagonal nodes of 64 or 128 this file
// factors and inverts in LDS (k_factor_node); k_lauum forms A^-1 = L^-T L^-1; the
// O(m^2) slot replacement updates A^-1 in place between refactors; and the
// coefficient kernel applies it. A is padded to a multiple of 64 with an
// identity block so no kernel needs edge handling.
//
// Dense 64 x 64 x 64 tile products (k_lauum) run on fp64 MFMA
// (v_mfma_f64_16x16x4f64): 4 waves, each a 32 x 32 quadrant of 2 x 2 16x16
// tiles, operands from LDS. They are written as C[r][c] = sum_k a[r][k] *
// b[c][k]; a tile that enters as b[k][c] is transposed while it is staged.
#include "internal.h"
#include "tile_util.h"

namespace mfac {
namespace {

constexpr int P = 68;  // LDS pitch of a 64 x 64 fp64 tile

__device__ __forceinline__ void stage_tile_t(double (*S)[P], const double* __restrict__ src, int64_t ld) {
    for (int e = threadIdx.x; e < 64 * 64; e += blockDim.x) {
        const int r = e >> 6, c = e & 63;
        S[c][r] = src[(int64_t)r * ld + c];
    }
}

__device__ __forceinline__ void zero_acc(v4d (&acc)[2][2]) {
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y) acc[x][y] = v4d{0.0, 0.0, 0.0, 0.0};
}

// acc += a * b^T over k in [0, 64) for this wave's quadrant (256 threads).
__device__ __forceinline__ void mma_nt(const double (*a)[P], const double (*b)[P], v4d (&acc)[2][2]) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wr = wave >> 1, wc = wave & 1;
    const int rl = lane & 15, kl = lane >> 4;
#pragma unroll 4
    for (int kk = 0; kk < 16; ++kk) {
        double av[2], bv[2];
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            av[s] = a[wr * 32 + s * 16 + rl][kk * 4 + kl];
            bv[s] = b[wc * 32 + s * 16 + rl][kk * 4 + kl];
        }
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
            for (int y = 0; y < 2; ++y)
                acc[x][y] = __builtin_amdgcn_mfma_f64_16x16x4f64(av[x], bv[y], acc[x][y], 0, 0, 0);
    }
}

// Visit this thread's accumulator entries: f(row, col, value). In the fp64
// 16x16x4 MFMA result, lane l register r holds row (l/16) + 4r, column l%16.
template <typename F>
__device__ __forceinline__ void for_acc(v4d (&acc)[2][2], F f) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wr = wave >> 1, wc = wave & 1;
    const int rl = lane & 15, kl = lane >> 4;
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y)
#pragma unroll
            for (int r = 0; r < 4; ++r) f(wr * 32 + x * 16 + kl + 4 * r, wc * 32 + y * 16 + rl, acc[x][y][r]);
}

// ------------------------------------------------------------------ assemble
__global__ __launch_bounds__(256) void k_assemble(double* __restrict__ K, int m,
                                                  const double* __restrict__ p, int pstride, int k,
                                                  double mu, double* __restrict__ A, int mp,
                                                  int* __restrict__ err) {
    const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (e >= (int64_t)mp * mp) return;
    const int i = (int)(e / mp), j = (int)(e % mp);
    double v;
    if (i < m && j < m) {
        if (k >= 0 && i == k)
            v = p[(int64_t)j * pstride];
        else if (k >= 0 && j == k)
            v = p[(int64_t)i * pstride];
        else
            v = K[(int64_t)i * m + j];
        if (k >= 0 && i == k) {
            K[(int64_t)k * m + j] = v;
            K[(int64_t)j * m + k] = v;
            if (!isfinite(v)) atomicOr(err, 1);
        }
        if (i == j) v += mu;
    } else {
        v = (i == j) ? 1.0 : 0.0;
    }
    A[e] = v;
}

// ------------------------------------------------------------------ diagonal nodes
__device__ __forceinline__ double rsqrt_of(double x) { return rsqrt(x); }
__device__ __forceinline__ float rsqrt_of(float x) { return rsqrtf(x); }

// v of lane src (src the same in every lane)
__device__ __forceinline__ float lane_value(float v, int src) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), src));
}
__device__ __forceinline__ double lane_value(double v, int src) {
    const long long b = __double_as_longlong(v);
    const unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)b, src);
    const unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)(b >> 32), src);
    return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}

// Orders LDS traffic between the lanes of one wave: a wave's LDS operations
// complete in issue order, so this only has to keep the compiler from moving
// them across the point.
__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// 16x16x4 MFMA per element type: accumulator and the row of register r
template <typename R>
struct NodeMfma;
template <>
struct NodeMfma<double> {
    typedef v4d acc;
    static __device__ __forceinline__ acc mfma(double a, double b, acc c) {
        return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
    }
    static __device__ __forceinline__ int row(int lane, int r) { return mfma64_row(lane, r); }
};
template <>
struct NodeMfma<float> {
    typedef v4f acc;
    static __device__ __forceinline__ acc mfma(float a, float b, acc c) {
        return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
    }
    static __device__ __forceinline__ int row(int lane, int r) { return mfma32_row(lane, r); }
};

constexpr int NPX = 132;  // LDS pitch of the node (rows of 16-row MFMA reads on distinct banks)
constexpr int NSP = 20;   // LDS pitch of the 16-column product scratch

// Factor and invert the diagonal node [o, o+n) (n = 64 or 128) of every batch
// item in one launch: one work-group of four waves per item, the node's lower
// 64 x 64 tiles resident in LDS (fp64: 153 KB). Blocked in 16 x 16 tiles so
// that every loop is short and the code stays small:
//   Cholesky, 16-column panels left to right: wave 0 factors the panel's
//     diagonal block and inverts it in the same column sweep (a lane per row
//     of L and per column of the inverse D); the rows below are A D^T, and
//     the four waves apply the panel's rank-16 update to the lower tiles to
//     its right, both on MFMA;
//   inverse of the factor in place, block columns right to left:
//     Linv[below j][j] = -Linv[below j][below j] L[below j][j] D_j,
//     where the first factor is already the inverse (two MFMA products).
// Writes the node's lower tiles of Linv, zeros above the diagonal of its
// diagonal 64 x 64 tiles; A is only read. Only lower-triangle values of A
// enter the result. err |= 2 on a non-positive or non-finite pivot (which
// then continues as 1).
template <typename R>
__global__ __launch_bounds__(256) void k_factor_node(const R* __restrict__ A, R* __restrict__ Linv, int mp,
                                                     int64_t bstride, int o, int n, int* __restrict__ err) {
    __shared__ R X[128][NPX];
    __shared__ R S[112][NSP];
    __shared__ __align__(16) R colv[2][16];  // the current column of L (double-buffered)
    typedef NodeMfma<R> M;
    typedef typename M::acc acc_t;
    const R* Ab = A + (int64_t)blockIdx.x * bstride;
    R* Lb = Linv + (int64_t)blockIdx.x * bstride;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int rl = lane & 15, kl = lane >> 4;
    const int np = n >> 4;
    // the lower 64 x 64 tiles (00, 10, 11; 00 alone when n = 64): thread t
    // moves row t/4, columns 16 (t%4) .. +15 of each, all loads in flight
    // before the first LDS store
    constexpr int VE = 16 / sizeof(R);  // elements per 16-byte access
    typedef R vec_t __attribute__((ext_vector_type(VE)));
    const int lr = tid >> 2, lc = (tid & 3) * 16;
    const int ntile = n == 128 ? 3 : 1;
    {
        vec_t buf[3][16 / VE];
#pragma unroll
        for (int tl = 0; tl < 3; ++tl) {
            if (tl < ntile) {
                const int tr = tl == 0 ? 0 : 64, tc = tl == 2 ? 64 : 0;
                const vec_t* src = reinterpret_cast<const vec_t*>(Ab + (int64_t)(o + tr + lr) * mp + o + tc + lc);
#pragma unroll
                for (int v = 0; v < 16 / VE; ++v) buf[tl][v] = src[v];
            }
        }
#pragma unroll
        for (int tl = 0; tl < 3; ++tl) {
            if (tl < ntile) {
                const int tr = tl == 0 ? 0 : 64, tc = tl == 2 ? 64 : 0;
#pragma unroll
                for (int v = 0; v < 16 / VE; ++v) *reinterpret_cast<vec_t*>(&X[tr + lr][tc + lc + v * VE]) = buf[tl][v];
            }
        }
    }
    __syncthreads();

    int bad = 0;
    for (int p = 0; p < np; ++p) {
        const int j0 = p * 16;
        if (wave == 0) {
            // the 16 x 16 diagonal block: lane l < 16 keeps row l of it (r) and
            // column l of its inverse (x, by forward substitution folded into
            // the same column sweep); column k of L goes to every lane through
            // LDS. Lanes 16..63 and entries above the diagonal carry values
            // that nothing reads.
            R r[16], x[16];
#pragma unroll
            for (int c = 0; c < 16; ++c) {
                r[c] = lane < 16 ? X[j0 + lane][j0 + c] : R(0);
                x[c] = (c == lane) ? R(1) : R(0);
            }
#pragma unroll
            for (int k = 0; k < 16; ++k) {
                R pk = lane_value(r[k], k);
                if (!(pk > R(0)) || !isfinite(pk)) {
                    bad = 1;
                    pk = R(1);
                }
                const R rs = rsqrt_of(pk);
                r[k] = lane == k ? pk * rs : r[k] * rs;
                if (lane < 16) colv[k & 1][lane] = r[k];
                wave_sync();
                R lc[16];
#pragma unroll
                for (int c = 0; c < 16; ++c) lc[c] = colv[k & 1][c];
                // x_k = (e_l - sum_{i<k} L[k][i] x_i)_k / L[k][k], then the
                // rows below take their L[.][k] x_k terms
                x[k] = x[k] * rs;
#pragma unroll
                for (int c = k + 1; c < 16; ++c) {
                    r[c] -= r[k] * lc[c];
                    x[c] -= lc[c] * x[k];
                }
                wave_sync();
            }
            // the inverse block (zeros above its diagonal) over the block
            if (lane < 16) {
#pragma unroll
                for (int c = 0; c < 16; ++c) X[j0 + c][j0 + lane] = x[c];
            }
        }
        __syncthreads();
        const int nt = np - 1 - p;  // 16-row tiles below the diagonal block
        // panel rows below: L = A D^T (D the diagonal block's inverse), into S
        for (int t = wave; t < nt; t += 4) {
            acc_t acc = acc_t{0, 0, 0, 0};
            const int ra = j0 + 16 + 16 * t;
#pragma unroll
            for (int kk = 0; kk < 4; ++kk)
                acc = M::mfma(X[ra + rl][j0 + kk * 4 + kl], X[j0 + rl][j0 + kk * 4 + kl], acc);
#pragma unroll
            for (int rr = 0; rr < 4; ++rr) S[16 * t + M::row(lane, rr)][rl] = acc[rr];
        }
        __syncthreads();
        // lower 16 x 16 tiles (a, b), a >= b, of the trailing block -= P P^T,
        // and the panel rows back into X
        const int ntl = nt * (nt + 1) / 2;
        for (int q = wave; q < ntl; q += 4) {
            int a = 0;
            while ((a + 1) * (a + 2) / 2 <= q) ++a;
            const int b = q - a * (a + 1) / 2;
            const int ra = j0 + 16 + 16 * a, cb = j0 + 16 + 16 * b;
            acc_t acc;
#pragma unroll
            for (int rr = 0; rr < 4; ++rr) acc[rr] = X[ra + M::row(lane, rr)][cb + rl];
#pragma unroll
            for (int kk = 0; kk < 4; ++kk)
                acc = M::mfma(-S[16 * a + rl][kk * 4 + kl], S[16 * b + rl][kk * 4 + kl], acc);
#pragma unroll
            for (int rr = 0; rr < 4; ++rr) X[ra + M::row(lane, rr)][cb + rl] = acc[rr];
        }
        for (int e = tid; e < nt * 256; e += 256) X[j0 + 16 + (e >> 4)][j0 + (e & 15)] = S[e >> 4][e & 15];
        __syncthreads();
    }

    // block columns right to left
    for (int j = np - 2; j >= 0; --j) {
        const int nt = np - 1 - j, rb = 16 * (j + 1);
        for (int t = wave; t < nt; t += 4) {
            acc_t acc = acc_t{0, 0, 0, 0};
            for (int s = 0; s <= t; ++s)
#pragma unroll
                for (int kk = 0; kk < 4; ++kk)
                    acc = M::mfma(X[rb + 16 * t + rl][rb + 16 * s + kk * 4 + kl],
                                  X[rb + 16 * s + kk * 4 + kl][16 * j + rl], acc);
#pragma unroll
            for (int r = 0; r < 4; ++r) S[16 * t + M::row(lane, r)][rl] = acc[r];
        }
        __syncthreads();
        for (int t = wave; t < nt; t += 4) {
            acc_t acc = acc_t{0, 0, 0, 0};
#pragma unroll
            for (int kk = 0; kk < 4; ++kk)
                acc = M::mfma(-S[16 * t + rl][kk * 4 + kl], X[16 * j + kk * 4 + kl][16 * j + rl], acc);
#pragma unroll
            for (int r = 0; r < 4; ++r) X[rb + 16 * t + M::row(lane, r)][16 * j + rl] = acc[r];
        }
        __syncthreads();
    }

#pragma unroll
    for (int tl = 0; tl < 3; ++tl) {
        if (tl < ntile) {
            const int tr = tl == 0 ? 0 : 64, tc = tl == 2 ? 64 : 0;
            vec_t* dst = reinterpret_cast<vec_t*>(Lb + (int64_t)(o + tr + lr) * mp + o + tc + lc);
#pragma unroll
            for (int v = 0; v < 16 / VE; ++v) {
                vec_t w;
#pragma unroll
                for (int q = 0; q < VE; ++q) {
                    const int r = tr + lr, c = tc + lc + v * VE + q;
                    w[q] = (c <= r) ? X[r][c] : R(0);
                }
                dst[v] = w;
            }
        }
    }
    if (tid == 0 && bad) atomicOr(err, 2);
}

template <typename R>
__global__ __launch_bounds__(256) void k_zero_superdiag(R* __restrict__ Linv, int mp, int64_t bstride) {
    // zero the first superdiagonal of 64 x 64 tiles, (t, t+1); grid (T-1, nbatch)
    const int t = blockIdx.x;
    R* C = Linv + (int64_t)blockIdx.y * bstride + (int64_t)t * 64 * mp + (t + 1) * 64;
    for (int e = threadIdx.x; e < 4096; e += 256) C[(int64_t)(e >> 6) * mp + (e & 63)] = R(0);
}

// ------------------------------------------------------------------ explicit inverse
// Ainv = (A)^-1 = Linv^T Linv, tile (I, J) = sum_{K >= max(I,J)} Linv[K,I]^T Linv[K,J].
// grid (T*T, nbatch).
__global__ __launch_bounds__(256) void k_lauum(const double* __restrict__ Linv, double* __restrict__ Ainv, int mp,
                                               int64_t bstride) {
    __shared__ double Sa[64][P];
    __shared__ double Sb[64][P];
    const int T = mp / 64;
    const int I = blockIdx.x / T, J = blockIdx.x % T;
    const double* Lb = Linv + (int64_t)blockIdx.y * bstride;
    v4d acc[2][2];
    zero_acc(acc);
    for (int K = (I > J ? I : J); K < T; ++K) {
        stage_tile_t(Sa, Lb + (int64_t)K * 64 * mp + I * 64, mp);
        stage_tile_t(Sb, Lb + (int64_t)K * 64 * mp + J * 64, mp);
        __syncthreads();
        mma_nt(Sa, Sb, acc);
        __syncthreads();
    }
    double* C = Ainv + (int64_t)blockIdx.y * bstride + (int64_t)I * 64 * mp + J * 64;
    for_acc(acc, [&](int row, int col, double v) { C[(int64_t)row * mp + col] = v; });
}

__device__ __forceinline__ double wave_sum_d(double x) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
    return x;
}

// Slot k takes a new gradient whose Gram column is p (p[j*pstride], p_k = |g|^2).
// Writes row/column k of K, z = Ainv b (b = p off slot k, 0 at k) and
// v = row k of Ainv (the old inverse's column k). One wave per row of Ainv.
__global__ __launch_bounds__(256) void k_inv_gemv(double* __restrict__ K, int m, const double* __restrict__ p,
                                                  int pstride, int k, const double* __restrict__ Ainv, int mp,
                                                  double* __restrict__ z, double* __restrict__ v,
                                                  int* __restrict__ err) {
    const int lane = threadIdx.x & 63;
    const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (i >= mp) return;
    const double* row = Ainv + (int64_t)i * mp;
    double s = 0.0;
#pragma unroll 4
    for (int j = lane; j < m; j += 64)
        if (j != k) s += row[j] * p[(int64_t)j * pstride];
    s = wave_sum_d(s);
    if (lane == 0) z[i] = s;
    if (i == k) {
        for (int j = lane; j < mp; j += 64) v[j] = row[j];
    }
    if (i < m && lane == 0) {
        const double pi = p[(int64_t)i * pstride];
        K[(int64_t)k * m + i] = pi;
        K[(int64_t)i * m + k] = pi;
        if (!isfinite(pi)) atomicOr(err, 1);
    }
}

// Block-wide scalars of the slot update, computed identically by every
// work-group (fixed order): t = v_k, zk = z_k, s = c - b^T u with
// u = z - v zk / t and c = p_k + mu.
__device__ void inv_update_scalars(const double* __restrict__ p, int pstride, int k, int m, double mu,
                                   const double* __restrict__ z, const double* __restrict__ v, double* sh,
                                   double& t, double& zk, double& s) {
    t = v[k];
    zk = z[k];
    double acc = 0.0;
    for (int j = threadIdx.x; j < m; j += 256)
        if (j != k) acc += p[(int64_t)j * pstride] * (z[j] - v[j] * (zk / t));
    acc = wave_sum_d(acc);
    if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = acc;
    __syncthreads();
    const double bu = (sh[0] + sh[1]) + (sh[2] + sh[3]);
    s = p[(int64_t)k * pstride] + mu - bu;
}

// Ainv <- Ainv - v v^T / v_k + w w^T / s,  w = u - e_k, u = z - v z_k / v_k:
// the inverse with slot k removed (Schur complement of its old pivot) plus
// the new column inserted (new pivot s >= m*lambda). grid (T*T).
__global__ __launch_bounds__(256) void k_inv_update(const double* __restrict__ p, int pstride, int k, int m,
                                                    double mu, const double* __restrict__ z,
                                                    const double* __restrict__ v, double* __restrict__ Ainv,
                                                    int mp, int* __restrict__ err) {
    __shared__ double sh[4];
    double t, zk, s;
    inv_update_scalars(p, pstride, k, m, mu, z, v, sh, t, zk, s);
    if (blockIdx.x == 0 && threadIdx.x == 0 && (!(s > 0.0) || !isfinite(s) || !(t > 0.0))) atomicOr(err, 16);
    const int T = mp / 64;
    const int I = blockIdx.x / T, J = blockIdx.x % T;
    const double r = zk / t, it = 1.0 / t, is = 1.0 / s;
    for (int e = threadIdx.x; e < 4096; e += 256) {
        const int i = I * 64 + (e >> 6), j = J * 64 + (e & 63);
        const double wi = z[i] - v[i] * r - (i == k ? 1.0 : 0.0);
        const double wj = z[j] - v[j] * r - (j == k ? 1.0 : 0.0);
        double* a = Ainv + (int64_t)i * mp + j;
        *a = *a - v[i] * v[j] * it + wi * wj * is;
    }
}

// k_inv_update and k_coef_from_inv in one pass over Ainv: one wave per row i
// updates the row (the same expression per entry) and, for i < m, forms the
// row's coefficients from the new values (the same per-lane order and wave
// sums), so both results are those of the two kernels. The column k of the
// coefficient matrix (kc >= 0) is the new Ainv[i][kc]; the other columns take
// rhs[j*rstride + c]. grid ceil(mp / 4).
__global__ __launch_bounds__(256) void k_inv_update_coef(const double* __restrict__ p, int pstride, int k, int m,
                                                         double mu, const double* __restrict__ z,
                                                         const double* __restrict__ v, double* __restrict__ Ainv,
                                                         int mp, const double* __restrict__ rhs, int rstride, int nv,
                                                         int kc, double s0, double s1, double* __restrict__ coef,
                                                         int* __restrict__ err) {
    __shared__ double sh[4];
    double t, zk, s;
    inv_update_scalars(p, pstride, k, m, mu, z, v, sh, t, zk, s);
    if (blockIdx.x == 0 && threadIdx.x == 0 && (!(s > 0.0) || !isfinite(s) || !(t > 0.0))) atomicOr(err, 16);
    const int lane = threadIdx.x & 63;
    const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (i >= mp) return;
    const double r = zk / t, it = 1.0 / t, is = 1.0 / s;
    const double vi = v[i], wi = z[i] - v[i] * r - (i == k ? 1.0 : 0.0);
    double* row = Ainv + (int64_t)i * mp;
    double acc[MAXNV];
#pragma unroll
    for (int c = 0; c < MAXNV; ++c) acc[c] = 0.0;
    const int c0 = kc >= 0 ? 1 : 0;
    double akc = 0.0;
#pragma unroll 4
    for (int j = lane; j < mp; j += 64) {
        const double wj = z[j] - v[j] * r - (j == k ? 1.0 : 0.0);
        const double a = row[j] - vi * v[j] * it + wi * wj * is;
        row[j] = a;
        if (j == kc) akc = a;
        if (j < m) {
#pragma unroll
            for (int c = 0; c < MAXNV; ++c)
                if (c >= c0 && c < nv) acc[c] += a * rhs[(int64_t)j * rstride + c];
        }
    }
    if (i >= m) return;
    if (c0) akc = wave_sum_d(akc);  // the one lane holding it, exact
#pragma unroll
    for (int c = 0; c < MAXNV; ++c) {
        if (c < nv) {
            double x = (c < c0) ? akc : wave_sum_d(acc[c]);
            x *= (c == 0 ? s0 : s1);
            if (lane == 0) {
                if (!isfinite(x)) atomicOr(err, 4);
                coef[i * nv + c] = x;
            }
        }
    }
}

// coef[i*nv + c] = scale_c * (Ainv rhs_c)_i with rhs_0 = e_k when k >= 0,
// the other columns p[j*pstride + c]; one wave per row i, lanes along the row.
__global__ __launch_bounds__(256) void k_coef_from_inv(const double* __restrict__ Ainv, int mp, int m,
                                                       const double* __restrict__ p, int pstride, int nv, int k,
                                                       double s0, double s1, double* __restrict__ coef,
                                                       int* __restrict__ err) {
    const int lane = threadIdx.x & 63;
    const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (i >= m) return;
    const double* row = Ainv + (int64_t)i * mp;
    double acc[MAXNV];
#pragma unroll
    for (int c = 0; c < MAXNV; ++c) acc[c] = 0.0;
    const int c0 = k >= 0 ? 1 : 0;
#pragma unroll 4
    for (int j = lane; j < m; j += 64) {
        const double a = row[j];
#pragma unroll
        for (int c = 0; c < MAXNV; ++c)
            if (c >= c0 && c < nv) acc[c] += a * p[(int64_t)j * pstride + c];
    }
#pragma unroll
    for (int c = 0; c < MAXNV; ++c) {
        if (c < nv) {
            double x = (c < c0) ? row[k] : wave_sum_d(acc[c]);
            x *= (c == 0 ? s0 : s1);
            if (lane == 0) {
                if (!isfinite(x)) atomicOr(err, 4);
                coef[i * nv + c] = x;
            }
        }
    }
}

}  // namespace

hipError_t launch_assemble(double* K, int m, const double* p, int pstride, int k, double mu, double* A,
                           int mp, int* err, hipStream_t st) {
    const int64_t n = (int64_t)mp * mp;
    hipLaunchKernelGGL(k_assemble, dim3((unsigned)ceil_div(n, 256)), dim3(256), 0, st, K, m, p, pstride, k,
                       mu, A, mp, err);
    return hipGetLastError();
}

template <typename R>
hipError_t launch_factor_node(R* A, R* Linv, int mp, int nbatch, int64_t bstride, int o, int n, int* err,
                              hipStream_t st) {
    if (n != 64 && n != 128) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_factor_node<R>, dim3(nbatch), dim3(256), 0, st, A, Linv, mp, bstride, o, n, err);
    return hipGetLastError();
}
template hipError_t launch_factor_node<double>(double*, double*, int, int, int64_t, int, int, int*, hipStream_t);
template hipError_t launch_factor_node<float>(float*, float*, int, int, int64_t, int, int, int*, hipStream_t);

template <typename R>
hipError_t launch_zero_superdiag(R* M, int mp, int nbatch, int64_t bstride, hipStream_t st) {
    const int T = mp / 64;
    if (T < 2) return hipSuccess;
    hipLaunchKernelGGL(k_zero_superdiag<R>, dim3(T - 1, nbatch), dim3(256), 0, st, M, mp, bstride);
    return hipGetLastError();
}
template hipError_t launch_zero_superdiag<double>(double*, int, int, int64_t, hipStream_t);
template hipError_t launch_zero_superdiag<float>(float*, int, int, int64_t, hipStream_t);

hipError_t launch_lauum(const double* Linv, double* Ainv, int mp, int nbatch, int64_t bstride, hipStream_t st) {
    const int T = mp / 64;
    hipLaunchKernelGGL(k_lauum, dim3(T * T, nbatch), dim3(256), 0, st, Linv, Ainv, mp, bstride);
    return hipGetLastError();
}

hipError_t launch_inv_replace(double* K, int m, const double* p, int pstride, int k, double mu, double* Ainv,
                              int mp, double* z, double* v, int* err, hipStream_t st) {
    hipLaunchKernelGGL(k_inv_gemv, dim3((unsigned)ceil_div(mp, 4)), dim3(256), 0, st, K, m, p, pstride, k, Ainv, mp,
                       z, v, err);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int T = mp / 64;
    hipLaunchKernelGGL(k_inv_update, dim3(T * T), dim3(256), 0, st, p, pstride, k, m, mu, z, v, Ainv, mp, err);
    return hipGetLastError();
}

hipError_t launch_inv_replace_coef(double* K, int m, const double* p, int pstride, int k, double mu, double* Ainv,
                                  int mp, double* z, double* v, const double* rhs, int rstride, int nv, int kc,
                                  double s0, double s1, double* coef, int* err, hipStream_t st) {
    hipLaunchKernelGGL(k_inv_gemv, dim3((unsigned)ceil_div(mp, 4)), dim3(256), 0, st, K, m, p, pstride, k, Ainv, mp,
                       z, v, err);
    hipLaunchKernelGGL(k_inv_update_coef, dim3((unsigned)ceil_div(mp, 4)), dim3(256), 0, st, p, pstride, k, m, mu, z,
                       v, Ainv, mp, rhs, rstride, nv, kc, s0, s1, coef, err);
    return hipGetLastError();
}

hipError_t launch_coef_from_inv(const double* Ainv, int mp, int m, const double* p, int pstride, int nv, int k,
                                double s0, double s1, double* coef, int* err, hipStream_t st) {
    hipLaunchKernelGGL(k_coef_from_inv, dim3((unsigned)ceil_div(m, 4)), dim3(256), 0, st, Ainv, mp, m, p, pstride, nv,
                       k, s0, s1, coef, err);
    return hipGetLastError();
}

}  // namespace mfac
