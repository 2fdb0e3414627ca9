// The m x m coefficient phase, in fp64.
//
// The paper's D (Section 3.2) is the upper LU factor, without pivoting, of
// K/lambda + m I minus m I (Appendix B); equivalently D and B come from the
// Cholesky factor R of A = K + m*lambda*I: A = lambda * Ru Ru^T with
// D = diag(Ru) Ru^T - m I and B = lambda^-1 (Ru diag(Ru)^-1)^-1. The
// coefficients of Theorem 1 are then c = lambda^-1 A^-1 G x. The library
// keeps the explicit inverse A^-1 (the paper's remark that a modified
// Cholesky kernel would beat its LU): factor.hip computes L and L^-1 with a
// recursive blocked algorithm whose 64 x 64 leaves this file factors and
// inverts in registers (k_potrf_diag); k_lauum forms A^-1 = L^-T L^-1; the
// O(m^2) slot replacement updates A^-1 in place between refactors; and the
// coefficient kernel applies it. A is padded to a multiple of 64 with an
// identity block so no kernel needs edge handling.
//
// Dense 64 x 64 x 64 tile products (k_lauum) run on fp64 MFMA
// (v_mfma_f64_16x16x4f64): 4 waves, each a 32 x 32 quadrant of 2 x 2 16x16
// tiles, operands from LDS. They are written as C[r][c] = sum_k a[r][k] *
// b[c][k]; a tile that enters as b[k][c] is transposed while it is staged.
#include "internal.h"

namespace mfac {
namespace {

typedef double v4d __attribute__((ext_vector_type(4)));
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

// ------------------------------------------------------------------ potrf
__device__ __forceinline__ double rsqrt_of(double x) { return rsqrt(x); }
__device__ __forceinline__ float rsqrt_of(float x) { return rsqrtf(x); }

// One 64-thread wave per batch item (fp64, or fp32 for the fast static mode): factor diagonal tile t in place (lower)
// and write its inverse into the diagonal tile of Linv. Lane i keeps row i of
// the tile in registers; each column step broadcasts the new column through a
// double-buffered LDS vector (reads of step j and writes of step j+2 are
// separated by the barriers of step j+1), so the trailing update is a run of
// independent FMAs on registers.
template <typename R>
__global__ __launch_bounds__(64) void k_potrf_diag(R* __restrict__ A, R* __restrict__ Linv, int mp, int64_t bstride,
                                                   int t, int* __restrict__ err) {
    __shared__ R col[2][64];
    __shared__ R T[64][65];
    __shared__ R rdiag[64];  // 1 / L[j][j]
    R* Ab = A + (int64_t)blockIdx.x * bstride + (int64_t)t * 64 * mp + t * 64;
    R* Lb = Linv + (int64_t)blockIdx.x * bstride + (int64_t)t * 64 * mp + t * 64;
    const int i = threadIdx.x;
    R a[64];
#pragma unroll
    for (int c = 0; c < 64; ++c) a[c] = Ab[(int64_t)i * mp + c];
    int bad = 0;
#pragma unroll
    for (int j = 0; j < 64; ++j) {
        R* cb = col[j & 1];
        // the pivot lane publishes 1 / L[j][j] = rsqrt(pivot); the column below
        // it scales by that reciprocal (no division on the per-column chain)
        if (i == j) {
            R piv = a[j];
            if (!(piv > R(0)) || !isfinite(piv)) {
                bad = 1;
                piv = R(1);
            }
            const R r = rsqrt_of(piv);
            a[j] = piv * r;
            cb[j] = r;
            rdiag[j] = r;
        }
        __syncthreads();
        if (i > j) {
            a[j] = a[j] * cb[j];
            cb[i] = a[j];
        }
        __syncthreads();
        if (i > j) {
            const R lij = a[j];
#pragma unroll
            for (int c = j + 1; c < 64; ++c) a[c] -= lij * cb[c];
        }
    }
    if (bad) atomicOr(err, 2);
    // the factor (lower part of the registers) into LDS and back to A
#pragma unroll
    for (int c = 0; c < 64; ++c) {
        const R v = (c <= i) ? a[c] : R(0);
        T[i][c] = v;
        Ab[(int64_t)i * mp + c] = v;
    }
    __syncthreads();
    // Column i of the inverse of the lower factor by forward substitution,
    // kept in registers: x_r = (delta_ri - sum_{l<r} T[r][l] x_l) / T[r][r]
    // (as a product with the stored reciprocal).
    // Rows above i come out as exact zeros. Reads of T[r][l] are the same
    // address across the wave (LDS broadcast); the dot products use four
    // partial sums so consecutive FMAs do not wait on each other.
    {
        R x[64];
#pragma unroll
        for (int r = 0; r < 64; ++r) {
            R s0 = (r == i) ? R(1) : R(0), s1 = 0, s2 = 0, s3 = 0;
#pragma unroll
            for (int l = 0; l + 3 < r; l += 4) {
                s0 -= T[r][l] * x[l];
                s1 -= T[r][l + 1] * x[l + 1];
                s2 -= T[r][l + 2] * x[l + 2];
                s3 -= T[r][l + 3] * x[l + 3];
            }
#pragma unroll
            for (int l = r & ~3; l < r; ++l) s0 -= T[r][l] * x[l];
            x[r] = ((s0 + s1) + (s2 + s3)) * rdiag[r];
        }
        __syncthreads();
        // transpose through LDS so each lane writes a row of the inverse
#pragma unroll
        for (int r = 0; r < 64; ++r) T[r][i] = x[r];
    }
    __syncthreads();
#pragma unroll
    for (int c = 0; c < 64; ++c) Lb[(int64_t)i * mp + c] = T[i][c];
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
hipError_t launch_potrf_tile(R* A, R* Linv, int mp, int nbatch, int64_t bstride, int t, int* err, hipStream_t st) {
    hipLaunchKernelGGL(k_potrf_diag<R>, dim3(nbatch), dim3(64), 0, st, A, Linv, mp, bstride, t, err);
    return hipGetLastError();
}
template hipError_t launch_potrf_tile<double>(double*, double*, int, int, int64_t, int, int*, hipStream_t);
template hipError_t launch_potrf_tile<float>(float*, float*, int, int, int64_t, int, int*, hipStream_t);

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

hipError_t launch_coef_from_inv(const double* Ainv, int mp, int m, const double* p, int pstride, int nv, int k,
                                double s0, double s1, double* coef, int* err, hipStream_t st) {
    hipLaunchKernelGGL(k_coef_from_inv, dim3((unsigned)ceil_div(m, 4)), dim3(256), 0, st, Ainv, mp, m, p, pstride, nv,
                       k, s0, s1, coef, err);
    return hipGetLastError();
}

}  // namespace mfac
