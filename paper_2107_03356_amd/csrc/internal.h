// Internal declarations shared by the HIP translation units of libmfac.
// Not part of the public ABI (include/mfac.h is).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mfac {

// Window storage: the m x d window is kept as column slabs of SLAB floats;
// slab s holds columns [s*SLAB, (s+1)*SLAB) of all m rows, row i of the slab
// at offset i*SLAB (so one slab is a contiguous m*SLAB block). Columns past d
// in the last slab are zero.
constexpr int SLAB = 2048;
// Coefficient matrices are padded to a multiple of NB with an identity block.
constexpr int NB = 64;
constexpr int MAXNV = 17;  // 1 inserted gradient + up to 16 extra queries
constexpr int PASS1_MAX_GRID = 512;

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int64_t round_up(int64_t a, int64_t b) { return ceil_div(a, b) * b; }

// Pointer/scale sets for the multi-vector passes (passed by value).
struct VecIn {
    const float* v[MAXNV];
};
struct VecOut {
    const float* x[MAXNV];  // x_v, or nullptr when alpha_v == 0
    float* y[MAXNV];
    float alpha[MAXNV];
};

// ---------------------------------------------------------------- passes
// Fill n floats with zero.
hipError_t launch_fill_zero(float* p, int64_t n, hipStream_t st);
// rows (count x d, row-major, leading dimension ld) -> window rows [first, first+count)
hipError_t launch_set_rows(float* G, int m, int64_t d, int64_t nslab, int first, int count,
                           const float* rows, int64_t ld, hipStream_t st);
hipError_t launch_get_rows(const float* G, int m, int64_t d, int first, int count,
                           float* rows, int64_t ld, hipStream_t st);
// Row k of the window <- g (d floats; zero padding past d).
hipError_t launch_write_row(float* G, int m, int64_t d, int64_t nslab, int k, const float* g, hipStream_t st);
// Pass-1 launch shape: gx work-groups per row group, ng row groups of mg rows
// (the last may hold fewer); gx * ng <= PASS1_MAX_GRID.
struct Pass1Grid {
    int gx, ng, mg;
};
// Pass 1: partial sums of G[i,:] . vec_v over the chunks of each work-group,
// part[(g * gx + b) * mg * nv + (i - g * mg) * nv + v] for work-group b of
// row group g = i / mg. Returns the launch shape.
hipError_t launch_pass1(const float* G, int m, int64_t d, int64_t nslab, int nv,
                        const VecIn& vin, bool aligned, double* part, Pass1Grid* grid_out, hipStream_t st);
// p[i*nv + v] = sum over the work-groups of row i's group (fixed order, fp64)
hipError_t launch_reduce_partials(const double* part, const Pass1Grid& pg, int m, int nv, double* p,
                                  hipStream_t st);
// Pass 2: y_v = alpha_v x_v - sum_i coef[i*nv+v] G[i,:] (fp64 coefficients and
// accumulation, fp32 output)
hipError_t launch_pass2(const float* G, int m, int64_t d, int64_t nslab, int nv,
                        const double* coef, const VecOut& vout, bool aligned, hipStream_t st);

// Pass 2 of one step fused with pass 1 of the next (one vector each, m <=
// PASS21_MAX_M): y = -G^T coef and the partial dots of the rows with gn, row
// knext counted as gn . gn; partials in the layout of launch_pass1 (returned
// shape: one row group).
constexpr int PASS21_MAX_M = 2048;  // coefficients, row sums and 2 x 4 x SLAB fp64 partials: 160 KB of LDS
hipError_t launch_pass2_next(const float* G, int m, int64_t d, int64_t nslab, const double* coef, float* y,
                             const float* gn, int knext, bool aligned, double* part, Pass1Grid* grid_out,
                             hipStream_t st);

// ---------------------------------------------------------------- Gram
// Window Gram: K (m x m, fp64, full symmetric) = sum over slabs of G_s G_s^T,
// fp64 MFMA tiles; part must hold gram_window_part_doubles().
int64_t gram_window_part_doubles(int m, int64_t nslab);
hipError_t launch_gram_window(const float* G, int m, int64_t nslab, double* part, double* K,
                              hipStream_t st);
// Static blocks: A_b = G_b G_b^T + mu I (fp64 MFMA), padded to mp with identity;
// blocks [b0, b0+nb) of the m x d row-major G (row stride d), block width B.
// Batches with few tiles split the columns over work-groups: part must then
// hold gram_blocks_part_doubles(nb, mp, B) doubles (0 when no split is used).
// accumulate: A_b += G_b G_b^T instead (the lower tiles), no mu or padding;
// a wide block paged through the device in column pages sums its pages so.
int64_t gram_blocks_part_doubles(int nb, int mp, int B);
hipError_t launch_gram_blocks(const float* G, int m, int64_t d, int B, int b0, int nb,
                              double mu, double* A, int mp, double* part, hipStream_t st,
                              bool accumulate = false);
// The same on fp32 MFMA in 256 x 256 tiles (fp32 sums over at most 2048
// columns, longer blocks split and the splits summed in fp64), stored as fp32
// A; no accumulate mode. part: gram_blocks32_part_doubles(nb, mp, B).
int64_t gram_blocks32_part_doubles(int nb, int mp, int B);
hipError_t launch_gram_blocks32(const float* G, int m, int64_t d, int B, int b0, int nb, double mu, float* A,
                                int mp, double* part, hipStream_t st);

// ---------------------------------------------------------------- coefficients
// A (mp x mp) = K (m x m) + mu I, identity padding; optionally first replaces
// row/column k of K with p (dynamic replace).
hipError_t launch_assemble(double* K, int m, const double* p, int pstride, int k, double mu,
                           double* A, int mp, int* err, hipStream_t st);
// Cholesky factor and inverse of nbatch SPD matrices (mp x mp, mp a multiple
// of 64, batch stride bstride): the lower triangle of Linv <- L^-1 (the
// diagonal 64 x 64 tiles carry zeros above their diagonals; the strictly
// upper tiles are left unspecified: readers use the lower triangle only). A is
// consumed (its contents afterwards are scratch). err |= 2 on a non-positive
// pivot. Recursive blocked algorithm on batched fp64 MFMA GEMMs.
// part (part_elems doubles, or nullptr): room for the K segments of GEMMs
// with few tasks (one matrix), which then split K over more work-groups;
// splitk_part_doubles(mp) covers every GEMM of an mp factor.
hipError_t launch_factor_invert(double* A, double* Linv, int mp, int nbatch, int64_t bstride, int* err,
                                hipStream_t st, double* part = nullptr, int64_t part_elems = 0);
int64_t splitk_part_doubles(int mp);
// The same in fp32 (fp32 matrix cores and leaves), for the fast static mode.
hipError_t launch_factor_invert32(float* A, float* Linv, int mp, int nbatch, int64_t bstride, int* err,
                                  hipStream_t st);
// Ainv = Linv^T Linv (the explicit inverse of A = L L^T), full mp x mp.
hipError_t launch_lauum(const double* Linv, double* Ainv, int mp, int nbatch, int64_t bstride, hipStream_t st);
// O(m^2) slot replacement: K row/column k <- p and Ainv <- (A with column k
// replaced)^-1; z, v: mp-double scratch vectors.
hipError_t launch_inv_replace(double* K, int m, const double* p, int pstride, int k, double mu, double* Ainv,
                              int mp, double* z, double* v, int* err, hipStream_t st);
// launch_inv_replace, then the coefficients of launch_coef_from_inv (rhs at
// stride rstride, nv columns, column kc the new Ainv's column if kc >= 0)
// formed in the same pass over Ainv.
hipError_t launch_inv_replace_coef(double* K, int m, const double* p, int pstride, int k, double mu, double* Ainv,
                                  int mp, double* z, double* v, const double* rhs, int rstride, int nv, int kc,
                                  double s0, double s1, double* coef, int* err, hipStream_t st);
// coef[i*nv+c] = scale_c (Ainv rhs_c)_i: rhs_0 = e_k if k >= 0 (scale s0); the
// other columns rhs_c[j] = p[j*pstride + c] (scale s1; also column 0 if k < 0).
hipError_t launch_coef_from_inv(const double* Ainv, int mp, int m, const double* p, int pstride, int nv, int k,
                                double s0, double s1, double* coef, int* err, hipStream_t st);

// ---------------------------------------------------------------- static
// W_b = Linv_b G_b in place over G (fp32), colsum of squares in fp64 -> diag
hipError_t launch_trmm_diag(const double* Linv, int mp, int64_t bstride, float* G, int m,
                            int64_t d, int B, int b0, int nb, double lam, double* diag,
                            hipStream_t st);
// W_b = Linv_b G_b on fp32 MFMA for blocks [b0, b0+nb): Linv the fp32 L^-1
// of each block at batch stride lstride; G is read only. diag (or nullptr):
// (1 - colsum(W^2)) / lam in fp64 from the fp32 W. Wout (or nullptr): W, row
// stride d.
hipError_t launch_trmm32(const float* Linv, int mp, int64_t lstride, const float* G, int m, int64_t d, int B, int b0,
                         int nb, double lam, double* diag, float* Wout, hipStream_t st);
hipError_t launch_diag_to_f32(const double* diag, int64_t d, float* out, hipStream_t st);
hipError_t launch_scores(const float* theta, const double* diag, int64_t d, double* scores,
                         int* err, hipStream_t st);
// Radix selection of the keep-th largest score and the keep-mask
struct SelectScratch {
    unsigned int* hist;       // 256 bins
    unsigned long long* state;  // prefix, mask, remaining rank, (unused)
    unsigned int* chunk_cnt;  // per-chunk tie counts
    int nchunk;
};
int64_t select_scratch_bytes(int64_t d);
SelectScratch select_scratch_carve(void* base, int64_t d);
// The band step of the fast static mode: selects the keep-th largest score t,
// lists the coordinates with |s - t| <= tau t (s != 0) and recomputes their
// diagonal exactly (fp64 iterative refinement against G with the fp32 L^-1
// as preconditioner), writing diag and scores of those coordinates.
// list: d entries; count: one word; work: band_work_doubles(m, B) doubles.
// m <= 4096.
int64_t band_work_doubles(int m, int B);
hipError_t launch_band_refine(const double* scores_in, int64_t d, int64_t keep, SelectScratch sc, double tau,
                              unsigned int* count, unsigned int* list, double* work, const float* G, int m, int B,
                              const float* L32, int mp, int64_t lstride, double lam, const float* theta,
                              double* diag, double* scores, int* err, hipStream_t st);
hipError_t launch_topk_mask(const double* scores, int64_t d, int64_t keep, SelectScratch sc,
                            uint8_t* mask, hipStream_t st);

// ---------------------------------------------------------------- static queries
int64_t static_query_part_doubles(int64_t d, int B, int m);
// Y = alpha X - W_b^T (pscale W_b X) per block, n <= 4 vectors (row-major, stride d)
hipError_t launch_static_ihvp(const float* W, int m, int64_t d, int B, int n, const float* X, float alpha,
                              double pscale, float* Y, double* part, double* coef, hipStream_t st);
hipError_t launch_obs_x(const float* theta, const uint8_t* keep, const double* diag, int64_t d, float* x,
                        hipStream_t st);
hipError_t launch_static_element(const float* W, int m, int64_t d, int B, int64_t nq, const int64_t* ij, double lam,
                                 double* out, int* err, hipStream_t st);

}  // namespace mfac
