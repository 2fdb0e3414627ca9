/*
 * mfac.h - C ABI of the MI355X M-FAC IHVP library (gfx950, HIP).
 *
 * Matrix-free inverse-Hessian-vector products under the damped empirical
 * Fisher of a window of m gradients g_1..g_m in R^d (Frantar, Kurtic, Alistarh,
 * "M-FAC: Efficient Matrix-Free Approximations of Second-Order Information"):
 *
 *     F = lambda * I_d + (1/m) * sum_i g_i g_i^T            (Theorem 1)
 *
 * Two families of calls:
 *   - the dynamic sliding window (Section 3.2; optimizer of Section 4.2):
 *     replace one gradient, refresh the Gram row, recompute the m x m
 *     coefficients, and return F^-1 applied to the new gradient (and to up to
 *     max_queries extra vectors in the same two passes over the window);
 *   - the static block-wise precompute (Section 3.1, block-wise paragraph;
 *     Appendix C) with the inverse-diagonal query and the OBD keep-mask
 *     (Section 4.1).
 *
 * Conventions for every call:
 *   - Pointers are HIP device pointers unless marked (host).
 *   - Vectors of length d are fp32 and contiguous; a batch of n vectors is n
 *     rows of length d with row stride d (row-major). The window calls accept
 *     4-byte aligned vectors and take 128-bit accesses when every vector is
 *     16-byte aligned (and d % 4 == 0 for batches); the static calls state
 *     their own alignment below.
 *   - The library never allocates or frees device memory. Window storage,
 *     workspaces and outputs are owned by the caller and must outlive the
 *     handle (storage/workspace) or the call's stream work (inputs/outputs).
 *   - Calls only enqueue work on the handle's stream and return at once; the
 *     *_status calls and mfac_window_get_rows synchronise that stream.
 *   - Argument errors are detected on the host before anything is enqueued:
 *     the call returns MFAC_EINVAL or MFAC_EWORKSPACE and the handle is
 *     unchanged. A failed HIP launch returns MFAC_EHIP. A non-finite or
 *     non-positive pivot met on the device latches an error word in the
 *     workspace, reported as MFAC_ENONFINITE by the next *_status call.
 *   - A handle is used by one host thread and one stream at a time.
 *   - Calls are not meant for stream capture into HIP graphs: the ring head,
 *     the step count and the refactor counter advance on the host when a call
 *     is made, so a replayed graph would repeat the captured slot and policy.
 */
#ifndef MFAC_H
#define MFAC_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    MFAC_OK = 0,
    MFAC_EINVAL = -1,      /* invalid argument (null pointer, size, range, alignment) */
    MFAC_EWORKSPACE = -2,  /* storage or workspace smaller than the *_bytes query   */
    MFAC_EHIP = -3,        /* a HIP runtime call or kernel launch failed              */
    MFAC_ENONFINITE = -4,  /* non-finite data or non-positive pivot seen on device    */
    MFAC_ESTATE = -5,      /* call not valid in the handle's current state            */
    MFAC_EPRECISION = -6,  /* fast static mode: the keep-mask could not be certified   */
    /* not a status: widens the enum to the full int32 range, so any code a C
       caller passes (e.g. to mfac_status_string) is a valid value of the type */
    MFAC_STATUS_INT32_ = 0x7fffffff
} mfac_status;

typedef struct mfac_window_s* mfac_window;
typedef struct mfac_static_s* mfac_static;

/* Text for a status code (static storage, never NULL). */
const char* mfac_status_string(mfac_status s);

/* Library version as MAJOR*10000 + MINOR*100 + PATCH. */
int32_t mfac_version(void);

/* ======================================================================
 * Dynamic sliding window (Section 3.2; Appendix B; Section 4.2)
 * ====================================================================== */

/* Bytes of window storage for an m x d window. The storage holds the m
 * gradients in a library-chosen layout (column slabs of the window, each slab
 * m rows x a fixed width, zero padded past d); read rows back with
 * mfac_window_get_rows. Returns 0 for d < 1 or m < 1. */
size_t mfac_window_storage_bytes(int64_t d, int32_t m);

/* Bytes of device workspace for the window (Gram matrix and coefficient
 * factor in fp64, per-call partial sums, error word). max_queries bounds the
 * n of mfac_window_replace (n extra queries) and mfac_ihvp. Returns 0 on
 * invalid sizes. */
size_t mfac_window_workspace_bytes(int64_t d, int32_t m, int32_t max_queries);

/* Create a window handle.
 *   1 <= d <= 2^34, m >= 1, lambda > 0 finite (kept in fp64: the
 *   coefficient phase runs in fp64), 0 <= max_queries <= 16,
 *   m * (max_queries + 1) <= 16384.
 *   storage:   >= mfac_window_storage_bytes(d, m), 256-byte aligned.
 *   workspace: >= mfac_window_workspace_bytes(d, m, max_queries), 256-byte aligned.
 *   G0:        m x d row-major initial gradients, or NULL for an empty window
 *              (all rows zero; Theorem 1 keeps the 1/m scale for the capacity
 *              m, so empty slots contribute nothing).
 * Enqueues: copy of G0 into the storage (or zero fill), Gram K = G G^T
 * (fp64 MFMA tiles on the exact fp32 values, fp64 reduction), and the
 * coefficient factor. The ring head starts at slot 0. *out receives a
 * host-allocated handle. */
mfac_status mfac_window_init(mfac_window* out, int64_t d, int32_t m, double lambda,
                             int32_t max_queries, void* storage, size_t storage_bytes,
                             void* workspace, size_t workspace_bytes,
                             const float* G0, hipStream_t stream);

/* Overwrite rows [first, first+count) of the window with count x d row-major
 * rows (no Gram update: call mfac_window_rebuild after the last batch). */
mfac_status mfac_window_set_rows(mfac_window w, int32_t first, int32_t count, const float* rows);

/* Recompute the Gram matrix from the stored rows and refactor the
 * coefficients (the O(d m^2 + m^3) setup of Section 3.2). Also the recovery
 * path after a latched non-finite error once the data is fixed. */
mfac_status mfac_window_rebuild(mfac_window w);

/* The sliding step (Section 3.2 update and multiplication; Appendix B's
 * combined update-multiply; Section 4.2's optimizer step):
 *   1. slot k (k = slot, or the ring head if slot == -1) takes g_new;
 *   2. p = G g_new gives row and column k of the Gram matrix;
 *   3. the m x m coefficients are refactored from the Gram matrix;
 *   4. y_out = F^-1 g_new for the window that now holds g_new, evaluated as
 *      m * G^T (G G^T + m*lambda*I)^-1 e_k (free of the cancellation of the
 *      direct form lambda^-1 g - G^T c), and Y = F^-1 X for the n extra rows.
 * X/Y (n x d) are read/written in the same two passes over the window as g.
 * y_out may be NULL (then only the window is updated); X and Y may be NULL iff
 * n == 0. g_new, X must not alias the window storage or y_out/Y.
 * When slot == -1 the ring head advances to (k + 1) mod m. */
mfac_status mfac_window_replace(mfac_window w, int32_t slot, const float* g_new,
                                float* y_out, int32_t n, const float* X, float* Y);

/* A sequence of sliding steps whose gradients are all known in advance:
 * gradient t of Gn (n x d row-major) enters the ring head, then Yn row t =
 * F_t^-1 Gn[t] for the window F_t that holds gradients 0..t of the sequence
 * (Section 3.2 update and multiplication, as n calls of mfac_window_replace
 * with slot -1, no extra queries). The window read that forms Yn[t] also
 * forms the Gram column of Gn[t+1] (Appendix B reuses one product of the
 * window for the update and the multiplication; here the reuse spans two
 * consecutive steps): the row Gn[t+1] replaces is still read for Yn[t], and
 * its dot with Gn[t+1] is taken as Gn[t+1] . Gn[t+1], its value after the
 * replacement. One read of the window per step instead of two for m <= 2048;
 * larger m runs the two passes per step of mfac_window_replace. Results equal
 * those of the separate calls up to the order of fp64 sums in the Gram
 * column. Not for an optimizer loop, whose next gradient depends on this
 * step's output. n >= 1; Gn and Yn must not alias each other or the window
 * storage. The ring head and step count advance by n. */
mfac_status mfac_window_replace_seq(mfac_window w, int32_t n, const float* Gn, float* Yn);

/* Y = F^-1 X for n x d row-major X (Section 3.2 multiplication; Algorithm 2's
 * role): two passes over the window and an O(m^2) solve with the cached
 * factor. 1 <= n <= max_queries + 1 (the vectors one replace carries). */
mfac_status mfac_ihvp(mfac_window w, int32_t n, const float* X, float* Y);

/* mfac_ihvp for callers that cannot allocate device memory or pass a
 * workspace per call (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): the same computation and results, with
 * the call's scratch (pass-1 partial sums, their reduction and the
 * coefficients) in a fixed 16 MiB device array inside the library instead of
 * the window's workspace. Allocates nothing; no hipMalloc, hipFree or
 * allocating library routine. The array exists once per GPU (held until the
 * process ends; its address is resolved at mfac_window_init) and is shared by
 * every call on that GPU, so calls that overlap on one GPU (several streams
 * or host threads) race and must be serialised by the caller; it keeps the
 * last call's contents, which later calls overwrite before reading.
 * Limit: (512 + 2) * m * n * 8 bytes (each part rounded up to 256) <= 16 MiB,
 * i.e. m * n <= 4080; larger returns MFAC_EWORKSPACE before anything is
 * enqueued. Other arguments and errors as mfac_ihvp. */
mfac_status mfac_ihvp_noalloc(mfac_window w, int32_t n, const float* X, float* Y);

/* Copy rows [first, first+count) back as count x d row-major fp32 (device
 * pointer). Synchronises the stream. */
mfac_status mfac_window_get_rows(mfac_window w, int32_t first, int32_t count, float* rows_out);

/* Current ring head (the slot the next replace with slot == -1 overwrites) and
 * number of replaces so far (host values; no device access). */
mfac_status mfac_window_info(mfac_window w, int32_t* head_out /* host */, int64_t* steps_out /* host */);

/* Set the ring head and step count (resume from a checkpoint of the rows). */
mfac_status mfac_window_set_head(mfac_window w, int32_t head, int64_t steps);

/* How the m x m coefficients follow a replace. The library keeps the explicit
 * fp64 inverse of A = G G^T + m*lambda*I.
 *   period == 0: refactor A from the Gram matrix on every replace (blocked
 *                Cholesky, triangular inverse, L^-T L^-1: the O(m^3) per-replace
 *                cost of Section 3.2's complexity analysis);
 *   period >= 1: O(m^2) update of the inverse on a replace (slot k's old
 *                pivot removed through its Schur complement, the new column
 *                inserted), with a full refactor from the Gram matrix every
 *                `period` replaces to bound rounding drift.
 * Default: max(m, 1024). */
mfac_status mfac_window_set_refactor_period(mfac_window w, int32_t period);

/* Change the stream later calls enqueue on. */
mfac_status mfac_window_set_stream(mfac_window w, hipStream_t stream);

/* Phase timing with HIP events recorded on the handle's stream (a tracing aid,
 * off by default). Phases: 0 = pass-1 kernel (G x), 1 = coefficient phase
 * (partial-sum reduction, Gram row, inverse update or refactor, coefficients),
 * 2 = pass-2 kernel (G^T c), 3 = the write of the new gradient into its slot.
 * enable != 0 starts recording around every replace, replace_seq and ihvp;
 * 0 stops (recorded events are kept until read). In mfac_window_replace_seq
 * phase 2 is the fused pass (G^T c of one step with G x of the next) for all
 * but the last step, and phase 0 runs once, for the first gradient. Each
 * recorded event costs a few microseconds of queue time between launches. */
#define MFAC_NPHASES 4
mfac_status mfac_window_trace(mfac_window w, int32_t enable);

/* Synchronise the stream, add up the recorded phase times: ms_out and
 * count_out (host arrays of MFAC_NPHASES) receive milliseconds and launch
 * counts per phase; the recorded events are then released. */
mfac_status mfac_window_trace_read(mfac_window w, double* ms_out /* host */, int64_t* count_out /* host */);

/* Synchronise the stream and report (then clear) a latched device error. */
mfac_status mfac_window_status(mfac_window w);

/* Free the host handle (device buffers stay with the caller). NULL is a no-op. */
mfac_status mfac_window_destroy(mfac_window w);

/* ======================================================================
 * Static block-wise precompute (Section 3.1; Appendix C) and OBD queries
 * (Section 4.1)
 * ====================================================================== */

/* Bytes of workspace for the static path: per-block fp64 Gram/factor/inverse
 * buffers for a batch of blocks processed together, plus the fp64 inverse
 * diagonal (d values). block must divide d. Returns 0 on invalid sizes. */
size_t mfac_static_workspace_bytes(int64_t d, int32_t block, int32_t m);

/* Precompute for the block-wise Fisher: d/B independent blocks, block b
 * covering columns [bB, (b+1)B) with
 *     F_b = lambda * I_B + (1/m) G_b^T G_b.
 * G is the caller's m x d row-major gradient matrix; it is overwritten in
 * place by W with W_b = R_b^-1 G_b, R_b the Cholesky factor of
 * G_b G_b^T + m*lambda*I (the same role as the paper's V, which Algorithm 3
 * also writes over G: V_i = sqrt(q_i / lambda) W_i). The inverse diagonal
 * diag(F_b^-1) = (1 - sum_i W_b[i,:]^2) / lambda is formed in fp64 from the
 * unrounded W and kept in the workspace.
 * With MFAC_STATIC_FP32 the precompute leaves G intact instead (see the flag).
 * Requirements: 1 <= m <= 8192, 4 <= block, block % 4 == 0,
 * d % block == 0, d <= 2^32 - 256, lambda > 0 finite, G 16-byte aligned,
 * workspace 256-byte aligned (at least mfac_static_workspace_bytes_flags for
 * the flags given), flags a combination of MFAC_STATIC_* bits. */
mfac_status mfac_static_precompute(mfac_static* out, int64_t d, int32_t block, int32_t m,
                                   double lambda, float* G, void* workspace,
                                   size_t workspace_bytes, uint32_t flags, hipStream_t stream);

/* flags of mfac_static_precompute and mfac_static_precompute_paged */
#define MFAC_STATIC_TRACE 1u /* record HIP events around the precompute's stages and
                                mfac_obs_mask; read with mfac_static_trace_read */
/* Fast mode (mfac_static_precompute only; m <= 4096, block <= 65536): the
 * Gram matrices, their Cholesky factors and inverses, and W on fp32 matrix
 * cores (fp32 products and sums: a Gram entry over at most 2048 columns,
 * wider blocks adding their 2048-column splits in fp64; W over the m rows;
 * the squares of W summed in fp64 for the diagonal). The inverse diagonal then
 * carries the fp32 rounding (on gradient-like data with a well-conditioned
 * G_b G_b^T + m*lambda*I, a largest entry error of 4.1e-6 relative measured
 * at d = 4.19M, B = 2048, m = 1024). G is left intact: the fp32 L^-1 of
 * every block is kept in the workspace, and W is formed into the workspace by
 * the first query that reads it (mfac_static_ihvp, mfac_static_element,
 * mfac_obs_update). mfac_obs_mask stays exact: coordinates whose fp64 score
 * lies within 1e-5 relative of the cut get their diagonal recomputed in fp64
 * (iterative refinement against G, see mfac_obs_mask), so the mask equals the
 * fp64 mask whenever the fp32 path's score error is below about 1e-5. */
#define MFAC_STATIC_FP32 2u

/* Workspace bytes for mfac_static_precompute with these flags (the fast mode
 * needs more: the fp32 L^-1 of every block, m*d floats for W, and the band
 * list). 0 on invalid sizes or flags. */
size_t mfac_static_workspace_bytes_flags(int64_t d, int32_t block, int32_t m, uint32_t flags);

/* Host-paged static precompute, for a G larger than the device should hold
 * (Appendix C, swapping gradient blocks between host and GPU memory; here
 * the pages are column ranges, which the block structure makes independent).
 * Computes the same W (written back over G on the host), inverse diagonal
 * and handle as mfac_static_precompute.
 *   G_host:    m x d row-major fp32 in pinned host memory (hipHostMalloc or
 *              a pinned torch tensor), 16-byte aligned; overwritten by W.
 *              Pageable memory is rejected (MFAC_EINVAL).
 *   page_cols: columns per page, a multiple of 4 and, when block < d, of
 *              block (a page holds whole blocks, at most 65535); values above
 *              d mean d; the page width (after that) at most 2^30. Three
 *              device page buffers of m * page_cols floats live in the
 *              workspace.
 * block < d: one sweep; each page is uploaded, its blocks go through Gram,
 * factor and W, and W is downloaded (G crosses the host link twice).
 * block == d: the one block's Gram is summed page by page, factored, and a
 * second sweep forms W page by page, starting with the (up to) three last
 * pages, still on the device (G crosses up to three times).
 * Uploads and downloads run on two streams the handle creates (default
 * priority) and overlap each other and the kernels on `stream`, which waits
 * for the last download before any later call on the handle. The queries
 * (mfac_static_ihvp, mfac_static_element, mfac_obs_update) of a paged
 * handle read W directly from the pinned host buffer over the host link;
 * mfac_inv_diag, mfac_inv_diag64 and mfac_obs_mask use the device diagonal.
 * Other requirements as mfac_static_precompute. */
size_t mfac_static_paged_workspace_bytes(int64_t d, int32_t block, int32_t m, int64_t page_cols);
mfac_status mfac_static_precompute_paged(mfac_static* out, int64_t d, int32_t block, int32_t m,
                                         double lambda, float* G_host, int64_t page_cols, void* workspace,
                                         size_t workspace_bytes, uint32_t flags, hipStream_t stream);

/* Per-stage device time of a static handle created with MFAC_STATIC_TRACE,
 * since creation or the last read (synchronises the stream). ms_out and
 * count_out (host arrays of MFAC_STATIC_NPHASES) receive milliseconds and
 * launch counts for: 0 batched Gram (one launch per batch of blocks), 1
 * factor and inverse, 2 W and inverse diagonal, 3 scores and keep-mask.
 * Without the flag every entry is 0. */
#define MFAC_STATIC_NPHASES 4
mfac_status mfac_static_trace_read(mfac_static s, double* ms_out /* host */, int64_t* count_out /* host */);

/* diag(F^-1) for all d coordinates (Appendix C, row-selected extraction with
 * the identity selection), rounded to fp32. */
mfac_status mfac_inv_diag(mfac_static s, float* diag_out);

/* Same, in fp64 (fp64-accurate in the default mode; in the fast mode it has
 * the fp32 path's error, except coordinates that an mfac_obs_mask call
 * recomputed in its band). */
mfac_status mfac_inv_diag64(mfac_static s, double* diag_out);

/* OBD saliency rho_j = theta_j^2 / (2 [F^-1]_jj) in fp64 (Section 4.1) and a
 * global keep-mask over all blocks: keep_mask[j] = 1 for the `keep` largest
 * rho, ties broken by the lower index; 0 <= keep <= d. scores_out may be
 * NULL. theta 4-byte aligned. Uses workspace scratch; output is exact given
 * the fp64 diagonal. In the fast mode (MFAC_STATIC_FP32) the scores come from
 * the fp32-path diagonal; the keep-th largest score t is selected, every
 * coordinate with a nonzero score within [t(1 - 1e-5), t(1 + 1e-5)] has
 * [F^-1]_jj recomputed in fp64 (x = A_b^-1 g_j by iterative refinement: the
 * residual g_j - A_b x formed from G in fp64, the kept fp32 L^-1 as
 * preconditioner, until the estimated remaining error is below 1e-13 of x;
 * then (1 - g_j.x) /
 * lambda), stored into the diagonal, and the selection runs again. The mask
 * then equals the fp64 mask: a coordinate outside the band is on the same side
 * of the fp64 cut as long as the fp32 scores are within 1e-5 / (1 + 1e-5)
 * relative of the fp64 ones. The refinement measures that error on the band
 * (the coordinates at the cut); if any exceeds 2.5e-6 (a quarter of the band's
 * half-width: the fp32 path is then too inaccurate for this G, e.g. blocks
 * whose Fisher term dwarfs m*lambda), the mask is not certified and the next
 * mfac_static_status returns MFAC_EPRECISION: use the default (fp64) mode. A
 * refinement that does not settle within 12 steps latches MFAC_ENONFINITE. */
mfac_status mfac_obs_mask(mfac_static s, const float* theta, int64_t keep,
                          double* scores_out, uint8_t* keep_mask_out);

/* Y = F^-1 X for the block-wise Fisher, n x d row-major fp32 X and Y,
 * 1 <= n <= 4 (Appendix C eq. 9; with W in place of V and q:
 * F_b^-1 x_b = (x_b - W_b^T (W_b x_b)) / lambda). Two passes over W (the
 * precompute's output in G's storage). X and Y 16-byte aligned and must not
 * alias G. */
mfac_status mfac_static_ihvp(mfac_static s, int32_t n, const float* X, float* Y);

/* Element queries [F^-1]_ij, O(m) each (Section 3.1, eq. 5):
 * (delta_ij - sum_k W[k,i] W[k,j]) / lambda when i and j share a block, 0
 * otherwise; fp64 sums of the fp32 W. ij: device array of 2*nq int64 indices
 * (i_0, j_0, i_1, j_1, ...); out: nq fp64 values. An index outside [0, d)
 * yields NaN and latches MFAC_ENONFINITE. */
mfac_status mfac_static_element(mfac_static s, int64_t nq, const int64_t* ij, double* out);

/* OBS correction (Section 4.1) for removing every coordinate j with
 * keep_mask[j] == 0 at once: delta = -F^-1 x with x_j = theta_j / [F^-1]_jj on
 * removed coordinates and 0 elsewhere, i.e. the sum of the single-weight OBS
 * updates -theta_j F^-1 e_j / [F^-1]_jj (the paper's approximate
 * multi-weight OBS). theta + delta zeroes a removed weight that is the only
 * removed one in its block. theta, delta_out: d fp32 (theta 4-byte,
 * delta_out 16-byte aligned); keep_mask: d uint8. */
mfac_status mfac_obs_update(mfac_static s, const float* theta, const uint8_t* keep_mask, float* delta_out);

mfac_status mfac_static_set_stream(mfac_static s, hipStream_t stream);
mfac_status mfac_static_status(mfac_static s);
mfac_status mfac_static_destroy(mfac_static s);

#ifdef __cplusplus
}
#endif

#endif /* MFAC_H */
