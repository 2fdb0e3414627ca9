// C ABI of libmfac (include/mfac.h): host-side validation, workspace layout
// and the launch sequences of the dynamic and static paths. Nothing here
// computes on the host; every step of the method runs in the kernels of
// pass.hip, gram.hip, chol.hip, factor.hip, static.hip and static_query.hip.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>
#include <vector>

#include "../../include/mfac.h"
#include "internal.h"

#define MFAC_API extern "C" __attribute__((visibility("default")))

using namespace mfac;

namespace {

constexpr int MAX_QUERIES = 16;
constexpr int64_t MAX_MNV = 16384;  // m * (max_queries + 1): the pass LDS stays within 128 KB
constexpr int64_t STATIC_BATCH_BYTES = int64_t(8) << 30;

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

struct Carve {
    char* base;
    size_t off = 0;
    template <typename T>
    T* take(size_t count) {
        T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
        off += align256(count * sizeof(T));
        return p;
    }
};

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }
bool aligned4(const void* p) { return ((uintptr_t)p & 3u) == 0; }

int64_t nslab_of(int64_t d) { return ceil_div(d, SLAB); }
int padded_m(int m) { return (int)round_up(m, NB); }

// ---------------------------------------------------------------- allocation-free IHVP
// Scratch of mfac_ihvp_noalloc: a file-scope device array, one per GPU the
// library runs on, held until the process ends. Host code never uses the
// array's name as an address: it takes the device address from
// hipGetSymbolAddress, once per device (at window init, with the window's
// device current), and passes that pointer on.
constexpr size_t NOALLOC_SCRATCH_BYTES = size_t(16) << 20;
__device__ __align__(256) unsigned char scratch[NOALLOC_SCRATCH_BYTES];

constexpr int MAX_DEVICES = 64;
std::mutex scratch_mu;
void* scratch_dev[MAX_DEVICES];

// Device address of this device's scratch (resolved on first use per device).
hipError_t scratch_address(int device, void** out) {
    *out = nullptr;
    if (device < 0 || device >= MAX_DEVICES) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(scratch_mu);
    if (!scratch_dev[device]) {
        int cur = -1;
        hipError_t e = hipGetDevice(&cur);
        if (e != hipSuccess) return e;
        if (cur != device && (e = hipSetDevice(device)) != hipSuccess) return e;
        void* ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (cur != device) (void)hipSetDevice(cur);
        if (e != hipSuccess) return e;
        scratch_dev[device] = ptr;
    }
    *out = scratch_dev[device];
    return hipSuccess;
}


}  // namespace

struct mfac_window_s {
    int64_t d;
    int m, mp, max_q;
    int device;  // the device of the handle's stream at init
    double lambda;
    int64_t nslab;
    float* G;
    hipStream_t st;
    int* err;
    double *K, *A, *Linv, *Ainv, *part, *p, *zv, *gpart, *coef;
    int64_t gpart_elems;  // the window Gram's partials, and the factor's K segments
    int head;
    int64_t steps;
    // coefficient policy: 0 = refactor from K on every replace; R > 0 = O(m^2)
    // update of the explicit inverse, refactored from K every R replaces
    int32_t period;
    int32_t since_refactor;
    // phase tracing (host side): events recorded around the phases
    bool trace;
    struct Mark {
        int phase;
        hipEvent_t a, b;
    };
    std::vector<Mark>* marks;
    hipEvent_t open_ev;
};

struct mfac_static_s {
    int64_t d;
    int B, m, mp, nblocks, batch;
    double lambda;
    float* G;
    // fast mode (MFAC_STATIC_FP32): fp32 MFMA Gram and W, the fp32 L^-1 of every
    // block kept, G left intact, W formed on the first query into its own
    // buffer; the keep-mask's band recomputed exactly in fp64
    bool fast, w_ready;
    float* W;  // where the queries read W: G (fp64 mode) or the W buffer (fast mode)
    float* A32;  // fast mode: the batch of fp32 Gram matrices, factored in place
    float* L32;  // fast mode: fp32 L^-1 of every block (the factor writes it here)
    unsigned int *band_count, *band_list;
    double* band_work;  // fast mode: the wide band refinement's vectors
    hipStream_t st;
    int* err;
    double *A, *Linv, *gpart, *diag, *scores, *qpart;
    int64_t gpart_elems;  // the Gram's partials, and the factor's K segments when a batch is small
    double* qcoef;
    float* xobs;
    SelectScratch sel;
    // stage tracing (MFAC_STATIC_TRACE): events recorded around the stages
    bool trace;
    std::vector<mfac_window_s::Mark>* marks;
    hipEvent_t open_ev;
    // host-paged precompute: G lives in pinned host memory (G above is its
    // device-visible address), pages of it pass through three device buffers
    bool paged;
    float* Ghost;
    float* page[3];
    hipStream_t up, down;  // host-to-device and device-to-host copy streams
    hipEvent_t pev[12];    // fork, factor done, join, uploaded[3], computed[3], downloaded[3]
};

namespace {

template <typename W>
size_t window_layout(int64_t d, int m, int max_q, char* base, W* w) {
    const int mp = padded_m(m);
    const int nvmax = 1 + max_q;
    Carve c{base};
    int* err = c.take<int>(64);
    double* K = c.take<double>((size_t)m * m);
    double* A = c.take<double>((size_t)mp * mp);
    double* Linv = c.take<double>((size_t)mp * mp);
    double* part = c.take<double>((size_t)PASS1_MAX_GRID * m * nvmax);
    double* Ainv = c.take<double>((size_t)mp * mp);
    double* p = c.take<double>((size_t)m * nvmax);
    double* zv = c.take<double>((size_t)mp * 2);
    double* coef = c.take<double>((size_t)m * nvmax);
    // the init Gram's partials and, later, the refactor's split-K segments
    const int64_t gw = gram_window_part_doubles(m, nslab_of(d)), gk = splitk_part_doubles(mp);
    double* gpart = c.take<double>((size_t)(gw > gk ? gw : gk));
    if (w) {
        w->err = err;
        w->K = K;
        w->A = A;
        w->Linv = Linv;
        w->part = part;
        w->Ainv = Ainv;
        w->p = p;
        w->zv = zv;
        w->coef = coef;
        w->gpart = gpart;
        w->gpart_elems = gw > gk ? gw : gk;
    }
    return c.off;
}

bool window_sizes_ok(int64_t d, int32_t m, int32_t max_q) {
    // d <= 2^34: the row copy kernels launch d/4 work-items (a 32-bit count)
    return d >= 1 && m >= 1 && max_q >= 0 && max_q <= MAX_QUERIES && (int64_t)m * (max_q + 1) <= MAX_MNV &&
           d <= (int64_t(1) << 34);
}

#define HIPCHK(x)                                  \
    do {                                           \
        hipError_t e_ = (x);                       \
        if (e_ != hipSuccess) return MFAC_EHIP;    \
    } while (0)

// Tracing: mark_begin before a phase's first launch, mark_end after its last.
// A phase whose launch failed leaves its begin event open: the next
// mark_begin (or marks_free) releases it. The marks of a phase are recorded
// on the stream it runs on (the handle's, unless given).
template <typename H>
hipError_t mark_begin(H* h, hipStream_t st) {
    if (!h->trace) return hipSuccess;
    if (h->open_ev) {
        (void)hipEventDestroy(h->open_ev);
        h->open_ev = nullptr;
    }
    hipError_t e = hipEventCreate(&h->open_ev);
    if (e != hipSuccess) {
        h->open_ev = nullptr;
        return e;
    }
    return hipEventRecord(h->open_ev, st);
}

template <typename H>
hipError_t mark_end(H* h, int phase, hipStream_t st) {
    if (!h->trace) return hipSuccess;
    hipEvent_t b;
    hipError_t e = hipEventCreate(&b);
    if (e != hipSuccess) return e;
    e = hipEventRecord(b, st);
    h->marks->push_back({phase, h->open_ev, b});
    h->open_ev = nullptr;
    return e;
}

template <typename H>
hipError_t mark_begin(H* h) {
    return mark_begin(h, h->st);
}

template <typename H>
hipError_t mark_end(H* h, int phase) {
    return mark_end(h, phase, h->st);
}

// Sum and release the recorded marks of a handle into ms/count (nph phases).
template <typename H>
mfac_status marks_read(H* h, int nph, double* ms_out, int64_t* count_out) {
    for (int i = 0; i < nph; ++i) {
        ms_out[i] = 0.0;
        count_out[i] = 0;
    }
    if (!h->marks) return MFAC_OK;
    if (hipStreamSynchronize(h->st) != hipSuccess) return MFAC_EHIP;
    mfac_status rc = MFAC_OK;
    for (auto& mk : *h->marks) {
        float ms = 0.f;
        if (hipEventElapsedTime(&ms, mk.a, mk.b) != hipSuccess) rc = MFAC_EHIP;
        ms_out[mk.phase] += ms;
        count_out[mk.phase] += 1;
        (void)hipEventDestroy(mk.a);
        (void)hipEventDestroy(mk.b);
    }
    h->marks->clear();
    return rc;
}

template <typename H>
void marks_free(H* h) {
    if (h->open_ev) {
        (void)hipEventDestroy(h->open_ev);
        h->open_ev = nullptr;
    }
    if (!h->marks) return;
    for (auto& mk : *h->marks) {
        (void)hipEventDestroy(mk.a);
        (void)hipEventDestroy(mk.b);
    }
    delete h->marks;
    h->marks = nullptr;
}

// Full refactor from K (optionally after replacing row/column k with p):
// A = K + m*lambda*I, A = L L^T, Linv = L^-1, Ainv = Linv^T Linv.
mfac_status window_factor(mfac_window w, const double* p, int pstride, int k) {
    HIPCHK(launch_assemble(w->K, w->m, p, pstride, k, (double)w->m * w->lambda, w->A, w->mp, w->err, w->st));
    HIPCHK(launch_factor_invert(w->A, w->Linv, w->mp, 1, 0, w->err, w->st, w->gpart, w->gpart_elems));
    HIPCHK(launch_lauum(w->Linv, w->Ainv, w->mp, 1, 0, w->st));
    w->since_refactor = 0;
    return MFAC_OK;
}

// Coefficients after slot k took a gradient with Gram column p: O(m^2) update
// of the inverse, or a full refactor when the policy asks for one.
mfac_status window_slot_update(mfac_window w, int pstride, int k) {
    if (w->period == 0 || w->since_refactor + 1 >= w->period) return window_factor(w, w->p, pstride, k);
    HIPCHK(launch_inv_replace(w->K, w->m, w->p, pstride, k, (double)w->m * w->lambda, w->Ainv, w->mp, w->zv,
                              w->zv + w->mp, w->err, w->st));
    w->since_refactor += 1;
    return MFAC_OK;
}

// window_slot_update followed by the coefficients coef[i*nv + c] = scale_c
// (Ainv rhs_c)_i (see launch_coef_from_inv); the O(m^2) update forms them in
// the same pass over Ainv.
mfac_status window_slot_update_coef(mfac_window w, int pstride, int k, const double* rhs, int rstride, int nv, int kc,
                                    double s0, double s1) {
    if (w->period == 0 || w->since_refactor + 1 >= w->period) {
        mfac_status rc = window_factor(w, w->p, pstride, k);
        if (rc != MFAC_OK) return rc;
        HIPCHK(launch_coef_from_inv(w->Ainv, w->mp, w->m, rhs, rstride, nv, kc, s0, s1, w->coef, w->err, w->st));
        return MFAC_OK;
    }
    HIPCHK(launch_inv_replace_coef(w->K, w->m, w->p, pstride, k, (double)w->m * w->lambda, w->Ainv, w->mp, w->zv,
                                   w->zv + w->mp, rhs, rstride, nv, kc, s0, s1, w->coef, w->err, w->st));
    w->since_refactor += 1;
    return MFAC_OK;
}

// The coefficient phase of a replace whose pass 1 left its partials in
// w->part (shape grid, nv vectors): p, then the slot update (or refactor) and,
// with nvc > 0, the coefficients (see window_slot_update_coef).
mfac_status window_coef_phase(mfac_window w, const Pass1Grid& grid, int nv, int k, const double* rhs, int rstride,
                              int nvc, int kc, double s0, double s1) {
    HIPCHK(launch_reduce_partials(w->part, grid, w->m, nv, w->p, w->st));
    if (nvc > 0) return window_slot_update_coef(w, nv, k, rhs, rstride, nvc, kc, s0, s1);
    return window_slot_update(w, nv, k);
}

}  // namespace

// ====================================================================== misc

MFAC_API const char* mfac_status_string(mfac_status s) {
    switch (s) {
        case MFAC_OK: return "ok";
        case MFAC_EINVAL: return "invalid argument";
        case MFAC_EWORKSPACE: return "storage or workspace too small";
        case MFAC_EHIP: return "HIP runtime or launch failure";
        case MFAC_ENONFINITE: return "non-finite value or non-positive pivot on device";
        case MFAC_ESTATE: return "call not valid in the current state";
        case MFAC_EPRECISION: return "fast static mode could not certify the keep-mask; use the fp64 mode";
        default: break;
    }
    return "unknown status";
}

MFAC_API int32_t mfac_version(void) { return 100; }

// ====================================================================== window

MFAC_API size_t mfac_window_storage_bytes(int64_t d, int32_t m) {
    if (d < 1 || m < 1) return 0;
    return (size_t)nslab_of(d) * (size_t)m * SLAB * sizeof(float);
}

MFAC_API size_t mfac_window_workspace_bytes(int64_t d, int32_t m, int32_t max_queries) {
    if (!window_sizes_ok(d, m, max_queries)) return 0;
    return window_layout<mfac_window_s>(d, m, max_queries, nullptr, nullptr);
}

MFAC_API mfac_status mfac_window_init(mfac_window* out, int64_t d, int32_t m, double lambda, int32_t max_queries,
                                      void* storage, size_t storage_bytes, void* workspace, size_t workspace_bytes,
                                      const float* G0, hipStream_t stream) {
    if (!out) return MFAC_EINVAL;
    *out = nullptr;
    if (!window_sizes_ok(d, m, max_queries)) return MFAC_EINVAL;
    if (!(lambda > 0.0) || !isfinite(lambda)) return MFAC_EINVAL;
    if (!storage || !workspace) return MFAC_EINVAL;
    if (((uintptr_t)storage & 255u) || ((uintptr_t)workspace & 255u)) return MFAC_EINVAL;
    if (G0 && !aligned4(G0)) return MFAC_EINVAL;
    if (storage_bytes < mfac_window_storage_bytes(d, m)) return MFAC_EWORKSPACE;
    if (workspace_bytes < mfac_window_workspace_bytes(d, m, max_queries)) return MFAC_EWORKSPACE;

    mfac_window w = (mfac_window)calloc(1, sizeof(mfac_window_s));
    if (!w) return MFAC_EINVAL;
    w->d = d;
    w->m = m;
    w->mp = padded_m(m);
    w->max_q = max_queries;
    w->lambda = lambda;
    w->nslab = nslab_of(d);
    w->G = (float*)storage;
    w->st = stream;
    w->period = m > 1024 ? m : 1024;
    if (hipStreamGetDevice(stream, &w->device) != hipSuccess) {
        free(w);
        return MFAC_EHIP;
    }
    {
        // the allocation-free IHVP's scratch on this device, resolved once
        void* sp = nullptr;
        if (scratch_address(w->device, &sp) != hipSuccess) {
            free(w);
            return MFAC_EHIP;
        }
    }
    window_layout<mfac_window_s>(d, m, max_queries, (char*)workspace, w);

    mfac_status rc = MFAC_OK;
    if (launch_fill_zero((float*)w->err, 1, w->st) != hipSuccess) rc = MFAC_EHIP;
    if (rc == MFAC_OK) {
        hipError_t e = G0 ? launch_set_rows(w->G, m, d, w->nslab, 0, m, G0, d, w->st)
                          : launch_fill_zero(w->G, w->nslab * (int64_t)m * SLAB, w->st);
        if (e != hipSuccess) rc = MFAC_EHIP;
    }
    if (rc == MFAC_OK) {
        if (G0) {
            rc = mfac_window_rebuild(w);
        } else {
            // empty window: K = 0 without a Gram pass over the zero rows
            if (launch_fill_zero((float*)w->K, 2 * (int64_t)m * m, w->st) != hipSuccess) rc = MFAC_EHIP;
            if (rc == MFAC_OK) rc = window_factor(w, nullptr, 0, -1);
        }
    }
    if (rc != MFAC_OK) {
        free(w);
        return rc;
    }
    *out = w;
    return MFAC_OK;
}

MFAC_API mfac_status mfac_window_set_rows(mfac_window w, int32_t first, int32_t count, const float* rows) {
    if (!w || !rows || first < 0 || count < 1 || (int64_t)first + count > w->m || !aligned4(rows)) return MFAC_EINVAL;
    HIPCHK(launch_set_rows(w->G, w->m, w->d, w->nslab, first, count, rows, w->d, w->st));
    return MFAC_OK;
}

MFAC_API mfac_status mfac_window_rebuild(mfac_window w) {
    if (!w) return MFAC_EINVAL;
    HIPCHK(launch_gram_window(w->G, w->m, w->nslab, w->gpart, w->K, w->st));
    return window_factor(w, nullptr, 0, -1);
}

MFAC_API mfac_status mfac_window_replace(mfac_window w, int32_t slot, const float* g_new, float* y_out, int32_t n,
                                         const float* X, float* Y) {
    if (!w || !g_new) return MFAC_EINVAL;
    if (slot < -1 || slot >= w->m) return MFAC_EINVAL;
    if (n < 0 || n > w->max_q) return MFAC_EINVAL;
    if (n > 0 && (!X || !Y)) return MFAC_EINVAL;
    if (!aligned4(g_new) || (y_out && !aligned4(y_out)) || (n > 0 && (!aligned4(X) || !aligned4(Y))))
        return MFAC_EINVAL;
    const int k = slot < 0 ? w->head : slot;
    const int nv = 1 + n;
    const int64_t d = w->d;

    VecIn vin{};
    vin.v[0] = g_new;
    bool al = aligned16(g_new) && (y_out == nullptr || aligned16(y_out));
    for (int q = 0; q < n; ++q) vin.v[1 + q] = X + (int64_t)q * d;
    if (n > 0) al = al && aligned16(X) && aligned16(Y) && (d % 4 == 0);

    Pass1Grid grid{};
    HIPCHK(mark_begin(w));
    HIPCHK(launch_write_row(w->G, w->m, d, w->nslab, k, g_new, w->st));
    HIPCHK(mark_end(w, 3));
    HIPCHK(mark_begin(w));
    HIPCHK(launch_pass1(w->G, w->m, d, w->nslab, nv, vin, al, w->part, &grid, w->st));
    HIPCHK(mark_end(w, 0));
    HIPCHK(mark_begin(w));

    if (y_out || n > 0) {
        // column 0: c' = -m A^-1 e_k, so y = -G^T c' = m G^T A^-1 e_k;
        // queries: C = lambda^-1 A^-1 P, y = x / lambda - G^T C
        const double inv_lam = 1.0 / w->lambda;
        VecOut vout{};
        int v0 = 0;
        if (!y_out) v0 = 1;  // skip the inserted-gradient column
        int nv2 = 0;
        for (int v = v0; v < nv; ++v, ++nv2) {
            vout.x[nv2] = v == 0 ? nullptr : X + (int64_t)(v - 1) * d;
            vout.y[nv2] = v == 0 ? y_out : Y + (int64_t)(v - 1) * d;
            vout.alpha[nv2] = v == 0 ? 0.0f : (float)inv_lam;
        }
        // no y_out: coefficients of the queries only (columns 1..n of p)
        const mfac_status rc = v0 == 0 ? window_coef_phase(w, grid, nv, k, w->p, nv, nv, k, -(double)w->m, inv_lam)
                                       : window_coef_phase(w, grid, nv, k, w->p + 1, nv, nv2, -1, inv_lam, inv_lam);
        if (rc != MFAC_OK) return rc;
        HIPCHK(mark_end(w, 1));
        HIPCHK(mark_begin(w));
        HIPCHK(launch_pass2(w->G, w->m, d, w->nslab, nv2, w->coef, vout, al, w->st));
        HIPCHK(mark_end(w, 2));
    } else {
        const mfac_status rc = window_coef_phase(w, grid, nv, k, w->p, nv, 0, -1, 0.0, 0.0);
        if (rc != MFAC_OK) return rc;
        HIPCHK(mark_end(w, 1));
    }
    if (slot < 0) w->head = (k + 1) % w->m;
    w->steps += 1;
    return MFAC_OK;
}

MFAC_API mfac_status mfac_window_replace_seq(mfac_window w, int32_t n, const float* Gn, float* Yn) {
    if (!w || !Gn || !Yn || n < 1) return MFAC_EINVAL;
    if (!aligned4(Gn) || !aligned4(Yn)) return MFAC_EINVAL;
    const int64_t d = w->d;
    const int m = w->m;
    const bool al = aligned16(Gn) && aligned16(Yn) && (n == 1 || d % 4 == 0);
    const double inv_lam = 1.0 / w->lambda;
    const bool fused = m <= PASS21_MAX_M;

    // coefficients of gradient t once its Gram column is in p (slot k)
    auto coefficients = [&](const Pass1Grid& grid, int k) -> mfac_status {
        return window_coef_phase(w, grid, 1, k, w->p, 1, 1, k, -(double)m, inv_lam);
    };

    int k = w->head;
    Pass1Grid grid{};
    VecIn vin{};
    vin.v[0] = Gn;
    HIPCHK(mark_begin(w));
    HIPCHK(launch_write_row(w->G, m, d, w->nslab, k, Gn, w->st));
    HIPCHK(mark_end(w, 3));
    HIPCHK(mark_begin(w));
    HIPCHK(launch_pass1(w->G, m, d, w->nslab, 1, vin, al, w->part, &grid, w->st));
    HIPCHK(mark_end(w, 0));
    HIPCHK(mark_begin(w));
    w->head = (k + 1) % m;
    w->steps += 1;
    mfac_status rc = coefficients(grid, k);
    if (rc != MFAC_OK) return rc;
    HIPCHK(mark_end(w, 1));

    for (int32_t t = 0; t < n; ++t) {
        float* y = Yn + (int64_t)t * d;
        VecOut vout{};
        vout.x[0] = nullptr;
        vout.y[0] = y;
        vout.alpha[0] = 0.0f;
        if (t + 1 == n) {
            HIPCHK(mark_begin(w));
            HIPCHK(launch_pass2(w->G, m, d, w->nslab, 1, w->coef, vout, al, w->st));
            HIPCHK(mark_end(w, 2));
            break;
        }
        const float* gnext = Gn + (int64_t)(t + 1) * d;
        const int knext = (k + 1) % m;
        HIPCHK(mark_begin(w));
        if (fused) {
            // y_t and the next gradient's Gram column in one read of the
            // window; the next gradient enters its slot only after that read
            HIPCHK(launch_pass2_next(w->G, m, d, w->nslab, w->coef, y, gnext, knext, al, w->part, &grid, w->st));
            HIPCHK(mark_end(w, 2));
            HIPCHK(mark_begin(w));
            HIPCHK(launch_write_row(w->G, m, d, w->nslab, knext, gnext, w->st));
            HIPCHK(mark_end(w, 3));
        } else {
            HIPCHK(launch_pass2(w->G, m, d, w->nslab, 1, w->coef, vout, al, w->st));
            HIPCHK(mark_end(w, 2));
            HIPCHK(mark_begin(w));
            HIPCHK(launch_write_row(w->G, m, d, w->nslab, knext, gnext, w->st));
            HIPCHK(mark_end(w, 3));
            HIPCHK(mark_begin(w));
            vin.v[0] = gnext;
            HIPCHK(launch_pass1(w->G, m, d, w->nslab, 1, vin, al, w->part, &grid, w->st));
            HIPCHK(mark_end(w, 0));
        }
        HIPCHK(mark_begin(w));
        w->head = (knext + 1) % m;
        w->steps += 1;
        rc = coefficients(grid, knext);
        if (rc != MFAC_OK) return rc;
        HIPCHK(mark_end(w, 1));
        k = knext;
    }
    return MFAC_OK;
}

namespace {

// Y = F^-1 X for n rows: pass 1 into part, its reduction into p, the
// coefficients into coef, pass 2 (part, p, coef: scratch of the call).
mfac_status ihvp_run(mfac_window w, int32_t n, const float* X, float* Y, double* part, double* p, double* coef) {
    const int64_t d = w->d;
    const bool al = aligned16(X) && aligned16(Y) && (n == 1 || d % 4 == 0);
    VecIn vin{};
    VecOut vout{};
    const double inv_lam = 1.0 / w->lambda;
    for (int q = 0; q < n; ++q) {
        vin.v[q] = X + (int64_t)q * d;
        vout.x[q] = X + (int64_t)q * d;
        vout.y[q] = Y + (int64_t)q * d;
        vout.alpha[q] = (float)inv_lam;
    }
    Pass1Grid grid{};
    HIPCHK(mark_begin(w));
    HIPCHK(launch_pass1(w->G, w->m, d, w->nslab, n, vin, al, part, &grid, w->st));
    HIPCHK(mark_end(w, 0));
    HIPCHK(mark_begin(w));
    HIPCHK(launch_reduce_partials(part, grid, w->m, n, p, w->st));
    HIPCHK(launch_coef_from_inv(w->Ainv, w->mp, w->m, p, n, n, -1, inv_lam, inv_lam, coef, w->err, w->st));
    HIPCHK(mark_end(w, 1));
    HIPCHK(mark_begin(w));
    HIPCHK(launch_pass2(w->G, w->m, d, w->nslab, n, coef, vout, al, w->st));
    HIPCHK(mark_end(w, 2));
    return MFAC_OK;
}

bool ihvp_args_ok(mfac_window w, int32_t n, const float* X, float* Y) {
    return w && X && Y && n >= 1 && n <= w->max_q + 1 && aligned4(X) && aligned4(Y);
}

// Scratch layout of one call: pass-1 partials (at most PASS1_MAX_GRID
// work-groups x m rows x n vectors), the reduced sums p and the coefficients.
size_t noalloc_need(int m, int n, size_t* off_p, size_t* off_c) {
    const size_t mn = (size_t)m * n * sizeof(double);
    const size_t part = align256((size_t)PASS1_MAX_GRID * mn);
    *off_p = part;
    *off_c = part + align256(mn);
    return *off_c + align256(mn);
}

}  // namespace

MFAC_API mfac_status mfac_ihvp(mfac_window w, int32_t n, const float* X, float* Y) {
    if (!ihvp_args_ok(w, n, X, Y)) return MFAC_EINVAL;
    return ihvp_run(w, n, X, Y, w->part, w->p, w->coef);
}

MFAC_API mfac_status mfac_ihvp_noalloc(mfac_window w, int32_t n, const float* X, float* Y) {
    if (!ihvp_args_ok(w, n, X, Y)) return MFAC_EINVAL;
    size_t op, oc;
    if (noalloc_need(w->m, n, &op, &oc) > NOALLOC_SCRATCH_BYTES) return MFAC_EWORKSPACE;
    void* base = nullptr;
    HIPCHK(scratch_address(w->device, &base));
    char* b = (char*)base;
    return ihvp_run(w, n, X, Y, (double*)b, (double*)(b + op), (double*)(b + oc));
}

MFAC_API mfac_status mfac_window_get_rows(mfac_window w, int32_t first, int32_t count, float* rows_out) {
    if (!w || !rows_out || first < 0 || count < 1 || (int64_t)first + count > w->m || !aligned4(rows_out))
        return MFAC_EINVAL;
    HIPCHK(launch_get_rows(w->G, w->m, w->d, first, count, rows_out, w->d, w->st));
    HIPCHK(hipStreamSynchronize(w->st));
    return MFAC_OK;
}

MFAC_API mfac_status mfac_window_info(mfac_window w, int32_t* head_out, int64_t* steps_out) {
    if (!w) return MFAC_EINVAL;
    if (head_out) *head_out = w->head;
    if (steps_out) *steps_out = w->steps;
    return MFAC_OK;
}

MFAC_API mfac_status mfac_window_set_head(mfac_window w, int32_t head, int64_t steps) {
    if (!w || head < 0 || head >= w->m || steps < 0) return MFAC_EINVAL;
    w->head = head;
    w->steps = steps;
    return MFAC_OK;
}

MFAC_API mfac_status mfac_window_set_refactor_period(mfac_window w, int32_t period) {
    if (!w || period < 0) return MFAC_EINVAL;
    w->period = period;
    return MFAC_OK;
}

MFAC_API mfac_status mfac_window_set_stream(mfac_window w, hipStream_t stream) {
    if (!w) return MFAC_EINVAL;
    w->st = stream;
    return MFAC_OK;
}

MFAC_API mfac_status mfac_window_trace(mfac_window w, int32_t enable) {
    if (!w) return MFAC_EINVAL;
    if (enable && !w->marks) w->marks = new std::vector<mfac_window_s::Mark>();
    w->trace = enable != 0;
    return MFAC_OK;
}

MFAC_API mfac_status mfac_window_trace_read(mfac_window w, double* ms_out, int64_t* count_out) {
    if (!w || !ms_out || !count_out) return MFAC_EINVAL;
    return marks_read(w, MFAC_NPHASES, ms_out, count_out);
}

MFAC_API mfac_status mfac_window_status(mfac_window w) {
    if (!w) return MFAC_EINVAL;
    HIPCHK(hipStreamSynchronize(w->st));
    int e = 0;
    HIPCHK(hipMemcpy(&e, w->err, sizeof(int), hipMemcpyDeviceToHost));
    if (e != 0) {
        HIPCHK(launch_fill_zero((float*)w->err, 1, w->st));
        HIPCHK(hipStreamSynchronize(w->st));
        return MFAC_ENONFINITE;
    }
    return MFAC_OK;
}

MFAC_API mfac_status mfac_window_destroy(mfac_window w) {
    if (!w) return MFAC_OK;
    marks_free(w);
    free(w);
    return MFAC_OK;
}

// ====================================================================== static

namespace {

bool static_sizes_ok(int64_t d, int32_t B, int32_t m) {
    // d <= 2^32 - 256: the element-wise kernels launch one work-item per
    // coordinate (a 32-bit count)
    return d >= 1 && B >= 4 && m >= 1 && (B % 4) == 0 && d % B == 0 && m <= 8192 &&
           d <= (int64_t(1) << 32) - 256;
}

// the fast mode's band refinement keeps 3m + 2048 doubles in LDS and reads a
// whole block per band coordinate and step
constexpr int FAST_MAX_M = 4096;
constexpr int FAST_MAX_B = 65536;
// relative half-width of the band re-decided in fp64 (the fp32 path's score
// error must stay below tau / (1 + tau); measured near 1e-8 on the pruning
// workload)
constexpr double BAND_TAU = 1e-5;

bool static_flags_ok(int64_t d, int32_t B, int32_t m, uint32_t flags) {
    if (flags & ~(MFAC_STATIC_TRACE | MFAC_STATIC_FP32)) return false;
    if ((flags & MFAC_STATIC_FP32) && (m > FAST_MAX_M || B > FAST_MAX_B)) return false;
    return static_sizes_ok(d, B, m);
}

int static_batch(int64_t d, int B, int m) {
    const int mp = padded_m(m);
    const int64_t nblocks = d / B;
    const int64_t per = (int64_t)mp * mp * 8 * 2;
    int64_t b = STATIC_BATCH_BYTES / per;
    // MFAC_STATIC_BATCH_BLOCKS caps the blocks processed per batch (tests use it
    // to cover batch boundaries at small sizes); read by both the workspace
    // query and the precompute, so keep it fixed between the two calls.
    if (const char* env = getenv("MFAC_STATIC_BATCH_BLOCKS")) {
        const long cap = strtol(env, nullptr, 10);
        if (cap > 0 && cap < b) b = cap;
    }
    if (b < 1) b = 1;
    if (b > 65535) b = 65535;
    if (b > nblocks) b = nblocks;
    // batches of equal size up to rounding (the last one may be smaller)
    const int64_t nbatch = ceil_div(nblocks, b);
    return (int)ceil_div(nblocks, nbatch);
}

// partial-tile storage of the split block Gram, for the largest need among the
// batch sizes used (full batches and the last one); the fast mode's fp32
// kernel has its own tiles and splits
int64_t static_gram_part(int64_t nblocks, int batch, int mp, int B, bool fast) {
    const int last = (int)(nblocks - (ceil_div(nblocks, batch) - 1) * batch);
    auto need = [&](int nb) { return fast ? gram_blocks32_part_doubles(nb, mp, B) : gram_blocks_part_doubles(nb, mp, B); };
    const int64_t a = need(batch), b = need(last);
    return a > b ? a : b;
}

template <typename S>
size_t static_layout(int64_t d, int B, int m, bool fast, char* base, S* s) {
    const int mp = padded_m(m);
    const int batch = static_batch(d, B, m);
    Carve c{base};
    int* err = c.take<int>(64);
    double* diag = c.take<double>((size_t)d);
    double* scores = c.take<double>((size_t)d);
    char* sel = c.take<char>((size_t)select_scratch_bytes(d));
    // fp64 mode: a batch of fp64 A and L^-1; fast mode: a batch of fp32 A, and
    // the fp32 L^-1 of every block, W and the band list
    double* A = fast ? nullptr : c.take<double>((size_t)batch * mp * mp);
    double* Linv = fast ? nullptr : c.take<double>((size_t)batch * mp * mp);
    // the Gram's partials and, in the fp64 mode with small batches (few
    // GEMM tasks), the factor's split-K segments
    const int64_t ggp = static_gram_part(d / B, batch, mp, B, fast);
    const int64_t gsk = (!fast && batch < 256) ? splitk_part_doubles(mp) : 0;
    double* gpart = c.take<double>((size_t)(ggp > gsk ? ggp : gsk));
    double* qpart = c.take<double>((size_t)static_query_part_doubles(d, B, m));
    double* qcoef = c.take<double>((size_t)(d / B) * m * 4);
    float* xobs = c.take<float>((size_t)d);
    float *A32 = nullptr, *L32 = nullptr, *W = nullptr;
    unsigned int *bcount = nullptr, *blist = nullptr;
    double* bwork = nullptr;
    if (fast) {
        A32 = c.take<float>((size_t)batch * mp * mp);
        L32 = c.take<float>((size_t)(d / B) * mp * mp);
        W = c.take<float>((size_t)m * d);
        bcount = c.take<unsigned int>(64);
        blist = c.take<unsigned int>((size_t)d);
        bwork = c.take<double>((size_t)band_work_doubles(m, B));
    }
    if (s) {
        s->A32 = A32;
        s->L32 = L32;
        s->W = W;
        s->band_count = bcount;
        s->band_list = blist;
        s->band_work = bwork;
        s->qpart = qpart;
        s->qcoef = qcoef;
        s->xobs = xobs;
        s->err = err;
        s->diag = diag;
        s->scores = scores;
        s->sel = select_scratch_carve(sel, d);
        s->A = A;
        s->Linv = Linv;
        s->gpart = gpart;
        s->gpart_elems = ggp > gsk ? ggp : gsk;
        s->batch = batch;
    }
    return c.off;
}

// Frees the host-side handle: trace events, and for a paged handle its copy
// streams (after their work has finished) and events.
void static_release(mfac_static_s* s) {
    if (s->up) {
        (void)hipStreamSynchronize(s->up);
        (void)hipStreamDestroy(s->up);
    }
    if (s->down) {
        (void)hipStreamSynchronize(s->down);
        (void)hipStreamDestroy(s->down);
    }
    for (int i = 0; i < 12; ++i)
        if (s->pev[i]) (void)hipEventDestroy(s->pev[i]);
    marks_free(s);
    free(s);
}

}  // namespace

MFAC_API size_t mfac_static_workspace_bytes(int64_t d, int32_t block, int32_t m) {
    if (!static_sizes_ok(d, block, m)) return 0;
    return static_layout<mfac_static_s>(d, block, m, false, nullptr, nullptr);
}

MFAC_API size_t mfac_static_workspace_bytes_flags(int64_t d, int32_t block, int32_t m, uint32_t flags) {
    if (!static_flags_ok(d, block, m, flags)) return 0;
    return static_layout<mfac_static_s>(d, block, m, (flags & MFAC_STATIC_FP32) != 0, nullptr, nullptr);
}

MFAC_API mfac_status mfac_static_precompute(mfac_static* out, int64_t d, int32_t block, int32_t m, double lambda,
                                            float* G, void* workspace, size_t workspace_bytes, uint32_t flags,
                                            hipStream_t stream) {
    if (!out) return MFAC_EINVAL;
    *out = nullptr;
    if (!static_flags_ok(d, block, m, flags)) return MFAC_EINVAL;
    if (!(lambda > 0.0) || !isfinite(lambda)) return MFAC_EINVAL;
    if (!G || !workspace || !aligned16(G) || ((uintptr_t)workspace & 255u)) return MFAC_EINVAL;
    if (workspace_bytes < mfac_static_workspace_bytes_flags(d, block, m, flags)) return MFAC_EWORKSPACE;
    const bool fast = (flags & MFAC_STATIC_FP32) != 0;

    mfac_static s = (mfac_static)calloc(1, sizeof(mfac_static_s));
    if (!s) return MFAC_EINVAL;
    s->d = d;
    s->B = block;
    s->m = m;
    s->mp = padded_m(m);
    s->nblocks = (int)(d / block);
    s->lambda = lambda;
    s->G = G;
    s->st = stream;
    s->trace = (flags & MFAC_STATIC_TRACE) != 0;
    if (s->trace) s->marks = new std::vector<mfac_window_s::Mark>();
    static_layout<mfac_static_s>(d, block, m, fast, (char*)workspace, s);
    s->fast = fast;
    if (!fast) s->W = G;  // W is written over G

    const int64_t bstride = (int64_t)s->mp * s->mp;
    const double mu = (double)m * lambda;
    auto fail = [&]() {
        (void)hipStreamSynchronize(s->st);
        static_release(s);
        return MFAC_EHIP;
    };
    if (launch_fill_zero((float*)s->err, 1, s->st) != hipSuccess) return fail();
    for (int b0 = 0; b0 < s->nblocks; b0 += s->batch) {
        const int nb = (s->nblocks - b0) < s->batch ? (s->nblocks - b0) : s->batch;
        // fast mode: fp32 Gram, fp32 factor whose L^-1 goes to the kept
        // per-block store, and the diagonal from the fp32 W (not stored)
        float* L32b = fast ? s->L32 + (int64_t)b0 * bstride : nullptr;
        if (mark_begin(s) != hipSuccess) return fail();
        const hipError_t eg = fast ? launch_gram_blocks32(G, m, d, block, b0, nb, mu, s->A32, s->mp, s->gpart, s->st)
                                   : launch_gram_blocks(G, m, d, block, b0, nb, mu, s->A, s->mp, s->gpart, s->st);
        if (eg != hipSuccess) return fail();
        if (mark_end(s, 0) != hipSuccess || mark_begin(s) != hipSuccess) return fail();
        const hipError_t ef = fast ? launch_factor_invert32(s->A32, L32b, s->mp, nb, bstride, s->err, s->st)
                                   : launch_factor_invert(s->A, s->Linv, s->mp, nb, bstride, s->err, s->st, s->gpart,
                                                          s->gpart_elems);
        if (ef != hipSuccess) return fail();
        if (mark_end(s, 1) != hipSuccess || mark_begin(s) != hipSuccess) return fail();
        const hipError_t et =
            fast ? launch_trmm32(L32b, s->mp, bstride, G, m, d, block, b0, nb, lambda, s->diag, nullptr, s->st)
                 : launch_trmm_diag(s->Linv, s->mp, bstride, G, m, d, block, b0, nb, lambda, s->diag, s->st);
        if (et != hipSuccess) return fail();
        if (mark_end(s, 2) != hipSuccess) return fail();
    }
    *out = s;
    return MFAC_OK;
}

MFAC_API mfac_status mfac_static_trace_read(mfac_static s, double* ms_out, int64_t* count_out) {
    if (!s || !ms_out || !count_out) return MFAC_EINVAL;
    return marks_read(s, MFAC_STATIC_NPHASES, ms_out, count_out);
}

MFAC_API mfac_status mfac_inv_diag(mfac_static s, float* diag_out) {
    if (!s || !diag_out || !aligned4(diag_out)) return MFAC_EINVAL;
    HIPCHK(launch_diag_to_f32(s->diag, s->d, diag_out, s->st));
    return MFAC_OK;
}

MFAC_API mfac_status mfac_inv_diag64(mfac_static s, double* diag_out) {
    if (!s || !diag_out || ((uintptr_t)diag_out & 7u)) return MFAC_EINVAL;
    HIPCHK(hipMemcpyAsync(diag_out, s->diag, (size_t)s->d * sizeof(double), hipMemcpyDeviceToDevice, s->st));
    return MFAC_OK;
}

MFAC_API mfac_status mfac_obs_mask(mfac_static s, const float* theta, int64_t keep, double* scores_out,
                                   uint8_t* keep_mask_out) {
    if (!s || !theta || !keep_mask_out || keep < 0 || keep > s->d || !aligned4(theta)) return MFAC_EINVAL;
    if (scores_out && ((uintptr_t)scores_out & 7u)) return MFAC_EINVAL;
    double* sc = scores_out ? scores_out : s->scores;
    HIPCHK(mark_begin(s));
    HIPCHK(launch_scores(theta, s->diag, s->d, sc, s->err, s->st));
    if (s->fast)
        HIPCHK(launch_band_refine(sc, s->d, keep, s->sel, BAND_TAU, s->band_count, s->band_list, s->band_work, s->G, s->m, s->B,
                                  s->L32, s->mp, (int64_t)s->mp * s->mp, s->lambda, theta, s->diag, sc, s->err,
                                  s->st));
    HIPCHK(launch_topk_mask(sc, s->d, keep, s->sel, keep_mask_out, s->st));
    HIPCHK(mark_end(s, 3));
    return MFAC_OK;
}

namespace {
// Fast mode: W = L^-1 G for every block into the W buffer, once, from the kept
// fp32 L^-1 (G stays intact for later keep-masks).
mfac_status ensure_w(mfac_static s) {
    if (!s->fast || s->w_ready) return MFAC_OK;
    const int64_t bstride = (int64_t)s->mp * s->mp;
    HIPCHK(launch_trmm32(s->L32, s->mp, bstride, s->G, s->m, s->d, s->B, 0, s->nblocks, s->lambda, nullptr, s->W,
                         s->st));
    s->w_ready = true;
    return MFAC_OK;
}
}  // namespace

MFAC_API mfac_status mfac_static_ihvp(mfac_static s, int32_t n, const float* X, float* Y) {
    if (!s || !X || !Y || n < 1 || n > 4 || !aligned16(X) || !aligned16(Y)) return MFAC_EINVAL;
    const double inv_lam = 1.0 / s->lambda;
    const mfac_status rc = ensure_w(s);
    if (rc != MFAC_OK) return rc;
    HIPCHK(launch_static_ihvp(s->W, s->m, s->d, s->B, n, X, (float)inv_lam, inv_lam, Y, s->qpart, s->qcoef, s->st));
    return MFAC_OK;
}

MFAC_API mfac_status mfac_static_element(mfac_static s, int64_t nq, const int64_t* ij, double* out) {
    if (!s || nq < 0 || (nq > 0 && (!ij || !out)) || ((uintptr_t)ij & 7u) || ((uintptr_t)out & 7u))
        return MFAC_EINVAL;
    const mfac_status rc = ensure_w(s);
    if (rc != MFAC_OK) return rc;
    HIPCHK(launch_static_element(s->W, s->m, s->d, s->B, nq, ij, s->lambda, out, s->err, s->st));
    return MFAC_OK;
}

MFAC_API mfac_status mfac_obs_update(mfac_static s, const float* theta, const uint8_t* keep_mask, float* delta_out) {
    if (!s || !theta || !keep_mask || !delta_out || !aligned4(theta) || !aligned16(delta_out)) return MFAC_EINVAL;
    const double inv_lam = 1.0 / s->lambda;
    const mfac_status rc = ensure_w(s);
    if (rc != MFAC_OK) return rc;
    HIPCHK(launch_obs_x(theta, keep_mask, s->diag, s->d, s->xobs, s->st));
    // delta = -F^-1 x = -x / lambda + W^T (W x) / lambda
    HIPCHK(launch_static_ihvp(s->W, s->m, s->d, s->B, 1, s->xobs, (float)-inv_lam, -inv_lam, delta_out, s->qpart,
                              s->qcoef, s->st));
    return MFAC_OK;
}

MFAC_API mfac_status mfac_static_set_stream(mfac_static s, hipStream_t stream) {
    if (!s) return MFAC_EINVAL;
    s->st = stream;
    return MFAC_OK;
}

MFAC_API mfac_status mfac_static_status(mfac_static s) {
    if (!s) return MFAC_EINVAL;
    HIPCHK(hipStreamSynchronize(s->st));
    int e = 0;
    HIPCHK(hipMemcpy(&e, s->err, sizeof(int), hipMemcpyDeviceToHost));
    if (e != 0) {
        HIPCHK(launch_fill_zero((float*)s->err, 1, s->st));
        HIPCHK(hipStreamSynchronize(s->st));
        // bit 64: the band refinement measured an fp32 error too large for its band
        return e == 64 ? MFAC_EPRECISION : MFAC_ENONFINITE;
    }
    return MFAC_OK;
}

MFAC_API mfac_status mfac_static_destroy(mfac_static s) {
    if (!s) return MFAC_OK;
    static_release(s);
    return MFAC_OK;
}

// ====================================================================== paged static

namespace {

// Pages of a host-resident G: pc columns each (whole blocks when B < d, any
// multiple of 4 when the single block spans d), pb blocks per page.
struct PagedPlan {
    int64_t pc, npages;
    int pb;
};

bool paged_plan(int64_t d, int32_t B, int32_t m, int64_t page_cols, PagedPlan& pl) {
    if (!static_sizes_ok(d, B, m) || page_cols < 4 || page_cols % 4 != 0) return false;
    const int64_t pc = page_cols < d ? page_cols : d;
    if (pc > (int64_t(1) << 30)) return false;  // kernels take a page's width as int
    if (B < d) {
        if (pc % B != 0 || pc / B > 65535) return false;
        pl.pb = (int)(pc / B);
    } else {
        pl.pb = 1;
    }
    pl.pc = pc;
    pl.npages = ceil_div(d, pc);
    return true;
}

template <typename S>
size_t static_paged_layout(int64_t d, int B, int m, const PagedPlan& pl, char* base, S* s) {
    const int mp = padded_m(m);
    const int64_t nb_last = B < d ? (d - (pl.npages - 1) * pl.pc) / B : 1;
    const int wide = B < d ? B : (int)pl.pc;  // block width the page's Gram sees
    const int64_t pa = gram_blocks_part_doubles(pl.pb, mp, wide), pb2 = gram_blocks_part_doubles((int)nb_last, mp, wide);
    Carve c{base};
    int* err = c.take<int>(64);
    double* diag = c.take<double>((size_t)d);
    double* scores = c.take<double>((size_t)d);
    char* sel = c.take<char>((size_t)select_scratch_bytes(d));
    double* A = c.take<double>((size_t)pl.pb * mp * mp);
    double* Linv = c.take<double>((size_t)pl.pb * mp * mp);
    const int64_t gpp = pa > pb2 ? pa : pb2;
    const int64_t gsk = pl.pb < 256 ? splitk_part_doubles(mp) : 0;
    double* gpart = c.take<double>((size_t)(gpp > gsk ? gpp : gsk));
    double* qpart = c.take<double>((size_t)static_query_part_doubles(d, B, m));
    double* qcoef = c.take<double>((size_t)(d / B) * m * 4);
    float* xobs = c.take<float>((size_t)d);
    float* pg[3];
    for (int i = 0; i < 3; ++i) pg[i] = c.take<float>((size_t)m * pl.pc);
    if (s) {
        s->err = err;
        s->diag = diag;
        s->scores = scores;
        s->sel = select_scratch_carve(sel, d);
        s->A = A;
        s->Linv = Linv;
        s->gpart = gpart;
        s->gpart_elems = gpp > gsk ? gpp : gsk;
        s->qpart = qpart;
        s->qcoef = qcoef;
        s->xobs = xobs;
        for (int i = 0; i < 3; ++i) s->page[i] = pg[i];
        s->batch = pl.pb;
    }
    return c.off;
}

#define PCHK(x)                              \
    do {                                     \
        if ((x) != hipSuccess) return false; \
    } while (0)

// The page pipeline. Copies run on their own streams (uploads and downloads
// overlap each other and the kernels); the kernels run in order on the
// handle's stream; three device buffers rotate between pages, each reused
// once the page before in it has been downloaded (or, in a Gram-only sweep,
// consumed). With two, a buffer's upload-compute-download cycle, not the
// host link, set the pace.
bool paged_run(mfac_static s, const PagedPlan& pl, double mu) {
    const int64_t d = s->d;
    const int m = s->m, B = s->B, mp = s->mp;
    const int64_t bstride = (int64_t)mp * mp;
    hipStream_t st = s->st;
    hipEvent_t* E = s->pev;  // 0 fork, 1 factor done, 2 join, 3+b uploaded, 6+b computed, 9+b downloaded
    auto cols = [&](int64_t p, int64_t& c0) {
        c0 = p * pl.pc;
        return (d - c0) < pl.pc ? (d - c0) : pl.pc;
    };
    auto upload = [&](int64_t p, int b, hipEvent_t after) {
        int64_t c0;
        const int64_t nc = cols(p, c0);
        if (after) PCHK(hipStreamWaitEvent(s->up, after, 0));
        PCHK(hipMemcpy2DAsync(s->page[b], (size_t)pl.pc * 4, s->Ghost + c0, (size_t)d * 4, (size_t)nc * 4,
                              (size_t)m, hipMemcpyHostToDevice, s->up));
        PCHK(hipEventRecord(E[3 + b], s->up));
        PCHK(hipStreamWaitEvent(st, E[3 + b], 0));
        return true;
    };
    auto download = [&](int64_t p, int b) {
        int64_t c0;
        const int64_t nc = cols(p, c0);
        PCHK(hipEventRecord(E[6 + b], st));
        PCHK(hipStreamWaitEvent(s->down, E[6 + b], 0));
        PCHK(hipMemcpy2DAsync(s->Ghost + c0, (size_t)d * 4, s->page[b], (size_t)pl.pc * 4, (size_t)nc * 4,
                              (size_t)m, hipMemcpyDeviceToHost, s->down));
        PCHK(hipEventRecord(E[9 + b], s->down));
        return true;
    };
    PCHK(launch_fill_zero((float*)s->err, 1, st));
    PCHK(hipEventRecord(E[0], st));
    PCHK(hipStreamWaitEvent(s->up, E[0], 0));
    PCHK(hipStreamWaitEvent(s->down, E[0], 0));
    if (B < d) {
        // whole blocks per page: Gram, factor, W and diagonal, then back to the host
        for (int64_t p = 0; p < pl.npages; ++p) {
            const int b = (int)(p % 3);
            int64_t c0;
            const int nbp = (int)(cols(p, c0) / B);
            if (!upload(p, b, p >= 3 ? E[9 + b] : nullptr)) return false;
            PCHK(mark_begin(s));
            PCHK(launch_gram_blocks(s->page[b], m, pl.pc, B, 0, nbp, mu, s->A, mp, s->gpart, st));
            PCHK(mark_end(s, 0));
            PCHK(mark_begin(s));
            PCHK(launch_factor_invert(s->A, s->Linv, mp, nbp, bstride, s->err, st, s->gpart, s->gpart_elems));
            PCHK(mark_end(s, 1));
            PCHK(mark_begin(s));
            PCHK(launch_trmm_diag(s->Linv, mp, bstride, s->page[b], m, pl.pc, B, 0, nbp, s->lambda, s->diag + c0, st));
            PCHK(mark_end(s, 2));
            if (!download(p, b)) return false;
        }
    } else {
        // one block over all pages: its Gram summed page by page, the factor,
        // then a second sweep for W and the diagonal
        for (int64_t p = 0; p < pl.npages; ++p) {
            const int b = (int)(p % 3);
            int64_t c0;
            const int nc = (int)cols(p, c0);
            if (!upload(p, b, p >= 3 ? E[6 + b] : nullptr)) return false;
            PCHK(mark_begin(s));
            PCHK(launch_gram_blocks(s->page[b], m, pl.pc, nc, 0, 1, mu, s->A, mp, s->gpart, st, p > 0));
            PCHK(mark_end(s, 0));
            PCHK(hipEventRecord(E[6 + b], st));
        }
        PCHK(mark_begin(s));
        PCHK(launch_factor_invert(s->A, s->Linv, mp, 1, bstride, s->err, st, s->gpart, s->gpart_elems));
        PCHK(mark_end(s, 1));
        PCHK(hipEventRecord(E[1], st));
        PCHK(hipStreamWaitEvent(s->up, E[1], 0));
        // the last (up to) three pages are still in their buffers: they go
        // first, without a second upload; the others follow in order, each
        // in the buffer that the page processed three steps earlier freed
        const int64_t nres = pl.npages < 3 ? pl.npages : 3;
        int ring[3];
        for (int64_t q = 0; q < pl.npages; ++q) {
            const int64_t p = q < nres ? pl.npages - 1 - q : q - nres;
            int64_t c0;
            const int nc = (int)cols(p, c0);
            int b;
            if (q < nres) {
                b = (int)(p % 3);
                ring[q] = b;
            } else {
                b = ring[q % 3];
                if (!upload(p, b, E[9 + b])) return false;
            }
            PCHK(mark_begin(s));
            PCHK(launch_trmm_diag(s->Linv, mp, bstride, s->page[b], m, pl.pc, nc, 0, 1, s->lambda, s->diag + c0, st));
            PCHK(mark_end(s, 2));
            if (!download(p, b)) return false;
        }
    }
    PCHK(hipEventRecord(E[2], s->down));
    PCHK(hipStreamWaitEvent(st, E[2], 0));
    return true;
}

#undef PCHK

}  // namespace

MFAC_API size_t mfac_static_paged_workspace_bytes(int64_t d, int32_t block, int32_t m, int64_t page_cols) {
    PagedPlan pl;
    if (!paged_plan(d, block, m, page_cols, pl)) return 0;
    return static_paged_layout<mfac_static_s>(d, block, m, pl, nullptr, nullptr);
}

MFAC_API mfac_status mfac_static_precompute_paged(mfac_static* out, int64_t d, int32_t block, int32_t m,
                                                  double lambda, float* G_host, int64_t page_cols, void* workspace,
                                                  size_t workspace_bytes, uint32_t flags, hipStream_t stream) {
    if (!out) return MFAC_EINVAL;
    *out = nullptr;
    PagedPlan pl;
    if (!paged_plan(d, block, m, page_cols, pl)) return MFAC_EINVAL;
    if (flags & ~MFAC_STATIC_TRACE) return MFAC_EINVAL;
    if (!(lambda > 0.0) || !isfinite(lambda)) return MFAC_EINVAL;
    if (!G_host || !workspace || !aligned16(G_host) || ((uintptr_t)workspace & 255u)) return MFAC_EINVAL;
    // G must be pinned host memory (hipHostMalloc): the copies stream from it
    // and the queries read it in place
    hipPointerAttribute_t at;
    if (hipPointerGetAttributes(&at, G_host) != hipSuccess) {
        (void)hipGetLastError();
        return MFAC_EINVAL;
    }
    if (at.type != hipMemoryTypeHost || !at.devicePointer) return MFAC_EINVAL;
    if (workspace_bytes < mfac_static_paged_workspace_bytes(d, block, m, page_cols)) return MFAC_EWORKSPACE;

    mfac_static s = (mfac_static)calloc(1, sizeof(mfac_static_s));
    if (!s) return MFAC_EINVAL;
    s->d = d;
    s->B = block;
    s->m = m;
    s->mp = padded_m(m);
    s->nblocks = (int)(d / block);
    s->lambda = lambda;
    s->G = (float*)at.devicePointer;
    s->W = s->G;
    s->Ghost = G_host;
    s->paged = true;
    s->st = stream;
    s->trace = (flags & MFAC_STATIC_TRACE) != 0;
    if (s->trace) s->marks = new std::vector<mfac_window_s::Mark>();
    static_paged_layout<mfac_static_s>(d, block, m, pl, (char*)workspace, s);
    bool ok = hipStreamCreateWithFlags(&s->up, hipStreamNonBlocking) == hipSuccess &&
              hipStreamCreateWithFlags(&s->down, hipStreamNonBlocking) == hipSuccess;
    for (int i = 0; ok && i < 12; ++i) ok = hipEventCreateWithFlags(&s->pev[i], hipEventDisableTiming) == hipSuccess;
    if (ok) ok = paged_run(s, pl, (double)m * lambda);
    if (!ok) {
        (void)hipStreamSynchronize(s->st);
        static_release(s);
        return MFAC_EHIP;
    }
    *out = s;
    return MFAC_OK;
}
