// Host-side check of libmfac's C ABI (csrc/capi.hip) under AddressSanitizer
// and UndefinedBehaviorSanitizer, without a GPU.
//
// capi.hip is linked against stubs of the HIP runtime and of the kernel
// launchers (mfac::launch_* and the size helpers of the other translation
// units). Device buffers are fake address ranges that nothing dereferences;
// every launcher stub checks that the buffers it receives lie inside the
// ranges the caller handed to the library (storage, workspace, inputs,
// outputs), which bounds-checks the workspace carving on the host. Handles
// are created, driven through every entry point and destroyed; a launch
// failure is injected at every position of init, rebuild and the static
// precomputes, and each failing call must return MFAC_EHIP and release what
// it created. LeakSanitizer and the stream/event counters catch what is not
// released. Exit status 0 and "host check ok" on success.
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <vector>

#include "../../include/mfac.h"
#include "../../paper_2107_03356_amd/csrc/internal.h"

// ------------------------------------------------------------------ fake device memory
namespace {

struct Region {
    uintptr_t base;
    size_t bytes;
    const char* name;
};
std::vector<Region> regions;
uintptr_t next_base = uintptr_t(1) << 44;  // far from any host mapping; never dereferenced
int failures = 0;
long launches = 0;
long fail_at = -1;  // the launch (1-based count) that returns an error, or -1
long streams_live = 0, events_live = 0;

#define CHECK(c)                                                                    \
    do {                                                                            \
        if (!(c)) {                                                                 \
            fprintf(stderr, "host check failed: %s (%s:%d)\n", #c, __FILE__, __LINE__); \
            ++failures;                                                             \
        }                                                                           \
    } while (0)

void* fake_alloc(size_t bytes, const char* name) {
    const uintptr_t b = next_base;
    next_base += (bytes + (1u << 20) + 4095) & ~uintptr_t(4095);  // a gap after each range
    regions.push_back({b, bytes, name});
    return (void*)b;
}

// Forget the buffers of one case; the library's scratch (its address is
// resolved once per device and kept) stays registered.
void fake_reset() {
    std::vector<Region> keep;
    for (const Region& r : regions)
        if (strcmp(r.name, "scratch") == 0) keep.push_back(r);
    regions = keep;
}

// [p, p + bytes) inside one registered range
bool inside(const void* p, size_t bytes) {
    const uintptr_t a = (uintptr_t)p;
    for (const Region& r : regions)
        if (a >= r.base && a + bytes <= r.base + r.bytes && a + bytes >= a) return true;
    return false;
}

#define IN(p, bytes)                                                                           \
    do {                                                                                       \
        if (!inside((p), (size_t)(bytes))) {                                                   \
            fprintf(stderr, "host check failed: %s [%zu bytes] outside every buffer (%s:%d)\n", #p, \
                    (size_t)(bytes), __FILE__, __LINE__);                                      \
            ++failures;                                                                        \
        }                                                                                      \
    } while (0)

hipError_t launched() {
    ++launches;
    return launches == fail_at ? hipErrorInvalidValue : hipSuccess;
}

}  // namespace

// ------------------------------------------------------------------ HIP runtime stubs
extern "C" {
void** __hipRegisterFatBinary(const void*) {
    static void* module = nullptr;
    return &module;
}
void __hipRegisterVar(void**, void*, char*, char*, int, size_t, int, int) {}
void __hipUnregisterFatBinary(void**) {}

hipError_t hipGetLastError(void) { return hipSuccess; }
hipError_t hipGetDevice(int* d) {
    *d = 0;
    return hipSuccess;
}
hipError_t hipSetDevice(int) { return hipSuccess; }
hipError_t hipStreamGetDevice(hipStream_t, hipDevice_t* d) {
    *d = 0;
    return hipSuccess;
}
hipError_t hipGetSymbolAddress(void** p, const void*) {
    static void* scratch = nullptr;
    if (!scratch) scratch = fake_alloc(16u << 20, "scratch");
    *p = scratch;
    return hipSuccess;
}
hipError_t hipStreamSynchronize(hipStream_t) { return hipSuccess; }
hipError_t hipStreamCreateWithFlags(hipStream_t* s, unsigned int) {
    *s = (hipStream_t) new char[8];
    ++streams_live;
    return hipSuccess;
}
hipError_t hipStreamDestroy(hipStream_t s) {
    delete[](char*) s;
    --streams_live;
    return hipSuccess;
}
hipError_t hipStreamWaitEvent(hipStream_t, hipEvent_t, unsigned int) { return hipSuccess; }
hipError_t hipEventCreate(hipEvent_t* e) {
    *e = (hipEvent_t) new char[8];
    ++events_live;
    return hipSuccess;
}
hipError_t hipEventCreateWithFlags(hipEvent_t* e, unsigned) { return hipEventCreate(e); }
hipError_t hipEventDestroy(hipEvent_t e) {
    delete[](char*) e;
    --events_live;
    return hipSuccess;
}
hipError_t hipEventRecord(hipEvent_t, hipStream_t) { return hipSuccess; }
hipError_t hipEventElapsedTime(float* ms, hipEvent_t, hipEvent_t) {
    *ms = 1.0f;
    return hipSuccess;
}
hipError_t hipMemcpy(void* dst, const void* src, size_t bytes, hipMemcpyKind kind) {
    if (kind == hipMemcpyDeviceToHost) {
        IN(src, bytes);
        memset(dst, 0, bytes);  // the latched error word reads as clear
    }
    return hipSuccess;
}
hipError_t hipMemcpyAsync(void* dst, const void* src, size_t bytes, hipMemcpyKind, hipStream_t) {
    IN(dst, bytes);
    IN(src, bytes);
    return launched();
}
hipError_t hipMemcpy2DAsync(void* dst, size_t dpitch, const void* src, size_t spitch, size_t width, size_t height,
                            hipMemcpyKind, hipStream_t) {
    if (height > 0) {
        IN(dst, dpitch * (height - 1) + width);
        IN(src, spitch * (height - 1) + width);
    }
    return launched();
}
hipError_t hipPointerGetAttributes(hipPointerAttribute_t* at, const void* p) {
    memset(at, 0, sizeof(*at));
    for (const Region& r : regions)
        if ((uintptr_t)p == r.base && strcmp(r.name, "pinned") == 0) {
            at->type = hipMemoryTypeHost;
            at->devicePointer = (void*)p;
            at->hostPointer = (void*)p;
            return hipSuccess;
        }
    at->type = hipMemoryTypeDevice;
    at->devicePointer = (void*)p;
    return hipSuccess;
}
}  // extern "C"

// ------------------------------------------------------------------ launcher stubs
namespace mfac {

hipError_t launch_fill_zero(float* p, int64_t n, hipStream_t) {
    IN(p, n * 4);
    return launched();
}
hipError_t launch_set_rows(float* G, int m, int64_t, int64_t nslab, int first, int count, const float* rows,
                           int64_t ld, hipStream_t) {
    IN(G, nslab * m * SLAB * 4);
    IN(rows, ((int64_t)(count - 1) * ld + ld) * 4);
    CHECK(first >= 0 && first + count <= m);
    return launched();
}
hipError_t launch_get_rows(const float* G, int m, int64_t d, int first, int count, float* rows, int64_t ld,
                           hipStream_t) {
    IN(G, ceil_div(d, SLAB) * m * SLAB * 4);
    IN(rows, ((int64_t)(count - 1) * ld + d) * 4);
    CHECK(first >= 0 && first + count <= m);
    return launched();
}
hipError_t launch_write_row(float* G, int m, int64_t d, int64_t nslab, int k, const float* g, hipStream_t) {
    IN(G, nslab * m * SLAB * 4);
    IN(g, d * 4);
    CHECK(k >= 0 && k < m);
    return launched();
}
hipError_t launch_pass1(const float* G, int m, int64_t d, int64_t nslab, int nv, const VecIn& vin, bool,
                        double* part, Pass1Grid* grid, hipStream_t) {
    IN(G, nslab * m * SLAB * 4);
    for (int v = 0; v < nv; ++v) IN(vin.v[v], d * 4);
    IN(part, (int64_t)PASS1_MAX_GRID * m * nv * 8);
    CHECK(nv >= 1 && nv <= MAXNV);
    *grid = Pass1Grid{PASS1_MAX_GRID, 1, m};
    return launched();
}
hipError_t launch_reduce_partials(const double* part, const Pass1Grid& pg, int m, int nv, double* p, hipStream_t) {
    IN(part, (int64_t)pg.gx * pg.ng * pg.mg * nv * 8);
    IN(p, (int64_t)m * nv * 8);
    return launched();
}
hipError_t launch_pass2(const float* G, int m, int64_t d, int64_t nslab, int nv, const double* coef,
                        const VecOut& vout, bool, hipStream_t) {
    IN(G, nslab * m * SLAB * 4);
    IN(coef, (int64_t)m * nv * 8);
    for (int v = 0; v < nv; ++v) {
        if (vout.x[v]) IN(vout.x[v], d * 4);
        IN(vout.y[v], d * 4);
    }
    return launched();
}
hipError_t launch_pass2_next(const float* G, int m, int64_t d, int64_t nslab, const double* coef, float* y,
                             const float* gn, int knext, bool, double* part, Pass1Grid* grid, hipStream_t) {
    IN(G, nslab * m * SLAB * 4);
    IN(coef, (int64_t)m * 8);
    IN(y, d * 4);
    IN(gn, d * 4);
    IN(part, (int64_t)PASS1_MAX_GRID * m * 8);
    CHECK(knext >= 0 && knext < m);
    *grid = Pass1Grid{PASS1_MAX_GRID, 1, m};
    return launched();
}
int64_t gram_window_part_doubles(int m, int64_t nslab) { return (int64_t)m * m * (nslab < 8 ? nslab : 8); }
hipError_t launch_gram_window(const float* G, int m, int64_t nslab, double* part, double* K, hipStream_t) {
    IN(G, nslab * m * SLAB * 4);
    IN(part, gram_window_part_doubles(m, nslab) * 8);
    IN(K, (int64_t)m * m * 8);
    return launched();
}
int64_t gram_blocks_part_doubles(int nb, int mp, int B) { return B > 4096 ? (int64_t)nb * mp * mp * 2 : 0; }
hipError_t launch_gram_blocks(const float* G, int m, int64_t d, int B, int b0, int nb, double, double* A, int mp,
                              double* part, hipStream_t, bool) {
    IN(G, ((int64_t)(m - 1) * d + (int64_t)(b0 + nb) * B) * 4);
    IN(A, (int64_t)nb * mp * mp * 8);
    if (gram_blocks_part_doubles(nb, mp, B)) IN(part, gram_blocks_part_doubles(nb, mp, B) * 8);
    return launched();
}
int64_t gram_blocks32_part_doubles(int nb, int mp, int B) { return B > 2048 ? (int64_t)nb * mp * mp * 3 : 0; }
hipError_t launch_gram_blocks32(const float* G, int m, int64_t d, int B, int b0, int nb, double, float* A, int mp,
                                double* part, hipStream_t) {
    IN(G, ((int64_t)(m - 1) * d + (int64_t)(b0 + nb) * B) * 4);
    IN(A, (int64_t)nb * mp * mp * 4);
    if (gram_blocks32_part_doubles(nb, mp, B)) IN(part, gram_blocks32_part_doubles(nb, mp, B) * 8);
    return launched();
}
hipError_t launch_trmm32(const float* Linv, int mp, int64_t lstride, const float* G, int m, int64_t d, int B, int b0,
                         int nb, double, double* diag, float* Wout, hipStream_t) {
    IN(Linv, ((int64_t)(nb - 1) * lstride + (int64_t)mp * mp) * 4);
    IN(G, ((int64_t)(m - 1) * d + (int64_t)(b0 + nb) * B) * 4);
    if (diag) IN(diag + (int64_t)b0 * B, (int64_t)nb * B * 8);
    if (Wout) IN(Wout, ((int64_t)(m - 1) * d + (int64_t)(b0 + nb) * B) * 4);
    return launched();
}
int64_t band_work_doubles(int m, int B) { return 64 * (3 * (int64_t)((m + 3) & ~3) + B) + 2 * 6 * 64; }
hipError_t launch_band_refine(const double* scores_in, int64_t d, int64_t keep, SelectScratch sc, double tau,
                              unsigned int* count, unsigned int* list, double* work, const float* G, int m, int B,
                              const float* L32, int mp, int64_t lstride, double, const float* theta, double* diag,
                              double* scores, int* err, hipStream_t) {
    IN(work, band_work_doubles(m, B) * 8);
    IN(scores_in, d * 8);
    IN(scores, d * 8);
    IN(diag, d * 8);
    IN(theta, d * 4);
    IN(count, 4);
    IN(list, d * 4);
    IN(G, (int64_t)m * d * 4);
    IN(L32, ((d / B - 1) * lstride + (int64_t)mp * mp) * 4);
    IN(sc.hist, 1024);
    IN(err, 4);
    CHECK(tau > 0.0 && tau < 1e-3 && keep >= 0 && keep <= d && m <= 4096 && B <= 65536);
    return launched();
}
hipError_t launch_assemble(double* K, int m, const double* p, int pstride, int k, double, double* A, int mp, int* err,
                           hipStream_t) {
    IN(K, (int64_t)m * m * 8);
    if (k >= 0) IN(p, ((int64_t)(m - 1) * pstride + 1) * 8);
    IN(A, (int64_t)mp * mp * 8);
    IN(err, 4);
    return launched();
}
int64_t splitk_part_doubles(int mp) { return mp <= 128 ? 0 : (int64_t)512 * 128 * 128; }
hipError_t launch_factor_invert(double* A, double* Linv, int mp, int nbatch, int64_t bstride, int* err, hipStream_t,
                                double* part, int64_t part_elems) {
    IN(A, ((int64_t)(nbatch - 1) * bstride + (int64_t)mp * mp) * 8);
    IN(Linv, ((int64_t)(nbatch - 1) * bstride + (int64_t)mp * mp) * 8);
    IN(err, 4);
    if (part) IN(part, part_elems * 8);
    // one matrix (the refactor, the one-block precompute) brings room for its split-K segments
    if (nbatch == 1 && mp > 128) CHECK(part && part_elems >= splitk_part_doubles(mp));
    CHECK(mp % NB == 0);
    return launched();
}
hipError_t launch_factor_invert32(float* A, float* Linv, int mp, int nbatch, int64_t bstride, int* err, hipStream_t) {
    IN(A, ((int64_t)(nbatch - 1) * bstride + (int64_t)mp * mp) * 4);
    IN(Linv, ((int64_t)(nbatch - 1) * bstride + (int64_t)mp * mp) * 4);
    IN(err, 4);
    CHECK(mp % NB == 0);
    return launched();
}
hipError_t launch_lauum(const double* Linv, double* Ainv, int mp, int nbatch, int64_t bstride, hipStream_t) {
    IN(Linv, ((int64_t)(nbatch - 1) * bstride + (int64_t)mp * mp) * 8);
    IN(Ainv, ((int64_t)(nbatch - 1) * bstride + (int64_t)mp * mp) * 8);
    return launched();
}
hipError_t launch_inv_replace(double* K, int m, const double* p, int pstride, int k, double, double* Ainv, int mp,
                              double* z, double* v, int* err, hipStream_t) {
    IN(K, (int64_t)m * m * 8);
    IN(p, ((int64_t)(m - 1) * pstride + 1) * 8);
    IN(Ainv, (int64_t)mp * mp * 8);
    IN(z, (int64_t)mp * 8);
    IN(v, (int64_t)mp * 8);
    IN(err, 4);
    CHECK(k >= 0 && k < m);
    return launched();
}
hipError_t launch_inv_replace_coef(double* K, int m, const double* p, int pstride, int k, double, double* Ainv, int mp,
                                  double* z, double* v, const double* rhs, int rstride, int nv, int kc, double, double,
                                  double* coef, int* err, hipStream_t) {
    IN(K, (int64_t)m * m * 8);
    IN(p, ((int64_t)(m - 1) * pstride + 1) * 8);
    IN(Ainv, (int64_t)mp * mp * 8);
    IN(z, (int64_t)mp * 8);
    IN(v, (int64_t)mp * 8);
    IN(rhs, ((int64_t)(m - 1) * rstride + nv) * 8);
    IN(coef, (int64_t)m * nv * 8);
    IN(err, 4);
    CHECK(k >= 0 && k < m && kc < m && nv >= 1 && nv <= 17);
    return launched();
}
hipError_t launch_coef_from_inv(const double* Ainv, int mp, int m, const double* p, int pstride, int nv, int k, double,
                                double, double* coef, int* err, hipStream_t) {
    IN(Ainv, (int64_t)mp * mp * 8);
    IN(p, ((int64_t)(m - 1) * pstride + nv) * 8);
    IN(coef, (int64_t)m * nv * 8);
    IN(err, 4);
    CHECK(k < m);
    return launched();
}
hipError_t launch_trmm_diag(const double* Linv, int mp, int64_t bstride, float* G, int m, int64_t d, int B, int b0,
                            int nb, double, double* diag, hipStream_t) {
    IN(Linv, ((int64_t)(nb - 1) * bstride + (int64_t)mp * mp) * 8);
    IN(G, ((int64_t)(m - 1) * d + (int64_t)(b0 + nb) * B) * 4);
    IN(diag + (int64_t)b0 * B, (int64_t)nb * B * 8);
    return launched();
}
hipError_t launch_diag_to_f32(const double* diag, int64_t d, float* out, hipStream_t) {
    IN(diag, d * 8);
    IN(out, d * 4);
    return launched();
}
hipError_t launch_scores(const float* theta, const double* diag, int64_t d, double* s, int* err, hipStream_t) {
    IN(theta, d * 4);
    IN(diag, d * 8);
    IN(s, d * 8);
    IN(err, 4);
    return launched();
}
int64_t select_scratch_bytes(int64_t d) { return 2048 + ceil_div(d, 1024) * 4; }
SelectScratch select_scratch_carve(void* base, int64_t d) {
    SelectScratch s;
    s.hist = (unsigned int*)base;
    s.state = (unsigned long long*)((char*)base + 1024);
    s.chunk_cnt = (unsigned int*)((char*)base + 2048);
    s.nchunk = (int)ceil_div(d, 1024);
    return s;
}
hipError_t launch_topk_mask(const double* s, int64_t d, int64_t keep, SelectScratch sc, uint8_t* mask, hipStream_t) {
    IN(s, d * 8);
    IN(mask, d);
    IN(sc.hist, 1024);
    IN(sc.chunk_cnt, (int64_t)sc.nchunk * 4);
    CHECK(keep >= 0 && keep <= d);
    return launched();
}
int64_t static_query_part_doubles(int64_t d, int B, int m) { return (d / B) * m * 4 + d / 64; }
hipError_t launch_static_ihvp(const float* W, int m, int64_t d, int B, int n, const float* X, float, double, float* Y,
                              double* part, double* coef, hipStream_t) {
    IN(W, (int64_t)m * d * 4);
    IN(X, (int64_t)n * d * 4);
    IN(Y, (int64_t)n * d * 4);
    IN(part, static_query_part_doubles(d, B, m) * 8);
    IN(coef, (d / B) * m * 4 * 8);
    return launched();
}
hipError_t launch_obs_x(const float* theta, const uint8_t* keep, const double* diag, int64_t d, float* x, hipStream_t) {
    IN(theta, d * 4);
    IN(keep, d);
    IN(diag, d * 8);
    IN(x, d * 4);
    return launched();
}
hipError_t launch_static_element(const float* W, int m, int64_t d, int, int64_t nq, const int64_t* ij, double,
                                 double* out, int* err, hipStream_t) {
    IN(W, (int64_t)m * d * 4);
    if (nq > 0) {
        IN(ij, nq * 16);
        IN(out, nq * 8);
    }
    IN(err, 4);
    return launched();
}

}  // namespace mfac

// ------------------------------------------------------------------ the checks
namespace {

hipStream_t const ST = nullptr;

void check_rejections() {
    mfac_window w = nullptr;
    CHECK(mfac_window_init(nullptr, 4096, 16, 1e-3, 0, (void*)256, 1 << 30, (void*)512, 1 << 30, nullptr, ST) ==
          MFAC_EINVAL);
    CHECK(mfac_window_init(&w, 0, 16, 1e-3, 0, (void*)256, 1 << 30, (void*)512, 1 << 30, nullptr, ST) == MFAC_EINVAL);
    CHECK(w == nullptr);
    CHECK(mfac_window_replace(nullptr, -1, (float*)256, nullptr, 0, nullptr, nullptr) == MFAC_EINVAL);
    CHECK(mfac_ihvp(nullptr, 1, (float*)256, (float*)512) == MFAC_EINVAL);
    CHECK(mfac_ihvp_noalloc(nullptr, 1, (float*)256, (float*)512) == MFAC_EINVAL);
    CHECK(mfac_window_destroy(nullptr) == MFAC_OK);
    CHECK(mfac_static_destroy(nullptr) == MFAC_OK);
    // size queries at the edges of what is accepted (UBSan: no overflow)
    CHECK(mfac_window_storage_bytes(int64_t(1) << 34, 16384) > 0);
    CHECK(mfac_window_workspace_bytes(int64_t(1) << 34, 16384, 0) > 0);
    CHECK(mfac_window_workspace_bytes(int64_t(1) << 34, 1024, 16) == 0);
    CHECK(mfac_window_workspace_bytes(INT64_MAX, 1 << 30, 16) == 0);
    CHECK(mfac_static_workspace_bytes((int64_t(1) << 32) - 256, 64, 8192) > 0);
    CHECK(mfac_static_workspace_bytes(INT64_MAX, 1 << 30, 1 << 30) == 0);
    CHECK(mfac_static_paged_workspace_bytes((int64_t(1) << 32) - 256, 64, 8192, int64_t(64) * 65535) > 0);
    CHECK(mfac_static_paged_workspace_bytes((int64_t(1) << 32) - 256, 64, 8192, int64_t(64) * 65536) == 0);
    CHECK(mfac_static_paged_workspace_bytes((int64_t(1) << 32) - 256, 64, 8192, INT64_MAX & ~int64_t(3)) == 0);
    CHECK(mfac_static_paged_workspace_bytes(4096, 4096, 64, INT64_MAX & ~int64_t(3)) > 0);
    CHECK(mfac_static_paged_workspace_bytes(4096, 4096, 64, INT64_MAX) == 0);  // not a multiple of 4
    CHECK(strcmp(mfac_status_string((mfac_status)12345), "unknown status") == 0);
}

// A window through every entry point; returns the number of launches it made.
void drive_window(int64_t d, int m, int q) {
    fake_reset();
    const size_t sb = mfac_window_storage_bytes(d, m), wb = mfac_window_workspace_bytes(d, m, q);
    CHECK(sb > 0 && wb > 0);
    void* storage = fake_alloc(sb, "storage");
    void* ws = fake_alloc(wb, "workspace");
    float* G0 = (float*)fake_alloc((size_t)m * d * 4, "G0");
    float* g = (float*)fake_alloc((size_t)d * 4 + 16, "g");  // one case reads it from g + 1
    float* y = (float*)fake_alloc((size_t)d * 4, "y");
    float* X = (float*)fake_alloc((size_t)(q + 1) * d * 4, "X");
    float* Y = (float*)fake_alloc((size_t)(q + 1) * d * 4, "Y");
    float* Gn = (float*)fake_alloc((size_t)5 * d * 4, "Gn");
    float* Yn = (float*)fake_alloc((size_t)5 * d * 4, "Yn");
    mfac_window w = nullptr;
    // too small storage / workspace
    CHECK(mfac_window_init(&w, d, m, 1e-3, q, storage, sb - 1, ws, wb, G0, ST) == MFAC_EWORKSPACE);
    CHECK(mfac_window_init(&w, d, m, 1e-3, q, storage, sb, ws, wb - 1, G0, ST) == MFAC_EWORKSPACE);
    for (const float* init : {(const float*)nullptr, (const float*)G0}) {
        CHECK(mfac_window_init(&w, d, m, 1e-3, q, storage, sb, ws, wb, init, ST) == MFAC_OK);
        if (!w) return;
        CHECK(mfac_window_replace(w, -1, g, y, 0, nullptr, nullptr) == MFAC_OK);
        CHECK(mfac_window_replace(w, m - 1, g, nullptr, q, q ? X : nullptr, q ? Y : nullptr) == MFAC_OK);
        CHECK(mfac_window_replace(w, m, g, y, 0, nullptr, nullptr) == MFAC_EINVAL);
        CHECK(mfac_window_replace(w, -1, g, y, q + 1, X, Y) == MFAC_EINVAL);
        CHECK(mfac_window_replace(w, -1, g + 1, y, 0, nullptr, nullptr) == MFAC_OK);  // 4-byte aligned is accepted
        CHECK(mfac_window_replace(w, -1, (const float*)((char*)g + 2), y, 0, nullptr, nullptr) == MFAC_EINVAL);
        CHECK(mfac_window_replace_seq(w, 5, Gn, Yn) == MFAC_OK);
        CHECK(mfac_ihvp(w, q + 1, X, Y) == MFAC_OK);
        CHECK(mfac_ihvp(w, q + 2, X, Y) == MFAC_EINVAL);
        CHECK(mfac_ihvp_noalloc(w, 1, X, Y) == ((int64_t)m * 1 <= 4080 ? MFAC_OK : MFAC_EWORKSPACE));
        CHECK(mfac_window_set_rows(w, 0, m, G0) == MFAC_OK);
        CHECK(mfac_window_set_rows(w, 1, m, G0) == MFAC_EINVAL);
        CHECK(mfac_window_rebuild(w) == MFAC_OK);
        CHECK(mfac_window_get_rows(w, 0, m, G0) == MFAC_OK);
        int32_t head = -1;
        int64_t steps = -1;
        CHECK(mfac_window_info(w, &head, &steps) == MFAC_OK);
        CHECK(steps == 8 && head == (7 % m));
        CHECK(mfac_window_set_head(w, m, 0) == MFAC_EINVAL);
        CHECK(mfac_window_set_head(w, 0, 3) == MFAC_OK);
        CHECK(mfac_window_set_refactor_period(w, -1) == MFAC_EINVAL);
        for (int period : {0, 1, 3}) {
            CHECK(mfac_window_set_refactor_period(w, period) == MFAC_OK);
            for (int t = 0; t < 4; ++t) CHECK(mfac_window_replace(w, -1, g, y, 0, nullptr, nullptr) == MFAC_OK);
        }
        CHECK(mfac_window_trace(w, 1) == MFAC_OK);
        CHECK(mfac_window_replace(w, -1, g, y, q, q ? X : nullptr, q ? Y : nullptr) == MFAC_OK);
        CHECK(mfac_window_replace_seq(w, 3, Gn, Yn) == MFAC_OK);
        double ms[MFAC_NPHASES];
        int64_t cnt[MFAC_NPHASES];
        CHECK(mfac_window_trace_read(w, ms, cnt) == MFAC_OK);
        CHECK(cnt[0] >= 2 && cnt[1] >= 4 && cnt[2] >= 4 && cnt[3] >= 4);
        CHECK(mfac_window_replace(w, -1, g, y, 0, nullptr, nullptr) == MFAC_OK);  // marks left for destroy
        CHECK(mfac_window_set_stream(w, ST) == MFAC_OK);
        CHECK(mfac_window_status(w) == MFAC_OK);
        CHECK(mfac_window_destroy(w) == MFAC_OK);
        w = nullptr;
    }
    // a launch failure at every position of init (with G0) and of rebuild
    const long before = launches;
    mfac_window w0 = nullptr;
    CHECK(mfac_window_init(&w0, d, m, 1e-3, q, storage, sb, ws, wb, G0, ST) == MFAC_OK);
    const long n_init = launches - before;
    CHECK(mfac_window_destroy(w0) == MFAC_OK);
    for (long f = 1; f <= n_init; ++f) {
        fail_at = launches + f;
        mfac_window wf = nullptr;
        CHECK(mfac_window_init(&wf, d, m, 1e-3, q, storage, sb, ws, wb, G0, ST) == MFAC_EHIP);
        CHECK(wf == nullptr);
    }
    fail_at = -1;
    CHECK(mfac_window_init(&w0, d, m, 1e-3, q, storage, sb, ws, wb, nullptr, ST) == MFAC_OK);
    CHECK(mfac_window_trace(w0, 1) == MFAC_OK);
    fail_at = launches + 2;
    CHECK(mfac_window_replace(w0, -1, g, y, 0, nullptr, nullptr) == MFAC_EHIP);
    fail_at = -1;
    CHECK(mfac_window_destroy(w0) == MFAC_OK);
}

void drive_static(int64_t d, int B, int m, bool paged, bool fast = false) {
    fake_reset();
    mfac_static s0_unused = nullptr;
    const int64_t page = paged ? (B < d ? 2 * (int64_t)B : (d / 3 + 3) / 4 * 4) : 0;
    const uint32_t fl = fast ? MFAC_STATIC_FP32 : 0u;
    const size_t wb = paged ? mfac_static_paged_workspace_bytes(d, B, m, page)
                            : mfac_static_workspace_bytes_flags(d, B, m, fl);
    if (!paged) CHECK(mfac_static_workspace_bytes_flags(d, B, m, 0) == mfac_static_workspace_bytes(d, B, m));
    if (fast) CHECK(wb > (size_t)m * d * 4 + (size_t)(d / B) * m * m * 4);  // W and the per-block L^-1
    CHECK(wb > 0);
    void* ws = fake_alloc(wb, "workspace");
    float* G = (float*)fake_alloc((size_t)m * d * 4, paged ? "pinned" : "G");
    float* theta = (float*)fake_alloc((size_t)d * 4, "theta");
    float* diag = (float*)fake_alloc((size_t)d * 4, "diag");
    double* diag64 = (double*)fake_alloc((size_t)d * 8, "diag64");
    double* scores = (double*)fake_alloc((size_t)d * 8, "scores");
    uint8_t* mask = (uint8_t*)fake_alloc((size_t)d, "mask");
    float* X = (float*)fake_alloc((size_t)4 * d * 4, "X");
    float* Y = (float*)fake_alloc((size_t)4 * d * 4, "Y");
    int64_t* ij = (int64_t*)fake_alloc(64 * 16, "ij");
    double* out = (double*)fake_alloc(64 * 8, "out");
    auto make = [&](mfac_static* s, uint32_t flags) {
        return paged ? mfac_static_precompute_paged(s, d, B, m, 1e-4, G, page, ws, wb, flags, ST)
                     : mfac_static_precompute(s, d, B, m, 1e-4, G, ws, wb, flags | fl, ST);
    };
    if (paged) CHECK(mfac_static_precompute_paged(&s0_unused, d, B, m, 1e-4, G, page, ws, wb, MFAC_STATIC_FP32, ST) ==
                     MFAC_EINVAL);
    if (fast) CHECK(mfac_static_precompute(&s0_unused, d, B, m, 1e-4, G, ws, wb - 1, fl, ST) == MFAC_EWORKSPACE);
    mfac_static s = nullptr;
    for (uint32_t flags : {0u, (uint32_t)MFAC_STATIC_TRACE}) {
        const long before = launches;
        CHECK(make(&s, flags) == MFAC_OK);
        const long n_pre = launches - before;
        if (!s) return;
        CHECK(mfac_inv_diag(s, diag) == MFAC_OK);
        CHECK(mfac_inv_diag64(s, diag64) == MFAC_OK);
        CHECK(mfac_obs_mask(s, theta, d / 2, scores, mask) == MFAC_OK);
        CHECK(mfac_obs_mask(s, theta, d / 2, nullptr, mask) == MFAC_OK);
        CHECK(mfac_obs_mask(s, theta, d + 1, nullptr, mask) == MFAC_EINVAL);
        CHECK(mfac_static_ihvp(s, 4, X, Y) == MFAC_OK);
        CHECK(mfac_static_ihvp(s, 5, X, Y) == MFAC_EINVAL);
        CHECK(mfac_static_element(s, 64, ij, out) == MFAC_OK);
        CHECK(mfac_obs_update(s, theta, mask, Y) == MFAC_OK);
        double ms[MFAC_STATIC_NPHASES];
        int64_t cnt[MFAC_STATIC_NPHASES];
        CHECK(mfac_static_trace_read(s, ms, cnt) == MFAC_OK);
        CHECK(mfac_static_set_stream(s, ST) == MFAC_OK);
        CHECK(mfac_static_status(s) == MFAC_OK);
        CHECK(mfac_static_destroy(s) == MFAC_OK);
        s = nullptr;
        // a launch failure at every position of the precompute
        for (long f = 1; f <= n_pre; ++f) {
            fail_at = launches + f;
            mfac_static sf = nullptr;
            CHECK(make(&sf, flags) == MFAC_EHIP);
            CHECK(sf == nullptr);
        }
        fail_at = -1;
    }
    CHECK(mfac_static_precompute(&s, d, B, m, 1e-4, G, ws, wb, 6, ST) == MFAC_EINVAL);
}

}  // namespace

int main() {
    check_rejections();
    for (int q : {0, 3}) {
        drive_window(4096, 16, q);
        drive_window(3 * 2048 + 5, 70, q);
        drive_window(1000, 4081, 0);
    }
    drive_static(4096, 256, 64, false);
    drive_static(8192, 8192, 100, false);    // one wide block: split Gram
    drive_static(3000, 100, 300, false);     // m > B
    drive_static(8192, 1024, 64, true);      // paged, whole blocks per page
    drive_static(12000, 12000, 64, true);    // paged, one block over all pages
    drive_static(4096, 256, 64, false, true);     // fast mode
    drive_static(3000, 100, 300, false, true);    // fast mode, m > B
    drive_static(65536, 65536, 128, false, true); // fast mode, the widest block it accepts
    {
        mfac_static s = nullptr;
        CHECK(mfac_static_workspace_bytes_flags(4096, 256, 4097, MFAC_STATIC_FP32) == 0);     // m past the fast limit
        CHECK(mfac_static_workspace_bytes_flags(131072, 131072, 64, MFAC_STATIC_FP32) == 0);  // block past it
        CHECK(mfac_static_workspace_bytes_flags(4096, 256, 64, 4u) == 0);                     // unknown flag
        CHECK(mfac_static_precompute(&s, 4096, 256, 4097, 1e-4, (float*)256, (void*)512, size_t(1) << 40,
                                     MFAC_STATIC_FP32, ST) == MFAC_EINVAL);
    }
    CHECK(streams_live == 0);
    CHECK(events_live == 0);
    if (failures) {
        fprintf(stderr, "host check: %d failure(s)\n", failures);
        return 1;
    }
    printf("host check ok (%ld launches)\n", launches);
    return 0;
}
