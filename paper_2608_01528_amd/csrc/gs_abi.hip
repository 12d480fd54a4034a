// C-ABI entry points of the Gram-Space library: argument validation, error
// reporting and dispatch to the kernels.  Every check runs on the host before
// any HIP call, so a rejected call touches neither the device nor its outputs.
#include <atomic>
#include <mutex>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <string>
#include <algorithm>
#include <vector>

#include "gs_internal.h"

using namespace gs;

namespace {

thread_local std::string g_err;

// GS_LOG set (to anything but "0"): one line on stderr per rejected call
// (its status and message) and per launched call (its name).
bool logging() {
    static const bool on = [] {
        const char *v = getenv("GS_LOG");
        return v && *v && !(v[0] == '0' && v[1] == 0);
    }();
    return on;
}

gs_status fail(gs_status st, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    if (logging()) fprintf(stderr, "[gramspace] status %d: %s\n", (int)st, buf);
    return st;
}

gs_status ok() {
    g_err.clear();
    return GS_OK;
}

size_t esize(gs_dtype t) { return t == GS_F64 ? 8 : (t == GS_F32 ? 4 : 2); }
bool valid_dtype(int t) { return t == GS_F32 || t == GS_BF16 || t == GS_F64; }
const char *dname(gs_dtype t) { return t == GS_F32 ? "f32" : (t == GS_BF16 ? "bf16" : "f64"); }

// Byte range occupied by a rows x cols matrix with leading dimension ld.
struct Span {
    const char *lo = nullptr, *hi = nullptr;
    const char *name = "";
};

Span span(const void *p, int64_t rows, int64_t cols, int64_t ld, size_t es, const char *name) {
    Span s;
    s.name = name;
    if (!p || rows <= 0 || cols <= 0) return s;
    s.lo = static_cast<const char *>(p);
    s.hi = s.lo + ((rows - 1) * ld + cols) * (int64_t)es;
    return s;
}

bool overlap(const Span &a, const Span &b) {
    return a.lo && b.lo && a.lo < b.hi && b.lo < a.hi;
}

// Outputs must overlap neither inputs nor each other.
gs_status check_overlaps(const std::vector<Span> &in, const std::vector<Span> &out) {
    for (size_t a = 0; a < out.size(); ++a) {
        for (const Span &i : in)
            if (overlap(out[a], i)) return fail(GS_ERR_ARG, "output %s overlaps input %s", out[a].name, i.name);
        for (size_t b = a + 1; b < out.size(); ++b)
            if (overlap(out[a], out[b]))
                return fail(GS_ERR_ARG, "outputs %s and %s overlap", out[a].name, out[b].name);
    }
    return GS_OK;
}

gs_status check_aligned(const void *p, size_t es, const char *name) {
    if (p && (reinterpret_cast<uintptr_t>(p) % es) != 0)
        return fail(GS_ERR_ALIGN, "%s is not aligned to its %zu-byte element", name, es);
    return GS_OK;
}

#define GS_CHECK(x) do { gs_status s_ = (x); if (s_ != GS_OK) return s_; } while (0)

gs_status check_matrix(const void *p, const char *name, int64_t rows, int64_t cols, int64_t ld,
                       gs_dtype t, bool nullable) {
    if (!p) {
        // an empty batch may come without storage
        if (nullable || rows == 0) return GS_OK;
        return fail(GS_ERR_ARG, "%s is null", name);
    }
    if (ld < cols) return fail(GS_ERR_SHAPE, "leading dimension of %s (%lld) is smaller than its %lld columns",
                                name, (long long)ld, (long long)cols);
    return check_aligned(p, esize(t), name);
}

gs_status check_device() {
    static std::atomic<int> state{-1};   // -1 unknown, 0 none, 1 ok
    int s = state.load();
    if (s < 0) {
        int n = 0;
        hipError_t e = hipGetDeviceCount(&n);
        s = (e == hipSuccess && n > 0) ? 1 : 0;
        state.store(s);
    }
    if (!s) return fail(GS_ERR_DEVICE, "no HIP device is available");
    return GS_OK;
}

gs_status launched(hipError_t e, const char *what) {
    if (e != hipSuccess) return fail(GS_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
    if (logging()) fprintf(stderr, "[gramspace] %s: launched\n", what);
    if (getenv("GS_DEBUG")) {
        hipError_t e2 = hipDeviceSynchronize();
        if (e2 != hipSuccess) return fail(GS_ERR_DEVICE, "%s (GS_DEBUG sync): %s", what, hipGetErrorString(e2));
    }
    return ok();
}

bool is_batch_type(gs_dtype t) { return t == GS_F32 || t == GS_BF16; }

}  // namespace

extern "C" {

int gs_abi_version(void) { return GS_ABI_VERSION; }

const char *gs_last_error(void) { return g_err.c_str(); }

size_t gs_compress_workspace(int64_t M, int64_t D) {
    if (M < 1 || D < 1 || M > D) return 0;
    return compress_workspace(M, D);
}

}  // extern "C"

namespace {

// Checks shared by gs_compress and gs_compress_noalloc (everything but the
// workspace).
gs_status check_compress(const char *fn, const void *C, gs_dtype ct, int64_t M, int64_t D, int64_t ldc,
                         double tol, void *Q, gs_dtype qt, int64_t ldq, void *R, gs_dtype rt, int64_t ldr,
                         int32_t *kept, float *cnorm, int32_t *rank, const Span &ws_span) {
    if (!valid_dtype(ct) || !valid_dtype(qt) || !valid_dtype(rt))
        return fail(GS_ERR_DTYPE, "%s: unknown element type", fn);
    if (!rank) return fail(GS_ERR_ARG, "%s: rank (host) is null", fn);
    if (M < 1 || D < 1) return fail(GS_ERR_SHAPE, "%s: M and D must be >= 1 (M=%lld, D=%lld)", fn,
                                    (long long)M, (long long)D);
    if (M > D) return fail(GS_ERR_SHAPE, "%s: M=%lld > D=%lld needs partitioned bases (gs_compress_partitioned)",
                           fn, (long long)M, (long long)D);
    if (!(tol >= 0.0 && tol < 1.0)) return fail(GS_ERR_ARG, "%s: tol must be in [0, 1)", fn);
    GS_CHECK(check_matrix(C, "C", M, D, ldc, ct, false));
    GS_CHECK(check_matrix(Q, "Q", M, D, ldq, qt, false));
    GS_CHECK(check_matrix(R, "R", M, M, ldr, rt, false));
    GS_CHECK(check_aligned(kept, 4, "kept"));
    GS_CHECK(check_aligned(cnorm, 4, "cnorm"));
    const Span sC = span(C, M, D, ldc, esize(ct), "C");
    GS_CHECK(check_overlaps({sC, ws_span}, {span(Q, M, D, ldq, esize(qt), "Q"), span(R, M, M, ldr, esize(rt), "R"),
                                           span(kept, 1, M, M, 4, "kept"), span(cnorm, 1, M, M, 4, "cnorm")}));
    return GS_OK;
}

gs_status finish_compress(const char *fn, hipError_t e, int nonfinite, int32_t r, int32_t *rank) {
    if (e != hipSuccess) return fail(GS_ERR_DEVICE, "%s: %s", fn, hipGetErrorString(e));
    if (nonfinite & 1) return fail(GS_ERR_NUMERIC, "%s: codebook holds a NaN or infinity", fn);
    if (nonfinite) return fail(GS_ERR_NUMERIC, "%s: the orthogonalisation broke down", fn);
    *rank = r;
    return ok();
}

// Scratch memory of gs_compress_noalloc: one array per GPU, held by the
// loaded code object until the process ends.  Host code never uses the
// array's name as an address: its device address is looked up once per
// device (with that device current) and kept in scratch_ptr.
constexpr size_t kScratchBytes = (size_t)GS_NOALLOC_SCRATCH_BYTES;
__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

gs_status scratch_for_current_device(void **out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(GS_ERR_DEVICE, "gs_compress_noalloc: hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxDevices)
        return fail(GS_ERR_DEVICE, "gs_compress_noalloc: device %d beyond the %d supported", dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(GS_ERR_DEVICE, "gs_compress_noalloc: hipGetSymbolAddress: %s", hipGetErrorString(e));
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return GS_OK;
}

// The second stream of the allocating compression calls: one per GPU,
// created on first use with that device current and kept until the process
// ends, shared by every call on the GPU (its work is ordered against each
// call's own stream by that call's events).  gs_compress_noalloc does not use
// it: creating a stream or an event can allocate.
std::mutex g_aux_mu;
hipStream_t g_aux_stream[kMaxDevices] = {};
bool g_aux_made[kMaxDevices] = {};

class OverlapScope {
public:
    // Sets up ov for the current device; a failure is reported as an error.
    gs_status open(const char *fn) {
        int dev = -1;
        hipError_t e = hipGetDevice(&dev);
        if (e != hipSuccess) return fail(GS_ERR_DEVICE, "%s: hipGetDevice: %s", fn, hipGetErrorString(e));
        if (dev < 0 || dev >= kMaxDevices)
            return fail(GS_ERR_DEVICE, "%s: device %d beyond the %d supported", fn, dev, kMaxDevices);
        {
            std::lock_guard<std::mutex> lock(g_aux_mu);
            if (!g_aux_made[dev]) {
                hipStream_t st = nullptr;
                e = hipStreamCreateWithFlags(&st, hipStreamNonBlocking);
                if (e != hipSuccess)
                    return fail(GS_ERR_DEVICE, "%s: hipStreamCreateWithFlags: %s", fn, hipGetErrorString(e));
                g_aux_stream[dev] = st;
                g_aux_made[dev] = true;
            }
            ov_.aux = g_aux_stream[dev];
        }
        e = hipEventCreateWithFlags(&ov_.fork, hipEventDisableTiming);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&ov_.join, hipEventDisableTiming);
        if (e != hipSuccess) return fail(GS_ERR_DEVICE, "%s: hipEventCreateWithFlags: %s", fn, hipGetErrorString(e));
        return GS_OK;
    }
    const gs::CompressOverlap *get() const { return &ov_; }
    ~OverlapScope() {
        if (ov_.fork) (void)hipEventDestroy(ov_.fork);
        if (ov_.join) (void)hipEventDestroy(ov_.join);
    }

private:
    gs::CompressOverlap ov_{nullptr, nullptr, nullptr};
};

}  // namespace

extern "C" {

gs_status gs_compress(const void *C, gs_dtype ct, int64_t M, int64_t D, int64_t ldc, double tol,
                      void *Q, gs_dtype qt, int64_t ldq, void *R, gs_dtype rt, int64_t ldr,
                      int32_t *kept, float *cnorm, int32_t *rank, void *ws, size_t ws_bytes,
                      void *stream) {
    GS_CHECK(check_compress("gs_compress", C, ct, M, D, ldc, tol, Q, qt, ldq, R, rt, ldr, kept, cnorm, rank,
                            Span{}));
    if (!ws) return fail(GS_ERR_WORKSPACE, "gs_compress: workspace is null");
    if ((reinterpret_cast<uintptr_t>(ws) & 255u) != 0)
        return fail(GS_ERR_ALIGN, "gs_compress: workspace must be 256-byte aligned");
    const size_t need = compress_workspace(M, D);
    if (ws_bytes < need)
        return fail(GS_ERR_WORKSPACE, "gs_compress: workspace of %zu bytes, %zu needed", ws_bytes, need);
    {
        // the workspace overlaps neither the codebook nor an output
        const Span sW = span(ws, 1, (int64_t)need, (int64_t)need, 1, "workspace");
        GS_CHECK(check_overlaps({sW}, {span(C, M, D, ldc, esize(ct), "C"), span(Q, M, D, ldq, esize(qt), "Q"),
                                       span(R, M, M, ldr, esize(rt), "R"), span(kept, 1, M, M, 4, "kept"),
                                       span(cnorm, 1, M, M, 4, "cnorm")}));
    }
    GS_CHECK(check_device());
    OverlapScope ovs;
    GS_CHECK(ovs.open("gs_compress"));
    int nonfinite = 0;
    int32_t r = 0;
    hipError_t e = run_compress(C, ct, M, D, ldc, tol, Q, qt, ldq, R, rt, ldr, kept, cnorm, &r,
                                &nonfinite, ws, (hipStream_t)stream, 0, ovs.get());
    return finish_compress("gs_compress", e, nonfinite, r, rank);
}

gs_status gs_compress_partitioned(const void *C, gs_dtype ct, int64_t M, int64_t D, int64_t ldc, double tol,
                                  int64_t subset, void *Q, gs_dtype qt, int64_t ldq, void *R, gs_dtype rt,
                                  int64_t ldr, int32_t *kept, float *cnorm, int32_t *ranks, int32_t *rank,
                                  void *ws, size_t ws_bytes, void *stream) {
    const char *fn = "gs_compress_partitioned";
    if (!valid_dtype(ct) || !valid_dtype(qt) || !valid_dtype(rt))
        return fail(GS_ERR_DTYPE, "%s: unknown element type", fn);
    if (!rank || !ranks) return fail(GS_ERR_ARG, "%s: rank or ranks (host) is null", fn);
    if (M < 1 || D < 1) return fail(GS_ERR_SHAPE, "%s: M and D must be >= 1", fn);
    if (subset < 1 || subset > D)
        return fail(GS_ERR_SHAPE, "%s: subset must be in [1, D] (subset=%lld, D=%lld)", fn, (long long)subset,
                    (long long)D);
    if (!(tol >= 0.0 && tol < 1.0)) return fail(GS_ERR_ARG, "%s: tol must be in [0, 1)", fn);
    GS_CHECK(check_matrix(C, "C", M, D, ldc, ct, false));
    GS_CHECK(check_matrix(Q, "Q", M, D, ldq, qt, false));
    GS_CHECK(check_matrix(R, "R", M, M, ldr, rt, false));
    GS_CHECK(check_aligned(kept, 4, "kept"));
    GS_CHECK(check_aligned(cnorm, 4, "cnorm"));
    GS_CHECK(check_overlaps({span(C, M, D, ldc, esize(ct), "C")},
                            {span(Q, M, D, ldq, esize(qt), "Q"), span(R, M, M, ldr, esize(rt), "R"),
                             span(kept, 1, M, M, 4, "kept"), span(cnorm, 1, M, M, 4, "cnorm")}));
    const int64_t ms = subset < M ? subset : M;
    if (!ws) return fail(GS_ERR_WORKSPACE, "%s: workspace is null", fn);
    if ((reinterpret_cast<uintptr_t>(ws) & 255u) != 0)
        return fail(GS_ERR_ALIGN, "%s: workspace must be 256-byte aligned", fn);
    const size_t need = compress_workspace(ms, D);
    if (ws_bytes < need) return fail(GS_ERR_WORKSPACE, "%s: workspace of %zu bytes, %zu needed", fn, ws_bytes, need);
    {
        const Span sW = span(ws, 1, (int64_t)need, (int64_t)need, 1, "workspace");
        GS_CHECK(check_overlaps({sW}, {span(C, M, D, ldc, esize(ct), "C"), span(Q, M, D, ldq, esize(qt), "Q"),
                                       span(R, M, M, ldr, esize(rt), "R"), span(kept, 1, M, M, 4, "kept"),
                                       span(cnorm, 1, M, M, 4, "cnorm")}));
    }
    GS_CHECK(check_device());
    OverlapScope ovs;
    GS_CHECK(ovs.open(fn));
    int nonfinite = 0;
    int32_t total = 0;
    hipError_t e = run_compress_partitioned(C, ct, M, D, ldc, tol, subset, Q, qt, ldq, R, rt, ldr, kept, cnorm,
                                            ranks, &total, &nonfinite, ws, (hipStream_t)stream, ovs.get());
    return finish_compress(fn, e, nonfinite, total, rank);
}

size_t gs_compress_padded_workspace(int64_t M, int64_t D, int64_t k) {
    if (M < 1 || D < 1 || k < M || M + k > D) return 0;
    return compress_padded_workspace(M, D, k);
}

gs_status gs_compress_padded(const void *C, gs_dtype ct, int64_t M, int64_t D, int64_t ldc, double tol,
                             int64_t k, const double *H, int64_t ldh, void *Q, gs_dtype qt, int64_t ldq,
                             void *R, gs_dtype rt, int64_t ldr, int32_t *kept, float *cnorm, int32_t *rank,
                             void *ws, size_t ws_bytes, void *stream) {
    const char *fn = "gs_compress_padded";
    if (!valid_dtype(ct) || !valid_dtype(qt) || !valid_dtype(rt))
        return fail(GS_ERR_DTYPE, "%s: unknown element type", fn);
    if (!rank) return fail(GS_ERR_ARG, "%s: rank (host) is null", fn);
    if (M < 1 || D < 1) return fail(GS_ERR_SHAPE, "%s: M and D must be >= 1", fn);
    if (k < M || M + k > D)
        return fail(GS_ERR_SHAPE, "%s: need M <= k and M + k <= D (M=%lld, k=%lld, D=%lld)", fn, (long long)M,
                    (long long)k, (long long)D);
    if (!(tol >= 0.0 && tol < 1.0)) return fail(GS_ERR_ARG, "%s: tol must be in [0, 1)", fn);
    GS_CHECK(check_matrix(C, "C", M, D, ldc, ct, false));
    GS_CHECK(check_matrix(H, "H", k, k, ldh, GS_F64, true));
    GS_CHECK(check_matrix(Q, "Q", k, D, ldq, qt, false));
    GS_CHECK(check_matrix(R, "R", M, k, ldr, rt, false));
    GS_CHECK(check_aligned(kept, 4, "kept"));
    GS_CHECK(check_aligned(cnorm, 4, "cnorm"));
    GS_CHECK(check_overlaps({span(C, M, D, ldc, esize(ct), "C"), span(H, k, k, ldh, 8, "H")},
                            {span(Q, k, D, ldq, esize(qt), "Q"), span(R, M, k, ldr, esize(rt), "R"),
                             span(kept, 1, M, M, 4, "kept"), span(cnorm, 1, M, M, 4, "cnorm")}));
    if (!ws) return fail(GS_ERR_WORKSPACE, "%s: workspace is null", fn);
    if ((reinterpret_cast<uintptr_t>(ws) & 255u) != 0)
        return fail(GS_ERR_ALIGN, "%s: workspace must be 256-byte aligned", fn);
    const size_t need = compress_padded_workspace(M, D, k);
    if (ws_bytes < need) return fail(GS_ERR_WORKSPACE, "%s: workspace of %zu bytes, %zu needed", fn, ws_bytes, need);
    {
        const Span sW = span(ws, 1, (int64_t)need, (int64_t)need, 1, "workspace");
        GS_CHECK(check_overlaps({sW}, {span(C, M, D, ldc, esize(ct), "C"), span(H, k, k, ldh, 8, "H"),
                                       span(Q, k, D, ldq, esize(qt), "Q"), span(R, M, k, ldr, esize(rt), "R"),
                                       span(kept, 1, M, M, 4, "kept"), span(cnorm, 1, M, M, 4, "cnorm")}));
    }
    GS_CHECK(check_device());
    OverlapScope ovs;
    GS_CHECK(ovs.open(fn));
    int nonfinite = 0;
    int32_t r = 0;
    hipError_t e = run_compress_padded(C, ct, M, D, ldc, tol, k, H, ldh, Q, qt, ldq, R, rt, ldr, kept, cnorm, &r,
                                       &nonfinite, ws, (hipStream_t)stream, ovs.get());
    return finish_compress(fn, e, nonfinite, r, rank);
}

gs_status gs_compress_noalloc(const void *C, gs_dtype ct, int64_t M, int64_t D, int64_t ldc, double tol,
                              void *Q, gs_dtype qt, int64_t ldq, void *R, gs_dtype rt, int64_t ldr,
                              int32_t *kept, float *cnorm, int32_t *rank, void *stream) {
    GS_CHECK(check_compress("gs_compress_noalloc", C, ct, M, D, ldc, tol, Q, qt, ldq, R, rt, ldr, kept, cnorm,
                            rank, Span{}));
    const size_t need = compress_workspace(M, D);
    if (need > kScratchBytes)
        return fail(GS_ERR_WORKSPACE, "gs_compress_noalloc: a %lld x %lld codebook needs %zu bytes of scratch, "
                    "beyond the %zu of the library's static array (use gs_compress with a workspace)",
                    (long long)M, (long long)D, need, kScratchBytes);
    GS_CHECK(check_device());
    void *ws = nullptr;
    GS_CHECK(scratch_for_current_device(&ws));
    int nonfinite = 0;
    int32_t r = 0;
    hipError_t e = run_compress(C, ct, M, D, ldc, tol, Q, qt, ldq, R, rt, ldr, kept, cnorm, &r,
                                &nonfinite, ws, (hipStream_t)stream);
    return finish_compress("gs_compress_noalloc", e, nonfinite, r, rank);
}

gs_status gs_project(const void *X, gs_dtype xt, int64_t B, int64_t D, int64_t ldx,
                     const void *Q, gs_dtype qt, int64_t r, int64_t ldq,
                     void *T, gs_dtype tt, int64_t ldt, float *xnorm2, void *stream) {
    if (!is_batch_type(xt) || qt != xt || !is_batch_type(tt))
        return fail(GS_ERR_DTYPE, "gs_project: X/Q must be both f32 or both bf16 and T f32 or bf16 (got %s/%s/%s)",
                    dname(xt), dname(qt), valid_dtype(tt) ? dname(tt) : "?");
    if (B < 0 || D < 1 || r < 1) return fail(GS_ERR_SHAPE, "gs_project: need B >= 0, D >= 1, r >= 1");
    GS_CHECK(check_matrix(X, "X", B, D, ldx, xt, false));
    GS_CHECK(check_matrix(Q, "Q", r, D, ldq, qt, false));
    GS_CHECK(check_matrix(T, "T", B, r, ldt, tt, false));
    GS_CHECK(check_aligned(xnorm2, 4, "xnorm2"));
    GS_CHECK(check_overlaps({span(X, B, D, ldx, esize(xt), "X"), span(Q, r, D, ldq, esize(qt), "Q")},
                            {span(T, B, r, ldt, esize(tt), "T"), span(xnorm2, 1, B, B, 4, "xnorm2")}));
    if (B == 0) return ok();
    GS_CHECK(check_device());
    GemmArgs a{};
    a.A = X; a.lda = ldx; a.B = Q; a.ldb = ldq; a.C = T; a.ldc = ldt;
    a.M = B; a.N = r; a.K = D; a.rownorm2 = xnorm2;
    return launched(launch_gemm(xt, qt, tt, false, EPI_STORE, a, (hipStream_t)stream), "gs_project");
}

// Element type of a codebook-coordinate argument without the GS_ECHELON flag.
static gs_dtype coord_type(gs_dtype rt, bool *echelon) {
    *echelon = ((int)rt & GS_ECHELON) != 0;
    return (gs_dtype)((int)rt & ~GS_ECHELON);
}

gs_status gs_prob2vec(const void *P, gs_dtype pt, int64_t B, int64_t M, int64_t ldp,
                      const void *R, gs_dtype rt_in, int64_t r, int64_t ldr,
                      void *T, gs_dtype tt, int64_t ldt, void *stream) {
    bool ech;
    const gs_dtype rt = coord_type(rt_in, &ech);
    if (!is_batch_type(pt) || rt != pt || !is_batch_type(tt))
        return fail(GS_ERR_DTYPE, "gs_prob2vec: P/R must be both f32 or both bf16 and T f32 or bf16");
    if (B < 0 || M < 1 || r < 1) return fail(GS_ERR_SHAPE, "gs_prob2vec: need B >= 0, M >= 1 and r >= 1");
    GS_CHECK(check_matrix(P, "P", B, M, ldp, pt, false));
    GS_CHECK(check_matrix(R, "R", M, r, ldr, rt, false));
    GS_CHECK(check_matrix(T, "T", B, r, ldt, tt, false));
    GS_CHECK(check_overlaps({span(P, B, M, ldp, esize(pt), "P"), span(R, M, r, ldr, esize(rt), "R")},
                            {span(T, B, r, ldt, esize(tt), "T")}));
    if (B == 0) return ok();
    GS_CHECK(check_device());
    // small-codebook kernel for r <= M <= 64 (the codebook block is padded
    // to M's size); more coordinates than entries (a padded basis) and larger
    // codebooks take the matrix-core product
    if (M <= SMALL_MAX && r <= M) {
        SmallArgs a{};
        a.In = P; a.ldin = ldp; a.R = R; a.ldr = ldr; a.B = B; a.M = M; a.r = r; a.Out = T; a.ldout = ldt;
        return launched(launch_small_prob2vec(pt, tt, a, (hipStream_t)stream), "gs_prob2vec");
    }
    GemmArgs a{};
    a.A = P; a.lda = ldp; a.B = R; a.ldb = ldr; a.C = T; a.ldc = ldt; a.M = B; a.N = r; a.K = M;
    a.echelon = ech;
    return launched(launch_gemm(pt, rt, tt, true, EPI_STORE, a, (hipStream_t)stream), "gs_prob2vec");
}

gs_status gs_prob2vec_sparse(const int64_t *rowptr, const int32_t *cols, const void *vals, gs_dtype vt,
                             int64_t B, int64_t M, int64_t nnz,
                             const void *R, gs_dtype rt_in, int64_t r, int64_t ldr,
                             void *T, gs_dtype tt, int64_t ldt, void *stream) {
    bool ech;
    const gs_dtype rt = coord_type(rt_in, &ech);
    if (!is_batch_type(vt) || rt != vt || !is_batch_type(tt))
        return fail(GS_ERR_DTYPE, "gs_prob2vec_sparse: values/R must be both f32 or both bf16 and T f32 or bf16");
    if (B < 0 || M < 1 || r < 1 || nnz < 0)
        return fail(GS_ERR_SHAPE, "gs_prob2vec_sparse: need B >= 0, M >= 1, r >= 1 and nnz >= 0");
    if (B > 0 && !rowptr) return fail(GS_ERR_ARG, "gs_prob2vec_sparse: rowptr is null");
    if (nnz > 0 && (!cols || !vals)) return fail(GS_ERR_ARG, "gs_prob2vec_sparse: cols or vals is null");
    GS_CHECK(check_aligned(rowptr, 8, "rowptr"));
    GS_CHECK(check_aligned(cols, 4, "cols"));
    GS_CHECK(check_aligned(vals, esize(vt), "vals"));
    GS_CHECK(check_matrix(R, "R", M, r, ldr, rt, false));
    GS_CHECK(check_matrix(T, "T", B, r, ldt, tt, false));
    GS_CHECK(check_overlaps({span(rowptr, 1, B > 0 ? B + 1 : 0, B + 1, 8, "rowptr"),
                             span(cols, 1, nnz, nnz, 4, "cols"), span(vals, 1, nnz, nnz, esize(vt), "vals"),
                             span(R, M, r, ldr, esize(rt), "R")},
                            {span(T, B, r, ldt, esize(tt), "T")}));
    if (B == 0) return ok();
    GS_CHECK(check_device());
    SparseArgs a{};
    a.rowptr = rowptr; a.cols = cols; a.vals = vals; a.B = B; a.M = M; a.nnz = nnz;
    a.R = R; a.ldr = ldr; a.r = r; a.T = T; a.ldt = ldt;
    return launched(launch_sparse_prob2vec(vt, tt, a, (hipStream_t)stream), "gs_prob2vec_sparse");
}

static gs_status check_sim_common(const char *fn, const void *T, gs_dtype tt, int64_t B, int64_t r,
                                  int64_t ldt, const void *R, gs_dtype rt, int64_t M, int64_t ldr,
                                  const float *qnorm2, const float *cnorm, int mode) {
    if (!is_batch_type(tt) || rt != tt)
        return fail(GS_ERR_DTYPE, "%s: T/R must be both f32 or both bf16", fn);
    if (mode != GS_SIM_DOT && mode != GS_SIM_COSINE) return fail(GS_ERR_ARG, "%s: unknown similarity mode", fn);
    if (B < 0 || M < 1 || r < 1) return fail(GS_ERR_SHAPE, "%s: need B >= 0, M >= 1 and r >= 1", fn);
    GS_CHECK(check_matrix(T, "T", B, r, ldt, tt, false));
    GS_CHECK(check_matrix(R, "R", M, r, ldr, rt, false));
    GS_CHECK(check_aligned(qnorm2, 4, "qnorm2"));
    GS_CHECK(check_aligned(cnorm, 4, "cnorm"));
    return GS_OK;
}

gs_status gs_similarity(const void *T, gs_dtype tt, int64_t B, int64_t r, int64_t ldt,
                        const void *R, gs_dtype rt_in, int64_t M, int64_t ldr,
                        const float *qnorm2, const float *cnorm, gs_sim_mode mode, float scale,
                        float *S, int64_t lds, int32_t *argmax, void *stream) {
    bool ech;
    const gs_dtype rt = coord_type(rt_in, &ech);
    GS_CHECK(check_sim_common("gs_similarity", T, tt, B, r, ldt, R, rt, M, ldr, qnorm2, cnorm, mode));
    if (!S && !argmax && B > 0) return fail(GS_ERR_ARG, "gs_similarity: S and argmax are both null");
    GS_CHECK(check_matrix(S, "S", B, M, lds, GS_F32, true));
    GS_CHECK(check_aligned(argmax, 4, "argmax"));
    GS_CHECK(check_overlaps({span(T, B, r, ldt, esize(tt), "T"), span(R, M, r, ldr, esize(rt), "R"),
                             span(qnorm2, 1, B, B, 4, "qnorm2"), span(cnorm, 1, M, M, 4, "cnorm")},
                            {span(S, B, M, lds, 4, "S"), span(argmax, 1, B, B, 4, "argmax")}));
    if (B == 0) return ok();
    GS_CHECK(check_device());
    // small-codebook kernels (one thread per row of r <= M <= 64), unless a
    // few rows write their scores: those split the K reduction over work-groups
    if (M <= SMALL_MAX && r <= M && !(B <= FEW_ROWS && S)) {
        SmallArgs a{};
        a.In = T; a.ldin = ldt; a.R = R; a.ldr = ldr; a.B = B; a.M = M; a.r = r; a.Out = S; a.ldout = lds;
        a.qnorm2 = qnorm2; a.cnorm = cnorm; a.cosine = mode == GS_SIM_COSINE; a.scale = scale; a.argmax = argmax;
        return launched(launch_small_similarity(tt, a, (hipStream_t)stream), "gs_similarity");
    }
    GemmArgs a{};
    a.A = T; a.lda = ldt; a.B = R; a.ldb = ldr; a.C = S; a.ldc = lds; a.M = B; a.N = M; a.K = r;
    a.qnorm2 = qnorm2; a.cnorm = cnorm; a.cosine = mode == GS_SIM_COSINE; a.scale = scale;
    a.argmax = argmax; a.write_out = S != nullptr; a.echelon = ech;
    return launched(launch_gemm(tt, rt, GS_F32, false, EPI_SIM, a, (hipStream_t)stream), "gs_similarity");
}

gs_status gs_attention(const void *T, gs_dtype tt, int64_t B, int64_t r, int64_t ldt,
                       const void *R, gs_dtype rt_in, int64_t M, int64_t ldr,
                       const float *qnorm2, const float *cnorm, gs_sim_mode mode, float scale,
                       float beta, float *A, int64_t lda, void *O, gs_dtype ot, int64_t ldo,
                       void *stream) {
    bool ech;
    const gs_dtype rt = coord_type(rt_in, &ech);
    GS_CHECK(check_sim_common("gs_attention", T, tt, B, r, ldt, R, rt, M, ldr, qnorm2, cnorm, mode));
    GS_CHECK(check_matrix(A, "A", B, M, lda, GS_F32, false));
    if (O && !is_batch_type(ot)) return fail(GS_ERR_DTYPE, "gs_attention: O must be f32 or bf16");
    if (O) GS_CHECK(check_matrix(O, "O", B, r, ldo, ot, false));
    GS_CHECK(check_overlaps({span(T, B, r, ldt, esize(tt), "T"), span(R, M, r, ldr, esize(rt), "R"),
                             span(qnorm2, 1, B, B, 4, "qnorm2"), span(cnorm, 1, M, M, 4, "cnorm")},
                            {span(A, B, M, lda, 4, "A"), span(O, B, r, ldo, O ? esize(ot) : 1, "O")}));
    if (B == 0) return ok();
    GS_CHECK(check_device());
    hipStream_t s = (hipStream_t)stream;
    if (M <= SMALL_MAX && r <= M && B > FEW_ROWS) {   // small-codebook kernels, as in gs_similarity
        SmallArgs a{};
        a.In = T; a.ldin = ldt; a.R = R; a.ldr = ldr; a.B = B; a.M = M; a.r = r; a.Out = A; a.ldout = lda;
        a.O = O; a.ldo = ldo; a.qnorm2 = qnorm2; a.cnorm = cnorm; a.cosine = mode == GS_SIM_COSINE;
        a.scale = scale; a.beta = beta;
        return launched(launch_small_attention(tt, O ? ot : GS_F32, a, s), "gs_attention");
    }
    GemmArgs a{};
    a.A = T; a.lda = ldt; a.B = R; a.ldb = ldr; a.C = A; a.ldc = lda; a.M = B; a.N = M; a.K = r;
    a.qnorm2 = qnorm2; a.cnorm = cnorm; a.cosine = mode == GS_SIM_COSINE; a.scale = scale; a.beta = beta;
    a.echelon = ech;
    gs_status st = launched(launch_gemm(tt, rt, GS_F32, false, EPI_SOFTMAX, a, s), "gs_attention");
    if (st != GS_OK || !O) return st;
    GemmArgs o{};
    o.A = A; o.lda = lda; o.B = R; o.ldb = ldr; o.C = O; o.ldc = ldo; o.M = B; o.N = r; o.K = M;
    o.echelon = ech;
    return launched(launch_gemm(GS_F32, rt, ot, true, EPI_STORE, o, s), "gs_attention (weighted sum)");
}

gs_status gs_similarity_attention(const void *T, gs_dtype tt, int64_t B, int64_t r, int64_t ldt,
                                  const void *R, gs_dtype rt_in, int64_t M, int64_t ldr,
                                  const float *qnorm2, const float *cnorm, gs_sim_mode mode, float scale,
                                  float *S, int64_t lds, int32_t *argmax, float beta, float *A, int64_t lda,
                                  void *stream) {
    bool ech;
    const gs_dtype rt = coord_type(rt_in, &ech);
    const char *fn = "gs_similarity_attention";
    GS_CHECK(check_sim_common(fn, T, tt, B, r, ldt, R, rt, M, ldr, qnorm2, cnorm, mode));
    if (!S && !argmax && !A && B > 0) return fail(GS_ERR_ARG, "%s: S, argmax and A are all null", fn);
    GS_CHECK(check_matrix(S, "S", B, M, lds, GS_F32, true));
    GS_CHECK(check_matrix(A, "A", B, M, lda, GS_F32, true));
    GS_CHECK(check_aligned(argmax, 4, "argmax"));
    GS_CHECK(check_overlaps({span(T, B, r, ldt, esize(tt), "T"), span(R, M, r, ldr, esize(rt), "R"),
                             span(qnorm2, 1, B, B, 4, "qnorm2"), span(cnorm, 1, M, M, 4, "cnorm")},
                            {span(S, B, M, lds, 4, "S"), span(argmax, 1, B, B, 4, "argmax"),
                             span(A, B, M, lda, 4, "A")}));
    if (B == 0) return ok();
    GS_CHECK(check_device());
    hipStream_t s = (hipStream_t)stream;
    // argmax alone needs no score matrix: the similarity kernels' own
    if (!S && !A) return gs_similarity(T, tt, B, r, ldt, R, rt_in, M, ldr, qnorm2, cnorm, mode, scale,
                                       nullptr, M, argmax, stream);
    // the scores once, into S (or into A, replaced there by the weights)
    float *W = S ? S : A;
    const int64_t ldw = S ? lds : lda;
    if (M <= SMALL_MAX && r <= M && B > FEW_ROWS) {
        SmallArgs a{};
        a.In = T; a.ldin = ldt; a.R = R; a.ldr = ldr; a.B = B; a.M = M; a.r = r; a.Out = W; a.ldout = ldw;
        a.qnorm2 = qnorm2; a.cnorm = cnorm; a.cosine = mode == GS_SIM_COSINE; a.scale = scale;
        GS_CHECK(launched(launch_small_similarity(tt, a, s), fn));
    } else {
        GemmArgs a{};
        a.A = T; a.lda = ldt; a.B = R; a.ldb = ldr; a.C = W; a.ldc = ldw; a.M = B; a.N = M; a.K = r;
        a.qnorm2 = qnorm2; a.cnorm = cnorm; a.cosine = mode == GS_SIM_COSINE; a.scale = scale;
        a.write_out = true; a.echelon = ech;
        GS_CHECK(launched(launch_gemm(tt, rt, GS_F32, false, EPI_SIM, a, s), fn));
    }
    // one pass over the scores: the row argmax and the weights
    return launched(launch_sim_attn_pass(W, ldw, B, M, argmax, beta, A, lda, s), fn);
}

gs_status gs_reconstruct(const void *T, gs_dtype tt, int64_t B, int64_t r, int64_t ldt,
                         const void *T2, int64_t ldt2, gs_bind bind,
                         const void *Q, gs_dtype qt, int64_t D, int64_t ldq,
                         void *X, gs_dtype xt, int64_t ldx, void *stream) {
    if (!is_batch_type(tt) || qt != tt || !is_batch_type(xt))
        return fail(GS_ERR_DTYPE, "gs_reconstruct: T/Q must be both f32 or both bf16 and X f32 or bf16");
    if (bind != GS_BIND_NONE && bind != GS_BIND_MUL) return fail(GS_ERR_ARG, "gs_reconstruct: unknown bind");
    if (B < 0 || r < 1 || D < 1) return fail(GS_ERR_SHAPE, "gs_reconstruct: need B >= 0, r >= 1, D >= 1");
    GS_CHECK(check_matrix(T, "T", B, r, ldt, tt, false));
    if (bind == GS_BIND_MUL) GS_CHECK(check_matrix(T2, "T2", B, r, ldt2, tt, false));
    else if (T2) return fail(GS_ERR_ARG, "gs_reconstruct: T2 given without a bind operator");
    GS_CHECK(check_matrix(Q, "Q", r, D, ldq, qt, false));
    GS_CHECK(check_matrix(X, "X", B, D, ldx, xt, false));
    GS_CHECK(check_overlaps({span(T, B, r, ldt, esize(tt), "T"), span(T2, B, r, ldt2, esize(tt), "T2"),
                             span(Q, r, D, ldq, esize(qt), "Q")},
                            {span(X, B, D, ldx, esize(xt), "X")}));
    if (B == 0) return ok();
    GS_CHECK(check_device());
    GemmArgs a{};
    a.A = T; a.lda = ldt; a.A2 = T2; a.lda2 = ldt2; a.B = Q; a.ldb = ldq; a.C = X; a.ldc = ldx;
    a.M = B; a.N = D; a.K = r;
    return launched(launch_gemm(tt, qt, xt, true, bind == GS_BIND_MUL ? EPI_BIND : EPI_STORE, a,
                                (hipStream_t)stream), "gs_reconstruct");
}

gs_status gs_bind_coords(const void *T, gs_dtype tt, int64_t B, int64_t r, int64_t ldt,
                         const void *T2, int64_t ldt2, const void *Q, gs_dtype qt, int64_t D, int64_t ldq,
                         void *Z, gs_dtype zt, int64_t ldz, void *stream) {
    if (tt != GS_F32 || qt != GS_F32 || zt != GS_F32) return fail(GS_ERR_DTYPE, "gs_bind_coords: T, T2, Q and Z must be f32");
    if (B < 0 || r < 1 || D < 1) return fail(GS_ERR_SHAPE, "gs_bind_coords: need B >= 0, r >= 1, D >= 1");
    if (r > BIND_COORDS_MAX_R)
        return fail(GS_ERR_SHAPE, "gs_bind_coords: r = %lld exceeds %lld", (long long)r, (long long)BIND_COORDS_MAX_R);
    GS_CHECK(check_matrix(T, "T", B, r, ldt, tt, false));
    GS_CHECK(check_matrix(T2, "T2", B, r, ldt2, tt, false));
    GS_CHECK(check_matrix(Q, "Q", r, D, ldq, qt, false));
    GS_CHECK(check_matrix(Z, "Z", B, r, ldz, zt, false));
    GS_CHECK(check_overlaps({span(T, B, r, ldt, 4, "T"), span(T2, B, r, ldt2, 4, "T2"), span(Q, r, D, ldq, 4, "Q")},
                            {span(Z, B, r, ldz, 4, "Z")}));
    if (B == 0) return ok();
    GS_CHECK(check_device());
    BindCoordsArgs a{};
    a.T = static_cast<const float *>(T); a.ldt = ldt;
    a.T2 = static_cast<const float *>(T2); a.ldt2 = ldt2;
    a.Q = static_cast<const float *>(Q); a.ldq = ldq;
    a.Z = static_cast<float *>(Z); a.ldz = ldz;
    a.B = B; a.r = r; a.D = D;
    return launched(launch_bind_coords(a, (hipStream_t)stream), "gs_bind_coords");
}

gs_status gs_bind_restored(const void *X, gs_dtype xt, int64_t B, int64_t D, int64_t ldx,
                           const void *Y, int64_t ldy, gs_bind_op op, int64_t L,
                           void *Z, gs_dtype zt, int64_t ldz, void *stream) {
    if (!is_batch_type(xt) || !is_batch_type(zt)) return fail(GS_ERR_DTYPE, "gs_bind_restored: X/Y and Z must be f32 or bf16");
    if (op != GS_BINDOP_MUL && op != GS_BINDOP_XOR && op != GS_BINDOP_CONV && op != GS_BINDOP_CORR)
        return fail(GS_ERR_ARG, "gs_bind_restored: unknown operator");
    if (B < 0 || D < 1) return fail(GS_ERR_SHAPE, "gs_bind_restored: need B >= 0 and D >= 1");
    if (op == GS_BINDOP_CONV || op == GS_BINDOP_CORR) {
        if (L < 2 || L > 8192 || (L & (L - 1)) != 0 || D % L != 0)
            return fail(GS_ERR_SHAPE, "gs_bind_restored: L must be a power of two in [2, 8192] dividing D");
    }
    GS_CHECK(check_matrix(X, "X", B, D, ldx, xt, false));
    GS_CHECK(check_matrix(Y, "Y", B, D, ldy, xt, false));
    GS_CHECK(check_matrix(Z, "Z", B, D, ldz, zt, false));
    GS_CHECK(check_overlaps({span(X, B, D, ldx, esize(xt), "X"), span(Y, B, D, ldy, esize(xt), "Y")},
                            {span(Z, B, D, ldz, esize(zt), "Z")}));
    if (B == 0) return ok();
    GS_CHECK(check_device());
    BindArgs a{};
    a.X = X; a.ldx = ldx; a.Y = Y; a.ldy = ldy; a.Z = Z; a.ldz = ldz; a.B = B; a.D = D; a.L = L;
    return launched(launch_bind(xt, zt, (int)op, a, (hipStream_t)stream), "gs_bind_restored");
}

gs_status gs_soft_select(const gs_soft_group *groups, int ngroups, gs_dtype pt, gs_dtype tt,
                         gs_sim_mode mode, float scale, float beta, gs_soft_form form, void *stream) {
    if (!groups) return fail(GS_ERR_ARG, "gs_soft_select: groups is null");
    if (ngroups < 1 || ngroups > SOFT_MAX_GROUPS)
        return fail(GS_ERR_ARG, "gs_soft_select: ngroups must be in [1, %d]", SOFT_MAX_GROUPS);
    if (!is_batch_type(pt) || !is_batch_type(tt))
        return fail(GS_ERR_DTYPE, "gs_soft_select: P/R and T must be f32 or bf16");
    if (mode != GS_SIM_DOT && mode != GS_SIM_COSINE) return fail(GS_ERR_ARG, "gs_soft_select: unknown mode");
    if (form != GS_SOFT_AUTO && form != GS_SOFT_GRAM && form != GS_SOFT_COORDS)
        return fail(GS_ERR_ARG, "gs_soft_select: unknown form");
    std::vector<Span> in, out;
    SoftArgs a{};
    a.ngroups = ngroups;
    a.cosine = mode == GS_SIM_COSINE;
    a.scale = scale;
    a.beta = beta;
    int64_t tiles = 0;
    bool any_t = false;
    for (int i = 0; i < ngroups; ++i) {
        const gs_soft_group &g = groups[i];
        any_t = any_t || (g.T != nullptr && g.B > 0);
        if (g.B < 0 || g.M < 1 || g.M > SOFT_MAX_M || g.r < 1 || g.r > g.M)
            return fail(GS_ERR_SHAPE, "gs_soft_select: group %d needs B >= 0 and 1 <= r <= M <= %d", i, SOFT_MAX_M);
        GS_CHECK(check_matrix(g.P, "P", g.B, g.M, g.ldp, pt, false));
        GS_CHECK(check_matrix(g.R, "R", g.M, g.r, g.ldr, pt, false));
        GS_CHECK(check_aligned(g.cnorm, 4, "cnorm"));
        GS_CHECK(check_matrix(g.T, "T", g.B, g.r, g.ldt, tt, true));
        GS_CHECK(check_matrix(g.S, "S", g.B, g.M, g.lds, GS_F32, true));
        GS_CHECK(check_matrix(g.A, "A", g.B, g.M, g.lda, GS_F32, true));
        GS_CHECK(check_aligned(g.argmax, 4, "argmax"));
        in.push_back(span(g.P, g.B, g.M, g.ldp, esize(pt), "P"));
        in.push_back(span(g.R, g.M, g.r, g.ldr, esize(pt), "R"));
        in.push_back(span(g.cnorm, 1, g.M, g.M, 4, "cnorm"));
        out.push_back(span(g.T, g.B, g.r, g.ldt, esize(tt), "T"));
        out.push_back(span(g.S, g.B, g.M, g.lds, 4, "S"));
        out.push_back(span(g.argmax, 1, g.B, g.B, 4, "argmax"));
        out.push_back(span(g.A, g.B, g.M, g.lda, 4, "A"));
    }
    // Work-groups are dispatched in index order and the first ones get their
    // tiles first: the groups with the most work per row (the largest
    // codebooks) go first, so the longest work-groups start earliest.
    int order[SOFT_MAX_GROUPS];
    for (int i = 0; i < ngroups; ++i) order[i] = i;
    std::stable_sort(order, order + ngroups, [&](int x, int y) { return groups[x].M > groups[y].M; });
    for (int k = 0; k < ngroups; ++k) {
        const gs_soft_group &g = groups[order[k]];
        SoftGroup &d = a.g[k];
        d.P = g.P; d.ldp = g.ldp; d.R = g.R; d.ldr = g.ldr; d.cnorm = g.cnorm;
        d.B = g.B; d.M = g.M; d.r = g.r; d.T = g.T; d.ldt = g.ldt; d.S = g.S; d.lds = g.lds;
        d.argmax = g.argmax; d.A = g.A; d.lda = g.lda;
        a.tile_start[k] = tiles;
        tiles += soft_select_tiles(g.B);
    }
    a.tile_start[ngroups] = tiles;
    a.ntiles = tiles;
    if (form == GS_SOFT_GRAM && any_t)
        return fail(GS_ERR_ARG, "gs_soft_select: the Gram form forms no coordinates, but a group asks for T");
    a.coords = form == GS_SOFT_COORDS || (form == GS_SOFT_AUTO && any_t);
    GS_CHECK(check_overlaps(in, out));
    if (tiles == 0) return ok();
    GS_CHECK(check_device());
    return launched(launch_soft_select(pt, tt, a, (hipStream_t)stream), "gs_soft_select");
}

}  // extern "C"
