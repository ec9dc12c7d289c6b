// Host runtime behind the C ABI of include/tr.h: validation, budget plan
// (Algorithm 1), scratch ownership, launch orchestration and timing.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <dlfcn.h>

#include <algorithm>
#include <atomic>
#include <mutex>
#include <new>
#include <vector>

#include "tr.h"
#include "tr_internal.h"

using tr::CallPtrs;
using tr::check_params;
using tr::clear_error;
using tr::elem_bytes;
using tr::fail;
using tr::log_line;
using tr::ImageDesc;
using tr::make_plan;
using tr::Plan;

namespace {

tr_status hip_fail(hipError_t e, const char* what)
{
    return fail(TR_EDEVICE, "%s: %s", what, hipGetErrorString(e));
}

constexpr int kTimedCalls = 1024;
constexpr int64_t kFusedCopyBytes = 8 << 20;
constexpr int kLdsFallback = 65536;

int lds_limit_of(int dev)
{
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess || v <= 0)
        v = kLdsFallback;
    return v;
}

int capacity_for(int lds_limit)
{
    int lo = 0, hi = 65535;
    while (lo < hi) {
        const int mid = (lo + hi + 1) / 2;
        if (tr::select_lds_bytes(mid, tr::select_threads(mid)) <= (size_t)lds_limit) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Optional roctx ranges: with the environment variable TR_ROCTX = 1 the
// marker library is opened once (dlopen, no link-time dependency) and every
// entry point that enqueues work brackets its enqueue in a range named after
// itself, so a marker trace ties each call to the kernels it launched.
struct Roctx {
    int (*push)(const char*) = nullptr;
    int (*pop)() = nullptr;
};

const Roctx& roctx()
{
    static const Roctx r = [] {
        Roctx x;
        const char* v = getenv("TR_ROCTX");
        if (!v || strcmp(v, "1") != 0) return x;
        void* h = dlopen("librocprofiler-sdk-roctx.so.1", RTLD_NOW | RTLD_LOCAL);
        if (!h) h = dlopen("libroctx64.so.4", RTLD_NOW | RTLD_LOCAL);
        if (!h) {
            log_line("TR_ROCTX=1 but no roctx library could be opened");
            return x;
        }
        x.push = reinterpret_cast<int (*)(const char*)>(dlsym(h, "roctxRangePushA"));
        x.pop = reinterpret_cast<int (*)()>(dlsym(h, "roctxRangePop"));
        if (!x.push || !x.pop) {
            x.push = nullptr;
            x.pop = nullptr;
            log_line("TR_ROCTX=1 but the roctx library lacks its range functions");
        } else {
            log_line("roctx ranges on");
        }
        return x;
    }();
    return r;
}

struct Range {
    bool on;
    explicit Range(const char* name) : on(roctx().push != nullptr)
    {
        if (on) roctx().push(name);
    }
    ~Range()
    {
        if (on) roctx().pop();
    }
};

// The device allocations of one tr_create call.  Test hook: with the
// environment variable TR_FAIL_ALLOC = k (k >= 1), the k-th allocation fails
// as if the device were out of memory (nothing is allocated for it), so that
// the clean-up path of tr_create can be exercised on a real device.
struct CtxAlloc {
    int count = 0;
    int fail_at = 0;
    CtxAlloc()
    {
        const char* v = getenv("TR_FAIL_ALLOC");
        if (v) fail_at = atoi(v);
    }
    template <typename T>
    hipError_t operator()(T** ptr, size_t bytes)
    {
        if (++count == fail_at) {
            *ptr = nullptr;
            return hipErrorOutOfMemory;
        }
        return hipMalloc(reinterpret_cast<void**>(ptr), bytes);
    }
};

// Copies the context's count to a caller's word (and resets it if asked).
__global__ void take_kernel(uint32_t* src, uint32_t* dst, int32_t reset)
{
    if (threadIdx.x == 0) {
        *dst = *src;
        if (reset) *src = 0u;
    }
}

struct DeviceGuard {
    int prev = -1;
    bool ok = true;
    explicit DeviceGuard(int dev)
    {
        if (hipGetDevice(&prev) != hipSuccess) prev = -1;
        if (prev != dev) ok = hipSetDevice(dev) == hipSuccess;
    }
    ~DeviceGuard()
    {
        int cur = -1;
        if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
    }
};

}  // namespace

struct tr_ctx {
    tr_params p{};
    int device = 0;
    int Dc = 0;
    int eb = 4;
    int lds_limit = 0;
    int cap_n = 0;
    int cus = 256;                // compute units of the device
    float* key_imp = nullptr;
    float* key_s = nullptr;
    int32_t* rows = nullptr;
    uint32_t* gsel = nullptr;     // pick bitmaps of images shared by several workgroups
    uint32_t* gimp = nullptr;     // their X^imp bitmaps
    float* cos_part = nullptr;    // per-tile cosine partials of tr_mlp_out_cos (bf16, Dc % 128 == 0)
    uint32_t* nonfinite = nullptr;   // count of scored rows with a NaN or infinite element (TR_FLAG_CHECK_FINITE)
    bool timing = false;
    std::vector<hipEvent_t> events;   // 4 per timed call
    int timed = 0;
};

namespace {

// The kept rows' copy when the selection does it (every image of the call
// has at most kSmallSelectN tokens), or none.
struct FusedCopy {
    const void* X = nullptr;
    void* out = nullptr;
    int64_t row_bytes = 0;
    bool vec = false;
    int elem = 4;
};

// Launch the selection for every image of a plan (one launch when the batch is
// uniform, else groups of at most kMaxDescPerLaunch images).
hipError_t run_select(const tr_ctx* c, const Plan& pl, const float* key_imp, const float* key_s,
                      int32_t* out_idx, uint8_t* out_src, int32_t* out_rows, hipStream_t s,
                      const FusedCopy& fc = FusedCopy())
{
    tr::SelectArgs a;
    memset(&a, 0, sizeof a);
    a.key_imp = key_imp;
    a.key_s = key_s;
    a.out_idx = out_idx;
    a.out_src = out_src;
    a.out_rows = out_rows;
    a.gsel = c->gsel;
    a.gimp = c->gimp;
    a.stride_real = (c->p.flags & TR_FLAG_STRIDE_REAL) ? 1 : 0;
    const int B = (int)pl.desc.size();
    if (B == 0) return hipSuccess;
    if (fc.X) {
        int kmin = INT32_MAX;
        for (int b = 0; b < B; ++b) kmin = std::min(kmin, pl.desc[(size_t)b].k1 + pl.desc[(size_t)b].k2);
        a.gX = fc.X;
        a.gout = fc.out;
        a.grow_bytes = fc.row_bytes;
        a.gvec = fc.vec ? 1 : 0;
        a.gelem = fc.elem;
        a.ggroups = tr::select_small_groups(B, kmin, c->cus);
    }
    if (pl.uniform) {
        a.uniform = 1;
        a.nimg = B;
        a.img0 = 0;
        a.desc[0] = pl.desc[0];
        a.groups = tr::select_groups(tr::select_shares(pl.desc[0]) ? B : 0, c->cus);
        return tr::launch_select(a, pl.nmax, s);
    }
    for (int b0 = 0; b0 < B; b0 += tr::kMaxDescPerLaunch) {
        const int nb = B - b0 < tr::kMaxDescPerLaunch ? B - b0 : tr::kMaxDescPerLaunch;
        a.uniform = 0;
        a.nimg = nb;
        a.img0 = b0;
        int nmax = 0, large = 0;
        for (int i = 0; i < nb; ++i) {
            a.desc[i] = pl.desc[(size_t)(b0 + i)];
            if (a.desc[i].n > nmax) nmax = a.desc[i].n;
            if (tr::select_shares(a.desc[i])) ++large;
        }
        a.groups = tr::select_groups(large, c->cus);
        hipError_t e = tr::launch_select(a, nmax, s);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

tr_status check_ctx_plan(tr_ctx* c, int32_t B, const int32_t* N, const int32_t* K, Plan& pl)
{
    tr_status st = make_plan(&c->p, B, N, K, pl);
    if (st != TR_OK) return st;
    if (pl.nmax > c->cap_n)
        return fail(TR_EUNSUPPORTED, "N = %d exceeds the selection capacity %d", pl.nmax, c->cap_n);
    return TR_OK;
}

}  // namespace

extern "C" {

int32_t tr_capacity_N(void)
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    return capacity_for(lds_limit_of(dev));
}

tr_status tr_create(const tr_params* p, tr_ctx** out)
{
    clear_error();
    if (!out) return fail(TR_EINVAL, "out is NULL");
    *out = nullptr;
    tr_status st = check_params(p, true);
    if (st != TR_OK) return st;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    const int lds = lds_limit_of(dev);
    const int cap = capacity_for(lds);
    if (p->max_N > cap)
        return fail(TR_EUNSUPPORTED, "max_N = %d exceeds the selection capacity %d of this device",
                    p->max_N, cap);
    tr_ctx* c = new (std::nothrow) tr_ctx;
    if (!c) return fail(TR_ENOMEM, "host allocation failed");
    c->p = *p;
    c->device = dev;
    c->Dc = p->Dc ? p->Dc : p->D;
    c->eb = elem_bytes(p->dtype);
    c->lds_limit = lds;
    c->cap_n = cap;
    if ((e = hipDeviceGetAttribute(&c->cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) {
        tr_destroy(c);
        return hip_fail(e, "hipDeviceGetAttribute");
    }
    const size_t n = (size_t)p->max_tokens;
    const size_t gw = tr::select_gsel_words(p->max_tokens, p->max_images);
    CtxAlloc al;
    if ((e = al(&c->key_imp, n * sizeof(float))) != hipSuccess ||
        (e = al(&c->key_s, n * sizeof(float))) != hipSuccess ||
        (e = al(&c->rows, n * sizeof(int32_t))) != hipSuccess ||
        (e = al(&c->gsel, gw * sizeof(uint32_t))) != hipSuccess ||
        (e = al(&c->gimp, gw * sizeof(uint32_t))) != hipSuccess) {
        tr_destroy(c);
        return fail(TR_ENOMEM, "hipMalloc of %zu-token scratch failed: %s", n, hipGetErrorString(e));
    }
    // The split selection leaves the pick bitmaps zero after every call.  The
    // key scratch starts at zero so that a call that needs neither key (every
    // image keeps all its tokens of a stage) selects from defined values.
    if ((e = hipMemset(c->gsel, 0, gw * sizeof(uint32_t))) != hipSuccess ||
        (e = hipMemset(c->key_imp, 0, n * sizeof(float))) != hipSuccess ||
        (e = hipMemset(c->key_s, 0, n * sizeof(float))) != hipSuccess ||
        (e = hipDeviceSynchronize()) != hipSuccess) {
        tr_destroy(c);
        return hip_fail(e, "scratch initialisation");
    }
    if ((e = tr::select_prepare(lds)) != hipSuccess || (e = tr::gemm_prepare()) != hipSuccess) {
        tr_destroy(c);
        return hip_fail(e, "hipFuncSetAttribute");
    }
    if (p->flags & TR_FLAG_CHECK_FINITE) {
        if ((e = al(&c->nonfinite, sizeof(uint32_t))) != hipSuccess) {
            tr_destroy(c);
            return fail(TR_ENOMEM, "hipMalloc of the non-finite row count failed");
        }
        if ((e = hipMemset(c->nonfinite, 0, sizeof(uint32_t))) != hipSuccess ||
            (e = hipDeviceSynchronize()) != hipSuccess) {
            tr_destroy(c);
            return hip_fail(e, "non-finite row count initialisation");
        }
    }
    if (p->dtype == TR_BF16 && c->Dc % 128 == 0) {
        const size_t words = n * (size_t)tr::gemm_part_cols(c->Dc) * 3;
        if ((e = al(&c->cos_part, words * sizeof(float))) != hipSuccess) {
            tr_destroy(c);
            return fail(TR_ENOMEM, "hipMalloc of %zu cosine partials failed", words);
        }
    }
    log_line("context on device %d: D %d, Dc %d, %s, lambda %.6g, flags 0x%x, up to %d images / %lld tokens / "
             "N %d (device selection capacity %d)",
             dev, p->D, c->Dc, p->dtype == TR_BF16 ? "bf16" : "fp32", p->lambda, (unsigned)p->flags, p->max_images,
             (long long)p->max_tokens, p->max_N, cap);
    *out = c;
    return TR_OK;
}

void tr_destroy(tr_ctx* c)
{
    if (!c) return;
    DeviceGuard g(c->device);
    if (c->key_imp) (void)hipFree(c->key_imp);
    if (c->key_s) (void)hipFree(c->key_s);
    if (c->rows) (void)hipFree(c->rows);
    if (c->gsel) (void)hipFree(c->gsel);
    if (c->gimp) (void)hipFree(c->gimp);
    if (c->cos_part) (void)hipFree(c->cos_part);
    if (c->nonfinite) (void)hipFree(c->nonfinite);
    for (hipEvent_t ev : c->events) (void)hipEventDestroy(ev);
    delete c;
}

tr_status tr_timing_enable(tr_ctx* c, int32_t enable)
{
    clear_error();
    if (!c) return fail(TR_EINVAL, "ctx is NULL");
    DeviceGuard g(c->device);
    if (enable && c->events.empty()) {
        c->events.resize((size_t)kTimedCalls * 4, nullptr);
        for (hipEvent_t& ev : c->events) {
            hipError_t e = hipEventCreate(&ev);
            if (e != hipSuccess) return hip_fail(e, "hipEventCreate");
        }
    }
    c->timing = enable != 0;
    c->timed = 0;
    return TR_OK;
}

tr_status tr_timing_read(tr_ctx* c, double* ms, int64_t* calls)
{
    clear_error();
    if (!c || !ms) return fail(TR_EINVAL, "ctx or ms is NULL");
    DeviceGuard g(c->device);
    double acc[3] = {0, 0, 0};
    for (int i = 0; i < c->timed; ++i) {
        hipEvent_t* ev = &c->events[(size_t)i * 4];
        hipError_t e = hipEventSynchronize(ev[3]);
        if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
        for (int k = 0; k < 3; ++k) {
            float t = 0.f;
            e = hipEventElapsedTime(&t, ev[k], ev[k + 1]);
            if (e != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
            acc[k] += t;
        }
    }
    ms[0] = acc[0];
    ms[1] = acc[1];
    ms[2] = acc[2];
    if (calls) *calls = c->timed;
    c->timed = 0;
    return TR_OK;
}

}  // extern "C"

namespace {

// One call of the module: tr_reduce, or one of its two fused forms (Stage II
// key supplied; projection of the kept rows instead of their copy).
struct ReduceCall {
    const void* X = nullptr;
    const void* X_pre = nullptr;
    const void* X_post = nullptr;
    const float* key_s = nullptr;   // supplied Stage II key, or nullptr
    int32_t B = 0;
    const int32_t* N = nullptr;
    const int32_t* K = nullptr;
    void* out = nullptr;
    int32_t* out_idx = nullptr;
    uint8_t* out_src = nullptr;
    float* out_h2 = nullptr;
    float* out_s = nullptr;
    const void* W = nullptr;        // projector weight [Nout, D], or nullptr: gather
    int64_t ldw = 0;
    int32_t Nout = 0;
    void* stream = nullptr;
};

tr_status reduce_impl(tr_ctx* c, ReduceCall r)
{
    if (!c) return fail(TR_EINVAL, "ctx is NULL");
    Plan pl;
    tr_status st = check_ctx_plan(c, r.B, r.N, r.K, pl);
    if (st != TR_OK) return st;
    if (r.B == 0) return TR_OK;
    // Pointer rules, and which scores the call needs (lambda = 1 never needs
    // s, lambda = 0 never needs H2; a supplied Stage II key replaces s).  A
    // score that is not needed is not computed and its inputs are not read.
    CallPtrs cp;
    cp.X = r.X;
    cp.X_pre = r.X_pre;
    cp.X_post = r.X_post;
    cp.key_s = r.key_s;
    cp.out = r.out;
    cp.out_idx = r.out_idx;
    cp.out_src = r.out_src;
    cp.out_h2 = r.out_h2;
    cp.out_s = r.out_s;
    bool need_x = false, need_c = false;
    st = tr::check_call(&c->p, pl, cp, need_x, need_c);
    if (st != TR_OK) return st;
    r.X_pre = cp.X_pre;
    r.X_post = cp.X_post;
    int mode = (need_x ? tr::kScoreImp : 0) | (need_c ? tr::kScoreSim : 0);
    if (need_x && (c->p.flags & TR_FLAG_SHANNON)) mode |= tr::kScoreShannon;

    const int64_t row_bytes = (int64_t)c->p.D * c->eb;
    const int64_t rowc_bytes = (int64_t)c->Dc * c->eb;
    const bool vec_score = aligned16(r.X) && aligned16(r.X_pre) && aligned16(r.X_post) &&
                           row_bytes % 16 == 0 && rowc_bytes % 16 == 0;
    const bool vec_gather = aligned16(r.X) && aligned16(r.out) && row_bytes % 16 == 0;
    tr::GemmArgs ga{};
    if (r.W) {
        if (c->p.dtype != TR_BF16) return fail(TR_EUNSUPPORTED, "the projection needs a bf16 context");
        if (!tr::gemm_shape_ok((int)pl.sum_k, r.Nout, c->p.D))
            return fail(TR_EUNSUPPORTED, "projection needs Nout %% 128 == 0 and D %% 64 == 0 (Nout = %d, D = %d)",
                        r.Nout, c->p.D);
        if (!aligned16(r.X) || row_bytes % 16 || !aligned16(r.W) || (r.ldw * 2) % 16 || r.ldw < c->p.D)
            return fail(TR_EINVAL, "X, W and their row strides must be 16-byte aligned (ldw >= D)");
        ga.A = r.X;
        ga.arows = c->rows;
        ga.arow_count = pl.sum_n;
        ga.B = r.W;
        ga.C = r.out;
        ga.M = (int32_t)pl.sum_k;
        ga.N = r.Nout;
        ga.K = c->p.D;
        ga.lda = c->p.D;
        ga.ldb = r.ldw;
        ga.ldc = r.Nout;
    }

    DeviceGuard g(c->device);
    if (!g.ok) return fail(TR_EDEVICE, "hipSetDevice(%d) failed", c->device);
    hipStream_t s = static_cast<hipStream_t>(r.stream);
    // A timed call takes the next free slot of four events; the slot counts
    // only once every launch of the call is enqueued, so a call that fails
    // part-way leaves no half-recorded slot for tr_timing_read.
    hipEvent_t* ev = nullptr;
    if (c->timing && c->timed < kTimedCalls) ev = &c->events[(size_t)c->timed * 4];
    hipError_t e;
    if (ev && (e = hipEventRecord(ev[0], s)) != hipSuccess) return hip_fail(e, "hipEventRecord");

    if (mode) {
        tr::ScoreArgs sa;
        sa.X = r.X;
        sa.P = r.X_pre;
        sa.Q = r.X_post;
        sa.rows = pl.sum_n;
        sa.D = c->p.D;
        sa.Dc = c->Dc;
        sa.key_imp = c->key_imp;
        sa.key_s = r.key_s ? nullptr : c->key_s;
        sa.out_h2 = r.out_h2;
        sa.out_s = r.out_s;
        sa.logD = (float)log((double)c->p.D);
        sa.nonfinite = c->nonfinite;
        if ((e = tr::launch_score(sa, c->p.dtype == TR_BF16, vec_score, mode, s)) != hipSuccess)
            return hip_fail(e, "score kernel launch");
    }
    if (ev && (e = hipEventRecord(ev[1], s)) != hipSuccess) return hip_fail(e, "hipEventRecord");

    // Small calls (images of at most kSmallSelectN tokens, at most
    // kFusedCopyBytes of kept rows): the selection copies the kept rows itself,
    // saving the gather launch on a latency-bound call.  Larger copies are
    // bound by HBM bandwidth and run faster in the gather kernel (64 x 576 x
    // 4096 bf16: step 150.7 us fused, 149.1-150.6 us with the gather kernel).
    FusedCopy fc;
    if (!r.W && pl.nmax <= tr::kSmallSelectN && pl.sum_k * row_bytes <= kFusedCopyBytes) {
        fc.X = r.X;
        fc.out = r.out;
        fc.row_bytes = row_bytes;
        fc.vec = vec_gather;
        fc.elem = c->eb;
    }
    if ((e = run_select(c, pl, c->key_imp, r.key_s ? r.key_s : c->key_s, r.out_idx, r.out_src,
                        fc.X ? nullptr : c->rows, s, fc)) != hipSuccess)
        return hip_fail(e, "select kernel launch");
    if (ev && (e = hipEventRecord(ev[2], s)) != hipSuccess) return hip_fail(e, "hipEventRecord");

    if (r.W) e = tr::launch_gemm(ga, s);
    else if (!fc.X) e = tr::launch_gather(r.X, r.out, c->rows, pl.sum_k, pl.sum_n, row_bytes, c->eb, vec_gather, s);
    if (e != hipSuccess) return hip_fail(e, r.W ? "projection kernel launch" : "gather kernel launch");
    if (ev && (e = hipEventRecord(ev[3], s)) != hipSuccess) return hip_fail(e, "hipEventRecord");
    if (ev) ++c->timed;
    return TR_OK;
}

}  // namespace

extern "C" {

tr_status tr_reduce(tr_ctx* c, const void* X, const void* X_pre, const void* X_post, int32_t B,
                    const int32_t* N, const int32_t* K, void* out, int32_t* out_idx,
                    uint8_t* out_src, float* out_h2, float* out_s, void* stream)
{
    clear_error();
    Range range("tr_reduce");
    ReduceCall r;
    r.X = X;
    r.X_pre = X_pre;
    r.X_post = X_post;
    r.B = B;
    r.N = N;
    r.K = K;
    r.out = out;
    r.out_idx = out_idx;
    r.out_src = out_src;
    r.out_h2 = out_h2;
    r.out_s = out_s;
    r.stream = stream;
    return reduce_impl(c, r);
}

tr_status tr_reduce_given_s(tr_ctx* c, const void* X, const float* key_s, int32_t B, const int32_t* N,
                            const int32_t* K, void* out, int32_t* out_idx, uint8_t* out_src, float* out_h2,
                            void* stream)
{
    clear_error();
    Range range("tr_reduce_given_s");
    if (!key_s) return fail(TR_EINVAL, "key_s must be non-NULL");
    ReduceCall r;
    r.X = X;
    r.key_s = key_s;
    r.B = B;
    r.N = N;
    r.K = K;
    r.out = out;
    r.out_idx = out_idx;
    r.out_src = out_src;
    r.out_h2 = out_h2;
    r.stream = stream;
    return reduce_impl(c, r);
}

tr_status tr_reduce_project(tr_ctx* c, const void* X, const void* X_pre, const void* X_post, int32_t B,
                            const int32_t* N, const int32_t* K, const void* W, int64_t ldw, int32_t Nout,
                            void* out, int32_t* out_idx, uint8_t* out_src, void* stream)
{
    clear_error();
    Range range("tr_reduce_project");
    if (!W) return fail(TR_EINVAL, "W must be non-NULL");
    ReduceCall r;
    r.X = X;
    r.X_pre = X_pre;
    r.X_post = X_post;
    r.B = B;
    r.N = N;
    r.K = K;
    r.W = W;
    r.ldw = ldw;
    r.Nout = Nout;
    r.out = out;
    r.out_idx = out_idx;
    r.out_src = out_src;
    r.stream = stream;
    return reduce_impl(c, r);
}

tr_status tr_gemm_bf16(tr_ctx* c, const void* A, int64_t lda, const int32_t* a_rows, int64_t a_row_count,
                       const void* B, int64_t ldb, void* C, int64_t ldc, int32_t M, int32_t N, int32_t K,
                       void* stream)
{
    clear_error();
    Range range("tr_gemm_bf16");
    if (!c) return fail(TR_EINVAL, "ctx is NULL");
    if (M < 0) return fail(TR_EINVAL, "M must be >= 0");
    if (!tr::gemm_shape_ok(M, N, K))
        return fail(TR_EUNSUPPORTED, "GEMM needs N %% 128 == 0 and K %% 64 == 0 (N = %d, K = %d)", N, K);
    if (M == 0) return TR_OK;
    if (!A || !B || !C) return fail(TR_EINVAL, "A, B and C must be non-NULL");
    if (!aligned16(A) || !aligned16(B) || (lda * 2) % 16 || (ldb * 2) % 16 || lda < K || ldb < K || ldc < N ||
        ((uintptr_t)C & 1u) || ((uintptr_t)a_rows & 3u))
        return fail(TR_EINVAL, "A and B need 16-byte aligned bases and row strides >= K; C stride >= N");
    if (a_rows && a_row_count < 1) return fail(TR_EINVAL, "a_row_count must be >= 1 with a_rows");
    DeviceGuard g(c->device);
    if (!g.ok) return fail(TR_EDEVICE, "hipSetDevice(%d) failed", c->device);
    tr::GemmArgs ga{};
    ga.A = A;
    ga.arows = a_rows;
    ga.arow_count = a_rows ? a_row_count : M;
    ga.B = B;
    ga.C = C;
    ga.M = M;
    ga.N = N;
    ga.K = K;
    ga.lda = lda;
    ga.ldb = ldb;
    ga.ldc = ldc;
    hipError_t e = tr::launch_gemm(ga, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "GEMM launch");
    return TR_OK;
}

tr_status tr_mlp_out_cos(tr_ctx* c, const void* Hact, int64_t ldh, const void* W2, int64_t ldw,
                         const void* X_pre, void* X_post, int32_t M, int32_t Hd, float* key_s, void* stream)
{
    clear_error();
    Range range("tr_mlp_out_cos");
    if (!c) return fail(TR_EINVAL, "ctx is NULL");
    if (c->p.dtype != TR_BF16) return fail(TR_EUNSUPPORTED, "tr_mlp_out_cos needs a bf16 context");
    if (!c->cos_part) return fail(TR_EUNSUPPORTED, "tr_mlp_out_cos needs Dc %% 128 == 0 (Dc = %d)", c->Dc);
    if (M < 0 || (int64_t)M > c->p.max_tokens) return fail(TR_EINVAL, "M must be in [0, max_tokens]");
    if (!tr::gemm_shape_ok(M, c->Dc, Hd)) return fail(TR_EUNSUPPORTED, "Hd must be a positive multiple of 64");
    if (M == 0) return TR_OK;
    if (!Hact || !W2 || !X_pre || !X_post || !key_s)
        return fail(TR_EINVAL, "Hact, W2, X_pre, X_post and key_s must be non-NULL");
    if (!aligned16(Hact) || !aligned16(W2) || (ldh * 2) % 16 || (ldw * 2) % 16 || ldh < Hd || ldw < Hd ||
        ((uintptr_t)X_pre & 1u) || ((uintptr_t)X_post & 1u) || ((uintptr_t)key_s & 3u))
        return fail(TR_EINVAL, "Hact and W2 need 16-byte aligned bases and row strides >= Hd");
    DeviceGuard g(c->device);
    if (!g.ok) return fail(TR_EDEVICE, "hipSetDevice(%d) failed", c->device);
    tr::GemmArgs ga{};
    ga.A = Hact;
    ga.arow_count = M;
    ga.B = W2;
    ga.C = X_post;
    ga.M = M;
    ga.N = c->Dc;
    ga.K = Hd;
    ga.lda = ldh;
    ga.ldb = ldw;
    ga.ldc = c->Dc;
    ga.P = X_pre;
    ga.ldp = c->Dc;
    ga.part = c->cos_part;
    ga.part_cols = tr::gemm_part_cols(c->Dc);
    ga.s_out = key_s;
    hipError_t e = tr::launch_gemm(ga, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "GEMM launch");
    return TR_OK;
}

tr_status tr_read_bandwidth(const void* const* p, const int64_t* bytes, int32_t n, uint32_t* sink,
                            int32_t sink_words, void* stream)
{
    clear_error();
    Range range("tr_read_bandwidth");
    if (n < 1 || n > tr::kReadBuffers || !p || !bytes)
        return fail(TR_EINVAL, "n must be in [1, %d] with host arrays p and bytes", tr::kReadBuffers);
    int64_t total = 0;
    for (int i = 0; i < n; ++i) {
        if (bytes[i] < 0 || bytes[i] % 16) return fail(TR_EINVAL, "bytes[%d] must be a non-negative multiple of 16", i);
        if (bytes[i] && (!p[i] || !aligned16(p[i]))) return fail(TR_EINVAL, "p[%d] must be 16-byte aligned", i);
        total += bytes[i];
    }
    if (total == 0) return TR_OK;
    if (!sink || sink_words < 1 || ((uintptr_t)sink & 3u))
        return fail(TR_EINVAL, "sink must be a 4-byte aligned buffer of >= 1 word");
    hipError_t e = tr::launch_read(p, bytes, n, sink, sink_words, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "read kernel launch");
    return TR_OK;
}

tr_status tr_nonfinite_rows(tr_ctx* c, uint32_t* count, int32_t reset, void* stream)
{
    clear_error();
    if (!c) return fail(TR_EINVAL, "ctx is NULL");
    if (!c->nonfinite) return fail(TR_EUNSUPPORTED, "the context was created without TR_FLAG_CHECK_FINITE");
    if (!count || ((uintptr_t)count & 3u)) return fail(TR_EINVAL, "count must be a 4-byte aligned device word");
    DeviceGuard g(c->device);
    if (!g.ok) return fail(TR_EDEVICE, "hipSetDevice(%d) failed", c->device);
    hipLaunchKernelGGL(take_kernel, dim3(1), dim3(64), 0, static_cast<hipStream_t>(stream), c->nonfinite, count,
                       reset);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "count copy launch");
    return TR_OK;
}

tr_status tr_score(tr_ctx* c, const void* X, const void* X_pre, const void* X_post, int64_t rows,
                   float* key_imp, float* key_s, float* out_h2, void* stream)
{
    clear_error();
    Range range("tr_score");
    if (!c) return fail(TR_EINVAL, "ctx is NULL");
    if (rows < 0) return fail(TR_EINVAL, "rows must be >= 0");
    if (rows == 0) return TR_OK;
    const bool want_x = X || key_imp || out_h2;
    const bool want_c = X_pre || X_post || key_s;
    if (!want_x && !want_c) return fail(TR_EINVAL, "nothing to compute: every tensor is NULL");
    if (want_x && (!X || !key_imp)) return fail(TR_EINVAL, "X and key_imp go together (out_h2 needs both)");
    if (want_c && (!X_pre || !X_post || !key_s))
        return fail(TR_EINVAL, "X_pre, X_post and key_s go together");
    const uintptr_t em = (uintptr_t)c->eb - 1;
    if (((uintptr_t)X | (uintptr_t)X_pre | (uintptr_t)X_post) & em)
        return fail(TR_EUNSUPPORTED, "X, X_pre and X_post must be aligned to the element size (%d bytes)", c->eb);
    if (((uintptr_t)key_imp | (uintptr_t)key_s | (uintptr_t)out_h2) & 3u)
        return fail(TR_EUNSUPPORTED, "score outputs must be 4-byte aligned");
    const int64_t row_bytes = (int64_t)c->p.D * c->eb;
    const int64_t rowc_bytes = (int64_t)c->Dc * c->eb;
    const bool vec = aligned16(X) && aligned16(X_pre) && aligned16(X_post) && row_bytes % 16 == 0 &&
                     rowc_bytes % 16 == 0;
    DeviceGuard g(c->device);
    if (!g.ok) return fail(TR_EDEVICE, "hipSetDevice(%d) failed", c->device);
    tr::ScoreArgs sa;
    sa.X = X;
    sa.P = X_pre;
    sa.Q = X_post;
    sa.rows = rows;
    sa.D = c->p.D;
    sa.Dc = c->Dc;
    sa.key_imp = key_imp;
    sa.key_s = key_s;
    sa.out_h2 = out_h2;
    sa.out_s = nullptr;
    sa.logD = (float)log((double)c->p.D);
    sa.nonfinite = c->nonfinite;
    int mode = (want_x ? tr::kScoreImp : 0) | (want_c ? tr::kScoreSim : 0);
    if (want_x && (c->p.flags & TR_FLAG_SHANNON)) mode |= tr::kScoreShannon;
    hipError_t e = tr::launch_score(sa, c->p.dtype == TR_BF16, vec, mode, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "score kernel launch");
    return TR_OK;
}

tr_status tr_select(tr_ctx* c, const float* key_imp, const float* key_s, int32_t B, const int32_t* N,
                    const int32_t* K, int32_t* out_idx, uint8_t* out_src, void* stream)
{
    clear_error();
    Range range("tr_select");
    if (!c) return fail(TR_EINVAL, "ctx is NULL");
    Plan pl;
    tr_status st = check_ctx_plan(c, B, N, K, pl);
    if (st != TR_OK) return st;
    if (B == 0) return TR_OK;
    if (!key_imp || !key_s || !out_idx) return fail(TR_EINVAL, "key_imp, key_s and out_idx must be non-NULL");
    if (((uintptr_t)key_imp | (uintptr_t)key_s | (uintptr_t)out_idx) & 3u)
        return fail(TR_EUNSUPPORTED, "key and index arrays must be 4-byte aligned");
    DeviceGuard g(c->device);
    if (!g.ok) return fail(TR_EDEVICE, "hipSetDevice(%d) failed", c->device);
    hipError_t e = run_select(c, pl, key_imp, key_s, out_idx, out_src, nullptr, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "select kernel launch");
    return TR_OK;
}

}  // extern "C"

// ---- tr_reduce without a context, for callers that cannot allocate ------------
namespace {

constexpr int64_t kStaticTokens = TR_NOALLOC_MAX_TOKENS;
constexpr int32_t kStaticImages = TR_NOALLOC_MAX_IMAGES;
constexpr size_t kStaticGselWords = (size_t)(kStaticTokens / 32) + 2 * (size_t)kStaticImages + 2;
// Stage I keys, Stage II keys and kept-row list (a word per token each),
// then the two split-selection bitmaps: 6.4 MB.
constexpr size_t kStaticWords = 3 * (size_t)kStaticTokens + 2 * kStaticGselWords;
static_assert(kStaticGselWords >= 2 + kStaticTokens / 32 + 2 * (size_t)kStaticImages,
              "bitmap words of every image of a full call");

// The scratch of tr_reduce_noalloc, one copy per device for the life of the
// process.  In host code `scratch` names the symbol only; its device address
// is taken once per device with hipGetSymbolAddress and used from then on.
static __device__ __align__(256) uint32_t scratch[kStaticWords];

__global__ __launch_bounds__(256) void fill_kernel(uint32_t* p, int64_t n, uint32_t v)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

constexpr int kMaxDevices = 64;

struct StaticDev {
    uint32_t* ptr = nullptr;   // device address of `scratch` on this device
    int lds = 0;
    int cap_n = 0;
    int cus = 256;
};

StaticDev g_static[kMaxDevices];
std::atomic<int> g_static_ready[kMaxDevices];
std::mutex g_static_mu;

// Set-up on the first call on a device (that device current): the array's
// address on this device, the selection's LDS limit, and one clear of the
// array on the caller's stream (the split selection needs its bitmaps zero;
// the keys start defined).  A fill kernel, not a memset, so that a first call
// under graph capture records only kernels.
tr_status static_setup(int dev, hipStream_t stream, const StaticDev*& out)
{
    if (dev < 0 || dev >= kMaxDevices) return fail(TR_EUNSUPPORTED, "device %d beyond %d devices", dev, kMaxDevices);
    if (!g_static_ready[dev].load(std::memory_order_acquire)) {
        std::lock_guard<std::mutex> lock(g_static_mu);
        if (!g_static_ready[dev].load(std::memory_order_relaxed)) {
            StaticDev sd;
            void* ptr = nullptr;
            hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
            if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
            sd.ptr = static_cast<uint32_t*>(ptr);
            sd.lds = lds_limit_of(dev);
            sd.cap_n = capacity_for(sd.lds);
            if ((e = hipDeviceGetAttribute(&sd.cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess)
                return hip_fail(e, "hipDeviceGetAttribute");
            if ((e = tr::select_prepare(sd.lds)) != hipSuccess) return hip_fail(e, "hipFuncSetAttribute");
            hipLaunchKernelGGL(fill_kernel, dim3(1024), dim3(256), 0, stream, sd.ptr, (int64_t)kStaticWords, 0u);
            if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "scratch clear launch");
            g_static[dev] = sd;
            g_static_ready[dev].store(1, std::memory_order_release);
        }
    }
    out = &g_static[dev];
    return TR_OK;
}

}  // namespace

extern "C" tr_status tr_reduce_noalloc(const tr_params* p, const void* X, const void* X_pre, const void* X_post,
                                       int32_t B, const int32_t* N, const int32_t* K, void* out,
                                       int32_t* out_idx, uint8_t* out_src, float* out_h2, float* out_s,
                                       void* stream)
{
    clear_error();
    tr_status st = check_params(p, false);
    if (st != TR_OK) return st;
    if (p->flags & TR_FLAG_CHECK_FINITE)
        return fail(TR_EUNSUPPORTED, "TR_FLAG_CHECK_FINITE needs a context (tr_create) to hold its count");
    if (B > kStaticImages)
        return fail(TR_EINVAL, "B = %d exceeds the %d images of the no-allocation scratch", B, kStaticImages);
    if (B > 0 && N) {
        int64_t rows = 0;
        for (int32_t b = 0; b < B; ++b) rows += N[b] > 0 ? N[b] : 0;
        if (rows > kStaticTokens)
            return fail(TR_EINVAL, "sum of N = %lld exceeds the %lld tokens of the no-allocation scratch",
                        (long long)rows, (long long)kStaticTokens);
    }
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    const StaticDev* sd = nullptr;
    if ((st = static_setup(dev, static_cast<hipStream_t>(stream), sd)) != TR_OK) return st;

    // A context view on the device's copy of the array (allocates nothing).
    tr_ctx c;
    c.p = *p;
    c.p.max_images = kStaticImages;
    c.p.max_tokens = kStaticTokens;
    c.p.max_N = p->max_N > 0 ? p->max_N : 0;
    c.device = dev;
    c.Dc = p->Dc ? p->Dc : p->D;
    c.eb = elem_bytes(p->dtype);
    c.lds_limit = sd->lds;
    c.cap_n = sd->cap_n;
    c.cus = sd->cus;
    uint32_t* base = sd->ptr;
    c.key_imp = reinterpret_cast<float*>(base);
    c.key_s = reinterpret_cast<float*>(base + kStaticTokens);
    c.rows = reinterpret_cast<int32_t*>(base + 2 * kStaticTokens);
    c.gsel = base + 3 * kStaticTokens;
    c.gimp = c.gsel + kStaticGselWords;

    ReduceCall r;
    r.X = X;
    r.X_pre = X_pre;
    r.X_post = X_post;
    r.B = B;
    r.N = N;
    r.K = K;
    r.out = out;
    r.out_idx = out_idx;
    r.out_src = out_src;
    r.out_h2 = out_h2;
    r.out_s = out_s;
    r.stream = stream;
    return reduce_impl(&c, r);
}
