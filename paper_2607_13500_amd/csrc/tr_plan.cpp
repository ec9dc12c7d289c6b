// Host-only part of the library (see tr_plan.h): parameter checks, the budget
// plan of Algorithm 1, the synchronous argument rules of a reduce call, and
// the error reporting of the C ABI.  No HIP dependency.
#include "tr_plan.h"

#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

namespace tr {

namespace {
thread_local char g_err[512];
}  // namespace

void clear_error() { g_err[0] = '\0'; }

bool log_enabled()
{
    const char* v = getenv("TR_LOG");
    return v && strcmp(v, "1") == 0;
}

void log_line(const char* fmt, ...)
{
    if (!log_enabled()) return;
    char line[640];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(line, sizeof line, fmt, ap);
    va_end(ap);
    fprintf(stderr, "tr: %s\n", line);
}

tr_status fail(tr_status st, const char* fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    if (log_enabled()) fprintf(stderr, "tr: %s: %s\n", tr_strerror(st), g_err);
    return st;
}

const char* last_error() { return g_err; }

int elem_bytes(int32_t dtype) { return dtype == TR_BF16 ? 2 : 4; }

tr_status check_params(const tr_params* p, bool need_caps)
{
    if (!p) return fail(TR_EINVAL, "params is NULL");
    if (p->D <= 0) return fail(TR_EINVAL, "D must be > 0 (got %d)", p->D);
    if (p->Dc < 0) return fail(TR_EINVAL, "Dc must be >= 0 (got %d)", p->Dc);
    if (p->dtype != TR_FP32 && p->dtype != TR_BF16)
        return fail(TR_EINVAL, "dtype must be TR_FP32 or TR_BF16 (got %d)", p->dtype);
    if (p->flags & ~(int32_t)(TR_FLAG_STRIDE_REAL | TR_FLAG_SHANNON | TR_FLAG_CHECK_FINITE))
        return fail(TR_EINVAL, "unknown flags 0x%x", (unsigned)p->flags);
    if (!(p->lambda >= 0.0 && p->lambda <= 1.0))
        return fail(TR_EINVAL, "lambda must be in [0, 1] (got %g)", p->lambda);
    if (!(p->keep_ratio == 0.0 || (p->keep_ratio > 0.0 && p->keep_ratio <= 1.0)))
        return fail(TR_EINVAL, "keep_ratio must be 0 (unused) or in (0, 1] (got %g)", p->keep_ratio);
    const int64_t eb = elem_bytes(p->dtype);
    const int64_t dc = p->Dc ? p->Dc : p->D;
    if ((int64_t)p->D * eb > (int64_t)INT32_MAX || dc * eb > (int64_t)INT32_MAX)
        return fail(TR_EINVAL, "row too wide");
    if (need_caps) {
        if (p->max_images < 1) return fail(TR_EINVAL, "max_images must be >= 1");
        if (p->max_tokens < 1 || p->max_tokens > (int64_t)INT32_MAX)
            return fail(TR_EINVAL, "max_tokens must be in [1, 2^31 - 1]");
        if (p->max_N < 1) return fail(TR_EINVAL, "max_N must be >= 1");
    }
    return TR_OK;
}

tr_status make_plan(const tr_params* p, int32_t B, const int32_t* N, const int32_t* K, Plan& out)
{
    if (B < 0) return fail(TR_EINVAL, "B must be >= 0 (got %d)", B);
    if (p->max_images > 0 && B > p->max_images)
        return fail(TR_EINVAL, "B = %d exceeds max_images = %d", B, p->max_images);
    if (B > 0 && !N) return fail(TR_EINVAL, "N is NULL");
    if (B > 0 && !K && !(p->keep_ratio > 0.0))
        return fail(TR_EINVAL, "K is NULL and no keep_ratio was set");
    out.desc.resize((size_t)B);
    int64_t rows = 0, outs = 0;
    for (int32_t b = 0; b < B; ++b) {
        const int32_t n = N[b];
        if (n < 1) return fail(TR_EINVAL, "N[%d] = %d must be >= 1", b, n);
        if (n > 65535) return fail(TR_EINVAL, "N[%d] = %d exceeds 65535", b, n);
        if (p->max_N > 0 && n > p->max_N)
            return fail(TR_EINVAL, "N[%d] = %d exceeds max_N = %d", b, n, p->max_N);
        int32_t k;
        if (K) {
            k = K[b];
        } else {
            const double kr = floor(p->keep_ratio * (double)n);
            k = kr < 1.0 ? 1 : (kr > (double)n ? n : (int32_t)kr);
        }
        if (k < 1 || k > n) return fail(TR_EINVAL, "K[%d] = %d must be in [1, N = %d]", b, k, n);
        const int32_t k1 = (int32_t)floor(p->lambda * (double)k);
        const int32_t k2 = k - k1;
        int32_t t = 0;
        if (k2 > 0) {
            t = (n - k1) / k2;
            if (t < 1) t = 1;
        }
        ImageDesc& d = out.desc[(size_t)b];
        d.row_off = (int32_t)rows;
        d.n = n;
        d.k1 = k1;
        d.k2 = k2;
        d.t = t;
        d.out_off = (int32_t)outs;
        if (k1 > 0 && k1 < n) out.keys_imp = true;
        if (k2 > 0 && k2 < n - k1) out.keys_s = true;
        rows += n;
        outs += k;
        if (rows > (int64_t)INT32_MAX) return fail(TR_EINVAL, "sum of N exceeds 2^31 - 1");
        if (n > out.nmax) out.nmax = n;
        if (b > 0) {
            const ImageDesc& d0 = out.desc[0];
            if (d.n != d0.n || d.k1 != d0.k1 || d.k2 != d0.k2) out.uniform = false;
        }
    }
    if (p->max_tokens > 0 && rows > p->max_tokens)
        return fail(TR_EINVAL, "sum of N = %lld exceeds max_tokens = %lld", (long long)rows,
                    (long long)p->max_tokens);
    out.sum_n = rows;
    out.sum_k = outs;
    return TR_OK;
}

tr_status check_call(const tr_params* p, const Plan& pl, CallPtrs& r, bool& need_x, bool& need_c)
{
    if (!r.X || !r.out || !r.out_idx) return fail(TR_EINVAL, "X, out and out_idx must be non-NULL");
    need_x = pl.keys_imp || r.out_h2;
    need_c = !r.key_s && (pl.keys_s || r.out_s);
    if (need_c && (!r.X_pre || !r.X_post))
        return fail(TR_EINVAL, "X_pre and X_post must be non-NULL when Stage II ranks tokens or out_s is set");
    if (!need_c) r.X_pre = r.X_post = nullptr;
    const uintptr_t em = (uintptr_t)elem_bytes(p->dtype) - 1;
    if (((uintptr_t)r.X | (uintptr_t)r.X_pre | (uintptr_t)r.X_post | (uintptr_t)r.out) & em)
        return fail(TR_EUNSUPPORTED, "X, X_pre, X_post and out must be aligned to the element size (%d bytes)",
                    elem_bytes(p->dtype));
    if (((uintptr_t)r.out_idx | (uintptr_t)r.out_h2 | (uintptr_t)r.out_s | (uintptr_t)r.key_s) & 3u)
        return fail(TR_EUNSUPPORTED, "out_idx, out_h2, out_s and key_s must be 4-byte aligned");
    return TR_OK;
}

}  // namespace tr

extern "C" {

const char* tr_strerror(tr_status s)
{
    switch (s) {
    case TR_OK: return "success";
    case TR_EINVAL: return "invalid argument";
    case TR_ENOMEM: return "out of memory";
    case TR_EUNSUPPORTED: return "unsupported request";
    case TR_EDEVICE: return "HIP device error";
    }
    return "unknown status";
}

const char* tr_last_error(void) { return tr::last_error(); }

tr_status tr_plan(const tr_params* p, int32_t B, const int32_t* N, const int32_t* K, int32_t* Kout,
                  int32_t* K1out, int32_t* K2out, int32_t* tout)
{
    tr::clear_error();
    tr_status st = tr::check_params(p, false);
    if (st != TR_OK) return st;
    tr::Plan pl;
    st = tr::make_plan(p, B, N, K, pl);
    if (st != TR_OK) return st;
    for (int32_t b = 0; b < B; ++b) {
        const tr::ImageDesc& d = pl.desc[(size_t)b];
        if (Kout) Kout[b] = d.k1 + d.k2;
        if (K1out) K1out[b] = d.k1;
        if (K2out) K2out[b] = d.k2;
        if (tout) tout[b] = d.t;
    }
    return TR_OK;
}

tr_status tr_check_reduce(const tr_params* p, const void* X, const void* X_pre, const void* X_post, int32_t B,
                          const int32_t* N, const int32_t* K, const void* out, const int32_t* out_idx,
                          const uint8_t* out_src, const float* out_h2, const float* out_s)
{
    tr::clear_error();
    tr_status st = tr::check_params(p, false);
    if (st != TR_OK) return st;
    tr::Plan pl;
    st = tr::make_plan(p, B, N, K, pl);
    if (st != TR_OK || B == 0) return st;
    tr::CallPtrs r;
    r.X = X;
    r.X_pre = X_pre;
    r.X_post = X_post;
    r.out = out;
    r.out_idx = out_idx;
    r.out_src = out_src;
    r.out_h2 = out_h2;
    r.out_s = out_s;
    bool need_x = false, need_c = false;
    return tr::check_call(p, pl, r, need_x, need_c);
}

}  // extern "C"
