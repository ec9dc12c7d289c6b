// Host-only part of the library: parameter checks, the budget plan of
// Algorithm 1 and the synchronous argument rules of a reduce call.  Plain
// C++ with no HIP dependency, so it also builds on its own (with the host
// sanitizers) for testing.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <vector>

#include "tr.h"

namespace tr {

struct ImageDesc {
    int32_t row_off;     // first row of the image in the packed batch
    int32_t n;           // tokens
    int32_t k1;          // Stage I budget
    int32_t k2;          // Stage II budget
    int32_t t;           // stride (>= 1 when k2 > 0)
    int32_t out_off;     // first output slot
};

// Per-image descriptors of a call: held inline up to kInlineImages (so a
// call of that size allocates no host memory), on the heap beyond.
constexpr size_t kInlineImages = 256;

struct DescList {
    ImageDesc local[kInlineImages];
    std::vector<ImageDesc> heap;
    ImageDesc* p = local;
    size_t n = 0;
    void resize(size_t k)
    {
        if (k > kInlineImages) {
            heap.resize(k);
            p = heap.data();
        } else {
            p = local;
        }
        n = k;
    }
    size_t size() const { return n; }
    ImageDesc& operator[](size_t i) { return p[i]; }
    const ImageDesc& operator[](size_t i) const { return p[i]; }
};

struct Plan {
    DescList desc;
    int64_t sum_n = 0;
    int64_t sum_k = 0;
    int nmax = 0;
    bool uniform = true;
    bool keys_imp = false;   // some image's Stage I depends on the key order (0 < K1 < N)
    bool keys_s = false;     // some image's Stage II does (0 < K2 < N - K1)
};

// Latest failure of the calling thread, kept in a fixed buffer (reporting
// allocates nothing).  With the environment variable TR_LOG = 1 every failure
// is also written to stderr as one line, and log_line writes other lines
// (context creation); otherwise the library prints nothing.
void clear_error();
tr_status fail(tr_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
const char* last_error();
void log_line(const char* fmt, ...) __attribute__((format(printf, 1, 2)));

int elem_bytes(int32_t dtype);

// Checks of the problem statement shared by tr_create, tr_plan and the
// context-free calls; need_caps also requires the capacity fields.
tr_status check_params(const tr_params* p, bool need_caps);

// Algorithm 1, step 1 (K1 = floor(lambda K) in double, K2 = K - K1) and the
// stride t = max(1, floor((N - K1) / K2)) for every image, with every
// per-image check; capacities of p apply where they are > 0.
tr_status make_plan(const tr_params* p, int32_t B, const int32_t* N, const int32_t* K, Plan& out);

// The pointers of one reduce call.  check_call applies the rules tr_reduce
// states for them (after a plan with B > 0) and decides which scores the
// call computes: Stage I's when some image ranks by it or H2 is asked for,
// Stage II's likewise, unless its key is supplied.  A score that is not
// computed has its inputs cleared here, so they are never read.
struct CallPtrs {
    const void* X = nullptr;
    const void* X_pre = nullptr;
    const void* X_post = nullptr;
    const float* key_s = nullptr;   // supplied Stage II key, or nullptr
    const void* out = nullptr;
    const int32_t* out_idx = nullptr;
    const uint8_t* out_src = nullptr;
    const float* out_h2 = nullptr;
    const float* out_s = nullptr;
};

tr_status check_call(const tr_params* p, const Plan& pl, CallPtrs& r, bool& need_x, bool& need_c);

}  // namespace tr
