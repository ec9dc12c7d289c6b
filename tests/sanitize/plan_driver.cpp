// Host-only driver of the library's planner (tr_plan.cpp), built with the
// address and undefined-behaviour sanitizers by tests/test_abi_host.py.  It
// runs tr_plan and tr_check_reduce over valid and invalid calls, checks the
// statuses and the plan's invariants, and exits non-zero on any mismatch (a
// sanitizer report aborts it).  Device pointers are never dereferenced by
// these calls, so plain integers stand in for them.
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <vector>

#include "tr.h"

namespace {

int failures = 0;

void expect(bool ok, const char* what, int line)
{
    if (!ok) {
        fprintf(stderr, "line %d: %s (last error: %s)\n", line, what, tr_last_error());
        ++failures;
    }
}
#define EXPECT(c) expect((c), #c, __LINE__)

tr_params params(int dtype, double lam)
{
    tr_params p;
    memset(&p, 0, sizeof p);
    p.D = 64;
    p.dtype = dtype;
    p.lambda = lam;
    return p;
}

const void* at(uintptr_t a) { return reinterpret_cast<const void*>(a); }

uint32_t lcg(uint32_t& s)
{
    s = s * 1664525u + 1013904223u;
    return s >> 8;
}

}  // namespace

int main()
{
    // The paper's budget: 64 + 128 of 192 at lambda = 1/3, stride over N - K1.
    {
        tr_params p = params(TR_BF16, 1.0 / 3.0);
        const int32_t N[3] = {576, 576, 2880};
        const int32_t K[3] = {192, 64, 320};
        int32_t Ko[3], K1[3], K2[3], t[3];
        EXPECT(tr_plan(&p, 3, N, K, Ko, K1, K2, t) == TR_OK);
        EXPECT(K1[0] == 64 && K2[0] == 128 && t[0] == 4);
        EXPECT(K1[1] == 21 && K2[1] == 43 && t[1] == 12);
        EXPECT(K1[2] == 106 && K2[2] == 214 && t[2] == 12);
    }
    // Random batches, above and below the inline descriptor storage, with K
    // given or from a keep ratio: invariants of every image's plan.
    uint32_t seed = 7;
    for (int trial = 0; trial < 400; ++trial) {
        const int B = 1 + (int)(lcg(seed) % (trial % 10 == 0 ? 700 : 40));
        std::vector<int32_t> N(B), K(B), Ko(B), K1(B), K2(B), t(B);
        for (int b = 0; b < B; ++b) {
            N[b] = 1 + (int32_t)(lcg(seed) % 20000);
            K[b] = 1 + (int32_t)(lcg(seed) % (uint32_t)N[b]);
        }
        tr_params p = params(trial & 1 ? TR_FP32 : TR_BF16, (lcg(seed) % 1001) / 1000.0);
        const bool ratio = trial % 3 == 0;
        if (ratio) p.keep_ratio = (1 + lcg(seed) % 1000) / 1000.0;
        EXPECT(tr_plan(&p, B, N.data(), ratio ? nullptr : K.data(), Ko.data(), K1.data(), K2.data(), t.data()) ==
               TR_OK);
        for (int b = 0; b < B; ++b) {
            EXPECT(Ko[b] >= 1 && Ko[b] <= N[b] && K1[b] + K2[b] == Ko[b] && K1[b] >= 0 && K2[b] >= 0);
            EXPECT(K2[b] == 0 ? t[b] == 0 : (t[b] >= 1 && (int64_t)(K2[b] - 1) * t[b] < N[b] - K1[b]));
            if (!ratio) EXPECT(Ko[b] == K[b]);
        }
    }
    // Invalid calls: statuses and messages (long values exercise the fixed
    // error buffer).
    {
        tr_params p = params(TR_BF16, 0.5);
        const int32_t N[2] = {10, 65536}, K[2] = {11, 1};
        EXPECT(tr_plan(&p, 1, N, K, nullptr, nullptr, nullptr, nullptr) == TR_EINVAL);
        EXPECT(strstr(tr_last_error(), "K[0]") != nullptr);
        EXPECT(tr_plan(&p, 2, N, nullptr, nullptr, nullptr, nullptr, nullptr) == TR_EINVAL);
        EXPECT(tr_plan(&p, -1, N, K, nullptr, nullptr, nullptr, nullptr) == TR_EINVAL);
        EXPECT(tr_plan(nullptr, 1, N, K, nullptr, nullptr, nullptr, nullptr) == TR_EINVAL);
        p.lambda = 1.5;
        EXPECT(tr_plan(&p, 1, N, K, nullptr, nullptr, nullptr, nullptr) == TR_EINVAL);
        p.lambda = 0.5;
        p.flags = 0x40;
        EXPECT(tr_plan(&p, 1, N, K, nullptr, nullptr, nullptr, nullptr) == TR_EINVAL);
        p.flags = 0;
        p.D = 0x7fffffff;
        EXPECT(tr_plan(&p, 1, N, K, nullptr, nullptr, nullptr, nullptr) == TR_EINVAL);
        p.D = 64;
        p.max_tokens = 5;
        const int32_t N2[1] = {6}, K2[1] = {3};
        EXPECT(tr_plan(&p, 1, N2, K2, nullptr, nullptr, nullptr, nullptr) == TR_EINVAL);
        EXPECT(strstr(tr_last_error(), "max_tokens") != nullptr);
    }
    // tr_check_reduce: pointer presence and the alignment rule.
    {
        const uintptr_t g = 0x100000;
        const int32_t N[2] = {100, 50}, K[2] = {10, 5};
        for (int dtype = 0; dtype < 2; ++dtype) {
            tr_params p = params(dtype, 1.0 / 3.0);
            const uintptr_t e = dtype == TR_BF16 ? 2 : 4;
            auto chk = [&](uintptr_t X, uintptr_t P, uintptr_t Q, uintptr_t out, uintptr_t idx, uintptr_t h2) {
                return tr_check_reduce(&p, at(X), at(P), at(Q), 2, N, K, at(out),
                                       static_cast<const int32_t*>(at(idx)), nullptr,
                                       static_cast<const float*>(at(h2)), nullptr);
            };
            EXPECT(chk(g, g, g, g, g, 0) == TR_OK);
            EXPECT(chk(g + e, g + 3 * e, g, g + e, g, 0) == TR_OK);   // element-aligned: scalar path
            EXPECT(chk(g + 1, g, g, g, g, 0) == TR_EUNSUPPORTED);
            EXPECT(chk(g, g + 1, g, g, g, 0) == TR_EUNSUPPORTED);
            EXPECT(chk(g, g, g + 1, g, g, 0) == TR_EUNSUPPORTED);
            EXPECT(chk(g, g, g, g + 1, g, 0) == TR_EUNSUPPORTED);
            EXPECT(chk(g, g, g, g, g + 2, 0) == TR_EUNSUPPORTED);
            EXPECT(chk(g, g, g, g, g, g + 2) == TR_EUNSUPPORTED);
            EXPECT(chk(0, g, g, g, g, 0) == TR_EINVAL);
            EXPECT(chk(g, 0, g, g, g, 0) == TR_EINVAL);
            EXPECT(chk(g, g, g, 0, g, 0) == TR_EINVAL);
            EXPECT(chk(g, g, g, g, 0, 0) == TR_EINVAL);
            p.lambda = 1.0;   // no Stage II: X_pre / X_post are neither needed nor checked
            EXPECT(chk(g, 0, 0, g, g, 0) == TR_OK);
            EXPECT(chk(g, g + 1, g + 1, g, g, 0) == TR_OK);
            EXPECT(tr_check_reduce(&p, nullptr, nullptr, nullptr, 0, nullptr, nullptr, nullptr, nullptr, nullptr,
                                   nullptr, nullptr) == TR_OK);   // B = 0 is a no-op
        }
    }
    if (failures) {
        fprintf(stderr, "%d failures\n", failures);
        return 1;
    }
    printf("planner ok\n");
    return 0;
}
