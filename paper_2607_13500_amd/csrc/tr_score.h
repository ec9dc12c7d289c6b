// Interface of the scoring kernel (Eq. 3-4 and Eq. 6, one wavefront per
// token row).  Kept apart from the other kernels' declarations so that the
// scoring kernel's sources are exactly tr_score.hip, this file and tr_wave.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tr {

constexpr int kWave = 64;

struct ScoreArgs {
    const void* X;       // [rows, D]
    const void* P;       // [rows, Dc] pre-MLP states
    const void* Q;       // [rows, Dc] post-MLP states
    int64_t rows;
    int32_t D;
    int32_t Dc;
    float* key_imp;      // [rows] CV^2 of |x| (Shannon: log D - H1) (Stage I key, ascending), or nullptr
    float* key_s;        // [rows] s (Stage II key, ascending), or nullptr
    float* out_h2;       // [rows] H2 (Shannon: H1), or nullptr
    float* out_s;        // [rows] or nullptr
    float logD;          // log(D) in fp32
    uint32_t* nonfinite; // one is added per row holding a NaN or infinite element among the
                         // tensors the launch reads, or nullptr: no count
};

// Which scores a launch computes (a bit set, never 0).  A score left out
// reads nothing: its key (if the pointer is set) is written as 0, and its
// optional output is not written.
constexpr int kScoreImp = 1;   // Eq. (3)-(4) from X: key_imp, out_h2
constexpr int kScoreSim = 2;   // Eq. (6) from X_pre, X_post: key_s, out_s
constexpr int kScoreShannon = 4;   // with kScoreImp: Shannon variant (key KL = log D - H1, out H1)

// bf16: true for bfloat16 rows, false for fp32.  vec: every row start is
// 16-byte aligned (vector loads); otherwise element loads with the same
// per-lane arithmetic order.
hipError_t launch_score(const ScoreArgs& a, bool bf16, bool vec, int mode, hipStream_t s);

}  // namespace tr
