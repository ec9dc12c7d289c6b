// Internal declarations shared by the library's translation units (never by
// the oracle).  Kernels are launched only from the file that defines them.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "tr_plan.h"
#include "tr_score.h"

namespace tr {

// ---- per-image selection (top-K1, ordered remainder, sort, stride) --------
constexpr int kMaxDescPerLaunch = 32;

struct SelectArgs {
    const float* key_imp;   // packed [sum N]
    const float* key_s;     // packed [sum N]
    int32_t* out_idx;       // packed [sum K], image-local
    uint8_t* out_src;       // packed [sum K] or nullptr
    int32_t* out_rows;      // packed [sum K] global row of each kept token, or nullptr
    uint32_t* gsel;         // per-image pick bitmaps of split images (zero between calls)
    uint32_t* gimp;         // per-image X^imp bitmaps of split images
    int32_t uniform;        // 1: desc[0] holds n/k1/k2/t of every image
    int32_t nimg;           // images in this launch
    int32_t img0;           // index of the first image of this launch in the batch
    int32_t groups;         // workgroups per image (1, or more to split large images)
    int32_t stride_real;    // 1: X^div at floor(j R / K2) instead of j t
    // Gather fused into the small-image selection (images of at most
    // kSmallSelectN tokens): the kept rows of gX go to gout in output order.
    const void* gX;         // [sum N] rows of grow_bytes, or nullptr: no fused gather
    void* gout;             // [sum K] rows of grow_bytes
    int64_t grow_bytes;
    int32_t gvec;           // 1: 16-byte copies (bases and row pitch 16-byte aligned)
    int32_t gelem;          // element bytes (2 or 4) of the element-wise copy
    int32_t ggroups;        // workgroups per image of the small-image selection (>= 1)
    ImageDesc desc[kMaxDescPerLaunch];
};

// Images of at most this many tokens are selected one token per thread, and
// can have their gather fused into the selection.
constexpr int kSmallSelectN = 1024;
// Workgroups per image of the small-image selection when it also gathers:
// each repeats the (cheap) selection and copies a share of the kept rows.
int select_small_groups(int images, int k_min, int cus);

// Words of the split-image pick bitmaps for capacity (max_tokens, max_images).
size_t select_gsel_words(int64_t max_tokens, int max_images);
// Whether an image's selection is shared by several workgroups when its
// launch has more than one workgroup per image (large remainders).
bool select_shares(const ImageDesc& d);
// Workgroups per image for a launch with n_large such images on a device of
// `cus` compute units: the largest power of two (at most 64) with which they
// still fit the compute units in one round; 1 without such images.
int select_groups(int64_t n_large, int cus);

// Threads per selection workgroup for images of at most nmax tokens.
int select_threads(int nmax);
// Dynamic LDS bytes the selection needs for an image of n tokens.
size_t select_lds_bytes(int n, int threads);
hipError_t select_prepare(int lds_limit);
hipError_t launch_select(const SelectArgs& a, int nmax, hipStream_t s);

// ---- gather of kept rows ---------------------------------------------------
// rows[r] outside [0, nrows) are skipped (their output row is left as is).
hipError_t launch_gather(const void* X, void* out, const int32_t* rows, int64_t nout, int64_t nrows,
                         int64_t row_bytes, int elem_bytes, bool vec, hipStream_t s);

// ---- measurement: streaming-read ceiling --------------------------------------
// Reads bytes / 16 chunks of p (16-byte aligned) once; at most sink_words
// workgroups, each of which may write sink[its index].
// Buffers of one read-ceiling launch (at most kReadBuffers, each a whole
// number of 16-byte chunks; span_end: running count of 8 KB spans).
constexpr int kReadBuffers = 8;
struct ReadSet {
    const void* p[kReadBuffers];
    int64_t chunks[kReadBuffers];
    int64_t span_end[kReadBuffers];
    int n;
};
hipError_t launch_read(const void* const* p, const int64_t* bytes, int n, uint32_t* sink, int sink_words,
                       hipStream_t s);

// ---- bf16 matrix-core GEMM: C[M, N] = A[M, K] . B[N, K]^T -----------------
struct GemmArgs {
    const void* A;           // bf16, row m at A + row * lda (16-byte aligned rows)
    const int32_t* arows;    // [M] row of A for each row of C (gather), or nullptr: row m
    int64_t arow_count;      // rows of A (gathered indices outside [0, count) read as zeros)
    const void* B;           // bf16 [N, K], row stride ldb (16-byte aligned rows)
    void* C;                 // bf16 [M, N], row stride ldc
    int32_t M, N, K;         // N % 128 == 0, K % 64 == 0
    int64_t lda, ldb, ldc;   // elements
    const void* P;           // bf16 [M, N] (stride ldp) for the cosine epilogue, or nullptr
    int64_t ldp;
    float* part;             // [M, part_cols, 3] cosine partials (with P)
    int32_t part_cols;       // row stride of part: N / 128 (the wide kernel fills N / 256)
    float* s_out;            // [M] cosine of the rows of P and C (with P)
};

bool gemm_shape_ok(int M, int N, int K);
int gemm_part_cols(int N);
hipError_t gemm_prepare();
hipError_t launch_gemm(const GemmArgs& a, hipStream_t s);

}  // namespace tr
