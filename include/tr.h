/*
 * tr.h - C ABI of the MI355X (gfx950) ALTR visual-token reduction library.
 *
 * The operation (the paper's Sec. "Methodology", Eq. (3)-(7), Algorithm 1):
 * for every image b of a packed batch with N_b tokens x_i (rows of X) and the
 * pre-/post-MLP states x'_i, x''_i of the vision encoder's last MLP (rows of
 * X_pre and X_post, Eq. (5)), keep K_b tokens:
 *   1. K1 = floor(lambda K_b), K2 = K_b - K1                  (Algorithm 1)
 *   2. H2(x_i) = -log sum_j p_ij^2, p_ij = |x_ij| / sum_k |x_ik|   (Eq. 3-4)
 *   3. X^imp = the K1 tokens of highest H2 (ties: lower index)
 *   4. s_i = cos(x'_i, x''_i)                                      (Eq. 6)
 *   5. sort X^rem = X \ X^imp by s ascending (ties: lower index first)
 *   6. t = max(1, floor(|X^rem| / K2)); X^div = sorted positions 0, t, ...,
 *      (K2-1) t                                                (Algorithm 1)
 *   7. X* = X^imp U X^div (Eq. 7), listed in ascending token index, and the
 *      kept rows of X gathered into a compact output.
 *
 * Readings where the paper is silent: natural log; an all-zero row of X has
 * H2 = 0; a zero-norm x' or x'' gives s = 0; non-finite inputs give
 * unspecified (but memory-safe) results.
 *
 * Arithmetic: scores are accumulated in fp32 from exactly widened inputs.
 * Stage I ranks by the squared coefficient of variation of |x| (CV^2), which
 * orders tokens exactly as H2 does (H2 = log D - log(1 + CV^2)) and keeps
 * near-uniform rows apart in fp32.  Selection and gather are exact integer
 * and byte work.  A token row's scores depend only on its own bytes, so
 * identical rows tie exactly and resolve by index.
 *
 * Memory: every pointer named "device" is HIP device memory on the device
 * that was current at tr_create; host arrays are read during the call only.
 * The caller owns all tensors; a context owns only the scratch it allocates
 * in tr_create (and the HIP events tr_timing_enable creates).  No other call
 * allocates memory (tr_reduce_noalloc works in a static device array of the
 * library instead of a context's scratch).
 *
 * Layout: rows are packed back to back.  Image b's rows start at
 * sum_{b' < b} N[b'] in X, X_pre, X_post (and the score outputs), and its
 * kept entries start at sum_{b' < b} K[b'] in out, out_idx, out_src.
 * Row widths: X and out have D elements, X_pre and X_post have Dc.
 *
 * Asynchrony: work is enqueued on `stream` (a hipStream_t; NULL = the null
 * stream) and the call returns before it completes.  Buffers must stay valid
 * until the stream reaches that point.  A context must not be used by two
 * threads or two streams at once (its scratch is shared); distinct contexts
 * are independent.
 *
 * Errors: argument and capacity errors return TR_EINVAL (or TR_EUNSUPPORTED)
 * synchronously with nothing enqueued.  TR_EDEVICE reports a HIP failure at
 * launch.  tr_last_error gives a one-line description of the latest failure.
 *
 * Environment (all optional, for diagnosis): TR_LOG = 1 writes every failure
 * (and a one-line description of each context at tr_create) to stderr; the
 * library prints nothing otherwise.  TR_ROCTX = 1 opens the roctx marker
 * library at the first call that enqueues work and brackets each call of
 * tr_reduce, tr_reduce_given_s, tr_reduce_project, tr_score, tr_select,
 * tr_gemm_bf16, tr_mlp_out_cos and tr_read_bandwidth in a range named after
 * the entry point, so that a profiler's marker trace ties every call to its
 * kernels.  TR_FAIL_ALLOC and
 * TR_GEMM_TILE_ROWS are test hooks described at tr_create and tr_gemm_bf16.
 *
 * Alignment: every tensor base must be aligned to its element size (2 bytes
 * for bf16, 4 for fp32 and for the int32 / float outputs); a base that is not
 * is an unsupported alignment, TR_EUNSUPPORTED.  Beyond that, 16-byte aligned
 * bases and row pitches take the vector path and others a scalar path with
 * bit-identical results.
 */
#ifndef TR_H
#define TR_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct tr_ctx tr_ctx;

typedef enum {
    TR_OK = 0,
    TR_EINVAL = 1,        /* bad argument, size or capacity                   */
    TR_ENOMEM = 2,        /* device or host allocation failed in tr_create    */
    TR_EUNSUPPORTED = 3,  /* valid request this build cannot serve            */
    TR_EDEVICE = 4        /* HIP runtime error                                */
} tr_status;

typedef enum {
    TR_FP32 = 0,          /* IEEE binary32 elements                           */
    TR_BF16 = 1           /* bfloat16 elements (upper half of a binary32)     */
} tr_dtype;

/* Variants of the method, OR-ed into tr_params.flags (0 = Algorithm 1). */
typedef enum {
    /* Step 6 with the real-valued interval R / K2 (R = N - K1) that the
     * method's prose states (Sec. "Methodology", diversity stage) instead of
     * Algorithm 1's integer stride: X^div = sorted positions floor(j R / K2),
     * j = 0 .. K2-1, which spreads the picks over the whole of X^rem. */
    TR_FLAG_STRIDE_REAL = 1,
    /* Stage I ranks by the Shannon entropy H1 = -sum_j p_j log p_j of the
     * same distribution p (Eq. (3); 0 log 0 = 0, an all-zero row has H1 = 0)
     * instead of Eq. (4)'s Renyi-2 entropy: the measure the paper names as
     * the one its score improves on (Sec. "Stage I").  The Stage I key is
     * then KL = log D - H1 (ascending = descending H1) and out_h2 receives
     * H1.  Costs a logarithm per element of X. */
    TR_FLAG_SHANNON = 2,
    /* Count the scored rows that hold a NaN or an infinite element (the
     * paper defines the scores for finite tokens only; such rows still get
     * memory-safe, unspecified keys).  The context keeps a device count,
     * zero at tr_create, to which every scoring launch (tr_reduce and its
     * fused forms, tr_score) adds one per row that holds a non-finite
     * element in a tensor the launch reads: X when H2 is computed, X_pre or
     * X_post when s is computed (a row counts once).  tr_nonfinite_rows
     * reads it.  Finite rows cost nothing extra: a non-finite element always
     * sends its row to the scoring kernel's second read, where the check is
     * made.  Not available to tr_reduce_noalloc (TR_EUNSUPPORTED). */
    TR_FLAG_CHECK_FINITE = 4
} tr_flag;

/* Problem statement and capacities, fixed for the life of a context. */
typedef struct {
    int32_t D;            /* elements per row of X and out (> 0)                   */
    int32_t Dc;           /* elements per row of X_pre / X_post; 0 means D          */
    int32_t dtype;        /* tr_dtype of X, X_pre, X_post and out                  */
    int32_t max_images;   /* largest B accepted by tr_reduce / tr_select (>= 1)     */
    int64_t max_tokens;   /* largest sum of N[b] accepted (>= 1, < 2^31)            */
    int32_t max_N;        /* largest single N[b] accepted (>= 1)                    */
    int32_t flags;        /* OR of tr_flag values; 0 = the method as Algorithm 1 states */
    double lambda;        /* balance factor in [0, 1] (Algorithm 1; the paper's
                             efficiency setting is 1/3: 64 + 128 of 192)            */
    double keep_ratio;    /* used when K == NULL: K_b = clamp(floor(keep_ratio N_b),
                             1, N_b); must be in (0, 1] if used, else ignored      */
} tr_params;

/* Create a context on the current HIP device: validates p, allocates scratch
 * for max_tokens tokens (12 bytes each: two keys and a row index, plus two
 * bits each for the pick bitmaps of images shared by several workgroups; a
 * bf16 context with Dc a multiple of 128 also holds 12 x Dc / 128 bytes per
 * token for tr_mlp_out_cos's per-tile partial sums) and checks that max_N
 * fits the per-image selection's on-chip memory.  Returns TR_EINVAL for a bad
 * field, TR_EUNSUPPORTED when max_N exceeds the selection capacity
 * (tr_capacity_N), TR_ENOMEM or TR_EDEVICE on runtime failure.  *out is NULL
 * on failure and nothing stays allocated.  Test hook: the environment
 * variable TR_FAIL_ALLOC = k (k >= 1) makes the k-th device allocation of
 * each tr_create call fail as if the device were out of memory. */
tr_status tr_create(const tr_params* p, tr_ctx** out);

/* The whole module (steps 1-7 above) on a packed batch of B images.
 *   X      device [sum N, D]   tokens scored by Eq. (3)-(4) and gathered
 *   X_pre  device [sum N, Dc]  pre-MLP states x'  (Eq. 5-6), or NULL (below)
 *   X_post device [sum N, Dc]  post-MLP states x'' (Eq. 5-6), or NULL (below)
 *   B      number of images, 0 <= B <= max_images (B = 0 is a no-op)
 *   N      host [B], 1 <= N[b] <= max_N, sum N <= max_tokens
 *   K      host [B] with 1 <= K[b] <= N[b], or NULL to use keep_ratio
 *   out    device [sum K, D]   kept rows of X, byte copies, ascending index
 *   out_idx device int32 [sum K] kept token indices, image-local, strictly
 *          ascending within an image
 *   out_src device uint8 [sum K] or NULL: 0 = kept by Stage I, 1 = Stage II
 *   out_h2 device float [sum N] or NULL: H2 of every token (nats; H1 with
 *          TR_FLAG_SHANNON)
 *   out_s  device float [sum N] or NULL: s of every token
 *   stream hipStream_t or NULL
 * Bases not aligned to their element size give TR_EUNSUPPORTED (see
 * Alignment above).
 * A score that decides nothing is not computed and its inputs are not read:
 * H2 when every image has K1 = 0 or K1 = N (lambda = 0, the paper's ablation
 * without the importance stage) and out_h2 is NULL; s when every image has
 * K2 = 0 or K2 = N - K1 (lambda = 1, the ablation without the diversity
 * stage) and out_s is NULL.  In the latter case X_pre and X_post may be NULL
 * (and are ignored if given); otherwise NULL gives TR_EINVAL.  The kept set
 * is the same as with both scores computed. */
tr_status tr_reduce(tr_ctx* ctx, const void* X, const void* X_pre,
                    const void* X_post, int32_t B, const int32_t* N,
                    const int32_t* K, void* out, int32_t* out_idx,
                    uint8_t* out_src, float* out_h2, float* out_s,
                    void* stream);

/* Step 2 and step 4 alone (Eq. 3-4 and Eq. 6) over `rows` packed rows, with
 * the same kernel and bit-identical results as inside tr_reduce.
 *   key_imp device float [rows]: the Stage I key CV^2 = Var|x| / mean|x|^2
 *           (population variance over the D channels), D - 1 for an all-zero
 *           row; ascending CV^2 is descending H2.  With TR_FLAG_SHANNON:
 *           KL = log D - H1 (log D for an all-zero row)
 *   key_s   device float [rows]: s (Eq. 6)
 *   out_h2  device float [rows] or NULL: H2 = log D - log1p(CV^2) (with
 *           TR_FLAG_SHANNON: H1 = log D - KL)
 * Either score may be left out: X, key_imp (and out_h2) all NULL computes s
 * alone; X_pre, X_post and key_s all NULL computes the Stage I key alone.
 * A partly given group, or nothing to compute, is TR_EINVAL.
 * rows may be any value >= 0 (no capacity applies). */
tr_status tr_score(tr_ctx* ctx, const void* X, const void* X_pre,
                   const void* X_post, int64_t rows, float* key_imp,
                   float* key_s, float* out_h2, void* stream);

/* Steps 1, 3, 5, 6 and 7 (without the row gather) from given per-token keys:
 * the same selection tr_reduce runs, for callers that already hold scores.
 *   key_imp device float [sum N]: Stage I key, SMALLER is more important
 *           (tr_reduce uses CV^2; -H2 gives the same order)
 *   key_s   device float [sum N]: Stage II key (s), sorted ascending
 *   B, N, K as in tr_reduce; out_idx, out_src as in tr_reduce.
 * Keys are compared as IEEE values (-0 == +0); ties resolve by index.  NaN
 * keys give unspecified (memory-safe) order. */
tr_status tr_select(tr_ctx* ctx, const float* key_imp, const float* key_s,
                    int32_t B, const int32_t* N, const int32_t* K,
                    int32_t* out_idx, uint8_t* out_src, void* stream);

/* ---- The steps around the path, fused with it (bf16 contexts only) ------
 *
 * Matrix-core GEMM C[M, N] = A[M, K] . B[N, K]^T in bf16 with fp32
 * accumulation and bf16 output (round to nearest even), the building block
 * of the two entry points below.
 *   A      device bf16, row m of the product is A + r * lda with r = m, or
 *          r = a_rows[m] when a_rows (device int32 [M]) is given; rows
 *          outside [0, a_row_count) read as zeros (memory-safe)
 *   B      device bf16 [N, K] (row stride ldb), e.g. a Linear layer's weight
 *   C      device bf16 [M, N] (row stride ldc)
 * N must be a multiple of 128 and K of 64, and ceil(M / 256) * N / 128 must
 * stay below 2^31 (else TR_EUNSUPPORTED); A and B bases and row strides must
 * be 16-byte aligned (else TR_EINVAL).  Every tiling the library picks for a
 * shape gives the same bits (one fp32 accumulation order per element).  The
 * environment variable TR_GEMM_TILE_ROWS = 128, 192 or 256, read by
 * tr_create, pins the tile height of the tiling used when N % 256 == 0 and
 * K % 128 == 0 (otherwise the height that fills the CUs best is taken). */
tr_status tr_gemm_bf16(tr_ctx* ctx, const void* A, int64_t lda,
                       const int32_t* a_rows, int64_t a_row_count,
                       const void* B, int64_t ldb, void* C, int64_t ldc,
                       int32_t M, int32_t N, int32_t K, void* stream);

/* The encoder MLP's second layer with Eq. (6) fused into its epilogue (Sec.
 * "Stage II": x' and x'' are the input and output of the last MLP, Eq. 5):
 *   X_post[M, Dc] = Hact[M, Hd] . W2[Dc, Hd]^T   (bf16 out, as tr_gemm_bf16)
 *   key_s[M]      = cos(X_pre[m], X_post[m]) of the X_post values as stored
 *                   (rounded to bf16), summed in fp32 while the tile is in
 *                   registers
 * so the Stage II key is ready without another pass over X_pre or X_post.
 * It is Eq. (6) of the X_post the caller receives, as tr_reduce's scoring
 * computes it up to the order of the fp32 sums.
 *   Hact   device bf16 [M, Hd] hidden activations sigma(W1 x'), row stride ldh
 *   W2     device bf16 [Dc, Hd], row stride ldw
 *   X_pre  device bf16 [M, Dc] (x'), X_post device bf16 [M, Dc] (written)
 *   key_s  device float [M] (written; zero norm -> 0)
 * Dc is the context's; it must be a multiple of 128, Hd of 64; M <=
 * max_tokens (the per-tile partial sums live in the context's scratch). */
tr_status tr_mlp_out_cos(tr_ctx* ctx, const void* Hact, int64_t ldh,
                         const void* W2, int64_t ldw, const void* X_pre,
                         void* X_post, int32_t M, int32_t Hd, float* key_s,
                         void* stream);

/* tr_reduce with the Stage II key supplied (e.g. by tr_mlp_out_cos): X is
 * scored for Stage I only, key_s (device float [sum N]) orders Stage II.
 * Other arguments as tr_reduce. */
tr_status tr_reduce_given_s(tr_ctx* ctx, const void* X, const float* key_s,
                            int32_t B, const int32_t* N, const int32_t* K,
                            void* out, int32_t* out_idx, uint8_t* out_src,
                            float* out_h2, void* stream);

/* tr_reduce whose last step projects the kept tokens instead of copying
 * them (the step after the path: the kept tokens go through the projector):
 *   out[k, :] = X[kept row k] . W^T, W device bf16 [Nout, D] (row stride ldw),
 *   out device bf16 [sum K, Nout]
 * The kept rows are read from X by the GEMM itself; no gathered copy is made.
 * Nout must be a multiple of 128 and D of 64.  Other arguments as tr_reduce
 * (X_pre / X_post may be NULL under the same rule). */
tr_status tr_reduce_project(tr_ctx* ctx, const void* X, const void* X_pre,
                            const void* X_post, int32_t B, const int32_t* N,
                            const int32_t* K, const void* W, int64_t ldw,
                            int32_t Nout, void* out, int32_t* out_idx,
                            uint8_t* out_src, void* stream);

/* Host-only check of a tr_reduce call (Algorithm 1's REQUIRE: 1 <= K_b <=
 * N_b, lambda in [0, 1]; and the argument rules above): the status tr_reduce
 * would return for these arguments, without a device or a context.  p's
 * capacity fields apply where they are > 0; the device's selection capacity
 * (tr_capacity_N) is not checked.  Pointers are only inspected, never
 * dereferenced. */
tr_status tr_check_reduce(const tr_params* p, const void* X, const void* X_pre, const void* X_post,
                          int32_t B, const int32_t* N, const int32_t* K, const void* out,
                          const int32_t* out_idx, const uint8_t* out_src, const float* out_h2,
                          const float* out_s);

/* Host-only budget plan (Algorithm 1, step 1 and the stride of step 6) with
 * the same validation tr_reduce applies; needs no device.  p may carry zero
 * capacities (then only the per-image rules are checked).  For each image
 * writes the kept count, K1, K2 and the stride t (0 when K2 = 0) into the
 * optional host arrays Kout, K1out, K2out, tout (each [B] or NULL). */
tr_status tr_plan(const tr_params* p, int32_t B, const int32_t* N,
                  const int32_t* K, int32_t* Kout, int32_t* K1out,
                  int32_t* K2out, int32_t* tout);

/* With TR_FLAG_CHECK_FINITE: enqueue on `stream` a copy of the context's
 * count of non-finite rows (see the flag) into *count (device uint32, 4-byte
 * aligned), and, if reset != 0, set the count back to 0 in the same launch.
 * Ordered with the caller's other work on `stream`, so the count covers the
 * calls enqueued before it on that stream.  TR_EUNSUPPORTED for a context
 * created without the flag. */
tr_status tr_nonfinite_rows(tr_ctx* ctx, uint32_t* count, int32_t reset, void* stream);

/* Largest N a context on the current device can select in on-chip memory. */
int32_t tr_capacity_N(void);

/* Per-stage kernel timing for measurement: when enabled, tr_reduce (and
 * tr_reduce_given_s, tr_reduce_project) records HIP events around its score,
 * select and gather (or projection) kernels on the caller's stream.
 * tr_timing_read waits for the recorded calls, writes the summed milliseconds
 * of each stage into ms[3] (score, select, gather) and the number of calls
 * into *calls, then clears the record.  At most 1024 calls are kept between
 * reads (later calls are not timed); a call that returns an error is not
 * counted. */
tr_status tr_timing_enable(tr_ctx* ctx, int32_t enable);
tr_status tr_timing_read(tr_ctx* ctx, double* ms, int64_t* calls);

/* Measurement hook: read n buffers (1 <= n <= 8; host arrays p of device
 * addresses, 16-byte aligned, and bytes, each a multiple of 16) once, in one
 * kernel launch on `stream`, with 16-byte non-temporal loads and nothing
 * else: the streaming-read ceiling the scoring kernel's bandwidth is compared
 * with (the scoring kernel also reads its three tensors in one launch).  sink
 * is device scratch of sink_words uint32 (>= 1) that the kernel may write;
 * its contents are meaningless.  Needs no context. */
tr_status tr_read_bandwidth(const void* const* p, const int64_t* bytes, int32_t n,
                            uint32_t* sink, int32_t sink_words, void* stream);

/* ---- For callers that cannot allocate ------------------------------------
 *
 * tr_reduce without a context, for code that must not allocate device memory:
 * work recorded under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc.  The problem statement comes in p as for tr_create (its
 * capacity fields are optional limits, 0 = none); every other argument is as
 * in tr_reduce, and the results are bit-identical to tr_reduce's with the same
 * p.  The scratch is a static device array of the library: 6.4 MB on each GPU
 * it runs on, held until the process ends, for at most TR_NOALLOC_MAX_TOKENS
 * tokens (sum of N) in at most TR_NOALLOC_MAX_IMAGES images; larger calls
 * return TR_EINVAL with nothing enqueued.  The call allocates no device or
 * host memory; the first call on a device also enqueues one clear of the
 * array (a kernel) on `stream`.  All calls on one GPU share that GPU's array
 * and its contents persist between calls: calls that overlap on one GPU (two
 * streams, two host threads) race and give undefined results, so callers
 * serialise them. */
#define TR_NOALLOC_MAX_TOKENS 524288
#define TR_NOALLOC_MAX_IMAGES 256
tr_status tr_reduce_noalloc(const tr_params* p, const void* X, const void* X_pre,
                            const void* X_post, int32_t B, const int32_t* N,
                            const int32_t* K, void* out, int32_t* out_idx,
                            uint8_t* out_src, float* out_h2, float* out_s,
                            void* stream);

/* Release the context and its scratch (NULL is a no-op).  Freeing device
 * memory waits for the device to finish outstanding work first. */
void tr_destroy(tr_ctx* ctx);

/* Static description of a status code. */
const char* tr_strerror(tr_status s);

/* One-line description of the latest failure in this thread ("" if none). */
const char* tr_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* TR_H */
