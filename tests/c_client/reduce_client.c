/* A client of the library written in plain C99: it uses only include/tr.h
 * and the HIP runtime's C API (no C++, no torch), as a C caller of the
 * boundary would.  It builds a small ragged batch of fp32 tokens with a fixed
 * generator, runs tr_create / tr_reduce / tr_destroy on a stream of its own,
 * checks what C alone can check (per image: K strictly ascending in-range
 * indices, K1 = floor(lambda K) of them from Stage I, the kept rows equal to
 * X's rows byte for byte), and writes the inputs and outputs as raw arrays to
 * the directory given as its first argument, for the oracle comparison of the
 * test that builds it.  An optional second argument picks the element type
 * and variant: "fp32" (default), "bf16", "bf16-shannon" or "fp32-stride-real".
 * Exit status 0 when every call and check succeeded. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "tr.h"

#define NIMG 3
static const int32_t kN[NIMG] = {576, 300, 1000};
static const int32_t kK[NIMG] = {64, 40, 111};
enum { D = 1024, DC = 768 };

#define HIP_OK(call)                                                                      \
    do {                                                                                  \
        hipError_t e_ = (call);                                                           \
        if (e_ != hipSuccess) {                                                           \
            fprintf(stderr, "%s failed: %s\n", #call, hipGetErrorString(e_));             \
            return 1;                                                                     \
        }                                                                                 \
    } while (0)

#define TR_OK_OR_FAIL(call)                                                               \
    do {                                                                                  \
        tr_status s_ = (call);                                                            \
        if (s_ != TR_OK) {                                                                \
            fprintf(stderr, "%s: %s (%s)\n", #call, tr_strerror(s_), tr_last_error());  \
            return 1;                                                                     \
        }                                                                                 \
    } while (0)

static uint32_t g_state = 20261202u;

static float uniform01(void)   /* in (0, 1) */
{
    g_state = g_state * 1664525u + 1013904223u;
    return ((float)(g_state >> 8) + 0.5f) / 16777216.0f;
}

static float normal(void)   /* Box-Muller */
{
    const float u1 = uniform01(), u2 = uniform01();
    return sqrtf(-2.0f * logf(u1)) * cosf(6.28318531f * u2);
}

/* fp32 -> bf16, round to nearest even (finite inputs) */
static uint16_t to_bf16(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

static float from_bf16(uint16_t h)
{
    const uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

static int write_file(const char* dir, const char* name, const void* p, size_t bytes)
{
    char path[4096];
    snprintf(path, sizeof path, "%s/%s", dir, name);
    FILE* f = fopen(path, "wb");
    if (!f || fwrite(p, 1, bytes, f) != bytes) {
        fprintf(stderr, "cannot write %s\n", path);
        if (f) fclose(f);
        return 1;
    }
    fclose(f);
    return 0;
}

int main(int argc, char** argv)
{
    if (argc != 2 && argc != 3) {
        fprintf(stderr, "usage: %s <output directory> [fp32|bf16|bf16-shannon|fp32-stride-real]\n", argv[0]);
        return 2;
    }
    const char* mode = argc == 3 ? argv[2] : "fp32";
    const int bf16 = strncmp(mode, "bf16", 4) == 0;
    const int32_t flags = strcmp(mode, "bf16-shannon") == 0 ? TR_FLAG_SHANNON
                          : strcmp(mode, "fp32-stride-real") == 0 ? TR_FLAG_STRIDE_REAL : 0;
    if (!bf16 && strcmp(mode, "fp32") != 0 && strcmp(mode, "fp32-stride-real") != 0) {
        fprintf(stderr, "unknown mode %s\n", mode);
        return 2;
    }
    const size_t eb = bf16 ? 2 : 4;
    int64_t rows = 0, kept = 0;
    for (int b = 0; b < NIMG; ++b) {
        rows += kN[b];
        kept += kK[b];
    }
    float* X = malloc(sizeof(float) * (size_t)(rows * D));
    float* P = malloc(sizeof(float) * (size_t)(rows * DC));
    float* Q = malloc(sizeof(float) * (size_t)(rows * DC));
    float* out = malloc(sizeof(float) * (size_t)(kept * D));
    int32_t* idx = malloc(sizeof(int32_t) * (size_t)kept);
    uint8_t* src = malloc((size_t)kept);
    float* h2 = malloc(sizeof(float) * (size_t)rows);
    float* s = malloc(sizeof(float) * (size_t)rows);
    if (!X || !P || !Q || !out || !idx || !src || !h2 || !s) return 1;

    /* tokens: Gaussian rows of log-normal scale, every tenth one near-constant;
     * post-MLP states = pre-MLP states plus noise */
    for (int64_t i = 0; i < rows; ++i) {
        const float scale = expf(0.5f * normal());
        for (int j = 0; j < D; ++j)
            X[i * D + j] = (i % 10 == 3) ? scale * (1.0f + 1e-3f * normal()) : scale * normal();
        for (int j = 0; j < DC; ++j) {
            P[i * DC + j] = normal();
            Q[i * DC + j] = P[i * DC + j] + 0.5f * normal();
        }
    }

    /* the element arrays the library reads: fp32 as generated, or bf16 (and
     * the fp32 arrays set to the rounded values, for the checks below) */
    void* hX = X;
    void* hP = P;
    void* hQ = Q;
    uint16_t *bX = NULL, *bP = NULL, *bQ = NULL;
    if (bf16) {
        bX = malloc(2 * (size_t)(rows * D));
        bP = malloc(2 * (size_t)(rows * DC));
        bQ = malloc(2 * (size_t)(rows * DC));
        if (!bX || !bP || !bQ) return 1;
        for (int64_t i = 0; i < rows * D; ++i) X[i] = from_bf16(bX[i] = to_bf16(X[i]));
        for (int64_t i = 0; i < rows * DC; ++i) {
            P[i] = from_bf16(bP[i] = to_bf16(P[i]));
            Q[i] = from_bf16(bQ[i] = to_bf16(Q[i]));
        }
        hX = bX;
        hP = bP;
        hQ = bQ;
    }

    void *dX, *dP, *dQ, *dout, *didx, *dsrc, *dh2, *ds;
    HIP_OK(hipMalloc(&dX, eb * (size_t)(rows * D)));
    HIP_OK(hipMalloc(&dP, eb * (size_t)(rows * DC)));
    HIP_OK(hipMalloc(&dQ, eb * (size_t)(rows * DC)));
    HIP_OK(hipMalloc(&dout, eb * (size_t)(kept * D)));
    HIP_OK(hipMalloc(&didx, sizeof(int32_t) * (size_t)kept));
    HIP_OK(hipMalloc(&dsrc, (size_t)kept));
    HIP_OK(hipMalloc(&dh2, sizeof(float) * (size_t)rows));
    HIP_OK(hipMalloc(&ds, sizeof(float) * (size_t)rows));
    HIP_OK(hipMemcpy(dX, hX, eb * (size_t)(rows * D), hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(dP, hP, eb * (size_t)(rows * DC), hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(dQ, hQ, eb * (size_t)(rows * DC), hipMemcpyHostToDevice));
    hipStream_t stream;
    HIP_OK(hipStreamCreate(&stream));

    tr_params p;
    memset(&p, 0, sizeof p);
    p.D = D;
    p.Dc = DC;
    p.dtype = bf16 ? TR_BF16 : TR_FP32;
    p.max_images = NIMG;
    p.max_tokens = rows;
    p.max_N = 1000;
    p.flags = flags;
    p.lambda = 1.0 / 3.0;
    p.keep_ratio = 0.0;
    tr_ctx* ctx = NULL;
    TR_OK_OR_FAIL(tr_create(&p, &ctx));
    TR_OK_OR_FAIL(tr_reduce(ctx, dX, dP, dQ, NIMG, kN, kK, dout, (int32_t*)didx, (uint8_t*)dsrc, (float*)dh2,
                            (float*)ds, (void*)stream));
    HIP_OK(hipStreamSynchronize(stream));
    uint16_t* bout = bf16 ? malloc(2 * (size_t)(kept * D)) : NULL;
    if (bf16 && !bout) return 1;
    HIP_OK(hipMemcpy(bf16 ? (void*)bout : (void*)out, dout, eb * (size_t)(kept * D), hipMemcpyDeviceToHost));
    if (bf16)
        for (int64_t i = 0; i < kept * D; ++i) out[i] = from_bf16(bout[i]);
    HIP_OK(hipMemcpy(idx, didx, sizeof(int32_t) * (size_t)kept, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(src, dsrc, (size_t)kept, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(h2, dh2, sizeof(float) * (size_t)rows, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(s, ds, sizeof(float) * (size_t)rows, hipMemcpyDeviceToHost));
    tr_destroy(ctx);

    int bad = 0;
    int64_t r0 = 0, o0 = 0;
    for (int b = 0; b < NIMG; ++b) {
        const int32_t k1 = (int32_t)floor(p.lambda * (double)kK[b]);
        int32_t from1 = 0;
        for (int32_t k = 0; k < kK[b]; ++k) {
            const int32_t i = idx[o0 + k];
            if (i < 0 || i >= kN[b] || (k > 0 && i <= idx[o0 + k - 1])) ++bad;
            if (src[o0 + k] == 0) ++from1;
            if (i >= 0 && i < kN[b] && memcmp(out + (o0 + k) * D, X + (r0 + i) * D, sizeof(float) * D) != 0) ++bad;
        }
        if (from1 != k1) ++bad;
        r0 += kN[b];
        o0 += kK[b];
    }
    if (bad) {
        fprintf(stderr, "%d output checks failed\n", bad);
        return 1;
    }
    if (write_file(argv[1], "X.f32", X, sizeof(float) * (size_t)(rows * D)) ||
        write_file(argv[1], "P.f32", P, sizeof(float) * (size_t)(rows * DC)) ||
        write_file(argv[1], "Q.f32", Q, sizeof(float) * (size_t)(rows * DC)) ||
        write_file(argv[1], "out.f32", out, sizeof(float) * (size_t)(kept * D)) ||
        write_file(argv[1], "idx.i32", idx, sizeof(int32_t) * (size_t)kept) ||
        write_file(argv[1], "src.u8", src, (size_t)kept) ||
        write_file(argv[1], "h2.f32", h2, sizeof(float) * (size_t)rows) ||
        write_file(argv[1], "s.f32", s, sizeof(float) * (size_t)rows))
        return 1;
    HIP_OK(hipStreamDestroy(stream));
    HIP_OK(hipFree(dX));
    HIP_OK(hipFree(dP));
    HIP_OK(hipFree(dQ));
    HIP_OK(hipFree(dout));
    HIP_OK(hipFree(didx));
    HIP_OK(hipFree(dsrc));
    HIP_OK(hipFree(dh2));
    HIP_OK(hipFree(ds));
    free(X);
    free(P);
    free(Q);
    free(out);
    free(idx);
    free(src);
    free(h2);
    free(s);
    free(bX);
    free(bP);
    free(bQ);
    free(bout);
    printf("c client ok (%s): %d images, %lld tokens, %lld kept\n", mode, NIMG, (long long)rows, (long long)kept);
    return 0;
}
