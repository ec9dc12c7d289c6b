// bf16 matrix-core GEMM for the steps around the path:
//   C[M, N] = A[M, K] . B[N, K]^T      (bf16 in, fp32 accumulation, bf16 out)
// with two optional fusions:
//   * row gather of A (A row m is A[rows[m]]): the projector GEMM applied to
//     the kept tokens straight from X, without materialising the gathered
//     copy (the step after the path: the kept tokens are projected);
//   * cosine epilogue: while the fp32 tile of C is in registers, per-row
//     partial sums of P.C, P.P and C.C against a second [M, N] matrix P.  With
//     C = x'' the output of the encoder MLP's second layer (W2 applied to the
//     hidden activations) and P = x' its input, these are Eq. (6)'s three sums,
//     so the Stage II score needs no further pass over X_pre or X_post.
//
// Tiling for gfx950 (64-wide wavefronts, 32x32x16 bf16 MFMA):
//   * workgroup tile 256 x 128 x 64, four wavefronts in a 2 x 2 grid, each
//     owning 128 x 64 of C as 4 x 2 MFMA tiles (128 fp32 accumulators a lane);
//   * one LDS stage holding the A and B k-tiles, rows padded from 128 to 144
//     bytes so that the 16-byte fragment reads of a wavefront hit distinct
//     banks; the next k-tile is prefetched into registers while the current
//     one feeds the MFMAs (54 KB of LDS: two workgroups fit a CU);
//   * XCD-aware tile order: workgroup b runs on XCD b % 8; each XCD takes a
//     contiguous run of output tiles with the N tile fastest, so the
//     workgroups sharing an A block-row share that XCD's L2.
//
// MFMA operand layout (32x32x16 bf16, verified on the device): lane l holds
// A row l % 32 and B column l % 32, k = (l / 32) * 8 .. + 8; accumulator
// element v of lane l is C[(v / 4) * 8 + (l / 32) * 4 + v % 4][l % 32].
#include "tr_internal.h"
#include "tr_wave.h"

namespace tr {
namespace {

constexpr int kBM = 256, kBN = 128, kBK = 64;
constexpr int kThreads = 256;
constexpr int kRowBytes = 144;                       // 64 bf16 + 16 bytes of padding
constexpr int kLdsA = kBM * kRowBytes;               // 36864
constexpr int kLdsB = kBN * kRowBytes;               // 18432
constexpr int kLdsRed = 2 * kBM * 3 * 4;             // cosine partials of the two N-halves
constexpr int kXcds = 8;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }

// bf16 round-to-nearest-even of an fp32 value (finite inputs; NaN stays NaN).
__device__ __forceinline__ uint16_t to_bf16(float f)
{
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u) return (uint16_t)((u >> 16) | ((u & 0xffffu) ? 0x40u : 0u));
    return (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

template <bool GATHER, bool COS>
__global__ __launch_bounds__(kThreads, 2) void gemm_kernel(GemmArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char* lA = smem;
    unsigned char* lB = smem + kLdsA;

    // ---- tile of this workgroup (XCD-aware order) --------------------------
    const int mt = (a.M + kBM - 1) / kBM, nt = a.N / kBN;
    const int tiles = mt * nt;
    const int per_xcd = (tiles + kXcds - 1) / kXcds;
    const int t = (int)(blockIdx.x % kXcds) * per_xcd + (int)(blockIdx.x / kXcds);
    if (t >= tiles) return;   // whole workgroup leaves together
    const int m0 = (t / nt) * kBM, n0 = (t % nt) * kBN;

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int wm = w >> 1, wn = w & 1;   // 2 x 2 wavefront grid

    // ---- global -> register loads: thread owns 16-byte chunk (tid % 8) of
    // rows tid / 8 + 32 p.  A: 8 rows per thread, B: 4.
    const int ch = tid & 7, r0 = tid >> 3;
    // Rows outside the matrix (or gathered indices out of range) load row 0
    // and are zeroed when stored to LDS: the loads stay unconditional, so
    // nothing waits on them before the MFMAs of the current k-tile.
    const char* arow[8];
    uint32_t avalid = 0;
#pragma unroll
    for (int p = 0; p < 8; ++p) {
        const int m = m0 + r0 + 32 * p;
        int64_t src = -1;
        if (m < a.M) {
            src = m;
            if constexpr (GATHER) {
                const int32_t r = a.arows[m];
                src = (r >= 0 && r < a.arow_count) ? (int64_t)r : -1;
            }
        }
        if (src >= 0) avalid |= 1u << p;
        arow[p] = reinterpret_cast<const char*>(a.A) + (src >= 0 ? src : 0) * a.lda * 2 + ch * 16;
    }
    const char* brow[4];
#pragma unroll
    for (int p = 0; p < 4; ++p)
        brow[p] = reinterpret_cast<const char*>(a.B) + (int64_t)(n0 + r0 + 32 * p) * a.ldb * 2 + ch * 16;

    u32x4 ra[8], rb[4];
    auto load_tile = [&](int k0) {
#pragma unroll
        for (int p = 0; p < 8; ++p)
            ra[p] = *reinterpret_cast<const u32x4*>(arow[p] + (int64_t)k0 * 2);
#pragma unroll
        for (int p = 0; p < 4; ++p) rb[p] = *reinterpret_cast<const u32x4*>(brow[p] + (int64_t)k0 * 2);
    };
    auto store_tile = [&]() {
#pragma unroll
        for (int p = 0; p < 8; ++p)
            *reinterpret_cast<u32x4*>(lA + (r0 + 32 * p) * kRowBytes + ch * 16) =
                ((avalid >> p) & 1u) ? ra[p] : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
        for (int p = 0; p < 4; ++p)
            *reinterpret_cast<u32x4*>(lB + (r0 + 32 * p) * kRowBytes + ch * 16) = rb[p];
    };

    f32x16 acc[4][2];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    // fragment addresses inside the LDS tiles
    const int frow = lane & 31, fk = (lane >> 5) * 16;   // byte offset of the lane's 8 k values
    const unsigned char* fa = lA + (wm * 128 + frow) * kRowBytes + fk;
    const unsigned char* fb = lB + (wn * 64 + frow) * kRowBytes + fk;

    const int KT = a.K / kBK;
    load_tile(0);
    store_tile();
    __syncthreads();
    for (int kt = 0; kt < KT; ++kt) {
        if (kt + 1 < KT) load_tile((kt + 1) * kBK);
#pragma unroll
        for (int kk = 0; kk < kBK / 16; ++kk) {
            bf16x8 fA[4], fB[2];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                fA[i] = *reinterpret_cast<const bf16x8*>(fa + i * 32 * kRowBytes + kk * 32);
#pragma unroll
            for (int j = 0; j < 2; ++j)
                fB[j] = *reinterpret_cast<const bf16x8*>(fb + j * 32 * kRowBytes + kk * 32);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fA[i], fB[j], acc[i][j], 0, 0, 0);
        }
        __syncthreads();
        if (kt + 1 < KT) {
            store_tile();
            __syncthreads();
        }
    }

    // ---- epilogue ---------------------------------------------------------
    const int half = lane >> 5;
    uint16_t* C = reinterpret_cast<uint16_t*>(a.C);
    float* red = reinterpret_cast<float*>(smem + kLdsA + kLdsB);   // [2][kBM][3]
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int rl = wm * 128 + i * 32 + (v >> 2) * 8 + half * 4 + (v & 3);   // row in the tile
            const int m = m0 + rl;
            const bool ok = m < a.M;
            float dot = 0.f, pp = 0.f, cc = 0.f;
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int n = n0 + wn * 64 + j * 32 + (lane & 31);
                const float c = acc[i][j][v];
                if (ok) C[(int64_t)m * a.ldc + n] = to_bf16(c);
                if constexpr (COS) {
                    const float p = ok ? bf16_lo(reinterpret_cast<const uint16_t*>(a.P)[(int64_t)m * a.ldp + n]) : 0.f;
                    dot = fmaf(p, c, dot);
                    pp = fmaf(p, p, pp);
                    cc = fmaf(c, c, cc);
                }
            }
            if constexpr (COS) {
                // sum over the 32 lanes of this half (same row): lane 31 / 63 ends with it
                dot = half_sum(dot);
                pp = half_sum(pp);
                cc = half_sum(cc);
                if ((lane & 31) == 31) {
                    float* r = red + ((size_t)wn * kBM + rl) * 3;
                    r[0] = dot;
                    r[1] = pp;
                    r[2] = cc;
                }
            }
        }
    }
    if constexpr (COS) {
        __syncthreads();
        // one thread per tile row: the two N-halves, then this tile's partials
        const int rl = tid;
        const int m = m0 + rl;
        if (m < a.M) {
            const float* r0p = red + (size_t)rl * 3;
            const float* r1p = red + ((size_t)kBM + rl) * 3;
            float* out = a.part + ((int64_t)m * a.part_cols + n0 / kBN) * 3;
            out[0] = r0p[0] + r1p[0];
            out[1] = r0p[1] + r1p[1];
            out[2] = r0p[2] + r1p[2];
        }
    }
}

// s = dot / (|P| |C|) from the per-tile partials, summed in tile order; the
// same zero-norm reading as the scoring kernel (s = 0).
__global__ __launch_bounds__(256) void cos_finish_kernel(const float* part, int cols, int M, float* s)
{
    const int m = blockIdx.x * blockDim.x + threadIdx.x;
    if (m >= M) return;
    const float* p = part + (int64_t)m * cols * 3;
    float dot = 0.f, n1 = 0.f, n2 = 0.f;
    for (int c = 0; c < cols; ++c) {
        dot += p[3 * c];
        n1 += p[3 * c + 1];
        n2 += p[3 * c + 2];
    }
    float v = 0.f;
    if (n1 > 0.f && n2 > 0.f) v = dot / (sqrtf(n1) * sqrtf(n2));
    s[m] = v;
}

}  // namespace

int gemm_part_cols(int N) { return N / kBN; }

bool gemm_shape_ok(int M, int N, int K)
{
    if (M < 0 || N <= 0 || K <= 0 || N % kBN || K % kBK) return false;
    // output tiles (and the grid, rounded up to the XCD count) fit an int
    const int64_t tiles = (int64_t)((M + (int64_t)kBM - 1) / kBM) * (N / kBN);
    return tiles <= (int64_t)INT32_MAX - kXcds;
}

hipError_t gemm_prepare()
{
    hipError_t e;
    const int lds = kLdsA + kLdsB + kLdsRed;
    if ((e = hipFuncSetAttribute((const void*)gemm_kernel<false, false>,
                                 hipFuncAttributeMaxDynamicSharedMemorySize, lds)) != hipSuccess) return e;
    if ((e = hipFuncSetAttribute((const void*)gemm_kernel<true, false>,
                                 hipFuncAttributeMaxDynamicSharedMemorySize, lds)) != hipSuccess) return e;
    return hipFuncSetAttribute((const void*)gemm_kernel<false, true>,
                               hipFuncAttributeMaxDynamicSharedMemorySize, lds);
}

hipError_t launch_gemm(const GemmArgs& a, hipStream_t s)
{
    if (a.M == 0) return hipSuccess;
    const int tiles = ((a.M + kBM - 1) / kBM) * (a.N / kBN);
    const int grid = ((tiles + kXcds - 1) / kXcds) * kXcds;
    const bool gather = a.arows != nullptr, cos = a.P != nullptr;
    const size_t lds = kLdsA + kLdsB + (cos ? kLdsRed : 0);
    if (gather && cos) return hipErrorInvalidValue;
    if (gather)
        hipLaunchKernelGGL((gemm_kernel<true, false>), dim3(grid), dim3(kThreads), lds, s, a);
    else if (cos)
        hipLaunchKernelGGL((gemm_kernel<false, true>), dim3(grid), dim3(kThreads), lds, s, a);
    else
        hipLaunchKernelGGL((gemm_kernel<false, false>), dim3(grid), dim3(kThreads), lds, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !cos) return e;
    hipLaunchKernelGGL(cos_finish_kernel, dim3((a.M + 255) / 256), dim3(256), 0, s, a.part, a.part_cols, a.M,
                       a.s_out);
    return hipGetLastError();
}

}  // namespace tr
