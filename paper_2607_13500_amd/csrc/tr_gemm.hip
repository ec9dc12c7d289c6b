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
//     so the Stage II score needs no further pass over X_pre or X_post.  The
//     sums use C as stored (rounded to bf16), so the score is Eq. (6) on the
//     x'' the caller receives, as an unfused scoring pass would compute it.
//
// Two tilings for gfx950 (64-wide wavefronts, 32x32x16 bf16 MFMA), both with
// the same per-element MFMA sequence (k ascending in steps of 16), so they give
// bit-identical C:
//   * wide (N % 256 == 0, K % 128 == 0): workgroup tile (64 MT) x 256 x 64
//     with MT = 4, 3 or 2 picked per shape so the tiles fill the CUs in whole
//     waves; eight wavefronts in a 2 x 4 grid, each owning 32 MT x 64 of C
//     (MT x 2 MFMA tiles, 32 MT fp32 accumulators a lane).
//     Operands go from global memory straight into LDS (buffer loads with the
//     LDS-destination form, 16 bytes a lane), two LDS stages of 64 KB, so the
//     next k-tile streams in while the current one feeds the MFMAs with no
//     staging registers.  LDS rows are 128 bytes with the 16-byte chunks
//     XOR-swizzled by (row / 2) % 8, which keeps the fragment reads of any 16
//     consecutive rows on distinct banks.  Buffer range checking reads rows
//     past the end of A (or invalid gathered rows) as zeros.  The cosine
//     epilogue stages its block of P through the freed LDS stages.
//   * narrow (every other shape, or operands beyond 31-bit buffer offsets):
//     workgroup tile 256 x 128 x 64, four wavefronts of 128 x 64, rows padded
//     from 128 to 144 bytes for conflict-free fragment reads, the next k-tile
//     prefetched into registers (54 KB of LDS: two workgroups fit a CU).
// Both use an XCD-aware tile order: workgroup b runs on XCD b % 8; each XCD
// takes a contiguous run of output tiles with the N tile fastest, so the
// workgroups sharing an A block-row share that XCD's L2.
//
// MFMA operand layout (32x32x16 bf16, verified on the device): lane l holds
// A row l % 32 and B column l % 32, k = (l / 32) * 8 .. + 8; accumulator
// element v of lane l is C[(v / 4) * 8 + (l / 32) * 4 + v % 4][l % 32].
#include <cstdlib>

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
                const uint16_t cb = to_bf16(acc[i][j][v]);
                const float c = bf16_lo(cb);   // the value stored
                if (ok) C[(int64_t)m * a.ldc + n] = cb;
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

// ---- wide tiling -----------------------------------------------------------
constexpr int kWBN = 256;
constexpr int kWThreads = 512;
constexpr int kWStage = kBM * kBK * 2;              // one operand k-tile: 256 rows x 128 B
constexpr int kWRed = 4 * kBM * 3;                  // cosine partials of the four N-quarters (floats)
constexpr uint32_t kBufWord3 = 0x00020000u;        // raw buffer resource, 32-bit elements
constexpr uint32_t kBadRow = 0x80000000u;          // a buffer offset past every resource

typedef __attribute__((address_space(3))) unsigned char lds_t;
typedef __attribute__((address_space(3))) bf16x8 lds_frag;
typedef __attribute__((address_space(3))) void lds_void;

// MT: MFMA tiles per wavefront along M (4, 3 or 2), so the workgroup tile is
// 64 MT rows by 256 columns.
template <int MT, bool GATHER, bool COS>
__global__ __launch_bounds__(kWThreads, 1) void gemm_wide_kernel(GemmArgs a)
{
    constexpr int BMW = 64 * MT;
    __shared__ __attribute__((aligned(1024))) unsigned char sA0[kWStage], sA1[kWStage], sB0[kWStage], sB1[kWStage];
    __shared__ float red[COS ? kWRed : 1];
    lds_t* const a0 = (lds_t*)sA0;
    lds_t* const a1 = (lds_t*)sA1;
    lds_t* const b0 = (lds_t*)sB0;
    lds_t* const b1 = (lds_t*)sB1;

    const int mt = (a.M + BMW - 1) / BMW, nt = a.N / kWBN;
    const int tiles = mt * nt;
    const int per_xcd = (tiles + kXcds - 1) / kXcds;
    const int t = (int)(blockIdx.x % kXcds) * per_xcd + (int)(blockIdx.x / kXcds);
    if (t >= tiles) return;   // whole workgroup leaves together
    const int m0 = (t / nt) * BMW, n0 = (t % nt) * kWBN;

    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = w >> 2, wn = w & 3;   // 2 x 4 wavefront grid

    // ---- global -> LDS.  Wavefront w fills row blocks MT w .. MT w + MT-1 of
    // the A tile and 4w .. 4w+3 of the B tile (blocks of 8 rows of 128 B);
    // lane l writes physical chunk l % 8 of row l / 8 of a block, which holds
    // logical chunk (l % 8) ^ ((row / 2) % 8).
    // Offsets are 32-bit bytes from the resource base; the k offset of a
    // k-tile is the scalar offset.  The host routes larger operands to the
    // narrow kernel.
    const uint16_t* A = reinterpret_cast<const uint16_t*>(a.A);
    const uint16_t* B = reinterpret_cast<const uint16_t*>(a.B);
    int64_t a_bytes;
    const uint16_t* abase;
    if constexpr (GATHER) {
        abase = A;
        a_bytes = a.arow_count * a.lda * 2;
    } else {
        abase = A + (int64_t)m0 * a.lda;
        a_bytes = (int64_t)(a.M - m0) * a.lda * 2;
    }
    const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(
        (void*)abase, (short)0, (int)(a_bytes < (int64_t)kBadRow ? a_bytes : (int64_t)kBadRow - 1), kBufWord3);
    const __amdgpu_buffer_rsrc_t rb = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(B + (int64_t)n0 * a.ldb), (short)0, (int)(kWBN * a.ldb * 2), kBufWord3);
    // ao has room for the tallest tile (an array bound that depends on MT,
    // captured by the lambdas below, makes the host pass drop the kernel).
    uint32_t ao[4], bo[4];
#pragma unroll
    for (int i = 0; i < MT; ++i) {
        const int row = (w * MT + i) * 8 + (lane >> 3);
        const int c = (lane & 7) ^ ((row >> 1) & 7);
        if constexpr (GATHER) {
            const int m = m0 + row;
            int32_t r = m < a.M ? a.arows[m] : -1;
            ao[i] = (r >= 0 && r < a.arow_count) ? (uint32_t)((int64_t)r * a.lda * 2 + c * 16) : kBadRow;
        } else {
            ao[i] = (uint32_t)(row * a.lda * 2 + c * 16);
        }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int row = (w * 4 + i) * 8 + (lane >> 3);
        const int c = (lane & 7) ^ ((row >> 1) & 7);
        bo[i] = (uint32_t)(row * a.ldb * 2 + c * 16);
    }
    const int dsta = w * MT * 1024, dstb = w * 4 * 1024;
    auto issue = [&](lds_t* sa, lds_t* sb, int k0) {
#pragma unroll
        for (int i = 0; i < MT; ++i)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void*)(sa + dsta + i * 1024), 16, ao[i], k0 * 2, 0, 0);
#pragma unroll
        for (int i = 0; i < 4; ++i)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_void*)(sb + dstb + i * 1024), 16, bo[i], k0 * 2, 0, 0);
    };

    // ---- fragment reads: lane l reads row l % 32 of a 32-row block, logical
    // chunk 2 kk + l / 32, which sits at physical chunk (2 kk + l / 32) ^ sw.
    const int l31 = lane & 31, half = lane >> 5;
    const int sw = (l31 >> 1) & 7, shi = sw >> 1, slo = sw & 1;
    int offA[4], offB[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
        const int cb = 32 * (kk ^ shi) + 16 * (half ^ slo);
        offA[kk] = (wm * 32 * MT + l31) * 128 + cb;
        offB[kk] = (wn * 64 + l31) * 128 + cb;
    }

    f32x16 acc[MT][2];
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    // One k-tile: the fragments of step kk+1 are read before the MFMAs of step
    // kk (the scheduling barriers keep that order).
    auto compute = [&](const lds_t* sa, const lds_t* sb) {
        bf16x8 fa[2][MT], fb[2][2];
#pragma unroll
        for (int i = 0; i < MT; ++i) fa[0][i] = *(const lds_frag*)(sa + offA[0] + i * 4096);
#pragma unroll
        for (int j = 0; j < 2; ++j) fb[0][j] = *(const lds_frag*)(sb + offB[0] + j * 4096);
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            const int cur = kk & 1, nxt = cur ^ 1;
            if (kk < 3) {
#pragma unroll
                for (int i = 0; i < MT; ++i) fa[nxt][i] = *(const lds_frag*)(sa + offA[kk + 1] + i * 4096);
#pragma unroll
                for (int j = 0; j < 2; ++j) fb[nxt][j] = *(const lds_frag*)(sb + offB[kk + 1] + j * 4096);
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int i = 0; i < MT; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[cur][i], fb[cur][j], acc[i][j], 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    // Two stages.  Before each k-tile every wavefront waits for its own
    // LDS-destination loads, then the barrier makes all of them visible and
    // guarantees the other stage is no longer read: the next k-tile's loads go
    // there while this one is computed.
    // The host sends only an even number of k-tiles (K % 128 == 0) here: a
    // loop with a single exit keeps the accumulators in place.
    //
    // Cosine epilogue: the tile's [64 MT, 256] block of P (at most 128 KB) is
    // staged through the two freed stages.  Rows 0-127 (all those of
    // wavefronts 0-3) go into stage 0 during the last k-tile; rows 128 and up
    // into stage 1 while wavefronts 0-3 form their sums.  Stage h holds row
    // 64 g + r of its 128 rows at array g (A or B part of the stage), byte
    // r * 512.
    const int KT = a.K / kBK;
    [[maybe_unused]] __amdgpu_buffer_rsrc_t rp;
    if constexpr (COS) {
        const int64_t p_bytes = (int64_t)(a.M - m0) * a.ldp * 2;
        rp = __builtin_amdgcn_make_buffer_rsrc(
            (void*)(reinterpret_cast<const uint16_t*>(a.P) + (int64_t)m0 * a.ldp + n0), (short)0,
            (int)(p_bytes < (int64_t)kBadRow ? p_bytes : (int64_t)kBadRow - 1), kBufWord3);
    }
    auto issue_p = [&](int h, lds_t* sa, lds_t* sb) {
        lds_t* arr = w < 4 ? sa : sb;
        const int rows = BMW - 128 * h < 128 ? BMW - 128 * h : 128;   // rows of P in this stage
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int q = (w & 3) * 8 + i;   // 1 KB block of the array: rows 2q, 2q+1
            const int rh = (w >> 2) * 64 + 2 * q;   // first of the two rows within the stage
            if (rh < rows)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    rp, (lds_void*)(arr + q * 1024), 16,
                    (uint32_t)((h * 128 + rh + (lane >> 5)) * a.ldp * 2 + (lane & 31) * 16), 0, 0, 0);
        }
    };

    issue(a0, b0, 0);
    for (int kt = 0; kt < KT; kt += 2) {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        issue(a1, b1, (kt + 1) * kBK);
        compute(a0, b0);
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        if (kt + 2 < KT) {
            issue(a0, b0, (kt + 2) * kBK);
        } else {
            if constexpr (COS) issue_p(0, a0, b0);
        }
        compute(a1, b1);
    }

    // ---- epilogue ----------------------------------------------------------
    // The row stride passes through an empty asm so that no output address is
    // formed before the main loop (64 row offsets held across it would spill).
    int64_t ldc = a.ldc;
    asm volatile("" : "+s"(ldc));
    uint16_t* C = reinterpret_cast<uint16_t*>(a.C);
    auto store_c = [&]() {
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int m = m0 + wm * 32 * MT + i * 32 + (v >> 2) * 8 + half * 4 + (v & 3);
                if (m < a.M) {
#pragma unroll
                    for (int j = 0; j < 2; ++j)
                        C[(int64_t)m * ldc + n0 + wn * 64 + j * 32 + l31] = to_bf16(acc[i][j][v]);
                }
            }
    };
    // Per-row sums P.C, P.P and C.C over this wavefront's 64 columns, from P
    // staged in LDS; rows past M have P = 0 and C = 0 (their A rows read as
    // zeros) and are never used.
    auto cos_part = [&]() {
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int r0 = wm * 32 * MT + i * 32;   // first row of this 32-row block (uniform)
                const int rr = (r0 & 127) + (v >> 2) * 8 + half * 4 + (v & 3);   // row within its stage
                const lds_t* arr = r0 >= 128 ? ((r0 & 127) >= 64 ? b1 : a1) : ((r0 & 127) >= 64 ? b0 : a0);
                float dot = 0.f, pp = 0.f, cc = 0.f;
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    const int col = wn * 64 + j * 32 + l31;
                    const float pv = bf16_lo(*(const __attribute__((address_space(3))) uint16_t*)(
                        arr + (rr & 63) * 512 + col * 2));
                    const float c = bf16_lo(to_bf16(acc[i][j][v]));   // the value stored
                    dot = fmaf(pv, c, dot);
                    pp = fmaf(pv, pv, pp);
                    cc = fmaf(c, c, cc);
                }
                dot = half_sum(dot);
                pp = half_sum(pp);
                cc = half_sum(cc);
                if (l31 == 31) {
                    float* r = red + ((size_t)wn * kBM + r0 + (v >> 2) * 8 + half * 4 + (v & 3)) * 3;
                    r[0] = dot;
                    r[1] = pp;
                    r[2] = cc;
                }
            }
    };

    if constexpr (!COS) {
        store_c();
    } else {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();   // P rows 0-127 in stage 0; stage 1 no longer read
        issue_p(1, a1, b1);
        if (wm == 0) cos_part();
        store_c();
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();   // P rows 128 and up in stage 1
        if (wm == 1) cos_part();
        __syncthreads();
        // one thread per tile row: the four N-quarters in order, then this
        // tile's partials
        if (tid < BMW) {
            const int m = m0 + tid;
            if (m < a.M) {
                float d = 0.f, p = 0.f, q = 0.f;
#pragma unroll
                for (int qn = 0; qn < 4; ++qn) {
                    const float* r = red + ((size_t)qn * kBM + tid) * 3;
                    d += r[0];
                    p += r[1];
                    q += r[2];
                }
                float* out = a.part + ((int64_t)m * a.part_cols + n0 / kWBN) * 3;
                out[0] = d;
                out[1] = p;
                out[2] = q;
            }
        }
    }
}

// s = dot / (|P| |C|) from the per-tile partials, summed in tile order; the
// same zero-norm reading as the scoring kernel (s = 0).
__global__ __launch_bounds__(256) void cos_finish_kernel(const float* part, int stride, int cols, int M, float* s)
{
    const int m = blockIdx.x * blockDim.x + threadIdx.x;
    if (m >= M) return;
    const float* p = part + (int64_t)m * stride * 3;
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

// The wide kernel takes the shape when N is a multiple of 256, K of 128 (an
// even number of k-tiles) and every buffer offset it forms fits 31 bits.
bool use_wide(const GemmArgs& a)
{
    if (a.N % kWBN || a.K % (2 * kBK)) return false;
    const int64_t lim = (int64_t)kBadRow;
    if ((int64_t)kBM * a.lda * 2 >= lim || (int64_t)kWBN * a.ldb * 2 >= lim) return false;
    if (a.arows && a.arow_count * a.lda * 2 >= lim) return false;
    if (a.P && (int64_t)kBM * a.ldp * 2 >= lim) return false;
    return true;
}

int g_cus = 256;         // compute units of the device (set by gemm_prepare)
int g_force_mt = 0;      // tile height override: 0 = model, else 2, 3 or 4

// Tile height of the wide kernel (MFMA tiles per wavefront along M): the one
// with the least modelled time, (tile waves over the CUs) x (rows per tile),
// where shorter tiles pay for their higher LDS traffic per MFMA.
int wide_mt(int M, int N)
{
    if (g_force_mt) return g_force_mt;
    const double cost_per_row[5] = {0, 0, 1.2, 1.05, 1.0};
    int best = 4;
    double best_t = 0;
    for (int mtw = 4; mtw >= 2; --mtw) {
        const int64_t tiles = (int64_t)((M + 64 * mtw - 1) / (64 * mtw)) * (N / kWBN);
        const int64_t waves = (tiles + g_cus - 1) / g_cus;
        const double t = (double)waves * mtw * cost_per_row[mtw];
        if (mtw == 4 || t < best_t) {
            best = mtw;
            best_t = t;
        }
    }
    return best;
}

void launch_wide(const GemmArgs& a, int mtw, bool gather, bool cos, int grid, hipStream_t s)
{
    const dim3 g(grid), b(kWThreads);
    if (mtw == 4) {
        if (gather)
            hipLaunchKernelGGL((gemm_wide_kernel<4, true, false>), g, b, 0, s, a);
        else if (cos)
            hipLaunchKernelGGL((gemm_wide_kernel<4, false, true>), g, b, 0, s, a);
        else
            hipLaunchKernelGGL((gemm_wide_kernel<4, false, false>), g, b, 0, s, a);
    } else if (mtw == 3) {
        if (gather)
            hipLaunchKernelGGL((gemm_wide_kernel<3, true, false>), g, b, 0, s, a);
        else if (cos)
            hipLaunchKernelGGL((gemm_wide_kernel<3, false, true>), g, b, 0, s, a);
        else
            hipLaunchKernelGGL((gemm_wide_kernel<3, false, false>), g, b, 0, s, a);
    } else {
        if (gather)
            hipLaunchKernelGGL((gemm_wide_kernel<2, true, false>), g, b, 0, s, a);
        else if (cos)
            hipLaunchKernelGGL((gemm_wide_kernel<2, false, true>), g, b, 0, s, a);
        else
            hipLaunchKernelGGL((gemm_wide_kernel<2, false, false>), g, b, 0, s, a);
    }
}

}  // namespace

// capacity (row stride of the partials): the narrow kernel's column count
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
    int dev = 0;
    if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
    if ((e = hipDeviceGetAttribute(&g_cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
    // TR_GEMM_TILE_ROWS = 128, 192 or 256 pins the wide kernel's tile height
    // (tuning and tests); anything else leaves the choice to the model.
    const char* env = getenv("TR_GEMM_TILE_ROWS");
    const int rows = env ? atoi(env) : 0;
    g_force_mt = (rows == 128 || rows == 192 || rows == 256) ? rows / 64 : 0;
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
    const bool gather = a.arows != nullptr, cos = a.P != nullptr;
    if (gather && cos) return hipErrorInvalidValue;
    const bool wide = use_wide(a);
    const int mtw = wide ? wide_mt(a.M, a.N) : 4;
    const int bm = wide ? 64 * mtw : kBM, bn = wide ? kWBN : kBN;
    const int tiles = ((a.M + bm - 1) / bm) * (a.N / bn);
    const int grid = ((tiles + kXcds - 1) / kXcds) * kXcds;
    if (wide) {
        launch_wide(a, mtw, gather, cos, grid, s);
    } else {
        const size_t lds = kLdsA + kLdsB + (cos ? kLdsRed : 0);
        if (gather)
            hipLaunchKernelGGL((gemm_kernel<true, false>), dim3(grid), dim3(kThreads), lds, s, a);
        else if (cos)
            hipLaunchKernelGGL((gemm_kernel<false, true>), dim3(grid), dim3(kThreads), lds, s, a);
        else
            hipLaunchKernelGGL((gemm_kernel<false, false>), dim3(grid), dim3(kThreads), lds, s, a);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !cos) return e;
    hipLaunchKernelGGL(cos_finish_kernel, dim3((a.M + 255) / 256), dim3(256), 0, s, a.part, a.part_cols, a.N / bn,
                       a.M, a.s_out);
    return hipGetLastError();
}

}  // namespace tr
