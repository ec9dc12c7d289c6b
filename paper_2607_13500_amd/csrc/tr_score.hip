// Fused per-token scoring: one HBM pass over X, X_pre and X_post.
//
// One wavefront scores one token row.  The row is cut into chunks of 16 bytes
// (8 bf16 or 4 fp32 elements); chunk c belongs to lane c % 64 and every lane
// walks its chunks in ascending c, so a row's arithmetic never depends on
// where the row sits in the batch (identical rows score identically).
//
// Eq. (3)-(4): with m = mean |x| and V = M2 / D (M2 = sum (|x| - m)^2),
//   sum_j p_j^2 = (1 + V / m^2) / D,  H2 = log D - log1p(CV^2),
//   CV^2 = M2 / (D m^2).
// Stage I ranks ascending CV^2 (= descending H2): near-uniform rows have H2
// within an fp32 ulp of log D but well-separated CV^2.  M2 is accumulated
// around one shift c shared by the whole row, the mean |x| of its first
// min(D, 64 * 16 / elem) elements (every lane's first chunk, summed by a
// butterfly before any other work): d = |x| - c is exact when |x| is within a
// factor 2 of c (near-uniform rows), and M2 = sum d^2 - (sum d)^2 / D has
// little cancellation because c lies close to m.
//
// Range: both scores are invariant to scaling a row by a positive constant
// (Eq. 3 divides by sum |x|, Eq. 6 by both norms), so X is scored as
// |x| 2^-e with 2^e the binade of the probe mean: the power of two is applied
// by the same fused multiply-add that subtracts the shift (exact for normal
// values, no extra instruction), and the sums of squares stay far from fp32
// overflow and underflow whatever the row's magnitude.  A row whose probe
// mean lies outside [2^-120, 2^120] (an all-zero probe included) or whose
// scaled sums leave [0, 2^100] is scored again from a second read of its
// bytes, scaled from its exact maximum |x| and shifted by its exact mean.
//
// Eq. (6): fp32 sums of x'x'', x'^2 and x''^2 (bf16 rows: hardware bf16 dot
// products of element pairs, accumulated in fp32), unscaled.  When both
// squared norms lie in [2^-60, FLT_MAX], products that underflow (or
// denormal inputs) move s by less than 2^-40 and nothing overflowed; any
// other row is scored again from a second read, each of x' and x'' scaled by
// the power of two of its own maximum |x|, in fp32 fused multiply-adds.
//
// Non-finite elements: a NaN or an infinity makes the first pass's sums NaN
// or infinite, so such a row always takes the second read, which is where it
// is detected; with a count requested, lane 0 adds one per such row.
//
// Lane partial sums are combined by a fixed DPP scan tree (the total is read
// from lane 63 into every lane) and lane 0 writes the results.
//
// A launch may compute only one of the two scores (Stage I's key alone, or
// Stage II's alone): the other tensor is then never read and its key is
// written as 0.  The scores that are computed are bit-identical to those of a
// launch that computes both, because each score's arithmetic is independent.
//
// Shannon variant of Stage I (H1 = -sum p log p of the same p): the key is
// KL = log D - H1 >= 0 (ascending = descending H1), accumulated without
// cancellation as a sum of non-negative terms.  With u = |x| / c for the same
// row shift c and g(u) = u log u - u + 1 >= 0, and r = mean|x| / c,
//   D KL = sum_j (|x_j|/m) log(|x_j|/m) = (sum_j g(u_j) - D g(r)) / r,
// where the subtracted D g(r) is small because c lies close to the mean.
// Every u is formed as 1 + e with e = (|x| - c) (1/c) + delta, delta =
// c (1/c) - 1 taken exactly by a fused multiply-add, so all terms (and r)
// refer to the same effective shift 1 / (1/c) and e keeps full relative
// accuracy for near-uniform rows.  The terms are summed in base-2 units
// (e / ln 2 and g / ln 2), which saves a multiply per element; the row's sum
// is scaled by ln 2 once.
#include "tr_score.h"
#include "tr_wave.h"

namespace tr {
namespace {

// 16 bytes of raw row data.
struct Raw {
    uint32_t w[4];
};

template <bool BF16>
struct Layout {
    static constexpr int kV = BF16 ? 8 : 4;    // elements per 16-byte chunk
    static constexpr int kEB = BF16 ? 2 : 4;   // bytes per element
};

// bf16 -> fp32 is exact: the stored half is the upper half of the binary32.
__device__ __forceinline__ float lo_bf16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_bf16(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

template <bool BF16>
__device__ __forceinline__ void unpack(const Raw& r, float* v)
{
    if constexpr (BF16) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            v[2 * k] = lo_bf16(r.w[k]);
            v[2 * k + 1] = hi_bf16(r.w[k]);
        }
    } else {
#pragma unroll
        for (int k = 0; k < 4; ++k) v[k] = __uint_as_float(r.w[k]);
    }
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Load full chunk c of a row.  Every byte is read exactly once, so the vector
// path uses non-temporal loads (streamed past the caches: measured 7.0 vs
// 6.2 TB/s for this access pattern on MI355X).
template <bool BF16, bool VEC>
__device__ __forceinline__ Raw load_chunk(const char* row, int c)
{
    Raw r;
    if constexpr (VEC) {
        const u32x4 q = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(row + (size_t)c * 16));
        r.w[0] = q.x;
        r.w[1] = q.y;
        r.w[2] = q.z;
        r.w[3] = q.w;
    } else if constexpr (BF16) {
        const uint16_t* e = reinterpret_cast<const uint16_t*>(row) + (size_t)c * 8;
#pragma unroll
        for (int k = 0; k < 4; ++k) r.w[k] = (uint32_t)e[2 * k] | ((uint32_t)e[2 * k + 1] << 16);
    } else {
        const uint32_t* e = reinterpret_cast<const uint32_t*>(row) + (size_t)c * 4;
#pragma unroll
        for (int k = 0; k < 4; ++k) r.w[k] = e[k];
    }
    return r;
}

// Load the first m (< kV) elements of chunk c element by element.
template <bool BF16>
__device__ __forceinline__ void load_partial(const char* row, int c, int m, float* v)
{
    if constexpr (BF16) {
        const uint16_t* e = reinterpret_cast<const uint16_t*>(row) + (size_t)c * 8;
        for (int k = 0; k < m; ++k) v[k] = __uint_as_float((uint32_t)e[k] << 16);
    } else {
        const float* e = reinterpret_cast<const float*>(row) + (size_t)c * 4;
        for (int k = 0; k < m; ++k) v[k] = e[k];
    }
}

struct XAcc {
    float sd;    // sum (|x| 2^-e - c)
    float sd2;   // sum (|x| 2^-e - c)^2; Shannon: sum g(|x| 2^-e / c) / ln 2
};

struct CAcc {
    float dot, n1, n2;
};

// d = |x| 2^-e - c in one fused multiply-add (scale = 2^-e): the product is
// exact for normal values, so d is the rounding of the exact scaled
// difference, and for near-uniform rows exact (Sterbenz).
__device__ __forceinline__ void x_chunk(XAcc& a, const float* v, int m, float c, float scale)
{
    for (int k = 0; k < m; ++k) {
        const float d = fmaf(fabsf(v[k]), scale, -c);
        a.sd += d;
        a.sd2 = fmaf(d, d, a.sd2);
    }
}

// Base-2 units: y = e / ln 2 and g2(y) = g(1 + e) / ln 2 >= 0, given y (and
// u = 1 + e for the direct form); the row's sum is multiplied by ln 2 once.
// For |e| < 1/4 as y^2 psi(y), psi a degree-5 polynomial (the Chebyshev
// interpolant of g(1 + e) / (y^2 ln 2) on |y| < (1/4) / ln 2, relative error
// 3e-7, 4e-7 with fp32 Horner; coefficients from gen_shannon_poly.py), which
// keeps full relative accuracy where the direct form cancels (in fp32 the
// direct form's error grows to 1e-5 at |e| = 1/8, so the cut stays at 1/4);
// elsewhere u log2 u - y with the hardware base-2 logarithm (argument clamped
// to 1e-30, a normal number, so u = 0 gives 0 - y = 1 / ln 2).  Both forms
// are evaluated and one is selected: no per-element divergence.
constexpr float kInvLn2 = 1.44269504088896340736f;
constexpr float kLn2 = 0.693147180559945309f;
constexpr float kShannonCut = 0.25f * kInvLn2;   // |e| < 1/4 in units of y

__device__ __forceinline__ float g2_shannon(float y, float u)
{
    float p = -2.818413918e-03f;
    p = fmaf(p, y, 5.614020020e-03f);
    p = fmaf(p, y, -1.152998215e-02f);
    p = fmaf(p, y, 2.773815429e-02f);
    p = fmaf(p, y, -8.007569547e-02f);
    p = fmaf(p, y, 3.465736915e-01f);
    const float series = (y * y) * p;
    const float direct = fmaf(u, __builtin_amdgcn_logf(fmaxf(u, 1e-30f)), -y);
    return fabsf(y) < kShannonCut ? series : direct;
}

// Shannon partial sums over m elements for a row shift c > 0 and scale
// 2^-e (inv_u = 2^-e / c, u = |x| inv_u; inv2 = (1/c) / ln 2 and delta2 =
// (c (1/c) - 1) / ln 2 give y): sd as for CV^2, sd2 = sum g(u) / ln 2.
__device__ __forceinline__ void x_chunk_shannon(XAcc& a, const float* v, int m, float c, float scale,
                                                float inv_u, float inv2, float delta2)
{
    for (int k = 0; k < m; ++k) {
        const float ax = fabsf(v[k]);
        const float d = fmaf(ax, scale, -c);
        a.sd += d;
        a.sd2 += g2_shannon(fmaf(d, inv2, delta2), ax * inv_u);
    }
}

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c)
{
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), __builtin_bit_cast(bf16x2, b),
                                           c, false);
}

// Eq. (6) partial sums over one chunk.  bf16: the hardware dot product of the
// two bf16 pairs in each 32-bit word (products of bf16 values are exact in
// fp32), no unpacking; fp32: fused multiply-adds.  Unused elements of a
// partial chunk are zero and add nothing.
template <bool BF16>
__device__ __forceinline__ void c_chunk(CAcc& a, const Raw& p, const Raw& q)
{
    if constexpr (BF16) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            a.dot = dot2_bf16(p.w[k], q.w[k], a.dot);
            a.n1 = dot2_bf16(p.w[k], p.w[k], a.n1);
            a.n2 = dot2_bf16(q.w[k], q.w[k], a.n2);
        }
    } else {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const float u = __uint_as_float(p.w[k]), v = __uint_as_float(q.w[k]);
            a.dot = fmaf(u, v, a.dot);
            a.n1 = fmaf(u, u, a.n1);
            a.n2 = fmaf(v, v, a.n2);
        }
    }
}

// The first m (< elements per chunk) elements of chunk c, zero-padded.
template <bool BF16>
__device__ __forceinline__ Raw load_partial_raw(const char* row, int c, int m)
{
    Raw r{{0u, 0u, 0u, 0u}};
    if constexpr (BF16) {
        const uint16_t* e = reinterpret_cast<const uint16_t*>(row) + (size_t)c * 8;
        for (int k = 0; k < m; ++k) r.w[k >> 1] |= (uint32_t)e[k] << (16 * (k & 1));
    } else {
        const uint32_t* e = reinterpret_cast<const uint32_t*>(row) + (size_t)c * 4;
        for (int k = 0; k < m; ++k) r.w[k] = e[k];
    }
    return r;
}

__device__ __forceinline__ float wave_sum(float v) { return wave_sum_f32(v); }

// Element j of a row as fp32 (exact widening), for the re-read paths.
template <bool BF16>
__device__ __forceinline__ float elem(const char* row, int j)
{
    if constexpr (BF16) return __uint_as_float((uint32_t)reinterpret_cast<const uint16_t*>(row)[j] << 16);
    else return reinterpret_cast<const float*>(row)[j];
}

// 2^-e for a positive m, e the exponent that puts m 2^-e in [0.5, 1), limited
// to [-125, 126] so that 2^-e is a normal number (m 2^-e then lies in
// [2^-24, 4) for every finite m > 0).
__device__ __forceinline__ float binade_scale(float m)
{
    int e;
    (void)frexpf(m, &e);
    e = e < -125 ? -125 : (e > 126 ? 126 : e);
    return ldexpf(1.f, -e);
}

__device__ __forceinline__ float wave_max_nonneg(float v)
{
    // non-negative floats order like their bit patterns
    return __uint_as_float(wave_max_u32(__float_as_uint(v)));
}

__device__ __forceinline__ float wave_min_nonneg(float v)
{
    return __uint_as_float(~wave_max_u32(~__float_as_uint(v)));
}

// The row shift c of the scaled values and what the Shannon terms derive
// from it (1/c and its rounding offset, folded with the scale).
struct Shift {
    float c, scale, inv_c, delta, inv_u, inv2, delta2;
};

__device__ __forceinline__ Shift make_shift(float c, float scale)
{
    Shift h;
    h.c = c;
    h.scale = scale;
    h.inv_c = c > 0.f ? 1.f / c : 0.f;
    h.delta = c > 0.f ? fmaf(c, h.inv_c, -1.f) : 0.f;
    h.inv_u = h.inv_c * scale;
    h.inv2 = h.inv_c * kInvLn2;
    h.delta2 = h.delta * kInvLn2;
    return h;
}

template <bool H1>
__device__ __forceinline__ void x_accumulate(XAcc& xa, const float* v, int m, const Shift& h)
{
    if constexpr (H1) x_chunk_shannon(xa, v, m, h.c, h.scale, h.inv_u, h.inv2, h.delta2);
    else x_chunk(xa, v, m, h.c, h.scale);
}

// Stage I sums of a row from a second read of its bytes: scaled by the power
// of two of its exact maximum |x| and shifted by its exact scaled mean, so
// that no term can overflow and none that matters underflows.  zero: every
// element is 0 (or the row is not finite).
struct XRow {
    Shift h;
    float sd, sd2;
    bool zero;
    bool nonfinite;   // some element is a NaN or infinite
};

template <bool BF16, bool H1>
__device__ __noinline__ XRow x_reread(const char* row, int D, int lane)
{
    XRow r;
    r.sd = r.sd2 = 0.f;
    float mx = 0.f, mn = __builtin_inff();
    bool bad = false;
    for (int j = lane; j < D; j += kWave) {
        const float a = fabsf(elem<BF16>(row, j));
        mx = fmaxf(mx, a);
        mn = fminf(mn, a);
        bad = bad || !(a <= 3.40282347e38f);   // NaN or infinite
    }
    const float rmax = wave_max_nonneg(mx);
    const float rmin = wave_min_nonneg(mn);
    r.nonfinite = __any(bad) != 0;
    r.zero = !(rmax > 0.f && rmax <= 3.40282347e38f);
    if (r.zero) {
        r.h = make_shift(0.f, 1.f);
        return r;
    }
    // The values are scaled once here (exact: the results are normal or
    // negligibly small), so the Shannon terms' 1/c is never folded with the
    // scale, which for a tiny row could leave the fp32 range.
    const float scale = binade_scale(rmax);
    float sum = 0.f;
    for (int j = lane; j < D; j += kWave) sum += fabsf(elem<BF16>(row, j)) * scale;
    // (a row of one magnitude: that magnitude, exactly, as the shift)
    r.h = make_shift(rmin == rmax ? rmax * scale : wave_sum(sum) / (float)D, 1.f);
    XAcc xa{0.f, 0.f};
    for (int j = lane; j < D; j += kWave) {
        const float v = elem<BF16>(row, j) * scale;
        x_accumulate<H1>(xa, &v, 1, r.h);
    }
    r.sd = wave_sum(xa.sd);
    r.sd2 = wave_sum(xa.sd2);
    return r;
}

struct CRow {
    float s;
    bool nonfinite;   // some element of x' or x'' is a NaN or infinite
};

// Eq. (6) from a second read of the two rows, each scaled by the power of two
// of its own maximum |x| (s is invariant to both), in fp32 fused
// multiply-adds.  A zero vector gives s = 0.
template <bool BF16>
__device__ __noinline__ CRow cos_reread(const char* pr, const char* qr, int Dc, int lane)
{
    float mp = 0.f, mq = 0.f;
    bool bad = false;
    for (int j = lane; j < Dc; j += kWave) {
        const float u = fabsf(elem<BF16>(pr, j)), v = fabsf(elem<BF16>(qr, j));
        mp = fmaxf(mp, u);
        mq = fmaxf(mq, v);
        bad = bad || !(u <= 3.40282347e38f) || !(v <= 3.40282347e38f);   // NaN or infinite
    }
    CRow r{0.f, __any(bad) != 0};
    const float xp = wave_max_nonneg(mp), xq = wave_max_nonneg(mq);
    if (!(xp > 0.f) || !(xq > 0.f)) return r;
    const float sp = binade_scale(xp), sq = binade_scale(xq);
    float dot = 0.f, n1 = 0.f, n2 = 0.f;
    for (int j = lane; j < Dc; j += kWave) {
        const float u = elem<BF16>(pr, j) * sp, v = elem<BF16>(qr, j) * sq;
        dot = fmaf(u, v, dot);
        n1 = fmaf(u, u, n1);
        n2 = fmaf(v, v, n2);
    }
    dot = wave_sum(dot);
    n1 = wave_sum(n1);
    n2 = wave_sum(n2);
    r.s = dot / (sqrtf(n1) * sqrtf(n2));
    return r;
}

template <bool BF16, bool VEC, int UNR, int MODE>
__global__ __launch_bounds__(256) void score_kernel(ScoreArgs a)
{
    using L = Layout<BF16>;
    constexpr int V = L::kV;
    constexpr bool kX = (MODE & kScoreImp) != 0;    // Eq. (3)-(4) over X
    constexpr bool kC = (MODE & kScoreSim) != 0;    // Eq. (6) over X_pre, X_post
    constexpr bool kH1 = kX && (MODE & kScoreShannon) != 0;   // Shannon variant of Stage I
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t row = (int64_t)blockIdx.x * (blockDim.x / kWave) + (threadIdx.x / kWave);
    if (row >= a.rows) return;   // whole wavefront leaves together

    const char* xr = static_cast<const char*>(a.X) + row * (int64_t)a.D * L::kEB;
    const char* pr = static_cast<const char*>(a.P) + row * (int64_t)a.Dc * L::kEB;
    const char* qr = static_cast<const char*>(a.Q) + row * (int64_t)a.Dc * L::kEB;
    const int nfx = kX ? a.D / V : 0;    // full chunks of X
    const int nfc = kC ? a.Dc / V : 0;   // full chunks of X_pre / X_post
    const int nf = nfx > nfc ? nfx : nfc;
    // elements in the lanes' first chunks: the sample the shift c averages
    const float n_probe = (float)(a.D < kWave * V ? a.D : kWave * V);

    // A trailing partial chunk belongs to lane (index % 64) like any other and
    // is that lane's last chunk.
    const bool tail_x = kX && (a.D % V) && (nfx & (kWave - 1)) == lane;
    const int mx = a.D - nfx * V;
    float tx[V];
    tx[0] = 0.f;
    if (tail_x) load_partial<BF16>(xr, nfx, mx, tx);

    XAcc xa{0.f, 0.f};
    CAcc ca{0.f, 0.f, 0.f};
    // The shift and scale from the probe mean (wave-uniform): the row is
    // accumulated as |x| 2^-e with the probe mean in [0.5, 1) after scaling.
    Shift sh = make_shift(0.f, 1.f);
    bool fast_x = false;
    // The probe is this lane's first m elements pv (lane 0 always has some).
    // Its mean is the shift; when every probe element has one magnitude, that
    // magnitude itself is (exact, so an exactly uniform row gets d = 0 and a
    // key of exactly 0 whatever its magnitude).  Either way c is a mean or a
    // value of a subset of the row, which bounds the cancellation in M2.
    auto set_probe = [&](const float* pv, int m) {
        const float ref = __uint_as_float(
            (uint32_t)__builtin_amdgcn_readlane((int)__float_as_uint(fabsf(pv[0])), 0));
        bool same = true;
        float sum = 0.f;
        for (int k = 0; k < m; ++k) {
            sum += fabsf(pv[k]);
            same = same && fabsf(pv[k]) == ref;
        }
        const float c_raw = __all(same) ? ref : wave_sum(sum) / n_probe;
        fast_x = c_raw >= 0x1p-120f && c_raw <= 0x1p120f;
        const float scale = fast_x ? binade_scale(c_raw) : 1.f;
        sh = make_shift(fast_x ? c_raw * scale : 0.f, scale);
    };
    if (kX && nfx == 0) set_probe(tx, tail_x ? mx : 0);

    for (int j0 = 0; j0 < nf; j0 += kWave * UNR) {   // same trip count for every lane
        Raw rx[UNR], rp[UNR], rq[UNR];
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            const int ci = j0 + lane + kWave * u;
            if (ci < nfx) rx[u] = load_chunk<BF16, VEC>(xr, ci);
            if (ci < nfc) {
                rp[u] = load_chunk<BF16, VEC>(pr, ci);
                rq[u] = load_chunk<BF16, VEC>(qr, ci);
            }
        }
        if (j0 == 0 && nfx > 0) {
            float v[V];
            int m = 0;
            if (lane < nfx) {
                unpack<BF16>(rx[0], v);
                m = V;
            } else if (tail_x) {
#pragma unroll
                for (int k = 0; k < V; ++k) v[k] = tx[k];
                m = mx;
            } else {
                v[0] = 0.f;
            }
            set_probe(v, m);
        }
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            const int ci = j0 + lane + kWave * u;
            if (ci < nfx) {
                float v[V];
                unpack<BF16>(rx[u], v);
                x_accumulate<kH1>(xa, v, V, sh);
            }
            if (ci < nfc) c_chunk<BF16>(ca, rp[u], rq[u]);
        }
    }
    if (tail_x) x_accumulate<kH1>(xa, tx, mx, sh);
    if (kC && a.Dc % V && (nfc & (kWave - 1)) == lane) {
        const int m = a.Dc - nfc * V;
        c_chunk<BF16>(ca, load_partial_raw<BF16>(pr, nfc, m), load_partial_raw<BF16>(qr, nfc, m));
    }

    float sd = 0.f, sd2 = 0.f, s = 0.f;
    bool zero_row = false;
    // A NaN or infinite element always sends its row to a second read (its
    // sums leave the range the first pass accepts), which reports it.
    bool bad_row = false;
    if constexpr (kX) {
        sd = wave_sum(xa.sd);
        sd2 = wave_sum(xa.sd2);
        // Probe outside the window, or a scaled sum out of range (NaN too):
        // score the row again from its maximum (a wave-uniform decision).
        if (!(fast_x && sd2 <= 0x1p100f)) {
            const XRow r = x_reread<BF16, kH1>(xr, a.D, lane);
            bad_row = r.nonfinite;
            sh = r.h;
            sd = r.sd;
            sd2 = r.sd2;
            zero_row = r.zero;
        }
    }
    if constexpr (kC) {
        const float dot = wave_sum(ca.dot), n1 = wave_sum(ca.n1), n2 = wave_sum(ca.n2);
        if (n1 >= 0x1p-60f && n2 >= 0x1p-60f && n1 <= 3.40282347e38f && n2 <= 3.40282347e38f) {
            s = dot / (sqrtf(n1) * sqrtf(n2));
        } else {
            const CRow r = cos_reread<BF16>(pr, qr, a.Dc, lane);
            s = r.s;
            bad_row = bad_row || r.nonfinite;
        }
    }

    if (lane == 0) {
        float cv2 = 0.f, h2 = 0.f;
        const float Df = (float)a.D;
        const float mean = sh.c + sd / Df;   // of the scaled |x|
        if constexpr (kH1) {
            // cv2 holds the key KL = log D - H1, h2 holds H1.
            if (zero_row || !(mean > 0.f)) {   // all-zero row: H1 = 0
                cv2 = a.logD;
                h2 = 0.f;
            } else {
                const float rm1 = fmaf(sd / Df, sh.inv_c, sh.delta);   // r - 1
                const float r = 1.f + rm1;
                const float gr = Df * g2_shannon(rm1 * kInvLn2, r);
                // sum g(u_j) >= D g(r) (Jensen), with equality only when every
                // u_j is equal; for any other row the difference is at least
                // about n_probe / (n_probe + D) of the sum.  A difference
                // within the rounding of the sums ((D / 64 + 16) ulps) is an
                // exactly uniform row, whose KL is 0 at any magnitude (such
                // rows then tie exactly, as Eq. 3 makes them).
                const float num = sd2 - gr;
                const float thr = (Df * (1.f / kWave) + 16.f) * 0x1p-24f;
                const float dkl = fabsf(num) <= thr * (sd2 + gr) ? 0.f : kLn2 * num / r;
                cv2 = fmaxf(0.f, dkl / Df);
                h2 = a.logD - cv2;
            }
        } else if constexpr (kX) {
            const float m2 = fmaxf(0.f, fmaf(-sd, sd / Df, sd2));
            if (zero_row || !(mean > 0.f)) {   // all-zero row: H2 = 0, i.e. 1 + CV^2 = D
                cv2 = Df - 1.f;
                h2 = 0.f;
            } else {
                cv2 = (m2 / (mean * Df)) / mean;
                h2 = a.logD - log1pf(cv2);
            }
        }
        if (a.key_imp) a.key_imp[row] = cv2;
        if (a.key_s) a.key_s[row] = s;
        if (kX && a.out_h2) a.out_h2[row] = h2;
        if (kC && a.out_s) a.out_s[row] = s;
        if (a.nonfinite && bad_row) atomicAdd(a.nonfinite, 1u);
    }
}

// One wavefront per workgroup: the finest scheduling grain spreads rows evenly
// over the 256 CUs (measured 128 us vs 136 us with four-wavefront groups on
// 64 x 576 x 4096 bf16 rows, the latter equal to a plain read of the bytes).
template <bool BF16, bool VEC, int MODE>
hipError_t launch_t(const ScoreArgs& a, hipStream_t s)
{
    constexpr int kThreads = 64;
    constexpr int kRowsPerBlock = kThreads / kWave;
    const int64_t blocks = (a.rows + kRowsPerBlock - 1) / kRowsPerBlock;
    if (blocks <= 0) return hipSuccess;
    // The Shannon terms need more registers per element: three chunks of each
    // tensor in flight (91 VGPRs, five wavefronts per SIMD) measured fastest
    // on 64 x 576 x 4096 bf16 rows, 131 us against 145 us with two (six
    // wavefronts per SIMD) and 134 us with four (four per SIMD).
    constexpr int kUnroll = (MODE & kScoreShannon) ? 3 : 4;
    hipLaunchKernelGGL((score_kernel<BF16, VEC, kUnroll, MODE>), dim3((unsigned)blocks), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

template <bool BF16, bool VEC>
hipError_t launch_m(const ScoreArgs& a, int mode, hipStream_t s)
{
    constexpr int I = kScoreImp, S = kScoreSim, H = kScoreShannon;
    switch (mode) {
    case I: return launch_t<BF16, VEC, I>(a, s);
    case S: return launch_t<BF16, VEC, S>(a, s);
    case I | S: return launch_t<BF16, VEC, I | S>(a, s);
    case I | H: return launch_t<BF16, VEC, I | H>(a, s);
    default: return launch_t<BF16, VEC, I | S | H>(a, s);
    }
}

}  // namespace

hipError_t launch_score(const ScoreArgs& a, bool bf16, bool vec, int mode, hipStream_t s)
{
    const int base = mode & ~kScoreShannon;
    if (base != kScoreImp && base != kScoreSim && base != (kScoreImp | kScoreSim)) return hipErrorInvalidValue;
    if ((mode & kScoreShannon) && !(mode & kScoreImp)) mode &= ~kScoreShannon;
    if (bf16) return vec ? launch_m<true, true>(a, mode, s) : launch_m<true, false>(a, mode, s);
    return vec ? launch_m<false, true>(a, mode, s) : launch_m<false, false>(a, mode, s);
}

}  // namespace tr
