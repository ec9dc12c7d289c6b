// Per-image selection (Algorithm 1 after the scores), everything resident in
// LDS.  Images of at most kSmallSelectN tokens take select_small_kernel (one
// token per thread, both stages ranked in the same passes; described where
// it is defined).  Larger images take select_kernel: one 1024-thread
// workgroup per image, or several sharing the ranking of a large image.
//
// Keys are fp32 scores mapped to order-preserving u32 (-0 == +0).  Stage I
// keeps the K1 smallest Stage I keys (ties: lower index); Stage II orders
// X^rem by the Stage II key (ties: lower index) and keeps sorted positions
// 0, t, ..., (K2-1) t (or floor(j R / K2) in the real-interval variant); the
// output lists X^imp U X^div in token order.
//
// Stage I buckets the keys by value (1024 equal-width buckets over their
// range, one pass) and a DPP scan finds the bucket holding the K1-th smallest
// key.  One more pass keeps every lower bucket and lists the members of that
// boundary bucket; one thread per listed member then counts the members
// smaller than itself in (key, index) order and keeps it if that rank is
// below the remaining budget.  When the boundary bucket holds more than 128
// keys (or the range is not finite), Stage I instead narrows a bucket
// {k : (k & pmask) == prefix} that contains the K1-th key with 8-bit digit
// passes over the highest still-undecided bits in which some key differs
// (bytes no key varies in cost nothing): each pass is a histogram (ballot
// "same digit" masks, one LDS atomic per distinct digit per tile) and a DPP
// scan that picks the digit holding the K1-th key.  It stops when
//   - the bucket holds a single key value T: keys < T are kept, then the first
//     keys == T in token order (ordered ballot counts), or
//   - the bucket holds at most 128 keys: ranked as above.
// Stage II buckets X^rem by value, 1024 buckets of equal width over the
// [min, max] of its keys, in one pass; every token's rank in the sorted
// X^rem is then its bucket's start plus the number of its bucket's members
// smaller in (key, index) order, counted exactly: per token for small images,
// a whole bucket per wavefront for large ones (shared by several workgroups
// that each rank a fixed share of the buckets).  If a bucket exceeds 256
// tokens or the range is not finite, Stage II falls back to a stable LSD radix
// sort of the 16-bit indices of X^rem (ordered compaction first, digits looked
// up by index, per-wavefront scatter offsets, passes over constant bytes
// skipped).
//
// Every wavefront owns a contiguous, 64-aligned range of tokens for the
// ordered steps (tie marking, compaction, output), so all results are exact
// and deterministic.
#include <type_traits>

#include "tr_internal.h"
#include "tr_wave.h"

namespace tr {
namespace {

constexpr int kThreads = 1024;
constexpr int kW = kThreads / kWave;
constexpr uint32_t kCountLimit = 128;    // Stage I: count exactly inside buckets this small
constexpr int kBuckets = kThreads;       // Stage II: value buckets (one per thread in the scan)
constexpr uint32_t kBucketLimit = 256;   // Stage II: largest bucket ranked by counting
constexpr int kDenseRem = 4096;          // Stage II: rank whole buckets per wavefront from here
constexpr int kMaxSplitGroups = 64;      // most workgroups sharing the ranking of one large image
constexpr uint16_t kNoBucket = 0xffff;   // Stage II bucket index of a token not in X^rem
static_assert(kCountLimit <= (uint32_t)kThreads && kCountLimit % kWave == 0,
              "one thread per listed Stage I member, in whole wavefronts");
static_assert((kMaxSplitGroups & (kMaxSplitGroups - 1)) == 0 && kMaxSplitGroups * kW <= kBuckets,
              "split ownership is a mask; every wavefront of the groups owns a bucket");
static_assert(kDenseRem / 2 >= 2 * kWave * kW, "dense ranking's pairs fit above the X^rem list");

// ---- LDS layout (same arithmetic on host and device) -----------------------
struct LdsLayout {
    size_t ks, ki, bimp, bsel, area, slots, misc, comp, total;
    bool has_comp;
};

__host__ __device__ inline size_t align_up(size_t v, size_t a) { return (v + a - 1) & ~(a - 1); }

//   ks    u32[n]        Stage II keys by token index
//   ki    u32[n]        Stage I keys; after Stage I the same bytes hold the
//                       u16 bucket list of X^rem (lower half) and each
//                       token's u16 bucket (upper half), then the dense
//                       ranking's per-wavefront pairs above the list; or the
//                       two u16[n] index buffers of the radix sort
//   bimp  u32[nw]       X^imp bitmap (nw = 2 ceil(n / 64))
//   bsel  u32[nw]       X^imp U X^div bitmap
//   area  u32[2048]     16-byte aligned, reused by phase:
//                         Stage I:  [0, 512) two 256-bin digit histograms,
//                                   [512, 768) u64[128] bucket members
//                         Stage II: [0, 1024) bucket counts, [1024, 2048)
//                                   bucket cursors; or u16[256][W] digit
//                                   counts / offsets of the radix sort
//   slots u32[8][W]     per-wavefront partial values, one row per use
//   misc  u32[16]       broadcast slots and counters
//   comp  u64[n]        only for n < kDenseRem: X^rem as (key << 32 | index)
//                       in bucket order, for the per-token ranking
__host__ __device__ inline LdsLayout lds_layout(int n)
{
    LdsLayout L;
    const size_t nw = 2 * (((size_t)n + 63) / 64);
    size_t o = 0;
    L.ks = o;
    o += 4 * (size_t)n;
    L.ki = o;
    o += 4 * (size_t)n;
    L.bimp = o;
    o += 4 * nw;
    L.bsel = o;
    o += 4 * nw;
    o = align_up(o, 16);
    L.area = o;
    o += 4 * 2048;
    L.slots = o;
    o += 4 * 8 * kW;
    L.misc = o;
    o += 4 * 16;
    L.has_comp = n < kDenseRem;
    L.comp = 0;
    if (L.has_comp) {
        o = align_up(o, 16);
        L.comp = o;
        o += 8 * (size_t)n;
    }
    L.total = o;
    return L;
}

// LDS a launch needs for images of at most nmax tokens: the layout's size is
// not monotonic in n (comp exists only below kDenseRem), so the largest over
// n <= nmax.
__host__ __device__ inline size_t launch_lds(int nmax)
{
    const size_t big = lds_layout(nmax).total;
    if (nmax < kDenseRem) return big;
    const size_t small = lds_layout(kDenseRem - 1).total;
    return big > small ? big : small;
}

// ---- helpers -------------------------------------------------------------------
// IEEE order -> unsigned order; -0 and +0 map to the same key.
__device__ __forceinline__ uint32_t order_key(float f)
{
    const uint32_t u = __float_as_uint(f + 0.0f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Inverse of order_key.
__device__ __forceinline__ float key_value(uint32_t k)
{
    return __uint_as_float((k & 0x80000000u) ? (k ^ 0x80000000u) : ~k);
}

__device__ __forceinline__ uint64_t lanes_below(int lane) { return (1ull << lane) - 1ull; }

// Mask of active lanes whose 8-bit digit equals this lane's digit.
__device__ __forceinline__ uint64_t same_digit(uint32_t digit, bool active)
{
    uint64_t m = __ballot(active);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
        const bool bit = (digit >> b) & 1u;
        const uint64_t set = __ballot(active && bit);
        m &= bit ? set : ~set;
    }
    return m;
}

__device__ __forceinline__ bool is_leader(uint64_t m, int lane)
{
    return m && (int)(__ffsll((long long)m) - 1) == lane;
}

__device__ __forceinline__ bool bit_of(const uint32_t* bm, int i) { return (bm[i >> 5] >> (i & 31)) & 1u; }

// A wavefront writes the 64-bit ballot of tile `base` into the tile's two
// bitmap words (base is a multiple of 64 and every bitmap starts 8-byte
// aligned, so the pair is one aligned 64-bit store).
__device__ __forceinline__ void put_tile_bits(uint32_t* bm, int base, uint64_t bits, int lane)
{
    if (lane == 0) *reinterpret_cast<uint64_t*>(bm + (base >> 5)) = bits;
}

// bsel's words of tile `base` = bimp's words | bits.
__device__ __forceinline__ void put_tile_union(uint32_t* bsel, const uint32_t* bimp, int base,
                                               uint64_t bits, int lane)
{
    if (lane == 0)
        *reinterpret_cast<uint64_t*>(bsel + (base >> 5)) =
            *reinterpret_cast<const uint64_t*>(bimp + (base >> 5)) | bits;
}

// A wavefront's passes over its token range read kTileUnr tiles of 64 from
// LDS before working on any of them, so the reads overlap.
constexpr int kTileUnr = 4;

// Keys base + 64 u + lane of v (u < kTileUnr); from `end` on, the key of
// 0.0f, so that bucket arithmetic on them stays finite (callers mask them).
__device__ __forceinline__ void load_tiles(const uint32_t* v, int base, int end, int lane,
                                           uint32_t (&out)[kTileUnr])
{
#pragma unroll
    for (int u = 0; u < kTileUnr; ++u) {
        const int i = base + u * kWave + lane;
        out[u] = i < end ? v[i] : 0x80000000u;
    }
}

// Whether each of the same tokens is in X^rem (before `end`, not in bimp).
__device__ __forceinline__ void rem_tiles(const uint32_t* bimp, int base, int end, int lane,
                                          bool (&out)[kTileUnr])
{
#pragma unroll
    for (int u = 0; u < kTileUnr; ++u) {
        const int i = base + u * kWave + lane;
        out[u] = i < end && !bit_of(bimp, i);
    }
}

// Contiguous 64-aligned token range of wavefront w.
__device__ __forceinline__ void wave_range(int n, int w, int& beg, int& end)
{
    const int seg = (((n + kW - 1) / kW) + 63) & ~63;
    beg = w * seg < n ? w * seg : n;
    end = beg + seg < n ? beg + seg : n;
}

// Cross-wavefront reductions of one LDS row of per-wavefront values: lane l
// reads entry l, the wavefront reduces in registers.
static_assert(kW <= kWave, "one row entry per lane");

// Sum of the entries of wavefronts 0 .. w-1.
__device__ __forceinline__ uint32_t sum_before(const uint32_t* row, int w, int lane)
{
    return wave_sum_u32(lane < w ? row[lane] : 0u);
}

__device__ __forceinline__ uint32_t max_all(const uint32_t* row, int lane)
{
    return wave_max_u32(lane < kW ? row[lane] : 0u);
}

__device__ __forceinline__ uint32_t or_all(const uint32_t* row, int lane)
{
    return wave_or_u32(lane < kW ? row[lane] : 0u);
}

// Exclusive prefix over wavefronts of a per-wavefront count (each row of
// slots is used once per kernel).
__device__ __forceinline__ uint32_t wave_prefix(uint32_t count, uint32_t* row)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int w = threadIdx.x / kWave;
    if (lane == 0) row[w] = count;
    __syncthreads();
    return sum_before(row, w, lane);
}

struct Img {
    int row_off, n, k1, k2, t, out_off;
};

__device__ __forceinline__ Img image_of(const SelectArgs& a, int local)
{
    ImageDesc d;
    if (a.uniform) {
        d = a.desc[0];
        const int img = a.img0 + local;
        d.row_off = img * d.n;
        d.out_off = img * (d.k1 + d.k2);
    } else {
        d = a.desc[local];
    }
    return Img{d.row_off, d.n, d.k1, d.k2, d.t, d.out_off};
}

// ---- phases ------------------------------------------------------------------
// Load the image's keys (all global loads of a batch issued before the LDS
// stores), zero `nzero` words at `zero`, and return the bits in which some key
// differs from token 0's key (each kind) and the range of the Stage I keys.
struct KeyStats {
    uint32_t k0i, VI, VS, kimin, kimax;
};

__device__ KeyStats load_keys(const SelectArgs& a, const Img& d, uint32_t* ki, uint32_t* ks,
                              uint32_t* zero, int nzero, uint32_t* slots)
{
    constexpr int kUnr = 8;   // keys of each kind in flight per thread
    const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
    const int N = d.n;
    KeyStats r;
    r.k0i = order_key(a.key_imp[d.row_off]);
    const uint32_t k0s = order_key(a.key_s[d.row_off]);
    uint32_t vi = 0, vs = 0, nlo = 0, hi = 0;
    for (int i0 = tid; i0 < N; i0 += kUnr * kThreads) {
        float fi[kUnr], fs[kUnr];
#pragma unroll
        for (int u = 0; u < kUnr; ++u) {
            const int i = i0 + u * kThreads;
            if (i < N) {
                fi[u] = a.key_imp[d.row_off + i];
                fs[u] = a.key_s[d.row_off + i];
            }
        }
#pragma unroll
        for (int u = 0; u < kUnr; ++u) {
            const int i = i0 + u * kThreads;
            if (i < N) {
                const uint32_t qi = order_key(fi[u]), qs = order_key(fs[u]);
                ki[i] = qi;
                ks[i] = qs;
                vi |= qi ^ r.k0i;
                vs |= qs ^ k0s;
                nlo = max(nlo, ~qi);
                hi = max(hi, qi);
            }
        }
    }
    for (int i = tid; i < nzero; i += kThreads) zero[i] = 0;
    vi = wave_or_u32(vi);
    vs = wave_or_u32(vs);
    nlo = wave_max_u32(nlo);
    hi = wave_max_u32(hi);
    if (lane == 0) {
        slots[w] = vi;
        slots[kW + w] = vs;
        slots[2 * kW + w] = nlo;
        slots[3 * kW + w] = hi;
    }
    __syncthreads();
    r.VI = or_all(slots, lane);
    r.VS = or_all(slots + kW, lane);
    nlo = max_all(slots + 2 * kW, lane);
    hi = max_all(slots + 3 * kW, lane);
    r.kimin = ~nlo;
    r.kimax = hi;
    return r;
}

// Append (key, index) of the lanes with `member` set to `list`, reserving the
// wavefront's slots with one atomic on the counter `cnt`.
__device__ __forceinline__ void append_member(bool member, uint32_t key, int i, uint64_t* list,
                                              uint32_t* cnt, int lane)
{
    const uint64_t bm = __ballot(member);
    if (!bm) return;
    const int leader = (int)__ffsll((long long)bm) - 1;
    uint32_t b0 = 0;
    if (lane == leader) b0 = atomicAdd(cnt, (uint32_t)__popcll(bm));
    b0 = (uint32_t)__builtin_amdgcn_readlane((int)b0, leader);
    if (member) list[b0 + __popcll(bm & lanes_below(lane))] = ((uint64_t)key << 16) | (uint32_t)i;
}

// Keep the `need` smallest of the m listed (key, index) members of the Stage I
// boundary bucket: thread j counts the entries below entry j (the entries are
// distinct, so the counts are the ranks) and sets the member's bits.  With ks
// given, the Stage II keys of the members left in X^rem are folded into the
// per-wavefront range rows (~min, max) of wavefronts 0 and 1.
__device__ void keep_ranked_members(const uint64_t* list, uint32_t m, uint32_t need, uint32_t* bimp,
                                    uint32_t* bsel, const uint32_t* ks, uint32_t* row_lo,
                                    uint32_t* row_hi)
{
    const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
    uint32_t nlo = 0, hi = 0;
    if (tid < (int)m) {
        const uint64_t mine = list[tid];
        uint32_t r = 0;
        for (uint32_t j = 0; j < m; ++j) r += list[j] < mine ? 1u : 0u;
        const int i = (int)(mine & 0xffffu);
        if (r < need) {
            atomicOr(&bimp[i >> 5], 1u << (i & 31));
            atomicOr(&bsel[i >> 5], 1u << (i & 31));
        } else if (ks) {
            nlo = ~ks[i];
            hi = ks[i];
        }
    }
    if (ks && tid < (int)kCountLimit) {   // whole wavefronts: every lane takes part
        nlo = wave_max_u32(nlo);
        hi = wave_max_u32(hi);
        if (lane == 0) {
            row_lo[w] = max(row_lo[w], nlo);
            row_hi[w] = max(row_hi[w], hi);
        }
    }
}

// Stage I digit passes (see the file comment).  On return the bucket
// {k : (k & pmask) == prefix} holds m keys and the K1-th smallest key overall
// is its need-th smallest; resolved means the bucket is a single key value.
__device__ void stage1_narrow(const uint32_t* ki, int N, uint32_t VI, uint32_t* hsh, uint32_t* misc,
                              uint32_t limit, uint32_t& prefix, uint32_t& pmask, uint32_t& need,
                              uint32_t& m, bool& resolved)
{
    const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
    int beg, end;
    wave_range(N, w, beg, end);
    resolved = false;
    for (int p = 0;; ++p) {
        const uint32_t vrem = VI & ~pmask;
        if (vrem == 0) {
            resolved = true;
            return;
        }
        if (m <= limit) return;
        const int hb = 31 - __clz((int)vrem);
        const int lo = hb >= 7 ? hb - 7 : 0;
        const uint32_t win = (hb == 31 ? 0xffffffffu : ((2u << hb) - 1u)) & ~((1u << lo) - 1u);
        uint32_t* H = hsh + (p & 1) * 256;
        if (tid < 256) hsh[((p + 1) & 1) * 256 + tid] = 0;   // the next pass's histogram
        for (int base = beg; base < end; base += kWave) {
            const int i = base + lane;
            bool act = i < end;
            const uint32_t key = act ? ki[i] : 0u;
            act = act && ((key & pmask) == prefix);
            const uint32_t dg = (key >> lo) & 255u;
            const uint64_t mm = same_digit(dg, act);
            if (act && is_leader(mm, lane)) atomicAdd(&H[dg], (uint32_t)__popcll(mm));
        }
        __syncthreads();
        if (w == 0) {
            const uint4 c4 = *reinterpret_cast<const uint4*>(H + lane * 4);
            const uint32_t c[4] = {c4.x, c4.y, c4.z, c4.w};
            const uint32_t sum = c[0] + c[1] + c[2] + c[3];
            uint32_t run = wave_scan_add(sum) - sum;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                if (run < need && need <= run + c[q]) {
                    misc[0] = (uint32_t)(lane * 4 + q);
                    misc[1] = need - run;
                    misc[2] = c[q];
                }
                run += c[q];
            }
        }
        __syncthreads();
        prefix |= misc[0] << lo;
        need = misc[1];
        m = misc[2];
        pmask |= win;
    }
}

// Value bucket of a key: floor((v - fmin) * scale) clamped to the last
// bucket, non-decreasing in the key.  Callers guarantee a finite width and
// scale, so for keys in [fmin, fmax] the product is finite and in range.
__device__ __forceinline__ int value_bucket(uint32_t key, float fmin, float scale)
{
    return min(kBuckets - 1, (int)((key_value(key) - fmin) * scale));
}

// Stage I by one bucketing pass: 1024 buckets of equal width over the key
// range; tokens in buckets below the one holding the K1-th key are kept, and
// members of that bucket (at most kCountLimit of them) are kept when fewer
// than the remaining budget of members precede them in (key, index) order.
// H (kBuckets words) must be zero; list holds kCountLimit u64; misc[8] must be
// 0.  On success row_lo / row_hi hold per-wavefront (~min, max) of the Stage II
// keys of X^rem, so Stage II needs no range pass of its own.  Returns false
// (having written only H, misc[0..2] and `row`) when the range is not finite
// or the boundary bucket is larger.
__device__ bool stage1_bucket(const uint32_t* ki, const uint32_t* ks, int N, uint32_t K1,
                              uint32_t kimin, uint32_t kimax, uint32_t* H, uint64_t* list,
                              uint32_t* misc, uint32_t* row, uint32_t* row_lo, uint32_t* row_hi,
                              uint32_t* bimp, uint32_t* bsel)
{
    const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
    int beg, end;
    wave_range(N, w, beg, end);
    const float fmin = key_value(kimin);
    const float width = key_value(kimax) - fmin;
    if (!(width > 0.f) || !(width < 3.0e38f)) return false;
    const float scale = (float)kBuckets / width;
    if (!(scale < 3.0e38f)) return false;   // a range of denormals: bucket arithmetic would overflow
    for (int base = beg; base < end; base += kTileUnr * kWave) {
        uint32_t k[kTileUnr];
        load_tiles(ki, base, end, lane, k);
#pragma unroll
        for (int u = 0; u < kTileUnr; ++u) {
            const int dg = value_bucket(k[u], fmin, scale);
            if (base + u * kWave + lane < end) atomicAdd(&H[dg], 1u);
        }
    }
    __syncthreads();
    {   // thread tid owns bucket tid: find the bucket holding the K1-th key
        const uint32_t c = H[tid];
        const uint32_t inc = wave_scan_add(c);
        if (lane == kWave - 1) row[w] = inc;
        __syncthreads();
        const uint32_t start = inc - c + sum_before(row, w, lane);
        if (start < K1 && K1 <= start + c) {
            misc[0] = (uint32_t)tid;
            misc[1] = K1 - start;
            misc[2] = c;
        }
    }
    __syncthreads();
    const int dstar = (int)misc[0];
    const uint32_t need = misc[1];
    if (misc[2] > kCountLimit) return false;
    uint32_t nlo = 0, hi = 0;   // Stage II key range of the tokens above the boundary bucket
    for (int base = beg; base < end; base += kTileUnr * kWave) {
        uint32_t k[kTileUnr], q[kTileUnr];
        load_tiles(ki, base, end, lane, k);
        load_tiles(ks, base, end, lane, q);
#pragma unroll
        for (int u = 0; u < kTileUnr; ++u) {
            const int tb = base + u * kWave;
            if (tb >= end) break;   // the next tiles belong to the next wavefront
            const int i = tb + lane;
            const int dv = value_bucket(k[u], fmin, scale);
            const int dg = i < end ? dv : kBuckets;
            const uint64_t bt = __ballot(dg < dstar);
            put_tile_bits(bimp, tb, bt, lane);
            put_tile_bits(bsel, tb, bt, lane);
            append_member(dg == dstar, k[u], i, list, &misc[8], lane);
            const bool above = i < end && dg > dstar;
            nlo = max(nlo, above ? ~q[u] : 0u);
            hi = max(hi, above ? q[u] : 0u);
        }
    }
    nlo = wave_max_u32(nlo);
    hi = wave_max_u32(hi);
    if (lane == 0) {
        row_lo[w] = nlo;
        row_hi[w] = hi;
    }
    __syncthreads();
    keep_ranked_members(list, misc[8], need, bimp, bsel, ks, row_lo, row_hi);
    return true;
}

// Stage I marking with a resolved threshold key T: keys < T, then the first
// `need` keys == T in token order.
__device__ void stage1_mark_resolved(const uint32_t* ki, int N, uint32_t T, uint32_t need,
                                     uint32_t* bimp, uint32_t* bsel, uint32_t* row)
{
    const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
    int beg, end;
    wave_range(N, w, beg, end);
    uint32_t eq = 0;
    for (int base = beg; base < end; base += kWave) {
        const int i = base + lane;
        eq += __popcll(__ballot(i < end && ki[i] == T));
    }
    uint32_t rank = wave_prefix(eq, row);
    for (int base = beg; base < end; base += kWave) {
        const int i = base + lane;
        const bool act = i < end;
        const uint32_t key = act ? ki[i] : 0xffffffffu;
        const bool is_eq = act && key == T;
        const uint64_t be = __ballot(is_eq);
        const uint32_t r = rank + (uint32_t)__popcll(be & lanes_below(lane));
        const bool take = act && (key < T || (is_eq && r < need));
        const uint64_t bt = __ballot(take);
        put_tile_bits(bimp, base, bt, lane);
        put_tile_bits(bsel, base, bt, lane);
        rank += (uint32_t)__popcll(be);
    }
}

// Stage I marking by exact counting inside a bucket of at most kCountLimit
// keys: keys below the bucket are kept, and a member is kept when fewer than
// `need` members precede it in (key, index) order.  misc[8] must be 0.
__device__ void stage1_mark_counted(const uint32_t* ki, int N, uint32_t prefix, uint32_t pmask,
                                    uint32_t need, uint64_t* list, uint32_t* misc, uint32_t* bimp,
                                    uint32_t* bsel)
{
    const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
    int beg, end;
    wave_range(N, w, beg, end);
    for (int base = beg; base < end; base += kWave) {
        const int i = base + lane;
        const bool act = i < end;
        const uint32_t key = act ? ki[i] : 0u;
        const uint64_t bt = __ballot(act && (key & pmask) < prefix);
        put_tile_bits(bimp, base, bt, lane);
        put_tile_bits(bsel, base, bt, lane);
        append_member(act && (key & pmask) == prefix, key, i, list, &misc[8], lane);
    }
    __syncthreads();
    keep_ranked_members(list, misc[8], need, bimp, bsel, nullptr, nullptr, nullptr);
}

// X^div positions in the ascending order of X^rem (R tokens, K2 picks).
// Algorithm 1: 0, t, ..., (K2 - 1) t.  Real-interval variant (the interval
// R / K2 of the method's prose): floor(j R / K2), j < K2.  Every product
// stays below 2^32 because R, K2 <= 65535.
struct Stride {
    uint32_t t, R, K2;
    bool real;
    // Is rank r a pick?  Real variant: the smallest j with floor(j R / K2) >=
    // r is ceil(r K2 / R); r is a pick iff that j is in range and lands on r.
    __device__ __forceinline__ bool picks(uint32_t r) const
    {
        if (!real) return r % t == 0 && r < K2 * t;
        const uint32_t j = (r * K2 + R - 1) / R;
        return j < K2 && (j * R) / K2 == r;
    }
    __device__ __forceinline__ uint32_t pos(uint32_t j) const { return real ? (j * R) / K2 : j * t; }
};

// Result of stage2_bucket.
constexpr int kS2Failed = 0;   // nothing decided: sort instead
constexpr int kS2Local = 1;    // every pick is in bsel
constexpr int kS2Global = 2;   // this group's picks are in the global bitmap

// Stage II by one bucketing pass and exact counting inside buckets.  Bucket
// d of a remaining token is floor((s - s_min) * B / (s_max - s_min)) (B =
// 1024 buckets over the remainder's key range: the image's whole range would
// be cheaper to get, but Stage I tends to keep the tokens with outlying keys
// and the rest would crowd into few buckets), a non-decreasing function of s
// in fp32 (every step rounds monotonically), so bucket order agrees with key
// order and counting inside a bucket the members smaller in (key, index)
// order gives the exact rank.
//   dgs   u16[n]  each token's bucket (kNoBucket outside X^rem), written by
//                 the histogram pass, read by the list pass
//   list  u16[n]  the indices of X^rem in bucket order; with `parts`
//                 workgroups on a dense image each lists only the buckets it
//                 ranks
//   pairs         2 kWave words per wavefront for the dense ranking (may
//                 overlap dgs, which is dead by then)
//   comp  u64[n]  or null: for the per-token ranking, X^rem as
//                 (key << 32 | index) in bucket order, listed instead of
//                 `list` (one LDS read per compared member instead of two
//                 dependent ones)
// H (B words) must be zero.  Returns kS2Failed, having written only H, cur,
// dgs, list and slot rows, when a bucket holds more than kBucketLimit tokens
// or the key range is not finite.
__device__ int stage2_bucket(const uint32_t* ks, const uint32_t* bimp, uint32_t* bsel, int N,
                              int R, const Stride& sp, uint32_t* H, uint32_t* cur, uint16_t* list,
                              uint16_t* dgs, uint32_t* pairs, uint32_t* row_lo, uint32_t* row_hi,
                              uint32_t* row_a, uint32_t* row_b, int part, int parts,
                              uint32_t* gpick, bool have_range, uint64_t* comp)
{
    const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
    int beg, end;
    wave_range(N, w, beg, end);

    // key range of X^rem (max of the complement gives the minimum), unless
    // Stage I left it in the rows (the same decision in every thread)
    if (!have_range) {
        uint32_t nlo = 0, hi = 0;
        for (int base = beg; base < end; base += kTileUnr * kWave) {
            uint32_t k[kTileUnr];
            bool rem[kTileUnr];
            load_tiles(ks, base, end, lane, k);
            rem_tiles(bimp, base, end, lane, rem);
#pragma unroll
            for (int u = 0; u < kTileUnr; ++u) {
                if (rem[u]) {
                    nlo = max(nlo, ~k[u]);
                    hi = max(hi, k[u]);
                }
            }
        }
        nlo = wave_max_u32(nlo);
        hi = wave_max_u32(hi);
        if (lane == 0) {
            row_lo[w] = nlo;
            row_hi[w] = hi;
        }
        __syncthreads();
    }
    const uint32_t kmin = ~max_all(row_lo, lane), kmax = max_all(row_hi, lane);

    if (kmin == kmax) {
        // Every remaining key is equal: the stable order is the token order of X^rem.
        uint32_t rc = 0;
        for (int base = beg; base < end; base += kWave) {
            const int i = base + lane;
            rc += __popcll(__ballot(i < end && !bit_of(bimp, i)));
        }
        uint32_t r0 = wave_prefix(rc, row_a);
        for (int base = beg; base < end; base += kWave) {
            const int i = base + lane;
            const bool rem = i < end && !bit_of(bimp, i);
            const uint64_t br = __ballot(rem);
            const uint32_t r = r0 + (uint32_t)__popcll(br & lanes_below(lane));
            const uint64_t bp = __ballot(rem && sp.picks(r));
            put_tile_union(bsel, bimp, base, bp, lane);
            r0 += (uint32_t)__popcll(br);
        }
        return kS2Local;
    }
    const float fmin = key_value(kmin);
    const float width = key_value(kmax) - fmin;
    if (!(width > 0.f) || !(width < 3.0e38f)) return kS2Failed;   // not finite: sort instead
    const float scale = (float)kBuckets / width;
    if (!(scale < 3.0e38f)) return kS2Failed;   // a range of denormals: sort instead

    for (int base = beg; base < end; base += kTileUnr * kWave) {
        uint32_t k[kTileUnr];
        bool rem[kTileUnr];
        load_tiles(ks, base, end, lane, k);
        rem_tiles(bimp, base, end, lane, rem);
#pragma unroll
        for (int u = 0; u < kTileUnr; ++u) {
            const int i = base + u * kWave + lane;
            const int dg = value_bucket(k[u], fmin, scale);
            if (rem[u]) atomicAdd(&H[dg], 1u);
            if (i < end) dgs[i] = rem[u] ? (uint16_t)dg : kNoBucket;
        }
    }
    __syncthreads();
    {   // exclusive bucket starts and the largest bucket; thread tid owns bucket tid
        const uint32_t c = H[tid];
        const uint32_t inc = wave_scan_add(c);
        const uint32_t mx = wave_max_u32(c);
        if (lane == kWave - 1) row_a[w] = inc;
        if (lane == 0) row_b[w] = mx;
        __syncthreads();
        const uint32_t start = inc - c + sum_before(row_a, w, lane);
        const uint32_t big = max_all(row_b, lane);
        cur[tid] = start;
        if (big > kBucketLimit) return kS2Failed;   // the same decision in every thread
    }
    __syncthreads();
    // Dense ranking gives bucket q to wavefront q % (parts W) across the
    // groups, so to group (q / W) % parts (parts is 1 or a power of two).
    // The per-token ranking reads X^rem packed as (key, index) when the
    // layout has room for it and buckets hold a member or more on average
    // (packing costs a wider store per member; with fewer members per bucket
    // there is little to compare: 576 tokens 0.56 -> 0.76 us of listing for
    // no ranking gain; 2880 tokens 4.4 -> 3.3 us of ranking).
    const bool dense = R >= kDenseRem;
    const bool pack = !dense && comp != nullptr && R >= kBuckets;
    auto list_pass = [&](auto packed) {   // one loop per form: the choice is per image
        for (int base = beg; base < end; base += kTileUnr * kWave) {
            uint32_t g[kTileUnr];
            bool own[kTileUnr];
#pragma unroll
            for (int u = 0; u < kTileUnr; ++u) {
                const int i = base + u * kWave + lane;
                g[u] = i < end ? dgs[i] : kNoBucket;
            }
#pragma unroll
            for (int u = 0; u < kTileUnr; ++u) {   // all cursor atomics, then the stores
                own[u] = g[u] != kNoBucket && (!dense || ((g[u] / kW) & (parts - 1)) == (uint32_t)part);
                if (own[u]) g[u] = atomicAdd(&cur[g[u]], 1u);
            }
#pragma unroll
            for (int u = 0; u < kTileUnr; ++u) {
                const int i = base + u * kWave + lane;
                if constexpr (decltype(packed)::value) {
                    if (own[u]) comp[g[u]] = ((uint64_t)ks[i] << 32) | (uint32_t)i;
                } else {
                    if (own[u]) list[g[u]] = (uint16_t)i;
                }
            }
        }
    };
    if (pack) list_pass(std::true_type{});
    else list_pass(std::false_type{});
    __syncthreads();
    if (dense) {
        // Dense buckets: a wavefront ranks a whole bucket at a time, one
        // member per lane (64 per chunk).  Each chunk of the bucket is
        // staged as (index, key) word pairs in the wavefront's own `pairs`
        // row, where every lane reads each pair with one broadcast LDS read
        // and compares (key, index) as one 64-bit value.  LDS operations of
        // one wavefront complete in order, so a pair written by any lane is
        // visible to the reads after it.  With `parts` workgroups on the
        // image, bucket q belongs to the wavefront numbered q % (parts W)
        // across them (lane q / (parts W)); picks then go to the image's
        // global pick bitmap gpick.
        uint32_t* wp = pairs + 2 * kWave * w;
        const int q = part * kW + w + parts * kW * lane;
        const bool mine = q < kBuckets;
        const uint32_t cnt = mine ? H[q] : 0u;
        const uint32_t stop = mine ? cur[q] : 0u;
        uint64_t todo = __ballot(cnt > 0);
        while (todo) {
            const int l = (int)__ffsll((long long)todo) - 1;
            todo &= todo - 1;
            const uint32_t b = (uint32_t)__builtin_amdgcn_readlane((int)cnt, l);
            const uint32_t start = (uint32_t)__builtin_amdgcn_readlane((int)stop, l) - b;
            for (uint32_t c0 = 0; c0 < b; c0 += kWave) {
                const bool have = c0 + lane < b;
                const uint32_t myid = have ? list[start + c0 + lane] : 0u;
                const uint64_t me = have ? ((uint64_t)ks[myid] << 32) | myid : 0ull;
                uint32_t r = 0;
                for (uint32_t c1 = 0; c1 < b; c1 += kWave) {
                    const bool oh = c1 + lane < b;
                    const uint32_t oid = oh ? list[start + c1 + lane] : 0u;
                    const uint32_t okey = oh ? ks[oid] : 0u;
                    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
                    wp[2 * lane] = oid;
                    wp[2 * lane + 1] = okey;
                    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
                    const uint32_t n1 = min((uint32_t)kWave, b - c1);
                    uint32_t j = 0;
                    for (; j + 4 <= n1; j += 4) {   // four reads in flight
                        uint64_t o[4];
#pragma unroll
                        for (int u = 0; u < 4; ++u)
                            o[u] = ((uint64_t)wp[2 * (j + u) + 1] << 32) | wp[2 * (j + u)];
#pragma unroll
                        for (int u = 0; u < 4; ++u) r += o[u] < me ? 1u : 0u;
                    }
                    for (; j < n1; ++j) {
                        const uint64_t o = ((uint64_t)wp[2 * j + 1] << 32) | wp[2 * j];
                        r += o < me ? 1u : 0u;
                    }
                }
                const uint32_t rr = start + r;
                if (have && sp.picks(rr)) {
                    if (gpick) atomicOr(&gpick[myid >> 5], 1u << (myid & 31));
                    else atomicOr(&bsel[myid >> 5], 1u << (myid & 31));
                }
            }
        }
        return gpick ? kS2Global : kS2Local;
    }
    for (int base = beg; base < end; base += kWave) {
        const int i = base + lane;
        const bool rem = i < end && !bit_of(bimp, i);
        bool picked = false;
        if (rem && pack) {
            const uint32_t key = ks[i];
            const uint64_t me = ((uint64_t)key << 32) | (uint32_t)i;
            const int dg = value_bucket(key, fmin, scale);
            const uint32_t stop = cur[dg];
            uint32_t j = stop - H[dg];
            uint32_t r = j;
            for (; j + 8 <= stop; j += 8) {   // eight independent reads in flight
                uint64_t c[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) c[u] = comp[j + u];
#pragma unroll
                for (int u = 0; u < 8; ++u) r += c[u] < me ? 1u : 0u;
            }
            for (; j < stop; ++j) r += comp[j] < me ? 1u : 0u;
            picked = sp.picks(r);
        } else if (rem) {
            const uint32_t key = ks[i];
            const int dg = value_bucket(key, fmin, scale);
            const uint32_t stop = cur[dg];
            uint32_t j = stop - H[dg];
            uint32_t r = j;
            for (; j + 4 <= stop; j += 4) {
                const uint32_t i0 = list[j], i1 = list[j + 1], i2 = list[j + 2], i3 = list[j + 3];
                const uint32_t k0 = ks[i0], k1 = ks[i1], k2 = ks[i2], k3 = ks[i3];
                r += (k0 < key || (k0 == key && i0 < (uint32_t)i)) ? 1u : 0u;
                r += (k1 < key || (k1 == key && i1 < (uint32_t)i)) ? 1u : 0u;
                r += (k2 < key || (k2 == key && i2 < (uint32_t)i)) ? 1u : 0u;
                r += (k3 < key || (k3 == key && i3 < (uint32_t)i)) ? 1u : 0u;
            }
            for (; j < stop; ++j) {
                const uint32_t ij = list[j], kj = ks[ij];
                r += (kj < key || (kj == key && ij < (uint32_t)i)) ? 1u : 0u;
            }
            picked = sp.picks(r);
        }
        const uint64_t bp = __ballot(picked);
        put_tile_union(bsel, bimp, base, bp, lane);
    }
    return kS2Local;
}

// Stage II by ordered compaction and a stable LSD radix sort of 16-bit
// indices; sets the X^div bits in bsel.  idx_a / idx_b hold n u16 each.
__device__ void stage2_radix(const uint32_t* ks, const uint32_t* bimp, uint32_t* bsel, int N, int K1,
                             const Stride& sp, uint32_t VS, uint16_t* idx_a, uint16_t* idx_b,
                             uint16_t* hist, uint32_t* row_c, uint32_t* row_s)
{
    const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
    int beg, end;
    wave_range(N, w, beg, end);
    uint32_t rc = 0;
    for (int base = beg; base < end; base += kWave) {
        const int i = base + lane;
        rc += __popcll(__ballot(i < end && !bit_of(bimp, i)));
    }
    uint32_t pos = wave_prefix(rc, row_c);
    for (int base = beg; base < end; base += kWave) {
        const int i = base + lane;
        const bool keep = i < end && !bit_of(bimp, i);
        const uint64_t bk = __ballot(keep);
        if (keep) idx_a[pos + __popcll(bk & lanes_below(lane))] = (uint16_t)i;
        pos += (uint32_t)__popcll(bk);
    }
    const int R = N - K1;
    int begR, endR;
    wave_range(R, w, begR, endR);
    uint16_t* src = idx_a;
    uint16_t* dst = idx_b;
    for (int shift = 0; shift < 32; shift += 8) {
        if (((VS >> shift) & 255u) == 0) continue;   // every key has the same byte here
        uint32_t* h32 = reinterpret_cast<uint32_t*>(hist);
        for (int i = tid; i < 128 * kW; i += kThreads) h32[i] = 0;
        __syncthreads();
        for (int base = begR; base < endR; base += kWave) {
            const int i = base + lane;
            const bool act = i < endR;
            const uint32_t id = act ? src[i] : 0u;
            const uint32_t dg = act ? (ks[id] >> shift) & 255u : 0u;
            const uint64_t m = same_digit(dg, act);
            if (act && is_leader(m, lane)) hist[dg * kW + w] = (uint16_t)(hist[dg * kW + w] + __popcll(m));
        }
        __syncthreads();
        {   // exclusive scan of hist in (digit, wavefront) order, 4 entries per thread
            const int e = tid * 4;
            const uint2 hv = *reinterpret_cast<const uint2*>(hist + e);
            const uint32_t h0 = hv.x & 0xffffu, h1 = hv.x >> 16, h2 = hv.y & 0xffffu, h3 = hv.y >> 16;
            const uint32_t v = h0 + h1 + h2 + h3;
            const uint32_t inc = wave_scan_add(v);
            if (lane == kWave - 1) row_s[w] = inc;
            __syncthreads();
            const uint32_t b0 = inc - v + sum_before(row_s, w, lane);
            const uint32_t o1 = b0 + h0, o2 = o1 + h1, o3 = o2 + h2;
            *reinterpret_cast<uint2*>(hist + e) = make_uint2(b0 | (o1 << 16), o2 | (o3 << 16));
        }
        __syncthreads();
        for (int base = begR; base < endR; base += kWave) {
            const int i = base + lane;
            const bool act = i < endR;
            const uint32_t id = act ? src[i] : 0u;
            const uint32_t dg = act ? (ks[id] >> shift) & 255u : 0u;
            const uint64_t m = same_digit(dg, act);
            const uint32_t off = act ? hist[dg * kW + w] : 0u;
            if (act) dst[off + __popcll(m & lanes_below(lane))] = (uint16_t)id;
            if (act && is_leader(m, lane)) hist[dg * kW + w] = (uint16_t)(off + __popcll(m));
        }
        __syncthreads();
        uint16_t* tmp = src;
        src = dst;
        dst = tmp;
    }
    __syncthreads();   // the compaction (or the last pass) is visible to every picker
    for (int j = tid; j < (int)sp.K2; j += kThreads) {
        const int id = src[sp.pos((uint32_t)j)];
        atomicOr(&bsel[id >> 5], 1u << (id & 31));
    }
}

// Lane t's value of a 64-bit register, on every lane (t wavefront-uniform).
__device__ __forceinline__ uint64_t lane_u64(uint64_t v, int t)
{
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, t);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), t);
    return ((uint64_t)hi << 32) | lo;
}

// X* in ascending token index: out_idx (image-local), out_src, out_rows.
// Lane t of each wavefront holds the 64-bit bsel and bimp words of the
// wavefront's t-th tile (a range has at most 64 tiles at the capacity's N),
// so the counts and the ordered writes read LDS once per wavefront.
__device__ void emit(const SelectArgs& a, const Img& d, const uint32_t* bimp, const uint32_t* bsel,
                     uint32_t* row)
{
    const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
    int beg, end;
    wave_range(d.n, w, beg, end);
    const int tiles = (end - beg + kWave - 1) / kWave;
    uint64_t sel = 0, imp = 0;
    if (lane < tiles) {
        sel = *reinterpret_cast<const uint64_t*>(bsel + ((beg >> 5) + 2 * lane));
        imp = *reinterpret_cast<const uint64_t*>(bimp + ((beg >> 5) + 2 * lane));
        const int valid = end - (beg + kWave * lane);   // tokens of this tile inside the image
        if (valid < kWave) sel &= (1ull << valid) - 1ull;
    }
    uint32_t opos = wave_prefix(wave_sum_u32((uint32_t)__popcll(sel)), row);
    const int K = d.k1 + d.k2;
    for (int t = 0; t < tiles; ++t) {
        const uint64_t m = lane_u64(sel, t), im = lane_u64(imp, t);
        const int i = beg + kWave * t + lane;
        const int slot = (int)opos + __popcll(m & lanes_below(lane));
        if (((m >> lane) & 1ull) && slot < K) {   // never more than K writes, whatever the keys
            const int o = d.out_off + slot;
            a.out_idx[o] = i;
            if (a.out_src) a.out_src[o] = ((im >> lane) & 1ull) ? 0 : 1;
            if (a.out_rows) a.out_rows[o] = d.row_off + i;
        }
        opos += (uint32_t)__popcll(m);
    }
}

__global__ __launch_bounds__(kThreads) void select_kernel(SelectArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int G = a.groups > 0 ? a.groups : 1;
    const int local = (int)blockIdx.x / G, part = (int)blockIdx.x % G;
    const int img = a.img0 + local;
    const Img d = image_of(a, local);
    const int N = d.n, K1 = d.k1, K2 = d.k2;
    // A large image is shared by G workgroups: each repeats the deterministic
    // Stage I and bucketing in its own LDS and ranks 1/G of the buckets into
    // the image's global pick bitmap; emit_kernel then writes the output.
    const bool split = G > 1 && K2 > 0 && N - K1 >= kDenseRem;   // as select_shares
    if (part > 0 && !split) return;
    const LdsLayout L = lds_layout(N);
    uint32_t* ks = reinterpret_cast<uint32_t*>(smem + L.ks);
    uint32_t* ki = reinterpret_cast<uint32_t*>(smem + L.ki);
    uint32_t* bimp = reinterpret_cast<uint32_t*>(smem + L.bimp);
    uint32_t* bsel = reinterpret_cast<uint32_t*>(smem + L.bsel);
    uint32_t* area = reinterpret_cast<uint32_t*>(smem + L.area);
    uint32_t* slots = reinterpret_cast<uint32_t*>(smem + L.slots);
    uint32_t* misc = reinterpret_cast<uint32_t*>(smem + L.misc);
    const int nw = 2 * ((N + 63) / 64);

    // Slot rows (each written, then read after a barrier, then not touched
    // again until further barriers have passed): 0-3 key ranges and varying
    // bits, 4 Stage I scans, 5 Stage I tie ranks, 6-7 Stage II ranges (from
    // Stage I's bucket path or Stage II's own pass), 2-3 Stage II scans, 4-5
    // the radix sort, 6 the output offsets.
    if (threadIdx.x < 16) misc[threadIdx.x] = 0;
    const KeyStats ksd = load_keys(a, d, ki, ks, area, kBuckets, slots);
    const uint32_t kimin = ksd.kimin, kimax = ksd.kimax;

    // ---- Stage I ---------------------------------------------------------------
    uint64_t* list1 = reinterpret_cast<uint64_t*>(area + kBuckets);   // kCountLimit u64
    bool s2_range = false;   // Stage I's bucket path leaves X^rem's key range in rows 6-7
    if (K1 == 0 || K1 == N) {
        const uint32_t fill = K1 ? 0xffffffffu : 0u;
        for (int i = threadIdx.x; i < nw; i += kThreads) {
            bimp[i] = fill;
            bsel[i] = fill;
        }
    } else if (kimin == kimax) {   // every key is equal: the first K1 tokens
        stage1_mark_resolved(ki, N, kimin, (uint32_t)K1, bimp, bsel, slots + 5 * kW);
    } else if (stage1_bucket(ki, ks, N, (uint32_t)K1, kimin, kimax, area, list1, misc, slots + 4 * kW,
                             slots + 6 * kW, slots + 7 * kW, bimp, bsel)) {
        s2_range = true;
    } else {
        __syncthreads();   // everyone is past the bucket attempt: reset its scratch
        area[threadIdx.x] = 0;
        if (threadIdx.x < 16) misc[threadIdx.x] = 0;
        __syncthreads();
        uint32_t prefix = ksd.k0i & ~ksd.VI, pmask = ~ksd.VI, need = (uint32_t)K1, m = (uint32_t)N;
        bool resolved;
        stage1_narrow(ki, N, ksd.VI, area, misc, kCountLimit, prefix, pmask, need, m, resolved);
        if (resolved) stage1_mark_resolved(ki, N, prefix, need, bimp, bsel, slots + 5 * kW);
        else stage1_mark_counted(ki, N, prefix, pmask, need, list1, misc, bimp, bsel);
    }
    __syncthreads();   // Stage I's histograms and list are read no more; ki is dead
    area[threadIdx.x] = 0;   // Stage II bucket counts
    __syncthreads();

    // ---- Stage II --------------------------------------------------------------
    if (K2 > 0) {
        uint16_t* idx = reinterpret_cast<uint16_t*>(ki);
        const size_t wbase = (size_t)(d.row_off >> 5) + 2 * (size_t)img;
        uint32_t* gpick = split ? a.gsel + wbase : nullptr;
        const Stride sp{(uint32_t)d.t, (uint32_t)(N - K1), (uint32_t)K2, a.stride_real != 0};
        // ki's bytes after Stage I: the u16 list of X^rem in the lower half;
        // the u16 bucket index of every token in the upper half (until the
        // list is built); then the dense ranking's pairs above the list, with
        // room for 2 kWave words per wavefront once N >= kDenseRem.
        int st = stage2_bucket(ks, bimp, bsel, N, N - K1, sp, area, area + kBuckets, idx, idx + N,
                               ki + (N + 1) / 2, slots + 6 * kW, slots + 7 * kW, slots + 2 * kW,
                               slots + 3 * kW, split ? part : 0, split ? G : 1, gpick, s2_range,
                               L.has_comp ? reinterpret_cast<uint64_t*>(smem + L.comp) : nullptr);
        if (st == kS2Failed) {
            if (part > 0) return;   // the same decision in every group: group 0 sorts
            __syncthreads();        // every thread is past the bucket attempt
            stage2_radix(ks, bimp, bsel, N, K1, sp, ksd.VS, idx, idx + N,
                         reinterpret_cast<uint16_t*>(area), slots + 4 * kW, slots + 5 * kW);
            st = kS2Local;
        }
        if (split) {
            // The output of a shared image is written by emit_kernel after this
            // launch: group 0 publishes X^imp (and picks it made alone).
            if (part == 0) {
                __syncthreads();
                for (int i = threadIdx.x; i < (N + 31) / 32; i += kThreads) {
                    a.gimp[wbase + i] = bimp[i];
                    if (st == kS2Local) {
                        const uint32_t extra = bsel[i] & ~bimp[i];
                        if (extra) atomicOr(&gpick[i], extra);
                    }
                }
            }
            return;
        }
    }
    __syncthreads();
    emit(a, d, bimp, bsel, slots + 6 * kW);
}

// Output of the images select_kernel shared between workgroups: X^imp and the
// picks from the global bitmaps (which are cleared for the next call), then
// the ordered output.  One workgroup per image of the launch.
__global__ __launch_bounds__(kThreads) void emit_kernel(SelectArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int G = a.groups > 0 ? a.groups : 1;
    const int local = (int)blockIdx.x;
    const int img = a.img0 + local;
    const Img d = image_of(a, local);
    const int N = d.n, K1 = d.k1, K2 = d.k2;
    if (!(G > 1 && K2 > 0 && N - K1 >= kDenseRem)) return;   // emitted by select_kernel
    const int nw = 2 * ((N + 63) / 64);
    uint32_t* bimp = reinterpret_cast<uint32_t*>(smem);
    uint32_t* bsel = bimp + nw;
    uint32_t* slots = bsel + nw;
    const size_t wbase = (size_t)(d.row_off >> 5) + 2 * (size_t)img;
    for (int i = threadIdx.x; i < (N + 31) / 32; i += kThreads) {
        const uint32_t im = a.gimp[wbase + i];
        bimp[i] = im;
        bsel[i] = im | a.gsel[wbase + i];
        a.gsel[wbase + i] = 0u;
    }
    __syncthreads();
    emit(a, d, bimp, bsel, slots);
}

// ---- images of at most kSmallSelectN tokens: one token per thread ------------
//
// Both stages are ranked in the same passes.  Every token gets its exact rank
// in (Stage II key, index) order among all N tokens, and its place relative
// to K1 in (Stage I key, index) order (counted exactly only inside the bucket
// that holds the K1 boundary); X^imp is the places below K1, and a token of X^rem ranks in X^rem as
// its Stage II rank minus the X^imp tokens ranked below it (read from a
// bitmap of X^imp in Stage II rank order), which decides the stride picks.
// Ranks come from value buckets and exact counting inside a bucket: bucket =
// clamp(floor((v - lo) nb / (hi - lo)), 0, nb - 1) is non-decreasing in the
// key, so rank = (tokens in lower buckets) + (members of the token's bucket
// smaller in (key, index) order).  lo and hi are about the 1.5 % and 98.5 %
// quantiles of a 64-key sample, so outliers (all-zero rows, zero-norm states)
// land in the two end buckets instead of crowding the bulk into a few; when
// the sample's range is not a finite positive float width, buckets are equal
// ranges of the order-preserving key itself.  All keys equal: rank = index.
// Phases are separated by eight workgroup barriers.  With a fused gather, G
// workgroups share an image: each repeats the selection and copies every G-th
// share of the kept rows (group 0 writes out_idx / out_src / out_rows).

struct SmallLayout {
    size_t hi, hs, si, ss, li, ls, samp, slots, misc, imps, kept, total;
};

__host__ __device__ inline SmallLayout small_layout(int T)
{
    SmallLayout L;
    size_t o = 0;
    L.hi = o;  o += 4 * (size_t)T;            // Stage I histogram, then cursors
    L.hs = o;  o += 4 * (size_t)T;            // Stage II histogram, then cursors
    L.si = o;  o += 4 * ((size_t)T + 1);      // Stage I bucket starts
    L.ss = o;  o += 4 * ((size_t)T + 1);      // Stage II bucket starts
    o = align_up(o, 16);
    L.li = o;  o += 8 * (size_t)T;            // (key << 32 | index) in Stage I bucket order
    L.ls = o;  o += 8 * (size_t)T;            // the same for Stage II
    L.samp = o; o += 8 * 128;                 // 64-key samples of both keys, (key << 6 | k)
    L.slots = o; o += 4 * 8 * kW;             // per-wavefront partial values
    L.misc = o; o += 4 * 16;                  // broadcast slots
    L.imps = o; o += 4 * 32;                  // X^imp bitmap in Stage II rank order
    L.kept = o; o += 4 * (size_t)T;           // token of each output slot (fused gather)
    L.total = o;
    return L;
}

// Bucketing of one key over [lo, hi] (order keys) into nb buckets.
struct Bucketing {
    int32_t mode;      // 0: value buckets; 1: order-key buckets; 2: every key equal
    float fmin, scale;
    uint32_t kmin;
    int32_t shift;
};

// kmin / kmax: the true range of the keys (order keys); value buckets need
// every key to be a number (NaN keys lie outside [-inf, +inf] in key order).
__device__ __forceinline__ Bucketing make_bucketing(uint32_t lo, uint32_t hi, uint32_t kmin, uint32_t kmax, int nb)
{
    Bucketing b;
    b.mode = 2;
    b.kmin = lo;
    b.fmin = key_value(lo);
    b.scale = 0.f;
    b.shift = 0;
    if (kmin == kmax) return b;
    const bool no_nan = kmin >= 0x007fffffu && kmax <= 0xff800000u;
    const float width = key_value(hi) - b.fmin;
    const float scale = (float)nb / width;
    if (no_nan && width > 0.f && width < 3.0e38f && scale < 3.0e38f) {
        b.mode = 0;
        b.scale = scale;
        return b;
    }
    b.mode = 1;
    const uint32_t span = hi - lo;
    int sh = 0;
    while (sh < 31 && (span >> sh) >= (uint32_t)nb) ++sh;
    b.shift = sh;
    return b;
}

// Non-decreasing in the key; always in [0, nb).
__device__ __forceinline__ int bucket_of(const Bucketing& b, uint32_t k, int nb)
{
    if (b.mode == 0) {
        const float x = (key_value(k) - b.fmin) * b.scale;   // NaN only if a key is NaN (then mode 1)
        return x <= 0.f ? 0 : (x >= (float)(nb - 1) ? nb - 1 : (int)x);
    }
    if (b.mode == 1) {
        if (k <= b.kmin) return 0;
        const uint32_t q = (k - b.kmin) >> b.shift;
        return q >= (uint32_t)nb ? nb - 1 : (int)q;
    }
    return 0;
}

// About the 1.5 % and 98.5 % quantiles of 64 sampled keys of an image (all
// of them for N <= 64), computed by one wavefront without the workgroup:
// lane k loads sample k (token floor(k N / 64)), the wave stages the samples
// as distinct (key << 6 | k) values in its own LDS row, every lane ranks its
// sample among the 64 (two per 16-byte broadcast read), and the lanes holding
// ranks lo_rank and hi_rank publish their keys in out[0], out[1].
__device__ __forceinline__ void sample_quantiles(const float* keys, int N, int lane, uint64_t* samp,
                                                 uint32_t* out)
{
    const int st = N > kWave ? (int)(((int64_t)lane * N) >> 6) : lane;
    const uint64_t mine = ((uint64_t)(st < N ? order_key(keys[st]) : 0xffffffffu) << 6) | (uint64_t)lane;
    samp[lane] = mine;
    // LDS operations of one wavefront complete in order: the row written
    // above is visible to the reads below
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const ulonglong2* sv = reinterpret_cast<const ulonglong2*>(samp);
    int r = 0;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        ulonglong2 q[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) q[j] = sv[16 * h + j];
#pragma unroll
        for (int j = 0; j < 16; ++j) r += (q[j].x < mine ? 1 : 0) + (q[j].y < mine ? 1 : 0);
    }
    const int lo_rank = N > kWave ? 1 : 0, hi_rank = N > kWave ? kWave - 2 : N - 1;
    if (r == lo_rank) out[0] = (uint32_t)(mine >> 6);
    if (r == hi_rank) out[1] = (uint32_t)(mine >> 6);
}

// Exact rank of `me` = (key << 32 | index) among the n > 1 members
// list[beg, beg + n) of its bucket, plus beg (the tokens of lower buckets).
__device__ __forceinline__ uint32_t rank_in(const uint64_t* list, uint32_t beg, uint32_t n, uint64_t me)
{
    const uint32_t end = beg + n;
    uint32_t r = beg, j = beg;
    for (; j + 4 <= end; j += 4) {
        const uint64_t m0 = list[j], m1 = list[j + 1], m2 = list[j + 2], m3 = list[j + 3];
        r += (m0 < me) + (m1 < me) + (m2 < me) + (m3 < me);
    }
    for (; j < end; ++j) r += list[j] < me ? 1u : 0u;
    return r;
}

typedef uint32_t u32x4s __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(kSmallSelectN) void select_small_kernel(SelectArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int T = (int)blockDim.x, nb = T, nw = T / kWave;
    const int G = a.ggroups > 0 ? a.ggroups : 1;
    const int local = (int)blockIdx.x / G, part = (int)blockIdx.x % G;
    const Img d = image_of(a, local);
    const int N = d.n, K1 = d.k1, K2 = d.k2, K = K1 + K2;
    const int tid = (int)threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
    const bool valid = tid < N;
    const SmallLayout L = small_layout(T);
    uint32_t* Hi = reinterpret_cast<uint32_t*>(smem + L.hi);
    uint32_t* Hs = reinterpret_cast<uint32_t*>(smem + L.hs);
    uint32_t* Si = reinterpret_cast<uint32_t*>(smem + L.si);
    uint32_t* Ss = reinterpret_cast<uint32_t*>(smem + L.ss);
    uint64_t* Li = reinterpret_cast<uint64_t*>(smem + L.li);
    uint64_t* Ls = reinterpret_cast<uint64_t*>(smem + L.ls);
    uint64_t* samp = reinterpret_cast<uint64_t*>(smem + L.samp);
    uint32_t* slots = reinterpret_cast<uint32_t*>(smem + L.slots);
    uint32_t* misc = reinterpret_cast<uint32_t*>(smem + L.misc);
    uint32_t* imps = reinterpret_cast<uint32_t*>(smem + L.imps);
    uint32_t* kept = reinterpret_cast<uint32_t*>(smem + L.kept);

    // ---- keys, samples, per-wavefront ranges ----------------------------------
    uint32_t ki = 0, ks = 0;
    if (valid) {
        ki = order_key(a.key_imp[d.row_off + tid]);
        ks = order_key(a.key_s[d.row_off + tid]);
    }
    // the quantiles of both keys, by wavefronts 0 and 1 (0 alone for N <= 64)
    if (w == 0) sample_quantiles(a.key_imp + d.row_off, N, lane, samp, &misc[0]);
    if (w == (nw > 1 ? 1 : 0)) sample_quantiles(a.key_s + d.row_off, N, lane, samp + kWave, &misc[2]);
    Hi[tid] = 0u;
    Hs[tid] = 0u;
    kept[tid] = 0xffffffffu;
    if (tid < 32) imps[tid] = 0u;
    {
        const uint32_t nlo_i = wave_max_u32(valid ? ~ki : 0u), hi_i = wave_max_u32(valid ? ki : 0u);
        const uint32_t nlo_s = wave_max_u32(valid ? ~ks : 0u), hi_s = wave_max_u32(valid ? ks : 0u);
        if (lane == 0) {
            slots[w] = nlo_i;
            slots[kW + w] = hi_i;
            slots[2 * kW + w] = nlo_s;
            slots[3 * kW + w] = hi_s;
        }
    }
    __syncthreads();   // B1
    auto max_of = [&](const uint32_t* row) { return wave_max_u32(lane < nw ? row[lane] : 0u); };
    const uint32_t kimin = ~max_of(slots), kimax = max_of(slots + kW);
    const uint32_t ksmin = ~max_of(slots + 2 * kW), ksmax = max_of(slots + 3 * kW);
    // Buckets over the sample quantiles (outliers clamp into the end buckets);
    // the histogram's atomic returns each token's place within its bucket.
    const Bucketing bi = make_bucketing(misc[0], misc[1], kimin, kimax, nb);
    const Bucketing bs = make_bucketing(misc[2], misc[3], ksmin, ksmax, nb);
    const int gi = valid ? bucket_of(bi, ki, nb) : 0;
    const int gs = valid ? bucket_of(bs, ks, nb) : 0;
    uint32_t li = 0, ls = 0;
    if (valid) {
        li = atomicAdd(&Hi[gi], 1u);
        ls = atomicAdd(&Hs[gs], 1u);
    }
    __syncthreads();   // B2
    // ---- bucket starts: thread t owns bucket t ----------------------------------
    const uint32_t ci = Hi[tid], cs = Hs[tid];
    const uint32_t inc_i = wave_scan_add(ci), inc_s = wave_scan_add(cs);
    if (lane == kWave - 1) {
        slots[4 * kW + w] = inc_i;
        slots[5 * kW + w] = inc_s;
    }
    __syncthreads();   // B3
    Si[tid] = inc_i - ci + sum_before(slots + 4 * kW, w, lane);
    Ss[tid] = inc_s - cs + sum_before(slots + 5 * kW, w, lane);
    if (tid == T - 1) {
        Si[T] = (uint32_t)N;
        Ss[T] = (uint32_t)N;
    }
    __syncthreads();   // B4
    // ---- members of shared buckets listed; exact ranks ------------------------
    const uint64_t me_i = ((uint64_t)ki << 32) | (uint32_t)tid;
    const uint64_t me_s = ((uint64_t)ks << 32) | (uint32_t)tid;
    uint32_t bi0 = 0, bi1 = 0, bs0 = 0, bs1 = 0;
    if (valid) {
        bi0 = Si[gi];
        bi1 = Si[gi + 1];
        bs0 = Ss[gs];
        bs1 = Ss[gs + 1];
        // Stage I needs exact ranks only in the bucket that holds the K1
        // boundary: a lower bucket's members are all in X^imp, a higher
        // one's all out, whatever their order inside it.
        if (bi1 - bi0 > 1u && bi0 < (uint32_t)K1 && bi1 > (uint32_t)K1) Li[bi0 + li] = me_i;
        if (bs1 - bs0 > 1u) Ls[bs0 + ls] = me_s;
    }
    __syncthreads();   // B5
    uint32_t ri = bi0, rs = bs0;
    if (valid) {
        if (bi.mode == 2) ri = (uint32_t)tid;
        else if (bi1 - bi0 > 1u && bi0 < (uint32_t)K1 && bi1 > (uint32_t)K1) ri = rank_in(Li, bi0, bi1 - bi0, me_i);
        if (bs.mode == 2) rs = (uint32_t)tid;
        else if (bs1 - bs0 > 1u) rs = rank_in(Ls, bs0, bs1 - bs0, me_s);
        rs = rs < (uint32_t)N ? rs : (uint32_t)N - 1u;   // a rank below N in every case (memory safety)
    }
    const bool imp = valid && ri < (uint32_t)K1;
    if (imp && K2 > 0) atomicOr(&imps[rs >> 5], 1u << (rs & 31));
    __syncthreads();   // B6
    // ---- stride picks on the rank in X^rem, union, output slots -------------------
    // X^imp tokens ranked below rs: a wave scan of the bitmap words' counts
    // (lane q holds word q), then the partial word.
    const uint32_t wc = lane < 32 ? (uint32_t)__popc(imps[lane]) : 0u;
    const uint32_t wex = wave_scan_add(wc) - wc;
    const uint32_t wbelow = (uint32_t)__shfl((int)wex, (int)(rs >> 5));   // every lane takes part
    bool pick = false;
    if (valid && !imp && K2 > 0) {
        const uint32_t below = wbelow + (uint32_t)__popc(imps[rs >> 5] & ((1u << (rs & 31)) - 1u));
        const Stride sp{(uint32_t)d.t, (uint32_t)(N - K1), (uint32_t)K2, a.stride_real != 0};
        pick = sp.picks(rs - below);
    }
    const bool sel = imp || pick;
    const uint64_t bm = __ballot(sel);
    if (lane == 0) slots[6 * kW + w] = (uint32_t)__popcll(bm);
    __syncthreads();   // B7
    const uint32_t slot = sum_before(slots + 6 * kW, w, lane) + (uint32_t)__popcll(bm & lanes_below(lane));
    if (sel && slot < (uint32_t)K) {   // never more than K writes, whatever the keys
        if (part == 0) {
            const int o = d.out_off + (int)slot;
            a.out_idx[o] = tid;
            if (a.out_src) a.out_src[o] = imp ? 0 : 1;
            if (a.out_rows) a.out_rows[o] = d.row_off + tid;
        }
        kept[slot] = (uint32_t)tid;
    }
    if (!a.gX) return;
    __syncthreads();   // B8
    // ---- fused gather: this group's share of the kept rows -------------------------
    const int s0 = (int)(((int64_t)part * K) / G), s1 = (int)(((int64_t)(part + 1) * K) / G);
    const char* X = static_cast<const char*>(a.gX);
    char* out = static_cast<char*>(a.gout);
    const int64_t rb = a.grow_bytes;
    if (a.gvec) {
        // Chunk j = r * cpr + c of the share, walked with (r, c) carried
        // from step to step (no division per chunk).
        const uint32_t cpr = (uint32_t)(rb / 16);
        const uint32_t rows = (uint32_t)(s1 - s0);
        const uint32_t qT = (uint32_t)T / cpr, mT = (uint32_t)T % cpr;
        uint32_t r = (uint32_t)tid / cpr, c = (uint32_t)tid % cpr;
        constexpr int kUnr = 8;
        while (r < rows) {
            u32x4s v[kUnr];
            uint32_t rr[kUnr], cc[kUnr];
#pragma unroll
            for (int u = 0; u < kUnr; ++u) {
                rr[u] = r;
                cc[u] = c;
                if (r < rows) {
                    const uint32_t k = kept[s0 + (int)r];
                    const uint32_t tk = k < (uint32_t)N ? k : 0u;   // always a filled slot
                    v[u] = __builtin_nontemporal_load(
                        reinterpret_cast<const u32x4s*>(X + (int64_t)(d.row_off + (int)tk) * rb) + c);
                }
                c += mT;
                r += qT;
                if (c >= cpr) {
                    c -= cpr;
                    ++r;
                }
            }
#pragma unroll
            for (int u = 0; u < kUnr; ++u) {
                if (rr[u] < rows)
                    __builtin_nontemporal_store(
                        v[u], reinterpret_cast<u32x4s*>(out + (int64_t)(d.out_off + s0 + (int)rr[u]) * rb) + cc[u]);
            }
        }
    } else if (a.gelem == 2) {
        const int64_t epr = rb / 2;
        for (int r = s0; r < s1; ++r) {
            const uint32_t tk = kept[r] < (uint32_t)N ? kept[r] : 0u;
            const uint16_t* src = reinterpret_cast<const uint16_t*>(X + (int64_t)(d.row_off + (int)tk) * rb);
            uint16_t* dst = reinterpret_cast<uint16_t*>(out + (int64_t)(d.out_off + r) * rb);
            for (int64_t c = tid; c < epr; c += T) dst[c] = src[c];
        }
    } else {
        const int64_t epr = rb / 4;
        for (int r = s0; r < s1; ++r) {
            const uint32_t tk = kept[r] < (uint32_t)N ? kept[r] : 0u;
            const uint32_t* src = reinterpret_cast<const uint32_t*>(X + (int64_t)(d.row_off + (int)tk) * rb);
            uint32_t* dst = reinterpret_cast<uint32_t*>(out + (int64_t)(d.out_off + r) * rb);
            for (int64_t c = tid; c < epr; c += T) dst[c] = src[c];
        }
    }
}

}  // namespace

int select_threads(int nmax)
{
    (void)nmax;
    return kThreads;
}

bool select_shares(const ImageDesc& d)
{
    return d.k2 > 0 && d.n - d.k1 >= kDenseRem;
}

int select_groups(int64_t n_large, int cus)
{
    if (n_large <= 0) return 1;
    int g = 1;
    while (g < kMaxSplitGroups && n_large * 2 * g <= (int64_t)cus) g *= 2;
    return g;
}

size_t select_gsel_words(int64_t max_tokens, int max_images)
{
    return (size_t)(max_tokens / 32) + 2 * (size_t)max_images + 2;
}

size_t select_lds_bytes(int n, int threads)
{
    (void)threads;
    return launch_lds(n);
}

hipError_t select_prepare(int lds_limit)
{
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&select_kernel),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, lds_limit);
    if (e != hipSuccess) return e;
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(&select_small_kernel),
                            hipFuncAttributeMaxDynamicSharedMemorySize, lds_limit);
    if (e != hipSuccess) return e;
    return hipFuncSetAttribute(reinterpret_cast<const void*>(&emit_kernel),
                               hipFuncAttributeMaxDynamicSharedMemorySize, lds_limit);
}

int select_small_groups(int images, int k_min, int cus)
{
    // enough workgroups to keep every compute unit copying, at most one per
    // kept row and 16 per image
    int g = (2 * cus + images - 1) / (images > 0 ? images : 1);
    if (g > 16) g = 16;
    if (g > k_min) g = k_min;
    return g < 1 ? 1 : g;
}

hipError_t launch_select(const SelectArgs& a, int nmax, hipStream_t s)
{
    if (a.nimg <= 0) return hipSuccess;
    if (nmax <= kSmallSelectN) {
        const int T = ((nmax > kWave ? nmax : kWave) + kWave - 1) / kWave * kWave;
        const int G = a.gX && a.ggroups > 0 ? a.ggroups : 1;
        SelectArgs b = a;
        b.ggroups = G;
        hipLaunchKernelGGL(select_small_kernel, dim3(a.nimg * G), dim3(T), small_layout(T).total, s, b);
        return hipGetLastError();
    }
    const size_t lds = launch_lds(nmax);
    const int groups = a.groups > 0 ? a.groups : 1;
    hipLaunchKernelGGL(select_kernel, dim3(a.nimg * groups), dim3(kThreads), lds, s, a);
    if (groups > 1) {
        const size_t elds = 8 * (2 * (((size_t)nmax + 63) / 64)) + 4 * 8 * kW;
        hipLaunchKernelGGL(emit_kernel, dim3(a.nimg), dim3(kThreads), elds, s, a);
    }
    return hipGetLastError();
}

}  // namespace tr
