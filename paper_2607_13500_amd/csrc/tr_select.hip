// Per-image selection, one workgroup per image, everything resident in LDS.
//
//   Stage I  (top-K1 smallest Stage I key, ties to the lower index):
//            4-pass MSB-first radix select over order-preserving 32-bit keys
//            finds the K1-th smallest key T and how many keys equal to T are
//            taken; an ordered pass then marks keys < T and the first of the
//            keys == T in index order.
//   Stage II (X^rem in index order, stable ascending sort by s, stride):
//            ordered compaction of the unmarked tokens, 4-pass stable LSD radix
//            sort of their 16-bit indices keyed by s, picks at positions
//            0, t, ..., (K2-1) t.
//   Output:  ordered compaction of X^imp U X^div (ascending token index).
//
// Every wavefront owns a contiguous, 64-aligned range of the array it walks,
// and ranks within a 64-token tile with ballots, so all orders are exact and
// ties are broken by index, deterministically.
//
// LDS layout for an image of n tokens (W = threads / 64, nw = 2 ceil(n/64)):
//   ks    u32[n]      Stage II keys by token index
//   ki    u32[n]      Stage I keys by token index; after Stage I the same bytes
//                     hold two u16[n] index buffers for the sort
//   bimp  u32[nw]     X^imp bitmap
//   bsel  u32[nw]     X^imp U X^div bitmap
//   hist  u16[256 W]  per-wavefront digit counts / scatter offsets
//   scan  u32[W + 4]  workgroup scan scratch and broadcast slots
#include "tr_internal.h"

namespace tr {
namespace {

// IEEE order -> unsigned order; -0 and +0 map to the same key.
__device__ __forceinline__ uint32_t order_key(float f)
{
    const uint32_t u = __float_as_uint(f + 0.0f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ uint64_t lanes_below(int lane)
{
    return (1ull << lane) - 1ull;
}

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

// Exclusive prefix over the wavefronts of a per-wavefront count (every lane of
// a wavefront passes the same value).  Returns the count of earlier waves.
template <int W>
__device__ __forceinline__ uint32_t wave_prefix(uint32_t count, uint32_t* scan)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int w = threadIdx.x / kWave;
    if (lane == 0) scan[w] = count;
    __syncthreads();
    uint32_t base = 0;
    for (int i = 0; i < w; ++i) base += scan[i];
    __syncthreads();
    return base;
}

// Exclusive prefix of one value per thread over the whole workgroup.
template <int THREADS>
__device__ __forceinline__ uint32_t block_prefix(uint32_t v, uint32_t* scan)
{
    constexpr int W = THREADS / kWave;
    const int lane = threadIdx.x & (kWave - 1);
    const int w = threadIdx.x / kWave;
    uint32_t x = v;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const uint32_t y = __shfl_up(x, o, kWave);
        if (lane >= o) x += y;
    }
    if (lane == kWave - 1) scan[w] = x;
    __syncthreads();
    uint32_t base = 0;
    for (int i = 0; i < W && i < w; ++i) base += scan[i];
    __syncthreads();
    return base + x - v;
}

__device__ __forceinline__ bool bit_of(const uint32_t* bm, int i)
{
    return (bm[i >> 5] >> (i & 31)) & 1u;
}

// A wavefront writes the 64-bit ballot of tile `base` into two bitmap words.
__device__ __forceinline__ void put_tile_bits(uint32_t* bm, int base, uint64_t bits, int lane)
{
    if (lane == 0) bm[base >> 5] = (uint32_t)bits;
    if (lane == 32) bm[(base >> 5) + 1] = (uint32_t)(bits >> 32);
}

template <int THREADS>
__global__ __launch_bounds__(THREADS) void select_kernel(SelectArgs a)
{
    constexpr int W = THREADS / kWave;
    extern __shared__ __align__(16) unsigned char smem[];
    const int lane = threadIdx.x & (kWave - 1);
    const int w = threadIdx.x / kWave;

    ImageDesc d;
    if (a.uniform) {
        d = a.desc[0];
        const int img = a.img0 + (int)blockIdx.x;
        d.row_off = img * d.n;
        d.out_off = img * (d.k1 + d.k2);
    } else {
        d = a.desc[blockIdx.x];
    }
    const int N = d.n, K1 = d.k1, K2 = d.k2, t = d.t;
    const int nw = 2 * ((N + 63) / 64);

    uint32_t* ks = reinterpret_cast<uint32_t*>(smem);
    uint32_t* ki = ks + N;
    uint16_t* idx_a = reinterpret_cast<uint16_t*>(ki);
    uint16_t* idx_b = idx_a + N;
    uint32_t* bimp = ki + N;
    uint32_t* bsel = bimp + nw;
    uint16_t* hist = reinterpret_cast<uint16_t*>(bsel + nw);
    uint32_t* scan = reinterpret_cast<uint32_t*>(hist + 256 * W);

    // Wavefront ranges over the n tokens.
    const int segN = (((N + W - 1) / W) + 63) & ~63;
    const int begN = w * segN < N ? w * segN : N;
    const int endN = begN + segN < N ? begN + segN : N;

    // ---- load keys ---------------------------------------------------------
    for (int i = threadIdx.x; i < N; i += THREADS) {
        ks[i] = order_key(a.key_s[d.row_off + i]);
        ki[i] = order_key(a.key_imp[d.row_off + i]);
    }
    __syncthreads();

    // ---- Stage I: radix select of the K1-th smallest key --------------------
    uint32_t T = 0;
    uint32_t need = 0;   // keys equal to T that are taken, in index order
    if (K1 > 0 && K1 < N) {
        uint32_t prefix = 0, pmask = 0;
        need = (uint32_t)K1;
        for (int shift = 24; shift >= 0; shift -= 8) {
            for (int i = threadIdx.x; i < 256 * W; i += THREADS) hist[i] = 0;
            __syncthreads();
            for (int base = begN; base < endN; base += kWave) {
                const int i = base + lane;
                bool act = i < endN;
                const uint32_t key = act ? ki[i] : 0u;
                act = act && ((key & pmask) == prefix);
                const uint32_t dg = (key >> shift) & 255u;
                const uint64_t m = same_digit(dg, act);
                if (act && (int)(__ffsll((long long)m) - 1) == lane)
                    hist[dg * W + w] = (uint16_t)(hist[dg * W + w] + __popcll(m));
            }
            __syncthreads();
            if (w == 0) {
                uint32_t cnt[4], sum = 0;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    uint32_t c = 0;
                    for (int ww = 0; ww < W; ++ww) c += hist[(lane * 4 + q) * W + ww];
                    cnt[q] = c;
                    sum += c;
                }
                uint32_t x = sum;
#pragma unroll
                for (int o = 1; o < kWave; o <<= 1) {
                    const uint32_t y = __shfl_up(x, o, kWave);
                    if (lane >= o) x += y;
                }
                uint32_t run = x - sum;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    if (run < need && need <= run + cnt[q]) {
                        scan[W] = (uint32_t)(lane * 4 + q);
                        scan[W + 1] = need - run;
                    }
                    run += cnt[q];
                }
            }
            __syncthreads();
            const uint32_t dsel = scan[W];
            need = scan[W + 1];
            prefix |= dsel << shift;
            pmask |= 255u << shift;
            __syncthreads();
        }
        T = prefix;
    }

    // ---- Stage I: mark X^imp (keys < T, then the first `need` keys == T) ----
    if (K1 == 0 || K1 == N) {
        const uint32_t fill = K1 ? 0xffffffffu : 0u;
        for (int i = threadIdx.x; i < nw; i += THREADS) bimp[i] = fill;
    } else {
        uint32_t eq = 0;
        for (int base = begN; base < endN; base += kWave) {
            const int i = base + lane;
            eq += __popcll(__ballot(i < endN && ki[i] == T));
        }
        uint32_t rank = wave_prefix<W>(eq, scan);
        for (int base = begN; base < endN; base += kWave) {
            const int i = base + lane;
            const bool act = i < endN;
            const uint32_t key = act ? ki[i] : 0xffffffffu;
            const bool is_eq = act && key == T;
            const uint64_t be = __ballot(is_eq);
            const uint32_t r = rank + (uint32_t)__popcll(be & lanes_below(lane));
            const bool take = act && (key < T || (is_eq && r < need));
            put_tile_bits(bimp, base, __ballot(take), lane);
            rank += (uint32_t)__popcll(be);
        }
    }
    __syncthreads();   // ki is dead from here on; its bytes become idx_a / idx_b

    // ---- Stage II: X^rem in index order, stable radix sort by s, stride -----
    for (int i = threadIdx.x; i < nw; i += THREADS) bsel[i] = bimp[i];
    if (K2 > 0) {
        uint32_t rc = 0;
        for (int base = begN; base < endN; base += kWave) {
            const int i = base + lane;
            rc += __popcll(__ballot(i < endN && !bit_of(bimp, i)));
        }
        uint32_t pos = wave_prefix<W>(rc, scan);
        for (int base = begN; base < endN; base += kWave) {
            const int i = base + lane;
            const bool keep = i < endN && !bit_of(bimp, i);
            const uint64_t bk = __ballot(keep);
            if (keep) idx_a[pos + __popcll(bk & lanes_below(lane))] = (uint16_t)i;
            pos += (uint32_t)__popcll(bk);
        }
        __syncthreads();

        const int R = N - K1;
        const int segR = (((R + W - 1) / W) + 63) & ~63;
        const int begR = w * segR < R ? w * segR : R;
        const int endR = begR + segR < R ? begR + segR : R;
        uint16_t* src = idx_a;
        uint16_t* dst = idx_b;
        for (int shift = 0; shift < 32; shift += 8) {
            for (int i = threadIdx.x; i < 256 * W; i += THREADS) hist[i] = 0;
            __syncthreads();
            for (int base = begR; base < endR; base += kWave) {
                const int i = base + lane;
                const bool act = i < endR;
                const uint32_t id = act ? src[i] : 0u;
                const uint32_t dg = act ? (ks[id] >> shift) & 255u : 0u;
                const uint64_t m = same_digit(dg, act);
                if (act && (int)(__ffsll((long long)m) - 1) == lane)
                    hist[dg * W + w] = (uint16_t)(hist[dg * W + w] + __popcll(m));
            }
            __syncthreads();
            {   // exclusive scan of hist in (digit, wavefront) order, 4 entries per thread
                const int e = threadIdx.x * 4;
                const uint32_t h0 = hist[e], h1 = hist[e + 1], h2 = hist[e + 2], h3 = hist[e + 3];
                const uint32_t b0 = block_prefix<THREADS>(h0 + h1 + h2 + h3, scan);
                hist[e] = (uint16_t)b0;
                hist[e + 1] = (uint16_t)(b0 + h0);
                hist[e + 2] = (uint16_t)(b0 + h0 + h1);
                hist[e + 3] = (uint16_t)(b0 + h0 + h1 + h2);
            }
            __syncthreads();
            for (int base = begR; base < endR; base += kWave) {
                const int i = base + lane;
                const bool act = i < endR;
                const uint32_t id = act ? src[i] : 0u;
                const uint32_t dg = act ? (ks[id] >> shift) & 255u : 0u;
                const uint64_t m = same_digit(dg, act);
                const uint32_t off = act ? hist[dg * W + w] : 0u;
                if (act) dst[off + __popcll(m & lanes_below(lane))] = (uint16_t)id;
                if (act && (int)(__ffsll((long long)m) - 1) == lane)
                    hist[dg * W + w] = (uint16_t)(off + __popcll(m));
            }
            __syncthreads();
            uint16_t* tmp = src;
            src = dst;
            dst = tmp;
        }
        for (int j = threadIdx.x; j < K2; j += THREADS) {
            const int id = src[j * t];
            atomicOr(&bsel[id >> 5], 1u << (id & 31));
        }
    }
    __syncthreads();

    // ---- X* in ascending token index ---------------------------------------
    uint32_t oc = 0;
    for (int base = begN; base < endN; base += kWave) {
        const int i = base + lane;
        oc += __popcll(__ballot(i < endN && bit_of(bsel, i)));
    }
    uint32_t opos = wave_prefix<W>(oc, scan);
    for (int base = begN; base < endN; base += kWave) {
        const int i = base + lane;
        const bool kept = i < endN && bit_of(bsel, i);
        const uint64_t bk = __ballot(kept);
        const int slot = (int)opos + __popcll(bk & lanes_below(lane));
        if (kept && slot < K1 + K2) {   // never more than K writes, whatever the keys
            const int o = d.out_off + slot;
            a.out_idx[o] = i;
            if (a.out_src) a.out_src[o] = bit_of(bimp, i) ? 0 : 1;
            if (a.out_rows) a.out_rows[o] = d.row_off + i;
        }
        opos += (uint32_t)__popcll(bk);
    }
}

}  // namespace

int select_threads(int nmax)
{
    return nmax > 4096 ? 1024 : 256;
}

size_t select_lds_bytes(int n, int threads)
{
    const size_t W = (size_t)threads / kWave;
    const size_t nw = 2 * (((size_t)n + 63) / 64);
    return 8 * (size_t)n + 8 * nw + 512 * W + 4 * (W + 4);
}

hipError_t select_prepare(int lds_limit)
{
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&select_kernel<1024>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, lds_limit);
    if (e != hipSuccess) return e;
    return hipFuncSetAttribute(reinterpret_cast<const void*>(&select_kernel<256>),
                               hipFuncAttributeMaxDynamicSharedMemorySize, lds_limit);
}

hipError_t launch_select(const SelectArgs& a, int nmax, hipStream_t s)
{
    if (a.nimg <= 0) return hipSuccess;
    const int threads = select_threads(nmax);
    const size_t lds = select_lds_bytes(nmax, threads);
    if (threads == 1024)
        hipLaunchKernelGGL(select_kernel<1024>, dim3(a.nimg), dim3(1024), lds, s, a);
    else
        hipLaunchKernelGGL(select_kernel<256>, dim3(a.nimg), dim3(256), lds, s, a);
    return hipGetLastError();
}

}  // namespace tr
