// Gather of the kept rows: out[r, :] = X[rows[r], :], byte for byte.
// With 16-byte aligned rows every lane moves UNR x 16 bytes per step.  Rows
// of at most 8 KiB (one step) go two to a wavefront, the second row's loads
// in flight while the first is stored (64 x 576 x 4096 bf16 step: 150.4 ->
// 148.8 us; four rows to a wavefront: 151.6 us); longer rows take one
// wavefront each, all loads of a step issued before its stores.  Loads and
// stores are non-temporal: nothing is reused (non-temporal stores measured
// 8.6 vs 11.2 us for 4096 rows of 8 KiB).
#include "tr_internal.h"

namespace tr {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <int UNR>
__global__ __launch_bounds__(256) void gather_vec_kernel(const u32x4* __restrict__ X,
                                                          u32x4* __restrict__ out,
                                                          const int32_t* __restrict__ rows,
                                                          int64_t nout, int64_t nrows, int64_t vec_per_row)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t r = (int64_t)blockIdx.x * (blockDim.x / kWave) + (threadIdx.x / kWave);
    if (r >= nout) return;
    if (rows[r] < 0 || rows[r] >= nrows) return;   // memory safety against a bad index
    const u32x4* s = X + (int64_t)rows[r] * vec_per_row;
    u32x4* d = out + r * vec_per_row;
    for (int64_t j0 = lane; j0 < vec_per_row; j0 += (int64_t)kWave * UNR) {
        u32x4 v[UNR];
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            const int64_t j = j0 + (int64_t)kWave * u;
            if (j < vec_per_row) v[u] = __builtin_nontemporal_load(s + j);
        }
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            const int64_t j = j0 + (int64_t)kWave * u;
            if (j < vec_per_row) __builtin_nontemporal_store(v[u], d + j);
        }
    }
}

// Rows of at most 64 x UNR chunks, RPW consecutive output rows per
// wavefront: the loads of row k + 1 are in flight while row k is stored.
template <int UNR, int RPW>
__global__ __launch_bounds__(256) void gather_pipe_kernel(const u32x4* __restrict__ X,
                                                           u32x4* __restrict__ out,
                                                           const int32_t* __restrict__ rows,
                                                           int64_t nout, int64_t nrows, int64_t vec_per_row)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t r0 = ((int64_t)blockIdx.x * (blockDim.x / kWave) + (threadIdx.x / kWave)) * RPW;
    if (r0 >= nout) return;
    u32x4 v[2][UNR];
    auto load = [&](int b, int64_t r) {
        const int32_t src = rows[r];
        const bool ok = src >= 0 && src < nrows;   // memory safety against a bad index
        const u32x4* s = X + (int64_t)(ok ? src : 0) * vec_per_row;
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            const int64_t j = lane + (int64_t)kWave * u;
            if (ok && j < vec_per_row) v[b][u] = __builtin_nontemporal_load(s + j);
        }
    };
    auto store = [&](int b, int64_t r) {
        const int32_t src = rows[r];
        if (src < 0 || src >= nrows) return;
        u32x4* d = out + r * vec_per_row;
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            const int64_t j = lane + (int64_t)kWave * u;
            if (j < vec_per_row) __builtin_nontemporal_store(v[b][u], d + j);
        }
    };
    load(0, r0);
#pragma unroll
    for (int k = 0; k < RPW; ++k) {
        const int64_t r = r0 + k;
        if (r >= nout) break;
        if (k + 1 < RPW && r + 1 < nout) load((k + 1) & 1, r + 1);
        store(k & 1, r);
    }
}

template <typename E>
__global__ __launch_bounds__(256) void gather_elem_kernel(const E* __restrict__ X, E* __restrict__ out,
                                                          const int32_t* __restrict__ rows,
                                                          int64_t nout, int64_t nrows, int64_t elems_per_row)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t r = (int64_t)blockIdx.x * (blockDim.x / kWave) + (threadIdx.x / kWave);
    if (r >= nout) return;
    if (rows[r] < 0 || rows[r] >= nrows) return;   // memory safety against a bad index
    const E* s = X + (int64_t)rows[r] * elems_per_row;
    E* d = out + r * elems_per_row;
    for (int64_t j = lane; j < elems_per_row; j += kWave) d[j] = s[j];
}

}  // namespace

hipError_t launch_gather(const void* X, void* out, const int32_t* rows, int64_t nout, int64_t nrows,
                         int64_t row_bytes, int elem_bytes, bool vec, hipStream_t s)
{
    if (nout <= 0) return hipSuccess;
    constexpr int kThreads = 256;
    const int64_t blocks = (nout + kThreads / kWave - 1) / (kThreads / kWave);
    constexpr int kUnr = 8, kRowsPerWave = 2;
    if (vec && row_bytes <= 16 * kWave * kUnr) {
        const int64_t waves = (nout + kRowsPerWave - 1) / kRowsPerWave;
        const int64_t pb = (waves + kThreads / kWave - 1) / (kThreads / kWave);
        hipLaunchKernelGGL((gather_pipe_kernel<kUnr, kRowsPerWave>), dim3((unsigned)pb), dim3(kThreads), 0, s,
                           static_cast<const u32x4*>(X), static_cast<u32x4*>(out), rows, nout, nrows,
                           row_bytes / 16);
    } else if (vec) {
        hipLaunchKernelGGL(gather_vec_kernel<kUnr>, dim3((unsigned)blocks), dim3(kThreads), 0, s,
                           static_cast<const u32x4*>(X), static_cast<u32x4*>(out), rows, nout,
                           nrows, row_bytes / 16);
    } else if (elem_bytes == 2) {
        hipLaunchKernelGGL(gather_elem_kernel<uint16_t>, dim3((unsigned)blocks), dim3(kThreads), 0, s,
                           static_cast<const uint16_t*>(X), static_cast<uint16_t*>(out), rows, nout,
                           nrows, row_bytes / 2);
    } else {
        hipLaunchKernelGGL(gather_elem_kernel<uint32_t>, dim3((unsigned)blocks), dim3(kThreads), 0, s,
                           static_cast<const uint32_t*>(X), static_cast<uint32_t*>(out), rows, nout,
                           nrows, row_bytes / 4);
    }
    return hipGetLastError();
}

}  // namespace tr
