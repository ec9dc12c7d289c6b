// Wavefront-level primitives for gfx950 (64 lanes): DPP scans and reductions.
//
// The scans use the GFX9 DPP pattern: row shifts by 1, 2, 4, 8 inside each
// row of 16 lanes, then row broadcasts of lane 15 and lane 31 into the later
// rows.  Lanes whose source falls outside the row read 0 (bound_ctrl), so the
// result is an exact inclusive prefix over the 64 lanes, always combined in
// the same order (deterministic for floats too).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tr {

__device__ __forceinline__ uint32_t dpp_u32(uint32_t x, int ctrl_sel)
{
    // The control must be a compile-time constant: dispatch on the few we use.
    switch (ctrl_sel) {
    case 1: return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xf, 0xf, true);
    case 2: return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xf, 0xf, true);
    case 4: return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xf, 0xf, true);
    case 8: return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xf, 0xf, true);
    case 15: return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xa, 0xf, false);
    default: return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xc, 0xf, false);
    }
}

// Inclusive prefix sum over the wavefront.
__device__ __forceinline__ uint32_t wave_scan_add(uint32_t x)
{
    x += dpp_u32(x, 1);
    x += dpp_u32(x, 2);
    x += dpp_u32(x, 4);
    x += dpp_u32(x, 8);
    x += dpp_u32(x, 15);
    x += dpp_u32(x, 31);
    return x;
}

// Inclusive prefix OR over the wavefront (lane 63 holds the OR of all lanes).
__device__ __forceinline__ uint32_t wave_scan_or(uint32_t x)
{
    x |= dpp_u32(x, 1);
    x |= dpp_u32(x, 2);
    x |= dpp_u32(x, 4);
    x |= dpp_u32(x, 8);
    x |= dpp_u32(x, 15);
    x |= dpp_u32(x, 31);
    return x;
}

__device__ __forceinline__ float dpp_f32(float x, int ctrl_sel)
{
    return __uint_as_float(dpp_u32(__float_as_uint(x), ctrl_sel));
}

// Sum over the wavefront, returned to every lane (lane 63's inclusive prefix,
// read back as a scalar).  The association order is fixed.
__device__ __forceinline__ float wave_sum_f32(float x)
{
    x += dpp_f32(x, 1);
    x += dpp_f32(x, 2);
    x += dpp_f32(x, 4);
    x += dpp_f32(x, 8);
    x += dpp_f32(x, 15);
    x += dpp_f32(x, 31);
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 63));
}

__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t x)
{
    return (uint32_t)__builtin_amdgcn_readlane((int)wave_scan_add(x), 63);
}

__device__ __forceinline__ uint32_t wave_or_u32(uint32_t x)
{
    return (uint32_t)__builtin_amdgcn_readlane((int)wave_scan_or(x), 63);
}

// Sum over each half of the wavefront: lane 31 ends with the sum of lanes
// 0-31 and lane 63 with the sum of lanes 32-63 (other lanes hold partial
// prefixes).  Row shifts inside each row of 16, then lane 15 of rows 0 and 2
// added into rows 1 and 3.
__device__ __forceinline__ float half_sum(float x)
{
    x += dpp_f32(x, 1);
    x += dpp_f32(x, 2);
    x += dpp_f32(x, 4);
    x += dpp_f32(x, 8);
    x += dpp_f32(x, 15);
    return x;
}

}  // namespace tr

namespace tr {

// Maximum over the wavefront (unsigned; 0 is the identity).
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x)
{
    x = max(x, dpp_u32(x, 1));
    x = max(x, dpp_u32(x, 2));
    x = max(x, dpp_u32(x, 4));
    x = max(x, dpp_u32(x, 8));
    x = max(x, dpp_u32(x, 15));
    x = max(x, dpp_u32(x, 31));
    return (uint32_t)__builtin_amdgcn_readlane((int)x, 63);
}

}  // namespace tr
