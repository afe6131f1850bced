// Buffer-resource loads and wave reductions for gfx950 (wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kla {

typedef __amdgpu_buffer_rsrc_t rsrc_t;

// Raw (unswizzled, stride 0) buffer over [base, base + bytes).  A load whose
// per-lane offset lies past the end returns zero instead of touching memory.
// The last word selects a 32-bit data format, which untyped loads require.
__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ uint16_t buf_ld16(rsrc_t r, uint32_t voff, uint32_t soff) {
    return __builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, 0);
}

__device__ __forceinline__ uint4 buf_ld128(rsrc_t r, uint32_t voff, uint32_t soff) {
    typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;
    const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
    return uint4{v[0], v[1], v[2], v[3]};
}

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, ROW_MASK,
                                                                 0xf, false));
}

// Sum over the 64 lanes of a wave with DPP moves (no LDS traffic); the total is
// returned in every lane through lane 63.
__device__ __forceinline__ float wave_sum(float x) {
    x += dpp<0xB1, 0xf>(x);    // quad_perm [1,0,3,2]
    x += dpp<0x4E, 0xf>(x);    // quad_perm [2,3,0,1]
    x += dpp<0x141, 0xf>(x);   // row_half_mirror
    x += dpp<0x140, 0xf>(x);   // row_mirror: every lane of a row holds the row sum
    x += dpp<0x142, 0xa>(x);   // row_bcast:15 into rows 1 and 3
    x += dpp<0x143, 0xc>(x);   // row_bcast:31 into rows 2 and 3
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 63));
}

}  // namespace kla
