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

typedef __attribute__((address_space(3))) void lds_void_t;

// Direct loads into LDS: lane i's 16 bytes land at dst + 16 i (one wave fills
// 1 KiB contiguously); lanes whose offset lies past the buffer end write zeros.
// The write completes with the wave's vector-memory counter, not lgkmcnt.
__device__ __forceinline__ void buf_ld128_lds(rsrc_t r, void* dst, uint32_t voff) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void_t*)dst, 16, voff, 0, 0, 0);
}

// 2-byte variant: lane i's value lands zero-extended in the word at dst + 4 i.
__device__ __forceinline__ void buf_ld16_lds(rsrc_t r, void* dst, uint32_t voff) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void_t*)dst, 2, voff, 0, 0, 0);
}

// 4-byte variant: lane i's word lands at dst + 4 i.
__device__ __forceinline__ void buf_ld32_lds(rsrc_t r, void* dst, uint32_t voff) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void_t*)dst, 4, voff, 0, 0, 0);
}

// s_waitcnt vmcnt(N): at most N vector memory accesses of this wave are still
// outstanding (they complete in issue order).
template <int N>
__device__ __forceinline__ void wait_vm_le() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | 0x70 | 0xF00);
}

// vmcnt(BASE + extra) for a wave-uniform extra in [0, 8).
template <int BASE>
__device__ __forceinline__ void wait_vm_le_rt(int extra) {
    switch (extra) {
        case 0: wait_vm_le<BASE>(); break;
        case 1: wait_vm_le<BASE + 1>(); break;
        case 2: wait_vm_le<BASE + 2>(); break;
        case 3: wait_vm_le<BASE + 3>(); break;
        case 4: wait_vm_le<BASE + 4>(); break;
        case 5: wait_vm_le<BASE + 5>(); break;
        case 6: wait_vm_le<BASE + 6>(); break;
        default: wait_vm_le<BASE + 7>(); break;
    }
}

// s_waitcnt vmcnt(0): every vector memory access of this wave has completed.
// Placed after loads whose results are carried into a prefetching loop, so the
// loop body does not wait on them (and thereby on the prefetch) at first use.
__device__ __forceinline__ void wait_vm_all() { __builtin_amdgcn_s_waitcnt(0xF70); }

// Workgroup barrier that orders LDS only: waits for this wave's LDS accesses
// (lgkmcnt) but leaves vector-memory requests in flight, so direct-to-LDS
// prefetches and global stores may cross it.  Data those requests bring into
// LDS is waited for by its consumer through vmcnt.
__device__ __forceinline__ void barrier_lds() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, ROW_MASK,
                                                                 0xf, false));
}

// dpp<> on a double: the same move applied to both 32-bit halves.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ double dpp(double x) {
    const uint64_t u = __builtin_bit_cast(uint64_t, x);
    const int lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)u, CTRL, ROW_MASK, 0xf, false);
    const int hi = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(u >> 32), CTRL, ROW_MASK, 0xf, false);
    return __builtin_bit_cast(double, (uint64_t)(uint32_t)lo | ((uint64_t)(uint32_t)hi << 32));
}

// Sums over the 32 lanes of each half of a wave (lanes 0..31 and 32..63) with
// DPP moves; the total of a half lands in its upper 16 lanes (16..31, 48..63).
template <typename A>
__device__ __forceinline__ A half_sum(A x) {
    x += dpp<0xB1, 0xf>(x);    // quad_perm [1,0,3,2]
    x += dpp<0x4E, 0xf>(x);    // quad_perm [2,3,0,1]
    x += dpp<0x141, 0xf>(x);   // row_half_mirror
    x += dpp<0x140, 0xf>(x);   // row_mirror: every lane of a row holds the row sum
    x += dpp<0x142, 0xa>(x);   // row_bcast:15 into rows 1 and 3
    return x;
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
