// MFMA helpers for gfx950 (CDNA4, wave64).
//
// v_mfma_f32_16x16x32_bf16 lane layout (lane l, g = l / 16):
//   A (16 x 32): lane l holds row l % 16, columns 8g .. 8g+7
//   B (32 x 16): lane l holds rows 8g .. 8g+7 of column l % 16
//   C (16 x 16): lane l holds rows 4g .. 4g+3 of column l % 16
// Because the contraction index may be permuted freely as long as A and B use
// the same permutation, an accumulator pair of two 16-row tiles can feed the B
// operand directly: lane group g then carries rows {4g..4g+3} and
// {16+4g..16+4g+3}, and the A operand is read with the same two 4-wide groups.
//
// Split-bf16 products: an fp32 operand x is carried as hi = bf16(x) and
// lo = bf16(x - hi); x*y ~ hi_x*hi_y + hi_x*lo_y + lo_x*hi_y keeps about 16
// significant bits per product, with fp32 accumulation.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kla_device.hpp"

namespace kla {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;

__device__ __forceinline__ f32x4 mfma_bf16(const bf16x8& a, const bf16x8& b, const f32x4& c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// split-bf16 product accumulate: c += (ah + al) * (bh + bl), dropping al * bl
__device__ __forceinline__ f32x4 mfma3(const bf16x8& ah, const bf16x8& al, const bf16x8& bh, const bf16x8& bl,
                                       f32x4 c) {
    c = mfma_bf16(al, bh, c);
    c = mfma_bf16(ah, bl, c);
    return mfma_bf16(ah, bh, c);
}

// c += (ah + al) * b for an exact bf16 operand b
__device__ __forceinline__ f32x4 mfma2a(const bf16x8& ah, const bf16x8& al, const bf16x8& b, f32x4 c) {
    c = mfma_bf16(al, b, c);
    return mfma_bf16(ah, b, c);
}

// c += a * (bh + bl) for an exact bf16 operand a
__device__ __forceinline__ f32x4 mfma2b(const bf16x8& a, const bf16x8& bh, const bf16x8& bl, f32x4 c) {
    c = mfma_bf16(a, bl, c);
    return mfma_bf16(a, bh, c);
}

__device__ __forceinline__ f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }

// 16-byte LDS read of 8 bf16 (address must be 16-byte aligned)
__device__ __forceinline__ bf16x8 lds8(const uint16_t* p) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
}

// two 8-byte LDS reads of 4 bf16 each, concatenated
__device__ __forceinline__ bf16x8 lds4x2(const uint16_t* p0, const uint16_t* p1) {
    const uint2 a = *reinterpret_cast<const uint2*>(p0);
    const uint2 b = *reinterpret_cast<const uint2*>(p1);
    return __builtin_bit_cast(bf16x8, uint4{a.x, a.y, b.x, b.y});
}

__device__ __forceinline__ uint32_t pack2(uint16_t lo16, uint16_t hi16) {
    return static_cast<uint32_t>(lo16) | (static_cast<uint32_t>(hi16) << 16);
}

typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4;
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4_t;

// MFMA operand read across the rows of a row-major bf16 LDS array X (row
// stride ld halfwords) with ds_read_b64_tr_b16: lane l (s = l % 16) receives
//   X[rowA + j][col0 + s] for j = 0..3 and X[rowB + j][col0 + s] for j = 0..3.
// Within each group of 16 lanes the instruction hands lane i element i % 4 of
// the 8 bytes addressed by lane 4 j + i / 4, so lane s addresses row
// rowA + s / 4 (resp. rowB + s / 4) at column col0 + 4 (s % 4).  Rows and
// columns may differ between the lane groups (rowA, rowB are per lane).
// col0 and ld must be multiples of 4 (8-byte aligned addresses).
__device__ __forceinline__ bf16x8 lds_tr8(const uint16_t* X, int ld, int rowA, int rowB, int col0, int s) {
    const uint16_t* p0 = X + (rowA + (s >> 2)) * ld + col0 + 4 * (s & 3);
    const uint16_t* p1 = X + (rowB + (s >> 2)) * ld + col0 + 4 * (s & 3);
    const bf16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t*)p0);
    const bf16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t*)p1);
    return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}

// fp32 -> (hi, lo) bf16 pair
__device__ __forceinline__ void split(float x, uint16_t& hi, uint16_t& lo) {
    hi = f32_to_bf16(x);
    lo = f32_to_bf16(x - bf16_to_f32(hi));
}

// Two fp32 -> packed hi pair and packed lo pair (x0 in the low halves).
__device__ __forceinline__ void split2(float x0, float x1, uint32_t& hi, uint32_t& lo) {
    hi = cvt_pk_bf16(x0, x1);
    lo = cvt_pk_bf16(x0 - __uint_as_float(hi << 16), x1 - __uint_as_float(hi & 0xffff0000u));
}

// Eight fp32 values (two accumulator quads) -> split-bf16 operand pair.
__device__ __forceinline__ void split8(const f32x4& x0, const f32x4& x1, bf16x8& hi, bf16x8& lo) {
    uint32_t h[4], l[4];
    split2(x0[0], x0[1], h[0], l[0]);
    split2(x0[2], x0[3], h[1], l[1]);
    split2(x1[0], x1[1], h[2], l[2]);
    split2(x1[2], x1[3], h[3], l[3]);
    hi = __builtin_bit_cast(bf16x8, uint4{h[0], h[1], h[2], h[3]});
    lo = __builtin_bit_cast(bf16x8, uint4{l[0], l[1], l[2], l[3]});
}

__device__ __forceinline__ float fast_rcp(float x) { return __builtin_amdgcn_rcpf(x); }

}  // namespace kla
