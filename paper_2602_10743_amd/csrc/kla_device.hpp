// Device-side helpers shared by the KLA kernels (gfx950, wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kla {

// Storage type tags: the element types the ABI accepts for per-token tensors.
struct f32_t {};
struct bf16_t {};

template <typename S> struct storage;
template <> struct storage<f32_t> { using type = float; };
template <> struct storage<bf16_t> { using type = uint16_t; };

__device__ __forceinline__ float bf16_to_f32(uint16_t u) {
    return __uint_as_float(static_cast<uint32_t>(u) << 16);
}

typedef __attribute__((__vector_size__(2 * sizeof(float)))) float f32x2_t;
typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2_t;

// Two fp32 -> packed bf16 pair (x0 in the low half), round to nearest even;
// one v_cvt_pk_bf16_f32 on gfx950.
__device__ __forceinline__ uint32_t cvt_pk_bf16(float x0, float x1) {
    const f32x2_t v = {x0, x1};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

// fp32 -> bf16, round to nearest even.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    return static_cast<uint16_t>(cvt_pk_bf16(f, 0.f));
}

// Gates of the exactly discretised OU prior (Sec. 4.1, eq. discretisation) for
// mean reversion a > 0, diffusion scale p and step delta > 0, formed in fp64:
//   abar = exp(-a delta),  pbar = p^2 (1 - exp(-2 a delta)) / (2 a).
__device__ __forceinline__ void ou_gates(float a, float p, float delta, float& abar, float& pbar) {
    const double ad = (double)a * (double)delta;
    abar = (float)exp(-ad);
    pbar = (float)((double)p * (double)p * -expm1(-2.0 * ad) / (2.0 * (double)a));
}

// Same gates left in fp64 (the fp32-input paths carry their filter arithmetic in fp64).
__device__ __forceinline__ void ou_gates(float a, float p, float delta, double& abar, double& pbar) {
    const double ad = (double)a * (double)delta;
    abar = exp(-ad);
    pbar = (double)p * (double)p * -expm1(-2.0 * ad) / (2.0 * (double)a);
}

// Arithmetic type of the token-recurrent and per-channel kernels for a storage type:
// fp32 inputs are filtered in fp64, so that the rounding accumulated over long
// recursions and reverse sums stays far below the single rounding of the outputs;
// bf16 inputs in fp32.
template <typename S> struct acc { using type = float; };
template <> struct acc<f32_t> { using type = double; };

__device__ __forceinline__ float ld(const float* p, size_t i) { return p[i]; }
__device__ __forceinline__ double ld(const double* p, size_t i) { return p[i]; }
__device__ __forceinline__ float ld(const uint16_t* p, size_t i) { return bf16_to_f32(p[i]); }
__device__ __forceinline__ void st(float* p, size_t i, float x) { p[i] = x; }
__device__ __forceinline__ void st(uint16_t* p, size_t i, float x) { p[i] = f32_to_bf16(x); }
__device__ __forceinline__ void st(float* p, size_t i, double x) { p[i] = (float)x; }
__device__ __forceinline__ void st(uint16_t* p, size_t i, double x) { p[i] = f32_to_bf16((float)x); }

// Reciprocal in the arithmetic type: v_rcp_f32 (about 1 ulp) for fp32; for fp64
// v_rcp_f64 refined by one Newton step, r + r (1 - x r), which squares its relative
// error (within a few ulp of the correctly rounded 1 / x, for the positive normal
// arguments the filters take; the IEEE division sequence costs about four times as
// many instructions).
__device__ __forceinline__ float rcpa(float x) { return __builtin_amdgcn_rcpf(x); }
__device__ __forceinline__ double rcpa(double x) {
    const double r = __builtin_amdgcn_rcp(x);
    return fma(r, fma(-x, r, 1.0), r);
}

}  // namespace kla
