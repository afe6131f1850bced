// Monte Carlo readout of KLA+ (the log-marginal-likelihood training loss of the
// paper's appendix, eqs. nmll_integral and nmll_logsumexp):
//
//   draws   y^(s)[b,t,h,d] = ymu[b,t,h,d] + sqrt(yvar[b,t,h]) eps[s,b,t,h,d]
//   loss    nll[i] = -logsumexp_s(logp[s,i]) + log S
//
// with eps from the counter-based generator Philox4x64-10 (Salmon et al., SC 2011)
// and the Box-Muller transform: for the flat index e of [S, B, T, H, dv], block
// j = e / 8 is Philox's output for counter (j, 0, 0, 0) and key (seed, 0); its four
// 64-bit words give eight 32-bit halves u_0..u_7 (low half first), and each pair
// (u_2p, u_2p+1) the normals r cos(pi a), r sin(pi a) with
// r = sqrt(-2 ln(((u_2p >> 8) + 1) 2^-24)), a = (u_2p+1 >> 8) 2^-23.  Nothing is
// stored: the backward draws eps again from the counter.
//
// Every dv is a multiple of 8, so a thread's 8 consecutive channels of one row are
// one Philox block per sample: it loads the row's ymu and yvar once, then per
// sample draws the block and stores 8 outputs (16-byte accesses in bf16).
#include <hip/hip_runtime.h>

#include "kla_device.hpp"
#include "kla_internal.hpp"

namespace kla {
namespace {

constexpr uint64_t kM0 = 0xD2E7470EE14C6C93ull, kM1 = 0xCA5A826395121157ull;   // round multipliers
constexpr uint64_t kW0 = 0x9E3779B97F4A7C15ull, kW1 = 0xBB67AE8584CAA73Bull;   // key increments

// The 128-bit product m x (m a constant) as its high and low 64-bit halves, from four
// 32 x 32 -> 64 partial products (v_mad_u64_u32) shared by both halves.
template <uint64_t M>
__device__ __forceinline__ void mul128(uint64_t x, uint64_t& hi, uint64_t& lo) {
    constexpr uint32_t m0 = (uint32_t)M, m1 = (uint32_t)(M >> 32);
    const uint32_t x0 = (uint32_t)x, x1 = (uint32_t)(x >> 32);
    const uint64_t p00 = (uint64_t)m0 * x0;                           // bits 0..63
    const uint64_t p01 = (uint64_t)m0 * x1 + (p00 >> 32);             // bits 32..95, no overflow
    const uint64_t p10 = (uint64_t)m1 * x0 + (uint32_t)p01;           // bits 32..95, no overflow
    hi = (uint64_t)m1 * x1 + (p01 >> 32) + (p10 >> 32);
    lo = (p10 << 32) | (uint32_t)p00;
}

__device__ __forceinline__ void philox4x64_10(uint64_t c0, uint64_t key, uint64_t w[4]) {
    uint64_t x0 = c0, x1 = 0, x2 = 0, x3 = 0, k0 = key, k1 = 0;
#pragma unroll
    for (int i = 0; i < 10; ++i) {
        uint64_t hi0, lo0, hi1, lo1;
        mul128<kM0>(x0, hi0, lo0);
        mul128<kM1>(x2, hi1, lo1);
        const uint64_t y0 = hi1 ^ x1 ^ k0, y2 = hi0 ^ x3 ^ k1;
        x0 = y0;
        x1 = lo1;
        x2 = y2;
        x3 = lo0;
        k0 += kW0;
        k1 += kW1;
    }
    w[0] = x0;
    w[1] = x1;
    w[2] = x2;
    w[3] = x3;
}

// the 8 normals of Philox block j.  The transcendentals are the hardware ones
// (v_log_f32, v_sqrt_f32, v_sin_f32 / v_cos_f32 in revolutions, each within a few
// ulp or 2^-20 absolute): the uniforms are exact multiples of 2^-24, the angle
// pi a with a in [0, 2) is a / 2 revolutions.
__device__ __forceinline__ void normals8(uint64_t j, uint64_t seed, float z[8]) {
    uint64_t w[4];
    philox4x64_10(j, seed, w);
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        const uint32_t ur = (uint32_t)w[p], ua = (uint32_t)(w[p] >> 32);
        const float u = (float)((ur >> 8) + 1u) * 0x1p-24f;                 // (0, 1], exact
        const float r = __builtin_amdgcn_sqrtf(-2.f * 0.69314718055994531f * __builtin_amdgcn_logf(u));
        const float rev = (float)(ua >> 8) * 0x1p-24f;                      // a / 2, exact
        z[2 * p] = r * __builtin_amdgcn_cosf(rev);
        z[2 * p + 1] = r * __builtin_amdgcn_sinf(rev);
    }
}

template <typename T_>
__device__ __forceinline__ void load8(const T_* p, float x[8]);
template <>
__device__ __forceinline__ void load8<float>(const float* p, float x[8]) {
    const float4 a = *reinterpret_cast<const float4*>(p), b = *reinterpret_cast<const float4*>(p + 4);
    x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w; x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}
template <>
__device__ __forceinline__ void load8<uint16_t>(const uint16_t* p, float x[8]) {
    const uint4 a = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        x[2 * i] = __uint_as_float(w[i] << 16);
        x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
}

__device__ __forceinline__ void store8(float* p, const float x[8]) {
    *reinterpret_cast<float4*>(p) = make_float4(x[0], x[1], x[2], x[3]);
    *reinterpret_cast<float4*>(p + 4) = make_float4(x[4], x[5], x[6], x[7]);
}
__device__ __forceinline__ void store8(uint16_t* p, const float x[8]) {
    *reinterpret_cast<uint4*>(p) =
        make_uint4(cvt_pk_bf16(x[0], x[1]), cvt_pk_bf16(x[2], x[3]), cvt_pk_bf16(x[4], x[5]), cvt_pk_bf16(x[6], x[7]));
}

// one thread per (row, 8 channels); rows = B T H, G = dv / 8 threads per row
template <typename T_>
__global__ __launch_bounds__(256) void mc_sample_kernel(int S, size_t nrow, int G, uint64_t seed,
                                                        const T_* __restrict__ ymu, const float* __restrict__ yvar,
                                                        T_* __restrict__ ys) {
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= nrow * G) return;
    const size_t row = i / G;
    float mu[8];
    load8(ymu + 8 * i, mu);
    const float sd = sqrtf(yvar[row]);
    const size_t per_s = nrow * G;   // Philox blocks per sample
    for (int s = 0; s < S; ++s) {
        float z[8];
        normals8((uint64_t)s * per_s + i, seed, z);
#pragma unroll
        for (int k = 0; k < 8; ++k) z[k] = fmaf(sd, z[k], mu[k]);
        store8(ys + ((size_t)s * per_s + i) * 8, z);
    }
}

// dymu = sum_s dys^(s); dyvar = sum_{s,d} dys^(s) eps^(s) / (2 sqrt(yvar)), the dot summed
// in fp64 over the thread's draws, then over the G lanes of the row (consecutive lanes of
// one wave), in a fixed order
template <typename T_>
__global__ __launch_bounds__(256) void mc_sample_bwd_kernel(int S, size_t nrow, int G, uint64_t seed,
                                                            const float* __restrict__ yvar, const T_* __restrict__ dys,
                                                            T_* __restrict__ dymu, float* __restrict__ dyvar) {
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const bool live = i < nrow * G;
    const size_t row = live ? i / G : 0;
    const size_t per_s = nrow * G;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    double dot = 0.0;
    if (live) {
        for (int s = 0; s < S; ++s) {
            float g[8], z[8];
            load8(dys + ((size_t)s * per_s + i) * 8, g);
            normals8((uint64_t)s * per_s + i, seed, z);
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                acc[k] += g[k];
                dot = fma((double)g[k], (double)z[k], dot);
            }
        }
        store8(dymu + 8 * i, acc);
    }
    // the G lanes of a row: G divides 64 and rows start at multiples of G
    for (int o = 1; o < G; o <<= 1) dot += __shfl_xor(dot, o, 64);
    if (live && i % G == 0) dyvar[row] = (float)(dot / (2.0 * sqrt((double)yvar[row])));
}

// nll[i] = -logsumexp_s(logp[s, i]) + log S
__global__ __launch_bounds__(256) void mc_nll_kernel(int S, size_t n, const float* __restrict__ logp,
                                                     float* __restrict__ nll) {
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    float m = logp[i];
    for (int s = 1; s < S; ++s) m = fmaxf(m, logp[(size_t)s * n + i]);
    float sum = 0.f;
    for (int s = 0; s < S; ++s) sum += expf(logp[(size_t)s * n + i] - m);
    nll[i] = logf((float)S) - m - logf(sum);
}

// dlogp[s, i] = -dnll[i] softmax_s(logp[., i])
__global__ __launch_bounds__(256) void mc_nll_bwd_kernel(int S, size_t n, const float* __restrict__ logp,
                                                         const float* __restrict__ dnll, float* __restrict__ dlogp) {
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    float m = logp[i];
    for (int s = 1; s < S; ++s) m = fmaxf(m, logp[(size_t)s * n + i]);
    float sum = 0.f;
    for (int s = 0; s < S; ++s) sum += expf(logp[(size_t)s * n + i] - m);
    const float c = -dnll[i] / sum;
    for (int s = 0; s < S; ++s) dlogp[(size_t)s * n + i] = c * expf(logp[(size_t)s * n + i] - m);
}

unsigned blocks(size_t n) { return (unsigned)((n + 255) / 256); }

}  // namespace

hipError_t launch_mc_sample(int S, size_t nrow, int dv, bool bf16, uint64_t seed, const void* ymu, const float* yvar,
                            void* ys, hipStream_t st) {
    const int G = dv / 8;
    if (nrow == 0) return hipSuccess;
    if (bf16)
        hipLaunchKernelGGL(mc_sample_kernel<uint16_t>, dim3(blocks(nrow * G)), dim3(256), 0, st, S, nrow, G, seed,
                           static_cast<const uint16_t*>(ymu), yvar, static_cast<uint16_t*>(ys));
    else
        hipLaunchKernelGGL(mc_sample_kernel<float>, dim3(blocks(nrow * G)), dim3(256), 0, st, S, nrow, G, seed,
                           static_cast<const float*>(ymu), yvar, static_cast<float*>(ys));
    return hipGetLastError();
}

hipError_t launch_mc_sample_bwd(int S, size_t nrow, int dv, bool bf16, uint64_t seed, const float* yvar,
                                const void* dys, void* dymu, float* dyvar, hipStream_t st) {
    const int G = dv / 8;
    if (nrow == 0) return hipSuccess;
    if (bf16)
        hipLaunchKernelGGL(mc_sample_bwd_kernel<uint16_t>, dim3(blocks(nrow * G)), dim3(256), 0, st, S, nrow, G, seed,
                           yvar, static_cast<const uint16_t*>(dys), static_cast<uint16_t*>(dymu), dyvar);
    else
        hipLaunchKernelGGL(mc_sample_bwd_kernel<float>, dim3(blocks(nrow * G)), dim3(256), 0, st, S, nrow, G, seed,
                           yvar, static_cast<const float*>(dys), static_cast<float*>(dymu), dyvar);
    return hipGetLastError();
}

hipError_t launch_mc_nll(int S, size_t n, const float* logp, float* nll, hipStream_t st) {
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(mc_nll_kernel, dim3(blocks(n)), dim3(256), 0, st, S, n, logp, nll);
    return hipGetLastError();
}

hipError_t launch_mc_nll_bwd(int S, size_t n, const float* logp, const float* dnll, float* dlogp, hipStream_t st) {
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(mc_nll_bwd_kernel, dim3(blocks(n)), dim3(256), 0, st, S, n, logp, dnll, dlogp);
    return hipGetLastError();
}

}  // namespace kla
