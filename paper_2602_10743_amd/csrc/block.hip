// Scaffolding of the KLA block (Mamba-style, Sec. 4.4 and the architecture
// paragraph of Appendix A): causal depthwise conv1d of kernel 4 fused with
// SiLU, RMS QK-norm, and the SiLU gate, forward and backward.
//
//   conv:  u[b,t,c] = silu(bias[c] + sum_j w[c,j] x[b,t-3+j,c])   (x = 0 before t = 0)
//   norm:  out = x / sqrt(mean(x^2) + eps) * w   over rows of n elements
//   gate:  out = y * silu(z)
//
// All are bound by HBM: every thread moves 16-byte vectors (8 bf16 or 4 fp32
// elements) along the contiguous dimension.  Reductions over tokens or rows
// (the weight gradients) go through per-block parts that a second kernel adds
// in a fixed order, so results are bitwise reproducible.
#include "kla_device.hpp"
#include "kla_internal.hpp"

namespace kla {
namespace {

template <typename S>
struct Vec;
template <>
struct Vec<bf16_t> {
    static constexpr int N = 8;
    using raw = uint4;
    __device__ static void load(const void* p, size_t i, float* f) {
        const uint4 u = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(p) + i);
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            f[2 * e] = __uint_as_float(w[e] << 16);
            f[2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u);
        }
    }
    __device__ static void store(void* p, size_t i, const float* f) {
        uint4 u;
        u.x = cvt_pk_bf16(f[0], f[1]);
        u.y = cvt_pk_bf16(f[2], f[3]);
        u.z = cvt_pk_bf16(f[4], f[5]);
        u.w = cvt_pk_bf16(f[6], f[7]);
        *reinterpret_cast<uint4*>(static_cast<uint16_t*>(p) + i) = u;
    }
};
template <>
struct Vec<f32_t> {
    static constexpr int N = 4;
    __device__ static void load(const void* p, size_t i, float* f) {
        const float4 v = *reinterpret_cast<const float4*>(static_cast<const float*>(p) + i);
        f[0] = v.x;
        f[1] = v.y;
        f[2] = v.z;
        f[3] = v.w;
    }
    __device__ static void store(void* p, size_t i, const float* f) {
        *reinterpret_cast<float4*>(static_cast<float*>(p) + i) = make_float4(f[0], f[1], f[2], f[3]);
    }
};

__device__ __forceinline__ float sigm(float x) { return __builtin_amdgcn_rcpf(1.f + __expf(-x)); }

// Conv threads: a block is 64 channel groups (16-byte vectors) x kSub token
// runs of kTT tokens; the backward adds its weight-gradient partials over the
// kSub runs in LDS before writing one part per block.
constexpr int kTT = 16;   // tokens per conv thread
constexpr int kSub = 4;   // token runs per block
constexpr int kCG = 64;   // channel groups per block
constexpr int kTB = kTT * kSub;

struct ConvTile {
    int b, c0, t0, t1, tile, cg;
    bool live;
    __device__ ConvTile(int B, int T, int C, int V) {
        const int ncg = C / V, ncb = (ncg + kCG - 1) / kCG, ntb = (T + kTB - 1) / kTB;
        const int cgl = threadIdx.x % kCG, sub = threadIdx.x / kCG;
        const int bx = blockIdx.x;
        const int cb = bx % ncb;
        tile = (bx / ncb) % ntb;
        b = bx / (ncb * ntb);
        cg = cb * kCG + cgl;
        c0 = cg * V;
        t0 = tile * kTB + sub * kTT;
        t1 = min(T, t0 + kTT);
        live = cg < ncg && t0 < T && b < B;
    }
};

// ---------------------------------------------------------------- conv + SiLU
template <typename S>
__global__ __launch_bounds__(256) void conv_fwd_kernel(int B, int T, int C, const void* __restrict__ x,
                                                       const float* __restrict__ w, const float* __restrict__ bias,
                                                       void* __restrict__ u) {
    constexpr int V = Vec<S>::N;
    const ConvTile ct(B, T, C, V);
    if (!ct.live) return;
    const int b = ct.b, c0 = ct.c0, t0 = ct.t0, t1 = ct.t1;
    float wk[4][V], bs[V];
#pragma unroll
    for (int e = 0; e < V; ++e) {
        const float4 ww = *reinterpret_cast<const float4*>(w + (size_t)(c0 + e) * 4);
        wk[0][e] = ww.x;
        wk[1][e] = ww.y;
        wk[2][e] = ww.z;
        wk[3][e] = ww.w;
        bs[e] = bias ? bias[c0 + e] : 0.f;
    }
    // history x[t-3], x[t-2], x[t-1]
    float h3[V], h2[V], h1[V];
    auto load_or_zero = [&](int t, float* f) {
        if (t >= 0) {
            Vec<S>::load(x, ((size_t)b * T + t) * C + c0, f);
        } else {
#pragma unroll
            for (int e = 0; e < V; ++e) f[e] = 0.f;
        }
    };
    if (t1 - t0 == kTT) {
        // a full run: every load of the run unconditional (history before token 0 read from
        // token 0 and replaced by zeros), so the unrolled loop can issue them all up front
        const size_t r0 = (size_t)b * T * C + c0;
        auto hist = [&](int t, float* f) {
            Vec<S>::load(x, r0 + (size_t)max(t, 0) * C, f);
#pragma unroll
            for (int e = 0; e < V; ++e) f[e] = t >= 0 ? f[e] : 0.f;
        };
        hist(t0 - 3, h3);
        hist(t0 - 2, h2);
        hist(t0 - 1, h1);
#pragma unroll
        for (int i = 0; i < kTT; ++i) {
            const int t = t0 + i;
            float cur[V], out[V];
            Vec<S>::load(x, r0 + (size_t)t * C, cur);
#pragma unroll
            for (int e = 0; e < V; ++e) {
                const float s = fmaf(wk[3][e], cur[e], fmaf(wk[2][e], h1[e], fmaf(wk[1][e], h2[e], fmaf(wk[0][e], h3[e], bs[e]))));
                out[e] = s * sigm(s);
                h3[e] = h2[e];
                h2[e] = h1[e];
                h1[e] = cur[e];
            }
            Vec<S>::store(u, r0 + (size_t)t * C, out);
        }
        return;
    }
    load_or_zero(t0 - 3, h3);
    load_or_zero(t0 - 2, h2);
    load_or_zero(t0 - 1, h1);
    for (int t = t0; t < t1; ++t) {
        float cur[V], out[V];
        Vec<S>::load(x, ((size_t)b * T + t) * C + c0, cur);
#pragma unroll
        for (int e = 0; e < V; ++e) {
            const float s = fmaf(wk[3][e], cur[e], fmaf(wk[2][e], h1[e], fmaf(wk[1][e], h2[e], fmaf(wk[0][e], h3[e], bs[e]))));
            out[e] = s * sigm(s);
            h3[e] = h2[e];
            h2[e] = h1[e];
            h1[e] = cur[e];
        }
        Vec<S>::store(u, ((size_t)b * T + t) * C + c0, out);
    }
}

// Reverse over the thread's tokens and 3 halo tokens after them: ds of each
// token from the recomputed pre-activation, dx[t] = sum_j w[j] ds[t+3-j], and
// the weight / bias gradient of the thread's own tokens, added over the
// block's token runs into part (b, token block).
template <typename S>
__global__ __launch_bounds__(256) void conv_bwd_kernel(int B, int T, int C, const void* __restrict__ x,
                                                       const float* __restrict__ w, const float* __restrict__ bias,
                                                       const void* __restrict__ du, void* __restrict__ dx,
                                                       float* __restrict__ part) {
    constexpr int V = Vec<S>::N;
    __shared__ float s_part[kSub][kCG][V * 5];
    const ConvTile ct(B, T, C, V);
    const int b = ct.b, c0 = ct.c0, t0 = ct.t0, t1 = ct.t1;
    const int cgl = threadIdx.x % kCG, sub = threadIdx.x / kCG;
    float gw[4][V], gb[V];
#pragma unroll
    for (int e = 0; e < V; ++e) gw[0][e] = gw[1][e] = gw[2][e] = gw[3][e] = gb[e] = 0.f;
    if (ct.live) {
        float wk[4][V], bs[V];
#pragma unroll
        for (int e = 0; e < V; ++e) {
            const float4 ww = *reinterpret_cast<const float4*>(w + (size_t)(c0 + e) * 4);
            wk[0][e] = ww.x;
            wk[1][e] = ww.y;
            wk[2][e] = ww.z;
            wk[3][e] = ww.w;
            bs[e] = bias ? bias[c0 + e] : 0.f;
        }
        auto load_or_zero = [&](const void* src, int t, float* f) {
            if (t >= 0 && t < T) {
                Vec<S>::load(src, ((size_t)b * T + t) * C + c0, f);
            } else {
#pragma unroll
                for (int e = 0; e < V; ++e) f[e] = 0.f;
            }
        };
        const int ts = min(T - 1, t1 + 2);   // the last token whose ds reaches this tile's dx
        // x window for token t: x[t], x[t-1], x[t-2], x[t-3]; ds of tokens t+1, t+2, t+3
        float x0[V], x1[V], x2[V], x3[V], d1[V], d2[V], d3[V];
        if (t1 - t0 == kTT && t1 + 3 <= T) {
            // a full run with its 3 halo tokens inside the sequence: the unrolled loop has
            // no branch (x before token 0 is read from token 0 and replaced by zeros), so
            // every load of the run can be issued up front
            const size_t r0 = (size_t)b * T * C + c0;
            auto xat = [&](int t, float* f) {
                Vec<S>::load(x, r0 + (size_t)max(t, 0) * C, f);
#pragma unroll
                for (int e = 0; e < V; ++e) f[e] = t >= 0 ? f[e] : 0.f;
            };
            xat(ts, x0);
            xat(ts - 1, x1);
            xat(ts - 2, x2);
            xat(ts - 3, x3);
#pragma unroll
            for (int e = 0; e < V; ++e) d1[e] = d2[e] = d3[e] = 0.f;
#pragma unroll
            for (int i = 0; i < kTT + 3; ++i) {
                const int t = ts - i;
                constexpr int kHalo = 3;
                float g[V], ds[V], xn[V], dxo[V];
                Vec<S>::load(du, r0 + (size_t)t * C, g);
                xat(t - 4, xn);
#pragma unroll
                for (int e = 0; e < V; ++e) {
                    const float s = fmaf(wk[3][e], x0[e], fmaf(wk[2][e], x1[e], fmaf(wk[1][e], x2[e], fmaf(wk[0][e], x3[e], bs[e]))));
                    const float sg = sigm(s);
                    ds[e] = g[e] * sg * fmaf(s, 1.f - sg, 1.f);
                    dxo[e] = fmaf(wk[3][e], ds[e], fmaf(wk[2][e], d1[e], fmaf(wk[1][e], d2[e], wk[0][e] * d3[e])));
                    if (i >= kHalo) {   // the run's own tokens
                        gw[3][e] = fmaf(ds[e], x0[e], gw[3][e]);
                        gw[2][e] = fmaf(ds[e], x1[e], gw[2][e]);
                        gw[1][e] = fmaf(ds[e], x2[e], gw[1][e]);
                        gw[0][e] = fmaf(ds[e], x3[e], gw[0][e]);
                        gb[e] += ds[e];
                    }
                    d3[e] = d2[e];
                    d2[e] = d1[e];
                    d1[e] = ds[e];
                    x0[e] = x1[e];
                    x1[e] = x2[e];
                    x2[e] = x3[e];
                    x3[e] = xn[e];
                }
                if (i >= kHalo) Vec<S>::store(dx, r0 + (size_t)t * C, dxo);
            }
        } else {
            load_or_zero(x, ts, x0);
            load_or_zero(x, ts - 1, x1);
            load_or_zero(x, ts - 2, x2);
            load_or_zero(x, ts - 3, x3);
#pragma unroll
            for (int e = 0; e < V; ++e) d1[e] = d2[e] = d3[e] = 0.f;
            for (int t = ts; t >= t0; --t) {
                float g[V], ds[V], xn[V];
                load_or_zero(du, t, g);
                load_or_zero(x, t - 4, xn);
                const bool own = t < t1;
                float dxo[V];
#pragma unroll
                for (int e = 0; e < V; ++e) {
                    const float s = fmaf(wk[3][e], x0[e], fmaf(wk[2][e], x1[e], fmaf(wk[1][e], x2[e], fmaf(wk[0][e], x3[e], bs[e]))));
                    const float sg = sigm(s);
                    ds[e] = g[e] * sg * fmaf(s, 1.f - sg, 1.f);
                    dxo[e] = fmaf(wk[3][e], ds[e], fmaf(wk[2][e], d1[e], fmaf(wk[1][e], d2[e], wk[0][e] * d3[e])));
                    if (own) {
                        gw[3][e] = fmaf(ds[e], x0[e], gw[3][e]);
                        gw[2][e] = fmaf(ds[e], x1[e], gw[2][e]);
                        gw[1][e] = fmaf(ds[e], x2[e], gw[1][e]);
                        gw[0][e] = fmaf(ds[e], x3[e], gw[0][e]);
                        gb[e] += ds[e];
                    }
                    d3[e] = d2[e];
                    d2[e] = d1[e];
                    d1[e] = ds[e];
                    x0[e] = x1[e];
                    x1[e] = x2[e];
                    x2[e] = x3[e];
                    x3[e] = xn[e];
                }
                if (own) Vec<S>::store(dx, ((size_t)b * T + t) * C + c0, dxo);
            }
        }
    }
#pragma unroll
    for (int e = 0; e < V; ++e) {
        s_part[sub][cgl][5 * e + 0] = gw[0][e];
        s_part[sub][cgl][5 * e + 1] = gw[1][e];
        s_part[sub][cgl][5 * e + 2] = gw[2][e];
        s_part[sub][cgl][5 * e + 3] = gw[3][e];
        s_part[sub][cgl][5 * e + 4] = gb[e];
    }
    __syncthreads();
    // part (b, token block): [C][5] = dw[c][0..3], dbias[c]; the sub-runs added in order
    const int ntb = (T + kTB - 1) / kTB;
    if (sub == 0 && ct.cg < C / V && b < B) {
        float* pp = part + ((size_t)b * ntb + ct.tile) * C * 5 + (size_t)c0 * 5;
        for (int i = 0; i < V * 5; ++i) {
            float acc = 0.f;
#pragma unroll
            for (int s2 = 0; s2 < kSub; ++s2) acc += s_part[s2][cgl][i];
            pp[i] = acc;
        }
    }
}

__global__ __launch_bounds__(256) void conv_wgrad_kernel(int nparts, int C, const float* __restrict__ part,
                                                         float* __restrict__ dw, float* __restrict__ dbias) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;   // c * 5 + j
    if (i >= C * 5) return;
    // eight interleaved partial sums keep eight loads in flight; added in a fixed order
    float a8[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    int p = 0;
    for (; p + 8 <= nparts; p += 8)
#pragma unroll
        for (int u = 0; u < 8; ++u) a8[u] += part[(size_t)(p + u) * C * 5 + i];
#pragma unroll
    for (int u = 0; u < 8; ++u)
        if (p + u < nparts) a8[u] += part[(size_t)(p + u) * C * 5 + i];
    const float acc = ((a8[0] + a8[1]) + (a8[2] + a8[3])) + ((a8[4] + a8[5]) + (a8[6] + a8[7]));
    const int c = i / 5, j = i % 5;
    if (j < 4)
        dw[c * 4 + j] = acc;
    else if (dbias)
        dbias[c] = acc;
}

// ---------------------------------------------------------------- RMS QK-norm
// A group of G = N / V lanes per row, one 16-byte vector each; the row sums
// are butterflies over the group's lanes.
template <int G>
__device__ __forceinline__ float group_sum(float v) {
#pragma unroll
    for (int m = G / 2; m >= 1; m /= 2) v += __shfl_xor(v, m, G);
    return v;
}

constexpr int kNormBlocks = 1024;   // fixed grid of the norm kernels (the weight-gradient parts)

template <typename S, int N>
__global__ __launch_bounds__(256) void norm_fwd_kernel(size_t rows, const void* __restrict__ x,
                                                       const float* __restrict__ w, float eps, void* __restrict__ out,
                                                       float* __restrict__ rstd) {
    constexpr int V = Vec<S>::N, G = N / V, RPB = 256 / G;
    const int gl = threadIdx.x % G, rl = threadIdx.x / G;
    float wv[V];
#pragma unroll
    for (int e = 0; e < V; ++e) wv[e] = w[gl * V + e];
    for (size_t row = (size_t)blockIdx.x * RPB + rl; row < rows; row += (size_t)gridDim.x * RPB) {
        float f[V];
        Vec<S>::load(x, row * N + gl * V, f);
        float ss = 0.f;
#pragma unroll
        for (int e = 0; e < V; ++e) ss = fmaf(f[e], f[e], ss);
        ss = group_sum<G>(ss);
        const float r = __builtin_amdgcn_rsqf(ss * (1.f / N) + eps);
#pragma unroll
        for (int e = 0; e < V; ++e) f[e] = f[e] * r * wv[e];
        Vec<S>::store(out, row * N + gl * V, f);
        if (gl == 0 && rstd) rstd[row] = r;
    }
}

// dx = rstd (w dout - xh mean(xh w dout)), xh = x rstd; the weight gradient
// sum_rows dout xh goes to one part per block.
template <typename S, int N>
__global__ __launch_bounds__(256) void norm_bwd_kernel(size_t rows, const void* __restrict__ x,
                                                       const float* __restrict__ w, const float* __restrict__ rstd,
                                                       const void* __restrict__ dout, void* __restrict__ dx,
                                                       float* __restrict__ part) {
    constexpr int V = Vec<S>::N, G = N / V, RPB = 256 / G;
    __shared__ float s_dw[RPB][N];
    const int gl = threadIdx.x % G, rl = threadIdx.x / G;
    float wv[V], acc[V];
#pragma unroll
    for (int e = 0; e < V; ++e) {
        wv[e] = w[gl * V + e];
        acc[e] = 0.f;
    }
    for (size_t row = (size_t)blockIdx.x * RPB + rl; row < rows; row += (size_t)gridDim.x * RPB) {
        float f[V], g[V];
        Vec<S>::load(x, row * N + gl * V, f);
        Vec<S>::load(dout, row * N + gl * V, g);
        const float r = rstd[row];
        float dot = 0.f;
#pragma unroll
        for (int e = 0; e < V; ++e) {
            f[e] *= r;   // xh
            dot = fmaf(f[e] * wv[e], g[e], dot);
            acc[e] = fmaf(g[e], f[e], acc[e]);
        }
        const float m = group_sum<G>(dot) * (1.f / N);
#pragma unroll
        for (int e = 0; e < V; ++e) g[e] = r * fmaf(-f[e], m, wv[e] * g[e]);
        Vec<S>::store(dx, row * N + gl * V, g);
    }
#pragma unroll
    for (int e = 0; e < V; ++e) s_dw[rl][gl * V + e] = acc[e];
    __syncthreads();
    for (int i = threadIdx.x; i < N; i += 256) {
        float sum = 0.f;
        for (int r2 = 0; r2 < RPB; ++r2) sum += s_dw[r2][i];
        part[(size_t)blockIdx.x * N + i] = sum;
    }
}

// one block per weight element: the parts spread over the block's threads, then a tree in LDS
__global__ __launch_bounds__(256) void norm_wgrad_kernel(int nparts, int N, const float* __restrict__ part,
                                                         float* __restrict__ dw) {
    __shared__ float s_acc[256];
    const int i = blockIdx.x;
    float acc = 0.f;
    for (int p = threadIdx.x; p < nparts; p += 256) acc += part[(size_t)p * N + i];
    s_acc[threadIdx.x] = acc;
    __syncthreads();
    for (int m = 128; m >= 1; m /= 2) {
        if ((int)threadIdx.x < m) s_acc[threadIdx.x] += s_acc[threadIdx.x + m];
        __syncthreads();
    }
    if (threadIdx.x == 0) dw[i] = s_acc[0];
}

// ---------------------------------------------------------------- gate
template <typename S>
__global__ __launch_bounds__(256) void gate_fwd_kernel(size_t n, const void* __restrict__ y,
                                                       const void* __restrict__ z, void* __restrict__ out) {
    constexpr int V = Vec<S>::N;
    for (size_t i = ((size_t)blockIdx.x * blockDim.x + threadIdx.x) * V; i < n; i += (size_t)gridDim.x * blockDim.x * V) {
        float a[V], b[V];
        Vec<S>::load(y, i, a);
        Vec<S>::load(z, i, b);
#pragma unroll
        for (int e = 0; e < V; ++e) a[e] = a[e] * b[e] * sigm(b[e]);
        Vec<S>::store(out, i, a);
    }
}

template <typename S>
__global__ __launch_bounds__(256) void gate_bwd_kernel(size_t n, const void* __restrict__ y,
                                                       const void* __restrict__ z, const void* __restrict__ dout,
                                                       void* __restrict__ dy, void* __restrict__ dz) {
    constexpr int V = Vec<S>::N;
    for (size_t i = ((size_t)blockIdx.x * blockDim.x + threadIdx.x) * V; i < n; i += (size_t)gridDim.x * blockDim.x * V) {
        float a[V], b[V], g[V], oy[V], oz[V];
        Vec<S>::load(y, i, a);
        Vec<S>::load(z, i, b);
        Vec<S>::load(dout, i, g);
#pragma unroll
        for (int e = 0; e < V; ++e) {
            const float sg = sigm(b[e]);
            oy[e] = g[e] * b[e] * sg;
            oz[e] = g[e] * a[e] * sg * fmaf(b[e], 1.f - sg, 1.f);
        }
        Vec<S>::store(dy, i, oy);
        Vec<S>::store(dz, i, oz);
    }
}

unsigned blocks_for(size_t threads) { return (unsigned)((threads + 255) / 256); }

unsigned stream_blocks(size_t n, int v) {
    const size_t want = (n / v + 255) / 256;
    return (unsigned)(want < 8192 ? (want > 0 ? want : 1) : 8192);
}

}  // namespace

int block_vec(bool bf16) { return bf16 ? 8 : 4; }

static unsigned conv_blocks(int B, int T, int C, int V) {
    const int ncb = (C / V + kCG - 1) / kCG, ntb = (T + kTB - 1) / kTB;
    return (unsigned)((size_t)B * ntb * ncb);
}

size_t conv_parts_bytes(int B, int T, int C) {
    const size_t ntb = (size_t)(T + kTB - 1) / kTB;
    return (size_t)B * ntb * C * 5 * sizeof(float);
}

size_t norm_parts_bytes(int n) { return (size_t)kNormBlocks * n * sizeof(float); }

hipError_t launch_conv_fwd(int B, int T, int C, bool bf16, const void* x, const float* w, const float* bias, void* u,
                           hipStream_t st) {
    const unsigned nb = conv_blocks(B, T, C, block_vec(bf16));
    if (nb == 0) return hipSuccess;
    if (bf16)
        hipLaunchKernelGGL(conv_fwd_kernel<bf16_t>, dim3(nb), dim3(256), 0, st, B, T, C, x, w, bias, u);
    else
        hipLaunchKernelGGL(conv_fwd_kernel<f32_t>, dim3(nb), dim3(256), 0, st, B, T, C, x, w, bias, u);
    return hipGetLastError();
}

hipError_t launch_conv_bwd(int B, int T, int C, bool bf16, const void* x, const float* w, const float* bias,
                           const void* du, void* dx, float* dw, float* dbias, float* part, hipStream_t st) {
    const int ntb = (T + kTB - 1) / kTB;
    const unsigned nb = conv_blocks(B, T, C, block_vec(bf16));
    if (nb > 0) {
        if (bf16)
            hipLaunchKernelGGL(conv_bwd_kernel<bf16_t>, dim3(nb), dim3(256), 0, st, B, T, C, x, w, bias, du, dx, part);
        else
            hipLaunchKernelGGL(conv_bwd_kernel<f32_t>, dim3(nb), dim3(256), 0, st, B, T, C, x, w, bias, du, dx, part);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(conv_wgrad_kernel, dim3(blocks_for((size_t)C * 5)), dim3(256), 0, st, B * ntb, C, part, dw,
                       dbias);
    return hipGetLastError();
}

template <int N>
static hipError_t norm_fwd_n(size_t rows, bool bf16, const void* x, const float* w, float eps, void* out, float* rstd,
                             hipStream_t st) {
    if (bf16)
        hipLaunchKernelGGL((norm_fwd_kernel<bf16_t, N>), dim3(kNormBlocks), dim3(256), 0, st, rows, x, w, eps, out, rstd);
    else
        hipLaunchKernelGGL((norm_fwd_kernel<f32_t, N>), dim3(kNormBlocks), dim3(256), 0, st, rows, x, w, eps, out, rstd);
    return hipGetLastError();
}

template <int N>
static hipError_t norm_bwd_n(size_t rows, bool bf16, const void* x, const float* w, const float* rstd,
                             const void* dout, void* dx, float* dw, float* part, hipStream_t st) {
    if (bf16)
        hipLaunchKernelGGL((norm_bwd_kernel<bf16_t, N>), dim3(kNormBlocks), dim3(256), 0, st, rows, x, w, rstd, dout,
                           dx, part);
    else
        hipLaunchKernelGGL((norm_bwd_kernel<f32_t, N>), dim3(kNormBlocks), dim3(256), 0, st, rows, x, w, rstd, dout,
                           dx, part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(norm_wgrad_kernel, dim3(N), dim3(256), 0, st, kNormBlocks, N, part, dw);
    return hipGetLastError();
}

hipError_t launch_norm_fwd(size_t rows, int n, bool bf16, const void* x, const float* w, float eps, void* out,
                           float* rstd, hipStream_t st) {
    switch (n) {
        case 16: return norm_fwd_n<16>(rows, bf16, x, w, eps, out, rstd, st);
        case 32: return norm_fwd_n<32>(rows, bf16, x, w, eps, out, rstd, st);
        case 64: return norm_fwd_n<64>(rows, bf16, x, w, eps, out, rstd, st);
        case 128: return norm_fwd_n<128>(rows, bf16, x, w, eps, out, rstd, st);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_norm_bwd(size_t rows, int n, bool bf16, const void* x, const float* w, const float* rstd,
                           const void* dout, void* dx, float* dw, float* part, hipStream_t st) {
    switch (n) {
        case 16: return norm_bwd_n<16>(rows, bf16, x, w, rstd, dout, dx, dw, part, st);
        case 32: return norm_bwd_n<32>(rows, bf16, x, w, rstd, dout, dx, dw, part, st);
        case 64: return norm_bwd_n<64>(rows, bf16, x, w, rstd, dout, dx, dw, part, st);
        case 128: return norm_bwd_n<128>(rows, bf16, x, w, rstd, dout, dx, dw, part, st);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_gate_fwd(size_t n, bool bf16, const void* y, const void* z, void* out, hipStream_t st) {
    if (n == 0) return hipSuccess;
    if (bf16)
        hipLaunchKernelGGL(gate_fwd_kernel<bf16_t>, dim3(stream_blocks(n, 8)), dim3(256), 0, st, n, y, z, out);
    else
        hipLaunchKernelGGL(gate_fwd_kernel<f32_t>, dim3(stream_blocks(n, 4)), dim3(256), 0, st, n, y, z, out);
    return hipGetLastError();
}

hipError_t launch_gate_bwd(size_t n, bool bf16, const void* y, const void* z, const void* dout, void* dy, void* dz,
                           hipStream_t st) {
    if (n == 0) return hipSuccess;
    if (bf16)
        hipLaunchKernelGGL(gate_bwd_kernel<bf16_t>, dim3(stream_blocks(n, 8)), dim3(256), 0, st, n, y, z, dout, dy, dz);
    else
        hipLaunchKernelGGL(gate_bwd_kernel<f32_t>, dim3(stream_blocks(n, 4)), dim3(256), 0, st, n, y, z, dout, dy, dz);
    return hipGetLastError();
}

}  // namespace kla
