// Per-channel precision: the filter with one observation precision per value
// channel, r_t[d] (Algorithm 1's Lambda^v of shape (B, T, 1, D)), so that the
// precision, the prior ratio and the forget gate are d_k x d_v arrays per head
// (eqs. kla-prec-mat and kla-mean-mat elementwise):
//   rho_t[n,d] = 1 / (abar_t[n]^2 + pbar_t[n] lam_{t-1}[n,d])
//   lam_t[n,d] = rho_t[n,d] lam_{t-1}[n,d] + k_t[n]^2 r_t[d]
//   H_t[n,d]   = abar_t[n] rho_t[n,d] H_{t-1}[n,d] + k_t[n] r_t[d] v_t[d]
//   y_t[d]     = sum_n q_t[n] H_t[n,d] / lam_t[n,d],  yvar_t[d] = sum_n q_t[n]^2 / lam_t[n,d]
// There is no shared gate to factor out of a chunk, so the scan is elementwise:
// every (n, d) runs its own recursion, token after token, with lam and H in
// registers.  It is bound by VALU issue (two quotients per element and token),
// not by HBM.
//
// Per element and token one reciprocal serves both quotients: with
// den = abar^2 + pbar lam and num = lam + k^2 r den (so lam_t = num / den),
//   R = 1 / (den num),  1 / den = num R,  1 / lam_t = den^2 R.
#include "kla_buf.hpp"
#include "kla_device.hpp"
#include "kla_internal.hpp"

namespace kla {
namespace {

constexpr int kNG = 8;    // lanes sharing one value channel, each with every 8th key slot
constexpr int kTB = 16;   // tokens per staged block

__device__ __forceinline__ float sum8(float x) {   // over the 8 lanes of a channel
    x += dpp<0xB1, 0xf>(x);    // quad_perm [1,0,3,2]
    x += dpp<0x4E, 0xf>(x);    // quad_perm [2,3,0,1]
    x += dpp<0x141, 0xf>(x);   // row_half_mirror
    return x;
}

// One workgroup per (b, h, CT value channels); lane l of the workgroup owns
// channel d0 + l / 8 and key slots n = l % 8 + 8 i.  Per block of kTB tokens the
// key-side inputs (abar, pbar, k, q as fp32 [t][n]) and the channel inputs
// (r, v as [t][c]) are staged in LDS, the elements are updated, the partial
// readouts summed over the 8 lanes of a channel and y, yvar written from LDS.
template <typename S, int DK, int DV>
__global__ __launch_bounds__(8 * (DV < 32 ? DV : 32)) void fwd_pc_kernel(Shape s, FwdArgs g) {
    using T_ = typename storage<S>::type;
    constexpr int CT = DV < 32 ? DV : 32;
    constexpr int NTHR = kNG * CT;
    constexpr int NPER = DK / kNG;
    __shared__ float4 s_k[kTB][DK];
    __shared__ float2 s_v[kTB][CT];
    __shared__ float s_y[kTB][CT], s_w[kTB][CT];

    const T_ *q = static_cast<const T_*>(g.q), *k = static_cast<const T_*>(g.k), *v = static_cast<const T_*>(g.v);
    const T_ *a = static_cast<const T_*>(g.a), *p = static_cast<const T_*>(g.p), *r = static_cast<const T_*>(g.r);
    T_* y = static_cast<T_*>(g.y);
    const int ntile = DV / CT;
    const int bh = blockIdx.x / ntile, d0 = (blockIdx.x % ntile) * CT;
    const int b = bh / s.H, h = bh % s.H;
    const int tid = threadIdx.x, ng = tid % kNG, c = tid / kNG, d = d0 + c;

    float lam[NPER], eta[NPER];
#pragma unroll
    for (int i = 0; i < NPER; ++i) {
        const size_t o = ((size_t)bh * DK + ng + kNG * i) * DV + d;
        lam[i] = g.lam0 ? g.lam0[o] : 1.f;
        eta[i] = g.eta0 ? g.eta0[o] : 0.f;
    }
    for (int t0 = 0; t0 < s.T; t0 += kTB) {
        const int nt = min(kTB, s.T - t0);
        for (int idx = tid; idx < nt * DK; idx += NTHR) {
            const int t = idx / DK, n = idx % DK;
            const size_t o = (((size_t)b * s.T + t0 + t) * s.H + h) * DK + n;
            s_k[t][n] = make_float4(ld(a, o), ld(p, o), ld(k, o), ld(q, o));
        }
        for (int idx = tid; idx < nt * CT; idx += NTHR) {
            const int t = idx / CT, cc = idx % CT;
            const size_t o = (((size_t)b * s.T + t0 + t) * s.H + h) * DV + d0 + cc;
            s_v[t][cc] = make_float2(ld(r, o), ld(v, o));
        }
        __syncthreads();
        for (int t = 0; t < nt; ++t) {
            const float2 rv = s_v[t][c];
            const float krv_s = rv.x * rv.y;   // r v: the evidence k r v over k
            float ya = 0.f, wa = 0.f;
#pragma unroll
            for (int i = 0; i < NPER; ++i) {
                const float4 in = s_k[t][ng + kNG * i];   // abar, pbar, k, q
                const float den = fmaf(in.y, lam[i], in.x * in.x);
                const float num = fmaf(in.z * in.z * rv.x, den, lam[i]);
                const float R = __builtin_amdgcn_rcpf(den * num);
                const float iden = num * R, ilam = den * (den * R);
                lam[i] = num * iden;
                eta[i] = fmaf(in.x * iden, eta[i], in.z * krv_s);
                ya = fmaf(in.w, eta[i] * ilam, ya);
                wa = fmaf(in.w * in.w, ilam, wa);
            }
            ya = sum8(ya);
            wa = sum8(wa);
            if (ng == 0) {
                s_y[t][c] = ya;
                s_w[t][c] = wa;
            }
        }
        __syncthreads();
        for (int idx = tid; idx < nt * CT; idx += NTHR) {
            const int t = idx / CT, cc = idx % CT;
            const size_t o = (((size_t)b * s.T + t0 + t) * s.H + h) * DV + d0 + cc;
            st(y, o, s_y[t][cc]);
            if (g.yvar) g.yvar[o] = s_w[t][cc];
        }
        // the next block's staging overwrites s_k, s_v only after every lane has read them,
        // and s_y, s_w only after the stores above
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < NPER; ++i) {
        const size_t o = ((size_t)bh * DK + ng + kNG * i) * DV + d;
        if (g.lamT) g.lamT[o] = lam[i];
        if (g.etaT) g.etaT[o] = eta[i];
    }
}

// Decode: one token for S sequences, belief [S, H, dk, dv] updated in place.
// One workgroup per (sequence, head); a thread owns 4 consecutive channels
// (16-byte accesses of lam and eta) of every NG-th key slot.
template <typename S, int DK, int DV>
__global__ __launch_bounds__(256) void decode_pc_kernel(int H, DecodeArgs g) {
    using T_ = typename storage<S>::type;
    constexpr int DV4 = DV / 4;
    constexpr int NG = (256 / DV4) < DK ? (256 / DV4) : DK;
    constexpr int NPER = DK / NG;
    __shared__ float4 s_k[DK];
    __shared__ float4 s_r[DV4], s_v[DV4];
    __shared__ float4 s_y[NG][DV4], s_w[NG][DV4];

    const T_ *q = static_cast<const T_*>(g.q), *k = static_cast<const T_*>(g.k), *v = static_cast<const T_*>(g.v);
    const T_ *a = static_cast<const T_*>(g.a), *p = static_cast<const T_*>(g.p), *r = static_cast<const T_*>(g.r);
    T_* y = static_cast<T_*>(g.y);
    const size_t sh = blockIdx.x;
    const int tid = threadIdx.x;
    for (int n = tid; n < DK; n += 256) {
        const size_t o = sh * DK + n;
        s_k[n] = make_float4(ld(a, o), ld(p, o), ld(k, o), ld(q, o));
    }
    for (int j = tid; j < DV4; j += 256) {
        const size_t o = sh * DV + 4 * j;
        s_r[j] = make_float4(ld(r, o), ld(r, o + 1), ld(r, o + 2), ld(r, o + 3));
        s_v[j] = make_float4(ld(v, o), ld(v, o + 1), ld(v, o + 2), ld(v, o + 3));
    }
    __syncthreads();
    const int d4 = tid % DV4, ng = tid / DV4;
    if (ng < NG) {
        const float4 rr = s_r[d4], vv = s_v[d4];
        const float rc[4] = {rr.x, rr.y, rr.z, rr.w};
        const float rv[4] = {rr.x * vv.x, rr.y * vv.y, rr.z * vv.z, rr.w * vv.w};
        float ya[4] = {0.f, 0.f, 0.f, 0.f}, wa[4] = {0.f, 0.f, 0.f, 0.f};
        float4* lam4 = reinterpret_cast<float4*>(g.lam + sh * DK * DV);
        float4* eta4 = reinterpret_cast<float4*>(g.eta + sh * DK * DV);
#pragma unroll 2
        for (int i = 0; i < NPER; ++i) {
            const int n = ng + NG * i;
            const float4 in = s_k[n];
            const float4 l4 = lam4[n * DV4 + d4], e4 = eta4[n * DV4 + d4];
            float lp[4] = {l4.x, l4.y, l4.z, l4.w}, ep[4] = {e4.x, e4.y, e4.z, e4.w};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const float den = fmaf(in.y, lp[j], in.x * in.x);
                const float num = fmaf(in.z * in.z * rc[j], den, lp[j]);
                const float R = __builtin_amdgcn_rcpf(den * num);
                const float iden = num * R, ilam = den * (den * R);
                lp[j] = num * iden;
                ep[j] = fmaf(in.x * iden, ep[j], in.z * rv[j]);
                ya[j] = fmaf(in.w, ep[j] * ilam, ya[j]);
                wa[j] = fmaf(in.w * in.w, ilam, wa[j]);
            }
            lam4[n * DV4 + d4] = make_float4(lp[0], lp[1], lp[2], lp[3]);
            eta4[n * DV4 + d4] = make_float4(ep[0], ep[1], ep[2], ep[3]);
        }
        s_y[ng][d4] = make_float4(ya[0], ya[1], ya[2], ya[3]);
        s_w[ng][d4] = make_float4(wa[0], wa[1], wa[2], wa[3]);
    }
    __syncthreads();
    for (int j = tid; j < DV4; j += 256) {
        float4 ys = s_y[0][j], ws = s_w[0][j];
        for (int gi = 1; gi < NG; ++gi) {
            const float4 y2 = s_y[gi][j], w2 = s_w[gi][j];
            ys.x += y2.x; ys.y += y2.y; ys.z += y2.z; ys.w += y2.w;
            ws.x += w2.x; ws.y += w2.y; ws.z += w2.z; ws.w += w2.w;
        }
        const size_t o = sh * DV + 4 * j;
        st(y, o, ys.x);
        st(y, o + 1, ys.y);
        st(y, o + 2, ys.z);
        st(y, o + 3, ys.w);
        if (g.yvar) {
            g.yvar[o] = ws.x;
            g.yvar[o + 1] = ws.y;
            g.yvar[o + 2] = ws.z;
            g.yvar[o + 3] = ws.w;
        }
    }
}

template <template <typename, int, int> class L, typename... A>
hipError_t dispatch_pc(const Shape& s, A&&... args) {
#define KLA_PC_CASE(DK_, DV_)                                                           \
    if (s.dk == DK_ && s.dv == DV_)                                                     \
        return s.bf16 ? L<bf16_t, DK_, DV_>::run(s, args...) : L<f32_t, DK_, DV_>::run(s, args...);
#define KLA_PC_ROW(DK_) KLA_PC_CASE(DK_, 16) KLA_PC_CASE(DK_, 32) KLA_PC_CASE(DK_, 64) KLA_PC_CASE(DK_, 128)
    KLA_PC_ROW(16) KLA_PC_ROW(32) KLA_PC_ROW(64) KLA_PC_ROW(128)
#undef KLA_PC_ROW
#undef KLA_PC_CASE
    return hipErrorInvalidValue;
}

template <typename S, int DK, int DV>
struct FwdPc {
    static hipError_t run(const Shape& s, const FwdArgs& a, hipStream_t st) {
        constexpr int CT = DV < 32 ? DV : 32;
        hipLaunchKernelGGL((fwd_pc_kernel<S, DK, DV>), dim3((unsigned)(s.B * s.H * (DV / CT))), dim3(kNG * CT), 0,
                           st, s, a);
        return hipGetLastError();
    }
};

template <typename S, int DK, int DV>
struct DecPc {
    static hipError_t run(const Shape& s, const DecodeArgs& a, hipStream_t st) {
        hipLaunchKernelGGL((decode_pc_kernel<S, DK, DV>), dim3((unsigned)(s.B * s.H)), dim3(256), 0, st, s.H, a);
        return hipGetLastError();
    }
};

}  // namespace

hipError_t launch_forward_pc(const Shape& s, const FwdArgs& a, hipStream_t st) { return dispatch_pc<FwdPc>(s, a, st); }

hipError_t launch_decode_pc(const Shape& s, const DecodeArgs& a, hipStream_t st) {
    return dispatch_pc<DecPc>(s, a, st);
}

}  // namespace kla
