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
//
// Backward: the exact reverse-mode derivative of each element's recursion (the
// per-element form of the adjoint in the oracle), with lam and H of every
// token recomputed in registers from checkpoints the forward stores every
// kCK tokens.  Per element and token, with ge, gl the adjoints of H_t and lam_t
// (gy = dy_t[d], gv = dyvar_t[d], mu = H_t / lam_t):
//   dq[n] += mu gy + 2 q gv / lam_t
//   ge    += q gy / lam_t,   gl -= (q gy mu + q^2 gv / lam_t) / lam_t
//   rho = 1 / (abar^2 + pbar lam_{t-1}),  f = abar rho,  df = ge H_{t-1}
//   dk[n] += ge r v + 2 gl k r,  dr[d] += ge k v + gl k^2,  dv[d] += ge k r
//   drho = df abar + gl lam_{t-1},  dden = -drho rho^2
//   dabar[n] += df rho + 2 abar dden,  dpbar[n] += dden lam_{t-1}
//   ge <- f ge,  gl <- gl rho + pbar dden
// and after the first token dlam0 = gl, deta0 = ge.
//
// Gates per (key slot, value channel) (TI instantiations): Algorithm 1's
// Abar, Pbar : (N, D), time-invariant, from OU parameters a, p, delta [H, dk, dv]
// by the exact discretisation of Sec. 4.1; every lane forms the gates of its
// elements once, the gates are not staged, and the backward sums each element's
// gate gradients over its tokens (one part per batch row) instead of storing them.
//
// Arithmetic type A (acc<S>): fp64 for fp32 inputs, fp32 for bf16 inputs; the
// per-element precision and state, their checkpoints and adjoints, and the partial
// sums up to their single rounding into an output are held in A.  The sums over n (dv, dr)
// are completed inside the workgroup, which holds every key slot of its
// channels; the sums over d (dq, dk, dabar, dpbar) inside the workgroup over
// its channels, then across the channel tiles by pc_key_combine_kernel, in a
// fixed order (the results are bitwise reproducible).
#include <type_traits>

#include "kla_buf.hpp"
#include "kla_device.hpp"
#include "kla_internal.hpp"

namespace kla {
namespace {

constexpr int kNG = 8;    // lanes sharing one value channel, each with every 8th key slot
constexpr int kTB = 16;   // tokens per staged block
constexpr int kCK = 8;    // tokens between checkpoints of the belief (saved context)
// The key-slot parts of the backward, [tile][4][B T H dk] fp32, lie part_stride(n)
// floats apart: n = B T H dk is a multiple of a large power of two at the usual
// shapes, and the combine kernel's streams that far apart would all fall on the
// same HBM channels; the pad (1280 bytes) spreads them.
constexpr int kKPad = 320;
__host__ __device__ inline size_t part_stride(size_t n) { return n + kKPad; }

template <typename A>
__device__ __forceinline__ A sum8(A x) {   // over the 8 lanes of a channel
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
template <typename S, int DK, int DV, bool TI>
__global__ __launch_bounds__(8 * (DV < 32 ? DV : 32)) void fwd_pc_kernel(Shape s, FwdArgs g,
                                                                       typename acc<S>::type* ck) {
    using T_ = typename storage<S>::type;
    using A = typename acc<S>::type;
    constexpr int CT = DV < 32 ? DV : 32;
    constexpr int NTHR = kNG * CT;
    constexpr int NPER = DK / kNG;
    __shared__ float4 s_k[kTB][DK];
    __shared__ float2 s_v[kTB][CT];
    __shared__ float s_y[kTB][CT], s_w[kTB][CT];
    __shared__ float s_junk[2][NTHR];   // the writes of the lanes that do not hold a channel's sum

    const T_ *q = static_cast<const T_*>(g.q), *k = static_cast<const T_*>(g.k), *v = static_cast<const T_*>(g.v);
    const T_ *a = static_cast<const T_*>(g.a), *p = static_cast<const T_*>(g.p), *r = static_cast<const T_*>(g.r);
    T_* y = static_cast<T_*>(g.y);
    const int ntile = DV / CT;
    const int bh = blockIdx.x / ntile, d0 = (blockIdx.x % ntile) * CT;
    const int b = bh / s.H, h = bh % s.H;
    const int tid = threadIdx.x, ng = tid % kNG, c = tid / kNG, d = d0 + c;

    A lam[NPER], eta[NPER], ga[NPER], gp[NPER];
#pragma unroll
    for (int i = 0; i < NPER; ++i) {
        const size_t o = ((size_t)bh * DK + ng + kNG * i) * DV + d;
        lam[i] = g.lam0 ? (A)g.lam0[o] : A(1);
        eta[i] = g.eta0 ? (A)g.eta0[o] : A(0);
        if constexpr (TI) {
            const size_t og = ((size_t)h * DK + ng + kNG * i) * DV + d;
            ou_gates(g.ou_a[og], g.ou_p[og], g.ou_d[og], ga[i], gp[i]);
        }
    }
    // checkpoints: the belief before tokens 0, kCK, 2 kCK, ... as lam [BH][nseg][DK][DV] then eta
    const int nseg = (s.T + kCK - 1) / kCK;
    A* ck_lam = ck;
    A* ck_eta = ck ? ck + (size_t)s.B * s.H * nseg * DK * DV : nullptr;
    for (int t0 = 0; t0 < s.T; t0 += kTB) {
        const int nt = min(kTB, s.T - t0);
        for (int idx = tid; idx < nt * DK; idx += NTHR) {
            const int t = idx / DK, n = idx % DK;
            const size_t o = (((size_t)b * s.T + t0 + t) * s.H + h) * DK + n;
            s_k[t][n] = TI ? make_float4(0.f, 0.f, ld(k, o), ld(q, o)) : make_float4(ld(a, o), ld(p, o), ld(k, o), ld(q, o));
        }
        for (int idx = tid; idx < nt * CT; idx += NTHR) {
            const int t = idx / CT, cc = idx % CT;
            const size_t o = (((size_t)b * s.T + t0 + t) * s.H + h) * DV + d0 + cc;
            s_v[t][cc] = make_float2(ld(r, o), ld(v, o));
        }
        __syncthreads();
        for (int t = 0; t < nt; ++t) {
            if (ck && (t0 + t) % kCK == 0) {
#pragma unroll
                for (int i = 0; i < NPER; ++i) {
                    const size_t o = (((size_t)bh * nseg + (t0 + t) / kCK) * DK + ng + kNG * i) * DV + d;
                    ck_lam[o] = lam[i];
                    ck_eta[o] = eta[i];
                }
            }
            const float2 rv = s_v[t][c];
            const A rc = rv.x, krv_s = (A)rv.x * (A)rv.y;   // r v: the evidence k r v over k
            A ya = 0, wa = 0;
#pragma unroll
            for (int i = 0; i < NPER; ++i) {
                const float4 in = s_k[t][ng + kNG * i];   // abar, pbar, k, q
                const A ax = TI ? ga[i] : (A)in.x, py = TI ? gp[i] : (A)in.y, kz = in.z, qw = in.w;
                const A den = fma(py, lam[i], ax * ax);
                const A num = fma(kz * kz * rc, den, lam[i]);
                const A R = rcpa(den * num);
                const A iden = num * R, ilam = den * (den * R);
                lam[i] = num * iden;
                eta[i] = fma(ax * iden, eta[i], kz * krv_s);
                ya = fma(qw, eta[i] * ilam, ya);
                wa = fma(qw * qw, ilam, wa);
            }
            ya = sum8(ya);
            wa = sum8(wa);
            // every lane writes (no lane mask): the channel's lane 0 its sums, the others a junk slot
            *(ng == 0 ? &s_y[t][c] : &s_junk[0][tid]) = (float)ya;
            *(ng == 0 ? &s_w[t][c] : &s_junk[1][tid]) = (float)wa;
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
        if (g.lamT) g.lamT[o] = (float)lam[i];
        if (g.etaT) g.etaT[o] = (float)eta[i];
    }
}

template <typename A>
struct alignas(4 * sizeof(A)) A4p {
    A x, y, z, w;
};

// Decode: one token for S sequences, belief [S, H, dk, dv] updated in place.
// One workgroup per (sequence, head); a thread owns 4 consecutive channels
// (16-byte accesses of lam and eta) of every NG-th key slot.
template <typename S, int DK, int DV, bool TI>
__global__ __launch_bounds__(256) void decode_pc_kernel(int H, DecodeArgs g) {
    using T_ = typename storage<S>::type;
    using A = typename acc<S>::type;
    constexpr int DV4 = DV / 4;
    constexpr int NG = (256 / DV4) < DK ? (256 / DV4) : DK;
    constexpr int NPER = DK / NG;
    __shared__ float4 s_k[DK];
    __shared__ float4 s_r[DV4], s_v[DV4];
    __shared__ A4p<A> s_y[NG][DV4], s_w[NG][DV4];

    const T_ *q = static_cast<const T_*>(g.q), *k = static_cast<const T_*>(g.k), *v = static_cast<const T_*>(g.v);
    const T_ *a = static_cast<const T_*>(g.a), *p = static_cast<const T_*>(g.p), *r = static_cast<const T_*>(g.r);
    T_* y = static_cast<T_*>(g.y);
    const size_t sh = blockIdx.x;
    const int tid = threadIdx.x;
    for (int n = tid; n < DK; n += 256) {
        const size_t o = sh * DK + n;
        s_k[n] = TI ? make_float4(0.f, 0.f, ld(k, o), ld(q, o)) : make_float4(ld(a, o), ld(p, o), ld(k, o), ld(q, o));
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
        const A rc[4] = {rr.x, rr.y, rr.z, rr.w};
        const A rv[4] = {(A)rr.x * vv.x, (A)rr.y * vv.y, (A)rr.z * vv.z, (A)rr.w * vv.w};
        A ya[4] = {0, 0, 0, 0}, wa[4] = {0, 0, 0, 0};
        float4* lam4 = reinterpret_cast<float4*>(g.lam + sh * DK * DV);
        float4* eta4 = reinterpret_cast<float4*>(g.eta + sh * DK * DV);
#pragma unroll 2
        for (int i = 0; i < NPER; ++i) {
            const int n = ng + NG * i;
            const float4 in = s_k[n];
            const A kz = in.z, qw = in.w;
            const float4 l4 = lam4[n * DV4 + d4], e4 = eta4[n * DV4 + d4];
            A lp[4] = {l4.x, l4.y, l4.z, l4.w}, ep[4] = {e4.x, e4.y, e4.z, e4.w};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                A ax = in.x, py = in.y;
                if constexpr (TI) {
                    const size_t og = ((size_t)(sh % H) * DK + n) * DV + 4 * d4 + j;
                    ou_gates(g.ou_a[og], g.ou_p[og], g.ou_d[og], ax, py);
                }
                const A den = fma(py, lp[j], ax * ax);
                const A num = fma(kz * kz * rc[j], den, lp[j]);
                const A R = rcpa(den * num);
                const A iden = num * R, ilam = den * (den * R);
                lp[j] = num * iden;
                ep[j] = fma(ax * iden, ep[j], kz * rv[j]);
                ya[j] = fma(qw, ep[j] * ilam, ya[j]);
                wa[j] = fma(qw * qw, ilam, wa[j]);
            }
            lam4[n * DV4 + d4] = make_float4((float)lp[0], (float)lp[1], (float)lp[2], (float)lp[3]);
            eta4[n * DV4 + d4] = make_float4((float)ep[0], (float)ep[1], (float)ep[2], (float)ep[3]);
        }
        s_y[ng][d4] = A4p<A>{ya[0], ya[1], ya[2], ya[3]};
        s_w[ng][d4] = A4p<A>{wa[0], wa[1], wa[2], wa[3]};
    }
    __syncthreads();
    for (int j = tid; j < DV4; j += 256) {
        A4p<A> ys = s_y[0][j], ws = s_w[0][j];
        for (int gi = 1; gi < NG; ++gi) {
            const A4p<A> y2 = s_y[gi][j], w2 = s_w[gi][j];
            ys.x += y2.x; ys.y += y2.y; ys.z += y2.z; ys.w += y2.w;
            ws.x += w2.x; ws.y += w2.y; ws.z += w2.z; ws.w += w2.w;
        }
        const size_t o = sh * DV + 4 * j;
        st(y, o, ys.x);
        st(y, o + 1, ys.y);
        st(y, o + 2, ys.z);
        st(y, o + 3, ys.w);
        if (g.yvar) {
            g.yvar[o] = (float)ws.x;
            g.yvar[o + 1] = (float)ws.y;
            g.yvar[o + 2] = (float)ws.z;
            g.yvar[o + 3] = (float)ws.w;
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
    static hipError_t run(const Shape& s, const FwdArgs& a, void* ck, hipStream_t st) {
        constexpr int CT = DV < 32 ? DV : 32;
        const dim3 grid((unsigned)(s.B * s.H * (DV / CT))), block(kNG * CT);
        auto* c = static_cast<typename acc<S>::type*>(ck);
        if (a.ou_a)
            hipLaunchKernelGGL((fwd_pc_kernel<S, DK, DV, true>), grid, block, 0, st, s, a, c);
        else
            hipLaunchKernelGGL((fwd_pc_kernel<S, DK, DV, false>), grid, block, 0, st, s, a, c);
        return hipGetLastError();
    }
};

// ----------------------------------------------------------------------------
// Backward.  One workgroup per (b, h, CB value channels: 32, 16 at dk = 128); LPC lanes per channel
// (32, or 16 at dk = 16), lane l owning key slots l % LPC + LPC i of channel
// l / LPC.  Segments of kCK tokens are taken last to first: stage the segment's
// inputs (fetched into registers one segment ahead), recompute lam and H of its
// tokens from the checkpoint into registers, then walk its tokens in reverse.
// Per token the channel sums (dv, dr) are completed by DPP over the LPC lanes of
// a channel; for the key-slot sums (dq, dk, dabar, dpbar) every channel writes
// its values to its own row of a double-buffered LDS slot, and after one barrier
// the rows are added in channel order and stored as this tile's part (no
// cross-lane shuffles, and the writes need no lane mask).
// At dk = 128 a lane's 4 elements keep 72 trajectory values in registers, so the
// workgroup takes 16 channels (2 waves per SIMD, room for them) instead of 32.
template <int DK, int DV, typename A = float>
struct PcLanes {
    static constexpr int LPC = DK < 32 ? DK : 32;
    static constexpr int NPER = DK / LPC;
    // fp64 arithmetic doubles the trajectory registers: 16 channels from dk = 64 on
    static constexpr int CBMAX = DK == 128 || (DK == 64 && sizeof(A) == 8) ? 16 : 32;
    static constexpr int CB = DV < CBMAX ? DV : CBMAX;
    static constexpr int NTHR = LPC * CB;
};

template <typename S, int DK, int DV, bool TI>
__global__ __launch_bounds__((PcLanes<DK, DV, typename acc<S>::type>::NTHR)) void bwd_pc_kernel(Shape s, BwdArgs g,
                                                                        const typename acc<S>::type* ck,
                                                                        float* kpart) {
    using T_ = typename storage<S>::type;
    using A = typename acc<S>::type;
    using PL = PcLanes<DK, DV, A>;
    constexpr int LPC = PL::LPC, NPER = PL::NPER;
    constexpr int CB = PL::CB;
    constexpr int NTHR = LPC * CB;
    static_assert(NTHR % 64 == 0 && (LPC == 16 || LPC == 32), "lane layout");
    __shared__ float4 s_k[kCK][DK];        // abar, pbar, k, q
    __shared__ float4 s_c[kCK][CB];        // r, v, dy, dyvar
    __shared__ float2 s_o[kCK][CB];        // dv, dr
    __shared__ float s_red[2][CB][4][DK];  // per-channel key-slot values of dq, dk, dabar, dpbar

    const T_ *q = static_cast<const T_*>(g.q), *k = static_cast<const T_*>(g.k), *v = static_cast<const T_*>(g.v);
    const T_ *a = static_cast<const T_*>(g.a), *p = static_cast<const T_*>(g.p), *r = static_cast<const T_*>(g.r);
    const T_* dy = static_cast<const T_*>(g.dy);
    T_* dv_out = static_cast<T_*>(g.dv);
    T_* dr_out = static_cast<T_*>(g.dr);
    const int ntile = DV / CB;
    const int bh = blockIdx.x / ntile, tile = blockIdx.x % ntile, d0 = tile * CB;
    const int b = bh / s.H, h = bh % s.H;
    const int tid = threadIdx.x;
    const int ln = tid % LPC, c = tid / LPC, d = d0 + c;
    const int T = s.T, nseg = (T + kCK - 1) / kCK;
    const size_t nck = (size_t)s.B * s.H * nseg * DK * DV;
    const size_t nkey = part_stride((size_t)s.B * T * s.H * DK);

    constexpr int NQ = TI ? 2 : 4;   // key-slot sums per token: dq, dk (, dabar, dpbar)
    A ge[NPER], gl[NPER], ga[NPER], gp[NPER], sum_da[NPER], sum_dp[NPER];
#pragma unroll
    for (int i = 0; i < NPER; ++i) {
        const size_t o = ((size_t)bh * DK + ln + LPC * i) * DV + d;
        ge[i] = g.detaT ? (A)g.detaT[o] : A(0);
        gl[i] = g.dlamT ? (A)g.dlamT[o] : A(0);
        sum_da[i] = sum_dp[i] = 0;
        if constexpr (TI) {
            const size_t og = ((size_t)h * DK + ln + LPC * i) * DV + d;
            ou_gates(g.ou_a[og], g.ou_p[og], g.ou_d[og], ga[i], gp[i]);
        }
    }
    // The inputs of a segment and its checkpoint are fetched into registers one segment
    // ahead (indices clamped to the segment's last token, so every load is issued) and
    // written to LDS at the start of the segment.
    constexpr int KPT = (kCK * DK + NTHR - 1) / NTHR, CPT = (kCK * CB + NTHR - 1) / NTHR;
    float4 nk[KPT], nc[CPT];
    A nl0[NPER], ne0[NPER];
    auto fetch = [&](int sg) {
        const int t0 = sg * kCK, tl = min(kCK, T - t0) - 1;
#pragma unroll
        for (int m = 0; m < KPT; ++m) {
            const int idx = min(tid + NTHR * m, kCK * DK - 1), t = min(idx / DK, tl), n = idx % DK;
            const size_t o = (((size_t)b * T + t0 + t) * s.H + h) * DK + n;
            nk[m] = TI ? make_float4(0.f, 0.f, ld(k, o), ld(q, o)) : make_float4(ld(a, o), ld(p, o), ld(k, o), ld(q, o));
        }
#pragma unroll
        for (int m = 0; m < CPT; ++m) {
            const int idx = min(tid + NTHR * m, kCK * CB - 1), t = min(idx / CB, tl), cc = idx % CB;
            const size_t o = (((size_t)b * T + t0 + t) * s.H + h) * DV + d0 + cc;
            nc[m] = make_float4(ld(r, o), ld(v, o), ld(dy, o), g.dyvar ? g.dyvar[o] : 0.f);
        }
#pragma unroll
        for (int i = 0; i < NPER; ++i) {
            const size_t o = (((size_t)bh * nseg + sg) * DK + ln + LPC * i) * DV + d;
            nl0[i] = ck[o];
            ne0[i] = ck[nck + o];
        }
    };
    wait_vm_all();   // the carries are complete before the segment loop
    if (nseg > 0) fetch(nseg - 1);
    for (int sg = nseg - 1; sg >= 0; --sg) {
        const int t0 = sg * kCK, nt = min(kCK, T - t0);
        barrier_lds();   // the previous segment's staging and outputs are no longer read
#pragma unroll
        for (int m = 0; m < KPT; ++m) {
            const int idx = tid + NTHR * m;
            if (KPT * NTHR == kCK * DK || idx < kCK * DK) s_k[idx / DK][idx % DK] = nk[m];
        }
#pragma unroll
        for (int m = 0; m < CPT; ++m) {
            const int idx = tid + NTHR * m;
            if (CPT * NTHR == kCK * CB || idx < kCK * CB) s_c[idx / CB][idx % CB] = nc[m];
        }
        // lam and H before each token of the segment and after its last
        A lt[kCK + 1][NPER], et[kCK + 1][NPER];
#pragma unroll
        for (int i = 0; i < NPER; ++i) {
            lt[0][i] = nl0[i];
            et[0][i] = ne0[i];
        }
        barrier_lds();   // the segment's inputs are in
        fetch(sg > 0 ? sg - 1 : 0);
#pragma unroll
        for (int j = 0; j < kCK; ++j) {
            const bool ok = j < nt;
            const float4 cv = s_c[ok ? j : 0][c];
            const A rc = cv.x, krv = (A)cv.x * (A)cv.y;
#pragma unroll
            for (int i = 0; i < NPER; ++i) {
                const float4 in = s_k[ok ? j : 0][ln + LPC * i];
                const A ax = TI ? ga[i] : (A)in.x, py = TI ? gp[i] : (A)in.y, kz = in.z;
                const A den = fma(py, lt[j][i], ax * ax);
                const A num = fma(kz * kz * rc, den, lt[j][i]);
                const A R = rcpa(den * num);
                const A iden = num * R;
                lt[j + 1][i] = ok ? num * iden : lt[j][i];
                et[j + 1][i] = ok ? fma(ax * iden, et[j][i], kz * krv) : et[j][i];
            }
        }
        // reverse over the segment's tokens
#pragma unroll
        for (int j = kCK - 1; j >= 0; --j) {
            if (j >= nt) continue;   // uniform: the tail of the last segment
            const float4 cv = s_c[j][c];   // r, v, gy, gv
            const A cr = cv.x, cvv = cv.y, gy = cv.z, gv = cv.w;
            float kq[4][NPER];             // this lane's dq, dk, dabar, dpbar of token j
            A cdv = 0, cdr = 0;
#pragma unroll
            for (int i = 0; i < NPER; ++i) {
                const float4 in = s_k[j][ln + LPC * i];   // abar, pbar, k, q
                const A av = TI ? ga[i] : (A)in.x, pv = TI ? gp[i] : (A)in.y, kv = in.z, qv = in.w;
                const A lp = lt[j][i], lc = lt[j + 1][i], ep = et[j][i], ec = et[j + 1][i];
                const A den = fma(pv, lp, av * av);
                const A R = rcpa(lc * den);
                const A ilc = den * R, rho = lc * R;
                const A mu = ec * ilc;
                const A qgy = qv * gy;
                kq[0][i] = (float)fma(mu, gy, A(2) * qv * gv * ilc);
                const A gei = fma(qgy, ilc, ge[i]);
                const A gli = gl[i] - fma(qgy, mu, qv * qv * gv * ilc) * ilc;
                const A df = gei * ep;
                const A kr = kv * cr;
                kq[1][i] = (float)fma(gei, cr * cvv, A(2) * gli * kr);
                cdr = fma(gei, kv * cvv, fma(gli, kv * kv, cdr));
                cdv = fma(gei, kr, cdv);
                const A drho = fma(df, av, gli * lp);
                const A dden = -drho * rho * rho;
                if constexpr (TI) {
                    sum_da[i] += fma(df, rho, A(2) * av * dden);
                    sum_dp[i] += dden * lp;
                } else {
                    kq[2][i] = (float)fma(df, rho, A(2) * av * dden);
                    kq[3][i] = (float)(dden * lp);
                }
                ge[i] = av * rho * gei;
                gl[i] = fma(gli, rho, pv * dden);
            }
            // channel sums over the LPC lanes of the channel
            if constexpr (LPC == 32) {
                cdv = half_sum(cdv);
                cdr = half_sum(cdr);
            } else {
                cdv += dpp<0xB1, 0xf>(cdv);
                cdv += dpp<0x4E, 0xf>(cdv);
                cdv += dpp<0x141, 0xf>(cdv);
                cdv += dpp<0x140, 0xf>(cdv);
                cdr += dpp<0xB1, 0xf>(cdr);
                cdr += dpp<0x4E, 0xf>(cdr);
                cdr += dpp<0x141, 0xf>(cdr);
                cdr += dpp<0x140, 0xf>(cdr);
            }
            if (ln == LPC - 1) s_o[j][c] = make_float2((float)cdv, (float)cdr);
            // key-slot sums over the channels of the workgroup: every channel's values go to
            // its own LDS row, summed in a fixed order after the barrier
            float* slot = &s_red[j & 1][c][0][0];
#pragma unroll
            for (int qi = 0; qi < NQ; ++qi)
#pragma unroll
                for (int i = 0; i < NPER; ++i) slot[qi * DK + ln + LPC * i] = kq[qi][i];
            barrier_lds();   // the channels' key-slot values of token j are in
            const size_t tk = ((size_t)b * T + t0 + j) * s.H + h;
            constexpr int RPT = (NQ * DK + NTHR - 1) / NTHR;
#pragma unroll
            for (int m = 0; m < RPT; ++m) {
                const int idx = tid + NTHR * m;
                if (RPT * NTHR != NQ * DK && idx >= NQ * DK) continue;
                float acc = 0.f;
#pragma unroll
                for (int cc = 0; cc < CB; ++cc) acc += (&s_red[j & 1][cc][0][0])[idx];
                const int qi = idx / DK, n = idx % DK;
                kpart[((size_t)tile * 4 + qi) * nkey + tk * DK + n] = acc;
            }
        }
        barrier_lds();   // the channel sums of the segment are in
        for (int idx = tid; idx < nt * CB; idx += NTHR) {
            const int t = idx / CB, cc = idx % CB;
            const size_t o = (((size_t)b * T + t0 + t) * s.H + h) * DV + d0 + cc;
            st(dv_out, o, s_o[t][cc].x);
            st(dr_out, o, s_o[t][cc].y);
        }
    }
#pragma unroll
    for (int i = 0; i < NPER; ++i) {
        const size_t o = ((size_t)bh * DK + ln + LPC * i) * DV + d;
        if (g.dlam0) g.dlam0[o] = (float)gl[i];
        if (g.deta0) g.deta0[o] = (float)ge[i];
        if constexpr (TI) {   // part b of the gate-gradient sums, [2][B][H][DK][DV]
            A* part = static_cast<A*>(g.ou_part);
            const size_t np = (size_t)s.B * s.H * DK * DV;
            part[o] = sum_da[i];
            part[np + o] = sum_dp[i];
        }
    }
}

// dq, dk, dabar, dpbar = sums of the NT channel tiles' parts (in tile order), in the
// input dtype.  A thread takes 4 consecutive elements (n is a multiple of 4; every
// array is 16-byte aligned) and issues all of its 4 NT part loads before the sums.
template <typename S, int NT, int NQ>
__global__ __launch_bounds__(256) void pc_key_combine_kernel(const float* __restrict__ kpart, size_t n, BwdArgs g) {
    const size_t i = ((size_t)blockIdx.x * blockDim.x + threadIdx.x) * 4, ns = part_stride(n);
    if (i >= n) return;
    void* out[4] = {g.dq, g.dk, g.da, g.dp};
    float4 x[NQ][NT];
#pragma unroll
    for (int qi = 0; qi < NQ; ++qi)
#pragma unroll
        for (int t = 0; t < NT; ++t) x[qi][t] = *reinterpret_cast<const float4*>(kpart + ((size_t)t * 4 + qi) * ns + i);
#pragma unroll
    for (int qi = 0; qi < NQ; ++qi) {
        float4 acc = x[qi][0];
#pragma unroll
        for (int t = 1; t < NT; ++t) {
            acc.x += x[qi][t].x;
            acc.y += x[qi][t].y;
            acc.z += x[qi][t].z;
            acc.w += x[qi][t].w;
        }
        if constexpr (std::is_same<S, bf16_t>::value)
            *reinterpret_cast<uint2*>(static_cast<uint16_t*>(out[qi]) + i) =
                make_uint2(cvt_pk_bf16(acc.x, acc.y), cvt_pk_bf16(acc.z, acc.w));
        else
            *reinterpret_cast<float4*>(static_cast<float*>(out[qi]) + i) = acc;
    }
}

template <typename S, int DK, int DV>
struct BwdPc {
    static hipError_t run(const Shape& s, const BwdArgs& a, const void* ck, float* kpart, hipStream_t st) {
        using PL = PcLanes<DK, DV, typename acc<S>::type>;
        constexpr int CB = PL::CB;
        constexpr int NTHR = PL::NTHR;
        const dim3 grid((unsigned)(s.B * s.H * (DV / CB))), block(NTHR);
        auto* c = static_cast<const typename acc<S>::type*>(ck);
        if (a.ou_a)
            hipLaunchKernelGGL((bwd_pc_kernel<S, DK, DV, true>), grid, block, 0, st, s, a, c, kpart);
        else
            hipLaunchKernelGGL((bwd_pc_kernel<S, DK, DV, false>), grid, block, 0, st, s, a, c, kpart);
        hipError_t e = hipGetLastError();
        const size_t n = (size_t)s.B * s.T * s.H * DK;   // dk is a multiple of 16, n of 4
        if (e != hipSuccess || n == 0) return e;
        constexpr int NT = DV / CB;
        static_assert(DK % 4 == 0 && (NT == 1 || NT == 2 || NT == 4 || NT == 8), "combine layout");
        const dim3 cgrid((unsigned)((n / 4 + 255) / 256));
        if (a.ou_a)   // the gate gradients went to the parameter parts
            hipLaunchKernelGGL((pc_key_combine_kernel<S, NT, 2>), cgrid, dim3(256), 0, st, kpart, n, a);
        else
            hipLaunchKernelGGL((pc_key_combine_kernel<S, NT, 4>), cgrid, dim3(256), 0, st, kpart, n, a);
        return hipGetLastError();
    }
};

template <typename S, int DK, int DV>
struct DecPc {
    static hipError_t run(const Shape& s, const DecodeArgs& a, hipStream_t st) {
        if (a.ou_a)
            hipLaunchKernelGGL((decode_pc_kernel<S, DK, DV, true>), dim3((unsigned)(s.B * s.H)), dim3(256), 0, st,
                               s.H, a);
        else
            hipLaunchKernelGGL((decode_pc_kernel<S, DK, DV, false>), dim3((unsigned)(s.B * s.H)), dim3(256), 0, st,
                               s.H, a);
        return hipGetLastError();
    }
};

}  // namespace

hipError_t launch_forward_pc(const Shape& s, const FwdArgs& a, void* ck, hipStream_t st) {
    return dispatch_pc<FwdPc>(s, a, ck, st);
}

size_t pc_saved_bytes(const Shape& s) {
    const size_t nseg = (size_t)(s.T + kCK - 1) / kCK;
    return 2 * (size_t)s.B * s.H * nseg * s.dk * s.dv * (s.bf16 ? sizeof(float) : sizeof(double));
}

// the per-batch-row parts of the gate-gradient sums of the OU entry points: [2][B][H][dk][dv]
size_t pc_ou_part_bytes(const Shape& s) {
    return 2 * (size_t)s.B * s.H * s.dk * s.dv * (s.bf16 ? sizeof(float) : sizeof(double));
}

size_t pc_bwd_workspace(const Shape& s) {
    const int cbmax = s.dk == 128 || (s.dk == 64 && !s.bf16) ? 16 : 32;   // as PcLanes
    const int cb = s.dv < cbmax ? s.dv : cbmax;
    return (size_t)(s.dv / cb) * 4 * part_stride((size_t)s.B * s.T * s.H * s.dk) * sizeof(float);
}

hipError_t launch_backward_pc(const Shape& s, const BwdArgs& a, const void* ck, float* kpart, hipStream_t st) {
    return dispatch_pc<BwdPc>(s, a, ck, kpart, st);
}

hipError_t launch_decode_pc(const Shape& s, const DecodeArgs& a, hipStream_t st) {
    return dispatch_pc<DecPc>(s, a, st);
}

}  // namespace kla
