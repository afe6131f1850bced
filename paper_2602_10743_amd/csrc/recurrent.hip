// Token-recurrent KLA kernels: forward, backward (two sweeps) and the decode step.
//
// These walk the filter one token at a time (Theorem 1 gate view for the
// precision, Theorem 2 for the information state, Algorithm 1 readout), with
// the d_k x d_v state held in registers across the token loop.  They are the
// reference HIP path of the library and the decode step's implementation.
// With OU parameters (ou_a set) every token of a head shares the gates of its
// key slot, formed once per lane; the backward then sums the gate gradients of
// a lane over its tokens into one part per batch row.
#include "kla_device.hpp"
#include "kla_internal.hpp"

namespace kla {
namespace {

constexpr int kThreads = 256;
constexpr int kTB = 16;  // tokens per LDS block in the forward

// ----------------------------------------------------------------------------
// Forward.  One workgroup per (b, h, value tile of DVT channels).  Threads
// tid < DK own the precision lane n = tid; every thread owns H[n, d] for
// n = ng + i*NG and one channel d = d0 + dl.
template <typename S, int DK, int DV>
__global__ __launch_bounds__(kThreads) void fwd_recurrent_kernel(Shape s, FwdArgs g) {
    using T_ = typename storage<S>::type;
    constexpr int DVT = DV < 32 ? DV : 32;
    constexpr int NTILE = DV / DVT;
    constexpr int NG = kThreads / DVT;
    constexpr int NPER = DK / NG > 0 ? DK / NG : 1;
    static_assert(DK % NG == 0 || NG > DK, "key width must be a multiple of the n-groups");

    __shared__ float sF[kTB][DK], sKh[kTB][DK], sQt[kTB][DK], sW[kTB][DK];
    __shared__ float sRed[kTB][NG][DVT];

    const T_* q = static_cast<const T_*>(g.q);
    const T_* k = static_cast<const T_*>(g.k);
    const T_* v = static_cast<const T_*>(g.v);
    const T_* a = static_cast<const T_*>(g.a);
    const T_* p = static_cast<const T_*>(g.p);
    const T_* r = static_cast<const T_*>(g.r);
    T_* y = static_cast<T_*>(g.y);

    const int tile = blockIdx.x % NTILE;
    const int bh = blockIdx.x / NTILE;
    const int b = bh / s.H, h = bh % s.H;
    const int tid = threadIdx.x;
    const int dl = tid % DVT, ng = tid / DVT;
    const int d = tile * DVT + dl;
    const bool owns = ng < DK;  // with NG > DK some n-groups are idle

    float Hs[NPER];
#pragma unroll
    for (int i = 0; i < NPER; ++i) {
        int n = ng + i * NG;
        Hs[i] = (owns && g.eta0) ? g.eta0[((size_t)bh * DK + n) * DV + d] : 0.f;
    }
    float lam = 1.f;
    if (tid < DK && g.lam0) lam = g.lam0[(size_t)bh * DK + tid];
    const bool ou = g.ou_a != nullptr;
    float oa = 0.f, op = 0.f;
    if (ou && tid < DK) ou_gates(g.ou_a[h * DK + tid], g.ou_p[h * DK + tid], g.ou_d[h * DK + tid], oa, op);

    for (int t0 = 0; t0 < s.T; t0 += kTB) {
        const int nt = min(kTB, s.T - t0);
        if (tid < DK) {
            for (int j = 0; j < nt; ++j) {
                const size_t base = ((size_t)b * s.T + t0 + j) * s.H + h;
                const float at = ou ? oa : ld(a, base * DK + tid), pt = ou ? op : ld(p, base * DK + tid);
                const float kt = ld(k, base * DK + tid), qt = ld(q, base * DK + tid);
                const float rt = ld(r, base);
                const float rho = 1.f / (at * at + pt * lam);
                sF[j][tid] = at * rho;
                lam = rho * lam + kt * kt * rt;
                const float inv = 1.f / lam;
                sKh[j][tid] = rt * kt;
                sQt[j][tid] = qt * inv;
                sW[j][tid] = qt * qt * inv;
            }
        }
        __syncthreads();
        for (int j = 0; j < nt; ++j) {
            const size_t base = ((size_t)b * s.T + t0 + j) * s.H + h;
            const float vd = ld(v, base * DV + d);
            float acc = 0.f;
#pragma unroll
            for (int i = 0; i < NPER; ++i) {
                const int n = ng + i * NG;
                if (owns) {
                    Hs[i] = sF[j][n] * Hs[i] + sKh[j][n] * vd;
                    acc += sQt[j][n] * Hs[i];
                }
            }
            sRed[j][ng][dl] = acc;
        }
        __syncthreads();
        for (int idx = tid; idx < nt * DVT; idx += kThreads) {
            const int j = idx / DVT, dd = idx % DVT;
            float acc = 0.f;
            for (int gi = 0; gi < NG; ++gi) acc += sRed[j][gi][dd];
            const size_t base = ((size_t)b * s.T + t0 + j) * s.H + h;
            st(y, base * DV + tile * DVT + dd, acc);
        }
        if (tile == 0 && g.yvar && tid >= kThreads - kTB && tid - (kThreads - kTB) < nt) {
            const int j = tid - (kThreads - kTB);
            float acc = 0.f;
            for (int n = 0; n < DK; ++n) acc += sW[j][n];
            g.yvar[((size_t)b * s.T + t0 + j) * s.H + h] = acc;
        }
        __syncthreads();
    }
    if (tile == 0 && g.lamT && tid < DK) g.lamT[(size_t)bh * DK + tid] = lam;
    if (g.etaT && owns) {
#pragma unroll
        for (int i = 0; i < NPER; ++i) g.etaT[((size_t)bh * DK + ng + i * NG) * DV + d] = Hs[i];
    }
}

// ----------------------------------------------------------------------------
// Backward, sweep 1 (forward in time).  Re-runs the filter and stores the
// precision trajectory lam_t and dqt_t = H_t dy_t (the gradient of the
// effective query q/lam_t), plus PT[n] = sum_d detaT[n,d] H_T[n,d].
// One workgroup per (b, h, 16 key slots); 16 lanes split the value channels.
template <typename S, int DK, int DV>
__global__ __launch_bounds__(kThreads) void bwd_sweep1_kernel(Shape s, BwdArgs g, float* wlam,
                                                               float* wdqt, float* wPT) {
    using T_ = typename storage<S>::type;
    constexpr int NT = 16, DL = 16, DPER = DV / DL;
    const T_* k = static_cast<const T_*>(g.k);
    const T_* v = static_cast<const T_*>(g.v);
    const T_* a = static_cast<const T_*>(g.a);
    const T_* p = static_cast<const T_*>(g.p);
    const T_* r = static_cast<const T_*>(g.r);
    const T_* dy = static_cast<const T_*>(g.dy);

    const int ntile = DK / NT;
    const int bh = blockIdx.x / ntile, nt = blockIdx.x % ntile;
    const int b = bh / s.H, h = bh % s.H;
    const int tid = threadIdx.x;
    const int n = nt * NT + tid / DL, dl = tid % DL;

    float Hs[DPER];
#pragma unroll
    for (int i = 0; i < DPER; ++i)
        Hs[i] = g.eta0 ? g.eta0[((size_t)bh * DK + n) * DV + dl + i * DL] : 0.f;
    float lam = g.lam0 ? g.lam0[(size_t)bh * DK + n] : 1.f;
    const bool ou = g.ou_a != nullptr;
    float oa = 0.f, op = 0.f;
    if (ou) ou_gates(g.ou_a[h * DK + n], g.ou_p[h * DK + n], g.ou_d[h * DK + n], oa, op);

    for (int t = 0; t < s.T; ++t) {
        const size_t base = ((size_t)b * s.T + t) * s.H + h;
        const float at = ou ? oa : ld(a, base * DK + n), pt = ou ? op : ld(p, base * DK + n);
        const float kt = ld(k, base * DK + n);
        const float rt = ld(r, base);
        const float rho = 1.f / (at * at + pt * lam);
        const float F = at * rho, kh = rt * kt;
        lam = rho * lam + kt * kt * rt;
        float acc = 0.f;
#pragma unroll
        for (int i = 0; i < DPER; ++i) {
            const size_t o = base * DV + dl + i * DL;
            Hs[i] = F * Hs[i] + kh * ld(v, o);
            acc += Hs[i] * ld(dy, o);
        }
#pragma unroll
        for (int off = DL / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off, DL);
        if (dl == 0) {
            wlam[base * DK + n] = lam;
            wdqt[base * DK + n] = acc;
        }
    }
    float acc = 0.f;
    if (g.detaT) {
#pragma unroll
        for (int i = 0; i < DPER; ++i) acc += g.detaT[((size_t)bh * DK + n) * DV + dl + i * DL] * Hs[i];
    }
#pragma unroll
    for (int off = DL / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off, DL);
    if (dl == 0) wPT[(size_t)bh * DK + n] = acc;
}

// ----------------------------------------------------------------------------
// Backward, sweep 2 (reverse in time), one workgroup per (b, h) holding the
// whole adjoint state dH.  Per token, with dG_t the adjoint of log F_t and
// g_t the adjoint of lam_t:
//   dH_t   = F_{t+1} dH_{t+1} + qt_t dy_t^T          (dH_T starts at detaT)
//   dkh_t  = dH_t v_t,  dv_t = dH_t^T kh_t
//   dG_t   = PT + sum_{s>=t} (qt_s dqt_s - kh_s dkh_s)
//   g_t    = c_t - q_t (dqt_t + q_t gv_t) / lam_t^2,  c_T = dlamT,
//            (gv_t: upstream gradient of the readout variance, zero if none)
//   c_{t-1}= abar_t^2 rho_t^2 g_t - pbar_t rho_t dG_t
// and the input gradients follow by the chain rule through rho, lam and F.
template <typename S, int DK, int DV>
__global__ __launch_bounds__(kThreads) void bwd_sweep2_kernel(Shape s, BwdArgs g, const float* wlam,
                                                               const float* wdqt, const float* wPT) {
    using T_ = typename storage<S>::type;
    constexpr int DVT = DV < 32 ? DV : 32;
    constexpr int NG = kThreads / DVT;
    constexpr int NPER = DK / NG > 0 ? DK / NG : 1;
    constexpr int DPER = DV / DVT;
    __shared__ float sQt[DK], sKh[DK], sFn[DK], sV[DV], sDy[DV], sDR[DK];
    __shared__ float sPK[DK][DVT + 1];
    __shared__ float sPV[NG][DV];

    const T_* q = static_cast<const T_*>(g.q);
    const T_* k = static_cast<const T_*>(g.k);
    const T_* v = static_cast<const T_*>(g.v);
    const T_* a = static_cast<const T_*>(g.a);
    const T_* p = static_cast<const T_*>(g.p);
    const T_* r = static_cast<const T_*>(g.r);
    const T_* dy = static_cast<const T_*>(g.dy);
    T_* dq = static_cast<T_*>(g.dq);
    T_* dk = static_cast<T_*>(g.dk);
    T_* dv = static_cast<T_*>(g.dv);
    T_* da = static_cast<T_*>(g.da);
    T_* dp = static_cast<T_*>(g.dp);
    T_* dr = static_cast<T_*>(g.dr);

    const int bh = blockIdx.x;
    const int b = bh / s.H, h = bh % s.H;
    const int tid = threadIdx.x;
    const int dl = tid % DVT, ng = tid / DVT;
    const bool owns = ng < DK;

    float dH[NPER][DPER];
#pragma unroll
    for (int i = 0; i < NPER; ++i)
#pragma unroll
        for (int j = 0; j < DPER; ++j)
            dH[i][j] = (owns && g.detaT) ? g.detaT[((size_t)bh * DK + ng + i * NG) * DV + dl + j * DVT] : 0.f;

    // per-slot scalars, live in threads tid < DK
    float Fnext = 1.f, cnext = 0.f, Sg = 0.f;
    const bool ou = g.ou_a != nullptr;
    float oa = 0.f, op = 0.f, sum_da = 0.f, sum_dp = 0.f;
    if (tid < DK) {
        cnext = g.dlamT ? g.dlamT[(size_t)bh * DK + tid] : 0.f;
        Sg = wPT[(size_t)bh * DK + tid];
        if (ou) ou_gates(g.ou_a[h * DK + tid], g.ou_p[h * DK + tid], g.ou_d[h * DK + tid], oa, op);
    }

    for (int t = s.T - 1; t >= 0; --t) {
        const size_t base = ((size_t)b * s.T + t) * s.H + h;
        float lam_t = 0.f, dqt = 0.f, qt = 0.f, kt = 0.f, rt = 0.f;
        if (tid < DK) {
            lam_t = wlam[base * DK + tid];
            dqt = wdqt[base * DK + tid];
            qt = ld(q, base * DK + tid);
            kt = ld(k, base * DK + tid);
            rt = ld(r, base);
            sQt[tid] = qt / lam_t;
            sKh[tid] = rt * kt;
            sFn[tid] = Fnext;
        }
        for (int i = tid; i < DV; i += kThreads) {
            sV[i] = ld(v, base * DV + i);
            sDy[i] = ld(dy, base * DV + i);
        }
        __syncthreads();
        float pv[DPER];
#pragma unroll
        for (int j = 0; j < DPER; ++j) pv[j] = 0.f;
#pragma unroll
        for (int i = 0; i < NPER; ++i) {
            const int n = ng + i * NG;
            if (!owns) break;
            float pk = 0.f;
#pragma unroll
            for (int j = 0; j < DPER; ++j) {
                const int dd = dl + j * DVT;
                dH[i][j] = sFn[n] * dH[i][j] + sQt[n] * sDy[dd];
                pk += dH[i][j] * sV[dd];
                pv[j] += dH[i][j] * sKh[n];
            }
            sPK[n][dl] = pk;
        }
#pragma unroll
        for (int j = 0; j < DPER; ++j) sPV[ng][dl + j * DVT] = pv[j];
        __syncthreads();
        if (tid < DK) {
            float dkh = 0.f;
            for (int i = 0; i < DVT; ++i) dkh += sPK[tid][i];
            const float at = ou ? oa : ld(a, base * DK + tid), pt = ou ? op : ld(p, base * DK + tid);
            const float lprev = t > 0 ? wlam[(base - s.H) * DK + tid] : (g.lam0 ? g.lam0[(size_t)bh * DK + tid] : 1.f);
            const float qtl = sQt[tid], kh = sKh[tid];
            const float qg = g.dyvar ? qt * g.dyvar[base] : 0.f;
            Sg += qtl * dqt - kh * dkh;                       // dG_t
            const float rho = 1.f / (at * at + pt * lprev);
            const float gl = cnext - qt * (dqt + qg) / (lam_t * lam_t);  // g_t
            const float drho = gl * lprev + Sg / rho;
            st(dq, base * DK + tid, (dqt + 2.f * qg) / lam_t);
            st(dk, base * DK + tid, rt * dkh + 2.f * kt * rt * gl);
            const float dav = Sg / at - 2.f * at * rho * rho * drho, dpv = -lprev * rho * rho * drho;
            if (ou) {
                sum_da += dav;
                sum_dp += dpv;
            } else {
                st(da, base * DK + tid, dav);
                st(dp, base * DK + tid, dpv);
            }
            sDR[tid] = kt * dkh + kt * kt * gl;
            cnext = at * at * rho * rho * gl - pt * rho * Sg;
            Fnext = at * rho;
        }
        if (tid < DV) {
            float acc = 0.f;
            for (int gi = 0; gi < NG && gi < DK; ++gi) acc += sPV[gi][tid];
            st(dv, base * DV + tid, acc);
        }
        __syncthreads();
        if (tid == 0) {
            float acc = 0.f;
            for (int n = 0; n < DK; ++n) acc += sDR[n];
            st(dr, base, acc);
        }
    }
    if (tid < DK && g.dlam0) g.dlam0[(size_t)bh * DK + tid] = cnext;
    if (ou && tid < DK) {   // part b of the token sums
        const size_t np = (size_t)s.B * s.H * DK;
        g.ou_part[(size_t)bh * DK + tid] = sum_da;
        g.ou_part[np + (size_t)bh * DK + tid] = sum_dp;
    }
    __syncthreads();
    if (tid < DK) sFn[tid] = Fnext;
    __syncthreads();
    if (g.deta0 && owns) {
#pragma unroll
        for (int i = 0; i < NPER; ++i)
#pragma unroll
            for (int j = 0; j < DPER; ++j) {
                const int n = ng + i * NG;
                g.deta0[((size_t)bh * DK + n) * DV + dl + j * DVT] = sFn[n] * dH[i][j];
            }
    }
}

// ----------------------------------------------------------------------------
// Decode: one token for S sequences, belief updated in place.  One workgroup
// per (sequence, head); the eta rows are streamed with 16-byte accesses.
template <typename S, int DK, int DV>
__global__ __launch_bounds__(kThreads) void decode_kernel(int H, DecodeArgs g) {
    using T_ = typename storage<S>::type;
    constexpr int DV4 = DV / 4;
    constexpr int NG = (kThreads / DV4) < DK ? (kThreads / DV4) : DK;
    constexpr int NPER = DK / NG;
    __shared__ float sF[DK], sKh[DK], sQt[DK], sW[DK], sV[DV];
    __shared__ float4 sRed[NG][DV4];

    const T_* q = static_cast<const T_*>(g.q);
    const T_* k = static_cast<const T_*>(g.k);
    const T_* v = static_cast<const T_*>(g.v);
    const T_* a = static_cast<const T_*>(g.a);
    const T_* p = static_cast<const T_*>(g.p);
    const T_* r = static_cast<const T_*>(g.r);
    T_* y = static_cast<T_*>(g.y);

    const size_t sh = blockIdx.x;
    const int tid = threadIdx.x;
    if (tid < DK) {
        const size_t o = sh * DK + tid;
        float at, pt;
        if (g.ou_a) {
            const int oh = (int)(sh % H) * DK + tid;
            ou_gates(g.ou_a[oh], g.ou_p[oh], g.ou_d[oh], at, pt);
        } else {
            at = ld(a, o);
            pt = ld(p, o);
        }
        const float kt = ld(k, o), qt = ld(q, o), rt = ld(r, sh);
        const float lam = g.lam[o];
        const float rho = 1.f / (at * at + pt * lam);
        const float ln = rho * lam + kt * kt * rt;
        g.lam[o] = ln;
        const float inv = 1.f / ln;
        sF[tid] = at * rho;
        sKh[tid] = rt * kt;
        sQt[tid] = qt * inv;
        sW[tid] = qt * qt * inv;
    }
    for (int i = tid; i < DV; i += kThreads) sV[i] = ld(v, sh * DV + i);
    __syncthreads();
    const int d4 = tid % DV4, ng = tid / DV4;
    if (ng < NG) {
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        const float4 vv = make_float4(sV[4 * d4], sV[4 * d4 + 1], sV[4 * d4 + 2], sV[4 * d4 + 3]);
        float4* eta4 = reinterpret_cast<float4*>(g.eta + sh * DK * DV);
#pragma unroll 4
        for (int i = 0; i < NPER; ++i) {
            const int n = ng + i * NG;
            float4 e = eta4[n * DV4 + d4];
            const float F = sF[n], kh = sKh[n], qt = sQt[n];
            e.x = F * e.x + kh * vv.x;
            e.y = F * e.y + kh * vv.y;
            e.z = F * e.z + kh * vv.z;
            e.w = F * e.w + kh * vv.w;
            eta4[n * DV4 + d4] = e;
            acc.x += qt * e.x;
            acc.y += qt * e.y;
            acc.z += qt * e.z;
            acc.w += qt * e.w;
        }
        sRed[ng][d4] = acc;
    }
    __syncthreads();
    if (tid < DV4) {
        float4 acc = sRed[0][tid];
        for (int gi = 1; gi < NG; ++gi) {
            const float4 x = sRed[gi][tid];
            acc.x += x.x;
            acc.y += x.y;
            acc.z += x.z;
            acc.w += x.w;
        }
        st(y, sh * DV + 4 * tid + 0, acc.x);
        st(y, sh * DV + 4 * tid + 1, acc.y);
        st(y, sh * DV + 4 * tid + 2, acc.z);
        st(y, sh * DV + 4 * tid + 3, acc.w);
    }
    if (g.yvar && tid == kThreads - 1) {
        float acc = 0.f;
        for (int n = 0; n < DK; ++n) acc += sW[n];
        g.yvar[sh] = acc;
    }
}

// ----------------------------------------------------------------------------
// (dk, dv) dispatch over {16, 32, 64, 128}^2 and the storage type.
template <template <typename, int, int> class L, typename... A>
hipError_t dispatch(const Shape& s, A&&... args) {
#define KLA_CASE(DK_, DV_)                                                              \
    if (s.dk == DK_ && s.dv == DV_)                                                     \
        return s.bf16 ? L<bf16_t, DK_, DV_>::run(s, args...) : L<f32_t, DK_, DV_>::run(s, args...);
#define KLA_ROW(DK_) KLA_CASE(DK_, 16) KLA_CASE(DK_, 32) KLA_CASE(DK_, 64) KLA_CASE(DK_, 128)
    KLA_ROW(16) KLA_ROW(32) KLA_ROW(64) KLA_ROW(128)
#undef KLA_ROW
#undef KLA_CASE
    return hipErrorInvalidValue;
}

template <typename S, int DK, int DV>
struct FwdL {
    static hipError_t run(const Shape& s, const FwdArgs& a, hipStream_t st) {
        constexpr int DVT = DV < 32 ? DV : 32;
        const unsigned grid = (unsigned)(s.B * s.H * (DV / DVT));
        hipLaunchKernelGGL((fwd_recurrent_kernel<S, DK, DV>), dim3(grid), dim3(kThreads), 0, st, s, a);
        return hipGetLastError();
    }
};

template <typename S, int DK, int DV>
struct BwdL {
    static hipError_t run(const Shape& s, const BwdArgs& a, void* ws, hipStream_t st) {
        const size_t ntok = (size_t)s.B * s.T * s.H * DK;
        float* wlam = static_cast<float*>(ws);
        float* wdqt = wlam + ntok;
        float* wPT = wdqt + ntok;
        hipLaunchKernelGGL((bwd_sweep1_kernel<S, DK, DV>), dim3(s.B * s.H * (DK / 16)), dim3(kThreads), 0, st,
                           s, a, wlam, wdqt, wPT);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL((bwd_sweep2_kernel<S, DK, DV>), dim3(s.B * s.H), dim3(kThreads), 0, st, s, a,
                           wlam, wdqt, wPT);
        return hipGetLastError();
    }
};

template <typename S, int DK, int DV>
struct DecL {
    static hipError_t run(const Shape& s, const DecodeArgs& a, hipStream_t st) {
        hipLaunchKernelGGL((decode_kernel<S, DK, DV>), dim3(s.B * s.H), dim3(kThreads), 0, st, s.H, a);
        return hipGetLastError();
    }
};

}  // namespace

hipError_t launch_forward_recurrent(const Shape& s, const FwdArgs& a, hipStream_t st) {
    return dispatch<FwdL>(s, a, st);
}

// one part per batch row: the recurrent backward walks a whole (b, h) in one workgroup
int recurrent_ou_parts(const Shape& s) { return s.B; }

size_t backward_recurrent_workspace(const Shape& s) {
    const size_t ntok = (size_t)s.B * s.T * s.H * s.dk;
    return (2 * ntok + (size_t)s.B * s.H * s.dk) * sizeof(float);
}

hipError_t launch_backward_recurrent(const Shape& s, const BwdArgs& a, void* ws, hipStream_t st) {
    return dispatch<BwdL>(s, a, ws, st);
}

hipError_t launch_decode_step(const Shape& s, const DecodeArgs& a, hipStream_t st) {
    return dispatch<DecL>(s, a, st);
}

}  // namespace kla
