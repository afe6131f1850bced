// Chunked backward of the KLA filter on MFMA (bf16 inputs, fp32 state).
//
// Notation per chunk of kC tokens (local t), with the precision walk redone
// from the saved chunk-start precision (see kla_scan.hpp for P, Qp, Kn):
//   H_t  = P_t (H0 + sum_{j<=t} Kn_j v_j^T)            (state, per key slot row)
//   G    = adjoint of the chunk's last state coming from later tokens
//          (detaT for the last chunk), Gs = diag(P_C) G
//   B    = dY V^T                                      (C x C)
//   A    = Qp Kn^T                                     (C x C, the forward attention)
// then, with M() keeping j <= t,
//   X    = dY H0^T + M(B) Kn     dqt = P * X   (gradient of q / lam_t)
//   Y    = M(B)^T Qp + V Gs^T    dkh = Y / P   (gradient of r k)
//   dV   = M(A)^T dY + Kn Gs
//   G'   = Qp^T dY + Gs                            (carry into the previous chunk)
// The adjoint of log F_t is the reverse running sum of qt*dqt - kh*dkh (plus
// the final-state term sum_d detaT H_T), and the adjoint g_t of lam_t follows
//   g_t = c_t - q_t dqt_t / lam_t^2,  c_T = dlamT,
//   c_{t-1} = abar_t^2 rho_t^2 g_t - pbar_t rho_t dlogF_t,
// from which the input gradients follow by the chain rule through rho, lam, F.
//
// (dv and deta0 come from the value-side kernel in chunk_bwd_dv.hip.)
// Kernel B2: one workgroup per (b, h, 64 key slots); walks chunks in reverse
//   keeping G^T[dv, 64] in registers; reads the saved chunk-start states H0;
//   writes dq, dk, dabar, dpbar, partial dr sums over its key slots and dlam0.
#include "kla_internal.hpp"
#include "kla_mfma.hpp"
#include "kla_scan.hpp"

namespace kla {
namespace {

constexpr int kC = 64;
constexpr int kThr = 256;

__device__ __forceinline__ void xcd_map(int i, int nbh, int ntile, int& bh, int& tile) {
    if (nbh % 8 == 0) {
        const int xcd = i % 8, slot = i / 8;
        tile = slot % ntile;
        bh = (slot / ntile) * 8 + xcd;
    } else {
        tile = i % ntile;
        bh = i / ntile;
    }
}

// ============================================================================ B2
template <int DK, int DV>
struct B2Cfg {
    static constexpr int NTN = DK < 64 ? DK : 64;   // key slots per workgroup
    static constexpr int NNT = DK / NTN;
    static constexpr int NCW = NTN / 16;            // waves owning 16 key-slot columns
    static constexpr int NRD = DV / 16;
    static constexpr int KSD = DV / 32;
    static constexpr int LD = DV + 8, LT = kC + 8, LS = NTN + 4;
    static constexpr int DY = 0, V = DY + kC * LD, DYT = V + kC * LD;
    static constexpr int BH = DYT + DV * LT, BL = BH + kC * LT, BTH = BL + kC * LT, BTL = BTH + kC * LT;
    static constexpr int QTH = BTL + kC * LT, QTL = QTH + NTN * LT, KTH = QTL + NTN * LT, KTL = KTH + NTN * LT;
    static constexpr int END16 = KTL + NTN * LT;
    // fp32 regions (float indices); X and Y alias the B / B^T buffers once those are consumed
    static constexpr int LAM = (END16 + 7) / 8 * 4, PP = LAM + kC * LS, DECAY = PP + kC * LS;
    // per-quarter affine summaries [4][4][NTN] alias the dY tile, dead by then
    static constexpr int QS = DY / 2;
    static constexpr int X = BH / 2, Y = X + kC * LS;
    static constexpr size_t BYTES = (size_t)(DECAY + NTN) * 4;
    static_assert((size_t)2 * kC * LS * 4 <= (size_t)4 * kC * LT * 2, "X/Y must fit in the B buffers");
    static_assert((size_t)16 * NTN * 4 <= (size_t)kC * LD * 2, "quarter summaries must fit in the dY tile");
    static_assert(BYTES <= 160 * 1024, "LDS budget of one workgroup");
    static_assert(BH % 8 == 0, "alignment");
};

template <int DK, int DV>
__global__ __launch_bounds__(kThr) void bwd_b2_kernel(Shape s, BwdArgs g, const float* __restrict__ saved_lam,
                                                       const float* __restrict__ saved_H, float* __restrict__ dr_part) {
    using Cfg = B2Cfg<DK, DV>;
    constexpr int NTN = Cfg::NTN, NCW = Cfg::NCW, NRD = Cfg::NRD, KSD = Cfg::KSD;
    constexpr int LD = Cfg::LD, LT = Cfg::LT, LS = Cfg::LS;
    extern __shared__ __align__(16) unsigned char smem_raw[];
    uint16_t* sm = reinterpret_cast<uint16_t*>(smem_raw);
    float* smf = reinterpret_cast<float*>(smem_raw);

    const uint16_t* q = static_cast<const uint16_t*>(g.q);
    const uint16_t* k = static_cast<const uint16_t*>(g.k);
    const uint16_t* v = static_cast<const uint16_t*>(g.v);
    const uint16_t* a = static_cast<const uint16_t*>(g.a);
    const uint16_t* p = static_cast<const uint16_t*>(g.p);
    const uint16_t* r = static_cast<const uint16_t*>(g.r);
    const uint16_t* dy = static_cast<const uint16_t*>(g.dy);
    uint16_t* dq = static_cast<uint16_t*>(g.dq);
    uint16_t* dk = static_cast<uint16_t*>(g.dk);
    uint16_t* da = static_cast<uint16_t*>(g.da);
    uint16_t* dp = static_cast<uint16_t*>(g.dp);

    int bh, ntile;
    xcd_map(blockIdx.x, s.B * s.H, Cfg::NNT, bh, ntile);
    const int b = bh / s.H, h = bh % s.H;
    const int n0 = ntile * NTN;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l16 = lane & 15, g4 = lane >> 4;
    const int T = s.T;
    const int nchunk = (T + kC - 1) / kC;
    const int nchunk32 = (T + 31) / 32;   // the saved lam is kept per 32-token chunk
    const size_t nbt = (size_t)s.B * T * s.H;
    const bool owns = wave < NCW;
    const int ncl = 16 * wave + l16;            // local key-slot column of this lane
    const int ncol = n0 + ncl;

    // G^T[d, n] for this wave's 16 key slots, all value channels
    f32x4 GT[NRD];
#pragma unroll
    for (int rd = 0; rd < NRD; ++rd)
#pragma unroll
        for (int rr = 0; rr < 4; ++rr)
            GT[rd][rr] = (owns && g.detaT) ? g.detaT[((size_t)bh * DK + ncol) * DV + 16 * rd + 4 * g4 + rr] : 0.f;

    // per-slot carries of the reverse recursions, kept (identically) by lane nl of every wave
    const bool glane = lane < NTN;
    const int nl = glane ? lane : 0;
    const int ng = n0 + nl;
    float cnext = 0.f, Sg = 0.f;
    if (glane) {
        cnext = g.dlamT ? g.dlamT[(size_t)bh * DK + ng] : 0.f;
        if (g.detaT) {
            const float* HT = saved_H + (((size_t)bh * (nchunk + 1) + nchunk) * DK + ng) * DV;
            const float* dT = g.detaT + ((size_t)bh * DK + ng) * DV;
            for (int d = 0; d < DV; ++d) Sg += dT[d] * HT[d];
        }
    }
    const bool scan_lane = tid < NTN;

    // the previous chunk's dY / V tiles, first scan inputs and saved state rows are
    // in flight while a chunk is processed
    TileStage<kC, DV, kThr> ystage, vstage;
    ScanPrefetch<4> spre;
    float4 h0pre[KSD][2];
    auto load_h0 = [&](int cc) {
        const float* H0 = saved_H + (((size_t)bh * (nchunk + 1) + cc) * DK + ncol) * DV;
#pragma unroll
        for (int ks = 0; ks < KSD; ++ks) {
            h0pre[ks][0] = *reinterpret_cast<const float4*>(H0 + 32 * ks + 8 * g4);
            h0pre[ks][1] = *reinterpret_cast<const float4*>(H0 + 32 * ks + 8 * g4 + 4);
        }
    };
    if (nchunk > 0) {
        const int cl = nchunk - 1;
        const size_t r0 = (size_t)b * T + (size_t)cl * kC;
        const int ntl = T - cl * kC;
        ystage.load(dy, r0, s.H, h, DV, 0, ntl, tid);
        vstage.load(v, r0, s.H, h, DV, 0, ntl, tid);
        if (wave == 0) scan_prefetch<4>(spre, a, p, k, q, r, r0, s.H, h, DK, scan_lane ? n0 + tid : n0, ntl);
        if (owns) load_h0(cl);
    }

    for (int c = nchunk - 1; c >= 0; --c) {
        const int t0 = c * kC;
        const int nt = min(kC, T - t0);
        const size_t row0 = (size_t)b * T + t0;
        const float lam_start = saved_lam[((size_t)bh * nchunk32 + 2 * c) * DK + ng];

        ystage.template store<LD, LT, true, true>(sm + Cfg::DY, sm + Cfg::DYT, tid);
        vstage.template store<LD, 0, true, false>(sm + Cfg::V, nullptr, tid);
        if (c > 0) {  // earlier chunks are full
            ystage.load(dy, row0 - kC, s.H, h, DV, 0, kC, tid);
            vstage.load(v, row0 - kC, s.H, h, DV, 0, kC, tid);
        }
        __syncthreads();

        if (wave == 0) {
            // precision walk of this workgroup's key slots
            float lam = saved_lam[((size_t)bh * nchunk32 + 2 * c) * DK + (scan_lane ? n0 + tid : n0)];
            ScanLds L{};
            L.qt_hi = sm + Cfg::QTH;
            L.qt_lo = sm + Cfg::QTL;
            L.kt_hi = sm + Cfg::KTH;
            L.kt_lo = sm + Cfg::KTL;
            L.lam = smf + Cfg::LAM;
            L.P = smf + Cfg::PP;
            const int n = scan_lane ? n0 + tid : n0;
            const float P = scan_chunk<kC, 0, LT, LS, false, false, true, true, true, 4>(
                a, p, k, q, r, row0, s.H, h, DK, n, scan_lane ? tid : 0, scan_lane, nt, lam, L, lane, spre);
            if (scan_lane) smf[Cfg::DECAY + tid] = P;
            if (c > 0) scan_prefetch<4>(spre, a, p, k, q, r, row0 - kC, s.H, h, DK, n, kC);
        } else {
            // meanwhile B[s, j] = dY_s . V_j for j <= s (exact bf16 products), kept as B and
            // B^T; tiles (0,1), (2,3) are the zeros read by the 32-deep K steps.
            for (int tk = wave - 1; tk < 12; tk += 3) {
                int st, jt;
                if (tk < 10) {
                    st = tk >= 6 ? 3 : tk >= 3 ? 2 : tk >= 1 ? 1 : 0;
                    jt = tk - st * (st + 1) / 2;
                } else {
                    st = tk == 10 ? 0 : 2;
                    jt = st + 1;
                }
                f32x4 acc = zero4();
                if (tk < 10) {
#pragma unroll
                    for (int ks = 0; ks < KSD; ++ks) {
                        const bf16x8 ya = lds8(sm + Cfg::DY + (16 * st + l16) * LD + 32 * ks + 8 * g4);
                        const bf16x8 vb = lds8(sm + Cfg::V + (16 * jt + l16) * LD + 32 * ks + 8 * g4);
                        acc = mfma_bf16(ya, vb, acc);
                    }
                }
#pragma unroll
                for (int rr = 0; rr < 4; ++rr) {
                    const int si = 16 * st + 4 * g4 + rr, j = 16 * jt + l16;
                    const float x = (tk < 10 && j <= si) ? acc[rr] : 0.f;
                    uint16_t hi, lo;
                    split(x, hi, lo);
                    sm[Cfg::BH + si * LT + j] = hi;
                    sm[Cfg::BL + si * LT + j] = lo;
                    sm[Cfg::BTH + j * LT + si] = hi;
                    sm[Cfg::BTL + j * LT + si] = lo;
                }
            }
        }
        __syncthreads();

        f32x4 accX[4], accY[4];
        if (owns) {
            // X = dY H0^T + M(B) Kn
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) accX[mt] = zero4();
#pragma unroll
            for (int ks = 0; ks < KSD; ++ks) {
                const float4 h0a = h0pre[ks][0], h0b = h0pre[ks][1];
                bf16x8 hh, hl;
                split8(f32x4{h0a.x, h0a.y, h0a.z, h0a.w}, f32x4{h0b.x, h0b.y, h0b.z, h0b.w}, hh, hl);
#pragma unroll
                for (int mt = 0; mt < 4; ++mt) {
                    const bf16x8 ya = lds8(sm + Cfg::DY + (16 * mt + l16) * LD + 32 * ks + 8 * g4);
                    accX[mt] = mfma2b(ya, hh, hl, accX[mt]);
                }
            }
            if (c > 0) load_h0(c - 1);
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) {
#pragma unroll
                for (int ks = 0; ks <= (mt >> 1); ++ks) {
                    const int bo = (16 * mt + l16) * LT + 32 * ks + 8 * g4;
                    const int ko = ncl * LT + 32 * ks + 8 * g4;
                    accX[mt] = mfma3(lds8(sm + Cfg::BH + bo), lds8(sm + Cfg::BL + bo), lds8(sm + Cfg::KTH + ko),
                                     lds8(sm + Cfg::KTL + ko), accX[mt]);
                }
            }
            // Y = M(B)^T Qp + V Gs^T
            const float Pc = smf[Cfg::DECAY + ncl];
#pragma unroll
            for (int rd = 0; rd < NRD; ++rd)
#pragma unroll
                for (int rr = 0; rr < 4; ++rr) GT[rd][rr] *= Pc;   // Gs^T in place
#pragma unroll
            for (int jt = 0; jt < 4; ++jt) accY[jt] = zero4();
#pragma unroll
            for (int jt = 0; jt < 4; ++jt) {
#pragma unroll
                for (int ks = jt >> 1; ks < 2; ++ks) {
                    const int bo = (16 * jt + l16) * LT + 32 * ks + 8 * g4;
                    const int qo = ncl * LT + 32 * ks + 8 * g4;
                    accY[jt] = mfma3(lds8(sm + Cfg::BTH + bo), lds8(sm + Cfg::BTL + bo), lds8(sm + Cfg::QTH + qo),
                                     lds8(sm + Cfg::QTL + qo), accY[jt]);
                }
            }
#pragma unroll
            for (int ks = 0; ks < KSD; ++ks) {
                bf16x8 gh, gl;
                split8(GT[2 * ks], GT[2 * ks + 1], gh, gl);
#pragma unroll
                for (int jt = 0; jt < 4; ++jt) {
                    const int vo = (16 * jt + l16) * LD + 32 * ks + 4 * g4;
                    accY[jt] = mfma2b(lds4x2(sm + Cfg::V + vo, sm + Cfg::V + vo + 16), gh, gl, accY[jt]);
                }
            }
            // G^T <- dY^T Qp + Gs^T
#pragma unroll
            for (int rd = 0; rd < NRD; ++rd) {
                f32x4 gacc = GT[rd];
#pragma unroll
                for (int ks = 0; ks < 2; ++ks) {
                    const bf16x8 ya = lds8(sm + Cfg::DYT + (16 * rd + l16) * LT + 32 * ks + 8 * g4);
                    const int qo = ncl * LT + 32 * ks + 8 * g4;
                    gacc = mfma2b(ya, lds8(sm + Cfg::QTH + qo), lds8(sm + Cfg::QTL + qo), gacc);
                }
                GT[rd] = gacc;
            }
        }
        __syncthreads();  // B buffers are dead: X and Y take their place
        if (owns) {
#pragma unroll
            for (int mt = 0; mt < 4; ++mt)
#pragma unroll
                for (int rr = 0; rr < 4; ++rr) {
                    const int t = 16 * mt + 4 * g4 + rr;
                    smf[Cfg::X + t * LS + ncl] = accX[mt][rr];
                    smf[Cfg::Y + t * LS + ncl] = accY[mt][rr];
                }
        }
        __syncthreads();

        // Reverse walk over the chunk's tokens, split into four 16-token quarters,
        // one per wave (lane = key slot).  With u_t = qt dqt - kh dkh and
        // w_t = q dqt / lam_t^2, the log-gate adjoint is S_t = S_in + sum_{s>=t} u_s
        // and the precision-adjoint carry obeys c_{t-1} = alpha_t (c_t - w_t) -
        // pbar_t rho_t S_t (alpha = abar^2 rho^2), affine in the quarter's incoming
        // (c_in, S_in).  Pass 1 composes each quarter into c_out = A c_in + B +
        // Gam S_in and S_out = S_in + U; the quarters are chained through LDS;
        // pass 2 re-walks each quarter from its incoming carries and writes the
        // gradients.
        if (lane < NTN) {
            const int tq1 = 16 * wave + 15;       // last token of this wave's quarter
            struct GIn {
                float av, pv, kv, qv, rv, lam_t, lam_p, Pt, Xv, Yv;
            };
            auto fetch = [&](int t) {
                GIn x;
                const int tc = min(t, nt - 1);
                const size_t rowi = (row0 + tc) * s.H + h;
                const size_t o = rowi * DK + ng;
                x.av = bf16_to_f32(a[o]);
                x.pv = bf16_to_f32(p[o]);
                x.kv = bf16_to_f32(k[o]);
                x.qv = bf16_to_f32(q[o]);
                x.rv = bf16_to_f32(r[rowi]);
                x.lam_t = smf[Cfg::LAM + t * LS + nl];
                const float lp = smf[Cfg::LAM + max(t - 1, 0) * LS + nl];
                x.lam_p = t > 0 ? lp : lam_start;
                x.Pt = smf[Cfg::PP + t * LS + nl];
                x.Xv = smf[Cfg::X + t * LS + nl];
                x.Yv = smf[Cfg::Y + t * LS + nl];
                return x;
            };
            // pass 1: affine summary of the quarter
            float A = 1.f, Bc = 0.f, Gam = 0.f, U = 0.f;
#pragma unroll 4
            for (int t = tq1; t > tq1 - 16; --t) {
                if (t >= nt) continue;
                const GIn x = fetch(t);
                const float den = fmaf(x.pv, x.lam_p, x.av * x.av);
                const float rr3 = fast_rcp(den * x.lam_t);
                const float rho = x.lam_t * rr3, ilam = den * rr3;
                const float dqt = x.Pt * x.Xv, dkh = x.Yv * fast_rcp(x.Pt);
                U += x.qv * ilam * dqt - x.rv * x.kv * dkh;           // L_t (local suffix sum)
                const float w = x.qv * dqt * ilam * ilam;
                const float alpha = x.av * x.av * rho * rho, prho = x.pv * rho;
                Bc = alpha * (Bc - w) - prho * U;
                A *= alpha;
                Gam = alpha * Gam - prho;
            }
            smf[Cfg::QS + (wave * 4 + 0) * NTN + nl] = A;
            smf[Cfg::QS + (wave * 4 + 1) * NTN + nl] = Bc;
            smf[Cfg::QS + (wave * 4 + 2) * NTN + nl] = Gam;
            smf[Cfg::QS + (wave * 4 + 3) * NTN + nl] = U;
        }
        __syncthreads();  // quarter summaries visible to every wave
        if (lane < NTN) {
            const int tq1 = 16 * wave + 15;
            float c_in = cnext, S_in = Sg;
            for (int w2 = 3; w2 > wave; --w2) {
                const float A2 = smf[Cfg::QS + (w2 * 4 + 0) * NTN + nl];
                const float B2 = smf[Cfg::QS + (w2 * 4 + 1) * NTN + nl];
                const float G2 = smf[Cfg::QS + (w2 * 4 + 2) * NTN + nl];
                const float U2 = smf[Cfg::QS + (w2 * 4 + 3) * NTN + nl];
                c_in = A2 * c_in + B2 + G2 * S_in;
                S_in += U2;
            }
            // carries into the previous chunk: through all four quarters
            {
                float c_all = cnext, S_all = Sg;
                for (int w2 = 3; w2 >= 0; --w2) {
                    const float A2 = smf[Cfg::QS + (w2 * 4 + 0) * NTN + nl];
                    const float B2 = smf[Cfg::QS + (w2 * 4 + 1) * NTN + nl];
                    const float G2 = smf[Cfg::QS + (w2 * 4 + 2) * NTN + nl];
                    const float U2 = smf[Cfg::QS + (w2 * 4 + 3) * NTN + nl];
                    c_all = A2 * c_all + B2 + G2 * S_all;
                    S_all += U2;
                }
                cnext = c_all;
                Sg = S_all;
            }
            // pass 2: gradients of the quarter's tokens
            float c = c_in, S = S_in;
#pragma unroll 4
            for (int t = tq1; t > tq1 - 16; --t) {
                if (t >= nt) continue;
                const int tc = t;
                const size_t rowi = (row0 + tc) * s.H + h;
                const size_t o = rowi * DK + ng;
                const float av = bf16_to_f32(a[o]), pv = bf16_to_f32(p[o]);
                const float kv = bf16_to_f32(k[o]), qv = bf16_to_f32(q[o]);
                const float rv = bf16_to_f32(r[rowi]);
                const float lam_t = smf[Cfg::LAM + t * LS + nl];
                const float lpl = smf[Cfg::LAM + max(t - 1, 0) * LS + nl];
                const float lam_p = t > 0 ? lpl : lam_start;
                const float Pt = smf[Cfg::PP + t * LS + nl];
                const float Xv = smf[Cfg::X + t * LS + nl], Yv = smf[Cfg::Y + t * LS + nl];
                const float den = fmaf(pv, lam_p, av * av);
                const float rr3 = fast_rcp(den * lam_t * av);   // one reciprocal for three
                const float rho = lam_t * av * rr3;
                const float ilam = den * av * rr3;
                const float ia = den * lam_t * rr3;
                const float dqt = Pt * Xv;
                const float dkh = Yv * fast_rcp(Pt);
                const float kh = rv * kv;
                S += qv * ilam * dqt - kh * dkh;                      // adjoint of log F_t
                const float gl = c - qv * dqt * ilam * ilam;          // adjoint of lam_t
                const float drho = fmaf(gl, lam_p, S * den);
                const float rho2 = rho * rho;
                dq[o] = f32_to_bf16(dqt * ilam);
                dk[o] = f32_to_bf16(rv * dkh + 2.f * kv * rv * gl);
                da[o] = f32_to_bf16(S * ia - 2.f * av * rho2 * drho);
                dp[o] = f32_to_bf16(-lam_p * rho2 * drho);
                smf[Cfg::X + t * LS + nl] = kv * dkh + kv * kv * gl;   // term of dr
                c = av * av * rho2 * gl - pv * rho * S;
            }
        }
        __syncthreads();
        // partial dr over this workgroup's key slots: 4 threads per token
        {
            const int t = tid >> 2, qd = tid & 3;
            float acc = 0.f;
            if (t < kC) {
#pragma unroll 4
                for (int i = qd; i < NTN; i += 4) acc += smf[Cfg::X + t * LS + i];
            }
            acc += __shfl_xor(acc, 1, 64);
            acc += __shfl_xor(acc, 2, 64);
            if (t < nt && qd == 0) dr_part[(size_t)ntile * nbt + (row0 + t) * s.H + h] = acc;
        }
        __syncthreads();
    }
    if (wave == 0 && glane && g.dlam0) g.dlam0[(size_t)bh * DK + ng] = cnext;
}

// dr = sum of the per-key-tile partials, stored in the input dtype
__global__ void dr_combine_kernel(const float* __restrict__ part, int ntile, size_t n, uint16_t* __restrict__ dr) {
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    float acc = 0.f;
    for (int t = 0; t < ntile; ++t) acc += part[(size_t)t * n + i];
    dr[i] = f32_to_bf16(acc);
}

template <int DK, int DV>
hipError_t launch_bwd(const Shape& s, const BwdArgs& a, const float* saved_lam, const float* saved_H, float* dr_part,
                      hipStream_t st) {
    using C2 = B2Cfg<DK, DV>;
    auto k2 = bwd_b2_kernel<DK, DV>;
    static const hipError_t e2 = hipFuncSetAttribute(reinterpret_cast<const void*>(k2),
                                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)C2::BYTES);
    if (e2 != hipSuccess) return e2;
    hipError_t e = launch_backward_dv(s, a, saved_lam, st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k2, dim3(s.B * s.H * C2::NNT), dim3(kThr), C2::BYTES, st, s, a, saved_lam, saved_H, dr_part);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const size_t n = (size_t)s.B * s.T * s.H;
    if (n > 0) {
        hipLaunchKernelGGL(dr_combine_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, dr_part, C2::NNT, n,
                           static_cast<uint16_t*>(a.dr));
        e = hipGetLastError();
    }
    return e;
}

}  // namespace

bool chunked_bwd_supported(const Shape& s) { return s.bf16 && s.dk >= 32 && s.dv >= 32; }

size_t chunked_bwd_workspace(const Shape& s) {
    const int ntn = s.dk < 64 ? s.dk : 64;
    return (size_t)(s.dk / ntn) * s.B * s.T * s.H * sizeof(float);
}

hipError_t launch_backward_chunked(const Shape& s, const BwdArgs& a, const void* saved, void* ws, hipStream_t st) {
    const size_t nchunk32 = (size_t)(s.T + 31) / 32;
    const float* saved_lam = static_cast<const float*>(saved);
    const float* saved_H = saved_lam + (size_t)s.B * s.H * nchunk32 * s.dk;
    float* dr_part = static_cast<float*>(ws);
#define KLA_BWD_CASE(DK_, DV_) \
    if (s.dk == DK_ && s.dv == DV_) return launch_bwd<DK_, DV_>(s, a, saved_lam, saved_H, dr_part, st);
#define KLA_BWD_ROW(DK_) KLA_BWD_CASE(DK_, 32) KLA_BWD_CASE(DK_, 64) KLA_BWD_CASE(DK_, 128)
    KLA_BWD_ROW(32) KLA_BWD_ROW(64) KLA_BWD_ROW(128)
#undef KLA_BWD_ROW
#undef KLA_BWD_CASE
    return hipErrorInvalidValue;
}

}  // namespace kla
