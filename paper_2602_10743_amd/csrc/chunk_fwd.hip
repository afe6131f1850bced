// Chunked forward of the KLA filter on MFMA (bf16 inputs, fp32 state).
//
// The sequence is cut into chunks of kC = 64 tokens.  Within a chunk, for each
// key slot n, the precision path (Theorem 1, gate view) is walked token by
// token from the carried lam, giving the gate F_t = abar_t rho_t (Theorem 2),
// its running product P_t = prod_{s<=t} F_s inside the chunk, the effective
// query qt_t = q_t / lam_t and the evidence key kh_t = r_t k_t.  With
//   Qp[t, n] = qt_t[n] P_t[n],   Kn[t, n] = kh_t[n] / P_t[n]
// the information-state recursion over the chunk is exactly
//   y    = mask(Qp Kn^T) V + Qp H                       (readout, Algorithm 1)
//   H   <- diag(P_C) (H + Kn^T V)                       (state at the chunk end)
// (the unrolled "attention matrix" of the paper's appendix, restricted to a
// chunk, plus the carried state).  The four contractions run on
// v_mfma_f32_16x16x32_bf16 with split-bf16 operands for the fp32 factors
// (see kla_mfma.hpp), accumulating in fp32.
//
// One workgroup (4 waves) per (batch, head, 64-wide value tile) walks the
// chunks in order with the state tile H[dk, 64] in registers: wave w owns the
// 16 value channels 16w..16w+15 of the tile for the readout and the state.
// Requirement (documented in the ABI): inside one chunk the product of gates
// P_t stays within fp32 range for every key slot.
#include "kla_internal.hpp"
#include "kla_mfma.hpp"
#include "kla_scan.hpp"

namespace kla {
namespace {

constexpr int kC = 64;
constexpr int kThreadsC = 256;

template <int DK, int DV>
struct FwdCfg {
    static constexpr int DVT = DV < 64 ? DV : 64;
    static constexpr int NTILE = DV / DVT;
    static constexpr int NCT = DVT / 16;
    static constexpr int NRT = DK / 16;
    static constexpr int KSN = DK / 32;
    static constexpr int NSCAN = DK < 64 ? 64 : DK;   // threads running the precision scan
    static constexpr int LQ = DK + 8;                  // row stride of [t][n] buffers
    static constexpr int LT = kC + 8;                  // row stride of [n][t], [d][t], [i][j]
    static constexpr int QH = 0, QL = QH + kC * LQ, KH = QL + kC * LQ, KL = KH + kC * LQ;
    static constexpr int KTH = KL + kC * LQ, KTL = KTH + DK * LT;
    static constexpr int VT = KTL + DK * LT;
    static constexpr int AH = VT + DVT * LT, AL = AH + kC * LT;
    static constexpr int END16 = AL + kC * LT;
    static constexpr int DECAY = (END16 + 7) / 8 * 4;      // float index
    static constexpr int YV = DECAY + DK;                  // [2][kC] floats
    static constexpr size_t BYTES = (size_t)(YV + 2 * kC) * 4;
    static_assert(DK >= 32 && DK % 32 == 0, "chunked path needs dk >= 32");
    static_assert(BYTES <= 160 * 1024, "LDS budget of one workgroup");
};

template <int DK, int DV, bool YV>
__global__ __launch_bounds__(kThreadsC) void fwd_chunk_kernel(Shape s, FwdArgs g, float* saved_lam,
                                                              float* saved_H) {
    using Cfg = FwdCfg<DK, DV>;
    constexpr int DVT = Cfg::DVT, NTILE = Cfg::NTILE, NCT = Cfg::NCT, NRT = Cfg::NRT, KSN = Cfg::KSN;
    constexpr int LQ = Cfg::LQ, LT = Cfg::LT;
    extern __shared__ __align__(16) unsigned char smem_raw[];
    uint16_t* sm = reinterpret_cast<uint16_t*>(smem_raw);
    float* smf = reinterpret_cast<float*>(smem_raw);
    float* sDecay = smf + Cfg::DECAY;
    float* sYV = smf + Cfg::YV;

    const uint16_t* q = static_cast<const uint16_t*>(g.q);
    const uint16_t* k = static_cast<const uint16_t*>(g.k);
    const uint16_t* v = static_cast<const uint16_t*>(g.v);
    const uint16_t* a = static_cast<const uint16_t*>(g.a);
    const uint16_t* p = static_cast<const uint16_t*>(g.p);
    const uint16_t* r = static_cast<const uint16_t*>(g.r);
    uint16_t* y = static_cast<uint16_t*>(g.y);

    // workgroup -> (b, h, value tile); the tiles of one (b, h) share an XCD (and its L2)
    const int nbh = s.B * s.H;
    int bh, tile;
    {
        const int i = blockIdx.x;
        if (nbh % 8 == 0) {
            const int xcd = i % 8, slot = i / 8;
            tile = slot % NTILE;
            bh = (slot / NTILE) * 8 + xcd;
        } else {
            tile = i % NTILE;
            bh = i / NTILE;
        }
    }
    const int b = bh / s.H, h = bh % s.H;
    const int d0 = tile * DVT;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l16 = lane & 15, g4 = lane >> 4;
    const int T = s.T;
    const int nchunk = (T + kC - 1) / kC;
    const bool want_yvar = YV && tile == 0;

    // state tile owned by this wave: rows n (all), columns d0 + 16*wave .. +15
    f32x4 Hs[NRT];
    const bool owns_cols = wave < NCT;
    const int dcol = d0 + 16 * wave + l16;
#pragma unroll
    for (int rt = 0; rt < NRT; ++rt) {
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
            const int n = 16 * rt + 4 * g4 + rr;
            Hs[rt][rr] = (owns_cols && g.eta0) ? g.eta0[((size_t)bh * DK + n) * DV + dcol] : 0.f;
        }
    }
    // precision lane n = tid (threads tid < DK)
    const bool scan_lane = tid < DK;
    float lam = 1.f;
    if (scan_lane && g.lam0) lam = g.lam0[(size_t)bh * DK + tid];

    // the next chunk's value tile and first scan inputs are in flight during a chunk
    TileStage<kC, DVT, kThreadsC> vstage;
    ScanPrefetch<8> spre;
    const int n_scan = scan_lane ? tid : DK - 1;
    if (nchunk > 0) {
        const int nt0 = min(kC, T);
        vstage.load(v, (size_t)b * T, s.H, h, DV, d0, nt0, tid);
        if (tid < Cfg::NSCAN) scan_prefetch<8>(spre, a, p, k, q, r, (size_t)b * T, s.H, h, DK, n_scan, nt0);
    }

    for (int c = 0; c < nchunk; ++c) {
        const int t0 = c * kC;
        const int nt = min(kC, T - t0);
        const size_t row0 = (size_t)b * T + t0;   // token index of t0 within batch b
        const int ntn = min(kC, T - t0 - kC);      // tokens of the next chunk (if any)

        if (saved_H) {
            if (scan_lane) saved_lam[((size_t)bh * nchunk + c) * DK + tid] = lam;
            if (owns_cols) {
                float* dst = saved_H + ((size_t)bh * (nchunk + 1) + c) * DK * DV;
#pragma unroll
                for (int rt = 0; rt < NRT; ++rt)
#pragma unroll
                    for (int rr = 0; rr < 4; ++rr) dst[(16 * rt + 4 * g4 + rr) * DV + dcol] = Hs[rt][rr];
            }
        }

        // ---- value tile, transposed into [d][t]; then the next chunk's is requested
        vstage.template store<0, LT, false, true>(nullptr, sm + Cfg::VT, tid);
        if (c + 1 < nchunk) vstage.load(v, row0 + kC, s.H, h, DV, d0, ntn, tid);

        // ---- precision walk, one key slot per lane
        if (tid < Cfg::NSCAN) {
            ScanLds L{};
            L.qn_hi = sm + Cfg::QH;
            L.qn_lo = sm + Cfg::QL;
            L.kn_hi = sm + Cfg::KH;
            L.kn_lo = sm + Cfg::KL;
            L.kt_hi = sm + Cfg::KTH;
            L.kt_lo = sm + Cfg::KTL;
            L.yv = sYV + wave * kC;
            const float P = scan_chunk<kC, LQ, LT, 0, true, true, false, true, false, 8, YV>(
                a, p, k, q, r, row0, s.H, h, DK, n_scan, n_scan, scan_lane, nt, lam, L, lane, spre);
            if (scan_lane) sDecay[n_scan] = P;
            if (c + 1 < nchunk) scan_prefetch<8>(spre, a, p, k, q, r, row0 + kC, s.H, h, DK, n_scan, ntn);
        }
        __syncthreads();

        // ---- attention tiles A[i, j] = sum_n Qp[i, n] Kn[j, n], j <= i, shared through LDS
        for (int tk = wave; tk < 12; tk += 4) {
            int it, jt;
            if (tk < 10) {
                it = tk >= 6 ? 3 : tk >= 3 ? 2 : tk >= 1 ? 1 : 0;
                jt = tk - it * (it + 1) / 2;
            } else {  // upper tiles read by the 32-deep K steps: zero them
                it = tk == 10 ? 0 : 2;
                jt = it + 1;
            }
            f32x4 acc = zero4();
            if (tk < 10) {
#pragma unroll
                for (int ks = 0; ks < KSN; ++ks) {
                    const int qo = (16 * it + l16) * LQ + 32 * ks + 8 * g4;
                    const int ko = (16 * jt + l16) * LQ + 32 * ks + 8 * g4;
                    acc = mfma3(lds8(sm + Cfg::QH + qo), lds8(sm + Cfg::QL + qo), lds8(sm + Cfg::KH + ko),
                                lds8(sm + Cfg::KL + ko), acc);
                }
            }
#pragma unroll
            for (int rr = 0; rr < 4; ++rr) {
                const int i = 16 * it + 4 * g4 + rr, j = 16 * jt + l16;
                const float x = (tk < 10 && j <= i) ? acc[rr] : 0.f;
                uint16_t hi, lo;
                split(x, hi, lo);
                sm[Cfg::AH + i * LT + j] = hi;
                sm[Cfg::AL + i * LT + j] = lo;
            }
        }
        __syncthreads();

        if (want_yvar && tid < nt) {
            float acc = 0.f;
            for (int w2 = 0; w2 < (Cfg::NSCAN + 63) / 64; ++w2) acc += sYV[w2 * kC + tid];
            g.yvar[(row0 + tid) * s.H + h] = acc;
        }

        if (owns_cols) {
            const int ct = wave;
            // ---- readout: y = mask(A) V + Qp H
            f32x4 acc[4];
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) acc[mt] = zero4();
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) {
#pragma unroll
                for (int ks = 0; ks <= (mt >> 1); ++ks) {
                    const int ao = (16 * mt + l16) * LT + 32 * ks + 8 * g4;
                    const bf16x8 vb = lds8(sm + Cfg::VT + (16 * ct + l16) * LT + 32 * ks + 8 * g4);
                    acc[mt] = mfma2a(lds8(sm + Cfg::AH + ao), lds8(sm + Cfg::AL + ao), vb, acc[mt]);
                }
            }
#pragma unroll
            for (int ks = 0; ks < KSN; ++ks) {
                bf16x8 hh, hl;
                split8(Hs[2 * ks], Hs[2 * ks + 1], hh, hl);
#pragma unroll
                for (int mt = 0; mt < 4; ++mt) {
                    const int qo = (16 * mt + l16) * LQ + 32 * ks + 4 * g4;
                    const bf16x8 qh = lds4x2(sm + Cfg::QH + qo, sm + Cfg::QH + qo + 16);
                    const bf16x8 ql = lds4x2(sm + Cfg::QL + qo, sm + Cfg::QL + qo + 16);
                    acc[mt] = mfma3(qh, ql, hh, hl, acc[mt]);
                }
            }
#pragma unroll
            for (int mt = 0; mt < 4; ++mt)
#pragma unroll
                for (int rr = 0; rr < 4; ++rr) {
                    const int t = 16 * mt + 4 * g4 + rr;
                    if (t < nt) y[((row0 + t) * s.H + h) * DV + dcol] = f32_to_bf16(acc[mt][rr]);
                }

            // ---- state: H <- diag(P_C) (H + Kn^T V)
#pragma unroll
            for (int rt = 0; rt < NRT; ++rt) {
                f32x4 hacc = Hs[rt];
#pragma unroll
                for (int ks = 0; ks < 2; ++ks) {
                    const int ko = (16 * rt + l16) * LT + 32 * ks + 8 * g4;
                    const bf16x8 vb = lds8(sm + Cfg::VT + (16 * ct + l16) * LT + 32 * ks + 8 * g4);
                    hacc = mfma2a(lds8(sm + Cfg::KTH + ko), lds8(sm + Cfg::KTL + ko), vb, hacc);
                }
#pragma unroll
                for (int rr = 0; rr < 4; ++rr) Hs[rt][rr] = hacc[rr] * sDecay[16 * rt + 4 * g4 + rr];
            }
        }
        __syncthreads();
    }

    if (saved_H && owns_cols) {  // the final state closes the saved sequence of chunk-start states
        float* dst = saved_H + ((size_t)bh * (nchunk + 1) + nchunk) * DK * DV;
#pragma unroll
        for (int rt = 0; rt < NRT; ++rt)
#pragma unroll
            for (int rr = 0; rr < 4; ++rr) dst[(16 * rt + 4 * g4 + rr) * DV + dcol] = Hs[rt][rr];
    }
    if (g.lamT && scan_lane && tile == 0) g.lamT[(size_t)bh * DK + tid] = lam;
    if (g.etaT && owns_cols) {
#pragma unroll
        for (int rt = 0; rt < NRT; ++rt)
#pragma unroll
            for (int rr = 0; rr < 4; ++rr)
                g.etaT[((size_t)bh * DK + 16 * rt + 4 * g4 + rr) * DV + dcol] = Hs[rt][rr];
    }
}

template <int DK, int DV, bool YV>
hipError_t launch_fwd_v(const Shape& s, const FwdArgs& a, float* saved_lam, float* saved_H, hipStream_t st) {
    using Cfg = FwdCfg<DK, DV>;
    auto kern = fwd_chunk_kernel<DK, DV, YV>;
    // more than 64 KiB of LDS must be opted into once per kernel (thread-safe static init)
    static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)Cfg::BYTES);
    if (attr != hipSuccess) return attr;
    const unsigned grid = (unsigned)(s.B * s.H * Cfg::NTILE);
    hipLaunchKernelGGL(kern, dim3(grid), dim3(kThreadsC), Cfg::BYTES, st, s, a, saved_lam, saved_H);
    return hipGetLastError();
}

// the readout variance adds a cross-lane sum per token, so it is a separate instantiation
template <int DK, int DV>
hipError_t launch_fwd(const Shape& s, const FwdArgs& a, float* saved_lam, float* saved_H, hipStream_t st) {
    return a.yvar ? launch_fwd_v<DK, DV, true>(s, a, saved_lam, saved_H, st)
                  : launch_fwd_v<DK, DV, false>(s, a, saved_lam, saved_H, st);
}

}  // namespace

bool chunked_supported(const Shape& s) { return s.bf16 && s.dk >= 32; }

// Saved context: lam at every chunk start [BH][nchunk][dk], then the information
// state at every chunk start and after the last token [BH][nchunk+1][dk][dv].
size_t chunked_saved_bytes(const Shape& s) {
    const size_t nchunk = (size_t)(s.T + kC - 1) / kC;
    return (size_t)s.B * s.H * s.dk * (nchunk + (nchunk + 1) * (size_t)s.dv) * sizeof(float);
}

hipError_t launch_forward_chunked(const Shape& s, const FwdArgs& a, void* saved, hipStream_t st) {
    float* saved_lam = nullptr;
    float* saved_H = nullptr;
    if (saved) {
        const size_t nchunk = (size_t)(s.T + kC - 1) / kC;
        saved_lam = static_cast<float*>(saved);
        saved_H = saved_lam + (size_t)s.B * s.H * nchunk * s.dk;
    }
#define KLA_FWD_CASE(DK_, DV_) \
    if (s.dk == DK_ && s.dv == DV_) return launch_fwd<DK_, DV_>(s, a, saved_lam, saved_H, st);
#define KLA_FWD_ROW(DK_) KLA_FWD_CASE(DK_, 16) KLA_FWD_CASE(DK_, 32) KLA_FWD_CASE(DK_, 64) KLA_FWD_CASE(DK_, 128)
    KLA_FWD_ROW(32) KLA_FWD_ROW(64) KLA_FWD_ROW(128)
#undef KLA_FWD_ROW
#undef KLA_FWD_CASE
    return hipErrorInvalidValue;
}

}  // namespace kla
