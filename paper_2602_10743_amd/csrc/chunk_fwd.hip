// Chunked forward of the KLA filter on MFMA (bf16 inputs, fp32 state).
//
// Per chunk of kC = 32 tokens, with Qp[t, n] = (q_t / lam_t) P_t and
// Kn[t, n] = (r_t k_t) / P_t from the precision walk (kla_chunk.hpp), the
// information-state recursion over the chunk is exactly
//   y    = mask(Qp Kn^T) V + Qp H                       (readout, Algorithm 1)
//   H   <- diag(P_C) (H + Kn^T V)                       (state at the chunk end)
// (the unrolled "attention matrix" of the paper's appendix, restricted to a
// chunk, plus the carried state).  The contractions run on
// v_mfma_f32_16x16x32_bf16 with split-bf16 operands for the fp32 factors
// (kla_mfma.hpp), accumulating in fp32.
//
// One workgroup per (batch, head, value tile of up to 64 channels): scan waves
// walk chunk c while MFMA waves (16 value channels each, the state H[dk, 16]
// in registers) consume chunk c - 1 -- attention tiles, readout, y, state
// update; operands that run across the rows of a tile (Kn^T, V) are read with
// transposing LDS reads (lds_tr8), so each tile is stored once.  The MFMA
// waves only store; all loads come from the scan waves.  TI: the gates come
// from OU parameters (time-invariant per key slot) instead of per-token tensors.
#include "kla_chunk.hpp"
#include "kla_internal.hpp"

namespace kla {
namespace {

template <int DK, int DV, bool YV, bool TI, bool NOY>
__global__ __launch_bounds__((ChunkCfg<DK, DV>::NTHR)) void fwd_chunk_kernel(Shape s, FwdArgs g, float* saved_lam,
                                                                         float* saved_H) {
    using Cfg = ChunkCfg<DK, DV>;
    constexpr int DVT = Cfg::DVT, NTILE = Cfg::NTILE, DCW = Cfg::DCW, NDT = Cfg::NDT, NSW = Cfg::NSW;
    constexpr int SW = Cfg::SW, NRT = Cfg::NRT, KSN = Cfg::KSN, LQ = Cfg::LQ;
    extern __shared__ __align__(16) unsigned char smem[];

    const uint16_t* q = static_cast<const uint16_t*>(g.q);
    const uint16_t* k = static_cast<const uint16_t*>(g.k);
    const uint16_t* v = static_cast<const uint16_t*>(g.v);
    const uint16_t* a = static_cast<const uint16_t*>(g.a);
    const uint16_t* p = static_cast<const uint16_t*>(g.p);
    const uint16_t* r = static_cast<const uint16_t*>(g.r);
    uint16_t* y = static_cast<uint16_t*>(g.y);

    int bh, tile;
    xcd_tile_map(blockIdx.x, s.B * s.H, NTILE, bh, tile);
    const int b = bh / s.H, h = bh % s.H;
    const int H = s.H, T = s.T;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform role
    const int l16 = lane & 15, g4 = lane >> 4;
    const int nchunk = (T + kC - 1) / kC;
    const size_t seq0 = (size_t)b * T;   // token index of this sequence's first token

    if (wave < NSW) {
        // ================================================================ scan waves
        const ScanSrc sc{a, p, k, q, r, v, tile * DVT, seq0, H, h, T, nchunk, bh, g.ou_a, g.ou_p, g.ou_d, g.range_flag};
        const float x = scan_wave<Cfg, YV, false, TI, NOY>(smem, wave, lane, sc, g.lam0, saved_lam != nullptr);
        if (g.lamT && lane < SW && tile == 0) g.lamT[(size_t)bh * DK + wave * SW + lane] = x;
    } else {
        // ================================================================ MFMA waves
        const int m = wave - NSW;
        const int dm0 = tile * DVT + m * DCW;   // first value channel of this wave
        const int dl0 = m * DCW;                // its first column within the value tile

        // state H[n, d] for n = 16 rt + 4 g4 + rr, d = dm0 + 16 dt + l16
        f32x4 Hs[NRT][NDT];
#pragma unroll
        for (int rt = 0; rt < NRT; ++rt)
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
                for (int rr = 0; rr < 4; ++rr)
                    Hs[rt][dt][rr] =
                        g.eta0 ? g.eta0[((size_t)bh * DK + 16 * rt + 4 * g4 + rr) * DV + dm0 + 16 * dt + l16] : 0.f;

        // state rows 16 rt .. 16 rt + 15 (this wave's columns) into saved slot `slot`
        auto save_rows = [&](int slot, int rt) {
            float* dst = saved_H + ((size_t)bh * (nchunk + 1) + slot) * DK * DV;
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
                for (int rr = 0; rr < 4; ++rr)
                    dst[(16 * rt + 4 * g4 + rr) * DV + dm0 + 16 * dt + l16] = Hs[rt][dt][rr];
        };
        for (int c = 0; c <= nchunk; ++c) {
            const int cc = c - 1;   // the chunk consumed in this round
            if (cc >= 0) {
                const int nt = min(kC, T - cc * kC);
                const size_t row0 = seq0 + (size_t)cc * kC;
                const unsigned char* buf = smem + (cc & 1) * Cfg::BUF;
                const uint16_t* sVS = reinterpret_cast<const uint16_t*>(buf + Cfg::VS);   // V [t][DVT]
                const uint16_t* sQH = reinterpret_cast<const uint16_t*>(buf + Cfg::QH);
                const uint16_t* sQL = reinterpret_cast<const uint16_t*>(buf + Cfg::QL);
                const uint16_t* sKH = reinterpret_cast<const uint16_t*>(buf + Cfg::KH);
                const uint16_t* sKL = reinterpret_cast<const uint16_t*>(buf + Cfg::KL);
                const float* sDec = reinterpret_cast<const float*>(buf + Cfg::DEC);

                if constexpr (!NOY) {   // the readout (skipped when only the final state is asked for)
                    // ---- S^T[j, i] = sum_n Kn[j, n] Qp[i, n], tiles (jt, it) = (0,0), (0,1), (1,1)
                    f32x4 S00 = zero4(), S01 = zero4(), S11 = zero4();
#pragma unroll
                    for (int ks = 0; ks < KSN; ++ks) {
                        const int o0 = l16 * LQ + 32 * ks + 8 * g4, o1 = o0 + 16 * LQ + kQPad;
                        const bf16x8 k0h = lds8(sKH + o0), k0l = lds8(sKL + o0);
                        const bf16x8 k1h = lds8(sKH + o1), k1l = lds8(sKL + o1);
                        const bf16x8 q0h = lds8(sQH + o0), q0l = lds8(sQL + o0);
                        const bf16x8 q1h = lds8(sQH + o1), q1l = lds8(sQL + o1);
                        S00 = mfma3(k0h, k0l, q0h, q0l, S00);
                        S01 = mfma3(k0h, k0l, q1h, q1l, S01);
                        S11 = mfma3(k1h, k1l, q1h, q1l, S11);
                    }
#pragma unroll
                    for (int rr = 0; rr < 4; ++rr) {   // causal mask j <= i inside the diagonal tiles
                        if (4 * g4 + rr > l16) {
                            S00[rr] = 0.f;
                            S11[rr] = 0.f;
                        }
                    }
                    // B operands over the 32-deep contraction j (rows {4g..4g+3} and {16+4g..16+4g+3})
                    bf16x8 sbh[2], sbl[2];
                    split8(S00, zero4(), sbh[0], sbl[0]);
                    split8(S01, S11, sbh[1], sbl[1]);

                    // ---- y^T[d, i] = sum_j V^T[d, j] S^T[j, i] + sum_n H^T[d, n] Qp^T[n, i]
                    f32x4 yacc[NDT][2];
#pragma unroll
                    for (int dt = 0; dt < NDT; ++dt) {
                        const bf16x8 va = lds_tr8(sVS, DVT, 4 * g4, 16 + 4 * g4, dl0 + 16 * dt, l16);
#pragma unroll
                        for (int it = 0; it < 2; ++it) yacc[dt][it] = mfma2b(va, sbh[it], sbl[it], zero4());
                    }
#pragma unroll
                    for (int ks = 0; ks < KSN; ++ks) {
                        bf16x8 qbh[2], qbl[2];
#pragma unroll
                        for (int it = 0; it < 2; ++it) {
                            const int qo = (16 * it + l16) * LQ + it * kQPad + 32 * ks + 4 * g4;
                            qbh[it] = lds4x2(sQH + qo, sQH + qo + 16);
                            qbl[it] = lds4x2(sQL + qo, sQL + qo + 16);
                        }
#pragma unroll
                        for (int dt = 0; dt < NDT; ++dt) {
                            bf16x8 hh, hl;
                            split8(Hs[2 * ks][dt], Hs[2 * ks + 1][dt], hh, hl);
#pragma unroll
                            for (int it = 0; it < 2; ++it) yacc[dt][it] = mfma3(hh, hl, qbh[it], qbl[it], yacc[dt][it]);
                        }
                        // the chunk-start state goes to the saved context a few rows at a time, between
                        // the products, so that the stores of all workgroups do not come in one burst
                        if (saved_H) {
                            save_rows(cc, 2 * ks);
                            save_rows(cc, 2 * ks + 1);
                        }
                    }
                    // y[t, d .. d+3] for t = 16 it + l16, d = dm0 + 16 dt + 4 g4
#pragma unroll
                    for (int it = 0; it < 2; ++it) {
                        const int t = 16 * it + l16;
                        if (t < nt) {
#pragma unroll
                            for (int dt = 0; dt < NDT; ++dt) {
                                const uint2 pk{cvt_pk_bf16(yacc[dt][it][0], yacc[dt][it][1]),
                                               cvt_pk_bf16(yacc[dt][it][2], yacc[dt][it][3])};
                                *reinterpret_cast<uint2*>(y + ((row0 + t) * H + h) * DV + dm0 + 16 * dt + 4 * g4) = pk;
                            }
                        }
                    }
                }

                // ---- state: H <- diag(P_C) (H + Kn^T V)
                const int tpad = g4 >= 2 ? kQPad : 0;   // tile rows 8 g4 .. 8 g4 + 7 past row 16
                bf16x8 vb[NDT];   // V rows t = 8 g4 .. 8 g4 + 7 of column d
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt) vb[dt] = lds_tr8(sVS, DVT, 8 * g4, 8 * g4 + 4, dl0 + 16 * dt, l16);
#pragma unroll
                for (int rt = 0; rt < NRT; ++rt) {
                    // Kn^T rows n = 16 rt + l16, tokens 8 g4 .. 8 g4 + 7
                    const bf16x8 kth = lds_tr8(sKH + tpad, LQ, 8 * g4, 8 * g4 + 4, 16 * rt, l16);
                    const bf16x8 ktl = lds_tr8(sKL + tpad, LQ, 8 * g4, 8 * g4 + 4, 16 * rt, l16);
                    const float4 dec = *reinterpret_cast<const float4*>(sDec + 16 * rt + 4 * g4);
#pragma unroll
                    for (int dt = 0; dt < NDT; ++dt) {
                        const f32x4 hacc = mfma2a(kth, ktl, vb[dt], Hs[rt][dt]);
                        Hs[rt][dt][0] = hacc[0] * dec.x;
                        Hs[rt][dt][1] = hacc[1] * dec.y;
                        Hs[rt][dt][2] = hacc[2] * dec.z;
                        Hs[rt][dt][3] = hacc[3] * dec.w;
                    }
                }

                // the chunk's walk state goes to the saved context (one value tile stores it)
                if (saved_lam && tile == 0) {
                    constexpr int NV4 = kLamRows * DK / 4;
                    const float4* src = reinterpret_cast<const float4*>(buf + Cfg::MIDS);
                    float4* dst = reinterpret_cast<float4*>(saved_lam + ((size_t)bh * nchunk + cc) * kLamRows * DK);
                    for (int i = m * 64 + lane; i < NV4; i += Cfg::NMW * 64) dst[i] = src[i];
                }

                if (YV && tile == 0 && m == 0 && lane < nt) {
                    const float* yv = reinterpret_cast<const float*>(buf + Cfg::YVP);
                    float acc = 0.f;
#pragma unroll
                    for (int w2 = 0; w2 < NSW; ++w2) acc += yv[w2 * kC + lane];
                    g.yvar[(row0 + lane) * H + h] = acc;
                }
            }
            barrier_lds();
        }

        if (saved_H)   // the final state closes the saved sequence
#pragma unroll
            for (int rt = 0; rt < NRT; ++rt) save_rows(nchunk, rt);
        if (g.etaT) {
#pragma unroll
            for (int rt = 0; rt < NRT; ++rt)
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
                    for (int rr = 0; rr < 4; ++rr)
                        g.etaT[((size_t)bh * DK + 16 * rt + 4 * g4 + rr) * DV + dm0 + 16 * dt + l16] = Hs[rt][dt][rr];
        }
    }
}

template <int DK, int DV, bool YV, bool TI, bool NOY = false>
hipError_t launch_fwd_v(const Shape& s, const FwdArgs& a, float* saved_lam, float* saved_H, hipStream_t st) {
    using Cfg = ChunkCfg<DK, DV>;
    auto kern = fwd_chunk_kernel<DK, DV, YV, TI, NOY>;
    // more than 64 KiB of LDS must be opted into once per kernel (thread-safe static init)
    static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                                       hipFuncAttributeMaxDynamicSharedMemorySize, Cfg::BYTES);
    if (attr != hipSuccess) return attr;
    const unsigned grid = (unsigned)(s.B * s.H * Cfg::NTILE);
    hipLaunchKernelGGL(kern, dim3(grid), dim3(Cfg::NTHR), Cfg::BYTES, st, s, a, saved_lam, saved_H);
    return hipGetLastError();
}

// the readout variance adds a cross-lane sum per token, so it is a separate
// instantiation, as are the time-invariant gates and the state-only pass (no y:
// the segment-parallel forward's first pass)
template <int DK, int DV>
hipError_t launch_fwd(const Shape& s, const FwdArgs& a, float* saved_lam, float* saved_H, hipStream_t st) {
    if (!a.y) return launch_fwd_v<DK, DV, false, false, true>(s, a, nullptr, nullptr, st);
    if (a.ou_a)
        return a.yvar ? launch_fwd_v<DK, DV, true, true>(s, a, saved_lam, saved_H, st)
                      : launch_fwd_v<DK, DV, false, true>(s, a, saved_lam, saved_H, st);
    return a.yvar ? launch_fwd_v<DK, DV, true, false>(s, a, saved_lam, saved_H, st)
                  : launch_fwd_v<DK, DV, false, false>(s, a, saved_lam, saved_H, st);
}

}  // namespace

bool chunked_supported(const Shape& s) { return s.bf16 && s.dk >= 32; }

// Saved context: the precision walk's state of every chunk [BH][nchunk][kLamRows][dk]
// (lam at the chunk start, lam_16 and P_16 after its first 16 tokens), then the
// information state at every chunk start and after the last token
// [BH][nchunk+1][dk][dv].
size_t chunked_saved_bytes(const Shape& s) {
    const size_t nchunk = (size_t)(s.T + kC - 1) / kC;
    return (size_t)s.B * s.H * s.dk * (kLamRows * nchunk + (nchunk + 1) * (size_t)s.dv) * sizeof(float);
}

hipError_t launch_forward_chunked(const Shape& s, const FwdArgs& a, void* saved, hipStream_t st) {
    float* saved_lam = nullptr;
    float* saved_H = nullptr;
    if (saved) {
        const size_t nchunk = (size_t)(s.T + kC - 1) / kC;
        saved_lam = static_cast<float*>(saved);
        saved_H = saved_lam + (size_t)s.B * s.H * nchunk * kLamRows * s.dk;
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
