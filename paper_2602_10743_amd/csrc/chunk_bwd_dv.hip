// Chunked backward, value side: dv and the adjoint of the information state.
//
// Walking the chunks (kC = 32 tokens, kla_chunk.hpp) from last to first, with
// G the adjoint of the chunk's last state coming from later tokens (detaT for
// the last chunk), Gs = diag(P_C) G and the forward attention
// A[i, j] = sum_n Qp[i, n] Kn[j, n] (j <= i):
//   dV = M(A)^T dY + Kn Gs          (gradient of the chunk's values)
//   G' = Qp^T dY + Gs               (carried into the previous chunk)
// the reverse-mode counterpart of the chunked readout and state update of the
// forward (Algorithm 1 unrolled over a chunk).  After the first chunk, G' is
// the gradient of the initial state eta0.
//
// One workgroup per (batch, head, value tile of up to 64 channels).  The scan
// waves redo the precision walk of each chunk, each half of it from its saved
// start state (lam_0; lam_16 and P_16), and stage the chunk's dY tile; the MFMA waves (16 value channels each, G[dk, 16]
// in registers) consume the previous round's chunk:
//   dV^T[d, j] = sum_i dY^T[d, i] A[i, j] + sum_n Gs^T[d, n] Kn^T[n, j]
//   G[n, d]   += sum_t Qp^T[n, t] dY[t, d]
// with the operands that run across tile rows (dY^T, Qp^T) read by
// transposing LDS reads.
#include "kla_chunk.hpp"
#include "kla_internal.hpp"

namespace kla {
namespace {

template <int DK, int DV, bool TI>
__global__ __launch_bounds__((ChunkCfg<DK, DV>::NTHR)) void bwd_dv_kernel(Shape s, BwdArgs g,
                                                                          const float* __restrict__ saved_lam) {
    using Cfg = ChunkCfg<DK, DV>;
    constexpr int DVT = Cfg::DVT, NTILE = Cfg::NTILE, DCW = Cfg::DCW, NDT = Cfg::NDT, NSW = Cfg::NSW;
    constexpr int NRT = Cfg::NRT, KSN = Cfg::KSN, LQ = Cfg::LQ;
    extern __shared__ __align__(16) unsigned char smem[];

    int bh, tile;
    xcd_tile_map(blockIdx.x, s.B * s.H, NTILE, bh, tile);
    const int b = bh / s.H, h = bh % s.H;
    const int H = s.H, T = s.T;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform role
    const int l16 = lane & 15, g4 = lane >> 4;
    const int nchunk = (T + kC - 1) / kC;
    const size_t seq0 = (size_t)b * T;

    if (wave < NSW) {
        const ScanSrc sc{static_cast<const uint16_t*>(g.a), static_cast<const uint16_t*>(g.p),
                         static_cast<const uint16_t*>(g.k), static_cast<const uint16_t*>(g.q),
                         static_cast<const uint16_t*>(g.r), static_cast<const uint16_t*>(g.dy),
                         tile * DVT, seq0, H, h, T, nchunk, bh, g.ou_a, g.ou_p, g.ou_d,
                         g.range_flag};
        scan_wave<Cfg, false, true, TI>(smem, wave, lane, sc, saved_lam, false);
        return;
    }

    // ==================================================================== MFMA waves
    uint16_t* dv = static_cast<uint16_t*>(g.dv);
    const int m = wave - NSW;
    const int dl0 = m * DCW;                // first column of this wave within the value tile
    const int dm0 = tile * DVT + dl0;       // its first value channel

    // G[n, d] for n = 16 rt + 4 g4 + rr, d = dm0 + 16 dt + l16
    f32x4 G[NRT][NDT];
#pragma unroll
    for (int rt = 0; rt < NRT; ++rt)
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
            for (int rr = 0; rr < 4; ++rr)
                G[rt][dt][rr] =
                    g.detaT ? g.detaT[((size_t)bh * DK + 16 * rt + 4 * g4 + rr) * DV + dm0 + 16 * dt + l16] : 0.f;

    for (int it = 0; it <= nchunk; ++it) {
        if (it >= 1) {
            const int c = nchunk - it;   // the chunk the scan waves walked in the previous round
            const int nt = min(kC, T - c * kC);
            const size_t row0 = seq0 + (size_t)c * kC;
            const unsigned char* buf = smem + ((it - 1) & 1) * Cfg::BUF;
            const uint16_t* sQH = reinterpret_cast<const uint16_t*>(buf + Cfg::QH);
            const uint16_t* sQL = reinterpret_cast<const uint16_t*>(buf + Cfg::QL);
            const uint16_t* sKH = reinterpret_cast<const uint16_t*>(buf + Cfg::KH);
            const uint16_t* sKL = reinterpret_cast<const uint16_t*>(buf + Cfg::KL);
            const uint16_t* sDY = reinterpret_cast<const uint16_t*>(buf + Cfg::VS);   // dY [t][DVT]
            const float* sDec = reinterpret_cast<const float*>(buf + Cfg::DEC);

            // ---- Gs = diag(P_C) G, in place
#pragma unroll
            for (int rt = 0; rt < NRT; ++rt) {
                const float4 dec = *reinterpret_cast<const float4*>(sDec + 16 * rt + 4 * g4);
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt) {
                    G[rt][dt][0] *= dec.x;
                    G[rt][dt][1] *= dec.y;
                    G[rt][dt][2] *= dec.z;
                    G[rt][dt][3] *= dec.w;
                }
            }

            // ---- A[i, j] = sum_n Qp[i, n] Kn[j, n], tiles (it, jt) = (0,0), (1,0), (1,1)
            f32x4 A00 = zero4(), A10 = zero4(), A11 = zero4();
#pragma unroll
            for (int ks = 0; ks < KSN; ++ks) {
                const int o0 = l16 * LQ + 32 * ks + 8 * g4, o1 = o0 + 16 * LQ + kQPad;
                const bf16x8 q0h = lds8(sQH + o0), q0l = lds8(sQL + o0);
                const bf16x8 q1h = lds8(sQH + o1), q1l = lds8(sQL + o1);
                const bf16x8 k0h = lds8(sKH + o0), k0l = lds8(sKL + o0);
                const bf16x8 k1h = lds8(sKH + o1), k1l = lds8(sKL + o1);
                A00 = mfma3(q0h, q0l, k0h, k0l, A00);
                A10 = mfma3(q1h, q1l, k0h, k0l, A10);
                A11 = mfma3(q1h, q1l, k1h, k1l, A11);
            }
#pragma unroll
            for (int rr = 0; rr < 4; ++rr) {   // causal mask i >= j inside the diagonal tiles
                if (4 * g4 + rr < l16) {
                    A00[rr] = 0.f;
                    A11[rr] = 0.f;
                }
            }
            // B operands over the 32-deep contraction i (rows {4g..4g+3} and {16+4g..16+4g+3})
            bf16x8 abh[2], abl[2];
            split8(A00, A10, abh[0], abl[0]);
            split8(zero4(), A11, abh[1], abl[1]);

            // ---- dV^T[d, j] = sum_i dY^T[d, i] A[i, j] + sum_n Gs^T[d, n] Kn^T[n, j]
            f32x4 vacc[NDT][2];
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) {
                const bf16x8 ya = lds_tr8(sDY, DVT, 4 * g4, 16 + 4 * g4, dl0 + 16 * dt, l16);
#pragma unroll
                for (int jt = 0; jt < 2; ++jt) vacc[dt][jt] = mfma2b(ya, abh[jt], abl[jt], zero4());
            }
#pragma unroll
            for (int ks = 0; ks < KSN; ++ks) {
                bf16x8 kbh[2], kbl[2];
#pragma unroll
                for (int jt = 0; jt < 2; ++jt) {
                    const int ko = (16 * jt + l16) * LQ + jt * kQPad + 32 * ks + 4 * g4;
                    kbh[jt] = lds4x2(sKH + ko, sKH + ko + 16);
                    kbl[jt] = lds4x2(sKL + ko, sKL + ko + 16);
                }
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt) {
                    bf16x8 gh, gl;
                    split8(G[2 * ks][dt], G[2 * ks + 1][dt], gh, gl);
#pragma unroll
                    for (int jt = 0; jt < 2; ++jt) vacc[dt][jt] = mfma3(gh, gl, kbh[jt], kbl[jt], vacc[dt][jt]);
                }
            }
            // dv[t, d .. d+3] for t = 16 jt + l16, d = dm0 + 16 dt + 4 g4
#pragma unroll
            for (int jt = 0; jt < 2; ++jt) {
                const int t = 16 * jt + l16;
                if (t < nt) {
#pragma unroll
                    for (int dt = 0; dt < NDT; ++dt) {
                        const uint2 pk{cvt_pk_bf16(vacc[dt][jt][0], vacc[dt][jt][1]),
                                       cvt_pk_bf16(vacc[dt][jt][2], vacc[dt][jt][3])};
                        *reinterpret_cast<uint2*>(dv + ((row0 + t) * H + h) * DV + dm0 + 16 * dt + 4 * g4) = pk;
                    }
                }
            }

            // ---- G <- Qp^T dY + Gs
            const int tpad = g4 >= 2 ? kQPad : 0;   // tile rows 8 g4 .. 8 g4 + 7 past row 16
            bf16x8 yb[NDT];   // dY rows t = 8 g4 .. 8 g4 + 7 of column d
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) yb[dt] = lds_tr8(sDY, DVT, 8 * g4, 8 * g4 + 4, dl0 + 16 * dt, l16);
#pragma unroll
            for (int rt = 0; rt < NRT; ++rt) {
                // Qp^T rows n = 16 rt + l16, tokens 8 g4 .. 8 g4 + 7
                const bf16x8 qth = lds_tr8(sQH + tpad, LQ, 8 * g4, 8 * g4 + 4, 16 * rt, l16);
                const bf16x8 qtl = lds_tr8(sQL + tpad, LQ, 8 * g4, 8 * g4 + 4, 16 * rt, l16);
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt) G[rt][dt] = mfma2a(qth, qtl, yb[dt], G[rt][dt]);
            }
        }
        barrier_lds();
    }

    if (g.deta0) {
#pragma unroll
        for (int rt = 0; rt < NRT; ++rt)
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
                for (int rr = 0; rr < 4; ++rr)
                    g.deta0[((size_t)bh * DK + 16 * rt + 4 * g4 + rr) * DV + dm0 + 16 * dt + l16] = G[rt][dt][rr];
    }
}

template <int DK, int DV, bool TI>
hipError_t launch_dv(const Shape& s, const BwdArgs& a, const float* saved_lam, hipStream_t st) {
    using Cfg = ChunkCfg<DK, DV>;
    auto kern = bwd_dv_kernel<DK, DV, TI>;
    static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                                       hipFuncAttributeMaxDynamicSharedMemorySize, Cfg::BYTES);
    if (attr != hipSuccess) return attr;
    hipLaunchKernelGGL(kern, dim3((unsigned)(s.B * s.H * Cfg::NTILE)), dim3(Cfg::NTHR), Cfg::BYTES, st, s, a,
                       saved_lam);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_backward_dv(const Shape& s, const BwdArgs& a, const float* saved_lam, hipStream_t st) {
#define KLA_DV_CASE(DK_, DV_)                                          \
    if (s.dk == DK_ && s.dv == DV_)                                    \
        return a.ou_a ? launch_dv<DK_, DV_, true>(s, a, saved_lam, st) \
                      : launch_dv<DK_, DV_, false>(s, a, saved_lam, st);
#define KLA_DV_ROW(DK_) KLA_DV_CASE(DK_, 32) KLA_DV_CASE(DK_, 64) KLA_DV_CASE(DK_, 128)
    KLA_DV_ROW(32) KLA_DV_ROW(64) KLA_DV_ROW(128)
#undef KLA_DV_ROW
#undef KLA_DV_CASE
    return hipErrorInvalidValue;
}

}  // namespace kla
