// Chunked forward of the KLA filter on MFMA (bf16 inputs, fp32 state).
//
// The sequence is cut into chunks of kC = 32 tokens.  Within a chunk, for each
// key slot n, the precision path (Theorem 1) is walked token by token in
// homogeneous coordinates.  The Moebius update
//   lam_t = (lam + phi (abar^2 + pbar lam)) / (abar^2 + pbar lam),  phi = k^2 r,
// acts linearly on (x, z) with lam = x / z:
//   z_t = pbar_t x_{t-1} + abar_t^2 z_{t-1}     (so rho_t = z_{t-1} / z_t)
//   x_t = x_{t-1} + phi_t z_t
// and, with A_t = prod_{s<=t} abar_s, the running product of the forget gates
// F = abar rho (Theorem 2) inside the chunk is P_t = A_t / z_t (x = lam, z = 1,
// A = 1 at the chunk start).  With one reciprocal R = 1 / (x_t A_t) per token,
//   Qp[t, n] = (q_t / lam_t) P_t = q_t A_t (A_t R)
//   Kn[t, n] = (r_t k_t) / P_t   = r_t k_t z_t (x_t R)
// and the information-state recursion over the chunk is exactly
//   y    = mask(Qp Kn^T) V + Qp H                       (readout, Algorithm 1)
//   H   <- diag(P_C) (H + Kn^T V)                       (state at the chunk end)
// (the unrolled "attention matrix" of the paper's appendix, restricted to a
// chunk, plus the carried state).  The contractions run on
// v_mfma_f32_16x16x32_bf16 with split-bf16 operands for the fp32 factors
// (kla_mfma.hpp), accumulating in fp32.
//
// One workgroup per (batch, head, value tile of up to 64 channels), with two
// kinds of waves that work one chunk apart through a double-buffered LDS
// exchange and one barrier per chunk:
//   scan waves (64 key slots each) walk chunk c and write Qp and Kn ([t][n]),
//     the chunk decay P_C and the variance partials into buffer c & 1; their inputs arrive in LDS by direct 16-byte buffer loads, each
//     block of tokens requested for chunk c + 1 as soon as chunk c has walked
//     past it; they also bring chunk c's value tile into the buffer;
//   MFMA waves (32 value channels each, the state H[dk, 32] in registers)
//     meanwhile consume chunk c - 1: attention tiles, readout, y, state update;
//     operands that run across the rows of a tile (Kn^T, V) are read with
//     transposing LDS reads (lds_tr8), so each tile is stored once.
// All loads are issued by the scan waves, whose request stream is fixed, so
// each wait names exactly the requests it needs (vmcnt counts in issue order);
// the MFMA waves only store.
// Requirement (documented in the ABI): inside one chunk, prod abar,
// prod (abar^2 + pbar lam) and lam prod (abar^2 + pbar lam) stay in fp32 range.
#include "kla_buf.hpp"
#include "kla_internal.hpp"
#include "kla_mfma.hpp"

namespace kla {
namespace {

constexpr int kC = 32;         // tokens per chunk
constexpr int kSaveEvery = 2;  // the saved context holds every second chunk start (64-token chunks)

template <int DK, int DV>
struct FwdCfg {
    static constexpr int DVT = DV < 64 ? DV : 64;    // value channels per workgroup
    static constexpr int NTILE = DV / DVT;
    static constexpr int DCW = DVT < 32 ? DVT : 32;  // value channels per MFMA wave
    static constexpr int NDT = DCW / 16;
    static constexpr int NMW = DVT / DCW;            // MFMA waves
    static constexpr int SW = DK < 64 ? DK : 64;     // key slots per scan wave
    static constexpr int NSW = DK / SW;              // scan waves
    static constexpr int NTHR = 64 * (NSW + NMW);
    static constexpr int NRT = DK / 16;
    static constexpr int KSN = DK / 32;
    static constexpr int LQ = DK + 8;                // row stride of [t][n] (halfwords)
    // one exchange buffer (byte offsets)
    static constexpr int QH = 0, QL = QH + kC * LQ * 2, KH = QL + kC * LQ * 2, KL = KH + kC * LQ * 2;
    static constexpr int DEC = KL + kC * LQ * 2;     // P_C [DK] fp32
    static constexpr int YVP = DEC + DK * 4;         // variance partials [NSW][kC] fp32
    static constexpr int VS = (YVP + NSW * kC * 4 + 15) / 16 * 16;   // value tile [kC][DVT] bf16
    static constexpr int BUF = VS + kC * DVT * 2;
    static constexpr int NVL = kC * DVT * 2 / 1024;  // 1 KiB wave loads of the value tile
    static constexpr int TPV = kC / NVL;             // tokens per value-tile load
    // per scan wave: abar, pbar, k, q [4][kC][SW] bf16, then r [2][64] as zero-extended words
    static constexpr int STG = 2 * BUF;
    static constexpr int STG_WAVE = 4 * kC * SW * 2 + 2 * 64 * 4;
    static constexpr int BYTES = STG + NSW * STG_WAVE;
    static constexpr int TPL = 512 / SW;             // tokens per 16-byte-per-lane load (one block)
    static constexpr int NBLK = kC / TPL;
    static_assert(DK >= 32 && DK % 32 == 0, "chunked path needs dk >= 32");
    static_assert(NBLK >= 1 && NVL >= 1, "tile sizes");
    static_assert(BYTES <= 160 * 1024, "LDS budget of one workgroup");
};

// Outputs of the precision walk in one exchange buffer.
struct ScanOut {
    uint16_t *qh, *ql, *kh, *kl;   // [t][n]
    float* yv;                     // per-token wave sums of q^2 / lam
};

// Staged inputs of one group of 8 tokens for one key slot (raw bf16 / r words).
struct ScanGroup {
    uint32_t a[8], p[8], k[8], q[8];
    uint4 r[2];
};

template <int SW>
__device__ __forceinline__ void read_group(ScanGroup& gr, const uint16_t* __restrict__ stg,
                                           const uint32_t* __restrict__ rw, int sl, int t8) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        gr.a[e] = stg[(0 * kC + t8 + e) * SW + sl];
        gr.p[e] = stg[(1 * kC + t8 + e) * SW + sl];
        gr.k[e] = stg[(2 * kC + t8 + e) * SW + sl];
        gr.q[e] = stg[(3 * kC + t8 + e) * SW + sl];
    }
    gr.r[0] = *reinterpret_cast<const uint4*>(rw + t8);
    gr.r[1] = *reinterpret_cast<const uint4*>(rw + t8 + 4);
}

// Walk the tokens of one chunk for key slot n (lane), from the staged inputs
// (stg: [4][kC][SW] bf16; rw: r as words [kC]).  FULL: all kC tokens are valid
// (no per-token guards).  The inputs of the next group of 8 tokens are read
// from LDS before the current group is processed.  before(G) runs before group
// G is read (the wait for its staged inputs); after(j) after token block j
// (TPL tokens) is done (the request of the next chunk's block j).
template <int SW, int TPL, int LQ, bool YV, bool FULL, class Before, class After>
__device__ __forceinline__ void scan_tokens(const uint16_t* __restrict__ stg, const uint32_t* __restrict__ rw, int sl,
                                            int nt, bool active, int n, float& x, float& z, float& A,
                                            const ScanOut& o, Before before, After after) {
    ScanGroup gr[2];
    before(0);
    read_group<SW>(gr[0], stg, rw, sl, 0);
#pragma unroll
    for (int t8 = 0; t8 < kC; t8 += 8) {
        const ScanGroup& cur = gr[(t8 / 8) & 1];
        if (t8 + 8 < kC) {
            before((t8 + 8) / 8);
            read_group<SW>(gr[((t8 / 8) + 1) & 1], stg, rw, sl, t8 + 8);
        }
#pragma unroll
        for (int j2 = 0; j2 < 4; ++j2) {
            float qp2[2], kn2[2];
#pragma unroll
            for (int e = 0; e < 2; ++e) {
                const int t = t8 + 2 * j2 + e, i = 2 * j2 + e;
                const float av = __uint_as_float(cur.a[i] << 16);
                const float pv = __uint_as_float(cur.p[i] << 16);
                const float kv = __uint_as_float(cur.k[i] << 16);
                const float qv = __uint_as_float(cur.q[i] << 16);
                const uint32_t rword = i < 4 ? (&cur.r[0].x)[i] : (&cur.r[1].x)[i - 4];
                const float rv = __uint_as_float(rword << 16);
                const float kr = kv * rv;
                const float zn = fmaf(pv, x, av * av * z);
                const float xn = fmaf(kr * kv, zn, x);
                const float An = A * av;
                const float R = fast_rcp(xn * An);
                const float AR = An * R;   // 1 / x_t
                const bool ok = FULL || t < nt;
                const float qp = ok ? (qv * An) * AR : 0.f;
                const float kn = ok ? (kr * zn) * (xn * R) : 0.f;
                x = ok ? xn : x;
                z = ok ? zn : z;
                A = ok ? An : A;
                qp2[e] = qp;
                kn2[e] = kn;
                if constexpr (YV) {
                    const float w = (ok && active) ? qv * qv * zn * AR : 0.f;   // q^2 / lam_t
                    const float ws = wave_sum(w);
                    if (sl == 0) o.yv[t] = ws;
                }
            }
            uint32_t qh, ql, kh, kl;
            split2(qp2[0], qp2[1], qh, ql);
            split2(kn2[0], kn2[1], kh, kl);
            const int t = t8 + 2 * j2;
            if (active) {
                o.qh[t * LQ + n] = static_cast<uint16_t>(qh);
                o.qh[(t + 1) * LQ + n] = static_cast<uint16_t>(qh >> 16);
                o.ql[t * LQ + n] = static_cast<uint16_t>(ql);
                o.ql[(t + 1) * LQ + n] = static_cast<uint16_t>(ql >> 16);
                o.kh[t * LQ + n] = static_cast<uint16_t>(kh);
                o.kh[(t + 1) * LQ + n] = static_cast<uint16_t>(kh >> 16);
                o.kl[t * LQ + n] = static_cast<uint16_t>(kl);
                o.kl[(t + 1) * LQ + n] = static_cast<uint16_t>(kl >> 16);
            }
        }
        if ((t8 + 8) % TPL == 0) after((t8 + 8) / TPL - 1);
    }
}

template <int DK, int DV, bool YV>
__global__ __launch_bounds__((FwdCfg<DK, DV>::NTHR)) void fwd_chunk_kernel(Shape s, FwdArgs g, float* saved_lam,
                                                                         float* saved_H) {
    using Cfg = FwdCfg<DK, DV>;
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
    const int H = s.H, T = s.T;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform role
    const int l16 = lane & 15, g4 = lane >> 4;
    const int nchunk = (T + kC - 1) / kC;
    const int nsave = (T + kC * kSaveEvery - 1) / (kC * kSaveEvery);
    const size_t seq0 = (size_t)b * T;   // token index of this sequence's first token

    if (wave < NSW) {
        // ================================================================ scan waves
        const bool active = lane < SW;
        const int sl = active ? lane : 0;     // slot within this wave's staged rows
        const int n = wave * SW + sl;
        float x = (active && g.lam0) ? g.lam0[(size_t)bh * DK + n] : 1.f;   // lam at the chunk start
        unsigned char* stw = smem + Cfg::STG + wave * Cfg::STG_WAVE;
        uint16_t* stg = reinterpret_cast<uint16_t*>(stw);
        uint32_t* rw = reinterpret_cast<uint32_t*>(stw + 4 * kC * SW * 2);   // [2][64]
        const uint32_t tok_bytes = (uint32_t)H * DK * 2;
        // lane -> (token within a block, 8 slots); the load of a block lands as [t][SW] rows
        const uint32_t blk_voff = (uint32_t)(lane / (SW / 8)) * tok_bytes + (lane % (SW / 8)) * 16;

        // buffer descriptors of chunk cn (empty past the sequence: such loads write zeros)
        rsrc_t rs[4];
        auto chunk_rsrc = [&](int cn) {
            const int t0 = cn * kC, nt = min(kC, T - t0);
            const size_t e0 = ((seq0 + t0) * H + h) * DK + wave * SW;
            const uint32_t bytes = nt > 0 ? (uint32_t)((nt - 1) * H * DK + SW) * 2 : 0u;
            rs[0] = make_rsrc(a + e0, bytes);
            rs[1] = make_rsrc(p + e0, bytes);
            rs[2] = make_rsrc(k + e0, bytes);
            rs[3] = make_rsrc(q + e0, bytes);
        };
        auto issue_block = [&](int j) {
#pragma unroll
            for (int ti = 0; ti < 4; ++ti)
                buf_ld128_lds(rs[ti], stg + (ti * kC + j * Cfg::TPL) * SW, blk_voff + (uint32_t)j * Cfg::TPL * tok_bytes);
        };
        // this wave's share of the value-tile loads of chunk cn (loads i = wave, wave + NSW, ...)
        const int nvw = wave < Cfg::NVL ? (Cfg::NVL - wave + NSW - 1) / NSW : 0;
        const uint32_t v_voff = (uint32_t)(lane / (DVT / 8)) * H * DV * 2 + (lane % (DVT / 8)) * 16;
        auto issue_v = [&](int cn) {
            const int t0 = cn * kC, nt = min(kC, T - t0);
            const rsrc_t rv = make_rsrc(v + ((seq0 + t0) * H + h) * DV + tile * DVT,
                                        nt > 0 ? (uint32_t)((nt - 1) * H * DV + DVT) * 2 : 0u);
            unsigned char* vs = smem + (cn & 1) * Cfg::BUF + Cfg::VS;
            for (int i = wave; i < Cfg::NVL; i += NSW)
                buf_ld128_lds(rv, vs + i * 1024, v_voff + (uint32_t)(i * Cfg::TPV) * H * DV * 2);
        };
        auto issue_r = [&](int cn) {
            const int t0 = cn * kC, nt = min(kC, T - t0);
            const rsrc_t rr = make_rsrc(r + (seq0 + t0) * H + h, nt > 0 ? (uint32_t)((nt - 1) * H + 1) * 2 : 0u);
            buf_ld16_lds(rr, rw + (cn & 1) * 64, (uint32_t)lane * H * 2);   // lanes >= nt read as 0
        };
        wait_vm_all();   // the carried lam is complete before the prefetch loop starts
        if (nchunk > 0) {
            chunk_rsrc(0);
            issue_r(0);
#pragma unroll
            for (int j = 0; j < Cfg::NBLK; ++j) issue_block(j);
        }

        for (int c = 0; c <= nchunk; ++c) {
            if (c < nchunk) {
                const int nt = min(kC, T - c * kC);
                issue_v(c);
                issue_r(c + 1);
                chunk_rsrc(c + 1);
                if (saved_lam && c % kSaveEvery == 0 && active)
                    saved_lam[((size_t)bh * nsave + c / kSaveEvery) * DK + n] = x;

                unsigned char* buf = smem + (c & 1) * Cfg::BUF;
                ScanOut o;
                o.qh = reinterpret_cast<uint16_t*>(buf + Cfg::QH);
                o.ql = reinterpret_cast<uint16_t*>(buf + Cfg::QL);
                o.kh = reinterpret_cast<uint16_t*>(buf + Cfg::KH);
                o.kl = reinterpret_cast<uint16_t*>(buf + Cfg::KL);
                o.yv = reinterpret_cast<float*>(buf + Cfg::YVP) + wave * kC;
                // Group G starting block j is read while block j - 1 is processed (after
                // the next chunk's blocks before j - 1 went out).  Younger than block j's
                // loads are then: its later blocks, this chunk's value-tile loads (nvw),
                // r of the next chunk, possibly the saved-lam store, and those requests:
                // 4 (NBLK - 1) + 1 + nvw for j = 0, 4 (NBLK - 2) + 1 + nvw otherwise.
                auto before = [&](int G) {
                    if (G == 0)
                        wait_vm_le_rt<4 * (Cfg::NBLK - 1) + 1>(nvw);
                    else if ((8 * G) % Cfg::TPL == 0)
                        wait_vm_le_rt<4 * (Cfg::NBLK - 2) + 1>(nvw);
                };
                auto after = [&](int j) { issue_block(j); };
                const uint32_t* rwc = rw + (c & 1) * 64;
                float z = 1.f, A = 1.f;
                if (nt == kC)
                    scan_tokens<SW, Cfg::TPL, LQ, YV, true>(stg, rwc, sl, nt, active, n, x, z, A, o, before, after);
                else
                    scan_tokens<SW, Cfg::TPL, LQ, YV, false>(stg, rwc, sl, nt, active, n, x, z, A, o, before, after);
                const float iz = fast_rcp(z);
                x *= iz;   // lam at the chunk end
                if (active) reinterpret_cast<float*>(buf + Cfg::DEC)[n] = A * iz;
                // the value tile has landed (younger: r, the saved-lam store, NBLK blocks)
                wait_vm_le<4 * Cfg::NBLK + 1>();
            }
            barrier_lds();
        }
        wait_vm_all();   // the requests for the chunk past the end have landed before exit
        if (g.lamT && active && tile == 0) g.lamT[(size_t)bh * DK + n] = x;
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

        auto save_state = [&](int slot) {
            float* dst = saved_H + ((size_t)bh * (nsave + 1) + slot) * DK * DV;
#pragma unroll
            for (int rt = 0; rt < NRT; ++rt)
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
                if (saved_H && cc % kSaveEvery == 0) save_state(cc / kSaveEvery);

                const uint16_t* sQH = reinterpret_cast<const uint16_t*>(buf + Cfg::QH);
                const uint16_t* sQL = reinterpret_cast<const uint16_t*>(buf + Cfg::QL);
                const uint16_t* sKH = reinterpret_cast<const uint16_t*>(buf + Cfg::KH);
                const uint16_t* sKL = reinterpret_cast<const uint16_t*>(buf + Cfg::KL);
                const float* sDec = reinterpret_cast<const float*>(buf + Cfg::DEC);

                // ---- S^T[j, i] = sum_n Kn[j, n] Qp[i, n], tiles (jt, it) = (0,0), (0,1), (1,1)
                f32x4 S00 = zero4(), S01 = zero4(), S11 = zero4();
#pragma unroll
                for (int ks = 0; ks < KSN; ++ks) {
                    const int o0 = l16 * LQ + 32 * ks + 8 * g4, o1 = o0 + 16 * LQ;
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
                        const int qo = (16 * it + l16) * LQ + 32 * ks + 4 * g4;
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

                // ---- state: H <- diag(P_C) (H + Kn^T V)
                bf16x8 vb[NDT];   // V rows t = 8 g4 .. 8 g4 + 7 of column d
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt) vb[dt] = lds_tr8(sVS, DVT, 8 * g4, 8 * g4 + 4, dl0 + 16 * dt, l16);
#pragma unroll
                for (int rt = 0; rt < NRT; ++rt) {
                    // Kn^T rows n = 16 rt + l16, tokens 8 g4 .. 8 g4 + 7
                    const bf16x8 kth = lds_tr8(sKH, LQ, 8 * g4, 8 * g4 + 4, 16 * rt, l16);
                    const bf16x8 ktl = lds_tr8(sKL, LQ, 8 * g4, 8 * g4 + 4, 16 * rt, l16);
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

        if (saved_H) save_state(nsave);   // the final state closes the saved sequence
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

template <int DK, int DV, bool YV>
hipError_t launch_fwd_v(const Shape& s, const FwdArgs& a, float* saved_lam, float* saved_H, hipStream_t st) {
    using Cfg = FwdCfg<DK, DV>;
    auto kern = fwd_chunk_kernel<DK, DV, YV>;
    // more than 64 KiB of LDS must be opted into once per kernel (thread-safe static init)
    static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                                       hipFuncAttributeMaxDynamicSharedMemorySize, Cfg::BYTES);
    if (attr != hipSuccess) return attr;
    const unsigned grid = (unsigned)(s.B * s.H * Cfg::NTILE);
    hipLaunchKernelGGL(kern, dim3(grid), dim3(Cfg::NTHR), Cfg::BYTES, st, s, a, saved_lam, saved_H);
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

// Saved context over 64-token chunks: lam at every chunk start [BH][nsave][dk],
// then the information state at every chunk start and after the last token
// [BH][nsave+1][dk][dv].
size_t chunked_saved_bytes(const Shape& s) {
    const size_t nsave = (size_t)(s.T + kC * kSaveEvery - 1) / (kC * kSaveEvery);
    return (size_t)s.B * s.H * s.dk * (nsave + (nsave + 1) * (size_t)s.dv) * sizeof(float);
}

hipError_t launch_forward_chunked(const Shape& s, const FwdArgs& a, void* saved, hipStream_t st) {
    float* saved_lam = nullptr;
    float* saved_H = nullptr;
    if (saved) {
        const size_t nsave = (size_t)(s.T + kC * kSaveEvery - 1) / (kC * kSaveEvery);
        saved_lam = static_cast<float*>(saved);
        saved_H = saved_lam + (size_t)s.B * s.H * nsave * s.dk;
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
