// Chunk geometry and the precision-walk ("scan") waves shared by the chunked
// forward and the chunked value-side backward.
//
// Chunks hold kC = 32 tokens.  For key slot n the precision path (Theorem 1)
// is walked token by token in homogeneous coordinates: the Moebius update
//   lam_t = (lam + phi (abar^2 + pbar lam)) / (abar^2 + pbar lam),  phi = k^2 r,
// acts linearly on (x, z) with lam = x / z:
//   z_t = pbar_t x_{t-1} + abar_t^2 z_{t-1}     (so rho_t = z_{t-1} / z_t)
//   x_t = x_{t-1} + phi_t z_t
// and, with A_t = prod_{s<=t} abar_s, the running product of the forget gates
// F = abar rho (Theorem 2) inside the chunk is P_t = A_t / z_t (x = lam, z = 1,
// A = 1 at the chunk start).  With one reciprocal R = 1 / (x_t A_t) per token,
//   Qp[t, n] = (q_t / lam_t) P_t = q_t A_t (A_t R)
//   Kn[t, n] = (r_t k_t) / P_t   = r_t k_t z_t (x_t R)
// Requirement (documented in the ABI): inside one chunk, prod abar,
// prod (abar^2 + pbar lam) and lam prod (abar^2 + pbar lam) stay in fp32 range.
//
// A workgroup runs NSW scan waves (64 key slots each) beside NMW MFMA waves
// (32 value channels each).  Round i of the chunk loop: the scan waves walk
// chunk c(i) into exchange buffer i & 1 -- Qp and Kn as split-bf16 [t][n]
// tiles, the chunk decay P_C, optionally the per-token variance partials --
// and bring that chunk's tile of a per-token value tensor (v or dy) into the
// same buffer, while the MFMA waves consume buffer (i - 1) & 1.  One
// LDS-ordering barrier ends each round.  The scan waves issue every load of
// the workgroup, straight into LDS (16-byte buffer loads), and request each
// token block of the next chunk as soon as the current chunk has walked past
// it; since their request stream is fixed, each wait names exactly the
// requests it needs.
#pragma once
#include "kla_buf.hpp"
#include "kla_mfma.hpp"

namespace kla {

constexpr int kC = 32;   // tokens per chunk

template <int DK_, int DV_>
struct ChunkCfg {
    static constexpr int DK = DK_, DV = DV_;
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
    static constexpr int LQ = DK + 8;                // row stride of [t][n] tiles (halfwords)
    // one exchange buffer (byte offsets)
    static constexpr int QH = 0, QL = QH + kC * LQ * 2, KH = QL + kC * LQ * 2, KL = KH + kC * LQ * 2;
    static constexpr int DEC = KL + kC * LQ * 2;     // P_C [DK] fp32
    static constexpr int YVP = DEC + DK * 4;         // variance partials [NSW][kC] fp32
    static constexpr int VS = (YVP + NSW * kC * 4 + 15) / 16 * 16;   // value tile [kC][DVT] bf16
    static constexpr int BUF = VS + kC * DVT * 2;
    static constexpr int NVL = kC * DVT * 2 / 1024;  // 1 KiB wave loads of the value tile
    static constexpr int TPV = kC / NVL;             // tokens per value-tile load
    // per scan wave: abar, pbar, k, q [4][kC][SW] bf16, r [2][64] and the chunk-start
    // lam [2][64] as words
    static constexpr int STG = 2 * BUF;
    static constexpr int STG_R = 4 * kC * SW * 2, STG_L = STG_R + 2 * 64 * 4;
    static constexpr int STG_WAVE = STG_L + 2 * 64 * 4;
    static constexpr int BYTES = STG + NSW * STG_WAVE;
    static constexpr int TPL = 512 / SW;             // tokens per 16-byte-per-lane load (one block)
    static constexpr int NBLK = kC / TPL;
    static_assert(DK >= 32 && DK % 32 == 0, "chunked path needs dk >= 32");
    static_assert(NBLK >= 2 && NVL >= 1, "tile sizes");
    static_assert(BYTES <= 160 * 1024, "LDS budget of one workgroup");
};

// workgroup -> (b * H + h, value tile); the tiles of one (b, h) share an XCD (and its L2)
__device__ __forceinline__ void xcd_tile_map(int i, int nbh, int ntile, int& bh, int& tile) {
    if (nbh % 8 == 0) {
        const int xcd = i % 8, slot = i / 8;
        tile = slot % ntile;
        bh = (slot / ntile) * 8 + xcd;
    } else {
        tile = i % ntile;
        bh = i / ntile;
    }
}

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

// Sequence and tensors of one scan-wave loop.
struct ScanSrc {
    const uint16_t *a, *p, *k, *q, *r;   // [B, T, H, DK] (r: [B, T, H])
    const uint16_t* tile;                 // per-token value tensor [B, T, H, DV] staged per chunk
    int tcol0;                            // first column of the value tile
    size_t seq0;                          // b * T
    int H, h, T, nchunk, bh;
};

// The scan-wave loop: nchunk + 1 rounds, each ended by barrier_lds().  The walk
// order is c = 0 .. nchunk-1 (REV = false: lam carried from lam_in, the
// chunk-start lam stored to save_lam when given) or c = nchunk-1 .. 0 (REV:
// the chunk-start lam read from lam_in [BH][nchunk][DK]).  Returns the lam
// after the last walked token (forward order) for key slot wave * SW + lane.
template <class Cfg, bool YV, bool REV>
__device__ __forceinline__ float scan_wave(unsigned char* smem, int wave, int lane, const ScanSrc& sc,
                                           const float* __restrict__ lam_in, float* __restrict__ save_lam) {
    constexpr int DK = Cfg::DK, DV = Cfg::DV, DVT = Cfg::DVT, SW = Cfg::SW, NSW = Cfg::NSW;
    constexpr int NL = REV ? 1 : 0;   // chunk-start lam requests per round
    const int H = sc.H, h = sc.h, T = sc.T, nchunk = sc.nchunk;
    const bool active = lane < SW;
    const int sl = active ? lane : 0;   // slot within this wave's staged rows
    const int n = wave * SW + sl;
    float x = 1.f;                      // lam at the chunk start
    if (!REV && active && lam_in) x = lam_in[(size_t)sc.bh * DK + n];
    unsigned char* stw = smem + Cfg::STG + wave * Cfg::STG_WAVE;
    uint16_t* stg = reinterpret_cast<uint16_t*>(stw);
    uint32_t* rw = reinterpret_cast<uint32_t*>(stw + Cfg::STG_R);   // [2][64]
    float* lw = reinterpret_cast<float*>(stw + Cfg::STG_L);         // [2][64]
    const uint32_t tok_bytes = (uint32_t)H * DK * 2;
    // lane -> (token within a block, 8 slots); the load of a block lands as [t][SW] rows
    const uint32_t blk_voff = (uint32_t)(lane / (SW / 8)) * tok_bytes + (lane % (SW / 8)) * 16;
    auto chunk_of = [&](int it) { return REV ? nchunk - 1 - it : it; };

    // buffer descriptors of chunk cn; chunks outside the sequence get empty
    // descriptors, whose loads write zeros
    rsrc_t rs[4];
    auto chunk_rsrc = [&](int cn) {
        const bool in = cn >= 0 && cn < nchunk;
        const int t0 = in ? cn * kC : 0, nt = in ? min(kC, T - t0) : 0;
        const size_t e0 = ((sc.seq0 + t0) * H + h) * DK + wave * SW;
        const uint32_t bytes = nt > 0 ? (uint32_t)((nt - 1) * H * DK + SW) * 2 : 0u;
        rs[0] = make_rsrc(sc.a + e0, bytes);
        rs[1] = make_rsrc(sc.p + e0, bytes);
        rs[2] = make_rsrc(sc.k + e0, bytes);
        rs[3] = make_rsrc(sc.q + e0, bytes);
    };
    auto issue_block = [&](int j) {
#pragma unroll
        for (int ti = 0; ti < 4; ++ti)
            buf_ld128_lds(rs[ti], stg + (ti * kC + j * Cfg::TPL) * SW, blk_voff + (uint32_t)j * Cfg::TPL * tok_bytes);
    };
    // this wave's share of the value-tile loads (loads i = wave, wave + NSW, ...)
    const int nvw = wave < Cfg::NVL ? (Cfg::NVL - wave + NSW - 1) / NSW : 0;
    const uint32_t v_voff = (uint32_t)(lane / (DVT / 8)) * H * DV * 2 + (lane % (DVT / 8)) * 16;
    auto issue_tile = [&](int cn, int it) {
        const int t0 = cn * kC, nt = min(kC, T - t0);
        const rsrc_t rv = make_rsrc(sc.tile + ((sc.seq0 + t0) * H + h) * DV + sc.tcol0,
                                    (uint32_t)((nt - 1) * H * DV + DVT) * 2);
        unsigned char* vs = smem + (it & 1) * Cfg::BUF + Cfg::VS;
        for (int i = wave; i < Cfg::NVL; i += NSW)
            buf_ld128_lds(rv, vs + i * 1024, v_voff + (uint32_t)(i * Cfg::TPV) * H * DV * 2);
    };
    // r of chunk cn (lanes >= nt read as 0) and, walking backwards, its start lam
    auto issue_rl = [&](int cn, int it) {
        const bool in = cn >= 0 && cn < nchunk;
        const int t0 = in ? cn * kC : 0, nt = in ? min(kC, T - t0) : 0;
        const rsrc_t rr = make_rsrc(sc.r + (sc.seq0 + t0) * H + h, nt > 0 ? (uint32_t)((nt - 1) * H + 1) * 2 : 0u);
        buf_ld16_lds(rr, rw + (it & 1) * 64, (uint32_t)lane * H * 2);
        if constexpr (REV) {
            const rsrc_t rl = make_rsrc(lam_in + ((size_t)sc.bh * nchunk + (in ? cn : 0)) * DK + wave * SW,
                                        in ? (uint32_t)SW * 4 : 0u);
            buf_ld32_lds(rl, lw + (it & 1) * 64, (uint32_t)lane * 4);
        }
    };
    wait_vm_all();   // the carried lam is complete before the prefetch loop starts
    if (nchunk > 0) {
        chunk_rsrc(chunk_of(0));
        issue_rl(chunk_of(0), 0);
#pragma unroll
        for (int j = 0; j < Cfg::NBLK; ++j) issue_block(j);
    }

    for (int it = 0; it <= nchunk; ++it) {
        if (it < nchunk) {
            const int c = chunk_of(it), cn = chunk_of(it + 1);
            const int nt = min(kC, T - c * kC);
            issue_tile(c, it);
            issue_rl(cn, it + 1);
            chunk_rsrc(cn);
            if (!REV && save_lam && active) save_lam[((size_t)sc.bh * nchunk + c) * DK + n] = x;

            unsigned char* buf = smem + (it & 1) * Cfg::BUF;
            ScanOut o;
            o.qh = reinterpret_cast<uint16_t*>(buf + Cfg::QH);
            o.ql = reinterpret_cast<uint16_t*>(buf + Cfg::QL);
            o.kh = reinterpret_cast<uint16_t*>(buf + Cfg::KH);
            o.kl = reinterpret_cast<uint16_t*>(buf + Cfg::KL);
            o.yv = reinterpret_cast<float*>(buf + Cfg::YVP) + wave * kC;
            // Group G starting block j is read while block j - 1 is processed (after
            // the next chunk's blocks before j - 1 went out).  Younger than block j's
            // loads are then: its later blocks, this chunk's value-tile loads (nvw),
            // r (and lam) of the next chunk, possibly the saved-lam store, and those
            // requests: 4 (NBLK - 1) + 1 + NL + nvw for j = 0, 4 (NBLK - 2) + 1 + NL +
            // nvw otherwise.  The chunk-start lam was requested before block 0.
            auto before = [&](int G) {
                if (G == 0) {
                    wait_vm_le_rt<4 * (Cfg::NBLK - 1) + 1 + NL>(nvw);
                    if constexpr (REV) x = lw[(it & 1) * 64 + sl];
                } else if ((8 * G) % Cfg::TPL == 0) {
                    wait_vm_le_rt<4 * (Cfg::NBLK - 2) + 1 + NL>(nvw);
                }
            };
            auto after = [&](int j) { issue_block(j); };
            const uint32_t* rwc = rw + (it & 1) * 64;
            float z = 1.f, A = 1.f;
            if (nt == kC)
                scan_tokens<SW, Cfg::TPL, Cfg::LQ, YV, true>(stg, rwc, sl, nt, active, n, x, z, A, o, before, after);
            else
                scan_tokens<SW, Cfg::TPL, Cfg::LQ, YV, false>(stg, rwc, sl, nt, active, n, x, z, A, o, before, after);
            const float iz = fast_rcp(z);
            x *= iz;   // lam at the chunk end
            if (active) reinterpret_cast<float*>(buf + Cfg::DEC)[n] = A * iz;
            // the value tile has landed (younger: r, lam, the saved-lam store, NBLK blocks)
            wait_vm_le<4 * Cfg::NBLK + 1 + NL>();
        }
        barrier_lds();
    }
    wait_vm_all();   // the requests for the chunk past the end have landed before exit
    return x;
}

}  // namespace kla
