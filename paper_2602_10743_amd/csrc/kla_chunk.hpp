// Chunk geometry and the precision-walk ("scan") waves shared by the chunked
// forward and the chunked value-side backward.
//
// Chunks hold kC = 32 tokens.  For key slot n the precision path (Theorem 1)
// is walked token by token in homogeneous coordinates: the Moebius update
//   lam_t = (lam + phi (abar^2 + pbar lam)) / (abar^2 + pbar lam),  phi = k^2 r,
// acts linearly on (x, z) with lam = x / z:
//   z_t = pbar_t x_{t-1} + abar_t^2 z_{t-1}     (so rho_t = z_{t-1} / z_t)
//   x_t = x_{t-1} + phi_t z_t
// i.e. (x, z) is multiplied by Theorem 1's matrix [[1 + pbar phi, abar^2 phi],
// [pbar, abar^2]].  With A_t = prod_{s<=t} abar_s, the running product of the
// forget gates F = abar rho (Theorem 2) inside the chunk is P_t = A_t / z_t
// (x = lam, z = 1, A = 1 at the chunk start).  With one reciprocal
// R = 1 / (x_t A_t) per token,
//   Qp[t, n] = (q_t / lam_t) P_t = q_t A_t (A_t R)
//   Kn[t, n] = (r_t k_t) / P_t   = r_t k_t z_t (x_t R)
// Requirement (documented in the ABI): inside one chunk, prod abar,
// prod (abar^2 + pbar lam) and lam prod (abar^2 + pbar lam) stay in fp32 range.
//
// A workgroup runs NSW scan waves (32 key slots each) beside NMW MFMA waves
// (16 value channels each).  A scan-wave lane owns one key slot and one half of
// the chunk (tokens 16 h .. 16 h + 15, h = lane / 32).  The second half needs
// the state after token 15 before it can start, so each lane first composes
// the 2x2 matrices of 8 tokens -- tokens 0..7 in half 0, 8..15 in half 1 --,
// the half-1 lane takes its partner's product through a cross-lane exchange and
// applies both to the chunk start (lam, 1); then both halves walk their 16
// tokens side by side, and the half-1 lanes end at the chunk end.
//
// Round i of the chunk loop: the scan waves walk chunk c(i) into exchange
// buffer i & 1 -- Qp and Kn as split-bf16 [t][n] tiles, the chunk decay P_C,
// optionally the per-token variance partials -- and bring that chunk's tile of
// a per-token value tensor (v or dy) into the same buffer, while the MFMA waves
// consume buffer (i - 1) & 1.  One LDS-ordering barrier ends each round.  The
// scan waves issue every load of the workgroup, straight into LDS (16-byte
// buffer loads); their input staging is double-buffered: at the start of round
// i they request all inputs of chunk c(i + 1) and then wait for those of chunk
// c(i), requested one round earlier.
//
// TI (time-invariant gates, from the OU parameters of Sec. 4.1): abar and pbar
// are the same for every token of a key slot; each lane forms them once and the
// staging carries only k, q and r.  NOQ (a pass that only carries the state):
// the query is neither staged nor turned into Qp.
#pragma once
#include <type_traits>

#include "kla_buf.hpp"
#include "kla_mfma.hpp"

namespace kla {

constexpr int kC = 32;   // tokens per chunk

// LDS placement of the per-chunk [t][...] tiles written by the two halves of a scan
// wave.  Lane l of a wave works on token rows of half l / 32; the rows 16 apart would
// otherwise fall on the same LDS banks, so the second 16 rows of every tile start
// 64 bytes (16 banks) further on: Qp / Kn tiles after kQPad extra halfwords, the
// staged inputs one spare row of SW = 32 slots later (kSR rows per input).
constexpr int kQPad = 32;
constexpr int kSR = kC + 1;
__device__ __forceinline__ constexpr int srow(int t) { return t + (t >> 4); }
constexpr int kLamRows = 3;   // saved walk state per chunk and key slot: lam_0, lam_16, P_16

// x of lane l ^ 32, as seen by the lanes of one half: hi32 is valid in lanes 32..63
// (the partner's value from lanes 0..31), lo32 in lanes 0..31.  One lane-swap
// instruction, no LDS round trip.
struct Swap32 {
    float hi32, lo32;
};
__device__ __forceinline__ Swap32 swap32(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return {__uint_as_float(r[0]), __uint_as_float(r[1])};
}

template <int DK_, int DV_>
struct ChunkCfg {
    static constexpr int DK = DK_, DV = DV_;
    static constexpr int DVT = DV < 64 ? DV : 64;    // value channels per workgroup
    static constexpr int NTILE = DV / DVT;
    static constexpr int DCW = 16;                   // value channels per MFMA wave
    static constexpr int NDT = DCW / 16;
    static constexpr int NMW = DVT / DCW;            // MFMA waves
    static constexpr int SW = 32;                    // key slots per scan wave
    static constexpr int NSW = DK / SW;              // scan waves
    static constexpr int NTHR = 64 * (NSW + NMW);
    static constexpr int NRT = DK / 16;
    static constexpr int KSN = DK / 32;
    static constexpr int LQ = DK + 8;                // row stride of [t][n] tiles (halfwords)
    static constexpr int QPAD = kQPad;               // extra halfwords before row 16 of a tile
    static constexpr int QT = kC * LQ + QPAD;        // one [t][n] tile (halfwords)
    // one exchange buffer (byte offsets)
    static constexpr int QH = 0, QL = QH + QT * 2, KH = QL + QT * 2, KL = KH + QT * 2;
    static constexpr int DEC = KL + QT * 2;          // P_C [DK] fp32
    static constexpr int MIDS = DEC + DK * 4;        // walk state [kLamRows][DK] fp32
    static constexpr int YVP = MIDS + kLamRows * DK * 4;   // variance partials [NSW][kC] fp32
    static constexpr int VS = (YVP + NSW * kC * 4 + 15) / 16 * 16;   // value tile [kC][DVT] bf16
    static constexpr int BUF = VS + kC * DVT * 2;
    static constexpr int NVL = kC * DVT * 2 / 1024;  // 1 KiB wave loads of the value tile
    static constexpr int TPV = kC / NVL;             // tokens per value-tile load
    // per scan wave: abar, pbar, k, q [2 buffers][4][kSR][SW] bf16 (token t in row
    // t + t / 16), then r [2][64] and the saved walk state [2][2][64] as words
    static constexpr int STG = 2 * BUF;
    static constexpr int STG_IN = 4 * kSR * SW * 2;  // one buffer of staged inputs
    static constexpr int STG_R = 2 * STG_IN, STG_L = STG_R + 2 * 64 * 4;
    static constexpr int STG_WAVE = STG_L + 2 * 128 * 4;
    static constexpr int BYTES = STG + NSW * STG_WAVE;
    static_assert(DK >= 32 && DK % 32 == 0, "chunked path needs dk >= 32");
    static_assert(DVT % 16 == 0 && NVL >= 1 && NVL * TPV == kC, "value tile sizes");
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
    float* dec;                    // P_C [n]
    float* yv;                     // per-token sums of q^2 / lam over this wave's slots
    float* mid;                    // the chunk's walk state [kLamRows][n] (see scan_wave)
};

// Staged inputs of 8 consecutive tokens for one key slot (raw bf16 / r words;
// a and p unused with time-invariant gates).
struct ScanGroup {
    uint32_t a[8], p[8], k[8], q[8];
    uint4 r[2];
};

template <int SW, bool TI, bool NOQ>
__device__ __forceinline__ void read_group(ScanGroup& gr, const uint16_t* __restrict__ stg,
                                           const uint32_t* __restrict__ rw, int sl, int t8) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const int row = srow(t8 + e);
        if constexpr (!TI) {
            gr.a[e] = stg[(0 * kSR + row) * SW + sl];
            gr.p[e] = stg[(1 * kSR + row) * SW + sl];
        }
        gr.k[e] = stg[(2 * kSR + row) * SW + sl];
        if constexpr (!NOQ) gr.q[e] = stg[(3 * kSR + row) * SW + sl];
    }
    gr.r[0] = *reinterpret_cast<const uint4*>(rw + t8);
    gr.r[1] = *reinterpret_cast<const uint4*>(rw + t8 + 4);
}

__device__ __forceinline__ float bf16w(uint32_t w) { return __uint_as_float(w << 16); }

// One chunk of the walk for key slot n (lane: slot sl, half hf) from the staged
// inputs (stg: [4][kC][SW] bf16; rw: r as words [kC]), starting from the chunk-
// start lam x.  FULL: all kC tokens are valid (no per-token guards).  TI: the
// gates are the lane's ca, cp for every token.  Returns the lam at the chunk end
// in every lane.  chk accumulates Qp Kn (= q r k / lam, of modest size) over the
// lane's tokens (NOQ: 0 Kn): it stays finite exactly while every Qp and Kn is.
// lm, pm: the walk's state after token 15 in half 1, as lam_16 and P_16 = A_16 /
// z_16 (the state (x, z, A) scaled by 1 / z_16, which leaves every Qp, Kn, lam
// and P of the later tokens unchanged).  MID: the walk starts from such a saved
// state instead, x = lam_0 in half 0 and lam_16 in half 1, pm = P_16 in half 1,
// so neither the 8-token products nor the exchanges between the halves are
// needed; the return value is then the half's own end lam (the chunk end in
// half 1 only).
template <int SW, int LQ, bool YV, bool FULL, bool TI, bool NOQ, bool MID = false>
__device__ __forceinline__ float scan_chunk(const uint16_t* __restrict__ stg, const uint32_t* __restrict__ rw,
                                            int sl, int hf, int n, int nt, float x, const ScanOut& o, float ca,
                                            float cp, float& chk, float& lm, float& pm) {
    float xw, zw, Aw;
    if constexpr (MID) {
        xw = x;
        zw = 1.f;
        Aw = hf ? pm : 1.f;
    } else {
        // ---- the 2x2 product of this lane's 8 tokens 8 hf .. 8 hf + 7, as the images of
        // (1, 0) and (0, 1), with the product of abar
        float m00 = 1.f, m10 = 0.f, m01 = 0.f, m11 = 1.f, aq = 1.f;
        {
            float ta[8], tp[8], tk[8], tr[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int t = 8 * hf + j;
                ta[j] = TI ? ca : bf16w(stg[(0 * kSR + t) * SW + sl]);
                tp[j] = TI ? cp : bf16w(stg[(1 * kSR + t) * SW + sl]);
                tk[j] = bf16w(stg[(2 * kSR + t) * SW + sl]);
                tr[j] = bf16w(rw[t]);
            }
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const float a2 = ta[j] * ta[j], phi = tk[j] * tk[j] * tr[j];
                const float z0 = fmaf(tp[j], m00, a2 * m10), z1 = fmaf(tp[j], m01, a2 * m11);
                const float x0 = fmaf(phi, z0, m00), x1 = fmaf(phi, z1, m01);
                const bool ok = FULL || 8 * hf + j < nt;
                m00 = ok ? x0 : m00;
                m10 = ok ? z0 : m10;
                m01 = ok ? x1 : m01;
                m11 = ok ? z1 : m11;
                aq = ok ? aq * ta[j] : aq;
            }
        }
        // ---- the start of this lane's half: (lam, 1, 1) in half 0; in half 1 the partner's
        // product (tokens 0..7) and then its own (8..15) applied to (lam, 1)
        const float p00 = swap32(m00).hi32, p10 = swap32(m10).hi32;   // used by half 1 only
        const float p01 = swap32(m01).hi32, p11 = swap32(m11).hi32;
        const float pa = swap32(aq).hi32;
        const float x8 = fmaf(p00, x, p01), z8 = fmaf(p10, x, p11);
        xw = hf ? fmaf(m00, x8, m01 * z8) : x;
        zw = hf ? fmaf(m10, x8, m11 * z8) : 1.f;
        Aw = hf ? aq * pa : 1.f;
        const float iz16 = fast_rcp(zw);
        lm = xw * iz16;
        pm = Aw * iz16;
    }

    // ---- walk tokens 16 hf .. 16 hf + 15 (inputs of the next 8 read before the current 8)
    const int tb = 16 * hf;
    ScanGroup gr[2];
    read_group<SW, TI, NOQ>(gr[0], stg, rw, sl, tb);
#pragma unroll
    for (int g = 0; g < 2; ++g) {
        const ScanGroup& cur = gr[g];
        if (g == 0) read_group<SW, TI, NOQ>(gr[1], stg, rw, sl, tb + 8);
#pragma unroll
        for (int j2 = 0; j2 < 4; ++j2) {
            float qp2[2], kn2[2];
#pragma unroll
            for (int e = 0; e < 2; ++e) {
                const int i = 2 * j2 + e, t = tb + 8 * g + i;
                const float av = TI ? ca : bf16w(cur.a[i]), pv = TI ? cp : bf16w(cur.p[i]);
                const float kv = bf16w(cur.k[i]), qv = NOQ ? 0.f : bf16w(cur.q[i]);
                const uint32_t rword = i < 4 ? (&cur.r[0].x)[i] : (&cur.r[1].x)[i - 4];
                const float rv = bf16w(rword);
                const float kr = kv * rv;
                const float zn = fmaf(pv, xw, av * av * zw);
                const float xn = fmaf(kr * kv, zn, xw);
                const float An = Aw * av;
                const float R = fast_rcp(xn * An);
                const float AR = An * R;   // 1 / x_t
                const bool ok = FULL || t < nt;
                qp2[e] = ok ? (qv * An) * AR : 0.f;
                kn2[e] = ok ? (kr * zn) * (xn * R) : 0.f;
                chk = fmaf(NOQ ? 0.f : qp2[e], kn2[e], chk);
                xw = ok ? xn : xw;
                zw = ok ? zn : zw;
                Aw = ok ? An : Aw;
                if constexpr (YV) {
                    const float w = ok ? qv * qv * zn * AR : 0.f;   // q^2 / lam_t
                    const float ws = half_sum(w);
                    if (sl == SW - 1) o.yv[t] = ws;
                }
            }
            uint32_t qh, ql, kh, kl;
            if constexpr (!NOQ) split2(qp2[0], qp2[1], qh, ql);
            split2(kn2[0], kn2[1], kh, kl);
            const int t = tb + 8 * g + 2 * j2;
            const int e0 = t * LQ + hf * kQPad + n, e1 = e0 + LQ;   // rows t, t + 1
            if constexpr (!NOQ) {
                o.qh[e0] = static_cast<uint16_t>(qh);
                o.qh[e1] = static_cast<uint16_t>(qh >> 16);
                o.ql[e0] = static_cast<uint16_t>(ql);
                o.ql[e1] = static_cast<uint16_t>(ql >> 16);
            }
            o.kh[e0] = static_cast<uint16_t>(kh);
            o.kh[e1] = static_cast<uint16_t>(kh >> 16);
            o.kl[e0] = static_cast<uint16_t>(kl);
            o.kl[e1] = static_cast<uint16_t>(kl >> 16);
        }
    }
    // ---- the half-1 lanes stand at the chunk end; their lam goes to both halves
    const float iz = fast_rcp(zw);
    const float lam_end = xw * iz;
    if (hf) o.dec[n] = Aw * iz;
    if constexpr (MID) {
        return lam_end;
    } else {
        const float other = swap32(lam_end).lo32;   // half 1's lam, in half 0
        return hf ? lam_end : other;
    }
}

// Sequence and tensors of one scan-wave loop.
struct ScanSrc {
    const uint16_t *a, *p, *k, *q, *r;   // [B, T, H, DK] (r: [B, T, H])
    const uint16_t* tile;                 // per-token value tensor [B, T, H, DV] staged per chunk
    int tcol0;                            // first column of the value tile
    size_t seq0;                          // b * T
    int H, h, T, nchunk, bh;
    const float *oa = nullptr, *op = nullptr, *od = nullptr;   // OU parameters [H, DK] (TI)
    int* range_flag = nullptr;   // set to 1 when the walk leaves fp32 range, or none
};

// The scan-wave loop: nchunk + 1 rounds, each ended by barrier_lds().  The walk
// order is c = 0 .. nchunk-1 (REV = false: lam carried from lam_in, and with
// save the chunk's walk state written to the exchange buffer's mid region, which
// the MFMA waves store) or c = nchunk-1 .. 0 (REV: the walk state read from
// lam_in).  The walk state of a chunk is [kLamRows][DK]: lam at the chunk start,
// lam_16 and P_16 after its first 16 tokens (the valid ones when fewer); the
// saved sequence holds it as [BH][nchunk][kLamRows][DK].  Returns, walking
// forwards, the lam after the last token for key slot wave * SW + lane % SW.
template <class Cfg, bool YV, bool REV, bool TI, bool NOQ = false>
__device__ __forceinline__ float scan_wave(unsigned char* smem, int wave, int lane, const ScanSrc& sc,
                                           const float* __restrict__ lam_in, bool save) {
    constexpr int DK = Cfg::DK, DV = Cfg::DV, DVT = Cfg::DVT, SW = Cfg::SW, NSW = Cfg::NSW;
    constexpr int NL = REV ? 2 : 0;    // walk-state requests per round
    // staging loads of the per-token key-side inputs per round: two per staged tensor
    constexpr int NI = 2 * ((TI ? 0 : 2) + 1 + (NOQ ? 0 : 1));
    static_assert(!(NOQ && YV), "the readout variance needs the query");
    const int H = sc.H, h = sc.h, T = sc.T, nchunk = sc.nchunk;
    const int sl = lane % SW, hf = lane / SW;   // key slot within the wave, half of the chunk
    const int n = wave * SW + sl;
    float x = 1.f;                              // lam at the chunk start
    float chk = 0.f;                            // range check of the walk (scan_chunk)
    float lm = 0.f, pm = 0.f;                   // half 1: lam_16, P_16 of the chunk walked last
    if (!REV && lam_in) x = lam_in[(size_t)sc.bh * DK + n];
    float ca = 0.f, cp = 0.f;                   // time-invariant gates of slot n
    if constexpr (TI) ou_gates(sc.oa[h * DK + n], sc.op[h * DK + n], sc.od[h * DK + n], ca, cp);
    unsigned char* stw = smem + Cfg::STG + wave * Cfg::STG_WAVE;
    uint32_t* rw = reinterpret_cast<uint32_t*>(stw + Cfg::STG_R);   // [2][64]
    float* lw = reinterpret_cast<float*>(stw + Cfg::STG_L);         // [2][2][64]
    const uint32_t tok_bytes = (uint32_t)H * DK * 2;
    // lane -> (token lane / 4, 8 slots); a load of 16 tokens lands as [t][SW] rows
    const uint32_t in_voff = (uint32_t)(lane >> 2) * tok_bytes + (lane & 3) * 16;
    auto chunk_of = [&](int it) { return REV ? nchunk - 1 - it : it; };

    // every input of chunk cn into staging buffer bb: abar, pbar, k, q (two loads of 16
    // tokens each), r and, walking backwards, the saved walk state (lane l: lam_0 of
    // slot l, or lam_16 of slot l - 32, then P_16).  Chunks outside the sequence get
    // empty descriptors, whose loads write zeros.
    auto issue_inputs = [&](int cn, int bb) {
        const bool in = cn >= 0 && cn < nchunk;
        const int t0 = in ? cn * kC : 0, nt = in ? min(kC, T - t0) : 0;
        const size_t e0 = ((sc.seq0 + t0) * H + h) * DK + wave * SW;
        const uint32_t bytes = nt > 0 ? (uint32_t)((nt - 1) * H * DK + SW) * 2 : 0u;
        uint16_t* stg = reinterpret_cast<uint16_t*>(stw) + bb * 4 * kSR * SW;
        auto one = [&](const uint16_t* src, int ti) {
            const rsrc_t rs = make_rsrc(src + e0, bytes);
            buf_ld128_lds(rs, stg + ti * kSR * SW, in_voff);
            buf_ld128_lds(rs, stg + (ti * kSR + srow(16)) * SW, in_voff + 16 * tok_bytes);
        };
        if constexpr (!TI) {
            one(sc.a, 0);
            one(sc.p, 1);
        }
        one(sc.k, 2);
        if constexpr (!NOQ) one(sc.q, 3);
        const rsrc_t rr = make_rsrc(sc.r + (sc.seq0 + t0) * H + h, nt > 0 ? (uint32_t)((nt - 1) * H + 1) * 2 : 0u);
        buf_ld16_lds(rr, rw + bb * 64, (uint32_t)lane * H * 2);
        if constexpr (REV) {
            const rsrc_t rl = make_rsrc(lam_in + ((size_t)sc.bh * nchunk + (in ? cn : 0)) * kLamRows * DK + wave * SW,
                                        in ? (uint32_t)(2 * DK + SW) * 4 : 0u);
            buf_ld32_lds(rl, lw + bb * 128, (uint32_t)(hf * DK + sl) * 4);
            buf_ld32_lds(rl, lw + bb * 128 + 64, (uint32_t)(2 * DK + sl) * 4);
        }
    };
    // this wave's share of the value-tile loads (loads i = wave, wave + NSW, ...)
    const int nvw = Cfg::NVL % NSW == 0 ? Cfg::NVL / NSW : wave < Cfg::NVL ? (Cfg::NVL - wave + NSW - 1) / NSW : 0;
    const uint32_t v_voff = (uint32_t)(lane / (DVT / 8)) * H * DV * 2 + (lane % (DVT / 8)) * 16;
    auto issue_tile = [&](int cn, int it) {
        const int t0 = cn * kC, nt = min(kC, T - t0);
        const rsrc_t rv = make_rsrc(sc.tile + ((sc.seq0 + t0) * H + h) * DV + sc.tcol0,
                                    (uint32_t)((nt - 1) * H * DV + DVT) * 2);
        unsigned char* vs = smem + (it & 1) * Cfg::BUF + Cfg::VS;
        for (int i = wave; i < Cfg::NVL; i += NSW)
            buf_ld128_lds(rv, vs + i * 1024, v_voff + (uint32_t)(i * Cfg::TPV) * H * DV * 2);
    };
    wait_vm_all();   // the carried lam is complete before the prefetch loop starts
    if (nchunk > 0) issue_inputs(chunk_of(0), 0);

    for (int it = 0; it <= nchunk; ++it) {
        if (it < nchunk) {
            const int c = chunk_of(it), bb = it & 1;
            const int nt = min(kC, T - c * kC);
            issue_tile(c, it);
            issue_inputs(chunk_of(it + 1), bb ^ 1);
            // this chunk's inputs, requested one round earlier, have landed: younger are the
            // requests just issued (the value-tile loads, NI + 1 + NL staging loads)
            wait_vm_le_rt<NI + 1 + NL>(nvw);
            if constexpr (REV) {
                x = lw[bb * 128 + lane];
                pm = lw[bb * 128 + 64 + lane];
            }

            unsigned char* buf = smem + (it & 1) * Cfg::BUF;
            ScanOut o;
            o.qh = reinterpret_cast<uint16_t*>(buf + Cfg::QH);
            o.ql = reinterpret_cast<uint16_t*>(buf + Cfg::QL);
            o.kh = reinterpret_cast<uint16_t*>(buf + Cfg::KH);
            o.kl = reinterpret_cast<uint16_t*>(buf + Cfg::KL);
            o.dec = reinterpret_cast<float*>(buf + Cfg::DEC);
            o.yv = reinterpret_cast<float*>(buf + Cfg::YVP) + wave * kC;
            o.mid = reinterpret_cast<float*>(buf + Cfg::MIDS);
            const float x0 = x;
            const uint16_t* stg = reinterpret_cast<const uint16_t*>(stw) + bb * 4 * kSR * SW;
            const uint32_t* rwc = rw + bb * 64;
            if (nt == kC)
                x = scan_chunk<SW, Cfg::LQ, YV, true, TI, NOQ, REV>(stg, rwc, sl, hf, n, nt, x, o, ca, cp, chk, lm,
                                                                  pm);
            else
                x = scan_chunk<SW, Cfg::LQ, YV, false, TI, NOQ, REV>(stg, rwc, sl, hf, n, nt, x, o, ca, cp, chk, lm,
                                                                   pm);
            if (!REV && save) {
                if (hf) {
                    o.mid[DK + n] = lm;
                    o.mid[2 * DK + n] = pm;
                } else {
                    o.mid[n] = x0;
                }
            }
            // the value tile has landed (younger: the NI + 1 + NL staging loads)
            wait_vm_le<NI + 1 + NL>();
        }
        barrier_lds();
    }
    wait_vm_all();   // the requests for the chunk past the end have landed before exit
    if (sc.range_flag && !(fabsf(chk) <= 3.0e38f)) *sc.range_flag = 1;   // NaN fails the test too
    return x;
}

}  // namespace kla
