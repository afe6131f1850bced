// Per-chunk precision walk of one key slot, shared by the chunked kernels.
//
// For key slot n and the tokens t < nt of one chunk, starting from the carried
// precision lam (Theorem 1, gate view):
//   den_t = abar_t^2 + pbar_t lam_{t-1}  (= 1 / rho_t)
//   lam_t = rho_t lam_{t-1} + k_t^2 r_t
//   F_t   = abar_t rho_t                  (forget gate, Theorem 2)
//   P_t   = prod_{s<=t} F_s               (inside the chunk)
//   Qp_t  = (q_t / lam_t) P_t,   Kn_t = (r_t k_t) / P_t
// With num = lam_{t-1} + k^2 r den (so lam_t = num / den), one reciprocal of
// den * num * abar yields rho_t, 1/lam_t and 1/abar.
//
// Qp and Kn are stored as split-bf16 (hi, lo) pairs in any of four LDS layouts
// selected at compile time: [t][n] (row stride LQ) and [n][t] (row stride LT,
// written 8 tokens per 16-byte store).  Optionally lam_t and P_t are stored in
// fp32 [t][n] (row stride LS), and (YV) the per-token wave sums of q^2/lam.
// Tokens t >= nt get zeros.  The inputs of the
// next NB tokens are loaded while the current NB are processed; loads are
// unconditional (clamped to the last valid token).
#pragma once
#include "kla_mfma.hpp"

namespace kla {

struct ScanLds {
    uint16_t *qn_hi, *qn_lo;   // Qp [t][n]
    uint16_t *kn_hi, *kn_lo;   // Kn [t][n]
    uint16_t *qt_hi, *qt_lo;   // Qp^T [n][t]
    uint16_t *kt_hi, *kt_lo;   // Kn^T [n][t]
    float *lam, *P;            // fp32 [t][n]
    float* yv;                 // per-token partial sums of q^2 / lam over the wave, [t]
};

template <int C, int LQ, int LT, int LS, bool QN, bool KN, bool QT, bool KT, bool ST, int NB, bool YV>
struct ChunkScan {
    static_assert(NB == 4 || NB == 8, "batches of 4 or 8 tokens");
    // raw bf16 inputs of NB tokens: abar, pbar, k, q, r
    struct Batch {
        uint16_t v[5][NB];
    };

    const uint16_t *a, *p, *k, *q, *r;
    size_t row0;
    int H, h, DK, n, nl, nt, lane;
    bool active;
    ScanLds L;
    float P = 1.f, iP = 1.f;
    uint32_t hp[8], lp[8];  // the current 8 tokens: packed (Qp, Kn) hi and lo halves

    __device__ __forceinline__ void load(Batch& b, int t4) const {
#pragma unroll
        for (int j = 0; j < NB; ++j) {
            const int tc = min(t4 + j, nt - 1);
            const size_t rowi = (row0 + tc) * H + h;
            const size_t o = rowi * DK + n;
            b.v[0][j] = a[o];
            b.v[1][j] = p[o];
            b.v[2][j] = k[o];
            b.v[3][j] = q[o];
            b.v[4][j] = r[rowi];
        }
    }

    // tokens t4 .. t4+NB-1 into slots OFF .. OFF+NB-1 of the current group of 8
    template <int OFF>
    __device__ __forceinline__ void step(const Batch& b, int t4, float& lam) {
#pragma unroll
        for (int j = 0; j < NB; ++j) {
            const int t = t4 + j;
            const float av = bf16_to_f32(b.v[0][j]), pv = bf16_to_f32(b.v[1][j]);
            const float kv = bf16_to_f32(b.v[2][j]), qv = bf16_to_f32(b.v[3][j]);
            const float rv = bf16_to_f32(b.v[4][j]);
            float qp = 0.f, kn = 0.f, w = 0.f;
            if (t < nt) {
                const float den = fmaf(pv, lam, av * av);
                const float num = fmaf(kv * kv * rv, den, lam);
                const float rr = fast_rcp(den * num * av);
                const float rho = num * av * rr;
                const float ilam = den * den * av * rr;
                const float ia = den * num * rr;
                lam = num * rho;
                P *= av * rho;
                iP *= den * ia;
                const float qt = qv * ilam;
                qp = qt * P;
                kn = rv * kv * iP;
                w = active ? qv * qt : 0.f;
            }
            split2(qp, kn, hp[OFF + j], lp[OFF + j]);
            if (active) {
                if constexpr (QN) {
                    L.qn_hi[t * LQ + nl] = static_cast<uint16_t>(hp[OFF + j]);
                    L.qn_lo[t * LQ + nl] = static_cast<uint16_t>(lp[OFF + j]);
                }
                if constexpr (KN) {
                    L.kn_hi[t * LQ + nl] = static_cast<uint16_t>(hp[OFF + j] >> 16);
                    L.kn_lo[t * LQ + nl] = static_cast<uint16_t>(lp[OFF + j] >> 16);
                }
                if constexpr (ST) {
                    L.lam[t * LS + nl] = lam;
                    L.P[t * LS + nl] = P;
                }
            }
            if constexpr (YV) {
#pragma unroll
                for (int off = 32; off > 0; off >>= 1) w += __shfl_xor(w, off, 64);
                if (lane == 0) L.yv[t] = w;
            }
        }
    }

    // the transposed rows [n][t8 .. t8+7], one 16-byte store each
    __device__ __forceinline__ void store8(int t8) const {
        if (!active) return;
        if constexpr (QT) {
            uint4 h4, l4;
            h4.x = (hp[0] & 0xffffu) | (hp[1] << 16);
            h4.y = (hp[2] & 0xffffu) | (hp[3] << 16);
            h4.z = (hp[4] & 0xffffu) | (hp[5] << 16);
            h4.w = (hp[6] & 0xffffu) | (hp[7] << 16);
            l4.x = (lp[0] & 0xffffu) | (lp[1] << 16);
            l4.y = (lp[2] & 0xffffu) | (lp[3] << 16);
            l4.z = (lp[4] & 0xffffu) | (lp[5] << 16);
            l4.w = (lp[6] & 0xffffu) | (lp[7] << 16);
            *reinterpret_cast<uint4*>(L.qt_hi + nl * LT + t8) = h4;
            *reinterpret_cast<uint4*>(L.qt_lo + nl * LT + t8) = l4;
        }
        if constexpr (KT) {
            uint4 h4, l4;
            h4.x = (hp[0] >> 16) | (hp[1] & 0xffff0000u);
            h4.y = (hp[2] >> 16) | (hp[3] & 0xffff0000u);
            h4.z = (hp[4] >> 16) | (hp[5] & 0xffff0000u);
            h4.w = (hp[6] >> 16) | (hp[7] & 0xffff0000u);
            l4.x = (lp[0] >> 16) | (lp[1] & 0xffff0000u);
            l4.y = (lp[2] >> 16) | (lp[3] & 0xffff0000u);
            l4.z = (lp[4] >> 16) | (lp[5] & 0xffff0000u);
            l4.w = (lp[6] >> 16) | (lp[7] & 0xffff0000u);
            *reinterpret_cast<uint4*>(L.kt_hi + nl * LT + t8) = h4;
            *reinterpret_cast<uint4*>(L.kt_lo + nl * LT + t8) = l4;
        }
    }

    // Walk the chunk from the carried lam; returns P at the chunk end.  The loop
    // over groups of 8 tokens is a runtime loop (LDS addresses advance with it
    // instead of being materialised per token); the loads of the next 4 tokens
    // are in flight while the current 4 are processed.
    // b0 holds the chunk's first NB tokens, loaded in advance by the caller.
    __device__ __forceinline__ float run(float& lam, const Batch& first) {
        Batch b0 = first, b1;
        if constexpr (NB == 4) {
#pragma unroll 1
            for (int t8 = 0; t8 < C; t8 += 8) {
                load(b1, t8 + 4);
                step<0>(b0, t8, lam);
                if (t8 + 8 < C) load(b0, t8 + 8);
                step<4>(b1, t8 + 4, lam);
                store8(t8);
            }
        } else {
#pragma unroll 1
            for (int t16 = 0; t16 < C; t16 += 16) {
                load(b1, t16 + 8);
                step<0>(b0, t16, lam);
                store8(t16);
                if (t16 + 16 < C) load(b0, t16 + 16);
                step<0>(b1, t16 + 8, lam);
                store8(t16 + 8);
            }
        }
        return P;
    }
};

// First NB tokens of a chunk for key slot n, issued ahead of the chunk's walk.
template <int NB>
struct ScanPrefetch {
    uint16_t v[5][NB];
};

template <int NB>
__device__ __forceinline__ void scan_prefetch(ScanPrefetch<NB>& b, const uint16_t* __restrict__ a,
                                              const uint16_t* __restrict__ p, const uint16_t* __restrict__ k,
                                              const uint16_t* __restrict__ q, const uint16_t* __restrict__ r,
                                              size_t row0, int H, int h, int DK, int n, int nt) {
#pragma unroll
    for (int j = 0; j < NB; ++j) {
        const int tc = min(j, nt - 1);
        const size_t rowi = (row0 + tc) * H + h;
        const size_t o = rowi * DK + n;
        b.v[0][j] = a[o];
        b.v[1][j] = p[o];
        b.v[2][j] = k[o];
        b.v[3][j] = q[o];
        b.v[4][j] = r[rowi];
    }
}

template <int C, int LQ, int LT, int LS, bool QN, bool KN, bool QT, bool KT, bool ST, int NB, bool YV = false>
__device__ __forceinline__ float scan_chunk(const uint16_t* __restrict__ a, const uint16_t* __restrict__ p,
                                            const uint16_t* __restrict__ k, const uint16_t* __restrict__ q,
                                            const uint16_t* __restrict__ r, size_t row0, int H, int h, int DK,
                                            int n, int nl, bool active, int nt, float& lam, const ScanLds& L,
                                            int lane, const ScanPrefetch<NB>& first) {
    using S = ChunkScan<C, LQ, LT, LS, QN, KN, QT, KT, ST, NB, YV>;
    S sc{a, p, k, q, r, row0, H, h, DK, n, nl, nt, lane, active, L};
    typename S::Batch b0;
#pragma unroll
    for (int i = 0; i < 5; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j) b0.v[i][j] = first.v[i][j];
    return sc.run(lam, b0);
}

// Register-staged copy of a chunk tile of a per-token bf16 tensor (row length
// rowlen, columns c0 .. c0+W): issued one chunk ahead, written to LDS later.
template <int C, int W, int NTHR>
struct TileStage {
    static constexpr int PER = (C * (W / 8) + NTHR - 1) / NTHR;
    uint4 x[PER];
    __device__ __forceinline__ void load(const uint16_t* __restrict__ src, size_t row0, int H, int h, int rowlen,
                                         int c0, int nt, int tid) {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int idx = tid + i * NTHR;
            const int t = idx / (W / 8), c8 = idx % (W / 8);
            const int tc = min(t, nt - 1);
            x[i] = *reinterpret_cast<const uint4*>(src + ((row0 + tc) * H + h) * rowlen + c0 + 8 * c8);
            if (t >= nt) x[i] = uint4{0u, 0u, 0u, 0u};
        }
    }
    // rows [t][c] with stride L and/or transposed [c][t] with stride LT
    template <int L, int LT, bool ROWS, bool COLS>
    __device__ __forceinline__ void store(uint16_t* rows, uint16_t* cols, int tid) const {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int idx = tid + i * NTHR;
            if (PER * NTHR != C * (W / 8) && idx >= C * (W / 8)) break;
            const int t = idx / (W / 8), c8 = idx % (W / 8);
            if constexpr (ROWS) *reinterpret_cast<uint4*>(rows + t * L + 8 * c8) = x[i];
            if constexpr (COLS) {
                const uint16_t* e = reinterpret_cast<const uint16_t*>(&x[i]);
#pragma unroll
                for (int j = 0; j < 8; ++j) cols[(8 * c8 + j) * LT + t] = e[j];
            }
        }
    }
};

// Chunk tile of a per-token bf16 tensor (row length rowlen, columns c0 .. c0+W)
// into LDS, row-major [t][c] (stride L) and/or transposed [c][t] (stride LT);
// rows past the sequence end are zero.
template <int C, int W, int L, int LT, bool ROWS, bool COLS>
__device__ __forceinline__ void load_tile(uint16_t* rows, uint16_t* cols, const uint16_t* __restrict__ src,
                                          size_t row0, int H, int h, int rowlen, int c0, int nt, int tid,
                                          int nthreads) {
    for (int idx = tid; idx < C * (W / 8); idx += nthreads) {
        const int t = idx / (W / 8), c8 = idx % (W / 8);
        const int tc = min(t, nt - 1);
        uint4 x = *reinterpret_cast<const uint4*>(src + ((row0 + tc) * H + h) * rowlen + c0 + 8 * c8);
        if (t >= nt) x = uint4{0u, 0u, 0u, 0u};
        if constexpr (ROWS) *reinterpret_cast<uint4*>(rows + t * L + 8 * c8) = x;
        if constexpr (COLS) {
            const uint16_t* e = reinterpret_cast<const uint16_t*>(&x);
#pragma unroll
            for (int i = 0; i < 8; ++i) cols[(8 * c8 + i) * LT + t] = e[i];
        }
    }
}

}  // namespace kla
