// Chunked forward and backward of the KLA filter for fp32 inputs, in fp64.
//
// The chunk form of the bf16 path (chunk_fwd.hip, chunk_bwd_dv.hip,
// chunk_bwd_dk.hip) with every quantity in fp64.  Per chunk of kC64 = 32 tokens
// and key slot n, the precision walk (Theorem 1 in homogeneous coordinates:
// z' = pbar x + abar^2 z, x' = x + k^2 r z', from (x, z) = (lam_0, 1), A the
// running product of abar) gives
//   lam_t = x_t / z_t,   P_t = A_t / z_t   (the product of the forget gates
//                                           F = abar rho over the chunk),
//   Qp[t, n] = q / lam_t * P_t = q A_t / x_t,   Kn[t, n] = k r / P_t = k r z_t / A_t,
// and the readout and state update of Algorithm 1 over the chunk are
//   y = M(Qp Kn^T) V + Qp H0,   H_C = diag(P_C) (H0 + Kn^T V)   (M: j <= t).
// The backward is their reverse-mode counterpart, chunk by chunk from the last:
//   S = M(Qp Kn^T),  B = M(dY V^T),  Gs = diag(P_C) G   (G: adjoint of the chunk's
//   last state from later tokens, detaT for the last chunk)
//   dV = S^T dY + Kn Gs,  X = dY H0^T + B Kn,  Y = B^T Qp + V Gs^T,
//   G' = Qp^T dY + Gs   (carried into the previous chunk; after the first, deta0),
// dqt = P X (gradient of qt = q / lam_t) and dkh = Y / P (gradient of kh = k r),
// then the adjoint walk of the precision, per slot over the chunk's tokens in
// reverse: with u_t = qt dqt - kh dkh summed from the end into S (the adjoint of
// log F, started at sum_d detaT H_T), g_t = c_t - q (dqt + q gv) / lam_t^2 and
// c_{t-1} = abar^2 rho^2 g_t - pbar rho S_t (c_T = dlamT, gv the upstream
// gradient of yvar), the input gradients
//   dq = (dqt + 2 q gv) / lam,  dk = r dkh + 2 k r g,  dr = sum_n (k dkh + k^2 g),
//   drho = g lam_{t-1} + S / rho,  dabar = S / abar - 2 abar rho^2 drho,
//   dpbar = -lam_{t-1} rho^2 drho,  dlam0 = c after the first token.
//
// Why fp64 in chunks: the fp32-input path is held to 1e-4 on every gradient, which
// its long adjoint chains only meet in fp64, and the token-recurrent fp64 kernels
// are bound by one dependent step per token; here the dependent steps are per
// chunk (the walk over 32 tokens, spread over token groups as in chunk_bwd_dk.hip),
// and the contractions run on v_mfma_f64_16x16x4_f64.
//
// One workgroup per (b, h), dk and dv in {16, 32}: 512 threads in the forward
// (walk waves and MFMA waves, see there), 256 in the backward.  The walk lanes
// are 256 threads (slot n = tid % dk, token group gq = tid / dk of TPG tokens); each
// lane forms its group's 2x2 transfer, the groups are chained through LDS from
// the chunk-start lam, and each lane then walks its own tokens.  Tokens past the
// sequence end enter with abar = 1, pbar = k = q = r = 0, which the walk, the
// contractions and the adjoint pass through unchanged.  The 16x16 tiles of the
// state (forward) or its adjoint (backward) live in the registers of one wave
// each.
//
// Saved context (c64_saved_bytes): lam at every chunk start [BH][nchunk][dk], then
// the information state at every chunk start and after the last token
// [BH][nchunk+1][dk][dv], fp64.
#include "kla_buf.hpp"
#include "kla_device.hpp"
#include "kla_internal.hpp"

namespace kla {
namespace {

constexpr int kC64 = 32;    // tokens per chunk
constexpr int kNT64 = 256;  // threads per backward workgroup

typedef double d4 __attribute__((ext_vector_type(4)));

// D += A B over four columns of A (v_mfma_f64_16x16x4_f64): lane l supplies
// A[l % 16][l / 16] and B[l / 16][l % 16]; D[i][j] is component i / 4 of lane
// j + 16 (i % 4).
__device__ __forceinline__ d4 mfma64(double a, double b, d4 c) {
    return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ d4 zero_d4() { return d4{0.0, 0.0, 0.0, 0.0}; }

// acc += sum_{k < K} A(i, k) B(k, j) for the 16x16 tile whose A rows start at pa and
// B columns at pb (LDS), A(i, k) = pa[i AI + k AK], B(k, j) = pb[k BK + j BJ].  The
// triangular products run over the whole chunk: the tile above the diagonal of the
// masked matrices is stored as zeros.
template <int K, int AI, int AK, int BK, int BJ>
__device__ __forceinline__ d4 tile_mm(d4 acc, const double* pa, const double* pb, int lane) {
    const int li = lane & 15, lk = lane >> 4;
    double av[K / 4], bv[K / 4];
#pragma unroll
    for (int s = 0; s < K / 4; ++s) {
        av[s] = pa[li * AI + (4 * s + lk) * AK];
        bv[s] = pb[(4 * s + lk) * BK + li * BJ];
    }
#pragma unroll
    for (int s = 0; s < K / 4; ++s) acc = mfma64(av[s], bv[s], acc);
    return acc;
}

// Sum over the DK lanes of one walk group (DK = 32: a half wave, DK = 16: a DPP row),
// valid in the group's last lane (n = DK - 1).
template <int DK>
__device__ __forceinline__ double slot_sum(double x) {
    if constexpr (DK == 32) {
        return half_sum(x);
    } else {
        x += dpp<0xB1, 0xf>(x);    // quad_perm [1,0,3,2]
        x += dpp<0x4E, 0xf>(x);    // quad_perm [2,3,0,1]
        x += dpp<0x141, 0xf>(x);   // row_half_mirror
        x += dpp<0x140, 0xf>(x);   // row_mirror
        return x;
    }
}

// row of component r of a D tile, relative to the tile (its column is lane % 16)
__device__ __forceinline__ int drow(int r, int lane) { return 4 * r + (lane >> 4); }

__device__ __forceinline__ float bld32(rsrc_t r, uint32_t voff) {
    return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, voff, 0, 0));
}

// Stores through a buffer: a lane whose offset lies past the end stores nothing.
__device__ __forceinline__ void bst32(rsrc_t r, uint32_t voff, float x) {
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(x), r, voff, 0, 0);
}

typedef __attribute__((__vector_size__(2 * sizeof(uint32_t)))) uint32_t u32x2;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;

__device__ __forceinline__ void bst64(rsrc_t r, uint32_t voff, double x) {
    __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, x), r, voff, 0, 0);
}

// N (2 or 4) consecutive floats through a buffer in one load (offset aligned to 4 N bytes)
template <int N>
__device__ __forceinline__ void bldN(rsrc_t r, uint32_t voff, float* out) {
    if constexpr (N == 4) {
        const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, voff, 0, 0);
#pragma unroll
        for (int i = 0; i < 4; ++i) out[i] = __uint_as_float(v[i]);
    } else {
        static_assert(N == 2, "2 or 4 floats");
        const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r, voff, 0, 0);
        out[0] = __uint_as_float(v[0]);
        out[1] = __uint_as_float(v[1]);
    }
}

// N (2 or 4) consecutive floats from LDS (aligned to 4 N bytes) stored through a buffer in one store
template <int N>
__device__ __forceinline__ void bstN_lds(rsrc_t r, uint32_t voff, const float* src) {
    if constexpr (N == 4) {
        const float4 v = *reinterpret_cast<const float4*>(src);
        __builtin_amdgcn_raw_buffer_store_b128(
            u32x4{__float_as_uint(v.x), __float_as_uint(v.y), __float_as_uint(v.z), __float_as_uint(v.w)}, r, voff, 0, 0);
    } else {
        static_assert(N == 2, "2 or 4 floats");
        const float2 v = *reinterpret_cast<const float2*>(src);
        __builtin_amdgcn_raw_buffer_store_b64(u32x2{__float_as_uint(v.x), __float_as_uint(v.y)}, r, voff, 0, 0);
    }
}

// Buffers over one chunk's rows of the per-token tensors of head h: [t][H][DK] rows
// (abar, pbar, k, q) and [t][H] (r), each ending at the chunk's last valid token, so
// that tokens past the sequence end read as zero.
struct ChunkBufs {
    rsrc_t a, p, k, q, r;
    __device__ ChunkBufs(const float* ga, const float* gp, const float* gk, const float* gq, const float* gr,
                         size_t tok0, int H, int h, int DK, int nt) {
        const size_t e0 = (tok0 * H + h) * DK;
        const uint32_t bytes = (uint32_t)((nt - 1) * H * DK + DK) * 4;
        a = make_rsrc(ga ? ga + e0 : gk, ga ? bytes : 0u);
        p = make_rsrc(gp ? gp + e0 : gk, gp ? bytes : 0u);
        k = make_rsrc(gk + e0, bytes);
        q = make_rsrc(gq + e0, bytes);
        r = make_rsrc(gr + tok0 * H + h, (uint32_t)((nt - 1) * H + 1) * 4);
    }
};

// Per-token inputs of a walk lane, slot n, tokens t0 .. t0 + TPG - 1 of a chunk
// (t0 = gq TPG), as loaded (fp32).  Tokens past the sequence end (j >= nv) read as
// zeros, and abar as 1: the identity step.
template <int DK, int TPG, bool TI>
struct WalkIn {
    float a[TPG], p[TPG], k[TPG], q[TPG], r[TPG];
    int nv;
    double ca, cp;   // time-invariant gates (TI)
    __device__ void load(const ChunkBufs& cb, int H, int n, int t0, int nt) {
        nv = min(max(nt - t0, 0), TPG);
#pragma unroll
        for (int j = 0; j < TPG; ++j) {
            const uint32_t vo = (uint32_t)((t0 + j) * H * DK + n) * 4;
            if constexpr (!TI) {
                a[j] = bld32(cb.a, vo);
                p[j] = bld32(cb.p, vo);
            }
            k[j] = bld32(cb.k, vo);
            q[j] = bld32(cb.q, vo);
            r[j] = bld32(cb.r, (uint32_t)((t0 + j) * H) * 4);
        }
    }
    __device__ double A(int j) const { return j < nv ? (TI ? ca : (double)a[j]) : 1.0; }
    __device__ double P(int j) const { return TI ? (j < nv ? cp : 0.0) : (double)p[j]; }
    __device__ double K(int j) const { return (double)k[j]; }
    __device__ double Q(int j) const { return (double)q[j]; }
    __device__ double R(int j) const { return (double)r[j]; }
};

// The 2x2 transfer of a lane's tokens (the images of (1, 0) and (0, 1) under the
// homogeneous precision map) and the product of abar, into qs[gq][5][DK].
template <int DK, int TPG, bool TI>
__device__ __forceinline__ void group_transfer(const WalkIn<DK, TPG, TI>& in, double* qs, int gq, int n) {
    double m00 = 1.0, m10 = 0.0, m01 = 0.0, m11 = 1.0, aq = 1.0;
#pragma unroll
    for (int j = 0; j < TPG; ++j) {
        const double av = in.A(j), kv = in.K(j);
        const double a2 = av * av, phi = kv * kv * in.R(j);
        const double z0 = fma(in.P(j), m00, a2 * m10), z1 = fma(in.P(j), m01, a2 * m11);
        m00 = fma(phi, z0, m00);
        m01 = fma(phi, z1, m01);
        m10 = z0;
        m11 = z1;
        aq *= av;
    }
    qs[(gq * 5 + 0) * DK + n] = m00;
    qs[(gq * 5 + 1) * DK + n] = m10;
    qs[(gq * 5 + 2) * DK + n] = m01;
    qs[(gq * 5 + 3) * DK + n] = m11;
    qs[(gq * 5 + 4) * DK + n] = aq;
}

// (x, z, A) before the lane's first token: the transfers of the earlier groups
// applied to the chunk start (lam, 1, 1).
template <int DK, int G>
__device__ __forceinline__ void chain_start(const double* qs, int gq, int n, double lam, double& x, double& z,
                                            double& A) {
    x = lam;
    z = 1.0;
    A = 1.0;
#pragma unroll
    for (int g2 = 0; g2 < G - 1; ++g2) {   // every lane the same steps, applied while g2 < gq
        const double m00 = qs[(g2 * 5 + 0) * DK + n], m10 = qs[(g2 * 5 + 1) * DK + n];
        const double m01 = qs[(g2 * 5 + 2) * DK + n], m11 = qs[(g2 * 5 + 3) * DK + n];
        const double aq = qs[(g2 * 5 + 4) * DK + n];
        const bool use = g2 < gq;
        const double xn = fma(m00, x, m01 * z), zn = fma(m10, x, m11 * z);
        x = use ? xn : x;
        z = use ? zn : z;
        A = use ? A * aq : A;
    }
}

// ============================================================================ forward
// Eight waves: waves 0..3 walk chunk c (stage, group transfers, walk: Qp, Kn, P_C
// and the next chunk-start lam into the LDS set of c's parity) while waves 4..7
// run the contractions of chunk c - 1 from the other set, each owning one state
// tile and one readout tile.  Two barriers per round: between the walk's group
// transfers and their chaining (the MFMA waves then go from S to the products
// that read it), and at the round's end.
constexpr int kWT = 256;   // walk threads of the forward (waves 0..3); waves 4..7 are MFMA waves

template <int DK, int DV, bool TI>
__global__ __launch_bounds__(2 * kWT) void fwd64_kernel(Shape s, FwdArgs g, double* saved_lam, double* saved_H) {
    constexpr int C = kC64, G = kWT / DK, TPG = C / G;
    constexpr int PQ = DK + 1, PV = DV + 1, PS = C + 1;
    constexpr int NTD = DV / 16, NTN = DK / 16, NTT = C / 16;
    constexpr int NVE = C * DV / kWT;   // value elements per walk thread and chunk
    // chunk c's walk results, in the set c & 1 (written by the walk waves in round c,
    // read by the MFMA waves in round c + 1)
    __shared__ double sQp[2][C * PQ], sKn[2][C * PQ], sV[2][C * PV], sPC[2][DK];
    __shared__ double sS[C * PS], sH[DK * PV];   // MFMA waves
    __shared__ double qs[G * 5 * DK], sLam[2 * DK];   // walk waves

    const int bh = blockIdx.x, b = bh / s.H, h = bh % s.H, H = s.H, T = s.T;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const bool walker = wave < 4;
    const int n = tid % DK, gq = (tid % kWT) / DK;   // walk lanes: slot, token group
    const int nchunk = (T + C - 1) / C;
    const size_t seq0 = (size_t)b * T;
    const float* fq = static_cast<const float*>(g.q);
    const float* fk = static_cast<const float*>(g.k);
    const float* fv = static_cast<const float*>(g.v);
    const float* fa = static_cast<const float*>(g.a);
    const float* fp = static_cast<const float*>(g.p);
    const float* fr = static_cast<const float*>(g.r);
    float* fy = static_cast<float*>(g.y);

    double ca = 0.0, cp = 0.0;   // time-invariant gates of slot n
    if constexpr (TI)
        if (walker) ou_gates(g.ou_a[h * DK + n], g.ou_p[h * DK + n], g.ou_d[h * DK + n], ca, cp);

    // MFMA wave mw's state tile (tn, td) = H[16 tn .. + 15][16 td .. + 15] and readout tile
    // (ti, tdy), if any (at dk = dv = 32 every MFMA wave owns one of each, known at compile time)
    constexpr bool FULL = NTN * NTD == 4 && NTT * NTD == 4;
    const int mw = wave - 4;
    const bool hown = !walker && (FULL || mw < NTN * NTD);
    const bool yown = !walker && (FULL || mw < NTT * NTD);
    const int tn = mw / NTD, td = mw % NTD, ti = mw / NTD, tdy = mw % NTD;
    d4 Hs = zero_d4();
    if (hown && g.eta0)
        for (int r = 0; r < 4; ++r)
            Hs[r] = g.eta0[((size_t)bh * DK + 16 * tn + drow(r, lane)) * DV + 16 * td + (lane & 15)];

    if (tid < DK) sLam[tid] = g.lam0 ? (double)g.lam0[(size_t)bh * DK + tid] : 1.0;
    double chk = 0.0;   // range check: sum of Qp Kn over the lane's tokens

    // a chunk's inputs, fetched by the walk waves one chunk ahead
    struct Pre {
        WalkIn<DK, TPG, TI> w;
        float v[NVE];
    };
    auto fetch = [&](Pre& P, int cn) {
        const int nt = min(C, T - cn * C);
        const size_t tok0 = seq0 + (size_t)cn * C;
        P.w.load(ChunkBufs(TI ? nullptr : fa, TI ? nullptr : fp, fk, fq, fr, tok0, H, h, DK, nt), H, n, gq * TPG, nt);
        const rsrc_t rv = make_rsrc(fv + (tok0 * H + h) * DV, (uint32_t)((nt - 1) * H * DV + DV) * 4);
#pragma unroll
        for (int m = 0; m < NVE; ++m) {
            const int e = tid + kWT * m, t = e / DV, d = e % DV;
            P.v[m] = bld32(rv, (uint32_t)(t * H * DV + d) * 4);
        }
    };

    // The walk waves' outputs of a round (yvar of its chunk) are stored at the start of
    // their next round, before that round's fetch: no store is then younger than a fetch,
    // and the wait for a fetched chunk does not also wait for the stores of the round before.
    float oyv[TPG];   // yvar of the lane's tokens (lane n = DK - 1)
    int oc = -1;      // the chunk they belong to (none: -1)
    auto flush = [&]() {
        if (oc < 0 || !g.yvar) return;
        const int nt = min(C, T - oc * C);
        const rsrc_t rw = make_rsrc(g.yvar + (seq0 + (size_t)oc * C) * H + h, (uint32_t)((nt - 1) * H + 1) * 4);
#pragma unroll
        for (int j = 0; j < TPG; ++j)   // tokens past the chunk's last one, and the other lanes, fall outside
            bst32(rw, n == DK - 1 ? (uint32_t)((gq * TPG + j) * H) * 4 : 0x7ffffff0u, oyv[j]);
    };

    // ---- walk waves, chunk c: stage and group transfers, then the next chunk's fetch
    auto walk1 = [&](int c, Pre& cur, Pre& nxt) {
        flush();
        const double* lam_s = sLam + (c & 1) * DK;
        if (saved_lam && tid < DK) saved_lam[((size_t)bh * nchunk + c) * DK + tid] = lam_s[tid];
        double* V = sV[c & 1];
#pragma unroll
        for (int m = 0; m < NVE; ++m) {
            const int e = tid + kWT * m, t = e / DV, d = e % DV;
            V[t * PV + d] = (double)cur.v[m];
        }
        group_transfer(cur.w, qs, gq, n);
        if (c + 1 < nchunk) fetch(nxt, c + 1);
    };
    // ---- walk waves, chunk c: the lane's own tokens from the chained start
    auto walk2 = [&](int c, Pre& cur) {
        double* Qp = sQp[c & 1];
        double* Kn = sKn[c & 1];
        double x, z, A;
        chain_start<DK, G>(qs, gq, n, sLam[(c & 1) * DK + n], x, z, A);
        double wv[TPG];   // q^2 / lam_t
#pragma unroll
        for (int j = 0; j < TPG; ++j) {
            const int t = gq * TPG + j;
            const double av = cur.w.A(j), kv = cur.w.K(j), qv = cur.w.Q(j);
            const double kr = kv * cur.w.R(j);
            const double zn = fma(cur.w.P(j), x, av * av * z);
            const double xn = fma(kr * kv, zn, x);
            const double An = A * av;
            const double R = rcpa(xn * An);
            const double AR = An * R;               // 1 / x_t
            const double qp = qv * An * AR;         // q A_t / x_t
            const double kn = kr * zn * (xn * R);   // k r z_t / A_t
            chk = fma(qp, kn, chk);
            Qp[t * PQ + n] = qp;
            Kn[t * PQ + n] = kn;
            wv[j] = qv * qv * zn * AR;
            x = xn;
            z = zn;
            A = An;
        }
        if (gq == G - 1) {   // the last group ends at the chunk end
            const double iz = rcpa(z);
            sLam[((c + 1) & 1) * DK + n] = x * iz;
            sPC[c & 1][n] = A * iz;
        }
        if (g.yvar)
#pragma unroll
            for (int j = 0; j < TPG; ++j) oyv[j] = (float)slot_sum<DK>(wv[j]);
        oc = c;
    };
    // ---- MFMA waves, chunk c: the chunk-start state into LDS (and the saved context), S =
    // M(Qp Kn^T) (tiles (0,0), (1,0), (1,1) from waves 4..6, wave 7 repeating the last,
    // unstored; wave 5 also writes the zero tile above the diagonal)
    auto mfma1 = [&](int c) {
        if (hown)
            for (int r = 0; r < 4; ++r) {
                const int row = 16 * tn + drow(r, lane), col = 16 * td + (lane & 15);
                sH[row * PV + col] = Hs[r];
                if (saved_H)
                    bst64(make_rsrc(saved_H + ((size_t)bh * (nchunk + 1) + c) * DK * DV, DK * DV * 8),
                          (uint32_t)(row * DV + col) * 8, Hs[r]);
            }
        const int st = mw < 3 ? mw : 2;
        const int si = st == 0 ? 0 : 1, sj = st == 2 ? 1 : 0;
        const d4 acc = tile_mm<DK, PQ, 1, 1, PQ>(zero_d4(), sQp[c & 1] + 16 * si * PQ, sKn[c & 1] + 16 * sj * PQ, lane);
        if (mw < 3) {
            for (int r = 0; r < 4; ++r) {
                const int i = drow(r, lane), j = lane & 15;
                sS[(16 * si + i) * PS + 16 * sj + j] = (si == sj && j > i) ? 0.0 : acc[r];
            }
            if (si != sj)
                for (int r = 0; r < 4; ++r) sS[drow(r, lane) * PS + 16 + (lane & 15)] = 0.0;
        }
    };
    // ---- MFMA waves, chunk c: y = S V + Qp H0 and the state update diag(P_C) (H0 + Kn^T V)
    auto mfma2 = [&](int c) {
        const double* Qp = sQp[c & 1];
        const double* V = sV[c & 1];
        if (yown) {
            d4 yacc = tile_mm<DK, PQ, 1, PV, 1>(zero_d4(), Qp + 16 * ti * PQ, sH + 16 * tdy, lane);
            yacc = tile_mm<C, PS, 1, PV, 1>(yacc, sS + 16 * ti * PS, V + 16 * tdy, lane);
            const int nt = min(C, T - c * C);
            const rsrc_t ry = make_rsrc(fy + ((seq0 + (size_t)c * C) * H + h) * DV, (uint32_t)((nt - 1) * H * DV + DV) * 4);
            for (int r = 0; r < 4; ++r)   // rows past the chunk's last token fall outside the buffer
                bst32(ry, (uint32_t)((16 * ti + drow(r, lane)) * H * DV + 16 * tdy + (lane & 15)) * 4, (float)yacc[r]);
        }
        if (hown) {
            Hs = tile_mm<C, 1, PQ, PV, 1>(Hs, sKn[c & 1] + 16 * tn, V + 16 * td, lane);
            for (int r = 0; r < 4; ++r) Hs[r] *= sPC[c & 1][16 * tn + drow(r, lane)];
        }
    };

    // round r: the walk waves take chunk r, the MFMA waves chunk r - 1
    auto round = [&](int r, Pre& cur, Pre& nxt) {
        if (walker) {
            if (r < nchunk) walk1(r, cur, nxt);
        } else if (r >= 1) {
            mfma1(r - 1);
        }
        barrier_lds();   // group transfers in; S and the chunk-start state in
        if (walker) {
            if (r < nchunk) walk2(r, cur);
        } else if (r >= 1) {
            mfma2(r - 1);
        }
        barrier_lds();   // chunk r's walk results in; chunk r - 1's LDS set free
    };

    Pre P0, P1;
    P0.w.ca = P1.w.ca = ca;
    P0.w.cp = P1.w.cp = cp;
    if (walker && nchunk > 0) fetch(P0, 0);
    for (int r = 0; r <= nchunk; r += 2) {
        round(r, P0, P1);
        if (r + 1 <= nchunk) round(r + 1, P1, P0);
    }

    // ---- the final belief
    if (walker) {
        flush();
        if (g.lamT && tid < DK) g.lamT[(size_t)bh * DK + tid] = (float)sLam[(nchunk & 1) * DK + tid];
        if (g.range_flag && !(fabs(chk) <= 1.0e300)) *g.range_flag = 1;
    } else if (hown) {
        for (int r = 0; r < 4; ++r) {
            const int row = 16 * tn + drow(r, lane), col = 16 * td + (lane & 15);
            if (g.etaT) g.etaT[((size_t)bh * DK + row) * DV + col] = (float)Hs[r];
            if (saved_H) saved_H[(((size_t)bh * (nchunk + 1) + nchunk) * DK + row) * DV + col] = Hs[r];
        }
    }
}

// ============================================================================ backward
// Four waves (one per SIMD) take each chunk, from the last, through every phase, with an
// LDS barrier after each: the chunk's inputs from the staging area and the group
// transfers | the walk (Qp, Kn, P_C; the next chunk's fetch issued) | S, B, Gs | dV, X, Y,
// G' | adjoint pass 1 | adjoint pass 2 (gradients staged; the next chunk's inputs staged).
// Overlapping the phases on eight waves, as the forward does, was slower: the fp64 walk and
// adjoint work and the fp64 MFMAs contend for the same units, and the two roles' state does
// not fit 256 registers per wave.
template <int DK, int DV, bool TI>
__global__ __launch_bounds__(kNT64) void bwd64_kernel(Shape s, BwdArgs g, const double* saved_lam,
                                                      const double* saved_H) {
    constexpr int C = kC64, G = kNT64 / DK, TPG = C / G;
    constexpr int PQ = DK + 1, PV = DV + 1, PS = C + 1;
    constexpr int NTD = DV / 16, NTN = DK / 16, NTT = C / 16;
    // values per thread of a chunk's [C][DV] and [C][DK] rows and of a [DK][DV] state
    constexpr int NVE = C * DV / kNT64, NKE = C * DK / kNT64, NHE = DK * DV / kNT64;
    constexpr int NIN = TI ? 2 : 4;    // staged input rows: abar, pbar (per-token gates only), k, q
    constexpr int NOUT = TI ? 2 : 4;   // staged gradient rows: dq, dk, dabar, dpbar (per-token gates only)
    constexpr int NINB = NIN * C * DK * 4 / 1024;   // 1 KiB direct loads of the input rows per chunk
    static_assert(NINB % 4 == 0 && (NVE == 2 || NVE == 4) && (NKE == 2 || NKE == 4), "staging shapes");
    // row strides of the staged gradients: the walk lanes' writes (rows TPG apart within a
    // wave) fall in distinct banks, and every row starts on 16 bytes
    constexpr int SO = 40, SVD = DV == 32 ? 48 : 16;
    __shared__ double sQp[C * PQ], sKn[C * PQ], sV[C * PV], sDY[C * PV], sS[C * PS], sB[C * PS];
    __shared__ double sH0[DK * PV], sGs[DK * PV], sX[C * PQ], sY[C * PQ];
    __shared__ double qs[G * 5 * DK];
    __shared__ double sPC[DK], sCar[2 * 2 * DK];   // carries (c, S) by round parity
    __shared__ __attribute__((aligned(16))) float sIn[NIN * C * DK];   // [NIN][C][DK]
    __shared__ __attribute__((aligned(16))) float sOut[NOUT * C * SO], sDv[C * SVD], sDr[C];

    const int bh = blockIdx.x, b = bh / s.H, h = bh % s.H, H = s.H, T = s.T;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n = tid % DK, gq = tid / DK;
    const int nchunk = (T + C - 1) / C;
    const size_t seq0 = (size_t)b * T;
    const float* fq = static_cast<const float*>(g.q);
    const float* fk = static_cast<const float*>(g.k);
    const float* fv = static_cast<const float*>(g.v);
    const float* fa = static_cast<const float*>(g.a);
    const float* fp = static_cast<const float*>(g.p);
    const float* fr = static_cast<const float*>(g.r);
    const float* fdy = static_cast<const float*>(g.dy);
    float* gdq = static_cast<float*>(g.dq);
    float* gdk = static_cast<float*>(g.dk);
    float* gdv = static_cast<float*>(g.dv);
    float* gda = static_cast<float*>(g.da);
    float* gdp = static_cast<float*>(g.dp);
    float* gdr = static_cast<float*>(g.dr);

    double ca = 0.0, cp = 0.0;
    if constexpr (TI) ou_gates(g.ou_a[h * DK + n], g.ou_p[h * DK + n], g.ou_d[h * DK + n], ca, cp);
    double sum_da = 0.0, sum_dp = 0.0;   // OU gates: the lane's sums of the gate gradients

    // this wave's adjoint tile (tn, td) of G, if any (at dk = dv = 32 every wave owns one
    // tile of G, dV, X and Y, known at compile time)
    constexpr bool FULL = NTN * NTD == 4 && NTT * NTD == 4 && NTT * NTN == 4;
    const bool gown = FULL || wave < NTN * NTD;
    const int tn = wave / NTD, td = wave % NTD;
    d4 Gt = zero_d4();
    if (gown && g.detaT)
        for (int r = 0; r < 4; ++r)
            Gt[r] = g.detaT[((size_t)bh * DK + 16 * tn + drow(r, lane)) * DV + 16 * td + (lane & 15)];
    // carries at the sequence end: c = dlamT, S = sum_d detaT H_T
    if (tid < DK) {
        double st = 0.0;
        if (g.detaT) {
            const double* HT = saved_H + (((size_t)bh * (nchunk + 1) + nchunk) * DK + tid) * DV;
            const float* dT = g.detaT + ((size_t)bh * DK + tid) * DV;
            for (int d = 0; d < DV; ++d) st = fma((double)dT[d], HT[d], st);
        }
        sCar[(nchunk & 1) * 2 * DK + tid] = g.dlamT ? (double)g.dlamT[(size_t)bh * DK + tid] : 0.0;
        sCar[(nchunk & 1) * 2 * DK + DK + tid] = st;
    }
    double chk = 0.0;

    // Chunk cn's inputs, fetched during the round before its own: abar, pbar, k, q by 16-byte
    // direct loads into sIn (row-major [C][DK] each), the rest into registers: v and dy (NVE
    // consecutive values of thread tid), the saved state (NHE consecutive values), r and gv of
    // token lane % 32, and lam of slot n.  Tokens past the sequence end read as zeros.
    float pv[NVE], pdy[NVE], pr, pgv;
    double ph0[NHE], plam;
    auto prefetch = [&](int cn) {
        const int nt = min(C, T - cn * C);
        const size_t tok0 = seq0 + (size_t)cn * C;
        const ChunkBufs cb(TI ? nullptr : fa, TI ? nullptr : fp, fk, fq, fr, tok0, H, h, DK, nt);
#pragma unroll
        for (int m = 0; m < NINB / 4; ++m) {
            const int blk = 4 * m + wave;                            // 1 KiB block of sIn
            const int x = blk * 1024 / (C * DK * 4);                 // its input row set
            const int o = blk * 1024 % (C * DK * 4) + 16 * lane;     // this lane's byte within the set
            const int t = o / (DK * 4), col = o % (DK * 4) / 4;
            const rsrc_t rs = TI ? (x == 0 ? cb.k : cb.q) : (x == 0 ? cb.a : x == 1 ? cb.p : x == 2 ? cb.k : cb.q);
            buf_ld128_lds(rs, sIn + blk * 256, (uint32_t)(t * H * DK + col) * 4);
        }
        pr = bld32(cb.r, (uint32_t)((lane & 31) * H) * 4);
        if (g.dyvar) {
            const rsrc_t rg = make_rsrc(g.dyvar + tok0 * H + h, (uint32_t)((nt - 1) * H + 1) * 4);
            pgv = bld32(rg, (uint32_t)((lane & 31) * H) * 4);
        } else {
            pgv = 0.f;
        }
        const size_t v0 = (tok0 * H + h) * DV;
        const uint32_t vbytes = (uint32_t)((nt - 1) * H * DV + DV) * 4;
        const int t = NVE * tid / DV, d = NVE * tid % DV;
        bldN<NVE>(make_rsrc(fv + v0, vbytes), (uint32_t)(t * H * DV + d) * 4, pv);
        bldN<NVE>(make_rsrc(fdy + v0, vbytes), (uint32_t)(t * H * DV + d) * 4, pdy);
        const double* hs = saved_H + ((size_t)bh * (nchunk + 1) + cn) * DK * DV + NHE * tid;
        if constexpr (NHE == 1) {
            ph0[0] = hs[0];
        } else {
#pragma unroll
            for (int i = 0; i < NHE / 2; ++i) {
                const double2 hv = reinterpret_cast<const double2*>(hs)[i];
                ph0[2 * i] = hv.x;
                ph0[2 * i + 1] = hv.y;
            }
        }
        plam = saved_lam[((size_t)bh * nchunk + cn) * DK + n];
    };
    // the fetched chunk becomes the next one: v, dy and the saved state into their fp64 tiles,
    // the per-lane values into the carried registers (after the wait for this wave's loads;
    // a barrier then publishes sIn and the tiles)
    double lam_c = 1.0;
    float rc = 0.f, gvc = 0.f;
    auto take = [&]() {
        wait_vm_le<0>();
        const int t = NVE * tid / DV, d = NVE * tid % DV;
#pragma unroll
        for (int i = 0; i < NVE; ++i) {
            sV[t * PV + d + i] = (double)pv[i];
            sDY[t * PV + d + i] = (double)pdy[i];
        }
        const int hr = NHE * tid / DV, hc = NHE * tid % DV;
#pragma unroll
        for (int i = 0; i < NHE; ++i) sH0[hr * PV + hc + i] = ph0[i];
        lam_c = plam;
        rc = pr;
        gvc = pgv;
    };

    // A round's gradients are staged in LDS (dV by the MFMA waves, the rest by the walk lanes,
    // dr by the last lane of each group) and stored at the start of the next round, 16 or 8
    // bytes per thread and row set, through buffers that drop the tokens past the end.
    const bool dvown = FULL || wave < NTT * NTD;
    const int tj = wave / NTD, dd = wave % NTD;   // this wave's dV tile
    int oc = -1;
    auto flush = [&]() {
        if (oc < 0) return;
        const int nt = min(C, T - oc * C);
        const size_t tok0 = seq0 + (size_t)oc * C;
        {
            const int t = NVE * tid / DV, d = NVE * tid % DV;
            const rsrc_t rv = make_rsrc(gdv + (tok0 * H + h) * DV, (uint32_t)((nt - 1) * H * DV + DV) * 4);
            bstN_lds<NVE>(rv, (uint32_t)(t * H * DV + d) * 4, sDv + t * SVD + d);
        }
        const size_t k0 = (tok0 * H + h) * DK;
        const uint32_t kbytes = (uint32_t)((nt - 1) * H * DK + DK) * 4;
        const int t = NKE * tid / DK, col = NKE * tid % DK;
        const uint32_t vo = (uint32_t)(t * H * DK + col) * 4;
        bstN_lds<NKE>(make_rsrc(gdq + k0, kbytes), vo, sOut + t * SO + col);
        bstN_lds<NKE>(make_rsrc(gdk + k0, kbytes), vo, sOut + C * SO + t * SO + col);
        if constexpr (!TI) {
            bstN_lds<NKE>(make_rsrc(gda + k0, kbytes), vo, sOut + 2 * C * SO + t * SO + col);
            bstN_lds<NKE>(make_rsrc(gdp + k0, kbytes), vo, sOut + 3 * C * SO + t * SO + col);
        }
        if (tid < C)
            bst32(make_rsrc(gdr + tok0 * H + h, (uint32_t)((nt - 1) * H + 1) * 4), (uint32_t)(tid * H) * 4, sDr[tid]);
    };

    auto round = [&](int c) {
        const int nt = min(C, T - c * C);
        flush();
        // ---- the lane's tokens from the staged rows, and their group transfer; then the fetch of
        // the previous chunk (sIn is free once every lane has read it)
        WalkIn<DK, TPG, TI> wi;
        wi.ca = ca;
        wi.cp = cp;
        wi.nv = min(max(nt - gq * TPG, 0), TPG);
        double gv[TPG];
#pragma unroll
        for (int j = 0; j < TPG; ++j) {
            const int t = gq * TPG + j;
            if constexpr (!TI) {
                wi.a[j] = sIn[t * DK + n];
                wi.p[j] = sIn[C * DK + t * DK + n];
            }
            wi.k[j] = sIn[(NIN - 2) * C * DK + t * DK + n];
            wi.q[j] = sIn[(NIN - 1) * C * DK + t * DK + n];
            wi.r[j] = __shfl(rc, t, 64);
            gv[j] = (double)__shfl(gvc, t, 64);
        }
        group_transfer(wi, qs, gq, n);
        barrier_lds();
        if (c >= 1) prefetch(c - 1);

        // ---- the walk over the lane's tokens: Qp, Kn, and what the adjoint walk needs
        // (kept across the contractions: lam_{t-1}, P_t, 1 / lam_t, rho_t and 1 / rho_t; the step
        // coefficients of the adjoint walk are formed in its first pass and kept for the second)
        double lam_p[TPG], P_t[TPG], il_t[TPG], rho[TPG], irho[TPG];
        {
            double x, z, A;
            chain_start<DK, G>(qs, gq, n, lam_c, x, z, A);
            double izp = rcpa(z);
#pragma unroll
            for (int j = 0; j < TPG; ++j) {
                const int t = gq * TPG + j;
                const double av = wi.A(j), kv = wi.K(j);
                const double kr = kv * wi.R(j);
                const double zn = fma(wi.P(j), x, av * av * z);
                const double xn = fma(kr * kv, zn, x);
                const double An = A * av;
                const double R = rcpa(xn * An), iz = rcpa(zn);
                const double AR = An * R, XR = xn * R;   // 1 / x_t, 1 / A_t
                const double qp = wi.Q(j) * An * AR, kn = kr * zn * XR;
                chk = fma(qp, kn, chk);
                sQp[t * PQ + n] = qp;
                sKn[t * PQ + n] = kn;
                lam_p[j] = x * izp;
                P_t[j] = An * iz;
                il_t[j] = zn * AR;
                rho[j] = z * iz;
                irho[j] = zn * izp;   // 1 / rho_t = z_t / z_{t-1}
                izp = iz;
                x = xn;
                z = zn;
                A = An;
            }
            if (gq == G - 1) sPC[n] = A * rcpa(z);
        }
        barrier_lds();   // Qp, Kn, P_C in

        // ---- S = M(Qp Kn^T) and B = M(dY V^T): tiles (0,0), (1,0), (1,1) of each from waves
        // 0..2 (wave 3 repeats the last, unstored); the tiles (1,0) also write the zero tile above
        // the diagonal.  Gs = diag(P_C) G
        {
            const int st = wave < 3 ? wave : 2;
            const int si = st == 0 ? 0 : 1, sj = st == 2 ? 1 : 0;
            const d4 sa = tile_mm<DK, PQ, 1, 1, PQ>(zero_d4(), sQp + 16 * si * PQ, sKn + 16 * sj * PQ, lane);
            const d4 ba = tile_mm<DV, PV, 1, 1, PV>(zero_d4(), sDY + 16 * si * PV, sV + 16 * sj * PV, lane);
            if (wave < 3) {
                for (int r = 0; r < 4; ++r) {
                    const int i = drow(r, lane), j = lane & 15;
                    const bool up = si == sj && j > i;
                    sS[(16 * si + i) * PS + 16 * sj + j] = up ? 0.0 : sa[r];
                    sB[(16 * si + i) * PS + 16 * sj + j] = up ? 0.0 : ba[r];
                }
                if (si != sj)
                    for (int r = 0; r < 4; ++r) {
                        sS[drow(r, lane) * PS + 16 + (lane & 15)] = 0.0;
                        sB[drow(r, lane) * PS + 16 + (lane & 15)] = 0.0;
                    }
            }
        }
        if (gown)
            for (int r = 0; r < 4; ++r) {
                const int row = 16 * tn + drow(r, lane);
                Gt[r] *= sPC[row];
                sGs[row * PV + 16 * td + (lane & 15)] = Gt[r];
            }
        barrier_lds();   // S, B, Gs in

        // ---- dV = S^T dY + Kn Gs (tiles (tj, td)); X = dY H0^T + B Kn and Y = B^T Qp + V Gs^T
        // (tiles (t, tn)); G' = Qp^T dY + Gs (this wave's tile)
        if (dvown) {
            d4 acc = tile_mm<C, 1, PS, PV, 1>(zero_d4(), sS + 16 * tj, sDY + 16 * dd, lane);
            acc = tile_mm<DK, PQ, 1, PV, 1>(acc, sKn + 16 * tj * PQ, sGs + 16 * dd, lane);
            for (int r = 0; r < 4; ++r) sDv[(16 * tj + drow(r, lane)) * SVD + 16 * dd + (lane & 15)] = (float)acc[r];
        }
        __builtin_amdgcn_sched_barrier(0);   // one job's operands in registers at a time
        if (FULL || wave < NTT * NTN) {
            const int tq = wave / NTN, nn = wave % NTN;
            d4 xa = tile_mm<DV, PV, 1, 1, PV>(zero_d4(), sDY + 16 * tq * PV, sH0 + 16 * nn * PV, lane);
            xa = tile_mm<C, PS, 1, PQ, 1>(xa, sB + 16 * tq * PS, sKn + 16 * nn, lane);
            d4 ya = tile_mm<C, 1, PS, PQ, 1>(zero_d4(), sB + 16 * tq, sQp + 16 * nn, lane);
            ya = tile_mm<DV, PV, 1, 1, PV>(ya, sV + 16 * tq * PV, sGs + 16 * nn * PV, lane);
            for (int r = 0; r < 4; ++r) {
                const int t = 16 * tq + drow(r, lane), col = 16 * nn + (lane & 15);
                sX[t * PQ + col] = xa[r];
                sY[t * PQ + col] = ya[r];
            }
        }
        __builtin_amdgcn_sched_barrier(0);
        if (gown) Gt = tile_mm<C, 1, PQ, PV, 1>(Gt, sQp + 16 * tn, sDY + 16 * td, lane);
        barrier_lds();   // X, Y in

        // ---- adjoint pass 1: the lane's tokens in reverse, each the affine step
        //   (c, S) -> (alpha (c - w) - beta (S + u), S + u),
        // composed into c_out = Am c_in + Bm S_in + Cm, S_out = S_in + Dm
        // per token of the lane: u, w and the step coefficients alpha = abar^2 rho^2, beta = pbar rho
        double dqt_[TPG], dkh_[TPG];
        auto coef = [&](int j, double& u, double& w, double& al, double& be) {
            const double qv = wi.Q(j), av = wi.A(j);
            const double qi = qv * il_t[j];
            u = qi * dqt_[j] - wi.K(j) * wi.R(j) * dkh_[j];
            w = qi * fma(qv, gv[j], dqt_[j]) * il_t[j];
            al = av * av * rho[j] * rho[j];
            be = wi.P(j) * rho[j];
        };
        double Am = 1.0, Bm = 0.0, Cm = 0.0, Dm = 0.0;
        double cu[TPG], cw[TPG], cal[TPG], cbe[TPG];   // the step coefficients, kept for pass 2
#pragma unroll
        for (int j = TPG - 1; j >= 0; --j) {
            const int t = gq * TPG + j;
            dqt_[j] = P_t[j] * sX[t * PQ + n];
            dkh_[j] = sY[t * PQ + n] * rcpa(P_t[j]);
            double u, w, al, be;
            coef(j, u, w, al, be);
            cu[j] = u;
            cw[j] = w;
            cal[j] = al;
            cbe[j] = be;
            Cm = al * Cm - be * Dm - (al * w + be * u);
            Bm = al * Bm - be;
            Am = al * Am;
            Dm = Dm + u;
        }
        qs[(gq * 4 + 0) * DK + n] = Am;   // the transfers were last read before two barriers
        qs[(gq * 4 + 1) * DK + n] = Bm;
        qs[(gq * 4 + 2) * DK + n] = Cm;
        qs[(gq * 4 + 3) * DK + n] = Dm;
        barrier_lds();

        // ---- pass 2: carries into the lane's group (through the later groups) and out of the
        // chunk, then the gradients of its tokens
        double cc, SS, drt[TPG];
        {
            const double* car = sCar + ((c + 1) & 1) * 2 * DK;
            double cT = car[n], ST = car[DK + n];
            cc = cT;
            SS = ST;
            for (int g2 = G - 1; g2 >= 0; --g2) {
                if (g2 == gq) {
                    cc = cT;
                    SS = ST;
                }
                const double A2 = qs[(g2 * 4 + 0) * DK + n], B2 = qs[(g2 * 4 + 1) * DK + n];
                const double C2 = qs[(g2 * 4 + 2) * DK + n], D2 = qs[(g2 * 4 + 3) * DK + n];
                const double cn = fma(A2, cT, fma(B2, ST, C2));
                ST += D2;
                cT = cn;
            }
            if (gq == 0) {
                sCar[(c & 1) * 2 * DK + n] = cT;
                sCar[(c & 1) * 2 * DK + DK + n] = ST;
            }
        }
#pragma unroll
        for (int j = TPG - 1; j >= 0; --j) {
            const int t = gq * TPG + j;
            const double u = cu[j], w = cw[j], al = cal[j], be = cbe[j];
            SS += u;
            const double gl = cc - w;
            const double kv = wi.K(j), rv = wi.R(j), av = wi.A(j), qv = wi.Q(j);
            const double r2 = rho[j] * rho[j];
            const double dkv = fma(2.0 * kv * rv, gl, rv * dkh_[j]);
            const double drho = fma(gl, lam_p[j], SS * irho[j]);
            const double dav = fma(-2.0 * av * r2, drho, SS * rcpa(av));
            const double dpv = -lam_p[j] * r2 * drho;
            const double dqv = fma(2.0 * qv, gv[j], dqt_[j]) * il_t[j];
            drt[j] = fma(kv * kv, gl, kv * dkh_[j]);
            cc = fma(al, gl, -be * SS);
            sOut[t * SO + n] = (float)dqv;
            sOut[C * SO + t * SO + n] = (float)dkv;
            if constexpr (!TI) {
                sOut[2 * C * SO + t * SO + n] = (float)dav;
                sOut[3 * C * SO + t * SO + n] = (float)dpv;
            }
            if (TI && t < nt) {
                sum_da += dav;
                sum_dp += dpv;
            }
        }
#pragma unroll
        for (int j = 0; j < TPG; ++j) {   // dr: the sum over the slots
            const double dr = slot_sum<DK>(drt[j]);
            if (n == DK - 1) sDr[gq * TPG + j] = (float)dr;
        }
        oc = c;
        if (c >= 1) take();
        barrier_lds();   // qs free for the next chunk's transfers; the next chunk staged
    };

    if (nchunk > 0) {
        prefetch(nchunk - 1);
        take();
    }
    barrier_lds();
    for (int c = nchunk - 1; c >= 0; --c) round(c);
    flush();

    // ---- gradients of the initial belief, and the OU gate sums
    if (g.dlam0 && tid < DK) g.dlam0[(size_t)bh * DK + tid] = (float)sCar[tid];
    if (g.deta0 && gown)
        for (int r = 0; r < 4; ++r)
            g.deta0[((size_t)bh * DK + 16 * tn + drow(r, lane)) * DV + 16 * td + (lane & 15)] = (float)Gt[r];
    if constexpr (TI) {
        double* part = static_cast<double*>(g.ou_part);
        const size_t np = (size_t)s.B * s.H * DK;
        // the slot's sum over all token groups (tids n, n + DK, ...), through LDS
        barrier_lds();
        sX[gq * PQ + n] = sum_da;
        sY[gq * PQ + n] = sum_dp;
        barrier_lds();
        if (tid < DK) {
            double sa = 0.0, sp = 0.0;
            for (int g2 = 0; g2 < G; ++g2) {
                sa += sX[g2 * PQ + tid];
                sp += sY[g2 * PQ + tid];
            }
            part[(size_t)bh * DK + tid] = sa;
            part[np + (size_t)bh * DK + tid] = sp;
        }
    }
    if (g.range_flag && !(fabs(chk) <= 1.0e300)) *g.range_flag = 1;
}

template <int DK, int DV>
hipError_t launch_fwd64(const Shape& s, const FwdArgs& a, void* saved, hipStream_t st) {
    double* slam = static_cast<double*>(saved);
    double* sH = slam ? slam + (size_t)s.B * s.H * ((s.T + kC64 - 1) / kC64) * DK : nullptr;
    const dim3 grid((unsigned)(s.B * s.H));
    if (a.ou_a)
        hipLaunchKernelGGL((fwd64_kernel<DK, DV, true>), grid, dim3(2 * kWT), 0, st, s, a, slam, sH);
    else
        hipLaunchKernelGGL((fwd64_kernel<DK, DV, false>), grid, dim3(2 * kWT), 0, st, s, a, slam, sH);
    return hipGetLastError();
}

template <int DK, int DV>
hipError_t launch_bwd64(const Shape& s, const BwdArgs& a, const void* saved, hipStream_t st) {
    if (!saved) return hipErrorInvalidValue;
    const double* slam = static_cast<const double*>(saved);
    const double* sH = slam + (size_t)s.B * s.H * ((s.T + kC64 - 1) / kC64) * DK;
    const dim3 grid((unsigned)(s.B * s.H));
    if (a.ou_a)
        hipLaunchKernelGGL((bwd64_kernel<DK, DV, true>), grid, dim3(kNT64), 0, st, s, a, slam, sH);
    else
        hipLaunchKernelGGL((bwd64_kernel<DK, DV, false>), grid, dim3(kNT64), 0, st, s, a, slam, sH);
    return hipGetLastError();
}

}  // namespace

bool c64_supported(const Shape& s) { return !s.bf16 && (s.dk == 16 || s.dk == 32) && (s.dv == 16 || s.dv == 32); }

size_t c64_saved_bytes(const Shape& s) {
    const size_t nchunk = (size_t)(s.T + kC64 - 1) / kC64;
    return (size_t)s.B * s.H * s.dk * (nchunk + (nchunk + 1) * (size_t)s.dv) * sizeof(double);
}

#define KLA_C64_CASES(F, ...)                                    \
    if (s.dk == 16 && s.dv == 16) return F<16, 16>(__VA_ARGS__); \
    if (s.dk == 16 && s.dv == 32) return F<16, 32>(__VA_ARGS__); \
    if (s.dk == 32 && s.dv == 16) return F<32, 16>(__VA_ARGS__); \
    if (s.dk == 32 && s.dv == 32) return F<32, 32>(__VA_ARGS__);

hipError_t launch_forward_c64(const Shape& s, const FwdArgs& a, void* saved, hipStream_t st) {
    KLA_C64_CASES(launch_fwd64, s, a, saved, st)
    return hipErrorInvalidValue;
}

hipError_t launch_backward_c64(const Shape& s, const BwdArgs& a, const void* saved, hipStream_t st) {
    KLA_C64_CASES(launch_bwd64, s, a, saved, st)
    return hipErrorInvalidValue;
}

}  // namespace kla
