// Chunked backward, key side: dq, dk, dabar, dpbar, dr and dlam0.
//
// Notation per chunk of kC = 32 tokens (local t), with P_t, Qp, Kn from the
// precision walk (kla_chunk.hpp) redone from the saved walk state:
//   H_t  = P_t (H0 + sum_{j<=t} Kn_j v_j^T)          (state rows, H0 = saved chunk-start state)
//   G    = adjoint of the chunk's last state from later tokens (detaT for the
//          last chunk), Gs = diag(P_C) G
//   B    = dY V^T                                    (kC x kC)
// then, with M() keeping j <= t,
//   X    = dY H0^T + M(B) Kn     dqt = P X   (gradient of qt = q / lam_t)
//   Y    = M(B)^T Qp + V Gs^T    dkh = Y / P (gradient of kh = r k)
//   G'   = Qp^T dY + Gs                          (carried into the previous chunk)
// The adjoint of log F_t is the reverse running sum S_t of qt dqt - kh dkh (plus
// the final-state term sum_d detaT H_T).  Over a whole chunk the attention parts of
// X and Y cancel exactly: the chunk's total of qt dqt - kh dkh is
// sum_t Qp_t (dY H0^T)_t - sum_j Kn_j (V Gs^T)_j, and S is carried from chunk to
// chunk by that total (per token, only within the chunk, by the running sum);
// summed token by token, the rounding of the large attention terms would add up
// over the sequence.  The adjoint c of lam follows
//   g_t = c_t - q_t dqt_t / lam_t^2,    c_T = dlamT,
//   c_{t-1} = abar_t^2 rho_t^2 g_t - pbar_t rho_t S_t,
// from which the input gradients follow by the chain rule through rho, lam, F
// (Theorem 1's update, differentiated by hand):
//   dq = dqt / lam,  dk = r dkh + 2 k r g,  dr = sum_n (k dkh + k^2 g),
//   drho = g lam_{t-1} + S / rho,  dabar = S / abar - 2 abar rho^2 drho,
//   dpbar = -lam_{t-1} rho^2 drho,  dlam0 = c after the first token.
// An upstream gradient gv_t of the readout variance yvar_t = sum_n q^2 / lam_t
// adds 2 q gv / lam to dq and -q^2 gv / lam^2 to g_t (YG instantiations; the
// others leave out its load and arithmetic).
//
// One workgroup per (batch, head, 64 key slots); a pair of waves owns 16 key
// slots n0 + 16 p .. + 15, and the pairs share only the dY / V tiles.  Wave e of
// a pair takes the tokens 16 e .. 16 e + 15 of each chunk in the walks:
//   walk   lanes = (slot nl = lane % 16, group g = lane / 16 of 4 tokens): each
//          lane forms its group's transfer -- the 2x2 map of (x, z) of
//          Theorem 1 over 4 tokens, with prod abar --, the four groups of each
//          half (the wave's four 16-lane rows) are chained by lane swaps from
//          the saved state at the start of the half (lam_0, or lam_16 and
//          P_16), and each lane walks its 4 tokens from the group start,
//          writing Qp and Kn ([t][16], split bf16) and keeping lam_t, P_t and
//          the reciprocals the adjoint walk needs;
//   MFMA   split by operand instead: wave 0 forms B^T and X^T (with the chunk's
//          saved start state H0 in registers), wave 1 forms B and Y^T and
//          carries G^T[dv, 16] in registers;
//   adjoint per lane: its group's tokens in reverse, once to summarise the
//          group as an affine map of the incoming (c, S), then -- the groups
//          chained through LDS -- once more for the gradients.
// The chunks are walked last to first, four LDS barriers per chunk separating
// the phases.  The next chunk's inputs go straight into LDS, requested during
// the first pass of a round's adjoint walk; the chunk's saved state rows come
// into wave 0's registers at the start of its round.
//
// TI (gates from OU parameters, the same for every token of a key slot): abar
// and pbar are formed once per lane and not loaded; dabar and dpbar are not
// stored per token but summed over the lane's tokens, one part per (batch row,
// wave of the pair), for the parameter gradients.
#include <type_traits>

#include "kla_chunk.hpp"
#include "kla_internal.hpp"

namespace kla {
namespace {

template <int DK, int DV>
struct DkCfg {
    static constexpr int NP = DK / 16 < 4 ? DK / 16 : 4;   // wave pairs, 16 key slots each
    static constexpr int NW = 2 * NP;                       // waves
    static constexpr int NTN = 16 * NP;                     // key slots per workgroup
    static constexpr int NNT = DK / NTN;                    // workgroups per (b, h)
    static constexpr int NTHR = 64 * NW;
    static constexpr int KSD = DV / 32;                     // 32-deep steps over the value channels
    static constexpr int NRD = DV / 16;                     // 16-row tiles over the value channels
    static constexpr int CPR = DV / 8;                      // 16-byte chunks per dY / V row
    static constexpr int TPV = 512 / DV;                    // rows per 1 KiB load of a dY / V tile
    static constexpr int NVL = kC / TPV;                    // 1 KiB loads per dY / V tile
    static constexpr int LQ2 = 24;                          // row stride of per-pair [t][16] bf16 tiles
    static constexpr int LX = 20;                           // row stride of per-pair [t][16] fp32 tiles
    static constexpr int NG = 8;                            // token groups per chunk (4 tokens each)
    // shared: dY and V tiles [2 buffers][2][kC][DV] (16-byte chunks swizzled by row)
    static constexpr int TILE = kC * DV * 2;
    static constexpr int PAIR0 = 2 * 2 * TILE;
    // per pair (offsets from the pair's base)
    static constexpr int STG = 0;                                   // [2][4][kC][16] bf16: abar, pbar, k, q
    static constexpr int RW = STG + 2 * 4 * kC * 16 * 2;            // [2][64] r words
    static constexpr int LW = RW + 2 * 64 * 4;                      // [2][64] walk state: lam_0, lam_16, P_16 [3][16]
    static constexpr int GV = LW + 2 * 64 * 4;                      // [2][64] yvar gradient (fp32)
    static constexpr int QH = GV + 2 * 64 * 4;                      // Qp, Kn split bf16 [kC][LQ2]
    static constexpr int QL = QH + kC * LQ2 * 2, KH = QL + kC * LQ2 * 2, KL = KH + kC * LQ2 * 2;
    static constexpr int XT = KL + kC * LQ2 * 2, YT = XT + kC * LX * 4;   // X, Y fp32 [kC][LX]
    static constexpr int QS = YT + kC * LX * 4;                     // adjoint group summaries [NG][4][16] fp32
    static constexpr int PC = QS + NG * 4 * 16 * 4;                 // chunk decay P_C [16] fp32
    static constexpr int WT = PC + 16 * 4;                          // chunk totals of the state parts [2][16]
    static constexpr int PAIR = (WT + 2 * 16 * 4 + 15) / 16 * 16;
    static constexpr int BYTES = PAIR0 + NP * PAIR;   // dynamic part
    // The gradient tiles dq, dk, dabar, dpbar [4][kC][16] bf16 and the dr terms
    // [kC][17] fp32 of each pair live in separate static arrays: they are read
    // back while the next chunk's direct-to-LDS loads are in flight, and as
    // distinct objects they are seen not to alias those loads' destinations.
    static constexpr int STATIC = NP * (4 * kC * 16 * 2 + kC * 17 * 4);
    static_assert(DK >= 32 && DK % 16 == 0 && DV >= 32 && DV % 32 == 0, "backward tile sizes");
    static_assert(NVL >= 1 && TPV * CPR == 64, "value tile loads");
    static_assert(4 + 2 * ((NVL + NW - 1) / NW) <= 8, "requests spread over 4 tokens, two each");
    static_assert(3 + 2 * ((NVL + NW - 1) / NW) <= 8, "requests spread over 4 tokens, two each");
    static_assert(BYTES + STATIC <= 160 * 1024, "LDS budget of one workgroup");
};

// Element (row t, column d) of a swizzled [kC][DV] bf16 tile: the 16-byte chunk
// d / 8 of row t sits at chunk (d / 8) ^ (t % CPR), so that 16 consecutive rows
// read at one column fall into distinct banks.
template <int DV>
__device__ __forceinline__ const uint16_t* swz(const uint16_t* tile, int t, int d) {
    constexpr int CPR = DV / 8;
    return tile + t * DV + ((((d >> 3) ^ (t % CPR)) << 3) | (d & 7));
}

template <int DV>
__device__ __forceinline__ bf16x8 lds8_swz(const uint16_t* tile, int t, int d0) {
    return lds8(swz<DV>(tile, t, d0));
}

template <int DV>
__device__ __forceinline__ bf16x8 lds4x2_swz(const uint16_t* tile, int t, int d0, int d1) {
    return lds4x2(swz<DV>(tile, t, d0), swz<DV>(tile, t, d1));
}

// lds_tr8 over a swizzled tile: lane s receives tile[rowA + j][col0 + s] and
// tile[rowB + j][col0 + s], j = 0..3 (col0 a multiple of 16)
template <int DV>
__device__ __forceinline__ bf16x8 lds_tr8_swz(const uint16_t* tile, int rowA, int rowB, int col0, int s) {
    const int col = col0 + 4 * (s & 3);
    const bf16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t*)swz<DV>(tile, rowA + (s >> 2), col));
    const bf16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t*)swz<DV>(tile, rowB + (s >> 2), col));
    return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}

// sum over each 16-lane row, held by every lane of the row
__device__ __forceinline__ float row_sum16f(float x) {
    x += dpp<0xB1, 0xf>(x);    // quad_perm [1,0,3,2]
    x += dpp<0x4E, 0xf>(x);    // quad_perm [2,3,0,1]
    x += dpp<0x141, 0xf>(x);   // row_half_mirror
    x += dpp<0x140, 0xf>(x);   // row_mirror
    return x;
}

__device__ __forceinline__ void buf_st128(uint4 v, rsrc_t r, uint32_t voff) {
    typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;
    __builtin_amdgcn_raw_buffer_store_b128(u32x4{v.x, v.y, v.z, v.w}, r, voff, 0, 0);
}

__device__ __forceinline__ void buf_st32(float v, rsrc_t r, uint32_t voff) {
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, voff, 0, 0);
}

template <int DK, int DV, bool TI, bool YG>
__global__ __launch_bounds__((DkCfg<DK, DV>::NTHR)) void bwd_dk_kernel(Shape s, BwdArgs g,
                                                                       const float* __restrict__ saved_lam,
                                                                       const float* __restrict__ saved_H,
                                                                       float* __restrict__ dr_part) {
    using Cfg = DkCfg<DK, DV>;
    constexpr int NP = Cfg::NP, NW = Cfg::NW, KSD = Cfg::KSD, NRD = Cfg::NRD, LQ2 = Cfg::LQ2, LX = Cfg::LX;
    constexpr int NG = Cfg::NG;
    constexpr int NST = TI ? 3 : 5;   // gradient stores per round: dq, dk(, dabar, dpbar) and dr
    extern __shared__ __align__(16) unsigned char smem[];
    __shared__ __align__(16) uint16_t s_out[NP * 4 * kC * 16];
    __shared__ __align__(16) float s_drc[NP * kC * 17];

    const uint16_t* a = static_cast<const uint16_t*>(g.a);
    const uint16_t* p = static_cast<const uint16_t*>(g.p);
    const uint16_t* k = static_cast<const uint16_t*>(g.k);
    const uint16_t* q = static_cast<const uint16_t*>(g.q);
    const uint16_t* r = static_cast<const uint16_t*>(g.r);
    const uint16_t* vv = static_cast<const uint16_t*>(g.v);
    const uint16_t* dy = static_cast<const uint16_t*>(g.dy);

    int bh, ntile;
    xcd_tile_map(blockIdx.x, s.B * s.H, Cfg::NNT, bh, ntile);
    const int b = bh / s.H, h = bh % s.H;
    const int H = s.H, T = s.T;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int pr = wave % NP, e = wave / NP;     // pair, half of the chunk (a pair shares a SIMD)
    const int l16 = lane & 15, g4 = lane >> 4;   // MFMA lane coordinates
    const int nl = l16, gg = 4 * e + g4;         // walk lanes: slot, token group (tokens 4 gg .. 4 gg + 3)
    const int n0w = ntile * Cfg::NTN + 16 * pr;  // the pair's first key slot
    const int nchunk = (T + kC - 1) / kC;
    const size_t seq0 = (size_t)b * T;
    const size_t nbt = (size_t)s.B * T * H;
    unsigned char* wb = smem + Cfg::PAIR0 + pr * Cfg::PAIR;
    const uint32_t tok_k = (uint32_t)H * DK * 2;   // bytes between tokens of a [.., H, DK] tensor
    const uint32_t tok_v = (uint32_t)H * DV * 2;

    // ---- carries of the reverse recursions (every lane of both waves holds its slot's values)
    float cT = g.dlamT ? g.dlamT[(size_t)bh * DK + n0w + nl] : 0.f;
    float ST = 0.f;
    if (g.detaT) {   // final-state term sum_d detaT H_T, split over the four lane groups
        const float* HT = saved_H + (((size_t)bh * (nchunk + 1) + nchunk) * DK + n0w + nl) * DV;
        const float* dT = g.detaT + ((size_t)bh * DK + n0w + nl) * DV;
        for (int d = g4 * (DV / 4); d < (g4 + 1) * (DV / 4); ++d) ST += dT[d] * HT[d];
    }
    ST += __shfl_xor(ST, 16, 64);
    ST += __shfl_xor(ST, 32, 64);
    // range check of the walk: Qp Kn (= q r k / lam) summed over the lane's tokens stays
    // finite exactly while every Qp and Kn is
    float chk = 0.f;
    // time-invariant gates of the slot and the lane's sums of their gradients
    float ca = 0.f, cp = 0.f, sum_da = 0.f, sum_dp = 0.f;
    if constexpr (TI) {
        const int o = h * DK + n0w + nl;
        ou_gates(g.ou_a[o], g.ou_p[o], g.ou_d[o], ca, cp);
    }

    // G^T[d, n] for d = 16 rd + 4 g4 + rr, n = n0w + l16 (carried by wave 1 of the pair)
    f32x4 GT[NRD];
#pragma unroll
    for (int rd = 0; rd < NRD; ++rd)
#pragma unroll
        for (int rr = 0; rr < 4; ++rr)
            GT[rd][rr] = (e == 1 && g.detaT) ? g.detaT[((size_t)bh * DK + n0w + l16) * DV + 16 * rd + 4 * g4 + rr] : 0.f;

    // ---- requests of chunk cn into buffer bb (chunks outside the sequence: empty, writing
    // zeros), one load per part so that they can be spread over a round:
    //   wave 0: 0..3  abar, pbar, k, q of the pair's slots (1 KiB each, lane -> (t = lane / 2, 8 slots));
    //                 TI: 0, 1  k, q
    //   wave 1: 0..2  r (lanes >= nt read as 0), the chunk-start lam of the 16 slots and (YG)
    //                 the yvar gradient
    //   then this wave's share of the dY and V tiles (loads i = wave, wave + NW, ...), swizzled
    const int nin = e == 0 ? (TI ? 2 : 4) : (YG ? 3 : 2);
    const int nvw = wave < Cfg::NVL ? (Cfg::NVL - wave + NW - 1) / NW : 0;
    const int nparts = nin + 2 * nvw;
    auto issue_part = [&](int cn, int bb, int part) {
        const bool in = cn >= 0 && cn < nchunk;
        const int t0 = in ? cn * kC : 0, nt = in ? min(kC, T - t0) : 0;
        const size_t tok0 = seq0 + t0;
        if (part < nin) {
            if (e == 0) {
                const int slot = TI ? part + 2 : part;   // staging slots: abar, pbar, k, q
                const uint16_t* src = slot == 0 ? a : slot == 1 ? p : slot == 2 ? k : q;
                const uint32_t kbytes = nt > 0 ? (uint32_t)((nt - 1) * H * DK + 16) * 2 : 0u;
                uint16_t* stg = reinterpret_cast<uint16_t*>(wb + Cfg::STG) + (bb * 4 + slot) * kC * 16;
                buf_ld128_lds(make_rsrc(src + (tok0 * H + h) * DK + n0w, kbytes), stg,
                              (uint32_t)(lane >> 1) * tok_k + (lane & 1) * 16);
            } else if (part == 0) {
                const rsrc_t rr = make_rsrc(r + tok0 * H + h, nt > 0 ? (uint32_t)((nt - 1) * H + 1) * 2 : 0u);
                buf_ld16_lds(rr, wb + Cfg::RW + bb * 256, (uint32_t)lane * H * 2);
            } else if (part == 2) {
                const rsrc_t rv = make_rsrc(g.dyvar + tok0 * H + h, nt > 0 ? (uint32_t)((nt - 1) * H + 1) * 4 : 0u);
                buf_ld32_lds(rv, wb + Cfg::GV + bb * 256, (uint32_t)lane * H * 4);
            } else {
                // lanes 16 i + l: row i of the saved walk state (lam_0, lam_16, P_16) for slot n0w + l
                const rsrc_t rl = make_rsrc(saved_lam + ((size_t)bh * nchunk + (in ? cn : 0)) * kLamRows * DK + n0w,
                                            in ? (uint32_t)(2 * DK + 16) * 4 : 0u);
                buf_ld32_lds(rl, wb + Cfg::LW + bb * 256, (uint32_t)((lane >> 4) * DK + (lane & 15)) * 4);
            }
        } else if (part < nparts) {
            const int m = (part - nin) >> 1, i = wave + NW * m, sel = (part - nin) & 1;
            const uint32_t vbytes = nt > 0 ? (uint32_t)((nt - 1) * H * DV + DV) * 2 : 0u;
            const rsrc_t rv = make_rsrc((sel ? vv : dy) + (tok0 * H + h) * DV, vbytes);
            const int row = i * Cfg::TPV + lane / Cfg::CPR, pch = lane % Cfg::CPR;
            const uint32_t off = (uint32_t)row * tok_v + (uint32_t)((pch ^ (row % Cfg::CPR)) * 16);
            buf_ld128_lds(rv, smem + (bb * 2 + sel) * Cfg::TILE + i * 1024, off);
        }
    };
    wait_vm_all();   // the carries and G^T are complete before the request stream starts
    if (nchunk > 0)
        for (int part = 0; part < nparts; ++part) issue_part(nchunk - 1, 0, part);

    for (int it = 0; it < nchunk; ++it) {
        const int c = nchunk - 1 - it, bb = it & 1;
        const int nt = min(kC, T - c * kC);
        const size_t row0 = seq0 + (size_t)c * kC;

        // the round's work for wave E of the pair; FULL: all kC tokens valid (no per-token guards)
        auto round_body = [&](auto full_tag, auto role_tag) {
            constexpr bool FULL = decltype(full_tag)::value;
            constexpr int E = decltype(role_tag)::value;
            // saved chunk-start state rows H0[n0w + l16][32 ks + 8 g4 .. + 7] (wave 0, for X)
            float4 h0[KSD][2];
            if constexpr (E == 0) {
                const float* H0 = saved_H + (((size_t)bh * (nchunk + 1) + c) * DK + n0w + l16) * DV;
#pragma unroll
                for (int ks = 0; ks < KSD; ++ks) {
                    h0[ks][0] = *reinterpret_cast<const float4*>(H0 + 32 * ks + 8 * g4);
                    h0[ks][1] = *reinterpret_cast<const float4*>(H0 + 32 * ks + 8 * g4 + 4);
                }
                // this chunk's requests (issued last round) have landed: younger are only the
                // last round's NST stores and the 2 KSD state loads just issued
                if (it == 0)
                    wait_vm_le<2 * KSD>();
                else
                    wait_vm_le<NST + 2 * KSD>();
            } else {
                if (it == 0)
                    wait_vm_le<0>();
                else
                    wait_vm_le<NST>();
            }
            barrier_lds();   // every wave's share of the dY / V tiles and staging is in

            const uint16_t* sDY = reinterpret_cast<const uint16_t*>(smem + bb * 2 * Cfg::TILE);
            const uint16_t* sV = sDY + kC * DV;
            const uint16_t* stg = reinterpret_cast<const uint16_t*>(wb + Cfg::STG) + bb * 4 * kC * 16;
            const uint32_t* rw = reinterpret_cast<const uint32_t*>(wb + Cfg::RW) + bb * 64;
            uint16_t* sQH = reinterpret_cast<uint16_t*>(wb + Cfg::QH);
            uint16_t* sQL = reinterpret_cast<uint16_t*>(wb + Cfg::QL);
            uint16_t* sKH = reinterpret_cast<uint16_t*>(wb + Cfg::KH);
            uint16_t* sKL = reinterpret_cast<uint16_t*>(wb + Cfg::KL);
            float* sX = reinterpret_cast<float*>(wb + Cfg::XT);
            float* sY = reinterpret_cast<float*>(wb + Cfg::YT);
            float* sPC = reinterpret_cast<float*>(wb + Cfg::PC);
            float* sWT = reinterpret_cast<float*>(wb + Cfg::WT);   // [2][16]: sum_t Qp X0, sum_j Kn Yg
            float* qs = reinterpret_cast<float*>(wb + Cfg::QS);
            auto in_a = [&](int t) {
                return TI ? ca : __uint_as_float((uint32_t)stg[(0 * kC + t) * 16 + nl] << 16);
            };
            auto in_p = [&](int t) {
                return TI ? cp : __uint_as_float((uint32_t)stg[(1 * kC + t) * 16 + nl] << 16);
            };
            auto in_k = [&](int t) { return __uint_as_float((uint32_t)stg[(2 * kC + t) * 16 + nl] << 16); };
            auto in_q = [&](int t) { return __uint_as_float((uint32_t)stg[(3 * kC + t) * 16 + nl] << 16); };
            auto in_r = [&](int t) { return __uint_as_float(rw[t] << 16); };
            const float* gvw = reinterpret_cast<const float*>(wb + Cfg::GV) + bb * 64;

            // ================================================================ phase 1
            // wave 0: B^T[j, t] = V_j . dY_t (j <= t), tiles (0,0), (0,1), (1,1), as operands over j;
            // wave 1: B[t, j] = dY_t . V_j (j <= t), tiles (0,0), (1,0), (1,1), as operands over t
            bf16x8 boh[2], bol[2];
            {
                f32x4 c0 = zero4(), c1 = zero4(), c2 = zero4();
#pragma unroll
                for (int ks = 0; ks < KSD; ++ks) {
                    const bf16x8 ya0 = lds8_swz<DV>(sDY, l16, 32 * ks + 8 * g4);
                    const bf16x8 ya1 = lds8_swz<DV>(sDY, 16 + l16, 32 * ks + 8 * g4);
                    const bf16x8 v0 = lds8_swz<DV>(sV, l16, 32 * ks + 8 * g4);
                    const bf16x8 v1 = lds8_swz<DV>(sV, 16 + l16, 32 * ks + 8 * g4);
                    if constexpr (E == 0) {
                        c0 = mfma_bf16(v0, ya0, c0);
                        c1 = mfma_bf16(v0, ya1, c1);
                        c2 = mfma_bf16(v1, ya1, c2);
                    } else {
                        c0 = mfma_bf16(ya0, v0, c0);
                        c1 = mfma_bf16(ya1, v0, c1);
                        c2 = mfma_bf16(ya1, v1, c2);
                    }
                }
#pragma unroll
                for (int rr = 0; rr < 4; ++rr) {
                    // B^T: row j = 4 g4 + rr, column t = l16; B: row t = 4 g4 + rr, column j = l16
                    const bool drop = E == 0 ? 4 * g4 + rr > l16 : l16 > 4 * g4 + rr;
                    if (drop) {
                        c0[rr] = 0.f;
                        c2[rr] = 0.f;
                    }
                }
                // rows {4g..}, {16+4g..} of the contraction
                if constexpr (E == 0) {
                    split8(c0, zero4(), boh[0], bol[0]);
                    split8(c1, c2, boh[1], bol[1]);
                } else {
                    split8(c0, c1, boh[0], bol[0]);
                    split8(zero4(), c2, boh[1], bol[1]);
                }
            }
            // the transfer of this lane's group: (x, z) -> M (x, z) over its valid tokens, as the
            // images of (1, 0) and (0, 1), and the product of abar
            float tr[5];
            {
                float x0 = 1.f, z0 = 0.f, x1 = 0.f, z1 = 1.f, Aq = 1.f;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int t = 4 * gg + j;
                    const float av = in_a(t), pv = in_p(t), kv = in_k(t), rv = in_r(t);
                    const float a2 = av * av, phi = kv * kv * rv;
                    const float z0n = fmaf(pv, x0, a2 * z0), z1n = fmaf(pv, x1, a2 * z1);
                    const bool ok = FULL || t < nt;
                    x0 = ok ? fmaf(phi, z0n, x0) : x0;
                    x1 = ok ? fmaf(phi, z1n, x1) : x1;
                    z0 = ok ? z0n : z0;
                    z1 = ok ? z1n : z1;
                    Aq = ok ? Aq * av : Aq;
                }
                tr[0] = x0;
                tr[1] = z0;
                tr[2] = x1;
                tr[3] = z1;
                tr[4] = Aq;
            }
            __builtin_amdgcn_sched_barrier(0);   // keep the phases apart in the schedule (register pressure)

            // ================================================================ phase 2
            // chain the wave's earlier groups from the saved state at the start of its half:
            // (x, z, A) = (lam_0, 1, 1) for tokens 0..15, (lam_16, 1, P_16) for 16..31.  A
            // wave's four groups are its four 16-lane rows, so the transfers of the earlier rows
            // are read across lanes (ds_bpermute), with no LDS store and no barrier.
            const float* lws = reinterpret_cast<const float*>(wb + Cfg::LW) + bb * 64;
            float x = lws[16 * E + nl], z = 1.f, A = E == 0 ? 1.f : lws[32 + nl];
#pragma unroll
            for (int q2 = 0; q2 < NG / 2 - 1; ++q2) {
                auto pick = [&](int i) { return __shfl(tr[i], 16 * q2 + nl, 64); };   // row q2, same column
                const float m00 = pick(0), m10 = pick(1), m01 = pick(2), m11 = pick(3), aq = pick(4);
                const bool use = q2 < g4;
                const float xn = fmaf(m00, x, m01 * z), zn = fmaf(m10, x, m11 * z);
                x = use ? xn : x;
                z = use ? zn : z;
                A = use ? A * aq : A;
            }
            float izp = fast_rcp(z);              // 1 / z before the group's first token
            const float lamq = x * izp;           // lam before the group's first token
            // per token of the group: lam_t, P_t and, for the adjoint walk, 1/P_t, 1/lam_t,
            // rho_t, 1/rho_t = abar^2 + pbar lam_{t-1}, 1/abar
            float lam_r[4], P_r[4], iP_r[4], il_r[4], rho_r[4], den_r[4], ia_r[4];
#pragma unroll
            for (int j2 = 0; j2 < 2; ++j2) {
                float qp2[2], kn2[2];
#pragma unroll
                for (int e2 = 0; e2 < 2; ++e2) {
                    const int j = 2 * j2 + e2, t = 4 * gg + j;
                    const float av = in_a(t), pv = in_p(t), kv = in_k(t), qv = in_q(t), rv = in_r(t);
                    const float kr = kv * rv;
                    const float zn = fmaf(pv, x, av * av * z);
                    const float xn = fmaf(kr * kv, zn, x);
                    const float An = A * av;
                    const float R = fast_rcp(xn * An);
                    const float iz = fast_rcp(zn);
                    const float AR = An * R, XR = xn * R;   // 1 / x_t, 1 / A_t
                    const bool ok = FULL || t < nt;
                    qp2[e2] = ok ? (qv * An) * AR : 0.f;
                    kn2[e2] = ok ? (kr * zn) * XR : 0.f;
                    chk = fmaf(qp2[e2], kn2[e2], chk);
                    lam_r[j] = xn * iz;
                    P_r[j] = An * iz;
                    iP_r[j] = zn * XR;
                    il_r[j] = zn * AR;
                    rho_r[j] = z * iz;
                    den_r[j] = zn * izp;
                    ia_r[j] = A * XR;
                    izp = iz;
                    x = ok ? xn : x;
                    z = ok ? zn : z;
                    A = ok ? An : A;
                }
                uint32_t qh, ql, kh, kl;
                split2(qp2[0], qp2[1], qh, ql);
                split2(kn2[0], kn2[1], kh, kl);
                const int t = 4 * gg + 2 * j2;
                sQH[t * LQ2 + nl] = static_cast<uint16_t>(qh);
                sQH[(t + 1) * LQ2 + nl] = static_cast<uint16_t>(qh >> 16);
                sQL[t * LQ2 + nl] = static_cast<uint16_t>(ql);
                sQL[(t + 1) * LQ2 + nl] = static_cast<uint16_t>(ql >> 16);
                sKH[t * LQ2 + nl] = static_cast<uint16_t>(kh);
                sKH[(t + 1) * LQ2 + nl] = static_cast<uint16_t>(kh >> 16);
                sKL[t * LQ2 + nl] = static_cast<uint16_t>(kl);
                sKL[(t + 1) * LQ2 + nl] = static_cast<uint16_t>(kl >> 16);
            }
            if (gg == NG - 1) sPC[nl] = A * fast_rcp(z);   // the last group ends at the chunk end
            barrier_lds();   // Qp, Kn of every token and P_C are in

            // ================================================================ phase 3
            if constexpr (E == 0) {
                // X^T[n, t] = sum_d H0[n, d] dY^T[d, t] + sum_j Kn^T[n, j] B^T[j, t]
                f32x4 xacc[2] = {zero4(), zero4()};
#pragma unroll
                for (int ks = 0; ks < KSD; ++ks) {
                    bf16x8 hh, hl;
                    split8(f32x4{h0[ks][0].x, h0[ks][0].y, h0[ks][0].z, h0[ks][0].w},
                           f32x4{h0[ks][1].x, h0[ks][1].y, h0[ks][1].z, h0[ks][1].w}, hh, hl);
#pragma unroll
                    for (int tt = 0; tt < 2; ++tt)
                        xacc[tt] = mfma2a(hh, hl, lds8_swz<DV>(sDY, 16 * tt + l16, 32 * ks + 8 * g4), xacc[tt]);
                }
                {   // chunk total of Qp X0 per slot n = 4 g4 + rr (tokens past the end have Qp = 0)
                    float w[4];
#pragma unroll
                    for (int rr = 0; rr < 4; ++rr) {
                        w[rr] = 0.f;
#pragma unroll
                        for (int tt = 0; tt < 2; ++tt) {
                            const int o = (16 * tt + l16) * LQ2 + 4 * g4 + rr;
                            const float qp = __uint_as_float((uint32_t)sQH[o] << 16) + __uint_as_float((uint32_t)sQL[o] << 16);
                            w[rr] = fmaf(qp, xacc[tt][rr], w[rr]);
                        }
                        w[rr] = row_sum16f(w[rr]);
                    }
                    if (l16 == 0)
#pragma unroll
                        for (int rr = 0; rr < 4; ++rr) sWT[4 * g4 + rr] = w[rr];
                }
                const bf16x8 knh = lds_tr8(sKH, LQ2, 4 * g4, 16 + 4 * g4, 0, l16);
                const bf16x8 knl = lds_tr8(sKL, LQ2, 4 * g4, 16 + 4 * g4, 0, l16);
#pragma unroll
                for (int tt = 0; tt < 2; ++tt) {
                    xacc[tt] = mfma3(knh, knl, boh[tt], bol[tt], xacc[tt]);
                    *reinterpret_cast<float4*>(sX + (16 * tt + l16) * LX + 4 * g4) =
                        float4{xacc[tt][0], xacc[tt][1], xacc[tt][2], xacc[tt][3]};
                }
            } else {
                // Y^T[n, j] = sum_d Gs[n, d] V^T[d, j] + sum_t Qp^T[n, t] B[t, j]: the state part
                // first, whose chunk total is taken before the attention part is added
                f32x4 yacc[2] = {zero4(), zero4()};
                const float pcn = sPC[l16];
#pragma unroll
                for (int rd = 0; rd < NRD; ++rd)
#pragma unroll
                    for (int rr = 0; rr < 4; ++rr) GT[rd][rr] *= pcn;   // Gs^T in place
#pragma unroll
                for (int ks = 0; ks < KSD; ++ks) {
                    bf16x8 gh, gl;
                    split8(GT[2 * ks], GT[2 * ks + 1], gh, gl);
#pragma unroll
                    for (int jt = 0; jt < 2; ++jt) {
                        const bf16x8 vb = lds4x2_swz<DV>(sV, 16 * jt + l16, 32 * ks + 4 * g4, 32 * ks + 16 + 4 * g4);
                        yacc[jt] = mfma2a(gh, gl, vb, yacc[jt]);
                    }
                }
                {   // chunk total of Kn Yg per slot n = 4 g4 + rr (tokens past the end have Kn = 0)
                    float w[4];
#pragma unroll
                    for (int rr = 0; rr < 4; ++rr) {
                        w[rr] = 0.f;
#pragma unroll
                        for (int jt = 0; jt < 2; ++jt) {
                            const int o = (16 * jt + l16) * LQ2 + 4 * g4 + rr;
                            const float kn = __uint_as_float((uint32_t)sKH[o] << 16) + __uint_as_float((uint32_t)sKL[o] << 16);
                            w[rr] = fmaf(kn, yacc[jt][rr], w[rr]);
                        }
                        w[rr] = row_sum16f(w[rr]);
                    }
                    if (l16 == 0)
#pragma unroll
                        for (int rr = 0; rr < 4; ++rr) sWT[16 + 4 * g4 + rr] = w[rr];
                }
                const bf16x8 qth = lds_tr8(sQH, LQ2, 4 * g4, 16 + 4 * g4, 0, l16);
                const bf16x8 qtl = lds_tr8(sQL, LQ2, 4 * g4, 16 + 4 * g4, 0, l16);
#pragma unroll
                for (int jt = 0; jt < 2; ++jt) yacc[jt] = mfma3(qth, qtl, boh[jt], bol[jt], yacc[jt]);
#pragma unroll
                for (int jt = 0; jt < 2; ++jt)
                    *reinterpret_cast<float4*>(sY + (16 * jt + l16) * LX + 4 * g4) =
                        float4{yacc[jt][0], yacc[jt][1], yacc[jt][2], yacc[jt][3]};
            }
            barrier_lds();   // X and Y of every token are in

            // ================================================================ phase 4
            // adjoint pass 1: the group's tokens in reverse; per token the affine step
            //   (c, S) -> (alpha (c - w) - beta (S + u), S + u)
            // composed into c_out = Am c_in + Bm S_in + Cm, S_out = S_in + Dm
            float u_[4], w_[4], al_[4], be_[4], dq_[4], rdk_[4], kr2_[4], ia_[4], a2r2_[4], lp_[4], den_[4], lpr2_[4],
                kdk_[4], kk_[4];
            float Am = 1.f, Bm = 0.f, Cm = 0.f, Dm = 0.f;
#pragma unroll
            for (int j = 3; j >= 0; --j) {
                const int t = 4 * gg + j;
                const float av = in_a(t), pv = in_p(t), kv = in_k(t), qv = in_q(t), rv = in_r(t);
                const float lam_p = j > 0 ? lam_r[j - 1] : lamq;
                const float Xv = sX[t * LX + nl], Yv = sY[t * LX + nl];
                const float rho = rho_r[j], ilam = il_r[j], ia = ia_r[j], den = den_r[j];
                const float dqt = P_r[j] * Xv, dkh = Yv * iP_r[j];
                const float kh = rv * kv;
                const float qi = qv * ilam, qg = YG ? qv * gvw[t] : 0.f;
                const bool ok = FULL || t < nt;
                const float u = ok ? qi * dqt - kh * dkh : 0.f;
                const float w = ok ? qi * (dqt + qg) * ilam : 0.f;
                const float rho2 = rho * rho;
                const float al = ok ? av * av * rho2 : 1.f;
                const float be = ok ? pv * rho : 0.f;
                u_[j] = u;
                w_[j] = w;
                al_[j] = al;
                be_[j] = be;
                dq_[j] = fmaf(2.f, qg, dqt) * ilam;
                rdk_[j] = rv * dkh;
                kr2_[j] = 2.f * kh;
                ia_[j] = ia;
                a2r2_[j] = 2.f * av * rho2;
                lp_[j] = lam_p;
                den_[j] = den;
                lpr2_[j] = lam_p * rho2;
                kdk_[j] = kv * dkh;
                kk_[j] = kv * kv;
                Cm = al * Cm - be * Dm - (al * w + be * u);
                Bm = al * Bm - be;
                Am = al * Am;
                Dm = Dm + u;
                // the next chunk's requests, two per token: they go out only after the
                // transposing LDS reads above (which would otherwise wait for them)
                issue_part(c - 1, bb ^ 1, 2 * (3 - j));
                issue_part(c - 1, bb ^ 1, 2 * (3 - j) + 1);
            }
            if constexpr (E == 1) {
                // G^T <- dY^T Qp + Gs^T
                const bf16x8 qbh = lds_tr8(sQH, LQ2, 8 * g4, 8 * g4 + 4, 0, l16);
                const bf16x8 qbl = lds_tr8(sQL, LQ2, 8 * g4, 8 * g4 + 4, 0, l16);
#pragma unroll
                for (int rd = 0; rd < NRD; ++rd) {
                    const bf16x8 yt = lds_tr8_swz<DV>(sDY, 8 * g4, 8 * g4 + 4, 16 * rd, l16);
                    GT[rd] = mfma2b(yt, qbh, qbl, GT[rd]);
                }
            }
            qs[(gg * 4 + 0) * 16 + nl] = Am;   // the last chunk's summaries were read before two barriers
            qs[(gg * 4 + 1) * 16 + nl] = Bm;
            qs[(gg * 4 + 2) * 16 + nl] = Cm;
            qs[(gg * 4 + 3) * 16 + nl] = Dm;
            barrier_lds();   // the group summaries are in

            // ================================================================ phase 5
            // carries into this group (through the later groups) and out of the chunk; S leaves
            // the chunk with the chunk's exact total, not the sum of its tokens' terms
            const float S_out = ST + (sWT[nl] - sWT[16 + nl]);
            float c_in = 0.f, S_in = 0.f;
#pragma unroll
            for (int q2 = NG - 1; q2 >= 0; --q2) {
                if (q2 == gg) {
                    c_in = cT;
                    S_in = ST;
                }
                const float A2 = qs[(q2 * 4 + 0) * 16 + nl], B2 = qs[(q2 * 4 + 1) * 16 + nl];
                const float C2 = qs[(q2 * 4 + 2) * 16 + nl], D2 = qs[(q2 * 4 + 3) * 16 + nl];
                const float cn = fmaf(A2, cT, fmaf(B2, ST, C2));
                ST += D2;
                cT = cn;
            }
            ST = S_out;
            // pass 2: gradients of the group's tokens
            uint16_t* so = s_out + pr * 4 * kC * 16;
            float* drc = s_drc + pr * kC * 17;
            float cc = c_in, SS = S_in;
#pragma unroll
            for (int j = 3; j >= 0; --j) {
                const int t = 4 * gg + j;
                SS += u_[j];
                const float gl = cc - w_[j];
                const float dkv = fmaf(kr2_[j], gl, rdk_[j]);
                const float drho = fmaf(gl, lp_[j], SS * den_[j]);
                const float dav = fmaf(-a2r2_[j], drho, SS * ia_[j]);
                const float dpv = -lpr2_[j] * drho;
                drc[t * 17 + nl] = fmaf(kk_[j], gl, kdk_[j]);
                cc = fmaf(al_[j], gl, -be_[j] * SS);
                const uint32_t pq = cvt_pk_bf16(dq_[j], dkv);
                so[(0 * kC + t) * 16 + nl] = static_cast<uint16_t>(pq);
                so[(1 * kC + t) * 16 + nl] = static_cast<uint16_t>(pq >> 16);
                if constexpr (TI) {
                    if (FULL || t < nt) {
                        sum_da += dav;
                        sum_dp += dpv;
                    }
                } else {
                    const uint32_t pa = cvt_pk_bf16(dav, dpv);
                    so[(2 * kC + t) * 16 + nl] = static_cast<uint16_t>(pa);
                    so[(3 * kC + t) * 16 + nl] = static_cast<uint16_t>(pa >> 16);
                }
            }

            // ---- stores of this wave's 16 tokens: [t][16] rows of dq, dk, dabar, dpbar (lanes
            // < 32: t = 16 E + lane / 2, 8 slots) and the pair's dr partial over its 16 slots
            // (lanes < 16: t = 16 E + lane); the other lanes address the end of the range and
            // are dropped, as are tokens past the sequence end
            {
                const int tl = 16 * E + ((lane >> 1) & 15);
                const uint32_t kbytes = (uint32_t)((nt - 1) * H * DK + 16) * 2;
                const size_t ek = (row0 * H + h) * DK + n0w;
                const uint32_t koff = lane < 32 ? (uint32_t)tl * tok_k + (lane & 1) * 16 : kbytes;
                const uint16_t* o = so + tl * 16 + (lane & 1) * 8;
                buf_st128(*reinterpret_cast<const uint4*>(o + 0 * kC * 16),
                          make_rsrc(static_cast<uint16_t*>(g.dq) + ek, kbytes), koff);
                buf_st128(*reinterpret_cast<const uint4*>(o + 1 * kC * 16),
                          make_rsrc(static_cast<uint16_t*>(g.dk) + ek, kbytes), koff);
                if constexpr (!TI) {
                    buf_st128(*reinterpret_cast<const uint4*>(o + 2 * kC * 16),
                              make_rsrc(static_cast<uint16_t*>(g.da) + ek, kbytes), koff);
                    buf_st128(*reinterpret_cast<const uint4*>(o + 3 * kC * 16),
                              make_rsrc(static_cast<uint16_t*>(g.dp) + ek, kbytes), koff);
                }
                const int t = 16 * E + l16;
                float acc = 0.f;
#pragma unroll
                for (int i = 0; i < 16; ++i) acc += drc[t * 17 + i];
                float* dst = dr_part + (size_t)(ntile * NP + pr) * nbt + row0 * H + h;
                const uint32_t dbytes = (uint32_t)((nt - 1) * H + 1) * 4;
                buf_st32(acc, make_rsrc(dst, dbytes), lane < 16 ? (uint32_t)t * H * 4 : dbytes);
            }
        };
        if (e == 0) {
            if (nt == kC)
                round_body(std::true_type{}, std::integral_constant<int, 0>{});
            else
                round_body(std::false_type{}, std::integral_constant<int, 0>{});
        } else {
            if (nt == kC)
                round_body(std::true_type{}, std::integral_constant<int, 1>{});
            else
                round_body(std::false_type{}, std::integral_constant<int, 1>{});
        }
    }
    wait_vm_all();   // the requests for the chunk before the first have landed before exit
    if (g.range_flag && !(fabsf(chk) <= 3.0e38f)) *g.range_flag = 1;
    if (g.dlam0 && e == 0 && g4 == 0) g.dlam0[(size_t)bh * DK + n0w + nl] = cT;
    if constexpr (TI) {   // part e * B + b of the token sums: the wave's four token groups added
        sum_da += __shfl_xor(sum_da, 16, 64);
        sum_da += __shfl_xor(sum_da, 32, 64);
        sum_dp += __shfl_xor(sum_dp, 16, 64);
        sum_dp += __shfl_xor(sum_dp, 32, 64);
        if (g4 == 0) {
            const size_t np = (size_t)2 * s.B * H * DK;
            const size_t o = ((size_t)(e * s.B + b) * H + h) * DK + n0w + nl;
            float* part = static_cast<float*>(g.ou_part);
            part[o] = sum_da;
            part[np + o] = sum_dp;
        }
    }
}

// dr = sum of the per-pair partials, stored in the input dtype
__global__ void dr_combine_kernel(const float* __restrict__ part, int nparts, size_t n, uint16_t* __restrict__ dr) {
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    float acc = 0.f;
    for (int t = 0; t < nparts; ++t) acc += part[(size_t)t * n + i];
    dr[i] = f32_to_bf16(acc);
}

template <int DK, int DV, bool TI, bool YG>
hipError_t launch_dk(const Shape& s, const BwdArgs& a, const float* saved_lam, const float* saved_H, float* dr_part,
                     hipStream_t st) {
    using Cfg = DkCfg<DK, DV>;
    auto kern = bwd_dk_kernel<DK, DV, TI, YG>;
    static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                                       hipFuncAttributeMaxDynamicSharedMemorySize, Cfg::BYTES);
    if (attr != hipSuccess) return attr;
    hipError_t e = launch_backward_dv(s, a, saved_lam, st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3((unsigned)(s.B * s.H * Cfg::NNT)), dim3(Cfg::NTHR), Cfg::BYTES, st, s, a,
                       saved_lam, saved_H, dr_part);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const size_t n = (size_t)s.B * s.T * s.H;
    if (n > 0) {
        hipLaunchKernelGGL(dr_combine_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, dr_part,
                           Cfg::NNT * Cfg::NP, n, static_cast<uint16_t*>(a.dr));
        e = hipGetLastError();
    }
    return e;
}

}  // namespace

bool chunked_bwd_supported(const Shape& s) { return s.bf16 && s.dk >= 32 && s.dv >= 32; }

// one part per (wave of a pair, batch row)
int chunked_ou_parts(const Shape& s) { return 2 * s.B; }

// per-pair dr partials: dk / 16 of them per token
size_t chunked_bwd_workspace(const Shape& s) { return (size_t)(s.dk / 16) * s.B * s.T * s.H * sizeof(float); }

hipError_t launch_backward_chunked(const Shape& s, const BwdArgs& a, const void* saved, void* ws, hipStream_t st) {
    const size_t nchunk = (size_t)(s.T + kC - 1) / kC;
    const float* saved_lam = static_cast<const float*>(saved);
    const float* saved_H = saved_lam + (size_t)s.B * s.H * nchunk * kLamRows * s.dk;
    float* dr_part = static_cast<float*>(ws);
#define KLA_DK_CASE(DK_, DV_)                                                    \
    if (s.dk == DK_ && s.dv == DV_) {                                            \
        if (a.dyvar)                                                             \
            return a.ou_a ? launch_dk<DK_, DV_, true, true>(s, a, saved_lam, saved_H, dr_part, st) \
                          : launch_dk<DK_, DV_, false, true>(s, a, saved_lam, saved_H, dr_part, st); \
        return a.ou_a ? launch_dk<DK_, DV_, true, false>(s, a, saved_lam, saved_H, dr_part, st)     \
                      : launch_dk<DK_, DV_, false, false>(s, a, saved_lam, saved_H, dr_part, st);    \
    }
#define KLA_DK_ROW(DK_) KLA_DK_CASE(DK_, 32) KLA_DK_CASE(DK_, 64) KLA_DK_CASE(DK_, 128)
    KLA_DK_ROW(32) KLA_DK_ROW(64) KLA_DK_ROW(128)
#undef KLA_DK_ROW
#undef KLA_DK_CASE
    return hipErrorInvalidValue;
}

}  // namespace kla
