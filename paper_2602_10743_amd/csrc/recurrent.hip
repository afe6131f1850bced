// Token-recurrent KLA kernels: forward, backward (two sweeps) and the decode step.
//
// These walk the filter one token at a time (Theorem 1 gate view for the
// precision, Theorem 2 for the information state, Algorithm 1 readout), with
// the d_k x d_v state held in registers across the token loop.  They take fp32
// inputs and the widths the chunked MFMA path does not, and implement the
// decode step.  With OU parameters (ou_a set) every token of a head shares the
// gates of its key slot; the backward then sums the gate gradients of a slot
// over its tokens into one part per batch row.  The forward can save the
// precision after every token, which the backward then reads instead of
// walking it again.
#include <type_traits>

#include "kla_buf.hpp"
#include "kla_device.hpp"
#include "kla_internal.hpp"

namespace kla {
namespace {

constexpr int kThreads = 256;
constexpr int kTB = 16;  // tokens per staged block of sweep 1
constexpr int kCKI = 64; // tokens between the information-state checkpoints of the saved context

// The saved context of this path: lam_t [B, T, H, dk], then the information state
// before every kCKI-th token [B, H, ceil(T / kCKI), dk, dv], fp32.
__host__ __device__ inline size_t saved_lam_floats(const Shape& s) { return (size_t)s.B * s.T * s.H * s.dk; }
__host__ __device__ inline int n_checkpoints(int T) { return (T + kCKI - 1) / kCKI; }

// Per-token inputs reach the kernels in blocks of ROWS tokens, staged in LDS as
// rows of floats.  A Part is one tensor's W values per token: each thread
// fetches elements tid + kThreads m of the next block into registers while the
// current block is worked on, and writes them to their LDS columns once that
// block is done, so a token's loads never wait in its recursion.  The kernels
// synchronise with barrier_lds (LDS ordering only): a full __syncthreads would
// wait for the prefetch at the first barrier after it is issued.
template <int ROWS, int W, int NT = kThreads>
struct Part {
    static constexpr int N = (ROWS * W + NT - 1) / NT;
    float x[N];
    // rows j < nt (nt >= 1): element c of row j at x0[j * ts + c].  Rows past nt and
    // elements past the block re-read the last valid element: they are never used,
    // and the loads stay unconditional, so nothing waits for them before the commit.
    template <typename T>
    __device__ __forceinline__ void fetch(const T* x0, int ts, int nt) {
#pragma unroll
        for (int m = 0; m < N; ++m) {
            const int e = min((int)threadIdx.x + NT * m, ROWS * W - 1);
            const int j = min(e / W, nt - 1), c = e % W;
            x[m] = ld(x0, (size_t)(j * ts + c));
        }
    }
    // row j of the block into dst[j * ROW + c0 + c]
    template <int ROW>
    __device__ __forceinline__ void commit(float* dst, int c0) const {
#pragma unroll
        for (int m = 0; m < N; ++m) {
            const int e = (int)threadIdx.x + NT * m;
            const int j = e / W, c = e % W;
            if (e < ROWS * W) dst[j * ROW + c0 + c] = x[m];
        }
    }
};

// Reciprocal on v_rcp_f32 (about 1 ulp), as in the chunked kernels: the IEEE division
// sequence would lengthen the per-token precision chain several times over.
__device__ __forceinline__ float rcp(float x) { return __builtin_amdgcn_rcpf(x); }

// Sum over each 16-lane row with DPP moves, held by every lane of the row.
__device__ __forceinline__ float row_sum16(float x) {
    x += dpp<0xB1, 0xf>(x);    // quad_perm [1,0,3,2]
    x += dpp<0x4E, 0xf>(x);    // quad_perm [2,3,0,1]
    x += dpp<0x141, 0xf>(x);   // row_half_mirror
    x += dpp<0x140, 0xf>(x);   // row_mirror
    return x;
}

// x of the lane D below within its 16-lane row (row_shr; lanes with none read 0)
template <int D>
__device__ __forceinline__ float row_shr(float x) {
    static_assert(D >= 1 && D <= 15, "row shift");
    return dpp<0x110 + D, 0xf>(x);
}

// Sum over groups of W consecutive lanes (W = 16 or 32), held by every lane of the
// group: W = 32 exchanges the two row sums with a swizzle (lane l reads lane l ^ 16).
template <int W>
__device__ __forceinline__ float group_sum_all(float x) {
    static_assert(W == 16 || W == 32, "group width");
    x = row_sum16(x);
    if constexpr (W == 32)
        x += __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, x), 0x401F));
    return x;
}

// value channels per forward workgroup: 16, so that even a small head spreads over
// several workgroups (each walks the precision of the head itself)
template <int DV>
constexpr int kFwdDVT = DV < 16 ? DV : 16;
// threads per forward workgroup and tokens per staged block: blocks of 32 tokens
// (half the barriers per token) where the LDS holds them, two waves per SIMD at
// dk = 64 (measured at the state-tracking shape, dk = 32: 256 threads and blocks
// of 32 tokens beat 512 threads and blocks of 16)
template <int DK>
constexpr int kFwdThreads = DK == 64 ? 512 : 256;
template <int DK>
constexpr int kFwdTB = DK <= 32 ? 32 : 16;

// ----------------------------------------------------------------------------
// Forward.  One workgroup per (b, h, value tile of DVT channels); every thread
// owns H[n, d] for n = ng + i*NG and one channel d = d0 + dl.  Per block of TBF
// tokens the precision walk is spread over all threads: GPS consecutive lanes per
// key slot, lane group g taking tokens g TPG .. g TPG + TPG - 1.  A lane composes
// the Moebius matrices of its tokens (Theorem 1 in homogeneous form:
// (x, z) -> ((1 + phi pbar) x + phi abar^2 z, pbar x + abar^2 z), lam = x / z,
// phi = k^2 r); an inclusive scan of these products over the slot's lanes (DPP,
// each product scaled by its largest entry: the map is projective) gives the
// product of every token before the lane's group, which applied to the block's
// starting lam starts the lane's own walk over its tokens.  The walk leaves F,
// r k, q / lam and q^2 / lam in the staged rows; then every thread updates its
// state entries over the block and the readout partials are summed.
template <typename S, int DK, int DV>
__global__ __launch_bounds__(kFwdThreads<DK>) void fwd_recurrent_kernel(Shape s, FwdArgs g, float* saved_lam) {
    using T_ = typename storage<S>::type;
    constexpr int NTH = kFwdThreads<DK>;
    constexpr int TBF = kFwdTB<DK>;   // tokens per staged block
    constexpr int DVT = kFwdDVT<DV>;
    constexpr int NTILE = DV / DVT;
    constexpr int NG = NTH / DVT;
    constexpr int NPER = DK / NG > 0 ? DK / NG : 1;
    static_assert(DK % NG == 0 || NG > DK, "key width must be a multiple of the n-groups");
    // staged row of a token: abar, pbar, k, q [DK] each, this tile's v [DVT], r
    constexpr int CA = 0, CP = DK, CK = 2 * DK, CQ = 3 * DK, CV = 4 * DK, CR = CV + DVT, ROW = CR + 1;
    constexpr int NY = (TBF * DVT + NTH - 1) / NTH;   // outputs per thread and block
    constexpr int GPS = NTH / DK, TPG = TBF / GPS;       // walk lanes per key slot, tokens per lane
    static_assert(GPS * DK == NTH && TPG * GPS == TBF && GPS <= 16 && (GPS & (GPS - 1)) == 0,
                  "the walk lanes of a slot split the block evenly within a DPP row");

    __shared__ float sIn[TBF * ROW];
    __shared__ float sRed[TBF][NG][DVT];

    const T_* q = static_cast<const T_*>(g.q);
    const T_* k = static_cast<const T_*>(g.k);
    const T_* v = static_cast<const T_*>(g.v);
    const T_* a = static_cast<const T_*>(g.a);
    const T_* p = static_cast<const T_*>(g.p);
    const T_* r = static_cast<const T_*>(g.r);
    T_* y = static_cast<T_*>(g.y);

    const int tile = blockIdx.x % NTILE;
    const int bh = blockIdx.x / NTILE;
    const int b = bh / s.H, h = bh % s.H;
    const int tid = threadIdx.x;
    const int dl = tid % DVT, ng = tid / DVT;
    const int d = tile * DVT + dl;
    const bool owns = ng < DK;  // with NG > DK some n-groups are idle
    const size_t row0 = (size_t)b * s.T;

    float Hs[NPER];
#pragma unroll
    for (int i = 0; i < NPER; ++i) {
        int n = ng + i * NG;
        Hs[i] = (owns && g.eta0) ? g.eta0[((size_t)bh * DK + n) * DV + d] : 0.f;
    }
    const int wn = tid / GPS, wg = tid % GPS;   // walk: key slot and token group of this lane
    float lam = g.lam0 ? g.lam0[(size_t)bh * DK + wn] : 1.f;   // lam before the block, in every lane of slot wn
    const bool ou = g.ou_a != nullptr;
    float oa = 0.f, op = 0.f;
    if (ou) ou_gates(g.ou_a[h * DK + wn], g.ou_p[h * DK + wn], g.ou_d[h * DK + wn], oa, op);

    Part<TBF, DK, NTH> xa, xp, xk, xq;
    Part<TBF, DVT, NTH> xv;
    Part<TBF, 1, NTH> xr;
    // with OU gates the abar / pbar columns are filled from k and not used
    const T_* ga = ou ? k : a;
    const T_* gp = ou ? k : p;
    auto fetch = [&](int t) {
        const int nt = min(TBF, s.T - t);
        const size_t o = (row0 + t) * s.H + h;
        xa.fetch(ga + o * DK, s.H * DK, nt);
        xp.fetch(gp + o * DK, s.H * DK, nt);
        xk.fetch(k + o * DK, s.H * DK, nt);
        xq.fetch(q + o * DK, s.H * DK, nt);
        xv.fetch(v + o * DV + tile * DVT, s.H * DV, nt);
        xr.fetch(r + o, s.H, nt);
    };
    auto commit = [&]() {
        wait_vm_all();   // the prefetch has landed (and stores issued before it are done)
        xa.template commit<ROW>(sIn, CA);
        xp.template commit<ROW>(sIn, CP);
        xk.template commit<ROW>(sIn, CK);
        xq.template commit<ROW>(sIn, CQ);
        xv.template commit<ROW>(sIn, CV);
        xr.template commit<ROW>(sIn, CR);
    };

    // Block blk is worked on from LDS while block blk + 1 is in registers; after its
    // outputs are formed, block blk + 1 goes to LDS, the outputs are stored and block
    // blk + 2 is fetched, a whole block ahead of its commit.  Fetches past the end fetch
    // the last block again (unused), so they stay unconditional.
    const int nblk = (s.T + TBF - 1) / TBF;
    wait_vm_all();   // the initial state is in: no first-use wait inside the loop
    if (nblk > 0) {
        fetch(0);
        commit();
        fetch(min(1, nblk - 1) * TBF);
    }
    barrier_lds();
    static_assert(kCKI % TBF == 0, "checkpoints fall on block starts");
    float* saved_H = saved_lam ? saved_lam + saved_lam_floats(s) : nullptr;
    const int nck = n_checkpoints(s.T);
    for (int blk = 0; blk < nblk; ++blk) {
        const int t0 = blk * TBF, nt = min(TBF, s.T - t0);
        if (saved_H && t0 % kCKI == 0 && owns) {   // the state before token t0
#pragma unroll
            for (int i = 0; i < NPER; ++i)
                saved_H[(((size_t)bh * nck + t0 / kCKI) * DK + ng + i * NG) * DV + d] = Hs[i];
        }
        float lsv[TPG];   // lam after each of this lane's tokens (the saved context)
        // Token loops carry no branch: rows past nt (the ragged last block) are worked on
        // as well, from the repeated last row, and only selects keep them out of the state.
        {
            float ta[TPG], tp[TPG], tk[TPG], tq[TPG], tr[TPG];
#pragma unroll
            for (int u = 0; u < TPG; ++u) {
                const float* row = sIn + (wg * TPG + u) * ROW;
                const float ra = row[CA + wn], rp = row[CP + wn];
                ta[u] = ou ? oa : ra;
                tp[u] = ou ? op : rp;
                tk[u] = row[CK + wn];
                tq[u] = row[CQ + wn];
                tr[u] = row[CR];
            }
            // this lane's product M_last ... M_first (tokens past nt: identity), scaled
            float m00 = 1.f, m01 = 0.f, m10 = 0.f, m11 = 1.f;
#pragma unroll
            for (int u = 0; u < TPG; ++u) {
                const float a2 = ta[u] * ta[u], phi = tk[u] * tk[u] * tr[u];
                const float z0 = fmaf(tp[u], m00, a2 * m10), z1 = fmaf(tp[u], m01, a2 * m11);
                const bool ok = wg * TPG + u < nt;
                m00 = ok ? fmaf(phi, z0, m00) : m00;
                m01 = ok ? fmaf(phi, z1, m01) : m01;
                m10 = ok ? z0 : m10;
                m11 = ok ? z1 : m11;
            }
            {
                const float sc = rcp(fmaxf(fmaxf(m00, m01), fmaxf(m10, m11)));
                m00 *= sc; m01 *= sc; m10 *= sc; m11 *= sc;
            }
            // inclusive scan over the slot's lanes: P_g = M_g ... M_0
            auto scan_step = [&](auto dd) {
                constexpr int D = decltype(dd)::value;
                if constexpr (D < GPS) {
                    const float b00 = row_shr<D>(m00), b01 = row_shr<D>(m01);
                    const float b10 = row_shr<D>(m10), b11 = row_shr<D>(m11);
                    const float c00 = fmaf(m00, b00, m01 * b10), c01 = fmaf(m00, b01, m01 * b11);
                    const float c10 = fmaf(m10, b00, m11 * b10), c11 = fmaf(m10, b01, m11 * b11);
                    const float sc = rcp(fmaxf(fmaxf(c00, c01), fmaxf(c10, c11)));
                    const bool take = wg >= D;
                    m00 = take ? c00 * sc : m00;
                    m01 = take ? c01 * sc : m01;
                    m10 = take ? c10 * sc : m10;
                    m11 = take ? c11 * sc : m11;
                }
            };
            scan_step(std::integral_constant<int, 1>{});
            scan_step(std::integral_constant<int, 2>{});
            scan_step(std::integral_constant<int, 4>{});
            scan_step(std::integral_constant<int, 8>{});
            // the product of the groups before this one (identity for group 0) applied to lam
            const float e00 = row_shr<1>(m00), e01 = row_shr<1>(m01);
            const float e10 = row_shr<1>(m10), e11 = row_shr<1>(m11);
            float lw = lam;
            if (wg > 0) lw = fmaf(e00, lam, e01) * rcp(fmaf(e10, lam, e11));
            // walk this lane's tokens
#pragma unroll
            for (int u = 0; u < TPG; ++u) {
                const int j = wg * TPG + u;
                float* row = sIn + j * ROW;
                const float rho = rcp(ta[u] * ta[u] + tp[u] * lw);
                const float ln = rho * lw + tk[u] * tk[u] * tr[u];
                lw = j < nt ? ln : lw;
                lsv[u] = ln;
                const float inv = rcp(ln);
                row[CA + wn] = ta[u] * rho;
                row[CP + wn] = tr[u] * tk[u];
                row[CK + wn] = tq[u] * inv;
                row[CQ + wn] = tq[u] * tq[u] * inv;
            }
            // lam after the block: the last group's, in every lane of the slot
            lam = __shfl(lw, (tid & 63 & ~(GPS - 1)) + GPS - 1, 64);
        }
        barrier_lds();
#pragma unroll
        for (int j = 0; j < TBF; ++j) {
            const float* row = sIn + j * ROW;
            const float vd = row[CV + dl];
            float acc = 0.f;
#pragma unroll
            for (int i = 0; i < NPER; ++i) {
                const int n = ng + i * NG;
                if (NG <= DK || owns) {
                    const float hn = row[CA + n] * Hs[i] + row[CP + n] * vd;
                    Hs[i] = j < nt ? hn : Hs[i];
                    acc += row[CK + n] * hn;
                }
            }
            sRed[j][ng][dl] = acc;
        }
        barrier_lds();
        // the block's outputs are formed in registers and stored after the commit, whose wait
        // then covers the prefetch only
        float yo[NY], yvo = 0.f;
#pragma unroll
        for (int u = 0; u < NY; ++u) {
            const int idx = tid + NTH * u, j = idx / DVT, dd = idx % DVT;
            float acc = 0.f;
            if (j < nt) {
#pragma unroll
                for (int gi = 0; gi < NG; ++gi) acc += sRed[j][gi][dd];
            }
            yo[u] = acc;
        }
        const int jv = tid - (NTH - TBF);   // the token whose readout variance this thread sums
        const bool wv = tile == 0 && g.yvar && jv >= 0 && jv < nt;
        if (wv) {
#pragma unroll
            for (int n = 0; n < DK; ++n) yvo += sIn[jv * ROW + CQ + n];
        }
        barrier_lds();
        commit();
#pragma unroll
        for (int u = 0; u < NY; ++u) {
            const int idx = tid + NTH * u, j = idx / DVT, dd = idx % DVT;
            if (j < nt) st(y, ((row0 + t0 + j) * s.H + h) * DV + tile * DVT + dd, yo[u]);
        }
        if (wv) g.yvar[(row0 + t0 + jv) * s.H + h] = yvo;
        if (saved_lam && tile == 0) {
#pragma unroll
            for (int u = 0; u < TPG; ++u) {
                const int j = wg * TPG + u;
                if (j < nt) saved_lam[((row0 + t0 + j) * s.H + h) * DK + wn] = lsv[u];
            }
        }
        fetch(min(blk + 2, nblk - 1) * TBF);
        barrier_lds();
    }
    wait_vm_all();   // the last (unused) prefetch has landed before the registers are released
    if (tile == 0 && g.lamT && wg == 0) g.lamT[(size_t)bh * DK + wn] = lam;
    if (g.etaT && owns) {
#pragma unroll
        for (int i = 0; i < NPER; ++i) g.etaT[((size_t)bh * DK + ng + i * NG) * DV + d] = Hs[i];
    }
}

// ----------------------------------------------------------------------------
// Backward, sweep 1 (forward in time).  From the saved context of the forward
// (lam_t after every token, the information state every kCKI tokens), re-runs the
// information state and stores dqt_t = H_t dy_t (the gradient of the effective
// query q/lam_t), plus PT[n] = sum_d detaT[n,d] H_T[n,d].  One workgroup per
// (b, h, 16 key slots, kCKI-token segment), started from the segment's
// checkpoint; 16 lanes split the value channels.  Every token's gates follow
// from the saved lam_{t-1}, for all (token, slot) pairs of a block in one
// parallel phase.
template <typename S, int DK, int DV>
__global__ __launch_bounds__(kThreads) void bwd_sweep1_kernel(Shape s, BwdArgs g, const float* slam, float* wdqt,
                                                               float* wPT) {
    using T_ = typename storage<S>::type;
    constexpr int NT = 16, DL = 16, DPER = DV / DL;
    static_assert(DL == kTB, "lane j of a slot's row holds token j of the block");
    static_assert(kThreads == kTB * NT, "one (token, slot) gate per thread");
    // staged row of a token: abar, pbar, k, saved lam of this workgroup's NT key slots, v [DV], dy [DV], r
    constexpr int CA = 0, CP = NT, CK = 2 * NT, CL = 3 * NT, CV = 4 * NT, CD = CV + DV, CR = CD + DV;
    constexpr int ROW = CR + 1;
    __shared__ float sIn[kTB * ROW];
    __shared__ float sLP[NT];          // lam of the token before the block
    __shared__ float2 sFK[kTB][NT];    // F and r k of every (token, slot) of the block

    const T_* k = static_cast<const T_*>(g.k);
    const T_* v = static_cast<const T_*>(g.v);
    const T_* a = static_cast<const T_*>(g.a);
    const T_* p = static_cast<const T_*>(g.p);
    const T_* r = static_cast<const T_*>(g.r);
    const T_* dy = static_cast<const T_*>(g.dy);

    const int ntile = DK / NT, nck = n_checkpoints(s.T);
    const int seg = blockIdx.x % nck, bt = blockIdx.x / nck;
    const int bh = bt / ntile, ktile = bt % ntile;
    const int b = bh / s.H, h = bh % s.H;
    const int tid = threadIdx.x;
    const int nl = tid / DL, n = ktile * NT + nl, dl = tid % DL;
    const size_t row0 = (size_t)b * s.T;
    const int ts0 = seg * kCKI, tend = min(ts0 + kCKI, s.T);   // this workgroup's tokens
    const float* ckH = slam + saved_lam_floats(s);

    float Hs[DPER];
#pragma unroll
    for (int i = 0; i < DPER; ++i) Hs[i] = ckH[(((size_t)bh * nck + seg) * DK + n) * DV + dl + i * DL];
    // the gate phase's (token, slot) pair of this thread
    const int gsl = tid % NT, gj = tid / NT;
    const bool ou = g.ou_a != nullptr;
    float goa = 0.f, gop = 0.f;
    if (ou) {
        const int gn = ktile * NT + gsl;
        ou_gates(g.ou_a[h * DK + gn], g.ou_p[h * DK + gn], g.ou_d[h * DK + gn], goa, gop);
    }

    Part<kTB, NT> xa, xp, xk, xl;
    Part<kTB, DV> xv, xdy;
    Part<kTB, 1> xr;
    Part<1, NT> xlp;
    // with OU gates the abar / pbar columns are filled from k and not used; with no initial
    // precision, token 0's lam_{t-1} is read from the saved lam and replaced by 1
    const T_* ga = ou ? k : a;
    const T_* gp = ou ? k : p;
    const bool lam0_one = g.lam0 == nullptr;
    auto fetch = [&](int t) {
        const int nt = min(kTB, tend - t);
        const size_t o = (row0 + t) * s.H + h;
        xa.fetch(ga + o * DK + ktile * NT, s.H * DK, nt);
        xp.fetch(gp + o * DK + ktile * NT, s.H * DK, nt);
        xk.fetch(k + o * DK + ktile * NT, s.H * DK, nt);
        xl.fetch(slam + o * DK + ktile * NT, s.H * DK, nt);
        xv.fetch(v + o * DV, s.H * DV, nt);
        xdy.fetch(dy + o * DV, s.H * DV, nt);
        xr.fetch(r + o, s.H, nt);
        const float* lp0 = t > 0 ? slam + (o - s.H) * DK : (lam0_one ? slam + o * DK : g.lam0 + (size_t)bh * DK);
        xlp.fetch(lp0 + ktile * NT, 0, 1);
    };
    auto commit = [&]() {
        wait_vm_all();   // the prefetch has landed (and stores issued before it are done)
        xa.template commit<ROW>(sIn, CA);
        xp.template commit<ROW>(sIn, CP);
        xk.template commit<ROW>(sIn, CK);
        xl.template commit<ROW>(sIn, CL);
        xv.template commit<ROW>(sIn, CV);
        xdy.template commit<ROW>(sIn, CD);
        xr.template commit<ROW>(sIn, CR);
        xlp.template commit<NT>(sLP, 0);
    };

    // blocks staged as in the forward: blk from LDS, blk + 1 in registers
    const int nblk = (tend - ts0 + kTB - 1) / kTB;
    wait_vm_all();   // the initial state is in: no first-use wait inside the loop
    if (nblk > 0) {
        fetch(ts0);
        commit();
        fetch(ts0 + min(1, nblk - 1) * kTB);
    }
    barrier_lds();
    for (int blk = 0; blk < nblk; ++blk) {
        const int t0 = ts0 + blk * kTB, nt = min(kTB, tend - t0);
        {   // the gates of every (token, slot) from the saved lam_{t-1}, in parallel
            const float* row = sIn + gj * ROW;
            const float ra = row[CA + gsl], rp = row[CP + gsl];
            const float at = ou ? goa : ra, pt = ou ? gop : rp;
            const float lp = gj > 0 ? row[CL + gsl - ROW] : (t0 == 0 && lam0_one ? 1.f : sLP[gsl]);
            const float rho = rcp(at * at + pt * lp);
            sFK[gj][gsl] = make_float2(at * rho, row[CR] * row[CK + gsl]);
        }
        barrier_lds();
        float odqt = 0.f;
#pragma unroll
        for (int j = 0; j < kTB; ++j) {   // no branch: rows past nt only reach selects
            const bool live = j < nt;
            const float* row = sIn + j * ROW;
            const float2 fk = sFK[j][nl];   // F, r k
            float acc = 0.f;
#pragma unroll
            for (int i = 0; i < DPER; ++i) {
                const float hn = fk.x * Hs[i] + fk.y * row[CV + dl + i * DL];
                Hs[i] = live ? hn : Hs[i];
                acc += hn * row[CD + dl + i * DL];
            }
            acc = row_sum16(acc);
            if (dl == j) odqt = acc;   // lane j of the slot's row keeps token j's result
        }
        barrier_lds();
        commit();
        if (dl < nt) wdqt[((row0 + t0 + dl) * s.H + h) * DK + n] = odqt;
        fetch(ts0 + min(blk + 2, nblk - 1) * kTB);
        barrier_lds();
    }
    wait_vm_all();   // the last (unused) prefetch has landed before the registers are released
    if (seg != nck - 1) return;   // the last segment ends at the final state
    float acc = 0.f;
    if (g.detaT) {
#pragma unroll
        for (int i = 0; i < DPER; ++i) acc += g.detaT[((size_t)bh * DK + n) * DV + dl + i * DL] * Hs[i];
    }
    acc = row_sum16(acc);
    if (dl == 0) wPT[(size_t)bh * DK + n] = acc;
}

// ----------------------------------------------------------------------------
// Backward, sweep 2 (reverse in time), one workgroup per (b, h) holding the
// whole adjoint state dH.  Per token, with dG_t the adjoint of log F_t and
// g_t the adjoint of lam_t:
//   dH_t   = F_{t+1} dH_{t+1} + qt_t dy_t^T          (dH_T starts at detaT)
//   dkh_t  = dH_t v_t,  dv_t = dH_t^T kh_t
//   dG_t   = PT + sum_{s>=t} (qt_s dqt_s - kh_s dkh_s)
//   g_t    = c_t - q_t (dqt_t + q_t gv_t) / lam_t^2,  c_T = dlamT,
//            (gv_t: upstream gradient of the readout variance, zero if none)
//   c_{t-1}= abar_t^2 rho_t^2 g_t - pbar_t rho_t dG_t
// and the input gradients follow by the chain rule through rho, lam and F.
// Per block of TB tokens (latest block first):
//   A  every (token, slot): rho, F, qt, kh and the coefficients of the c/g/dG
//      recursion, in parallel;
//   B  every thread: its dH entries over the block's tokens (latest first),
//      with the dkh sums (DPP) and dv partials per token;
//   C  one lane per slot: the dG / g / c recursion over the block;
//   D  every (token, slot): dq, dk, dabar, dpbar and the dr terms; dv sums;
//   E  dr sums, and the next block's inputs go to LDS.
template <int DK, int DV, int NTH_>
struct Sweep2Lay {
    static constexpr int NTH = NTH_;
    static constexpr int DVT = DV < 32 ? DV : 32, NG = NTH / DVT;
    static constexpr int NPER = DK / NG > 0 ? DK / NG : 1, DPER = DV / DVT;
    // staged row of token t: lam_t, dqt_t, q, k, abar, pbar [DK] each; v, dy [DV]; r; the
    // upstream gradient of the readout variance
    static constexpr int CL = 0, CDQ = DK, CQ = 2 * DK, CK = 3 * DK, CA = 4 * DK, CP = 5 * DK;
    static constexpr int CV = 6 * DK, CD = CV + DV, CR = CD + DV, CG = CR + 1, ROW = CG + 1;
    static constexpr int TB = ROW * 16 * 4 <= 48 * 1024 ? 16 : 8;
    // LDS, in floats: staged rows, then lam of the token before the block; {F_{t+1}, qt, kh,
    // rho} and {(abar rho)^2, pbar rho, q (dqt + q gv) / lam^2, qt dqt} per (token, slot);
    // dkh; dv partials per n-group; {dG, g} per (token, slot); dr terms; the carried forget
    // gate (two buffers); per-thread OU sums
    static constexpr int L_LP = TB * ROW, L_C0 = (L_LP + DK + 3) / 4 * 4, L_C1 = L_C0 + 4 * TB * DK;
    static constexpr int L_PK = L_C1 + 4 * TB * DK, L_PV = L_PK + TB * DK, L_SG = L_PV + TB * NG * DV;
    static constexpr int L_DR = L_SG + 2 * TB * DK, L_FC = L_DR + TB * DK, L_OU = L_FC + 2 * DK;
    static constexpr size_t BYTES = (size_t)(L_OU + 2 * NTH) * sizeof(float);
    static constexpr bool fits = NG <= DK && DK % NG == 0 && (TB * DK) % NTH == 0 && BYTES <= 160 * 1024;
};

// 512 threads (two waves per SIMD, half the dH entries per thread) for heads of up to
// 64 x 64 where the shape splits evenly over them and the LDS fits, else 256
template <int DK, int DV>
struct Sweep2Cfg : Sweep2Lay<DK, DV, (DK * DV <= 64 * 64 && Sweep2Lay<DK, DV, 512>::fits) ? 512 : 256> {
    static_assert(Sweep2Lay<DK, DV, Sweep2Cfg::NTH>::fits, "every thread owns dH entries; LDS budget");
};

template <typename S, int DK, int DV>
__global__ __launch_bounds__((Sweep2Cfg<DK, DV>::NTH)) void bwd_sweep2_kernel(Shape s, BwdArgs g, const float* wlam,
                                                               const float* wdqt, const float* wPT) {
    using T_ = typename storage<S>::type;
    using C = Sweep2Cfg<DK, DV>;
    constexpr int DVT = C::DVT, NG = C::NG, NPER = C::NPER, DPER = C::DPER, TB = C::TB, ROW = C::ROW;
    constexpr int NTH = C::NTH;
    constexpr int ND = TB * DK / NTH, NDV = (TB * DV + NTH - 1) / NTH;   // items per thread
    static_assert(ND * NTH == TB * DK, "(token, slot) items split evenly over the threads");
    extern __shared__ __align__(16) float sm[];
    float* sIn = sm;
    float* sLP = sm + C::L_LP;    // [DK]
    float* sC0 = sm + C::L_C0;    // [TB][DK][4]
    float* sC1 = sm + C::L_C1;    // [TB][DK][4]
    float* sPK = sm + C::L_PK;    // [TB][DK]
    float* sPV = sm + C::L_PV;    // [TB][NG][DV]
    float* sSG = sm + C::L_SG;    // [TB][DK][2]
    float* sDR = sm + C::L_DR;    // [TB][DK]
    float* sFC = sm + C::L_FC;    // [2][DK]
    float* sOU = sm + C::L_OU;    // [2][NTH]

    const T_* q = static_cast<const T_*>(g.q);
    const T_* k = static_cast<const T_*>(g.k);
    const T_* v = static_cast<const T_*>(g.v);
    const T_* a = static_cast<const T_*>(g.a);
    const T_* p = static_cast<const T_*>(g.p);
    const T_* r = static_cast<const T_*>(g.r);
    const T_* dy = static_cast<const T_*>(g.dy);
    T_* dq = static_cast<T_*>(g.dq);
    T_* dk = static_cast<T_*>(g.dk);
    T_* dv = static_cast<T_*>(g.dv);
    T_* da = static_cast<T_*>(g.da);
    T_* dp = static_cast<T_*>(g.dp);
    T_* dr = static_cast<T_*>(g.dr);

    const int bh = blockIdx.x;
    const int b = bh / s.H, h = bh % s.H;
    const int tid = threadIdx.x;
    const int dl = tid % DVT, ng = tid / DVT;
    const int nme = tid % DK;   // the key slot of this thread's (token, slot) items
    const size_t row0 = (size_t)b * s.T;

    float dH[NPER][DPER];
#pragma unroll
    for (int i = 0; i < NPER; ++i)
#pragma unroll
        for (int j = 0; j < DPER; ++j)
            dH[i][j] = g.detaT ? g.detaT[((size_t)bh * DK + ng + i * NG) * DV + dl + j * DVT] : 0.f;

    // the dG / c recursion lives in threads tid < DK
    float cnext = 0.f, Sg = 0.f;
    if (tid < DK) {
        cnext = g.dlamT ? g.dlamT[(size_t)bh * DK + tid] : 0.f;
        Sg = wPT[(size_t)bh * DK + tid];
        sFC[DK + tid] = 1.f;   // no forget gate after the last token
    }
    const bool ou = g.ou_a != nullptr;
    float oa = 0.f, op = 0.f, sum_da = 0.f, sum_dp = 0.f;
    if (ou) ou_gates(g.ou_a[h * DK + nme], g.ou_p[h * DK + nme], g.ou_d[h * DK + nme], oa, op);

    Part<TB, DK, NTH> xl, xdq, xq, xk, xa, xp;
    Part<TB, DV, NTH> xv, xdy;
    Part<TB, 1, NTH> xr, xg;
    Part<1, DK, NTH> xlp;
    // Loads stay unconditional: absent tensors are replaced by present ones whose values
    // are not used (OU gates: abar / pbar columns from k; no readout-variance gradient:
    // its column from lam, scaled by zero; no initial precision: token 0's lam_{t-1}
    // from lam_0, replaced by 1 where it is read).
    const T_* ga = ou ? k : a;
    const T_* gp = ou ? k : p;
    const float* gvar = g.dyvar ? g.dyvar : wlam;
    const float gscale = g.dyvar ? 1.f : 0.f;
    const float* glam0 = g.lam0 ? g.lam0 + (size_t)bh * DK : wlam + (row0 * s.H + h) * DK;
    const bool lam0_one = g.lam0 == nullptr;
    auto fetch = [&](int t) {
        const int nt = min(TB, s.T - t);
        const size_t o = (row0 + t) * s.H + h;
        const int ts = s.H * DK;
        xl.fetch(wlam + o * DK, ts, nt);
        xdq.fetch(wdqt + o * DK, ts, nt);
        xq.fetch(q + o * DK, ts, nt);
        xk.fetch(k + o * DK, ts, nt);
        xa.fetch(ga + o * DK, ts, nt);
        xp.fetch(gp + o * DK, ts, nt);
        xv.fetch(v + o * DV, s.H * DV, nt);
        xdy.fetch(dy + o * DV, s.H * DV, nt);
        xr.fetch(r + o, s.H, nt);
        xg.fetch(gvar + (g.dyvar ? o : o * DK), g.dyvar ? s.H : ts, nt);
        xlp.fetch(t > 0 ? wlam + (o - s.H) * DK : glam0, 0, 1);
    };
    auto commit = [&]() {
        wait_vm_all();   // the prefetch has landed (and stores issued before it are done)
        xl.template commit<ROW>(sIn, C::CL);
        xdq.template commit<ROW>(sIn, C::CDQ);
        xq.template commit<ROW>(sIn, C::CQ);
        xk.template commit<ROW>(sIn, C::CK);
        xa.template commit<ROW>(sIn, C::CA);
        xp.template commit<ROW>(sIn, C::CP);
        xv.template commit<ROW>(sIn, C::CV);
        xdy.template commit<ROW>(sIn, C::CD);
        xr.template commit<ROW>(sIn, C::CR);
        xg.template commit<ROW>(sIn, C::CG);
        xlp.template commit<DK>(sLP, 0);
    };

    // blocks staged as in the forward, latest first: blk from LDS, blk - 1 in registers
    const int nblk = (s.T + TB - 1) / TB;
    wait_vm_all();   // the initial state is in: no first-use wait inside the loop
    if (nblk > 0) {
        fetch((nblk - 1) * TB);
        commit();
        fetch(max(nblk - 2, 0) * TB);
    }
    int cur = 1;   // sFC buffer holding F of the token after the current block
    barrier_lds();
    for (int blk = nblk - 1; blk >= 0; --blk) {
        const int t0 = blk * TB, nt = min(TB, s.T - t0);
        // ---- A
        for (int idx = tid; idx < TB * DK; idx += NTH) {
            const int j = idx / DK, n = idx % DK;
            if (j < nt) {
                const float* row = sIn + j * ROW;
                const float lam = row[C::CL + n];
                const float lp = j > 0 ? row[C::CL + n - ROW] : (t0 == 0 && lam0_one ? 1.f : sLP[n]);
                const float dqt = row[C::CDQ + n], qv = row[C::CQ + n], kv = row[C::CK + n];
                const float ra = row[C::CA + n], rp = row[C::CP + n];
                const float at = ou ? oa : ra, pt = ou ? op : rp;
                const float rt = row[C::CR], gv = gscale * row[C::CG];
                const float rho = rcp(at * at + pt * lp);
                const float il = rcp(lam), qtl = qv * il, F = at * rho;
                float* c0 = sC0 + 4 * (j * DK + n);
                c0[1] = qtl;
                c0[2] = rt * kv;
                c0[3] = rho;
                if (j > 0) sC0[4 * ((j - 1) * DK + n)] = F;
                else sFC[(cur ^ 1) * DK + n] = F;
                if (j == nt - 1) c0[0] = sFC[cur * DK + n];
                *reinterpret_cast<float4*>(sC1 + 4 * (j * DK + n)) =
                    make_float4(F * F, pt * rho, qv * (dqt + qv * gv) * il * il, qtl * dqt);
            }
        }
        barrier_lds();
        // ---- B
        // tokens latest first, in runs of UB unrolled tokens: the whole block for small heads,
        // shorter runs where a thread holds many dH entries (keeps the loads in registers)
        constexpr int UB = NPER * DPER <= 2 ? TB : NPER * DPER <= 4 ? 8 : NPER * DPER <= 16 ? 4 : 2;
        static_assert(TB % UB == 0, "runs split the block");
#pragma unroll 1
        for (int jb = TB - UB; jb >= 0; jb -= UB)
#pragma unroll
        for (int jj = UB - 1; jj >= 0; --jj) {   // no branch: rows past nt only reach selects
            const int j = jb + jj;
            const bool live = j < nt;
            const float* row = sIn + j * ROW;
            float dyd[DPER], vd[DPER], pv[DPER];
#pragma unroll
            for (int jd = 0; jd < DPER; ++jd) {
                dyd[jd] = row[C::CD + dl + jd * DVT];
                vd[jd] = row[C::CV + dl + jd * DVT];
                pv[jd] = 0.f;
            }
#pragma unroll
            for (int i = 0; i < NPER; ++i) {
                const int n = ng + i * NG;
                const float4 co = *reinterpret_cast<const float4*>(sC0 + 4 * (j * DK + n));
                float pk = 0.f;
#pragma unroll
                for (int jd = 0; jd < DPER; ++jd) {
                    const float hn = co.x * dH[i][jd] + co.y * dyd[jd];
                    dH[i][jd] = live ? hn : dH[i][jd];
                    pk += hn * vd[jd];
                    pv[jd] += hn * co.z;
                }
                sPK[j * DK + n] = group_sum_all<DVT>(pk);   // the same value from every lane of the group
            }
#pragma unroll
            for (int jd = 0; jd < DPER; ++jd) sPV[(j * NG + ng) * DV + dl + jd * DVT] = pv[jd];
        }
        barrier_lds();
        // ---- C
        if (tid < DK) {
#pragma unroll
            for (int j = TB - 1; j >= 0; --j) {   // no branch: rows past nt only reach selects
                const bool live = j < nt;
                const float kh = sC0[4 * (j * DK + tid) + 2];
                const float4 c1 = *reinterpret_cast<const float4*>(sC1 + 4 * (j * DK + tid));
                const float dkh = sPK[j * DK + tid];
                const float sg = Sg + (c1.w - kh * dkh);   // dG_t
                const float gl = cnext - c1.z;              // g_t
                *reinterpret_cast<float2*>(sSG + 2 * (j * DK + tid)) = make_float2(sg, gl);
                Sg = live ? sg : Sg;
                cnext = live ? c1.x * gl - c1.y * sg : cnext;
            }
        }
        barrier_lds();
        // ---- D (results in registers: they are stored after the commit, whose wait then
        // covers the prefetch only)
        float o_dq[ND], o_dk[ND], o_da[ND], o_dp[ND], o_dv[NDV];
#pragma unroll
        for (int u = 0; u < ND; ++u) {
            const int idx = tid + NTH * u, j = idx / DK, n = idx % DK;
            const float* row = sIn + j * ROW;
            const float lam = row[C::CL + n];
            const float lp = j > 0 ? row[C::CL + n - ROW] : (t0 == 0 && lam0_one ? 1.f : sLP[n]);
            const float dqt = row[C::CDQ + n], qv = row[C::CQ + n], kv = row[C::CK + n];
            const float ra = row[C::CA + n], rp = row[C::CP + n];
            const float at = ou ? oa : ra, pt = ou ? op : rp;
            const float rt = row[C::CR], gv = gscale * row[C::CG];
            const float rho = sC0[4 * (j * DK + n) + 3];
            const float dkh = sPK[j * DK + n];
            const float2 sg = *reinterpret_cast<const float2*>(sSG + 2 * (j * DK + n));
            const float qg = qv * gv;
            const float drho = sg.y * lp + sg.x * (at * at + pt * lp);
            o_dq[u] = (dqt + 2.f * qg) * rcp(lam);
            o_dk[u] = rt * dkh + 2.f * kv * rt * sg.y;
            o_da[u] = sg.x * rcp(at) - 2.f * at * rho * rho * drho;
            o_dp[u] = -lp * rho * rho * drho;
            if (j < nt) {
                if (ou) {
                    sum_da += o_da[u];
                    sum_dp += o_dp[u];
                }
                sDR[j * DK + n] = kv * dkh + kv * kv * sg.y;
            }
        }
#pragma unroll
        for (int u = 0; u < NDV; ++u) {
            const int idx = tid + NTH * u, j = idx / DV, dd = idx % DV;
            float acc = 0.f;
            if (j < nt) {
#pragma unroll
                for (int gi = 0; gi < NG; ++gi) acc += sPV[(j * NG + gi) * DV + dd];
            }
            o_dv[u] = acc;
        }
        barrier_lds();
        // ---- E
        commit();
#pragma unroll
        for (int u = 0; u < ND; ++u) {
            const int idx = tid + NTH * u, j = idx / DK, n = idx % DK;
            if (j < nt) {
                const size_t o = ((row0 + t0 + j) * s.H + h) * DK + n;
                st(dq, o, o_dq[u]);
                st(dk, o, o_dk[u]);
                if (!ou) {
                    st(da, o, o_da[u]);
                    st(dp, o, o_dp[u]);
                }
            }
        }
#pragma unroll
        for (int u = 0; u < NDV; ++u) {
            const int idx = tid + NTH * u, j = idx / DV, dd = idx % DV;
            if (j < nt && idx < TB * DV) st(dv, ((row0 + t0 + j) * s.H + h) * DV + dd, o_dv[u]);
        }
        if (tid < nt) {
            float acc = 0.f;
#pragma unroll
            for (int n = 0; n < DK; ++n) acc += sDR[tid * DK + n];
            st(dr, (row0 + t0 + tid) * s.H + h, acc);
        }
        fetch(max(blk - 2, 0) * TB);
        cur ^= 1;
        barrier_lds();
    }
    wait_vm_all();   // the last (unused) prefetch has landed before the registers are released
    if (tid < DK && g.dlam0) g.dlam0[(size_t)bh * DK + tid] = cnext;
    if (ou) {   // part b of the token sums: the threads of one slot are combined in order
        sOU[tid] = sum_da;
        sOU[NTH + tid] = sum_dp;
        barrier_lds();
        if (tid < DK) {
            float sa = 0.f, sp = 0.f;
            for (int i = tid; i < NTH; i += DK) {
                sa += sOU[i];
                sp += sOU[NTH + i];
            }
            const size_t np = (size_t)s.B * s.H * DK;
            g.ou_part[(size_t)bh * DK + tid] = sa;
            g.ou_part[np + (size_t)bh * DK + tid] = sp;
        }
    }
    if (g.deta0) {   // sFC[cur] holds F of token 0
#pragma unroll
        for (int i = 0; i < NPER; ++i)
#pragma unroll
            for (int j = 0; j < DPER; ++j) {
                const int n = ng + i * NG;
                g.deta0[((size_t)bh * DK + n) * DV + dl + j * DVT] = sFC[cur * DK + n] * dH[i][j];
            }
    }
}

// ----------------------------------------------------------------------------
// Decode: one token for S sequences, belief updated in place.  One workgroup
// per (sequence, head); the eta rows are streamed with 16-byte accesses.
template <typename S, int DK, int DV>
__global__ __launch_bounds__(kThreads) void decode_kernel(int H, DecodeArgs g) {
    using T_ = typename storage<S>::type;
    constexpr int DV4 = DV / 4;
    constexpr int NG = (kThreads / DV4) < DK ? (kThreads / DV4) : DK;
    constexpr int NPER = DK / NG;
    __shared__ float sF[DK], sKh[DK], sQt[DK], sW[DK], sV[DV];
    __shared__ float4 sRed[NG][DV4];

    const T_* q = static_cast<const T_*>(g.q);
    const T_* k = static_cast<const T_*>(g.k);
    const T_* v = static_cast<const T_*>(g.v);
    const T_* a = static_cast<const T_*>(g.a);
    const T_* p = static_cast<const T_*>(g.p);
    const T_* r = static_cast<const T_*>(g.r);
    T_* y = static_cast<T_*>(g.y);

    const size_t sh = blockIdx.x;
    const int tid = threadIdx.x;
    if (tid < DK) {
        const size_t o = sh * DK + tid;
        float at, pt;
        if (g.ou_a) {
            const int oh = (int)(sh % H) * DK + tid;
            ou_gates(g.ou_a[oh], g.ou_p[oh], g.ou_d[oh], at, pt);
        } else {
            at = ld(a, o);
            pt = ld(p, o);
        }
        const float kt = ld(k, o), qt = ld(q, o), rt = ld(r, sh);
        const float lam = g.lam[o];
        const float rho = 1.f / (at * at + pt * lam);
        const float ln = rho * lam + kt * kt * rt;
        g.lam[o] = ln;
        const float inv = 1.f / ln;
        sF[tid] = at * rho;
        sKh[tid] = rt * kt;
        sQt[tid] = qt * inv;
        sW[tid] = qt * qt * inv;
    }
    for (int i = tid; i < DV; i += kThreads) sV[i] = ld(v, sh * DV + i);
    __syncthreads();
    const int d4 = tid % DV4, ng = tid / DV4;
    if (ng < NG) {
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        const float4 vv = make_float4(sV[4 * d4], sV[4 * d4 + 1], sV[4 * d4 + 2], sV[4 * d4 + 3]);
        float4* eta4 = reinterpret_cast<float4*>(g.eta + sh * DK * DV);
#pragma unroll 4
        for (int i = 0; i < NPER; ++i) {
            const int n = ng + i * NG;
            float4 e = eta4[n * DV4 + d4];
            const float F = sF[n], kh = sKh[n], qt = sQt[n];
            e.x = F * e.x + kh * vv.x;
            e.y = F * e.y + kh * vv.y;
            e.z = F * e.z + kh * vv.z;
            e.w = F * e.w + kh * vv.w;
            eta4[n * DV4 + d4] = e;
            acc.x += qt * e.x;
            acc.y += qt * e.y;
            acc.z += qt * e.z;
            acc.w += qt * e.w;
        }
        sRed[ng][d4] = acc;
    }
    __syncthreads();
    if (tid < DV4) {
        float4 acc = sRed[0][tid];
        for (int gi = 1; gi < NG; ++gi) {
            const float4 x = sRed[gi][tid];
            acc.x += x.x;
            acc.y += x.y;
            acc.z += x.z;
            acc.w += x.w;
        }
        st(y, sh * DV + 4 * tid + 0, acc.x);
        st(y, sh * DV + 4 * tid + 1, acc.y);
        st(y, sh * DV + 4 * tid + 2, acc.z);
        st(y, sh * DV + 4 * tid + 3, acc.w);
    }
    if (g.yvar && tid == kThreads - 1) {
        float acc = 0.f;
        for (int n = 0; n < DK; ++n) acc += sW[n];
        g.yvar[sh] = acc;
    }
}

// ----------------------------------------------------------------------------
// (dk, dv) dispatch over {16, 32, 64, 128}^2 and the storage type.
template <template <typename, int, int> class L, typename... A>
hipError_t dispatch(const Shape& s, A&&... args) {
#define KLA_CASE(DK_, DV_)                                                              \
    if (s.dk == DK_ && s.dv == DV_)                                                     \
        return s.bf16 ? L<bf16_t, DK_, DV_>::run(s, args...) : L<f32_t, DK_, DV_>::run(s, args...);
#define KLA_ROW(DK_) KLA_CASE(DK_, 16) KLA_CASE(DK_, 32) KLA_CASE(DK_, 64) KLA_CASE(DK_, 128)
    KLA_ROW(16) KLA_ROW(32) KLA_ROW(64) KLA_ROW(128)
#undef KLA_ROW
#undef KLA_CASE
    return hipErrorInvalidValue;
}

template <typename S, int DK, int DV>
struct FwdL {
    static hipError_t run(const Shape& s, const FwdArgs& a, float* saved_lam, hipStream_t st) {
        constexpr int DVT = kFwdDVT<DV>;
        const unsigned grid = (unsigned)(s.B * s.H * (DV / DVT));
        hipLaunchKernelGGL((fwd_recurrent_kernel<S, DK, DV>), dim3(grid), dim3(kFwdThreads<DK>), 0, st, s, a,
                           saved_lam);
        return hipGetLastError();
    }
};

template <typename S, int DK, int DV>
struct BwdL {
    static hipError_t run(const Shape& s, const BwdArgs& a, const float* saved_lam, void* ws, hipStream_t st) {
        if (!saved_lam) return hipErrorInvalidValue;
        const size_t ntok = (size_t)s.B * s.T * s.H * DK;
        float* wdqt = static_cast<float*>(ws);
        float* wPT = wdqt + ntok;
        // PT is written by the last segment's workgroups; with T == 0 it is detaT . eta0 summed over d,
        // which the reverse sweep does not need (no token reads it), so no workgroup is launched
        const unsigned grid1 = (unsigned)(s.B * s.H * (DK / 16) * n_checkpoints(s.T));
        if (grid1 > 0)
            hipLaunchKernelGGL((bwd_sweep1_kernel<S, DK, DV>), dim3(grid1), dim3(kThreads), 0, st, s, a, saved_lam,
                               wdqt, wPT);
        const float* lam_t = saved_lam;
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        auto kern = bwd_sweep2_kernel<S, DK, DV>;
        constexpr size_t bytes = Sweep2Cfg<DK, DV>::BYTES;
        // more than 64 KiB of LDS must be opted into once per kernel (thread-safe static init)
        static const hipError_t attr =
            hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
        if (attr != hipSuccess) return attr;
        hipLaunchKernelGGL(kern, dim3(s.B * s.H), dim3(Sweep2Cfg<DK, DV>::NTH), bytes, st, s, a, lam_t, wdqt, wPT);
        return hipGetLastError();
    }
};

template <typename S, int DK, int DV>
struct DecL {
    static hipError_t run(const Shape& s, const DecodeArgs& a, hipStream_t st) {
        hipLaunchKernelGGL((decode_kernel<S, DK, DV>), dim3(s.B * s.H), dim3(kThreads), 0, st, s.H, a);
        return hipGetLastError();
    }
};

}  // namespace

size_t recurrent_saved_bytes(const Shape& s) {
    return (saved_lam_floats(s) + (size_t)s.B * s.H * n_checkpoints(s.T) * s.dk * s.dv) * sizeof(float);
}

hipError_t launch_forward_recurrent(const Shape& s, const FwdArgs& a, float* saved_lam, hipStream_t st) {
    return dispatch<FwdL>(s, a, saved_lam, st);
}

// one part per batch row: the recurrent backward walks a whole (b, h) in one workgroup
int recurrent_ou_parts(const Shape& s) { return s.B; }

// dqt_t [B, T, H, dk] and PT [B, H, dk]
size_t backward_recurrent_workspace(const Shape& s) {
    const size_t ntok = (size_t)s.B * s.T * s.H * s.dk;
    return (ntok + (size_t)s.B * s.H * s.dk) * sizeof(float);
}

hipError_t launch_backward_recurrent(const Shape& s, const BwdArgs& a, const float* saved_lam, void* ws,
                                     hipStream_t st) {
    return dispatch<BwdL>(s, a, saved_lam, ws, st);
}

hipError_t launch_decode_step(const Shape& s, const DecodeArgs& a, hipStream_t st) {
    return dispatch<DecL>(s, a, st);
}

}  // namespace kla
