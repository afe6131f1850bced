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
//
// Arithmetic type A (acc<S>): fp64 for fp32 inputs, fp32 for bf16 inputs.  Every
// quantity that a recursion or a sum over tokens carries -- the precision walk,
// the forget gates, the information state and its adjoint, dqt, the log-gate and
// precision adjoints, and the saved context and workspace that hand them from
// kernel to kernel -- is held in A.  Only values used once per token (q / lam,
// q^2 / lam, partial sums that are rounded once into an output) pass through
// fp32.  With fp32 arithmetic the rounding accumulated along a 512-token adjoint
// chain alone exceeds the fp32 tolerance by a factor of four on the gate
// gradients; in fp64 it is negligible next to the final rounding of the outputs.
#include <type_traits>

#include "kla_buf.hpp"
#include "kla_device.hpp"
#include "kla_internal.hpp"

namespace kla {
namespace {

constexpr int kThreads = 256;
constexpr int kTB = 16;  // tokens per staged block of sweep 1
constexpr int kCKI = 64; // tokens between the information-state checkpoints of the saved context

// The saved context of this path, in the arithmetic type: lam_t [B, T, H, dk], then
// the information state before every kCKI-th token [B, H, ceil(T / kCKI), dk, dv].
__host__ __device__ inline size_t saved_lam_elems(const Shape& s) { return (size_t)s.B * s.T * s.H * s.dk; }
__host__ __device__ inline int n_checkpoints(int T) { return (T + kCKI - 1) / kCKI; }
__host__ __device__ inline size_t acc_bytes(const Shape& s) { return s.bf16 ? sizeof(float) : sizeof(double); }

// Per-token inputs reach the kernels in blocks of ROWS tokens, staged in LDS as
// rows of V.  A Part is one tensor's W values per token: each thread fetches
// elements tid + NT m of the next block into registers while the current block
// is worked on, and writes them to their LDS columns once that block is done,
// so a token's loads never wait in its recursion.  The kernels synchronise with
// barrier_lds (LDS ordering only): a full __syncthreads would wait for the
// prefetch at the first barrier after it is issued.
template <int ROWS, int W, int NT = kThreads, typename V = float>
struct Part {
    static constexpr int N = (ROWS * W + NT - 1) / NT;
    V x[N];
    // rows j < nt (nt >= 1): element c of row j at x0[j * ts + c].  Rows past nt and
    // elements past the block re-read the last valid element: they are never used,
    // and the loads stay unconditional, so nothing waits for them before the commit.
    template <typename T>
    __device__ __forceinline__ void fetch(const T* x0, int ts, int nt) {
#pragma unroll
        for (int m = 0; m < N; ++m) {
            const int e = min((int)threadIdx.x + NT * m, ROWS * W - 1);
            const int j = min(e / W, nt - 1), c = e % W;
            x[m] = (V)ld(x0, (size_t)(j * ts + c));
        }
    }
    // row j of the block into dst[j * ROW + c0 + c]
    template <int ROW>
    __device__ __forceinline__ void commit(V* dst, int c0) const {
#pragma unroll
        for (int m = 0; m < N; ++m) {
            const int e = (int)threadIdx.x + NT * m;
            const int j = e / W, c = e % W;
            if (e < ROWS * W) dst[j * ROW + c0 + c] = x[m];
        }
    }
};

// Sum over each 16-lane row with DPP moves, held by every lane of the row.
template <typename A>
__device__ __forceinline__ A row_sum16(A x) {
    x += dpp<0xB1, 0xf>(x);    // quad_perm [1,0,3,2]
    x += dpp<0x4E, 0xf>(x);    // quad_perm [2,3,0,1]
    x += dpp<0x141, 0xf>(x);   // row_half_mirror
    x += dpp<0x140, 0xf>(x);   // row_mirror
    return x;
}

// x of the lane D below within its 16-lane row (row_shr; lanes with none read 0)
template <int D, typename A>
__device__ __forceinline__ A row_shr(A x) {
    static_assert(D >= 1 && D <= 15, "row shift");
    return dpp<0x110 + D, 0xf>(x);
}

// lane l reads lane l ^ 16 (ds_swizzle, bitmask mode)
__device__ __forceinline__ float swz16(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, x), 0x401F));
}
__device__ __forceinline__ double swz16(double x) {
    const uint64_t u = __builtin_bit_cast(uint64_t, x);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_ds_swizzle((int)(uint32_t)u, 0x401F);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_ds_swizzle((int)(uint32_t)(u >> 32), 0x401F);
    return __builtin_bit_cast(double, (uint64_t)lo | ((uint64_t)hi << 32));
}

// Sum over groups of W consecutive lanes (W = 16 or 32), held by every lane of the
// group: W = 32 exchanges the two row sums with a swizzle (lane l reads lane l ^ 16).
template <int W, typename A>
__device__ __forceinline__ A group_sum_all(A x) {
    static_assert(W == 16 || W == 32, "group width");
    x = row_sum16(x);
    if constexpr (W == 32) x += swz16(x);
    return x;
}

template <typename A>
__device__ __forceinline__ A amax(A x, A y) { return x > y ? x : y; }

// value channels per forward workgroup: 16, so that even a small head spreads over
// several workgroups (each walks the precision of the head itself)
template <int DV>
constexpr int kFwdDVT = DV < 16 ? DV : 16;
// threads per forward workgroup and tokens per staged block: blocks of 32 tokens
// (half the barriers per token) where the LDS holds them, two waves per SIMD at
// dk = 64 (measured at the state-tracking shape, dk = 32: 256 threads and blocks
// of 32 tokens beat 512 threads and blocks of 16); fp64 arithmetic at dk = 128
// takes blocks of 8 tokens, within the LDS of a workgroup
template <int DK>
constexpr int kFwdThreads = DK == 64 ? 512 : 256;
template <typename A, int DK>
constexpr int kFwdTB = DK <= 32 ? 32 : (DK == 128 && sizeof(A) == 8) ? 8 : 16;

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
// starting lam starts the lane's own walk over its tokens.  The walk leaves F
// (arithmetic type), q / lam and q^2 / lam; then every thread updates its state
// entries over the block and the readout partials are summed.
template <typename S, int DK, int DV>
struct FwdLay {
    using A = typename acc<S>::type;
    static constexpr int NTH = kFwdThreads<DK>;
    static constexpr int TBF = kFwdTB<A, DK>;   // tokens per staged block
    static constexpr int DVT = kFwdDVT<DV>;
    static constexpr int NG = NTH / DVT;
    // staged row of a token: abar, pbar, k, q [DK] each, this tile's v [DVT], r; after the
    // walk the abar column holds q / lam and the pbar column q^2 / lam
    static constexpr int CA = 0, CP = DK, CK = 2 * DK, CQ = 3 * DK, CV = 4 * DK, CR = CV + DVT, ROW = CR + 1;
    // LDS (bytes): staged rows (fp32), forget gates [TBF][DK] (A), readout partials [TBF][NG][DVT] (fp32)
    static constexpr int L_IN = 0, L_F = (TBF * ROW * 4 + 15) / 16 * 16;
    static constexpr int L_RED = L_F + TBF * DK * (int)sizeof(A);
    static constexpr int BYTES = L_RED + TBF * NG * DVT * 4;
    static_assert(BYTES <= 160 * 1024, "LDS budget of one workgroup");
};

template <typename S, int DK, int DV>
__global__ __launch_bounds__(kFwdThreads<DK>) void fwd_recurrent_kernel(Shape s, FwdArgs g,
                                                                        typename acc<S>::type* saved_lam) {
    using T_ = typename storage<S>::type;
    using A = typename acc<S>::type;
    using L = FwdLay<S, DK, DV>;
    constexpr int NTH = L::NTH, TBF = L::TBF, DVT = L::DVT, NG = L::NG;
    constexpr int NTILE = DV / DVT;
    constexpr int NPER = DK / NG > 0 ? DK / NG : 1;
    static_assert(DK % NG == 0 || NG > DK, "key width must be a multiple of the n-groups");
    constexpr int CA = L::CA, CP = L::CP, CK = L::CK, CQ = L::CQ, CV = L::CV, CR = L::CR, ROW = L::ROW;
    constexpr int NY = (TBF * DVT + NTH - 1) / NTH;   // outputs per thread and block
    constexpr int GPS = NTH / DK, TPG = TBF / GPS;       // walk lanes per key slot, tokens per lane
    static_assert(GPS * DK == NTH && TPG * GPS == TBF && GPS <= 16 && (GPS & (GPS - 1)) == 0,
                  "the walk lanes of a slot split the block evenly within a DPP row");

    extern __shared__ __align__(16) unsigned char smem[];
    float* sIn = reinterpret_cast<float*>(smem + L::L_IN);
    A* sF = reinterpret_cast<A*>(smem + L::L_F);
    float* sRed = reinterpret_cast<float*>(smem + L::L_RED);   // [TBF][NG][DVT]

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

    A Hs[NPER];
#pragma unroll
    for (int i = 0; i < NPER; ++i) {
        int n = ng + i * NG;
        Hs[i] = (owns && g.eta0) ? (A)g.eta0[((size_t)bh * DK + n) * DV + d] : A(0);
    }
    const int wn = tid / GPS, wg = tid % GPS;   // walk: key slot and token group of this lane
    A lam = g.lam0 ? (A)g.lam0[(size_t)bh * DK + wn] : A(1);   // lam before the block, in every lane of slot wn
    const bool ou = g.ou_a != nullptr;
    A oa = 0, op = 0;
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
    A* saved_H = saved_lam ? saved_lam + saved_lam_elems(s) : nullptr;
    const int nck = n_checkpoints(s.T);
    for (int blk = 0; blk < nblk; ++blk) {
        const int t0 = blk * TBF, nt = min(TBF, s.T - t0);
        if (saved_H && t0 % kCKI == 0 && owns) {   // the state before token t0
#pragma unroll
            for (int i = 0; i < NPER; ++i)
                saved_H[(((size_t)bh * nck + t0 / kCKI) * DK + ng + i * NG) * DV + d] = Hs[i];
        }
        A lsv[TPG];   // lam after each of this lane's tokens (the saved context)
        // Token loops carry no branch: rows past nt (the ragged last block) are worked on
        // as well, from the repeated last row, and only selects keep them out of the state.
        {
            A ta[TPG], tp[TPG], tk[TPG], tq[TPG], tr[TPG];
#pragma unroll
            for (int u = 0; u < TPG; ++u) {
                const float* row = sIn + (wg * TPG + u) * ROW;
                const A ra = row[CA + wn], rp = row[CP + wn];
                ta[u] = ou ? oa : ra;
                tp[u] = ou ? op : rp;
                tk[u] = row[CK + wn];
                tq[u] = row[CQ + wn];
                tr[u] = row[CR];
            }
            // this lane's product M_last ... M_first (tokens past nt: identity), scaled
            A m00 = 1, m01 = 0, m10 = 0, m11 = 1;
#pragma unroll
            for (int u = 0; u < TPG; ++u) {
                const A a2 = ta[u] * ta[u], phi = tk[u] * tk[u] * tr[u];
                const A z0 = fma(tp[u], m00, a2 * m10), z1 = fma(tp[u], m01, a2 * m11);
                const bool ok = wg * TPG + u < nt;
                m00 = ok ? fma(phi, z0, m00) : m00;
                m01 = ok ? fma(phi, z1, m01) : m01;
                m10 = ok ? z0 : m10;
                m11 = ok ? z1 : m11;
            }
            {
                const A sc = rcpa(amax(amax(m00, m01), amax(m10, m11)));
                m00 *= sc; m01 *= sc; m10 *= sc; m11 *= sc;
            }
            // inclusive scan over the slot's lanes: P_g = M_g ... M_0
            auto scan_step = [&](auto dd) {
                constexpr int D = decltype(dd)::value;
                if constexpr (D < GPS) {
                    const A b00 = row_shr<D>(m00), b01 = row_shr<D>(m01);
                    const A b10 = row_shr<D>(m10), b11 = row_shr<D>(m11);
                    const A c00 = fma(m00, b00, m01 * b10), c01 = fma(m00, b01, m01 * b11);
                    const A c10 = fma(m10, b00, m11 * b10), c11 = fma(m10, b01, m11 * b11);
                    const A sc = rcpa(amax(amax(c00, c01), amax(c10, c11)));
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
            const A e00 = row_shr<1>(m00), e01 = row_shr<1>(m01);
            const A e10 = row_shr<1>(m10), e11 = row_shr<1>(m11);
            A lw = lam;
            if (wg > 0) lw = fma(e00, lam, e01) * rcpa(fma(e10, lam, e11));
            // walk this lane's tokens
#pragma unroll
            for (int u = 0; u < TPG; ++u) {
                const int j = wg * TPG + u;
                float* row = sIn + j * ROW;
                const A rho = rcpa(ta[u] * ta[u] + tp[u] * lw);
                const A ln = rho * lw + tk[u] * tk[u] * tr[u];
                lw = j < nt ? ln : lw;
                lsv[u] = ln;
                const A inv = rcpa(ln);
                sF[j * DK + wn] = ta[u] * rho;
                row[CA + wn] = (float)(tq[u] * inv);
                row[CP + wn] = (float)(tq[u] * tq[u] * inv);
            }
            // lam after the block: the last group's, in every lane of the slot
            lam = __shfl(lw, (tid & 63 & ~(GPS - 1)) + GPS - 1, 64);
        }
        barrier_lds();
#pragma unroll
        for (int j = 0; j < TBF; ++j) {
            const float* row = sIn + j * ROW;
            const A vr = (A)row[CV + dl] * (A)row[CR];   // v_d r
            A acc = 0;
#pragma unroll
            for (int i = 0; i < NPER; ++i) {
                const int n = ng + i * NG;
                if (NG <= DK || owns) {
                    const A hn = fma(sF[j * DK + n], Hs[i], (A)row[CK + n] * vr);
                    Hs[i] = j < nt ? hn : Hs[i];
                    acc = fma((A)row[CA + n], hn, acc);
                }
            }
            sRed[(j * NG + ng) * DVT + dl] = (float)acc;
        }
        barrier_lds();
        // the block's outputs are formed in registers and stored after the commit, whose wait
        // then covers the prefetch only
        A yo[NY], yvo = 0;
#pragma unroll
        for (int u = 0; u < NY; ++u) {
            const int idx = tid + NTH * u, j = idx / DVT, dd = idx % DVT;
            A acc = 0;
            if (j < nt) {
#pragma unroll
                for (int gi = 0; gi < NG; ++gi) acc += sRed[(j * NG + gi) * DVT + dd];
            }
            yo[u] = acc;
        }
        const int jv = tid - (NTH - TBF);   // the token whose readout variance this thread sums
        const bool wv = tile == 0 && g.yvar && jv >= 0 && jv < nt;
        if (wv) {
#pragma unroll
            for (int n = 0; n < DK; ++n) yvo += sIn[jv * ROW + CP + n];
        }
        barrier_lds();
        commit();
#pragma unroll
        for (int u = 0; u < NY; ++u) {
            const int idx = tid + NTH * u, j = idx / DVT, dd = idx % DVT;
            if (j < nt) st(y, ((row0 + t0 + j) * s.H + h) * DV + tile * DVT + dd, yo[u]);
        }
        if (wv) g.yvar[(row0 + t0 + jv) * s.H + h] = (float)yvo;
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
    if (tile == 0 && g.lamT && wg == 0) g.lamT[(size_t)bh * DK + wn] = (float)lam;
    if (g.etaT && owns) {
#pragma unroll
        for (int i = 0; i < NPER; ++i) g.etaT[((size_t)bh * DK + ng + i * NG) * DV + d] = (float)Hs[i];
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
__global__ __launch_bounds__(kThreads) void bwd_sweep1_kernel(Shape s, BwdArgs g, const typename acc<S>::type* slam,
                                                               typename acc<S>::type* wdqt,
                                                               typename acc<S>::type* wPT) {
    using T_ = typename storage<S>::type;
    using A = typename acc<S>::type;
    constexpr int NT = 16, DL = 16, DPER = DV / DL;
    static_assert(DL == kTB, "lane j of a slot's row holds token j of the block");
    static_assert(kThreads == kTB * NT, "one (token, slot) gate per thread");
    // staged row of a token: abar, pbar, k of this workgroup's NT key slots, v [DV], dy [DV], r
    constexpr int CA = 0, CP = NT, CK = 2 * NT, CV = 3 * NT, CD = CV + DV, CR = CD + DV;
    constexpr int ROW = CR + 1;
    __shared__ float sIn[kTB * ROW];
    __shared__ A sL[kTB * NT];          // saved lam_t of the block's tokens
    __shared__ A sLP[NT];               // lam of the token before the block
    __shared__ A sF[kTB][NT];           // F of every (token, slot) of the block
    __shared__ A sK[kTB][NT];           // r k

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
    const A* ckH = slam + saved_lam_elems(s);

    A Hs[DPER];
#pragma unroll
    for (int i = 0; i < DPER; ++i) Hs[i] = ckH[(((size_t)bh * nck + seg) * DK + n) * DV + dl + i * DL];
    // the gate phase's (token, slot) pair of this thread
    const int gsl = tid % NT, gj = tid / NT;
    const bool ou = g.ou_a != nullptr;
    A goa = 0, gop = 0;
    if (ou) {
        const int gn = ktile * NT + gsl;
        ou_gates(g.ou_a[h * DK + gn], g.ou_p[h * DK + gn], g.ou_d[h * DK + gn], goa, gop);
    }

    Part<kTB, NT> xa, xp, xk;
    Part<kTB, NT, kThreads, A> xl;
    Part<kTB, DV> xv, xdy;
    Part<kTB, 1> xr;
    Part<1, NT, kThreads, A> xlp;
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
        if (t > 0 || lam0_one)
            xlp.fetch(slam + (t > 0 ? o - s.H : o) * DK + ktile * NT, 0, 1);
        else
            xlp.fetch(g.lam0 + (size_t)bh * DK + ktile * NT, 0, 1);
    };
    auto commit = [&]() {
        wait_vm_all();   // the prefetch has landed (and stores issued before it are done)
        xa.template commit<ROW>(sIn, CA);
        xp.template commit<ROW>(sIn, CP);
        xk.template commit<ROW>(sIn, CK);
        xl.template commit<NT>(sL, 0);
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
            const A ra = row[CA + gsl], rp = row[CP + gsl];
            const A at = ou ? goa : ra, pt = ou ? gop : rp;
            const A lp = gj > 0 ? sL[(gj - 1) * NT + gsl] : (t0 == 0 && lam0_one ? A(1) : sLP[gsl]);
            const A rho = rcpa(at * at + pt * lp);
            sF[gj][gsl] = at * rho;
            sK[gj][gsl] = (A)row[CR] * (A)row[CK + gsl];
        }
        barrier_lds();
        A odqt = 0;
#pragma unroll
        for (int j = 0; j < kTB; ++j) {   // no branch: rows past nt only reach selects
            const bool live = j < nt;
            const float* row = sIn + j * ROW;
            const A F = sF[j][nl], kh = sK[j][nl];
            A acc = 0;
#pragma unroll
            for (int i = 0; i < DPER; ++i) {
                const A hn = fma(F, Hs[i], kh * (A)row[CV + dl + i * DL]);
                Hs[i] = live ? hn : Hs[i];
                acc = fma(hn, (A)row[CD + dl + i * DL], acc);
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
    A acc = 0;
    if (g.detaT) {
#pragma unroll
        for (int i = 0; i < DPER; ++i) acc = fma((A)g.detaT[((size_t)bh * DK + n) * DV + dl + i * DL], Hs[i], acc);
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
template <typename A>
struct alignas(4 * sizeof(A)) A4 {
    A x, y, z, w;
};
template <typename A>
struct alignas(2 * sizeof(A)) A2 {
    A x, y;
};

template <int DK, int DV, int NTH_, int TB_, typename A>
struct Sweep2Lay {
    static constexpr int NTH = NTH_, TB = TB_;
    static constexpr int DVT = DV < 32 ? DV : 32, NG = NTH / DVT;
    static constexpr int NPER = DK / NG > 0 ? DK / NG : 1, DPER = DV / DVT;
    // staged row of token t (fp32): q, k, abar, pbar [DK] each; v, dy [DV]; r; the upstream
    // gradient of the readout variance.  Staged in the arithmetic type: lam_t and dqt_t [DK] each.
    static constexpr int CQ = 0, CK = DK, CA = 2 * DK, CP = 3 * DK;
    static constexpr int CV = 4 * DK, CD = CV + DV, CR = CD + DV, CG = CR + 1, ROW = CG + 1;
    static constexpr int WL = 0, WDQ = DK, WROW = 2 * DK;
    static constexpr int SA = (int)sizeof(A);
    // LDS (bytes): {F_{t+1}, qt, kh, rho} and {(abar rho)^2, pbar rho, q (dqt + q gv) / lam^2,
    // qt dqt} per (token, slot); the staged A rows; lam of the token before the block; dkh;
    // {dG, g} per (token, slot); the carried forget gate (two buffers); per-thread OU sums;
    // the staged fp32 rows; dv partials per n-group; dr terms
    static constexpr int L_C0 = 0, L_C1 = L_C0 + 4 * TB * DK * SA, L_W = L_C1 + 4 * TB * DK * SA;
    static constexpr int L_LP = L_W + TB * WROW * SA, L_PK = L_LP + DK * SA, L_SG = L_PK + TB * DK * SA;
    static constexpr int L_FC = L_SG + 2 * TB * DK * SA, L_OU = L_FC + 2 * DK * SA;
    static constexpr int L_IN = L_OU + 2 * NTH * SA, L_PV = L_IN + (TB * ROW * 4 + 15) / 16 * 16;
    static constexpr int L_DR = L_PV + TB * NG * DV * 4;
    static constexpr size_t BYTES = (size_t)L_DR + TB * DK * 4;
    static constexpr bool fits = NG <= DK && DK % NG == 0 && (TB * DK) % NTH == 0 && BYTES <= 160 * 1024;
};

// tokens per staged block: 16 where the LDS holds them, else 8, else 4
template <int DK, int DV, int NTH, typename A>
constexpr int sweep2_tb() {
    return Sweep2Lay<DK, DV, NTH, 16, A>::fits ? 16 : Sweep2Lay<DK, DV, NTH, 8, A>::fits ? 8 : 4;
}

// 512 threads (two waves per SIMD, half the dH entries per thread) for heads of up to
// 64 x 64 where the shape splits evenly over them and the LDS fits, else 256
template <int DK, int DV, typename A>
constexpr int sweep2_nth() {
    return (DK * DV <= 64 * 64 && Sweep2Lay<DK, DV, 512, sweep2_tb<DK, DV, 512, A>(), A>::fits) ? 512 : 256;
}

template <int DK, int DV, typename A>
struct Sweep2Cfg : Sweep2Lay<DK, DV, sweep2_nth<DK, DV, A>(), sweep2_tb<DK, DV, sweep2_nth<DK, DV, A>(), A>(), A> {
    static_assert(Sweep2Cfg::fits, "every thread owns dH entries; LDS budget");
};

template <typename S, int DK, int DV>
__global__ __launch_bounds__((Sweep2Cfg<DK, DV, typename acc<S>::type>::NTH)) void bwd_sweep2_kernel(
    Shape s, BwdArgs g, const typename acc<S>::type* wlam, const typename acc<S>::type* wdqt,
    const typename acc<S>::type* wPT, typename acc<S>::type* ou_part) {
    using T_ = typename storage<S>::type;
    using A = typename acc<S>::type;
    using C = Sweep2Cfg<DK, DV, A>;
    constexpr int DVT = C::DVT, NG = C::NG, NPER = C::NPER, DPER = C::DPER, TB = C::TB, ROW = C::ROW;
    constexpr int WROW = C::WROW;
    constexpr int NTH = C::NTH;
    constexpr int ND = TB * DK / NTH, NDV = (TB * DV + NTH - 1) / NTH;   // items per thread
    static_assert(ND * NTH == TB * DK, "(token, slot) items split evenly over the threads");
    extern __shared__ __align__(16) unsigned char smem[];
    A4<A>* sC0 = reinterpret_cast<A4<A>*>(smem + C::L_C0);   // [TB][DK]
    A4<A>* sC1 = reinterpret_cast<A4<A>*>(smem + C::L_C1);   // [TB][DK]
    A* sW = reinterpret_cast<A*>(smem + C::L_W);              // [TB][WROW]
    A* sLP = reinterpret_cast<A*>(smem + C::L_LP);            // [DK]
    A* sPK = reinterpret_cast<A*>(smem + C::L_PK);            // [TB][DK]
    A2<A>* sSG = reinterpret_cast<A2<A>*>(smem + C::L_SG);   // [TB][DK]
    A* sFC = reinterpret_cast<A*>(smem + C::L_FC);            // [2][DK]
    A* sOU = reinterpret_cast<A*>(smem + C::L_OU);            // [2][NTH]
    float* sIn = reinterpret_cast<float*>(smem + C::L_IN);    // [TB][ROW]
    float* sPV = reinterpret_cast<float*>(smem + C::L_PV);    // [TB][NG][DV]
    float* sDR = reinterpret_cast<float*>(smem + C::L_DR);    // [TB][DK]

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

    A dH[NPER][DPER];
#pragma unroll
    for (int i = 0; i < NPER; ++i)
#pragma unroll
        for (int j = 0; j < DPER; ++j)
            dH[i][j] = g.detaT ? (A)g.detaT[((size_t)bh * DK + ng + i * NG) * DV + dl + j * DVT] : A(0);

    // the dG / c recursion lives in threads tid < DK
    A cnext = 0, Sg = 0;
    if (tid < DK) {
        cnext = g.dlamT ? (A)g.dlamT[(size_t)bh * DK + tid] : A(0);
        Sg = wPT[(size_t)bh * DK + tid];
        sFC[DK + tid] = 1;   // no forget gate after the last token
    }
    const bool ou = g.ou_a != nullptr;
    A oa = 0, op = 0, sum_da = 0, sum_dp = 0;
    if (ou) ou_gates(g.ou_a[h * DK + nme], g.ou_p[h * DK + nme], g.ou_d[h * DK + nme], oa, op);

    Part<TB, DK, NTH> xq, xk, xa, xp;
    Part<TB, DK, NTH, A> xl, xdq;
    Part<TB, DV, NTH> xv, xdy;
    Part<TB, 1, NTH> xr, xg;
    Part<1, DK, NTH, A> xlp;
    // Loads stay unconditional: absent tensors are replaced by present ones whose values
    // are not used (OU gates: abar / pbar columns from k; no readout-variance gradient:
    // its column from r, scaled by zero; no initial precision: token 0's lam_{t-1}
    // from the saved lam, replaced by 1 where it is read).
    const T_* ga = ou ? k : a;
    const T_* gp = ou ? k : p;
    const A gscale = g.dyvar ? A(1) : A(0);
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
        if (g.dyvar)
            xg.fetch(g.dyvar + o, s.H, nt);
        else
            xg.fetch(r + o, s.H, nt);
        if (t > 0 || lam0_one)
            xlp.fetch(wlam + (t > 0 ? o - s.H : o) * DK, 0, 1);
        else
            xlp.fetch(g.lam0 + (size_t)bh * DK, 0, 1);
    };
    auto commit = [&]() {
        wait_vm_all();   // the prefetch has landed (and stores issued before it are done)
        xl.template commit<WROW>(sW, C::WL);
        xdq.template commit<WROW>(sW, C::WDQ);
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
                const A* wrow = sW + j * WROW;
                const A lam = wrow[C::WL + n];
                const A lp = j > 0 ? wrow[C::WL + n - WROW] : (t0 == 0 && lam0_one ? A(1) : sLP[n]);
                const A dqt = wrow[C::WDQ + n], qv = row[C::CQ + n], kv = row[C::CK + n];
                const A ra = row[C::CA + n], rp = row[C::CP + n];
                const A at = ou ? oa : ra, pt = ou ? op : rp;
                const A rt = row[C::CR], gv = gscale * (A)row[C::CG];
                const A rho = rcpa(at * at + pt * lp);
                const A il = rcpa(lam), qtl = qv * il, F = at * rho;
                A4<A>& c0 = sC0[j * DK + n];
                c0.y = qtl;
                c0.z = rt * kv;
                c0.w = rho;
                if (j > 0) sC0[(j - 1) * DK + n].x = F;
                else sFC[(cur ^ 1) * DK + n] = F;
                if (j == nt - 1) c0.x = sFC[cur * DK + n];
                sC1[j * DK + n] = A4<A>{F * F, pt * rho, qv * (dqt + qv * gv) * il * il, qtl * dqt};
            }
        }
        barrier_lds();
        // ---- B
        // tokens latest first, in runs of UB unrolled tokens: the whole block for small heads,
        // shorter runs where a thread holds many dH entries (keeps the loads in registers)
        constexpr int UB0 = NPER * DPER <= 2 ? TB : NPER * DPER <= 4 ? 8 : NPER * DPER <= 16 ? 4 : 2;
        constexpr int UB = UB0 < TB ? UB0 : TB;
        static_assert(TB % UB == 0, "runs split the block");
#pragma unroll 1
        for (int jb = TB - UB; jb >= 0; jb -= UB)
#pragma unroll
        for (int jj = UB - 1; jj >= 0; --jj) {   // no branch: rows past nt only reach selects
            const int j = jb + jj;
            const bool live = j < nt;
            const float* row = sIn + j * ROW;
            A dyd[DPER], vd[DPER], pv[DPER];
#pragma unroll
            for (int jd = 0; jd < DPER; ++jd) {
                dyd[jd] = row[C::CD + dl + jd * DVT];
                vd[jd] = row[C::CV + dl + jd * DVT];
                pv[jd] = 0;
            }
#pragma unroll
            for (int i = 0; i < NPER; ++i) {
                const int n = ng + i * NG;
                const A4<A> co = sC0[j * DK + n];
                A pk = 0;
#pragma unroll
                for (int jd = 0; jd < DPER; ++jd) {
                    const A hn = fma(co.x, dH[i][jd], co.y * dyd[jd]);
                    dH[i][jd] = live ? hn : dH[i][jd];
                    pk = fma(hn, vd[jd], pk);
                    pv[jd] = fma(hn, co.z, pv[jd]);
                }
                sPK[j * DK + n] = group_sum_all<DVT>(pk);   // the same value from every lane of the group
            }
#pragma unroll
            for (int jd = 0; jd < DPER; ++jd) sPV[(j * NG + ng) * DV + dl + jd * DVT] = (float)pv[jd];
        }
        barrier_lds();
        // ---- C
        if (tid < DK) {
#pragma unroll
            for (int j = TB - 1; j >= 0; --j) {   // no branch: rows past nt only reach selects
                const bool live = j < nt;
                const A kh = sC0[j * DK + tid].z;
                const A4<A> c1 = sC1[j * DK + tid];
                const A dkh = sPK[j * DK + tid];
                const A sg = Sg + (c1.w - kh * dkh);   // dG_t
                const A gl = cnext - c1.z;              // g_t
                sSG[j * DK + tid] = A2<A>{sg, gl};
                Sg = live ? sg : Sg;
                cnext = live ? c1.x * gl - c1.y * sg : cnext;
            }
        }
        barrier_lds();
        // ---- D (results in registers: they are stored after the commit, whose wait then
        // covers the prefetch only)
        A o_dq[ND], o_dk[ND], o_da[ND], o_dp[ND], o_dv[NDV];
#pragma unroll
        for (int u = 0; u < ND; ++u) {
            const int idx = tid + NTH * u, j = idx / DK, n = idx % DK;
            const float* row = sIn + j * ROW;
            const A* wrow = sW + j * WROW;
            const A lam = wrow[C::WL + n];
            const A lp = j > 0 ? wrow[C::WL + n - WROW] : (t0 == 0 && lam0_one ? A(1) : sLP[n]);
            const A dqt = wrow[C::WDQ + n], qv = row[C::CQ + n], kv = row[C::CK + n];
            const A ra = row[C::CA + n], rp = row[C::CP + n];
            const A at = ou ? oa : ra, pt = ou ? op : rp;
            const A rt = row[C::CR], gv = gscale * (A)row[C::CG];
            const A rho = sC0[j * DK + n].w;
            const A dkh = sPK[j * DK + n];
            const A2<A> sg = sSG[j * DK + n];
            const A qg = qv * gv;
            const A drho = sg.y * lp + sg.x * (at * at + pt * lp);
            o_dq[u] = (dqt + A(2) * qg) * rcpa(lam);
            o_dk[u] = rt * dkh + A(2) * kv * rt * sg.y;
            o_da[u] = sg.x * rcpa(at) - A(2) * at * rho * rho * drho;
            o_dp[u] = -lp * rho * rho * drho;
            if (j < nt) {
                if (ou) {
                    sum_da += o_da[u];
                    sum_dp += o_dp[u];
                }
                sDR[j * DK + n] = (float)(kv * dkh + kv * kv * sg.y);
            }
        }
#pragma unroll
        for (int u = 0; u < NDV; ++u) {
            const int idx = tid + NTH * u, j = idx / DV, dd = idx % DV;
            A acc = 0;
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
            A acc = 0;
#pragma unroll
            for (int n = 0; n < DK; ++n) acc += sDR[tid * DK + n];
            st(dr, (row0 + t0 + tid) * s.H + h, acc);
        }
        fetch(max(blk - 2, 0) * TB);
        cur ^= 1;
        barrier_lds();
    }
    wait_vm_all();   // the last (unused) prefetch has landed before the registers are released
    if (tid < DK && g.dlam0) g.dlam0[(size_t)bh * DK + tid] = (float)cnext;
    if (ou) {   // part b of the token sums: the threads of one slot are combined in order
        sOU[tid] = sum_da;
        sOU[NTH + tid] = sum_dp;
        barrier_lds();
        if (tid < DK) {
            A sa = 0, sp = 0;
            for (int i = tid; i < NTH; i += DK) {
                sa += sOU[i];
                sp += sOU[NTH + i];
            }
            const size_t np = (size_t)s.B * s.H * DK;
            ou_part[(size_t)bh * DK + tid] = sa;
            ou_part[np + (size_t)bh * DK + tid] = sp;
        }
    }
    if (g.deta0) {   // sFC[cur] holds F of token 0
#pragma unroll
        for (int i = 0; i < NPER; ++i)
#pragma unroll
            for (int j = 0; j < DPER; ++j) {
                const int n = ng + i * NG;
                g.deta0[((size_t)bh * DK + n) * DV + dl + j * DVT] = (float)(sFC[cur * DK + n] * dH[i][j]);
            }
    }
}

// ----------------------------------------------------------------------------
// Decode: one token for S sequences, belief updated in place.  One workgroup
// per (sequence, head); the eta rows are streamed with 16-byte accesses.
template <typename S, int DK, int DV>
__global__ __launch_bounds__(kThreads) void decode_kernel(int H, DecodeArgs g) {
    using T_ = typename storage<S>::type;
    using A = typename acc<S>::type;
    constexpr int DV4 = DV / 4;
    constexpr int NG = (kThreads / DV4) < DK ? (kThreads / DV4) : DK;
    constexpr int NPER = DK / NG;
    __shared__ A sF[DK], sKh[DK], sQt[DK], sW[DK], sV[DV];
    __shared__ A4<A> sRed[NG][DV4];

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
        A at, pt;
        if (g.ou_a) {
            const int oh = (int)(sh % H) * DK + tid;
            ou_gates(g.ou_a[oh], g.ou_p[oh], g.ou_d[oh], at, pt);
        } else {
            at = ld(a, o);
            pt = ld(p, o);
        }
        const A kt = ld(k, o), qt = ld(q, o), rt = ld(r, sh);
        const A lam = g.lam[o];
        const A rho = A(1) / (at * at + pt * lam);
        const A ln = rho * lam + kt * kt * rt;
        g.lam[o] = (float)ln;
        const A inv = A(1) / ln;
        sF[tid] = at * rho;
        sKh[tid] = rt * kt;
        sQt[tid] = qt * inv;
        sW[tid] = qt * qt * inv;
    }
    for (int i = tid; i < DV; i += kThreads) sV[i] = ld(v, sh * DV + i);
    __syncthreads();
    const int d4 = tid % DV4, ng = tid / DV4;
    if (ng < NG) {
        A4<A> acc{0, 0, 0, 0};
        const A4<A> vv{sV[4 * d4], sV[4 * d4 + 1], sV[4 * d4 + 2], sV[4 * d4 + 3]};
        float4* eta4 = reinterpret_cast<float4*>(g.eta + sh * DK * DV);
#pragma unroll 4
        for (int i = 0; i < NPER; ++i) {
            const int n = ng + i * NG;
            const float4 e = eta4[n * DV4 + d4];
            const A F = sF[n], kh = sKh[n], qt = sQt[n];
            const A ex = fma(F, (A)e.x, kh * vv.x), ey = fma(F, (A)e.y, kh * vv.y);
            const A ez = fma(F, (A)e.z, kh * vv.z), ew = fma(F, (A)e.w, kh * vv.w);
            eta4[n * DV4 + d4] = make_float4((float)ex, (float)ey, (float)ez, (float)ew);
            acc.x = fma(qt, ex, acc.x);
            acc.y = fma(qt, ey, acc.y);
            acc.z = fma(qt, ez, acc.z);
            acc.w = fma(qt, ew, acc.w);
        }
        sRed[ng][d4] = acc;
    }
    __syncthreads();
    if (tid < DV4) {
        A4<A> acc = sRed[0][tid];
        for (int gi = 1; gi < NG; ++gi) {
            const A4<A> x = sRed[gi][tid];
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
        A acc = 0;
        for (int n = 0; n < DK; ++n) acc += sW[n];
        g.yvar[sh] = (float)acc;
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

// more than 64 KiB of LDS must be opted into once per kernel (thread-safe static init at the caller)
template <typename K>
hipError_t allow_lds(K kern, size_t bytes) {
    return hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                               (int)bytes);
}

template <typename S, int DK, int DV>
struct FwdL {
    static hipError_t run(const Shape& s, const FwdArgs& a, void* saved, hipStream_t st) {
        using A = typename acc<S>::type;
        using L = FwdLay<S, DK, DV>;
        auto kern = fwd_recurrent_kernel<S, DK, DV>;
        static const hipError_t attr = allow_lds(kern, L::BYTES);
        if (attr != hipSuccess) return attr;
        const unsigned grid = (unsigned)(s.B * s.H * (DV / L::DVT));
        hipLaunchKernelGGL(kern, dim3(grid), dim3(L::NTH), L::BYTES, st, s, a, static_cast<A*>(saved));
        return hipGetLastError();
    }
};

template <typename S, int DK, int DV>
struct BwdL {
    static hipError_t run(const Shape& s, const BwdArgs& a, const void* saved, void* ws, hipStream_t st) {
        using A = typename acc<S>::type;
        if (!saved) return hipErrorInvalidValue;
        const A* slam = static_cast<const A*>(saved);
        const size_t ntok = (size_t)s.B * s.T * s.H * DK;
        A* wdqt = static_cast<A*>(ws);
        A* wPT = wdqt + ntok;
        // PT is written by the last segment's workgroups; with T == 0 it is detaT . eta0 summed over d,
        // which the reverse sweep does not need (no token reads it), so no workgroup is launched
        const unsigned grid1 = (unsigned)(s.B * s.H * (DK / 16) * n_checkpoints(s.T));
        if (grid1 > 0)
            hipLaunchKernelGGL((bwd_sweep1_kernel<S, DK, DV>), dim3(grid1), dim3(kThreads), 0, st, s, a, slam, wdqt,
                               wPT);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        using C = Sweep2Cfg<DK, DV, A>;
        auto kern = bwd_sweep2_kernel<S, DK, DV>;
        static const hipError_t attr = allow_lds(kern, C::BYTES);
        if (attr != hipSuccess) return attr;
        hipLaunchKernelGGL(kern, dim3(s.B * s.H), dim3(C::NTH), C::BYTES, st, s, a, slam, wdqt, wPT,
                           static_cast<A*>(a.ou_part));
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
    return (saved_lam_elems(s) + (size_t)s.B * s.H * n_checkpoints(s.T) * s.dk * s.dv) * acc_bytes(s);
}

hipError_t launch_forward_recurrent(const Shape& s, const FwdArgs& a, void* saved, hipStream_t st) {
    return dispatch<FwdL>(s, a, saved, st);
}

// one part per batch row: the recurrent backward walks a whole (b, h) in one workgroup
int recurrent_ou_parts(const Shape& s) { return s.B; }
size_t recurrent_ou_part_bytes(const Shape& s) { return acc_bytes(s); }

// dqt_t [B, T, H, dk] and PT [B, H, dk], in the arithmetic type
size_t backward_recurrent_workspace(const Shape& s) {
    const size_t ntok = (size_t)s.B * s.T * s.H * s.dk;
    return (ntok + (size_t)s.B * s.H * s.dk) * acc_bytes(s);
}

hipError_t launch_backward_recurrent(const Shape& s, const BwdArgs& a, const void* saved, void* ws,
                                     hipStream_t st) {
    return dispatch<BwdL>(s, a, saved, ws, st);
}

hipError_t launch_decode_step(const Shape& s, const DecodeArgs& a, hipStream_t st) {
    return dispatch<DecL>(s, a, st);
}

}  // namespace kla
