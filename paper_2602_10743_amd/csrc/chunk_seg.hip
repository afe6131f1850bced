// Segment-parallel forward for few, long sequences.
//
// With B H small and T long, one workgroup per (b, h, value tile) leaves most
// of the chip idle.  The sequence is cut into NS equal segments and both
// recursions are carried across segment boundaries by their composition laws
// (Corollaries 1 and 2):
//   1. per piece of up to 256 tokens and key slot, the product of Theorem 1's
//      2x2 matrices over the piece's tokens (seg_prec_kernel), with prod abar,
//      then the product over each segment's pieces (seg_compose_kernel);
//   2. an exclusive scan over the segments gives the precision at every
//      segment start and the segment's gate product P_s = prod_t F_t
//      (seg_lam_scan_kernel);
//   3. the chunked forward over every segment at once from those precisions
//      and a zero state gives the state each segment adds on its own, U_s;
//   4. an exclusive scan of H_{s+1} = diag(P_s) H_s + U_s gives the state at
//      every segment start (seg_state_scan_kernel);
//   5. the chunked forward over every segment from the exact start belief
//      writes y (and yvar).
// Steps 3 and 5 run the chunked kernel on a virtual shape: batch B NS,
// length T / NS (token (b NS + s) T/NS + t is token b T + s T/NS + t), so every
// segment is its own sequence.
#include "kla_device.hpp"
#include "kla_internal.hpp"

namespace kla {
namespace {

// Per (b, h, piece of L tokens): lanes = key slots.  The images of (1, 0) and
// (0, 1) under the piece's matrices, with prod abar, rescaled together every
// 16 tokens by the largest entry (the matrix is projective and P = A / z is
// unchanged by a common scale).
template <typename S, int DK>
__global__ __launch_bounds__(DK) void seg_prec_kernel(int T, int H, int NP, const void* a_, const void* p_,
                                                      const void* k_, const void* r_, float* __restrict__ mseg) {
    using T_ = typename storage<S>::type;
    const T_ *a = static_cast<const T_*>(a_), *p = static_cast<const T_*>(p_), *k = static_cast<const T_*>(k_);
    const T_* r = static_cast<const T_*>(r_);
    const int seg = blockIdx.x % NP, bh = blockIdx.x / NP;
    const int b = bh / H, h = bh % H, n = threadIdx.x;
    const int L = T / NP;
    float x0 = 1.f, z0 = 0.f, x1 = 0.f, z1 = 1.f, A = 1.f;
    for (int t0 = 0; t0 < L; t0 += 16) {
#pragma unroll 4
        for (int j = 0; j < 16; ++j) {
            const size_t tok = ((size_t)b * T + (size_t)seg * L + t0 + j) * H + h;
            const float av = ld(a, tok * DK + n), pv = ld(p, tok * DK + n), kv = ld(k, tok * DK + n);
            const float phi = kv * kv * ld(r, tok);
            const float a2 = av * av;
            const float zn0 = fmaf(pv, x0, a2 * z0), zn1 = fmaf(pv, x1, a2 * z1);
            x0 = fmaf(phi, zn0, x0);
            x1 = fmaf(phi, zn1, x1);
            z0 = zn0;
            z1 = zn1;
            A *= av;
        }
        const float m = fmaxf(fmaxf(fabsf(x0), fabsf(z0)), fmaxf(fabsf(x1), fabsf(z1)));
        const float sc = 1.f / m;
        x0 *= sc;
        z0 *= sc;
        x1 *= sc;
        z1 *= sc;
        A *= sc;
    }
    float* o = mseg + ((size_t)bh * NP + seg) * 5 * DK;
    o[0 * DK + n] = x0;
    o[1 * DK + n] = z0;
    o[2 * DK + n] = x1;
    o[3 * DK + n] = z1;
    o[4 * DK + n] = A;
}

// Per (b, h, segment, key slot): the product of the segment's PPS piece matrices
// (later pieces on the left) with their abar products, rescaled by the largest
// entry after each piece; written over the segment's first piece.
__global__ __launch_bounds__(256) void seg_compose_kernel(int nbh, int DK, int NS, int PPS, float* __restrict__ mseg) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= nbh * NS * DK) return;
    const int n = i % DK, seg = (i / DK) % NS, bh = i / (DK * NS);
    float* m0 = mseg + ((size_t)bh * NS * PPS + (size_t)seg * PPS) * 5 * DK;
    float x0 = m0[0 * DK + n], z0 = m0[1 * DK + n], x1 = m0[2 * DK + n], z1 = m0[3 * DK + n], A = m0[4 * DK + n];
    for (int u = 1; u < PPS; ++u) {
        const float* m = m0 + (size_t)u * 5 * DK;
        const float mx0 = m[0 * DK + n], mz0 = m[1 * DK + n], mx1 = m[2 * DK + n], mz1 = m[3 * DK + n];
        const float nx0 = fmaf(mx0, x0, mx1 * z0), nz0 = fmaf(mz0, x0, mz1 * z0);
        const float nx1 = fmaf(mx0, x1, mx1 * z1), nz1 = fmaf(mz0, x1, mz1 * z1);
        A *= m[4 * DK + n];
        const float sc = 1.f / fmaxf(fmaxf(fabsf(nx0), fabsf(nz0)), fmaxf(fabsf(nx1), fabsf(nz1)));
        x0 = nx0 * sc;
        z0 = nz0 * sc;
        x1 = nx1 * sc;
        z1 = nz1 * sc;
        A *= sc;
    }
    m0[0 * DK + n] = x0;
    m0[1 * DK + n] = z0;
    m0[2 * DK + n] = x1;
    m0[3 * DK + n] = z1;
    m0[4 * DK + n] = A;
}

// Per (b, h, key slot): lam at every segment start (virtual layout
// [(b NS + s) H + h][DK]), each segment's gate product, and the final lam.
__global__ __launch_bounds__(256) void seg_lam_scan_kernel(int B, int H, int DK, int NS, int PPS,
                                                           const float* __restrict__ mseg,
                                                           const float* __restrict__ lam0, float* __restrict__ lam_start,
                                                           float* __restrict__ pseg, float* __restrict__ lamT) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= B * H * DK) return;
    const int n = i % DK, bh = i / DK, b = bh / H, h = bh % H;
    float lam = lam0 ? lam0[i] : 1.f;
    for (int s = 0; s < NS; ++s) {
        const size_t v = ((size_t)b * NS + s) * H + h;
        lam_start[v * DK + n] = lam;
        const float* m = mseg + ((size_t)bh * NS * PPS + (size_t)s * PPS) * 5 * DK;   // the composed segment
        const float x = fmaf(m[0 * DK + n], lam, m[2 * DK + n]);
        const float z = fmaf(m[1 * DK + n], lam, m[3 * DK + n]);
        pseg[v * DK + n] = m[4 * DK + n] / z;
        lam = x / z;
    }
    if (lamT) lamT[i] = lam;
}

// tokens per piece of the precision pass: the largest of 256, 128, 64, 32 dividing the segment
int piece_len(int L) {
    int sub = 256;
    while (L % sub) sub /= 2;
    return sub;
}

// Per element (b, h, n, d): H at every segment start, then the final state.
__global__ __launch_bounds__(256) void seg_state_scan_kernel(int B, int H, int DK, int DV, int NS,
                                                             const float* __restrict__ pseg,
                                                             const float* __restrict__ useg,
                                                             const float* __restrict__ eta0,
                                                             float* __restrict__ h_start, float* __restrict__ etaT) {
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const size_t per = (size_t)DK * DV;
    if (i >= (size_t)B * H * per) return;
    const size_t e = i % per, bh = i / per;
    const int n = (int)(e / DV), b = (int)(bh / H), h = (int)(bh % H);
    float st = eta0 ? eta0[i] : 0.f;
    for (int s = 0; s < NS; ++s) {
        const size_t v = ((size_t)b * NS + s) * H + h;
        h_start[v * per + e] = st;
        st = fmaf(pseg[v * DK + n], st, useg[v * per + e]);
    }
    if (etaT) etaT[i] = st;
}

}  // namespace

int forward_segments(const Shape& s) {
    if (!chunked_supported(s)) return 1;
    const int ntile = s.dv < 64 ? 1 : s.dv / 64;
    const long wg = (long)s.B * s.H * ntile;
    int ns = 1;
    // segments of at least 1024 tokens, a whole number of 32-token chunks each, until the
    // workgroups fill the chip once (one per CU)
    while (wg * ns * 2 <= 256 && s.T % (ns * 2 * 32) == 0 && s.T / (ns * 2) >= 1024) ns *= 2;
    return ns;
}

size_t forward_segmented_workspace(const Shape& s) {
    const int ns = forward_segments(s);
    if (ns < 2) return 0;
    const size_t np = (size_t)s.T / piece_len(s.T / ns);
    const size_t nl = (size_t)s.B * s.H * ns * s.dk, ne = nl * s.dv;
    // mseg (5 per piece and slot), lam_start, pseg (nl each), useg, h_start (ne each)
    return (5 * (size_t)s.B * s.H * np * s.dk + 2 * nl + 2 * ne) * sizeof(float) + 5 * 256;
}

hipError_t launch_forward_segmented(const Shape& s, const FwdArgs& a, void* ws, hipStream_t st) {
    const int ns = forward_segments(s);
    const int pps = (s.T / ns) / piece_len(s.T / ns), np = ns * pps;   // pieces per segment, in all
    const size_t nl = (size_t)s.B * s.H * ns * s.dk, ne = nl * s.dv;
    auto carve = [&](size_t count) {
        float* p = static_cast<float*>(ws);
        ws = static_cast<char*>(ws) + (count * sizeof(float) + 255) / 256 * 256;
        return p;
    };
    float* mseg = carve(5 * (size_t)s.B * s.H * np * s.dk);
    float* lam_start = carve(nl);
    float* pseg = carve(nl);
    float* useg = carve(ne);
    float* h_start = carve(ne);
    const int nbh = s.B * s.H;
#define KLA_SEG_PREC(DK_)                                                                                      \
    if (s.dk == DK_) {                                                                                         \
        hipLaunchKernelGGL((seg_prec_kernel<bf16_t, DK_>), dim3((unsigned)(nbh * np)), dim3(DK_), 0, st, s.T, \
                           s.H, np, a.a, a.p, a.k, a.r, mseg);                                                 \
    }
    KLA_SEG_PREC(32) KLA_SEG_PREC(64) KLA_SEG_PREC(128)
#undef KLA_SEG_PREC
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(seg_compose_kernel, dim3((unsigned)((nbh * ns * s.dk + 255) / 256)), dim3(256), 0, st, nbh,
                       s.dk, ns, pps, mseg);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(seg_lam_scan_kernel, dim3((unsigned)((nbh * s.dk + 255) / 256)), dim3(256), 0, st, s.B, s.H,
                       s.dk, ns, pps, mseg, a.lam0, lam_start, pseg, a.lamT);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // every segment as its own sequence
    const Shape v{s.B * ns, s.T / ns, s.H, s.dk, s.dv, s.bf16};
    FwdArgs zero = a;   // the state each segment adds from a zero start (no readout)
    zero.lam0 = lam_start;
    zero.eta0 = nullptr;
    zero.y = nullptr;
    zero.yvar = nullptr;
    zero.lamT = nullptr;
    zero.etaT = useg;
    if ((e = launch_forward_chunked(v, zero, nullptr, st)) != hipSuccess) return e;
    const size_t nel = (size_t)nbh * s.dk * s.dv;
    hipLaunchKernelGGL(seg_state_scan_kernel, dim3((unsigned)((nel + 255) / 256)), dim3(256), 0, st, s.B, s.H, s.dk,
                       s.dv, ns, pseg, useg, a.eta0, h_start, a.etaT);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    FwdArgs full = a;   // the exact pass: y and yvar from every segment's start belief
    full.lam0 = lam_start;
    full.eta0 = h_start;
    full.lamT = nullptr;
    full.etaT = nullptr;
    return launch_forward_chunked(v, full, nullptr, st);
}

}  // namespace kla
