// Domain validation of the filter inputs (enabled by KLA_CHECK=1): abar in
// (0, 1], pbar >= 0, r > 0 and lam0 > 0, everything finite; with OU parameters
// instead of per-token gates, a > 0, delta > 0 and p finite.  Any violation sets
// *flag to 1 with an ordinary vector store.
#include "kla_device.hpp"
#include "kla_internal.hpp"

namespace kla {
namespace {

__global__ void zero_flag(int* flag) {
    if (threadIdx.x == 0) *flag = 0;
}

template <typename S>
__global__ __launch_bounds__(256) void validate_kernel(size_t nk, size_t nv, size_t nr, size_t nb, size_t ne,
                                                       const void* q_, const void* k_, const void* v_,
                                                       const void* a_, const void* p_, const void* r_,
                                                       const float* lam0, const float* eta0, size_t nou,
                                                       const float* ou_a, const float* ou_p, const float* ou_d,
                                                       int* flag) {
    using T_ = typename storage<S>::type;
    const T_ *q = (const T_*)q_, *k = (const T_*)k_, *v = (const T_*)v_;
    const T_ *a = (const T_*)a_, *p = (const T_*)p_, *r = (const T_*)r_;
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    bool bad = false;
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < nk; i += stride) {
        const float qv = ld(q, i), kv = ld(k, i);
        bad |= !isfinite(qv) || !isfinite(kv);
        if (a) {
            const float av = ld(a, i), pv = ld(p, i);
            bad |= !(av > 0.f && av <= 1.f) || !(pv >= 0.f && pv <= 3.0e38f);
        }
    }
    if (ou_a)
        for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < nou; i += stride)
            bad |= !(ou_a[i] > 0.f && ou_a[i] <= 3.0e38f) || !(ou_d[i] > 0.f && ou_d[i] <= 3.0e38f) ||
                   !isfinite(ou_p[i]);
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < nv; i += stride) bad |= !isfinite(ld(v, i));
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < nr; i += stride) {
        const float rv = ld(r, i);
        bad |= !(rv > 0.f && rv <= 3.0e38f);
    }
    if (lam0)
        for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < nb; i += stride)
            bad |= !(lam0[i] > 0.f && lam0[i] <= 3.0e38f);
    if (eta0)
        for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < ne; i += stride) bad |= !isfinite(eta0[i]);
    if (bad) *flag = 1;
}

}  // namespace

hipError_t launch_validate(const Shape& s, const void* q, const void* k, const void* v, const void* a,
                           const void* p, const void* r, const float* lam0, const float* eta0, int T,
                           int* flag, hipStream_t st, const float* ou_a, const float* ou_p, const float* ou_d,
                           bool per_channel) {
    hipLaunchKernelGGL(zero_flag, dim3(1), dim3(64), 0, st, flag);
    const size_t tok = (size_t)s.B * T * s.H;
    const size_t nk = tok * s.dk, nv = tok * s.dv, ne = (size_t)s.B * s.H * s.dk * s.dv;
    // per-channel precision: r [B, T, H, dv] and lam0 [B, H, dk, dv]
    const size_t nr = per_channel ? nv : tok, nb = per_channel ? ne : (size_t)s.B * s.H * s.dk;
    // OU parameters: [H, dk], or [H, dk, dv] (gates per key slot and value channel) with the
    // per-channel precision
    const size_t nou = (size_t)s.H * s.dk * (per_channel ? s.dv : 1);
    const unsigned grid = 1024;
    if (s.bf16)
        hipLaunchKernelGGL(validate_kernel<bf16_t>, dim3(grid), dim3(256), 0, st, nk, nv, nr, nb, ne, q, k, v, a,
                           p, r, lam0, eta0, nou, ou_a, ou_p, ou_d, flag);
    else
        hipLaunchKernelGGL(validate_kernel<f32_t>, dim3(grid), dim3(256), 0, st, nk, nv, nr, nb, ne, q, k, v, a,
                           p, r, lam0, eta0, nou, ou_a, ou_p, ou_d, flag);
    return hipGetLastError();
}

}  // namespace kla
