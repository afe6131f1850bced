// Gradients of the OU parameters (Sec. 4.1, eq. discretisation) from the
// backward's per-part sums of the gate gradients.
//
// With abar = exp(-a delta), E = abar^2 and s = (1 - E) / (2 a), so that
// pbar = p^2 s, and G_a, G_p the gradients of the loss with respect to abar and
// pbar summed over every (b, t):
//   da     = G_a (-delta abar) + G_p p^2 (delta E - s) / a
//   dp     = G_p 2 p s
//   ddelta = G_a (-a abar) + G_p p^2 E
// The parts are added in a fixed order and the chain rule is taken in fp64
// ((delta E - s) / a cancels for small a delta).
#include "kla_device.hpp"
#include "kla_internal.hpp"

namespace kla {
namespace {

template <typename P>
__global__ __launch_bounds__(256) void ou_param_grads_kernel(int n, int nparts, const P* __restrict__ part,
                                                             const float* __restrict__ a, const float* __restrict__ p,
                                                             const float* __restrict__ d, float* __restrict__ da,
                                                             float* __restrict__ dp, float* __restrict__ dd) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    double ga = 0.0, gp = 0.0;
    for (int j = 0; j < nparts; ++j) {
        ga += part[(size_t)j * n + i];
        gp += part[((size_t)nparts + j) * n + i];
    }
    const double av = a[i], pv = p[i], dv = d[i];
    const double abar = exp(-av * dv), E = abar * abar;
    const double s = -expm1(-2.0 * av * dv) / (2.0 * av);
    da[i] = (float)(ga * (-dv * abar) + gp * pv * pv * (dv * E - s) / av);
    dp[i] = (float)(gp * 2.0 * pv * s);
    dd[i] = (float)(ga * (-av * abar) + gp * pv * pv * E);
}

}  // namespace

hipError_t launch_ou_param_grads(int H, int dk, int nparts, const void* part, bool part_f64, const float* a,
                                 const float* p, const float* d, float* da, float* dp, float* dd, hipStream_t st) {
    const int n = H * dk;
    const dim3 grid((unsigned)((n + 255) / 256));
    if (part_f64)
        hipLaunchKernelGGL(ou_param_grads_kernel<double>, grid, dim3(256), 0, st, n, nparts,
                           static_cast<const double*>(part), a, p, d, da, dp, dd);
    else
        hipLaunchKernelGGL(ou_param_grads_kernel<float>, grid, dim3(256), 0, st, n, nparts,
                           static_cast<const float*>(part), a, p, d, da, dp, dd);
    return hipGetLastError();
}

}  // namespace kla
