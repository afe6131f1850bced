// C ABI of the KLA filter layer: argument validation, workspace layout and
// launch sequencing.  Declarations and contracts are in include/kla.h.
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime.h>

#include "kla.h"
#include "kla_internal.hpp"

namespace {

constexpr size_t kAlign = 256;

size_t round_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool width_ok(int w) { return w == 16 || w == 32 || w == 64 || w == 128; }

bool aligned(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

kla_status check_desc(const kla_desc* d) {
    if (!d) return KLA_ERR_NULL;
    if (d->dtype != KLA_F32 && d->dtype != KLA_BF16) return KLA_ERR_DTYPE;
    if (d->B < 1 || d->H < 1 || d->T < 0 || !width_ok(d->dk) || !width_ok(d->dv)) return KLA_ERR_SHAPE;
    // every per-tensor element count must stay addressable with 32-bit grid math
    const double tok = (double)d->B * d->T * d->H * (d->dk > d->dv ? d->dk : d->dv);
    if (tok > 9.0e18 || (double)d->B * d->H * 8 > 2.0e9) return KLA_ERR_SHAPE;
    return KLA_OK;
}

kla::Shape shape_of(const kla_desc* d) { return kla::Shape{d->B, d->T, d->H, d->dk, d->dv, d->dtype == KLA_BF16}; }

// One predicate decides the saved-context layout on both sides: the context is in
// the chunked layout exactly when the chunked backward will consume it.
bool saves_chunked(const kla::Shape& s) { return kla::chunked_bwd_supported(s); }

bool check_mode() {
    const char* e = getenv("KLA_CHECK");
    return e && e[0] == '1';
}

template <typename... P>
bool all_aligned(P... ps) {
    return (aligned(ps) && ...);
}

}  // namespace

namespace kla {
hipError_t launch_validate(const Shape& s, const void* q, const void* k, const void* v, const void* a,
                           const void* p, const void* r, const float* lam0, const float* eta0, int T,
                           int* flag, hipStream_t st, const float* ou_a, const float* ou_p, const float* ou_d,
                           bool per_channel);
}

namespace {

// Domain check of the inputs (KLA_CHECK=1): synchronous; returns KLA_ERR_NUMERIC
// when any value is outside abar in (0,1], pbar >= 0, r > 0, lam0 > 0, finite
// (OU parameters: a > 0, delta > 0, p finite).
kla_status validate(const kla::Shape& s, int T, const void* q, const void* k, const void* v, const void* a,
                    const void* p, const void* r, const float* lam0, const float* eta0, void* flag_ws,
                    hipStream_t st, const float* ou_a = nullptr, const float* ou_p = nullptr,
                    const float* ou_d = nullptr, bool per_channel = false) {
    int* flag = static_cast<int*>(flag_ws);
    if (kla::launch_validate(s, q, k, v, a, p, r, lam0, eta0, T, flag, st, ou_a, ou_p, ou_d, per_channel) !=
        hipSuccess)
        return KLA_ERR_HIP;
    int host = 0;
    if (hipMemcpyAsync(&host, flag, sizeof(int), hipMemcpyDeviceToHost, st) != hipSuccess) return KLA_ERR_HIP;
    if (hipStreamSynchronize(st) != hipSuccess) return KLA_ERR_HIP;
    return host ? KLA_ERR_NUMERIC : KLA_OK;
}

// After a chunked call under KLA_CHECK=1: the walks set the flag (zeroed by validate)
// when a chunk's in-chunk gate products left fp32 range.  Synchronous.
kla_status range_status(const void* flag_ws, hipStream_t st) {
    int host = 0;
    if (hipMemcpyAsync(&host, flag_ws, sizeof(int), hipMemcpyDeviceToHost, st) != hipSuccess) return KLA_ERR_HIP;
    if (hipStreamSynchronize(st) != hipSuccess) return KLA_ERR_HIP;
    return host ? KLA_ERR_RANGE : KLA_OK;
}

}  // namespace

extern "C" {

size_t kla_forward_workspace(const kla_desc* desc) {
    if (check_desc(desc) != KLA_OK) return 0;
    // validation flag, then the segment-parallel forward's carries when the shape takes it
    return kAlign + round_up(kla::forward_segmented_workspace(shape_of(desc)));
}

size_t kla_saved_bytes(const kla_desc* desc) {
    if (check_desc(desc) != KLA_OK) return 0;
    const kla::Shape s = shape_of(desc);
    if (saves_chunked(s)) return kla::chunked_saved_bytes(s);
    return kla::c64_supported(s) ? kla::c64_saved_bytes(s) : kla::recurrent_saved_bytes(s);
}

size_t kla_backward_workspace(const kla_desc* desc, int with_saved) {
    if (check_desc(desc) != KLA_OK) return 0;
    const kla::Shape s = shape_of(desc);
    if (kla::chunked_bwd_supported(s)) {
        size_t bytes = kAlign + round_up(kla::chunked_bwd_workspace(s));
        if (!with_saved) {  // the context is recomputed: saved states plus a scratch output
            const size_t elt = s.bf16 ? 2 : 4;
            bytes += round_up(kla::chunked_saved_bytes(s)) + round_up((size_t)s.B * s.T * s.H * s.dv * elt);
        }
        return bytes;
    }
    if (kla::c64_supported(s)) {
        size_t bytes = kAlign;
        if (!with_saved)   // the context is recomputed: saved states plus a scratch output
            bytes += round_up(kla::c64_saved_bytes(s)) + round_up((size_t)s.B * s.T * s.H * s.dv * sizeof(float));
        return bytes;
    }
    size_t bytes = kAlign + round_up(kla::backward_recurrent_workspace(s));
    if (!with_saved) {  // the precision trajectory is recomputed by the forward, plus a scratch output
        const size_t elt = s.bf16 ? 2 : 4;
        bytes += round_up(kla::recurrent_saved_bytes(s)) + round_up((size_t)s.B * s.T * s.H * s.dv * elt);
    }
    return bytes;
}

}  // extern "C"

namespace {

// The forward behind both gate forms: per-token abar / pbar in a.a, a.p, or OU
// parameters in a.ou_a, a.ou_p, a.ou_d.
kla_status forward_impl(const kla_desc* desc, const kla::FwdArgs& a, bool ou, void* saved, void* ws,
                        size_t ws_bytes, hipStream_t stream) {
    kla_status st = check_desc(desc);
    if (st != KLA_OK) return st;
    if (ou && (!a.ou_a || !a.ou_p || !a.ou_d)) return KLA_ERR_NULL;
    // with T == 0 the per-token tensors are empty and may be NULL
    if (desc->T > 0 && (!a.q || !a.k || !a.v || (!ou && (!a.a || !a.p)) || !a.r || !a.y)) return KLA_ERR_NULL;
    if (!all_aligned(a.q, a.k, a.v, a.a, a.p, a.r, (const void*)a.lam0, (const void*)a.eta0, a.y, (void*)a.yvar,
                     (void*)a.lamT, (void*)a.etaT, saved, ws, (const void*)a.ou_a, (const void*)a.ou_p,
                     (const void*)a.ou_d))
        return KLA_ERR_ALIGN;
    if (!ws || ws_bytes < kla_forward_workspace(desc)) return KLA_ERR_WORKSPACE;
    const kla::Shape s = shape_of(desc);
    const bool check = check_mode();
    kla::FwdArgs fa = a;
    if (check) {
        st = validate(s, s.T, a.q, a.k, a.v, a.a, a.p, a.r, a.lam0, a.eta0, ws, stream, a.ou_a, a.ou_p, a.ou_d);
        if (st != KLA_OK) return st;
        fa.range_flag = static_cast<int*>(ws);
    }
    hipError_t e;
    // without a saved context any forward kernel may run; with one, the kernel whose
    // layout the backward reads (saves_chunked)
    const bool chunked = saved ? saves_chunked(s) : kla::chunked_supported(s);
    const bool c64 = kla::c64_supported(s);
    if (!saved && !ou && kla::forward_segments(s) > 1)
        e = kla::launch_forward_segmented(s, fa, static_cast<char*>(ws) + kAlign, stream);
    else if (chunked)
        e = kla::launch_forward_chunked(s, fa, saved, stream);
    else if (c64)
        e = kla::launch_forward_c64(s, fa, saved, stream);
    else
        e = kla::launch_forward_recurrent(s, fa, saved, stream);
    if (e != hipSuccess) return KLA_ERR_HIP;
    return check && (chunked || c64) ? range_status(ws, stream) : KLA_OK;
}

int ou_parts(const kla::Shape& s) {
    return kla::chunked_bwd_supported(s) ? kla::chunked_ou_parts(s) : kla::recurrent_ou_parts(s);
}

// bytes per OU part element: fp32 from the chunked backward, the arithmetic type from the
// token-recurrent one
size_t ou_part_bytes(const kla::Shape& s) {
    return kla::chunked_bwd_supported(s) ? sizeof(float) : kla::recurrent_ou_part_bytes(s);
}

// The backward behind both gate forms.  With OU parameters the gate gradients
// are summed into parts at the end of the workspace and reduced into the
// parameter gradients da, dp, dd.
kla_status backward_impl(const kla_desc* desc, kla::BwdArgs a, bool ou, const void* saved, float* da, float* dp,
                         float* dd, void* ws, size_t ws_bytes, hipStream_t stream) {
    kla_status st = check_desc(desc);
    if (st != KLA_OK) return st;
    if (ou && (!a.ou_a || !a.ou_p || !a.ou_d || !da || !dp || !dd)) return KLA_ERR_NULL;
    if (desc->T > 0 && (!a.q || !a.k || !a.v || (!ou && (!a.a || !a.p)) || !a.r || !a.dy || !a.dq || !a.dk ||
                        !a.dv || (!ou && (!a.da || !a.dp)) || !a.dr))
        return KLA_ERR_NULL;
    if (!all_aligned(a.q, a.k, a.v, a.a, a.p, a.r, (const void*)a.lam0, (const void*)a.eta0, saved, a.dy,
                     (const void*)a.dyvar, (const void*)a.dlamT, (const void*)a.detaT, a.dq, a.dk, a.dv, a.da, a.dp, a.dr,
                     (void*)a.dlam0, (void*)a.deta0, ws, (const void*)a.ou_a, (const void*)a.ou_p,
                     (const void*)a.ou_d, (void*)da, (void*)dp, (void*)dd))
        return KLA_ERR_ALIGN;
    const size_t need = ou ? kla_backward_ou_workspace(desc, saved != nullptr)
                           : kla_backward_workspace(desc, saved != nullptr);
    if (!ws || ws_bytes < need) return KLA_ERR_WORKSPACE;
    const kla::Shape s = shape_of(desc);
    const bool check = check_mode();
    if (check) {
        st = validate(s, s.T, a.q, a.k, a.v, a.a, a.p, a.r, a.lam0, a.eta0, ws, stream, a.ou_a, a.ou_p, a.ou_d);
        if (st != KLA_OK) return st;
        a.range_flag = static_cast<int*>(ws);
    }
    if (ou) a.ou_part = static_cast<char*>(ws) + kla_backward_workspace(desc, saved != nullptr);
    char* work = static_cast<char*>(ws) + kAlign;
    hipError_t e;
    if (kla::chunked_bwd_supported(s)) {
        if (!saved) {
            char* ctx = work + round_up(kla::chunked_bwd_workspace(s));
            void* yscratch = ctx + round_up(kla::chunked_saved_bytes(s));
            kla::FwdArgs f{a.q, a.k, a.v, a.a, a.p, a.r, a.lam0, a.eta0, yscratch, nullptr, nullptr, nullptr,
                           a.ou_a, a.ou_p, a.ou_d, a.range_flag};
            e = kla::launch_forward_chunked(s, f, ctx, stream);
            if (e != hipSuccess) return KLA_ERR_HIP;
            saved = ctx;
        }
        e = kla::launch_backward_chunked(s, a, saved, work, stream);
    } else if (kla::c64_supported(s)) {
        if (!saved) {
            char* ctx = work;
            void* yscratch = ctx + round_up(kla::c64_saved_bytes(s));
            kla::FwdArgs f{a.q, a.k, a.v, a.a, a.p, a.r, a.lam0, a.eta0, yscratch, nullptr, nullptr, nullptr,
                           a.ou_a, a.ou_p, a.ou_d, a.range_flag};
            e = kla::launch_forward_c64(s, f, ctx, stream);
            if (e != hipSuccess) return KLA_ERR_HIP;
            saved = ctx;
        }
        e = kla::launch_backward_c64(s, a, saved, stream);
    } else {
        if (!saved) {   // the same forward kernel fills the context, so both ways agree bit for bit
            char* ctx = work + round_up(kla::backward_recurrent_workspace(s));
            void* yscratch = ctx + round_up(kla::recurrent_saved_bytes(s));
            kla::FwdArgs f{a.q, a.k, a.v, a.a, a.p, a.r, a.lam0, a.eta0, yscratch, nullptr, nullptr, nullptr,
                           a.ou_a, a.ou_p, a.ou_d};
            e = kla::launch_forward_recurrent(s, f, ctx, stream);
            if (e != hipSuccess) return KLA_ERR_HIP;
            saved = ctx;
        }
        e = kla::launch_backward_recurrent(s, a, saved, work, stream);
    }
    if (e == hipSuccess && ou)
        e = kla::launch_ou_param_grads(s.H, s.dk, ou_parts(s), a.ou_part, ou_part_bytes(s) == sizeof(double), a.ou_a,
                                       a.ou_p, a.ou_d, da, dp, dd, stream);
    if (e != hipSuccess) return KLA_ERR_HIP;
    return check && (kla::chunked_bwd_supported(s) || kla::c64_supported(s)) ? range_status(ws, stream) : KLA_OK;
}

kla_status decode_impl(int32_t S, int32_t H, int32_t dk, int32_t dv, int32_t dtype, const kla::DecodeArgs& a,
                       bool ou, hipStream_t stream) {
    kla_desc d{S, 1, H, dk, dv, dtype};
    kla_status st = check_desc(&d);
    if (st != KLA_OK) return st;
    if (!a.q || !a.k || !a.v || (!ou && (!a.a || !a.p)) || !a.r || !a.lam || !a.eta || !a.y) return KLA_ERR_NULL;
    if (ou && (!a.ou_a || !a.ou_p || !a.ou_d)) return KLA_ERR_NULL;
    if (!all_aligned(a.q, a.k, a.v, a.a, a.p, a.r, (void*)a.lam, (void*)a.eta, a.y, (void*)a.yvar,
                     (const void*)a.ou_a, (const void*)a.ou_p, (const void*)a.ou_d))
        return KLA_ERR_ALIGN;
    return kla::launch_decode_step(shape_of(&d), a, stream) == hipSuccess ? KLA_OK : KLA_ERR_HIP;
}

}  // namespace

extern "C" {

kla_status kla_forward(const kla_desc* desc, const void* q, const void* k, const void* v, const void* abar,
                       const void* pbar, const void* r, const float* lam0, const float* eta0, void* y,
                       float* yvar, float* lamT, float* etaT, void* saved, void* ws, size_t ws_bytes,
                       hipStream_t stream) {
    return forward_impl(desc, kla::FwdArgs{q, k, v, abar, pbar, r, lam0, eta0, y, yvar, lamT, etaT}, false, saved,
                        ws, ws_bytes, stream);
}

kla_status kla_forward_ou(const kla_desc* desc, const void* q, const void* k, const void* v, const float* a,
                          const float* p, const float* delta, const void* r, const float* lam0, const float* eta0,
                          void* y, float* yvar, float* lamT, float* etaT, void* saved, void* ws, size_t ws_bytes,
                          hipStream_t stream) {
    return forward_impl(desc,
                        kla::FwdArgs{q, k, v, nullptr, nullptr, r, lam0, eta0, y, yvar, lamT, etaT, a, p, delta},
                        true, saved, ws, ws_bytes, stream);
}

kla_status kla_backward(const kla_desc* desc, const void* q, const void* k, const void* v, const void* abar,
                        const void* pbar, const void* r, const float* lam0, const float* eta0, const void* saved,
                        const void* dy, const float* dyvar, const float* dlamT, const float* detaT, void* dq,
                        void* dk, void* dv, void* dabar, void* dpbar, void* dr, float* dlam0, float* deta0,
                        void* ws, size_t ws_bytes, hipStream_t stream) {
    kla::BwdArgs a{q,  k,  v,  abar,  pbar,  r,  lam0, eta0,  dy, dlamT,
                   detaT, dq, dk, dv, dabar, dpbar, dr, dlam0, deta0};
    a.dyvar = dyvar;
    return backward_impl(desc, a, false, saved, nullptr, nullptr, nullptr, ws, ws_bytes, stream);
}

size_t kla_backward_ou_workspace(const kla_desc* desc, int with_saved) {
    if (check_desc(desc) != KLA_OK) return 0;
    const kla::Shape s = shape_of(desc);
    return kla_backward_workspace(desc, with_saved) + round_up((size_t)2 * ou_parts(s) * s.H * s.dk * ou_part_bytes(s));
}

kla_status kla_backward_ou(const kla_desc* desc, const void* q, const void* k, const void* v, const float* a,
                           const float* p, const float* delta, const void* r, const float* lam0, const float* eta0,
                           const void* saved, const void* dy, const float* dyvar, const float* dlamT,
                           const float* detaT, void* dq, void* dk, void* dv, float* da, float* dp, float* ddelta,
                           void* dr, float* dlam0, float* deta0, void* ws, size_t ws_bytes, hipStream_t stream) {
    kla::BwdArgs g{q,  k,  v,       nullptr, nullptr, r,  lam0,  eta0,  dy, dlamT,
                   detaT, dq, dk, dv, nullptr, nullptr, dr, dlam0, deta0};
    g.ou_a = a;
    g.ou_p = p;
    g.ou_d = delta;
    g.dyvar = dyvar;
    return backward_impl(desc, g, true, saved, da, dp, ddelta, ws, ws_bytes, stream);
}

size_t kla_saved_pc_bytes(const kla_desc* desc) {
    if (check_desc(desc) != KLA_OK) return 0;
    return kla::pc_saved_bytes(shape_of(desc));
}

size_t kla_backward_pc_workspace(const kla_desc* desc, int with_saved) {
    if (check_desc(desc) != KLA_OK) return 0;
    const kla::Shape s = shape_of(desc);
    size_t bytes = kAlign + round_up(kla::pc_bwd_workspace(s));
    if (!with_saved) {  // the checkpoints are recomputed: saved context plus a scratch output
        const size_t elt = s.bf16 ? 2 : 4;
        bytes += round_up(kla::pc_saved_bytes(s)) + round_up((size_t)s.B * s.T * s.H * s.dv * elt);
    }
    return bytes;
}

kla_status kla_forward_pc(const kla_desc* desc, const void* q, const void* k, const void* v, const void* abar,
                          const void* pbar, const void* r, const float* lam0, const float* eta0, void* y,
                          float* yvar, float* lamT, float* etaT, void* saved, void* ws, size_t ws_bytes,
                          hipStream_t stream) {
    kla_status st = check_desc(desc);
    if (st != KLA_OK) return st;
    if (desc->T > 0 && (!q || !k || !v || !abar || !pbar || !r || !y)) return KLA_ERR_NULL;
    if (!all_aligned(q, k, v, abar, pbar, r, (const void*)lam0, (const void*)eta0, y, (void*)yvar, (void*)lamT,
                     (void*)etaT, saved, ws))
        return KLA_ERR_ALIGN;
    if (!ws || ws_bytes < kla_forward_workspace(desc)) return KLA_ERR_WORKSPACE;
    const kla::Shape s = shape_of(desc);
    if (check_mode()) {
        st = validate(s, s.T, q, k, v, abar, pbar, r, lam0, eta0, ws, stream, nullptr, nullptr, nullptr, true);
        if (st != KLA_OK) return st;
    }
    const kla::FwdArgs a{q, k, v, abar, pbar, r, lam0, eta0, y, yvar, lamT, etaT};
    return kla::launch_forward_pc(s, a, saved, stream) == hipSuccess ? KLA_OK : KLA_ERR_HIP;
}

kla_status kla_backward_pc(const kla_desc* desc, const void* q, const void* k, const void* v, const void* abar,
                           const void* pbar, const void* r, const float* lam0, const float* eta0, const void* saved,
                           const void* dy, const float* dyvar, const float* dlamT, const float* detaT, void* dq,
                           void* dk, void* dv, void* dabar, void* dpbar, void* dr, float* dlam0, float* deta0,
                           void* ws, size_t ws_bytes, hipStream_t stream) {
    kla_status st = check_desc(desc);
    if (st != KLA_OK) return st;
    if (desc->T > 0 && (!q || !k || !v || !abar || !pbar || !r || !dy || !dq || !dk || !dv || !dabar || !dpbar ||
                        !dr))
        return KLA_ERR_NULL;
    if (!all_aligned(q, k, v, abar, pbar, r, (const void*)lam0, (const void*)eta0, saved, dy, (const void*)dyvar,
                     (const void*)dlamT, (const void*)detaT, dq, dk, dv, dabar, dpbar, dr, (void*)dlam0,
                     (void*)deta0, ws))
        return KLA_ERR_ALIGN;
    if (!ws || ws_bytes < kla_backward_pc_workspace(desc, saved != nullptr)) return KLA_ERR_WORKSPACE;
    const kla::Shape s = shape_of(desc);
    if (check_mode()) {
        st = validate(s, s.T, q, k, v, abar, pbar, r, lam0, eta0, ws, stream, nullptr, nullptr, nullptr, true);
        if (st != KLA_OK) return st;
    }
    char* work = static_cast<char*>(ws) + kAlign;
    float* kpart = reinterpret_cast<float*>(work);
    if (!saved) {
        char* ctx = work + round_up(kla::pc_bwd_workspace(s));
        void* yscratch = ctx + round_up(kla::pc_saved_bytes(s));
        const kla::FwdArgs f{q, k, v, abar, pbar, r, lam0, eta0, yscratch, nullptr, nullptr, nullptr};
        if (kla::launch_forward_pc(s, f, ctx, stream) != hipSuccess) return KLA_ERR_HIP;
        saved = ctx;
    }
    kla::BwdArgs a{q,  k,  v,  abar,  pbar,  r,  lam0, eta0,  dy, dlamT,
                   detaT, dq, dk, dv, dabar, dpbar, dr, dlam0, deta0};
    a.dyvar = dyvar;
    return kla::launch_backward_pc(s, a, saved, kpart, stream) == hipSuccess ? KLA_OK
                                                                                                      : KLA_ERR_HIP;
}

size_t kla_backward_pc_ou_workspace(const kla_desc* desc, int with_saved) {
    if (check_desc(desc) != KLA_OK) return 0;
    return kla_backward_pc_workspace(desc, with_saved) + round_up(kla::pc_ou_part_bytes(shape_of(desc)));
}

kla_status kla_forward_pc_ou(const kla_desc* desc, const void* q, const void* k, const void* v, const float* a,
                             const float* p, const float* delta, const void* r, const float* lam0, const float* eta0,
                             void* y, float* yvar, float* lamT, float* etaT, void* saved, void* ws, size_t ws_bytes,
                             hipStream_t stream) {
    kla_status st = check_desc(desc);
    if (st != KLA_OK) return st;
    if (!a || !p || !delta) return KLA_ERR_NULL;
    if (desc->T > 0 && (!q || !k || !v || !r || !y)) return KLA_ERR_NULL;
    if (!all_aligned(q, k, v, (const void*)a, (const void*)p, (const void*)delta, r, (const void*)lam0,
                     (const void*)eta0, y, (void*)yvar, (void*)lamT, (void*)etaT, saved, ws))
        return KLA_ERR_ALIGN;
    if (!ws || ws_bytes < kla_forward_workspace(desc)) return KLA_ERR_WORKSPACE;
    const kla::Shape s = shape_of(desc);
    if (check_mode()) {
        st = validate(s, s.T, q, k, v, nullptr, nullptr, r, lam0, eta0, ws, stream, a, p, delta, true);
        if (st != KLA_OK) return st;
    }
    const kla::FwdArgs f{q, k, v, nullptr, nullptr, r, lam0, eta0, y, yvar, lamT, etaT, a, p, delta};
    return kla::launch_forward_pc(s, f, saved, stream) == hipSuccess ? KLA_OK : KLA_ERR_HIP;
}

kla_status kla_backward_pc_ou(const kla_desc* desc, const void* q, const void* k, const void* v, const float* a,
                              const float* p, const float* delta, const void* r, const float* lam0,
                              const float* eta0, const void* saved, const void* dy, const float* dyvar,
                              const float* dlamT, const float* detaT, void* dq, void* dk, void* dv, float* da,
                              float* dp, float* ddelta, void* dr, float* dlam0, float* deta0, void* ws,
                              size_t ws_bytes, hipStream_t stream) {
    kla_status st = check_desc(desc);
    if (st != KLA_OK) return st;
    if (!a || !p || !delta || !da || !dp || !ddelta) return KLA_ERR_NULL;
    if (desc->T > 0 && (!q || !k || !v || !r || !dy || !dq || !dk || !dv || !dr)) return KLA_ERR_NULL;
    if (!all_aligned(q, k, v, (const void*)a, (const void*)p, (const void*)delta, r, (const void*)lam0,
                     (const void*)eta0, saved, dy, (const void*)dyvar, (const void*)dlamT, (const void*)detaT, dq,
                     dk, dv, (void*)da, (void*)dp, (void*)ddelta, dr, (void*)dlam0, (void*)deta0, ws))
        return KLA_ERR_ALIGN;
    if (!ws || ws_bytes < kla_backward_pc_ou_workspace(desc, saved != nullptr)) return KLA_ERR_WORKSPACE;
    const kla::Shape s = shape_of(desc);
    if (check_mode()) {
        st = validate(s, s.T, q, k, v, nullptr, nullptr, r, lam0, eta0, ws, stream, a, p, delta, true);
        if (st != KLA_OK) return st;
    }
    char* work = static_cast<char*>(ws) + kAlign;
    float* kpart = reinterpret_cast<float*>(work);
    void* ou_part = static_cast<char*>(ws) + kla_backward_pc_workspace(desc, saved != nullptr);
    if (!saved) {
        char* ctx = work + round_up(kla::pc_bwd_workspace(s));
        void* yscratch = ctx + round_up(kla::pc_saved_bytes(s));
        const kla::FwdArgs f{q, k, v, nullptr, nullptr, r, lam0, eta0, yscratch, nullptr, nullptr, nullptr, a, p,
                             delta};
        if (kla::launch_forward_pc(s, f, ctx, stream) != hipSuccess) return KLA_ERR_HIP;
        saved = ctx;
    }
    kla::BwdArgs g{q,  k,  v,  nullptr, nullptr, r,  lam0, eta0,  dy, dlamT,
                   detaT, dq, dk, dv, nullptr, nullptr, dr, dlam0, deta0};
    g.ou_a = a;
    g.ou_p = p;
    g.ou_d = delta;
    g.ou_part = ou_part;
    g.dyvar = dyvar;
    if (kla::launch_backward_pc(s, g, saved, kpart, stream) != hipSuccess) return KLA_ERR_HIP;
    // the parameters are per (head, key slot, value channel): H dk dv of them, one part per batch row
    return kla::launch_ou_param_grads(s.H, s.dk * s.dv, s.B, ou_part, !s.bf16, a, p, delta, da, dp, ddelta,
                                      stream) == hipSuccess
               ? KLA_OK
               : KLA_ERR_HIP;
}

kla_status kla_decode_step_pc_ou(int32_t S, int32_t H, int32_t dk, int32_t dv, int32_t dtype, const void* q,
                                 const void* k, const void* v, const float* a, const float* p, const float* delta,
                                 const void* r, float* lam, float* eta, void* y, float* yvar, hipStream_t stream) {
    kla_desc d{S, 1, H, dk, dv, dtype};
    kla_status st = check_desc(&d);
    if (st != KLA_OK) return st;
    if (!q || !k || !v || !a || !p || !delta || !r || !lam || !eta || !y) return KLA_ERR_NULL;
    if (!all_aligned(q, k, v, (const void*)a, (const void*)p, (const void*)delta, r, (void*)lam, (void*)eta, y,
                     (void*)yvar))
        return KLA_ERR_ALIGN;
    const kla::DecodeArgs g{q, k, v, nullptr, nullptr, r, lam, eta, y, yvar, a, p, delta};
    return kla::launch_decode_pc(shape_of(&d), g, stream) == hipSuccess ? KLA_OK : KLA_ERR_HIP;
}

kla_status kla_decode_step_pc(int32_t S, int32_t H, int32_t dk, int32_t dv, int32_t dtype, const void* q,
                              const void* k, const void* v, const void* abar, const void* pbar, const void* r,
                              float* lam, float* eta, void* y, float* yvar, hipStream_t stream) {
    kla_desc d{S, 1, H, dk, dv, dtype};
    kla_status st = check_desc(&d);
    if (st != KLA_OK) return st;
    if (!q || !k || !v || !abar || !pbar || !r || !lam || !eta || !y) return KLA_ERR_NULL;
    if (!all_aligned(q, k, v, abar, pbar, r, (void*)lam, (void*)eta, y, (void*)yvar)) return KLA_ERR_ALIGN;
    const kla::DecodeArgs a{q, k, v, abar, pbar, r, lam, eta, y, yvar};
    return kla::launch_decode_pc(shape_of(&d), a, stream) == hipSuccess ? KLA_OK : KLA_ERR_HIP;
}

kla_status kla_decode_step(int32_t S, int32_t H, int32_t dk, int32_t dv, int32_t dtype, const void* q,
                           const void* k, const void* v, const void* abar, const void* pbar, const void* r,
                           float* lam, float* eta, void* y, float* yvar, hipStream_t stream) {
    return decode_impl(S, H, dk, dv, dtype, kla::DecodeArgs{q, k, v, abar, pbar, r, lam, eta, y, yvar}, false,
                       stream);
}

kla_status kla_decode_step_ou(int32_t S, int32_t H, int32_t dk, int32_t dv, int32_t dtype, const void* q,
                              const void* k, const void* v, const float* a, const float* p, const float* delta,
                              const void* r, float* lam, float* eta, void* y, float* yvar, hipStream_t stream) {
    return decode_impl(S, H, dk, dv, dtype,
                       kla::DecodeArgs{q, k, v, nullptr, nullptr, r, lam, eta, y, yvar, a, p, delta}, true, stream);
}

// ---------------------------------------------------------------- block scaffolding

size_t kla_conv_silu_workspace(int32_t B, int32_t T, int32_t C) {
    if (B < 1 || T < 0 || C < 1) return 0;
    return kla::conv_parts_bytes(B, T, C);
}

kla_status kla_conv_silu_forward(int32_t B, int32_t T, int32_t C, int32_t dtype, const void* x, const float* w,
                                 const float* bias, void* u, hipStream_t stream) {
    if (dtype != KLA_F32 && dtype != KLA_BF16) return KLA_ERR_DTYPE;
    if (B < 1 || T < 0 || C < 1 || C % kla::block_vec(dtype == KLA_BF16) != 0) return KLA_ERR_SHAPE;
    if (!w || (T > 0 && (!x || !u))) return KLA_ERR_NULL;
    if (!all_aligned(x, (const void*)w, (const void*)bias, u)) return KLA_ERR_ALIGN;
    return kla::launch_conv_fwd(B, T, C, dtype == KLA_BF16, x, w, bias, u, stream) == hipSuccess ? KLA_OK
                                                                                                 : KLA_ERR_HIP;
}

kla_status kla_conv_silu_backward(int32_t B, int32_t T, int32_t C, int32_t dtype, const void* x, const float* w,
                                  const float* bias, const void* du, void* dx, float* dw, float* dbias, void* ws,
                                  size_t ws_bytes, hipStream_t stream) {
    if (dtype != KLA_F32 && dtype != KLA_BF16) return KLA_ERR_DTYPE;
    if (B < 1 || T < 0 || C < 1 || C % kla::block_vec(dtype == KLA_BF16) != 0) return KLA_ERR_SHAPE;
    if (!w || !dw || (T > 0 && (!x || !du || !dx))) return KLA_ERR_NULL;
    if (!all_aligned(x, (const void*)w, (const void*)bias, du, dx, (void*)dw, (void*)dbias, ws)) return KLA_ERR_ALIGN;
    if (!ws || ws_bytes < kla_conv_silu_workspace(B, T, C)) return KLA_ERR_WORKSPACE;
    return kla::launch_conv_bwd(B, T, C, dtype == KLA_BF16, x, w, bias, du, dx, dw, dbias, static_cast<float*>(ws),
                                stream) == hipSuccess
               ? KLA_OK
               : KLA_ERR_HIP;
}

size_t kla_qk_norm_workspace(int32_t n) { return width_ok(n) ? kla::norm_parts_bytes(n) : 0; }

kla_status kla_qk_norm_forward(int64_t rows, int32_t n, int32_t dtype, const void* x, const float* w, float eps,
                               void* out, float* rstd, hipStream_t stream) {
    if (dtype != KLA_F32 && dtype != KLA_BF16) return KLA_ERR_DTYPE;
    if (rows < 0 || !width_ok(n) || !(eps >= 0.f)) return KLA_ERR_SHAPE;
    if (!w || (rows > 0 && (!x || !out))) return KLA_ERR_NULL;
    if (!all_aligned(x, (const void*)w, out, (void*)rstd)) return KLA_ERR_ALIGN;
    return kla::launch_norm_fwd((size_t)rows, n, dtype == KLA_BF16, x, w, eps, out, rstd, stream) == hipSuccess
               ? KLA_OK
               : KLA_ERR_HIP;
}

kla_status kla_qk_norm_backward(int64_t rows, int32_t n, int32_t dtype, const void* x, const float* w,
                                const float* rstd, const void* dout, void* dx, float* dw, void* ws, size_t ws_bytes,
                                hipStream_t stream) {
    if (dtype != KLA_F32 && dtype != KLA_BF16) return KLA_ERR_DTYPE;
    if (rows < 0 || !width_ok(n)) return KLA_ERR_SHAPE;
    if (!w || !dw || (rows > 0 && (!x || !rstd || !dout || !dx))) return KLA_ERR_NULL;
    if (!all_aligned(x, (const void*)w, (const void*)rstd, dout, dx, (void*)dw, ws)) return KLA_ERR_ALIGN;
    if (!ws || ws_bytes < kla_qk_norm_workspace(n)) return KLA_ERR_WORKSPACE;
    return kla::launch_norm_bwd((size_t)rows, n, dtype == KLA_BF16, x, w, rstd, dout, dx, dw, static_cast<float*>(ws),
                                stream) == hipSuccess
               ? KLA_OK
               : KLA_ERR_HIP;
}

kla_status kla_gate_forward(int64_t n, int32_t dtype, const void* y, const void* z, void* out, hipStream_t stream) {
    if (dtype != KLA_F32 && dtype != KLA_BF16) return KLA_ERR_DTYPE;
    if (n < 0 || n % kla::block_vec(dtype == KLA_BF16) != 0) return KLA_ERR_SHAPE;
    if (n > 0 && (!y || !z || !out)) return KLA_ERR_NULL;
    if (!all_aligned(y, z, out)) return KLA_ERR_ALIGN;
    return kla::launch_gate_fwd((size_t)n, dtype == KLA_BF16, y, z, out, stream) == hipSuccess ? KLA_OK : KLA_ERR_HIP;
}

kla_status kla_gate_backward(int64_t n, int32_t dtype, const void* y, const void* z, const void* dout, void* dy,
                             void* dz, hipStream_t stream) {
    if (dtype != KLA_F32 && dtype != KLA_BF16) return KLA_ERR_DTYPE;
    if (n < 0 || n % kla::block_vec(dtype == KLA_BF16) != 0) return KLA_ERR_SHAPE;
    if (n > 0 && (!y || !z || !dout || !dy || !dz)) return KLA_ERR_NULL;
    if (!all_aligned(y, z, dout, dy, dz)) return KLA_ERR_ALIGN;
    return kla::launch_gate_bwd((size_t)n, dtype == KLA_BF16, y, z, dout, dy, dz, stream) == hipSuccess ? KLA_OK
                                                                                                      : KLA_ERR_HIP;
}

// ---------------------------------------------------------------- Monte Carlo readout

namespace {
kla_status mc_shape(int32_t S, int32_t B, int32_t T, int32_t H, int32_t dv, int32_t dtype) {
    if (dtype != KLA_F32 && dtype != KLA_BF16) return KLA_ERR_DTYPE;
    if (S < 1 || B < 1 || T < 0 || H < 1 || !width_ok(dv)) return KLA_ERR_SHAPE;
    if ((double)S * B * T * H * dv > 9.0e18) return KLA_ERR_SHAPE;
    return KLA_OK;
}
}  // namespace

kla_status kla_mc_sample(int32_t S, int32_t B, int32_t T, int32_t H, int32_t dv, int32_t dtype, uint64_t seed,
                         const void* ymu, const float* yvar, void* ys, hipStream_t stream) {
    const kla_status st = mc_shape(S, B, T, H, dv, dtype);
    if (st != KLA_OK) return st;
    if (T > 0 && (!ymu || !yvar || !ys)) return KLA_ERR_NULL;
    if (!all_aligned(ymu, (const void*)yvar, ys)) return KLA_ERR_ALIGN;
    return kla::launch_mc_sample(S, (size_t)B * T * H, dv, dtype == KLA_BF16, seed, ymu, yvar, ys, stream) ==
                   hipSuccess
               ? KLA_OK
               : KLA_ERR_HIP;
}

kla_status kla_mc_sample_backward(int32_t S, int32_t B, int32_t T, int32_t H, int32_t dv, int32_t dtype,
                                  uint64_t seed, const float* yvar, const void* dys, void* dymu, float* dyvar,
                                  hipStream_t stream) {
    const kla_status st = mc_shape(S, B, T, H, dv, dtype);
    if (st != KLA_OK) return st;
    if (T > 0 && (!yvar || !dys || !dymu || !dyvar)) return KLA_ERR_NULL;
    if (!all_aligned((const void*)yvar, dys, dymu, (void*)dyvar)) return KLA_ERR_ALIGN;
    return kla::launch_mc_sample_bwd(S, (size_t)B * T * H, dv, dtype == KLA_BF16, seed, yvar, dys, dymu, dyvar,
                                     stream) == hipSuccess
               ? KLA_OK
               : KLA_ERR_HIP;
}

kla_status kla_mc_nll(int32_t S, int64_t n, const float* logp, float* nll, hipStream_t stream) {
    if (S < 1 || n < 0) return KLA_ERR_SHAPE;
    if (n > 0 && (!logp || !nll)) return KLA_ERR_NULL;
    if (!all_aligned((const void*)logp, (void*)nll)) return KLA_ERR_ALIGN;
    return kla::launch_mc_nll(S, (size_t)n, logp, nll, stream) == hipSuccess ? KLA_OK : KLA_ERR_HIP;
}

kla_status kla_mc_nll_backward(int32_t S, int64_t n, const float* logp, const float* dnll, float* dlogp,
                               hipStream_t stream) {
    if (S < 1 || n < 0) return KLA_ERR_SHAPE;
    if (n > 0 && (!logp || !dnll || !dlogp)) return KLA_ERR_NULL;
    if (!all_aligned((const void*)logp, (const void*)dnll, (void*)dlogp)) return KLA_ERR_ALIGN;
    return kla::launch_mc_nll_bwd(S, (size_t)n, logp, dnll, dlogp, stream) == hipSuccess ? KLA_OK : KLA_ERR_HIP;
}

const char* kla_status_string(kla_status s) {
    switch (s) {
        case KLA_OK: return "KLA_OK";
        case KLA_ERR_NULL: return "KLA_ERR_NULL: a required pointer is NULL";
        case KLA_ERR_SHAPE: return "KLA_ERR_SHAPE: unsupported or inconsistent sizes";
        case KLA_ERR_DTYPE: return "KLA_ERR_DTYPE: unknown dtype";
        case KLA_ERR_ALIGN: return "KLA_ERR_ALIGN: a pointer is not 16-byte aligned";
        case KLA_ERR_WORKSPACE: return "KLA_ERR_WORKSPACE: workspace missing or too small";
        case KLA_ERR_NUMERIC: return "KLA_ERR_NUMERIC: an input lies outside the filter's domain";
        case KLA_ERR_HIP: return "KLA_ERR_HIP: a HIP launch or runtime call failed";
        case KLA_ERR_RANGE:
            return "KLA_ERR_RANGE: the gate products inside a 32-token chunk left fp32 range";
    }
    return "KLA_ERR_UNKNOWN";
}

}  // extern "C"
