// Internal launcher interface between the C ABI (kla_api.cpp) and the kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace kla {

struct Shape {
    int B, T, H, dk, dv;
    int bf16;  // 0: fp32 storage, 1: bf16 storage
};

// Gates: per token (a, p: abar, pbar [B, T, H, dk] in the storage type) or, when
// ou_a is set, time-invariant from the OU parameters ou_a, ou_p, ou_d [H, dk] fp32
// (a and p unused).
struct FwdArgs {
    const void *q, *k, *v, *a, *p, *r;
    const float *lam0, *eta0;
    void* y;
    float *yvar, *lamT, *etaT;
    const float *ou_a = nullptr, *ou_p = nullptr, *ou_d = nullptr;
    // chunked path: set to 1 when a chunk's walk leaves fp32 range (Qp or Kn not finite), or none
    int* range_flag = nullptr;
};

struct BwdArgs {
    const void *q, *k, *v, *a, *p, *r;
    const float *lam0, *eta0;
    const void* dy;
    const float *dlamT, *detaT;
    void *dq, *dk, *dv, *da, *dp, *dr;
    float *dlam0, *deta0;
    const float *ou_a = nullptr, *ou_p = nullptr, *ou_d = nullptr;
    // OU gates: per-part sums over tokens of the abar and pbar gradients,
    // [2][nparts][H][dk], fp32 from the chunked path, the arithmetic type from the
    // token-recurrent one (da, dp unused)
    void* ou_part = nullptr;
    const float* dyvar = nullptr;   // upstream gradient of yvar [B, T, H] fp32, or none
    int* range_flag = nullptr;        // as in FwdArgs
};

struct DecodeArgs {
    const void *q, *k, *v, *a, *p, *r;
    float *lam, *eta;
    void* y;
    float* yvar;
    const float *ou_a = nullptr, *ou_p = nullptr, *ou_d = nullptr;
};

// Token-recurrent kernels.  They compute in fp64 for fp32 inputs and in fp32 for
// bf16 inputs (the arithmetic type).  Their saved context (recurrent_saved_bytes(s)
// bytes, in the arithmetic type) is the precision after every token, lam_t
// [B, T, H, dk], followed by the information state before every 64th token,
// [B, H, ceil(T / 64), dk, dv]: optional for the forward, required by the backward.
size_t recurrent_saved_bytes(const Shape& s);
hipError_t launch_forward_recurrent(const Shape& s, const FwdArgs& a, void* saved, hipStream_t st);
size_t backward_recurrent_workspace(const Shape& s);
hipError_t launch_backward_recurrent(const Shape& s, const BwdArgs& a, const void* saved, void* ws,
                                     hipStream_t st);
// bytes per element of the recurrent backward's OU parts (the arithmetic type)
size_t recurrent_ou_part_bytes(const Shape& s);
hipError_t launch_decode_step(const Shape& s, const DecodeArgs& a, hipStream_t st);

// Chunked fp64 path for fp32 storage with dk, dv in {16, 32}: the chunk form on fp64
// MFMA.  Its saved context (c64_saved_bytes, fp64) is lam at every 32-token chunk
// start [B*H][nchunk][dk], then the information state at every chunk start and after
// the last token [B*H][nchunk+1][dk][dv]; the backward needs no other workspace and
// leaves the OU parts as the token-recurrent one does (per batch row, fp64).
bool c64_supported(const Shape& s);
size_t c64_saved_bytes(const Shape& s);
hipError_t launch_forward_c64(const Shape& s, const FwdArgs& a, void* saved, hipStream_t st);
hipError_t launch_backward_c64(const Shape& s, const BwdArgs& a, const void* saved, hipStream_t st);

// Chunked MFMA path (bf16 storage, dk >= 32).
bool chunked_supported(const Shape& s);
size_t chunked_saved_bytes(const Shape& s);
hipError_t launch_forward_chunked(const Shape& s, const FwdArgs& a, void* saved, hipStream_t st);
bool chunked_bwd_supported(const Shape& s);
size_t chunked_bwd_workspace(const Shape& s);
hipError_t launch_backward_chunked(const Shape& s, const BwdArgs& a, const void* saved, void* ws, hipStream_t st);
// Segment-parallel chunked forward for few long sequences (no saved context): the number of
// segments (1: not used), its workspace and launch.
int forward_segments(const Shape& s);
size_t forward_segmented_workspace(const Shape& s);
hipError_t launch_forward_segmented(const Shape& s, const FwdArgs& a, void* ws, hipStream_t st);
// value side of the chunked backward (dv, deta0); saved_lam: lam at every 32-token chunk start
hipError_t launch_backward_dv(const Shape& s, const BwdArgs& a, const float* saved_lam, hipStream_t st);
// token-sum parts of the OU gate gradients that the chunked / recurrent backward leave
int chunked_ou_parts(const Shape& s);
int recurrent_ou_parts(const Shape& s);

// Per-channel precision (r [B, T, H, dv], beliefs [B, H, dk, dv]): elementwise scan and decode.
// ck: NULL or pc_saved_bytes of belief checkpoints for launch_backward_pc; kpart: pc_bwd_workspace bytes
// The checkpoints are in the arithmetic type (fp64 for fp32 inputs, fp32 for bf16).
hipError_t launch_forward_pc(const Shape& s, const FwdArgs& a, void* ck, hipStream_t st);
size_t pc_saved_bytes(const Shape& s);
size_t pc_bwd_workspace(const Shape& s);
// OU parameters per (key slot, value channel), [H, dk, dv] (ou_a set in the arguments): the
// backward leaves per-batch-row parts of the gate-gradient sums in the arithmetic type
size_t pc_ou_part_bytes(const Shape& s);
hipError_t launch_backward_pc(const Shape& s, const BwdArgs& a, const void* ck, float* kpart, hipStream_t st);
hipError_t launch_decode_pc(const Shape& s, const DecodeArgs& a, hipStream_t st);

// Block scaffolding: causal conv1d (k = 4) + SiLU, RMS QK-norm, SiLU gate.
int block_vec(bool bf16);   // elements per 16-byte vector
size_t conv_parts_bytes(int B, int T, int C);
size_t norm_parts_bytes(int n);
hipError_t launch_conv_fwd(int B, int T, int C, bool bf16, const void* x, const float* w, const float* bias, void* u,
                           hipStream_t st);
hipError_t launch_conv_bwd(int B, int T, int C, bool bf16, const void* x, const float* w, const float* bias,
                           const void* du, void* dx, float* dw, float* dbias, float* part, hipStream_t st);
hipError_t launch_norm_fwd(size_t rows, int n, bool bf16, const void* x, const float* w, float eps, void* out,
                           float* rstd, hipStream_t st);
hipError_t launch_norm_bwd(size_t rows, int n, bool bf16, const void* x, const float* w, const float* rstd,
                           const void* dout, void* dx, float* dw, float* part, hipStream_t st);
hipError_t launch_gate_fwd(size_t n, bool bf16, const void* y, const void* z, void* out, hipStream_t st);
hipError_t launch_gate_bwd(size_t n, bool bf16, const void* y, const void* z, const void* dout, void* dy, void* dz,
                           hipStream_t st);

// Monte Carlo readout (KLA+): draws y = ymu + sqrt(yvar) eps over nrow = B T H rows of dv
// channels, their backward, and the logsumexp-over-samples loss and its backward.
hipError_t launch_mc_sample(int S, size_t nrow, int dv, bool bf16, uint64_t seed, const void* ymu, const float* yvar,
                            void* ys, hipStream_t st);
hipError_t launch_mc_sample_bwd(int S, size_t nrow, int dv, bool bf16, uint64_t seed, const float* yvar,
                                const void* dys, void* dymu, float* dyvar, hipStream_t st);
hipError_t launch_mc_nll(int S, size_t n, const float* logp, float* nll, hipStream_t st);
hipError_t launch_mc_nll_bwd(int S, size_t n, const float* logp, const float* dnll, float* dlogp, hipStream_t st);

// OU gates: gradients of the parameters from the per-part gate-gradient sums (fp32
// parts, or fp64 when part_f64)
hipError_t launch_ou_param_grads(int H, int dk, int nparts, const void* part, bool part_f64, const float* a,
                                 const float* p, const float* d, float* da, float* dp, float* dd, hipStream_t st);

}  // namespace kla
