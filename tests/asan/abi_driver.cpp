// Host sanitizer run of the C ABI layer (csrc/kla_api.cpp built with
// -fsanitize=address,undefined, linked with the library's other objects): every
// path that returns before any device work -- workspace and saved-context queries
// over all widths and dtypes, and the argument errors of every entry point (bad
// descriptors, NULL pointers, misaligned pointers, short workspaces) -- with the
// expected status each time.  No GPU is needed; the sanitizers abort on any invalid
// access.  Exit 0 on success.
#include <cstdint>
#include <cstdio>

#include "kla.h"

static int fails = 0;
#define EXPECT(expr, want)                                                                        \
    do {                                                                                          \
        const int got_ = (int)(expr);                                                             \
        if (got_ != (int)(want)) {                                                                \
            std::fprintf(stderr, "line %d: %s returned %d, expected %d\n", __LINE__, #expr, got_, \
                         (int)(want));                                                            \
            ++fails;                                                                              \
        }                                                                                         \
    } while (0)

int main() {
    // a fake, 16-byte aligned device address: every call below fails its checks
    // before dereferencing it
    alignas(16) static unsigned char buf[256];
    void* P = buf;
    void* M = buf + 1;   // misaligned
    float* F = reinterpret_cast<float*>(buf);
    const int widths[] = {16, 32, 64, 128};
    for (int dt = 0; dt < 2; ++dt)
        for (int dk : widths)
            for (int dv : widths) {
                kla_desc d{2, 100, 3, dk, dv, dt};
                if (kla_forward_workspace(&d) == 0) ++fails;
                if (kla_saved_bytes(&d) == 0) ++fails;
                if (kla_backward_workspace(&d, 0) < kla_backward_workspace(&d, 1)) ++fails;
                if (kla_backward_ou_workspace(&d, 1) < kla_backward_workspace(&d, 1)) ++fails;
                (void)kla_saved_pc_bytes(&d);
                (void)kla_backward_pc_workspace(&d, 0);
                (void)kla_backward_pc_ou_workspace(&d, 1);
            }
    // bad descriptors: the queries return 0, the calls KLA_ERR_SHAPE / KLA_ERR_DTYPE
    kla_desc bad_w{1, 8, 1, 48, 16, KLA_F32}, bad_t{1, -1, 1, 16, 16, KLA_F32}, bad_d{1, 8, 1, 16, 16, 7};
    if (kla_forward_workspace(&bad_w) || kla_saved_bytes(&bad_t) || kla_backward_workspace(&bad_d, 1)) ++fails;
    EXPECT(kla_forward(&bad_w, P, P, P, P, P, P, nullptr, nullptr, P, nullptr, nullptr, nullptr, nullptr, P, 1 << 20,
                       nullptr),
           KLA_ERR_SHAPE);
    EXPECT(kla_forward(&bad_d, P, P, P, P, P, P, nullptr, nullptr, P, nullptr, nullptr, nullptr, nullptr, P, 1 << 20,
                       nullptr),
           KLA_ERR_DTYPE);
    EXPECT(kla_forward(nullptr, P, P, P, P, P, P, nullptr, nullptr, P, nullptr, nullptr, nullptr, nullptr, P, 1 << 20,
                       nullptr),
           KLA_ERR_NULL);

    kla_desc d{2, 64, 2, 64, 32, KLA_BF16};
    const size_t fw = kla_forward_workspace(&d), bw = kla_backward_workspace(&d, 1);
    // forward: NULL input, misaligned input, short workspace
    EXPECT(kla_forward(&d, nullptr, P, P, P, P, P, nullptr, nullptr, P, nullptr, nullptr, nullptr, nullptr, P, fw,
                       nullptr),
           KLA_ERR_NULL);
    EXPECT(kla_forward(&d, P, M, P, P, P, P, nullptr, nullptr, P, nullptr, nullptr, nullptr, nullptr, P, fw, nullptr),
           KLA_ERR_ALIGN);
    EXPECT(kla_forward(&d, P, P, P, P, P, P, nullptr, nullptr, P, nullptr, nullptr, nullptr, nullptr, P, fw - 1,
                       nullptr),
           KLA_ERR_WORKSPACE);
    // backward
    EXPECT(kla_backward(&d, P, P, P, P, P, P, nullptr, nullptr, P, nullptr, nullptr, nullptr, nullptr, P, P, P, P, P,
                        P, nullptr, nullptr, P, bw, nullptr),
           KLA_ERR_NULL);
    EXPECT(kla_backward(&d, P, P, P, P, P, P, nullptr, nullptr, P, P, nullptr, nullptr, nullptr, P, P, P, P, P, M,
                        nullptr, nullptr, P, bw, nullptr),
           KLA_ERR_ALIGN);
    EXPECT(kla_backward(&d, P, P, P, P, P, P, nullptr, nullptr, P, P, nullptr, nullptr, nullptr, P, P, P, P, P, P,
                        nullptr, nullptr, P, bw - 1, nullptr),
           KLA_ERR_WORKSPACE);
    // allocation-free backward: a shape whose workspace exceeds the static limit
    kla_desc huge{64, 65536, 16, 128, 128, KLA_F32};
    EXPECT(kla_backward_noalloc(&huge, P, P, P, P, P, P, nullptr, nullptr, P, P, nullptr, nullptr, nullptr, P, P, P,
                                P, P, P, nullptr, nullptr, nullptr),
           KLA_ERR_WORKSPACE);
    EXPECT(kla_backward_noalloc(&d, P, P, P, P, P, P, nullptr, nullptr, nullptr, P, nullptr, nullptr, nullptr, P, P,
                                P, P, P, P, nullptr, nullptr, nullptr),
           KLA_ERR_NULL);
    // OU entry points
    EXPECT(kla_forward_ou(&d, P, P, P, nullptr, F, F, P, nullptr, nullptr, P, nullptr, nullptr, nullptr, nullptr, P,
                          fw, nullptr),
           KLA_ERR_NULL);
    // decode: bad width, NULL belief
    EXPECT(kla_decode_step(4, 2, 48, 16, KLA_F32, P, P, P, P, P, P, F, F, P, nullptr, nullptr), KLA_ERR_SHAPE);
    EXPECT(kla_decode_step(4, 2, 64, 16, KLA_F32, P, P, P, P, P, P, nullptr, F, P, nullptr, nullptr), KLA_ERR_NULL);
    EXPECT(kla_decode_step(4, 2, 64, 16, 9, P, P, P, P, P, P, F, F, P, nullptr, nullptr), KLA_ERR_DTYPE);
    // Monte Carlo readout
    EXPECT(kla_mc_sample(4, 1, 8, 2, 24, KLA_F32, 1, P, F, P, nullptr), KLA_ERR_SHAPE);
    EXPECT(kla_mc_sample(4, 1, 8, 2, 32, KLA_F32, 1, nullptr, F, P, nullptr), KLA_ERR_NULL);
    EXPECT(kla_mc_sample(4, 1, 8, 2, 32, KLA_F32, 1, M, F, P, nullptr), KLA_ERR_ALIGN);
    EXPECT(kla_mc_sample_backward(0, 1, 8, 2, 32, KLA_F32, 1, F, P, P, F, nullptr), KLA_ERR_SHAPE);
    EXPECT(kla_mc_nll(0, 16, F, F, nullptr), KLA_ERR_SHAPE);
    EXPECT(kla_mc_nll(4, 16, nullptr, F, nullptr), KLA_ERR_NULL);
    EXPECT(kla_mc_nll_backward(4, 16, F, nullptr, F, nullptr), KLA_ERR_NULL);
    // every status has a name
    for (int s = 0; s <= 9; ++s)
        if (!kla_status_string((kla_status)s)[0]) ++fails;
    if (fails == 0) std::printf("ABI sanitizer run: ok\n");
    return fails ? 1 : 0;
}
