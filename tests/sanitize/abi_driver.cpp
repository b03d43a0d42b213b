// Sanitizer driver for the host side of the C ABI (test infrastructure): calls every entry point of
// include/qta.h with arguments that host validation must reject (null pointers, bad shapes,
// unsupported sizes, misaligned pointers, too-small workspaces, options out of range) and the
// workspace queries with valid ones, so that AddressSanitizer and UndefinedBehaviorSanitizer see the
// validation and layout code. Nothing here reaches a device: every call returns before a launch.
// Built with the host code sanitized (hipcc -Xarch_host -fsanitize=...) and run by
// tests/test_sanitizers.py; exits 0 when every call returns the expected status.
#include <cstdint>
#include <cstdio>

#include "qta.h"

namespace {

int failures = 0;

void expect(const char* what, int got, int want)
{
    if (got != want) {
        std::fprintf(stderr, "%s: status %d, expected %d\n", what, got, want);
        ++failures;
    }
}

}  // namespace

int main()
{
    // aligned, never dereferenced addresses: validation fails before any use
    void* const P = reinterpret_cast<void*>(uintptr_t{0x100000});
    void* const MIS = reinterpret_cast<void*>(uintptr_t{0x100004});
    const float* const F = static_cast<const float*>(P);

    int Hl[QTA_MAX_LEVELS], Wl[QTA_MAX_LEVELS];
    expect("level dims", qta_level_dims(200, 336, 5, Hl, Wl), QTA_OK);
    expect("level dims null", qta_level_dims(200, 336, 5, nullptr, Wl), QTA_ERR_INVALID);
    expect("level dims too many", qta_level_dims(4, 4, 17, Hl, Wl), QTA_ERR_INVALID);
    expect("level above 1x1", qta_level_dims(2, 2, 3, Hl, Wl), QTA_ERR_INVALID);

    // workspace queries, plain and with every option
    qta_workspace_layout lay;
    expect("layout", qta_get_workspace_layout(2, 2, 200, 336, 32, 5, 16, QTA_BF16, &lay), QTA_OK);
    if (qta_workspace_bytes(2, 2, 200, 336, 32, 5, 16, QTA_BF16) != lay.total) ++failures;
    const int Kl[QTA_MAX_LEVELS] = {0, 8, 16, 32, 64};
    const void* vls[QTA_MAX_LEVELS] = {nullptr, P, P, P, P};
    qta_options opt{};
    opt.K_levels = Kl;
    opt.v_levels = vls;
    opt.pe_weight = F;
    expect("layout ex", qta_get_workspace_layout_ex(1, 8, 60, 80, 32, 5, 8, QTA_F32, &opt, &lay), QTA_OK);
    opt.epipolar = 1;
    expect("layout epipolar", qta_get_workspace_layout_ex(2, 8, 120, 160, 32, 4, 8, QTA_BF16, &opt, &lay), QTA_OK);
    opt = qta_options{};
    const int Kbad[QTA_MAX_LEVELS] = {0, 8, 65};
    opt.K_levels = Kbad;
    expect("K above max", qta_get_workspace_layout_ex(1, 1, 16, 16, 32, 3, 8, QTA_F32, &opt, &lay),
           QTA_ERR_UNSUPPORTED);
    opt.K_levels = nullptr;
    opt.pe_bias = F;
    expect("bias without kernels", qta_get_workspace_layout_ex(1, 1, 16, 16, 32, 3, 8, QTA_F32, &opt, &lay),
           QTA_ERR_INVALID);
    if (qta_workspace_bytes(1, 1, 16, 16, 48, 3, 8, QTA_F32) != 0) ++failures;
    if (qta_backward_workspace_bytes_ex(2, 2, 200, 336, 32, 5, 16, QTA_VARIANT_B, QTA_BF16, nullptr) == 0) ++failures;

    // forward: each argument wrong in turn
    const size_t ws = size_t{1} << 30;
    expect("fwd null q", qta_forward(nullptr, P, P, nullptr, 1, 1, 16, 16, 32, 3, 4, QTA_VARIANT_A, QTA_F32, 0.f, P,
                                     P, ws, nullptr), QTA_ERR_INVALID);
    expect("fwd d", qta_forward(P, P, P, nullptr, 1, 1, 16, 16, 48, 3, 4, QTA_VARIANT_A, QTA_F32, 0.f, P, P, ws,
                                nullptr), QTA_ERR_UNSUPPORTED);
    expect("fwd misaligned", qta_forward(MIS, P, P, nullptr, 1, 1, 16, 16, 32, 3, 4, QTA_VARIANT_A, QTA_F32, 0.f, P,
                                         P, ws, nullptr), QTA_ERR_INVALID);
    expect("fwd workspace", qta_forward(P, P, P, nullptr, 1, 1, 16, 16, 32, 3, 4, QTA_VARIANT_A, QTA_F32, 0.f, P, P,
                                        16, nullptr), QTA_ERR_WORKSPACE);
    expect("fwd variant", qta_forward(P, P, P, nullptr, 1, 1, 16, 16, 32, 3, 4, static_cast<qta_variant>(7),
                                      QTA_F32, 0.f, P, P, ws, nullptr), QTA_ERR_INVALID);
    expect("fwd coarse too big", qta_forward(P, P, P, nullptr, 1, 1, 64, 64, 32, 1, 4, QTA_VARIANT_B, QTA_F32, 0.f,
                                             P, P, ws, nullptr), QTA_ERR_UNSUPPORTED);
    expect("fwd K", qta_forward(P, P, P, nullptr, 1, 1, 16, 16, 32, 3, 0, QTA_VARIANT_A, QTA_F32, 0.f, P, P, ws,
                                nullptr), QTA_ERR_INVALID);
    const void* vnull[QTA_MAX_LEVELS] = {nullptr, nullptr, P};
    opt = qta_options{};
    opt.v_levels = vnull;
    expect("fwd ex missing V level", qta_forward_ex(P, P, P, nullptr, 1, 1, 16, 16, 32, 3, 4, QTA_VARIANT_A, QTA_F32,
                                                    0.f, &opt, P, P, ws, nullptr), QTA_ERR_INVALID);
    opt = qta_options{};
    opt.epipolar = 1;
    expect("fwd ex epipolar levels", qta_forward_ex(P, P, P, nullptr, 1, 1, 16, 4, 32, 4, 4, QTA_VARIANT_A, QTA_F32,
                                                    0.f, &opt, P, P, ws, nullptr), QTA_ERR_INVALID);
    expect("noalloc too big", qta_forward_ex_noalloc(P, P, P, nullptr, 64, 8, 120, 160, 32, 4, 8, QTA_VARIANT_B,
                                                     QTA_F32, 0.f, nullptr, P, nullptr), QTA_ERR_WORKSPACE);
    expect("noalloc null", qta_forward_ex_noalloc(P, nullptr, P, nullptr, 1, 1, 16, 16, 32, 3, 4, QTA_VARIANT_B,
                                                  QTA_F32, 0.f, nullptr, P, nullptr), QTA_ERR_INVALID);

    // backward
    float* const G = static_cast<float*>(P);
    expect("bwd v levels", qta_backward_ex(P, P, P, nullptr, P, 1, 1, 16, 16, 32, 3, 4, QTA_VARIANT_A, QTA_F32, 0.f,
                                           nullptr, P, 16, G, G, G, nullptr, P, ws, nullptr), QTA_ERR_WORKSPACE);
    expect("bwd null dout", qta_backward_ex(P, P, P, nullptr, nullptr, 1, 1, 16, 16, 32, 3, 4, QTA_VARIANT_A, QTA_F32,
                                            0.f, nullptr, P, ws, G, G, G, nullptr, P, ws, nullptr), QTA_ERR_INVALID);
    expect("bwd small bwd workspace", qta_backward_ex(P, P, P, nullptr, P, 1, 1, 16, 16, 32, 3, 4, QTA_VARIANT_A,
                                                      QTA_F32, 0.f, nullptr, P, ws, G, G, G, nullptr, P, 16, nullptr),
           QTA_ERR_WORKSPACE);
    expect("bwd finest one level", qta_backward_finest_ex(P, P, P, nullptr, P, 1, 1, 16, 16, 32, 1, 4, QTA_VARIANT_A,
                                                          QTA_F32, 0.f, nullptr, P, ws, G, G, G, nullptr, P, ws,
                                                          nullptr), QTA_ERR_INVALID);

    // stage calls
    expect("pyramid C", qta_build_pyramid(P, P, 1, 16, 16, 6, 3, QTA_BF16, nullptr), QTA_ERR_UNSUPPORTED);
    expect("pyramid null", qta_build_pyramid(nullptr, P, 1, 16, 16, 8, 3, QTA_BF16, nullptr), QTA_ERR_INVALID);
    expect("coarse too big", qta_coarse_attn(P, P, P, 1, 1, 40, 40, 32, 4, QTA_VARIANT_B, QTA_F32, 0.f,
                                             static_cast<float*>(P), static_cast<int32_t*>(P), G, nullptr),
           QTA_ERR_UNSUPPORTED);
    expect("coarse half selection", qta_coarse_attn(P, P, P, 1, 1, 4, 4, 32, 4, QTA_VARIANT_B, QTA_F32, 0.f,
                                                    static_cast<float*>(P), static_cast<int32_t*>(P), nullptr,
                                                    nullptr), QTA_ERR_INVALID);
    expect("topk n", qta_topk(F, nullptr, 4, 5000, 4, static_cast<int32_t*>(P), G, nullptr), QTA_ERR_UNSUPPORTED);
    expect("topk K", qta_topk(F, nullptr, 4, 50, 65, static_cast<int32_t*>(P), G, nullptr), QTA_ERR_UNSUPPORTED);
    expect("fine A needs scores", qta_fine_attn(P, P, P, 1, 1, 8, 8, 32, 4, QTA_VARIANT_A, QTA_F32, 0.f,
                                                static_cast<const int32_t*>(P), nullptr, G,
                                                static_cast<int32_t*>(P), G, nullptr), QTA_ERR_INVALID);
    const float* msgs[QTA_MAX_LEVELS] = {F, nullptr};
    expect("finest null message", qta_finest_attn(P, P, P, 1, 1, 8, 8, 32, 4, QTA_VARIANT_B, QTA_F32, 0.f,
                                                  static_cast<const int32_t*>(P), nullptr, 3, msgs, nullptr, P,
                                                  nullptr), QTA_ERR_INVALID);
    for (int s = 0; s < 6; ++s)
        if (!qta_status_str(static_cast<qta_status>(s))) ++failures;

    std::printf("host validation: %d failures\n", failures);
    return failures != 0;
}
