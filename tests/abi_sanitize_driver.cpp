// Test infrastructure: drives the host-side argument validation of every
// entry point of include/ffsl.h with invalid arguments (null pointers, bad
// sizes, bad types, misaligned buffers, a short workspace).  Every one of
// these calls must return its error code before anything touches a device,
// so the driver runs without a GPU.  tests/test_abi_sanitize.py builds the
// library's host code with AddressSanitizer and UndefinedBehaviorSanitizer
// (no device code) and runs this driver against it.
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "../include/ffsl.h"

static int failures = 0;

static void expect(const char *what, int got, int want) {
    if (got != want) {
        printf("FAIL %s: got %d, want %d (%s)\n", what, got, want, ffsl_last_error());
        ++failures;
    } else if (want != FFSL_OK && ffsl_last_error()[0] == '\0') {
        printf("FAIL %s: no error message\n", what);
        ++failures;
    }
}

int main() {
    // placeholders: never dereferenced, 256-byte aligned where that is checked
    void *p = (void *)(uintptr_t)(1u << 20);
    void *odd = (void *)(uintptr_t)((1u << 20) + 2);
    ffsl_layer *h = nullptr;
    const int BF = FFSL_BF16, F32 = FFSL_F32, I32 = FFSL_IDX_I32;

    // ------------------------------------------------------------ layers
    expect("create: out null",
           ffsl_create_layer_ex(nullptr, 100, 64, 8, BF, I32, p, p, nullptr, (float *)p, (float *)p, nullptr, nullptr, nullptr,
                                nullptr, p, 1 << 20, 8, 8),
           FFSL_EINVAL);
    struct {
        const char *what;
        int64_t L;
        int d, k, vt, it, B, nnz;
    } shapes[] = {
        {"L = 0", 0, 64, 8, BF, I32, 8, 8},         {"d = 0", 100, 0, 8, BF, I32, 8, 8},
        {"d too large", 100, FFSL_MAX_D + 1, 8, BF, I32, 8, 8},
        {"k = 0", 100, 64, 0, BF, I32, 8, 8},       {"k > d", 100, 8, 9, BF, I32, 8, 8},
        {"k too large", 100, 1024, FFSL_MAX_K + 1, BF, I32, 8, 8},
        {"B_max = 0", 100, 64, 8, BF, I32, 0, 8},   {"B_max too large", 100, 64, 8, BF, I32, FFSL_MAX_B + 1, 8},
        {"nnz_max < 0", 100, 64, 8, BF, I32, 8, -1}, {"L*k too large", (int64_t)1 << 40, 64, 8, BF, I32, 8, 8},
        {"value dtype", 100, 64, 8, 5, I32, 8, 8},   {"index dtype", 100, 64, 8, BF, 3, 8, 8},
    };
    for (auto &s : shapes)
        expect(s.what,
               ffsl_create_layer_ex(&h, s.L, s.d, s.k, s.vt, s.it, p, p, nullptr, (float *)p, (float *)p, nullptr, nullptr, nullptr,
                                    nullptr, p, 1 << 20, s.B, s.nnz),
               FFSL_EINVAL);
    expect("create: W null",
           ffsl_create_layer_ex(&h, 100, 64, 8, F32, I32, nullptr, p, nullptr, (float *)p, (float *)p, nullptr, nullptr, nullptr,
                                nullptr, p, 1 << 20, 8, 8),
           FFSL_EINVAL);
    expect("create: bias without moments",
           ffsl_create_layer_ex(&h, 100, 64, 8, F32, I32, p, p, (float *)p, (float *)p,
                                (float *)p, nullptr, nullptr, nullptr, nullptr, p, 1 << 20, 8, 8),
           FFSL_EINVAL);
    expect("create: dbias without bias",
           ffsl_create_layer_ex(&h, 100, 64, 8, F32, I32, p, p, nullptr, (float *)p, (float *)p, nullptr, nullptr,
                                nullptr, (float *)p, p, 1 << 20, 8, 8),
           FFSL_EINVAL);
    expect("create: workspace null",
           ffsl_create_layer_ex(&h, 100, 64, 8, F32, I32, p, p, nullptr, (float *)p, (float *)p, nullptr, nullptr,
                                nullptr, nullptr, nullptr, 1 << 20, 8, 8),
           FFSL_EINVAL);
    expect("create: workspace misaligned",
           ffsl_create_layer_ex(&h, 100, 64, 8, F32, I32, p, p, nullptr, (float *)p, (float *)p, nullptr, nullptr,
                                nullptr, nullptr, odd, 1 << 20, 8, 8),
           FFSL_EINVAL);
    expect("create: W misaligned",
           ffsl_create_layer_ex(&h, 100, 64, 8, F32, I32, odd, p, nullptr, (float *)p, (float *)p, nullptr, nullptr,
                                nullptr, nullptr, p, 1 << 20, 8, 8),
           FFSL_EINVAL);
    expect("create: u16 indices, d too wide",
           ffsl_create_layer_ex(&h, 100, 70000, 8, BF, FFSL_IDX_U16, p, p, nullptr, (float *)p, (float *)p, nullptr,
                                nullptr, nullptr, nullptr, p, 1 << 20, 8, 8),
           FFSL_EINVAL);
    if (ffsl_workspace_bytes(0, 64, 8, 8, 8) != 0 || ffsl_workspace_bytes_ex(100, 64, 8, 7, 8, 8) != 0) {
        printf("FAIL workspace bytes of an invalid shape\n");
        ++failures;
    }

    // ------------------------------------------------------------ calls on a null handle
    float f = 0.f;
    int32_t i = 0;
    expect("forward: null layer",
           ffsl_forward_loss(nullptr, p, 1, (int32_t *)p, (int32_t *)p, 1, 1.f, &f, nullptr, 0, nullptr),
           FFSL_EINVAL);
    expect("backward: null layer",
           ffsl_backward(nullptr, p, 1, (int32_t *)p, (int32_t *)p, 1, 1.f, nullptr, &f, 0, nullptr), FFSL_EINVAL);
    expect("adam: null layer", ffsl_adam_step(nullptr, 1, 1e-3f, 0.9f, 0.999f, 1e-8f, 0.f, nullptr), FFSL_EINVAL);
    expect("train: null layer",
           ffsl_train_step(nullptr, p, 1, (int32_t *)p, (int32_t *)p, 1, 1.f, 1, 1e-3f, 0.9f, 0.999f, 1e-8f, 0.f,
                           &f, &f, 0, nullptr),
           FFSL_EINVAL);
    expect("train+set: null layer",
           ffsl_train_step_set(nullptr, p, 1, (int32_t *)p, (int32_t *)p, 1, 1.f, 1, 1e-3f, 0.9f, 0.999f, 1e-8f,
                               0.f, &f, &f, 0, 0.1f, 1, 1, nullptr, &i, nullptr),
           FFSL_EINVAL);
    expect("set: null layer", ffsl_set_update(nullptr, 0.1f, 1, 1, nullptr, &i, nullptr), FFSL_EINVAL);
    expect("set threshold: null layer", ffsl_set_update_threshold(nullptr, 0.1f, 1, 1, nullptr, &i, nullptr),
           FFSL_EINVAL);
    expect("validate: null layer", ffsl_validate_indices(nullptr, &i, nullptr), FFSL_EINVAL);
    expect("timing: null layer", ffsl_set_timing_events(nullptr, nullptr, nullptr), FFSL_EINVAL);
    expect("topk: null layer",
           ffsl_infer_topk(nullptr, p, 1, 1, &i, &f, nullptr, nullptr, 0, nullptr, p, 1 << 20, nullptr),
           FFSL_EINVAL);
    if (ffsl_topk_workspace_bytes(nullptr, 8, 5) != 0) {
        printf("FAIL topk workspace of a null layer\n");
        ++failures;
    }

    // ------------------------------------------------------------ dense parts
    expect("gelu fwd: B = 0",
           ffsl_dense_gelu_fwd(p, 0, 64, 64, p, nullptr, &f, p, nullptr, 0, nullptr), FFSL_EINVAL);
    expect("gelu fwd: din not a multiple of 8",
           ffsl_dense_gelu_fwd(p, 4, 60, 64, p, nullptr, &f, p, nullptr, 0, nullptr), FFSL_EINVAL);
    expect("gelu fwd: X misaligned",
           ffsl_dense_gelu_fwd(odd, 4, 64, 64, p, nullptr, &f, p, nullptr, 0, nullptr), FFSL_EINVAL);
    expect("gelu fwd: outputs null",
           ffsl_dense_gelu_fwd(p, 4, 64, 64, p, nullptr, nullptr, p, nullptr, 0, nullptr), FFSL_EINVAL);
    expect("gelu fwd: workspace misaligned",
           ffsl_dense_gelu_fwd(p, 4, 64, 64, p, nullptr, &f, p, odd, 1 << 20, nullptr), FFSL_EINVAL);
    expect("gelu fwd: workspace short",
           ffsl_dense_gelu_fwd(p, 4, 64, 64, p, nullptr, &f, p, p, 16, nullptr), FFSL_EINVAL);
    expect("gelu bwd: workspace null",
           ffsl_dense_gelu_bwd(p, 4, 64, 64, p, &f, &f, &f, nullptr, nullptr, 0, nullptr, 0, nullptr), FFSL_EINVAL);
    expect("gelu bwd: dW1 null",
           ffsl_dense_gelu_bwd(p, 4, 64, 64, p, &f, &f, nullptr, nullptr, nullptr, 0, p, 1 << 20, nullptr),
           FFSL_EINVAL);
    expect("aux: n_labels = 0",
           ffsl_aux_bce_fwd_bwd(p, 4, 64, 32, 0, p, nullptr, (int32_t *)p, (int32_t *)p, 1, 1.f, &f, &f, nullptr,
                                nullptr, nullptr, 0, p, 1 << 20, nullptr),
           FFSL_EINVAL);
    expect("aux: tgt_off null",
           ffsl_aux_bce_fwd_bwd(p, 4, 64, 32, 100, p, nullptr, nullptr, (int32_t *)p, 1, 1.f, &f, &f, nullptr,
                                nullptr, nullptr, 0, p, 1 << 20, nullptr),
           FFSL_EINVAL);
    expect("aux: C not a multiple of 8",
           ffsl_aux_bce_fwd_bwd(p, 4, 64, 30, 100, p, nullptr, (int32_t *)p, (int32_t *)p, 1, 1.f, &f, &f,
                                nullptr, nullptr, nullptr, 0, p, 1 << 20, nullptr),
           FFSL_EINVAL);
    expect("aux: workspace short",
           ffsl_aux_bce_fwd_bwd(p, 4, 64, 32, 100, p, nullptr, (int32_t *)p, (int32_t *)p, 1, 1.f, &f, &f,
                                nullptr, nullptr, nullptr, 0, p, 64, nullptr),
           FFSL_EINVAL);
    expect("adam dense: n = 0", ffsl_adam_dense(p, F32, &f, &f, &f, 0, 1, 1e-3f, 0.9f, 0.999f, 1e-8f, 0.f, nullptr),
           FFSL_EINVAL);
    expect("adam dense: bad type",
           ffsl_adam_dense(p, 9, &f, &f, &f, 10, 1, 1e-3f, 0.9f, 0.999f, 1e-8f, 0.f, nullptr), FFSL_EUNSUPPORTED);
    expect("adam dense: t = 0", ffsl_adam_dense(p, F32, &f, &f, &f, 10, 0, 1e-3f, 0.9f, 0.999f, 1e-8f, 0.f, nullptr),
           FFSL_EINVAL);
    expect("adam dense: beta out of range",
           ffsl_adam_dense(p, F32, &f, &f, &f, 10, 1, 1e-3f, 1.5f, 0.999f, 1e-8f, 0.f, nullptr), FFSL_EINVAL);
    if (ffsl_dense_workspace_bytes(0, 64, 64) != 0 || ffsl_aux_workspace_bytes(4, 64, 7) != 0) {
        printf("FAIL dense workspace of an invalid shape\n");
        ++failures;
    }
    // a long message stays within the buffer
    expect("version", ffsl_version() >= 100 ? FFSL_OK : -99, FFSL_OK);
    printf("abi sanitize driver: %d failures\n", failures);
    return failures == 0 ? 0 : 1;
}
