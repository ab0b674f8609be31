// C ABI of libffsl: argument validation, workspace layout, dispatch.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>

#include <algorithm>
#include <new>
#include <string>

#include "ffsl_internal.h"

struct ffsl_layer {
    ffsl::Layer ly;
};

namespace ffsl {

static thread_local std::string g_err;

void set_error(const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_err = buf;
}

int fail(int code, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

int check_launch(const char *what) {
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(FFSL_EHIP, "%s launch failed: %s", what, hipGetErrorString(e));
    return FFSL_OK;
}

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

int max_parts_for(int num_cu) { return std::max(1, std::min(2 * num_cu, 1024)); }

WsLayout ws_layout(int64_t L, int32_t d, int32_t k, int32_t vt, int32_t B_max, int32_t nnz_max, int max_parts) {
    WsLayout w{};
    // the fused fast paths (bf16 only) and their buffers: the same shape
    // predicates as their dispatch (sweep_mx_eligible, sweep_wide_eligible)
    const bool bf16 = vt == FFSL_BF16;
    const bool wide = bf16 && wide_shape(L, d, k);
    const bool mx = bf16 && !wide && mx_shape(L, d, k);
    const int pass_b = wide ? WD_PASS_B : MX_PASS_B;
    const int passes = (B_max + pass_b - 1) / pass_b;
    size_t off = 0;
    w.loss_part = off;
    off = align256(off + sizeof(float) * (size_t)max_parts * (size_t)passes);
    w.tgt_b = off;
    off = align256(off + sizeof(int32_t) * (size_t)std::max(nnz_max, 1));
    w.dx_part = off;
    off = align256(off + sizeof(float) * (size_t)max_parts * (size_t)B_max * (size_t)d);
    w.has_partial = (mx && B_max > MX_PASS_B) || (wide && B_max > WD_PASS_B);
    w.dwp = off;
    if (w.has_partial) off = align256(off + sizeof(float) * (size_t)L * (size_t)k);
    w.dbp = off;
    if (w.has_partial) off = align256(off + sizeof(float) * (size_t)L);
    w.has_xt = wide || mx;
    w.keys = off;
    if (w.has_xt) off = align256(off + sizeof(uint32_t) * 1024 * (size_t)passes);
    w.xt = off;
    if (w.has_xt) off = align256(off + sizeof(uint16_t) * (size_t)passes * pass_b * (size_t)d);
    w.set_list = off;
    if (mx) off = align256(off + sizeof(int32_t) * (size_t)(L + 1));
    w.total = off;
    return w;
}

static int device_cu_count(int *cu, int *dev) {
    hipError_t e = hipGetDevice(dev);
    if (e != hipSuccess) return fail(FFSL_EHIP, "hipGetDevice: %s", hipGetErrorString(e));
    e = hipDeviceGetAttribute(cu, hipDeviceAttributeMultiprocessorCount, *dev);
    if (e != hipSuccess) return fail(FFSL_EHIP, "hipDeviceGetAttribute: %s", hipGetErrorString(e));
    return FFSL_OK;
}

static int check_shape(int64_t L, int32_t d, int32_t k, int32_t B_max, int32_t nnz_max) {
    if (L < 1) return fail(FFSL_EINVAL, "L must be >= 1 (got %lld)", (long long)L);
    if (d < 1 || d > FFSL_MAX_D) return fail(FFSL_EINVAL, "d must be in [1,%d] (got %d)", FFSL_MAX_D, d);
    if (k < 1 || k > d || k > FFSL_MAX_K)
        return fail(FFSL_EINVAL, "k must be in [1, min(d,%d)] (got k=%d, d=%d)", FFSL_MAX_K, k, d);
    if (B_max < 1 || B_max > FFSL_MAX_B)
        return fail(FFSL_EINVAL, "B_max must be in [1,%d] (got %d)", FFSL_MAX_B, B_max);
    if (nnz_max < 0) return fail(FFSL_EINVAL, "nnz_max must be >= 0");
    if (L > ((int64_t)1 << 40) / k) return fail(FFSL_EINVAL, "L*k too large");
    return FFSL_OK;
}

static int check_batch(const Layer &ly, const void *X, int32_t B, const int32_t *off, const int32_t *lab,
                       int32_t nnz) {
    if (!X) return fail(FFSL_EINVAL, "X is null");
    if (B < 1 || B > ly.B_max) return fail(FFSL_EINVAL, "B must be in [1,%d] (got %d)", ly.B_max, B);
    if (!off) return fail(FFSL_EINVAL, "tgt_off is null");
    if (nnz < 0 || nnz > ly.nnz_max)
        return fail(FFSL_EINVAL, "nnz must be in [0,%d] (got %d)", ly.nnz_max, nnz);
    if (nnz > 0 && !lab) return fail(FFSL_EINVAL, "tgt_lab is null");
    return FFSL_OK;
}

static int check_adam(int64_t t, float lr, float b1, float b2, float eps, float wd, AdamParams *p) {
    if (t < 1) return fail(FFSL_EINVAL, "Adam step t must be >= 1 (got %lld)", (long long)t);
    if (!(b1 >= 0.f && b1 < 1.f) || !(b2 >= 0.f && b2 < 1.f))
        return fail(FFSL_EINVAL, "betas must be in [0,1)");
    if (!(eps >= 0.f) || !isfinite(lr) || !isfinite(wd)) return fail(FFSL_EINVAL, "bad lr/eps/wd");
    p->lr = lr;
    p->b1 = b1;
    p->b2 = b2;
    p->eps = eps;
    p->wd = wd;
    p->bc1 = (float)(1.0 - pow((double)b1, (double)t));
    p->bc2 = (float)(1.0 - pow((double)b2, (double)t));
    if (!(p->bc1 > 0.f) || !(p->bc2 > 0.f)) return fail(FFSL_EINVAL, "bias correction underflows");
    return FFSL_OK;
}


static int check_width(const char *name, int64_t x, int64_t hi) {
    if (x < 8 || x > hi || x % 8 != 0)
        return fail(FFSL_EINVAL, "%s must be a multiple of 8 in [8,%lld] (got %lld)", name, (long long)hi,
                    (long long)x);
    return FFSL_OK;
}

static int check_aligned16(const char *name, const void *p) {
    if (!p) return fail(FFSL_EINVAL, "%s is null", name);
    if (reinterpret_cast<uintptr_t>(p) & 15u) return fail(FFSL_EINVAL, "%s must be 16-byte aligned", name);
    return FFSL_OK;
}

static int check_dense_batch(int32_t B) {
    if (B < 1 || B > FFSL_MAX_B) return fail(FFSL_EINVAL, "B must be in [1,%d] (got %d)", FFSL_MAX_B, B);
    return FFSL_OK;
}

static int current_cu_count(int *cu) {
    int dev = 0;
    return device_cu_count(cu, &dev);
}

}  // namespace ffsl

using namespace ffsl;

extern "C" {

const char *ffsl_last_error(void) { return g_err.c_str(); }

int ffsl_version(void) { return 100; }

size_t ffsl_workspace_bytes_ex(int64_t L, int32_t d, int32_t k, int32_t value_dtype, int32_t B_max,
                               int32_t nnz_max) {
    if (check_shape(L, d, k, B_max, nnz_max)) return 0;
    if (value_dtype != FFSL_F32 && value_dtype != FFSL_BF16) return 0;
    int cu = 0, dev = 0;
    if (device_cu_count(&cu, &dev)) return 0;
    return ws_layout(L, d, k, value_dtype, B_max, nnz_max, max_parts_for(cu)).total;
}

size_t ffsl_workspace_bytes(int64_t L, int32_t d, int32_t k, int32_t B_max, int32_t nnz_max) {
    // without the value type: the bf16 layout, which holds every buffer an
    // fp32 layer of the same shape needs
    return ffsl_workspace_bytes_ex(L, d, k, FFSL_BF16, B_max, nnz_max);
}

int ffsl_create_layer_ex(ffsl_layer **out, int64_t L, int32_t d, int32_t k, int32_t value_dtype,
                         int32_t index_dtype, void *W, void *I, float *bias, float *m, float *v, float *bias_m,
                         float *bias_v, float *dW, float *dbias, void *workspace, size_t workspace_bytes,
                         int32_t B_max, int32_t nnz_max) {
    g_err.clear();
    if (!out) return fail(FFSL_EINVAL, "out is null");
    *out = nullptr;
    int rc = check_shape(L, d, k, B_max, nnz_max);
    if (rc) return rc;
    if (value_dtype != FFSL_F32 && value_dtype != FFSL_BF16)
        return fail(FFSL_EINVAL, "value_dtype must be FFSL_F32 or FFSL_BF16");
    if (index_dtype != FFSL_IDX_I32 && index_dtype != FFSL_IDX_U16)
        return fail(FFSL_EINVAL, "index_dtype must be FFSL_IDX_I32 or FFSL_IDX_U16");
    if (index_dtype == FFSL_IDX_U16 && d > 65536)
        return fail(FFSL_EINVAL, "16-bit indices need d <= 65536 (got %d)", d);
    if (!W || !I || !m || !v) return fail(FFSL_EINVAL, "W, I, m and v are required");
    if (bias && (!bias_m || !bias_v)) return fail(FFSL_EINVAL, "bias needs bias_m and bias_v");
    if (dbias && !bias) return fail(FFSL_EINVAL, "dbias given without bias");
    if (!workspace) return fail(FFSL_EINVAL, "workspace is null");
    if (reinterpret_cast<uintptr_t>(workspace) & 255) return fail(FFSL_EINVAL, "workspace must be 256-byte aligned");
    if ((reinterpret_cast<uintptr_t>(W) | reinterpret_cast<uintptr_t>(I) | reinterpret_cast<uintptr_t>(m) |
         reinterpret_cast<uintptr_t>(v)) & 15)
        return fail(FFSL_EINVAL, "W, I, m, v must be 16-byte aligned");
    int cu = 0, dev = 0;
    rc = device_cu_count(&cu, &dev);
    if (rc) return rc;
    const int parts = max_parts_for(cu);
    const WsLayout wl = ws_layout(L, d, k, value_dtype, B_max, nnz_max, parts);
    if (workspace_bytes < wl.total)
        return fail(FFSL_EINVAL, "workspace too small: %zu < %zu bytes", workspace_bytes, wl.total);
    ffsl_layer *h = new (std::nothrow) ffsl_layer;
    if (!h) return fail(FFSL_EINVAL, "out of host memory");
    Layer &ly = h->ly;
    ly.L = L;
    ly.d = d;
    ly.k = k;
    ly.vt = value_dtype;
    ly.B_max = B_max;
    ly.nnz_max = nnz_max;
    ly.W = W;
    ly.I = static_cast<int32_t *>(I);
    ly.idx16 = index_dtype == FFSL_IDX_U16 ? 1 : 0;
    ly.bias = bias;
    ly.m = m;
    ly.v = v;
    ly.bm = bias_m;
    ly.bv = bias_v;
    ly.dW = dW;
    ly.dbias = dbias;
    ly.ws = static_cast<char *>(workspace);
    ly.ws_bytes = workspace_bytes;
    ly.num_cu = cu;
    ly.max_parts = parts;
    ly.device = dev;
    ly.ev_start = nullptr;
    ly.ev_stop = nullptr;
    *out = h;
    return FFSL_OK;
}

int ffsl_create_layer(ffsl_layer **out, int64_t L, int32_t d, int32_t k, int32_t value_dtype, void *W,
                      int32_t *I, float *bias, float *m, float *v, float *bias_m, float *bias_v, float *dW,
                      float *dbias, void *workspace, size_t workspace_bytes, int32_t B_max,
                      int32_t nnz_max) {
    return ffsl_create_layer_ex(out, L, d, k, value_dtype, FFSL_IDX_I32, W, I, bias, m, v, bias_m, bias_v, dW,
                                dbias, workspace, workspace_bytes, B_max, nnz_max);
}

int ffsl_destroy_layer(ffsl_layer *layer) {
    delete layer;
    return FFSL_OK;
}

int ffsl_forward_loss(ffsl_layer *layer, const void *X, int32_t B, const int32_t *tgt_off,
                      const int32_t *tgt_lab, int32_t nnz, float s, float *loss_out, float *logits_out,
                      uint32_t flags, void *stream) {
    g_err.clear();
    if (!layer) return fail(FFSL_EINVAL, "layer is null");
    int rc = check_batch(layer->ly, X, B, tgt_off, tgt_lab, nnz);
    if (rc) return rc;
    if (!loss_out) return fail(FFSL_EINVAL, "loss_out is null");
    SweepCall c{};
    c.layer = &layer->ly;
    c.X = X;
    c.B = B;
    c.tgt_off = tgt_off;
    c.tgt_lab = tgt_lab;
    c.nnz = nnz;
    c.s = s;
    c.mode = SWEEP_FWD;
    c.loss_out = loss_out;
    c.logits_out = logits_out;
    c.flags = flags;
    c.stream = static_cast<hipStream_t>(stream);
    return launch_sweep(c);
}

int ffsl_backward(ffsl_layer *layer, const void *X, int32_t B, const int32_t *tgt_off, const int32_t *tgt_lab,
                  int32_t nnz, float s, float *loss_out, float *dX_out, uint32_t flags, void *stream) {
    g_err.clear();
    if (!layer) return fail(FFSL_EINVAL, "layer is null");
    int rc = check_batch(layer->ly, X, B, tgt_off, tgt_lab, nnz);
    if (rc) return rc;
    if (!layer->ly.dW) return fail(FFSL_EINVAL, "layer was created without a dW buffer");
    if (!dX_out) return fail(FFSL_EINVAL, "dX_out is null");
    SweepCall c{};
    c.layer = &layer->ly;
    c.X = X;
    c.B = B;
    c.tgt_off = tgt_off;
    c.tgt_lab = tgt_lab;
    c.nnz = nnz;
    c.s = s;
    c.mode = SWEEP_BWD;
    c.loss_out = loss_out;
    c.dX_out = dX_out;
    c.flags = flags;
    c.stream = static_cast<hipStream_t>(stream);
    return launch_sweep(c);
}

int ffsl_adam_step(ffsl_layer *layer, int64_t t, float lr, float beta1, float beta2, float eps, float wd,
                   void *stream) {
    g_err.clear();
    if (!layer) return fail(FFSL_EINVAL, "layer is null");
    if (!layer->ly.dW) return fail(FFSL_EINVAL, "layer was created without a dW buffer");
    if (layer->ly.bias && !layer->ly.dbias) return fail(FFSL_EINVAL, "layer has a bias but no dbias buffer");
    AdamParams p{};
    int rc = check_adam(t, lr, beta1, beta2, eps, wd, &p);
    if (rc) return rc;
    return launch_adam(layer->ly, p, static_cast<hipStream_t>(stream));
}

int ffsl_train_step(ffsl_layer *layer, const void *X, int32_t B, const int32_t *tgt_off, const int32_t *tgt_lab,
                    int32_t nnz, float s, int64_t t, float lr, float beta1, float beta2, float eps, float wd,
                    float *loss_out, float *dX_out, uint32_t flags, void *stream) {
    g_err.clear();
    if (!layer) return fail(FFSL_EINVAL, "layer is null");
    int rc = check_batch(layer->ly, X, B, tgt_off, tgt_lab, nnz);
    if (rc) return rc;
    SweepCall c{};
    rc = check_adam(t, lr, beta1, beta2, eps, wd, &c.adam);
    if (rc) return rc;
    c.layer = &layer->ly;
    c.X = X;
    c.B = B;
    c.tgt_off = tgt_off;
    c.tgt_lab = tgt_lab;
    c.nnz = nnz;
    c.s = s;
    c.mode = SWEEP_FUSED;
    c.loss_out = loss_out;
    c.dX_out = dX_out;
    c.flags = flags;
    c.stream = static_cast<hipStream_t>(stream);
    return launch_sweep(c);
}

int ffsl_train_step_set(ffsl_layer *layer, const void *X, int32_t B, const int32_t *tgt_off,
                        const int32_t *tgt_lab, int32_t nnz, float s, int64_t t, float lr, float beta1, float beta2,
                        float eps, float wd, float *loss_out, float *dX_out, uint32_t flags, float frac,
                        uint64_t seed, uint64_t set_round, uint8_t *pruned_mask_out, int32_t *exhausted_out,
                        void *stream) {
    g_err.clear();
    if (!layer) return fail(FFSL_EINVAL, "layer is null");
    const Layer &ly = layer->ly;
    int rc = check_batch(ly, X, B, tgt_off, tgt_lab, nnz);
    if (rc) return rc;
    if (!(frac >= 0.f && frac <= 1.f)) return fail(FFSL_EINVAL, "frac must be in [0,1] (got %g)", (double)frac);
    const int32_t n = (int32_t)floor((double)frac * (double)ly.k + 1e-9);
    if (n > ly.d - ly.k)
        return fail(FFSL_EINVAL, "cannot regrow %d weights per row: only %d inactive columns", n, ly.d - ly.k);
    SweepCall c{};
    rc = check_adam(t, lr, beta1, beta2, eps, wd, &c.adam);
    if (rc) return rc;
    c.layer = &ly;
    c.X = X;
    c.B = B;
    c.tgt_off = tgt_off;
    c.tgt_lab = tgt_lab;
    c.nnz = nnz;
    c.s = s;
    c.mode = SWEEP_FUSED;
    c.loss_out = loss_out;
    c.dX_out = dX_out;
    c.flags = flags;
    c.stream = static_cast<hipStream_t>(stream);
    c.set_n = n;
    c.set_seed = seed;
    c.set_round = set_round;
    c.set_mask = pruned_mask_out;
    c.set_exhausted = exhausted_out;
    bool fused = false;
    c.set_fused = &fused;
    rc = launch_sweep(c);
    if (rc || fused) return rc;
    // the step's path has no fused SET: the same update as a separate call
    if (n == 0 && !pruned_mask_out) return FFSL_OK;
    return launch_set(ly, n, seed, set_round, pruned_mask_out, exhausted_out, static_cast<hipStream_t>(stream));
}

int ffsl_set_update(ffsl_layer *layer, float frac, uint64_t seed, uint64_t set_round, uint8_t *pruned_mask_out,
                    int32_t *exhausted_out, void *stream) {
    g_err.clear();
    if (!layer) return fail(FFSL_EINVAL, "layer is null");
    const Layer &ly = layer->ly;
    if (!(frac >= 0.f && frac <= 1.f)) return fail(FFSL_EINVAL, "frac must be in [0,1] (got %g)", (double)frac);
    const int32_t n = (int32_t)floor((double)frac * (double)ly.k + 1e-9);
    if (n > ly.d - ly.k)
        return fail(FFSL_EINVAL, "cannot regrow %d weights per row: only %d inactive columns", n, ly.d - ly.k);
    if (n == 0 && !pruned_mask_out) return FFSL_OK;
    return launch_set(ly, n, seed, set_round, pruned_mask_out, exhausted_out, static_cast<hipStream_t>(stream));
}

int ffsl_set_update_threshold(ffsl_layer *layer, float tau, uint64_t seed, uint64_t set_round,
                              uint8_t *pruned_mask_out, int32_t *exhausted_out, void *stream) {
    g_err.clear();
    if (!layer) return fail(FFSL_EINVAL, "layer is null");
    if (!(tau >= 0.f)) return fail(FFSL_EINVAL, "tau must be >= 0 (got %g)", (double)tau);
    return launch_set(layer->ly, 0, seed, set_round, pruned_mask_out, exhausted_out,
                      static_cast<hipStream_t>(stream), true, tau + 0.f);
}

int ffsl_set_timing_events(ffsl_layer *layer, void *start, void *stop) {
    g_err.clear();
    if (!layer) return fail(FFSL_EINVAL, "layer is null");
    if ((start == nullptr) != (stop == nullptr)) return fail(FFSL_EINVAL, "give both events or neither");
    layer->ly.ev_start = static_cast<hipEvent_t>(start);
    layer->ly.ev_stop = static_cast<hipEvent_t>(stop);
    return FFSL_OK;
}

size_t ffsl_topk_workspace_bytes(const ffsl_layer *layer, int32_t B_max, int32_t topk) {
    if (!layer || topk < 1 || (int64_t)topk > layer->ly.L) return 0;
    TopkPlan p{};
    if (!topk_shape(layer->ly, B_max, topk, &p)) return 0;
    return p.total;
}

int ffsl_infer_topk(ffsl_layer *layer, const void *X, int32_t B, int32_t topk, int32_t *top_labels,
                    float *top_scores, const int32_t *tgt_off, const int32_t *tgt_lab, int32_t nnz,
                    float *p_at_k, void *workspace, size_t workspace_bytes, void *stream) {
    g_err.clear();
    if (!layer) return fail(FFSL_EINVAL, "layer is null");
    const Layer &ly = layer->ly;
    if (!X) return fail(FFSL_EINVAL, "X is null");
    if (B < 1 || B > FFSL_MAX_B) return fail(FFSL_EINVAL, "B must be in [1,%d] (got %d)", FFSL_MAX_B, B);
    if (topk < 1 || topk > FFSL_MAX_TOPK || (int64_t)topk > ly.L)
        return fail(FFSL_EINVAL, "topk must be in [1, min(%d, L)] (got %d)", FFSL_MAX_TOPK, topk);
    if (!top_labels) return fail(FFSL_EINVAL, "top_labels is null");
    if (p_at_k) {
        if (!tgt_off) return fail(FFSL_EINVAL, "p_at_k needs tgt_off");
        if (nnz < 0) return fail(FFSL_EINVAL, "nnz must be >= 0");
        if (nnz > 0 && !tgt_lab) return fail(FFSL_EINVAL, "tgt_lab is null");
    }
    TopkPlan p{};
    if (!topk_shape(ly, B, topk, &p))
        return fail(FFSL_EUNSUPPORTED, "top-k inference does not support this shape (L=%lld, d=%d, %s)",
                    (long long)ly.L, ly.d, ly.vt == FFSL_BF16 ? "bf16" : "fp32");
    if (!workspace) return fail(FFSL_EINVAL, "workspace is null");
    if (reinterpret_cast<uintptr_t>(workspace) & 255u) return fail(FFSL_EINVAL, "workspace must be 256-byte aligned");
    if (workspace_bytes < p.total)
        return fail(FFSL_EINVAL, "workspace too small: %zu < %zu bytes", workspace_bytes, p.total);
    int rc = topk_grid(ly, &p);
    if (rc) return rc;
    return launch_topk(ly, X, B, topk, top_labels, top_scores, tgt_off, tgt_lab, p_at_k,
                       static_cast<char *>(workspace), p, static_cast<hipStream_t>(stream));
}

int ffsl_infer_topk_noalloc(ffsl_layer *layer, const void *X, int32_t B, int32_t topk, int32_t *top_labels,
                            float *top_scores, const int32_t *tgt_off, const int32_t *tgt_lab, int32_t nnz,
                            float *p_at_k, void *stream) {
    g_err.clear();
    if (!layer) return fail(FFSL_EINVAL, "layer is null");
    const Layer &ly = layer->ly;
    if (!X) return fail(FFSL_EINVAL, "X is null");
    if (B < 1 || B > FFSL_MAX_B) return fail(FFSL_EINVAL, "B must be in [1,%d] (got %d)", FFSL_MAX_B, B);
    if (topk < 1 || topk > FFSL_MAX_TOPK || (int64_t)topk > ly.L)
        return fail(FFSL_EINVAL, "topk must be in [1, min(%d, L)] (got %d)", FFSL_MAX_TOPK, topk);
    if (!top_labels) return fail(FFSL_EINVAL, "top_labels is null");
    if (p_at_k) {
        if (!tgt_off) return fail(FFSL_EINVAL, "p_at_k needs tgt_off");
        if (nnz < 0) return fail(FFSL_EINVAL, "nnz must be >= 0");
        if (nnz > 0 && !tgt_lab) return fail(FFSL_EINVAL, "tgt_lab is null");
    }
    TopkPlan p{};
    if (!topk_shape(ly, B, topk, &p))
        return fail(FFSL_EUNSUPPORTED, "top-k inference does not support this shape (L=%lld, d=%d, %s)",
                    (long long)ly.L, ly.d, ly.vt == FFSL_BF16 ? "bf16" : "fp32");
    if (p.total > (size_t)FFSL_TOPK_SCRATCH_BYTES)
        return fail(FFSL_EINVAL,
                    "B=%d, topk=%d need %zu bytes of scratch, more than the %zu of the no-allocation call "
                    "(use ffsl_infer_topk with a workspace, or a smaller batch)",
                    B, topk, p.total, (size_t)FFSL_TOPK_SCRATCH_BYTES);
    char *ws = nullptr;
    int rc = topk_scratch(ly.device, &ws);
    if (rc) return rc;
    rc = topk_grid(ly, &p);
    if (rc) return rc;
    return launch_topk(ly, X, B, topk, top_labels, top_scores, tgt_off, tgt_lab, p_at_k, ws, p,
                       static_cast<hipStream_t>(stream));
}

int ffsl_validate_indices(ffsl_layer *layer, int32_t *bad_rows_out, void *stream) {
    g_err.clear();
    if (!layer) return fail(FFSL_EINVAL, "layer is null");
    if (!bad_rows_out) return fail(FFSL_EINVAL, "bad_rows_out is null");
    return launch_validate(layer->ly, bad_rows_out, static_cast<hipStream_t>(stream));
}


size_t ffsl_dense_workspace_bytes(int32_t B_max, int32_t din, int32_t dout) {
    g_err.clear();
    if (check_dense_batch(B_max) || check_width("din", din, 65536) || check_width("dout", dout, 65536)) return 0;
    return dense_ws(B_max, din, dout).total;
}

int ffsl_dense_gelu_fwd(const void *X, int32_t B, int32_t din, int32_t dout, const void *W1, const float *c,
                        float *A_out, void *H_out, void *workspace, size_t workspace_bytes, void *stream) {
    g_err.clear();
    int rc;
    if ((rc = check_dense_batch(B)) || (rc = check_width("din", din, 65536)) ||
        (rc = check_width("dout", dout, 65536)) || (rc = check_aligned16("X", X)) ||
        (rc = check_aligned16("W1", W1)))
        return rc;
    if (!A_out || !H_out) return fail(FFSL_EINVAL, "A_out and H_out are required");
    if (workspace) {
        if (reinterpret_cast<uintptr_t>(workspace) & 255) return fail(FFSL_EINVAL, "workspace must be 256-byte aligned");
        const size_t need = dense_ws(B, din, dout).total;
        if (workspace_bytes < need)
            return fail(FFSL_EINVAL, "workspace too small: %zu < %zu bytes", workspace_bytes, need);
    }
    return launch_dense_gelu_fwd(static_cast<const uint16_t *>(X), B, din, dout, static_cast<const uint16_t *>(W1),
                                 c, A_out, static_cast<uint16_t *>(H_out), static_cast<char *>(workspace),
                                 static_cast<hipStream_t>(stream));
}

int ffsl_dense_gelu_bwd(const void *X, int32_t B, int32_t din, int32_t dout, const void *W1, const float *A,
                        const float *dH, float *dW1, float *dc, float *dX_out, uint32_t flags, void *workspace,
                        size_t workspace_bytes, void *stream) {
    g_err.clear();
    int rc;
    if ((rc = check_dense_batch(B)) || (rc = check_width("din", din, 65536)) ||
        (rc = check_width("dout", dout, 65536)) || (rc = check_aligned16("X", X)) ||
        (rc = check_aligned16("W1", W1)))
        return rc;
    if (!A || !dH || !dW1) return fail(FFSL_EINVAL, "A, dH and dW1 are required");
    if (!workspace) return fail(FFSL_EINVAL, "workspace is null");
    if ((reinterpret_cast<uintptr_t>(workspace) & 255u) != 0)
        return fail(FFSL_EINVAL, "workspace must be 256-byte aligned");
    const size_t need = dense_ws(B, din, dout).total;
    if (workspace_bytes < need)
        return fail(FFSL_EINVAL, "workspace too small: %zu < %zu bytes", workspace_bytes, need);
    return launch_dense_gelu_bwd(static_cast<const uint16_t *>(X), B, din, dout, static_cast<const uint16_t *>(W1),
                                 A, dH, dW1, dc, dX_out, (flags & FFSL_ACCUM_DX) != 0,
                                 static_cast<char *>(workspace), static_cast<hipStream_t>(stream));
}

size_t ffsl_aux_workspace_bytes(int32_t B_max, int32_t d, int32_t C) {
    g_err.clear();
    if (check_dense_batch(B_max) || check_width("d", d, 65536) || check_width("C", C, 1 << 20)) return 0;
    return aux_ws(B_max, d, C).total;
}

int ffsl_aux_bce_fwd_bwd(const void *X, int32_t B, int32_t d, int32_t C, int64_t n_labels, const void *Wa,
                         const float *ca,
                         const int32_t *tgt_off, const int32_t *tgt_lab, int32_t nnz, float s, float *loss_out,
                         float *dWa, float *dca, float *dX_out, float *logits_out, uint32_t flags, void *workspace,
                         size_t workspace_bytes, void *stream) {
    g_err.clear();
    int rc;
    if ((rc = check_dense_batch(B)) || (rc = check_width("d", d, 65536)) || (rc = check_width("C", C, 1 << 20)) ||
        (rc = check_aligned16("X", X)) || (rc = check_aligned16("Wa", Wa)))
        return rc;
    if (!tgt_off) return fail(FFSL_EINVAL, "tgt_off is null");
    if (nnz < 0) return fail(FFSL_EINVAL, "nnz must be >= 0");
    if (nnz > 0 && !tgt_lab) return fail(FFSL_EINVAL, "tgt_lab is null");
    if (n_labels < 1) return fail(FFSL_EINVAL, "n_labels must be >= 1 (got %lld)", (long long)n_labels);
    if (!dWa) return fail(FFSL_EINVAL, "dWa is required");
    if (!workspace) return fail(FFSL_EINVAL, "workspace is null");
    if ((reinterpret_cast<uintptr_t>(workspace) & 255u) != 0)
        return fail(FFSL_EINVAL, "workspace must be 256-byte aligned");
    const size_t need = aux_ws(B, d, C).total;
    if (workspace_bytes < need)
        return fail(FFSL_EINVAL, "workspace too small: %zu < %zu bytes", workspace_bytes, need);
    return launch_aux_bce(static_cast<const uint16_t *>(X), B, d, C, n_labels, static_cast<const uint16_t *>(Wa), ca,
                          tgt_off, tgt_lab, nnz, s, loss_out, dWa, dca, dX_out, logits_out, (flags & FFSL_ACCUM_DX) != 0,
                          (flags & FFSL_ACCUM_LOSS) != 0, static_cast<char *>(workspace),
                          static_cast<hipStream_t>(stream));
}

int ffsl_adam_dense(void *param, int32_t value_dtype, const float *grad, float *m, float *v, int64_t n, int64_t t,
                    float lr, float beta1, float beta2, float eps, float wd, void *stream) {
    g_err.clear();
    if (!param || !grad || !m || !v) return fail(FFSL_EINVAL, "param, grad, m and v are required");
    if (value_dtype != FFSL_F32 && value_dtype != FFSL_BF16)
        return fail(FFSL_EUNSUPPORTED, "value_dtype must be FFSL_F32 or FFSL_BF16");
    if (n < 1) return fail(FFSL_EINVAL, "n must be >= 1");
    AdamParams ap{};
    int rc = check_adam(t, lr, beta1, beta2, eps, wd, &ap);
    if (rc) return rc;
    int cu = 0;
    if ((rc = current_cu_count(&cu))) return rc;
    return launch_adam_flat(param, value_dtype, grad, m, v, n, ap, cu, static_cast<hipStream_t>(stream));
}

}  // extern "C"
