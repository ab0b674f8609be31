// Internal declarations of libffsl (HIP, gfx950).  Not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/ffsl.h"

namespace ffsl {

// ---------------------------------------------------------------- layer

struct Layer {
    int64_t L;
    int32_t d, k, vt, B_max, nnz_max;
    void *W;
    int32_t *I;      // int32 [L,k], or uint16 [L,k] bit patterns when idx16
    int idx16;       // 16-bit indices (d <= 65536)
    float *bias, *m, *v, *bm, *bv, *dW, *dbias;
    char *ws;
    size_t ws_bytes;
    int num_cu;      // compute units of the device the layer was created on
    int max_parts;   // per-workgroup partial buffers carved in the workspace
    int device;
    hipEvent_t ev_start, ev_stop;  // optional timing of the main sweep kernel
};

// Workspace carve-up (offsets in bytes, each 256-byte aligned).
struct WsLayout {
    size_t loss_part;   // float [max_parts * batch passes]
    size_t tgt_b;       // int32 [nnz_max]  sample of each positive pair
    size_t dx_part;     // float [max_parts][B_max][d]
    size_t dwp, dbp;    // float [L][k], [L]: dW / dbias carried between the
                        // batch passes of the fused fast path (B_max > 64, k = 32)
    size_t keys;        // uint32 [passes][1024]: each pass's sorted positives
    size_t xt;          // bf16 [passes][d][pass width]: the batch transposed per pass
    size_t set_list;    // int32 [1 + L]: the rows the fused step+SET sweep left
                        // to SET on a row list (count first), fan-in-32 path
    bool has_partial;
    bool has_xt;        // the shape may take a fused fast path (keys, xt allocated)
    size_t total;
};
// the workspace of a layer with values of type vt (FFSL_F32 / FFSL_BF16): the
// fast paths' buffers are carved only for shapes that can take a fast path
WsLayout ws_layout(int64_t L, int32_t d, int32_t k, int32_t vt, int32_t B_max, int32_t nnz_max, int max_parts);
// samples per pass of the fused fast path
constexpr int MX_PASS_B = 64;   // samples per pass of the fan-in-32 fast path
constexpr int WD_PASS_B = 16;   // samples per pass of the wide fan-in-64 fast path
// layers whose shape the wide fan-in-64 fast path serves (bf16 values)
inline bool wide_shape(int64_t L, int32_t d, int32_t k) {
    return k == 64 && d % 128 == 0 && d >= 128 && d <= 2048 && L < ((int64_t)1 << 24);
}
// layers whose shape the fan-in-32 fast path serves (bf16 values)
inline bool mx_shape(int64_t L, int32_t d, int32_t k) {
    return k == 32 && d % 128 == 0 && d >= 128 && d <= 768 && L < ((int64_t)1 << 25);
}
int max_parts_for(int num_cu);

// ---------------------------------------------------------------- errors

void set_error(const char *fmt, ...);
int fail(int code, const char *fmt, ...);
int check_launch(const char *what);

// ---------------------------------------------------------------- device helpers

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t h) {
    return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

// fp32 -> bf16 with round-to-nearest-even; NaN stays a quiet NaN.
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0u;
    u += 0x7fffu + ((u >> 16) & 1u);
    return static_cast<uint16_t>(u >> 16);
}

template <int VT> struct ValueT;
template <> struct ValueT<FFSL_F32> {
    using T = float;
    __device__ static __forceinline__ float load(const float *p, int64_t i) { return p[i]; }
    __device__ static __forceinline__ void store(float *p, int64_t i, float x) { p[i] = x; }
};
template <> struct ValueT<FFSL_BF16> {
    using T = uint16_t;
    __device__ static __forceinline__ float load(const uint16_t *p, int64_t i) {
        return bf16_bits_to_f32(p[i]);
    }
    __device__ static __forceinline__ void store(uint16_t *p, int64_t i, float x) {
        p[i] = f32_to_bf16_bits(x);
    }
};

// ---------------------------------------------------------------- launches

struct AdamParams {
    float lr, b1, b2, eps, wd;
    float bc1, bc2;   // 1 - b1^t, 1 - b2^t (computed in double on the host)
};

enum SweepMode { SWEEP_FWD = 0, SWEEP_BWD = 1, SWEEP_FUSED = 2 };

struct SweepCall {
    const Layer *layer;
    const void *X;
    int32_t B;
    const int32_t *tgt_off, *tgt_lab;
    int32_t nnz;
    float s;
    int mode;
    AdamParams adam;
    float *loss_out;
    float *logits_out;
    float *dX_out;
    uint32_t flags;
    hipStream_t stream;
    // SET after the update (ffsl_train_step_set): n pruned per row (0: none);
    // *set_fused is set when the sweep applied it
    int32_t set_n;
    uint64_t set_seed, set_round;
    uint8_t *set_mask;
    int32_t *set_exhausted;
    bool *set_fused;
};

int launch_sweep(const SweepCall &c);
// the fused fast paths' per-call batch preparation: sorted positives per pass
// (when nnz <= 1024) and the batch transposed per pass (batch_prep.hip)
// (and zero_word, when given, is set to 0: the deferred-row count of a fused
// step+SET sweep that follows)
int launch_batch_prep(const uint16_t *X, int32_t B, int32_t d, const int32_t *off, const int32_t *lab,
                      int32_t nnz, int64_t L, int pass_b, uint32_t *keys, uint16_t *xt, int32_t *zero_word,
                      hipStream_t st);
// what the fast sweeps read besides the layer and the call
struct FastBufs {
    const int32_t *tgt_b;     // sample of each positive (used when nnz > 1024)
    const uint32_t *keys;     // [passes][1024] sorted positives (nnz <= 1024)
    const uint16_t *xt;       // [passes][d][pass width] transposed batch
    float *loss_part, *dx_part, *dwp, *dbp;
    int32_t *set_list;        // [1 + L] rows left to SET on a row list (count first)
};
bool sweep_mx_eligible(const Layer &ly, int B, int mode);
int launch_sweep_mx(const SweepCall &c, const FastBufs &fb, int *grid_out, int *passes_out);
bool sweep_wide_eligible(const Layer &ly, int mode);
int launch_sweep_wide(const SweepCall &c, const FastBufs &fb, int *grid_out, int *passes_out);
int launch_adam(const Layer &ly, const AdamParams &p, hipStream_t st);
// SET; in threshold mode (tau >= 0) every slot with |W| < tau is pruned and n
// is ignored
int launch_set(const Layer &ly, int32_t n, uint64_t seed, uint64_t round,
               uint8_t *mask, int32_t *exhausted, hipStream_t st, bool threshold = false, float tau = 0.f);
// SET on the rows of list (list[0] = count, rows from list[1]); results as
// launch_set gives those rows
int launch_set_rows(const Layer &ly, int32_t n, uint64_t seed, uint64_t round, uint8_t *mask, int32_t *exhausted,
                    const int32_t *list, hipStream_t st);
int launch_validate(const Layer &ly, int32_t *bad_rows, hipStream_t st);
int launch_adam_flat(void *p, int vt, const float *g, float *m, float *v, int64_t n, const AdamParams &ap,
                     int num_cu, hipStream_t st);

// ---------------------------------------------------------------- inference

constexpr size_t TOPK_XS_MAX = 144 * 1024;   // LDS bytes of the staged X tile
constexpr int TOPK_MAX_WG_PER_CU = 4;         // scan workgroups per CU at most

struct TopkPlan {
    int spl;      // samples per lane (1, 2, 4)
    int kp;       // entries per lane list (1, 4, 8, 16)
    int bt;       // samples per batch tile (16 * spl)
    int tiles;    // batch tiles
    int nwg;      // scan workgroups per tile (set by topk_grid)
    size_t lds;   // dynamic LDS bytes of the scan kernel
    int thr_off;  // LDS byte offset of the per-sample bounds (after the X tile)
    const void *scan;
    size_t part, rel, total;   // workspace offsets and size
};
// shape of a top-k call (no HIP calls); false if the shape is unsupported
bool topk_shape(const Layer &ly, int B, int topk, TopkPlan *p);
// grid of the scan kernel on the current device
int topk_grid(const Layer &ly, TopkPlan *p);
// device address of the static scratch of the no-allocation inference call
// on `device`, which must be the current device (FFSL_TOPK_SCRATCH_BYTES bytes)
int topk_scratch(int device, char **ptr);
int launch_topk(const Layer &ly, const void *X, int B, int topk, int32_t *top_lab, float *top_sc,
                const int32_t *off, const int32_t *lab, float *p_at_k, char *ws, const TopkPlan &p,
                hipStream_t st);

// ---------------------------------------------------------------- dense parts

// workspace of the intermediate layer's backward (byte offsets, 256-aligned)
struct DenseWs {
    size_t fwd_part; // fp32 [splits, B_max, dout] split-K partials of the forward
    size_t dA16;     // bf16 [B_max, dout]
    size_t dx_part;  // fp32 [splits, B_max, din]
    size_t total;
};
// workspace of the auxiliary head
struct AuxWs {
    size_t dz16;       // bf16 [B_max, C] dlogits
    size_t loss_part;  // fp32, one per forward workgroup (64 samples x 64 clusters)
    size_t csum_part;  // fp32 [ceil(B_max/64), C] column sums of the dlogits per row block
    size_t dx_part;    // fp32 [splits, B_max, d]
    size_t total;
};
DenseWs dense_ws(int B_max, int din, int dout);
AuxWs aux_ws(int B_max, int d, int C);
int launch_dense_gelu_fwd(const uint16_t *X, int B, int din, int dout, const uint16_t *W1, const float *c,
                          float *A_out, uint16_t *H_out, char *ws, hipStream_t st);
int launch_dense_gelu_bwd(const uint16_t *X, int B, int din, int dout, const uint16_t *W1, const float *A,
                          const float *dH, float *dW1, float *dc, float *dX, bool accum, char *ws,
                          hipStream_t st);
int launch_aux_bce(const uint16_t *X, int B, int d, int C, int64_t n_labels, const uint16_t *Wa, const float *ca,
                   const int32_t *off, const int32_t *lab, int nnz, float s, float *loss, float *dWa, float *dca,
                   float *dX, float *Zout, bool accum_dx, bool accum_loss, char *ws, hipStream_t st);

}  // namespace ffsl
