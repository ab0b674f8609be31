// Unfused Adam / AdamW step over the layer's [L,k] weights and [L] bias,
// reading the gradients the backward sweep wrote (Kingma & Ba 2015,
// Algorithm 1; decoupled decay of Loshchilov & Hutter 2019).  Elementwise,
// grid-stride, 4 slots per thread per iteration.
#include "ffsl_internal.h"

namespace ffsl {

namespace {

__device__ __forceinline__ float adam_elem(float p, float g, float &mm, float &vv, const AdamParams &ap,
                                           float decay) {
    p *= decay;
    mm = ap.b1 * mm + (1.f - ap.b1) * g;
    vv = ap.b2 * vv + (1.f - ap.b2) * g * g;
    return p - ap.lr * (mm / ap.bc1) / (sqrtf(vv / ap.bc2) + ap.eps);
}

template <int VT>
__global__ void __launch_bounds__(256) k_adam(void *Wv, const float *g, float *m, float *v, int64_t n,
                                               float *bias, const float *dbias, float *bm, float *bv,
                                               int64_t L, AdamParams ap) {
    using VTy = typename ValueT<VT>::T;
    VTy *W = static_cast<VTy *>(Wv);
    const float decay = 1.f - ap.lr * ap.wd;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += stride) {
        float mm = m[e], vv = v[e];
        const float p = adam_elem(ValueT<VT>::load(W, e), g[e], mm, vv, ap, decay);
        m[e] = mm;
        v[e] = vv;
        ValueT<VT>::store(W, e, p);
    }
    if (bias) {
        for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < L; e += stride) {
            float mm = bm[e], vv = bv[e];
            bias[e] = adam_elem(bias[e], dbias[e], mm, vv, ap, decay);
            bm[e] = mm;
            bv[e] = vv;
        }
    }
}

}  // namespace

int launch_adam(const Layer &ly, const AdamParams &p, hipStream_t st) {
    const int64_t n = ly.L * ly.k;
    const int blocks = (int)std::min<int64_t>((n + 255) / 256, (int64_t)ly.num_cu * 16);
    if (ly.vt == FFSL_BF16)
        hipLaunchKernelGGL(k_adam<FFSL_BF16>, dim3(blocks), dim3(256), 0, st, ly.W, ly.dW, ly.m, ly.v, n,
                           ly.bias, ly.dbias, ly.bm, ly.bv, ly.L, p);
    else
        hipLaunchKernelGGL(k_adam<FFSL_F32>, dim3(blocks), dim3(256), 0, st, ly.W, ly.dW, ly.m, ly.v, n,
                           ly.bias, ly.dbias, ly.bm, ly.bv, ly.L, p);
    return check_launch("adam");
}

// the same update over a flat parameter array (the dense layers' weights and
// biases)
int launch_adam_flat(void *p, int vt, const float *g, float *m, float *v, int64_t n, const AdamParams &ap,
                     int num_cu, hipStream_t st) {
    const int blocks = (int)std::max<int64_t>(1, std::min<int64_t>((n + 255) / 256, (int64_t)num_cu * 16));
    if (vt == FFSL_BF16)
        hipLaunchKernelGGL(k_adam<FFSL_BF16>, dim3(blocks), dim3(256), 0, st, p, g, m, v, n, nullptr, nullptr,
                           nullptr, nullptr, (int64_t)0, ap);
    else
        hipLaunchKernelGGL(k_adam<FFSL_F32>, dim3(blocks), dim3(256), 0, st, p, g, m, v, n, nullptr, nullptr,
                           nullptr, nullptr, (int64_t)0, ap);
    return check_launch("adam_flat");
}

}  // namespace ffsl
