// Sweep kernels of the fixed fan-in layer: gathered forward, fused BCE,
// both backward products and (fused mode) Adam, in one pass over the
// [L,k] arrays (Sec. 2.2 of the paper: ELLPACK rows of exactly k weights).
//
// Mapping (general path):
//   - a persistent grid of workgroups, 256 threads each; a workgroup walks
//     chunks of 256 consecutive label rows, one row per thread, and keeps
//     the row's k weights, indices and (backward) gradient in registers;
//   - the batch is cut into tiles of Bt samples; a tile of X is staged in LDS
//     as fp32 [Bt][d] so every gather X[b, I[l,j]] is an LDS read;
//   - dX contributions of a tile are accumulated in an LDS fp32 [Bt][d]
//     array with LDS float adds and flushed, at a tile switch and at the
//     end, into a per-workgroup partial; a separate kernel sums the partials
//     in workgroup order.  The four waves add their contributions of a
//     sample one after the other (a barrier between them), and the adds of
//     one wave instruction that meet at one address are applied in lane
//     order, so every sum is formed in the same order in every run.  Tile
//     order alternates between consecutive chunks so a chunk starts on the
//     tile the previous one ended with.
//   - the loss is a per-thread sum reduced per workgroup in a fixed tree and
//     then over workgroups in order.
#include "ffsl_internal.h"

namespace ffsl {

namespace {

constexpr int SW_THREADS = 256;
constexpr int SW_MAXT = 1024;   // max batch tiles (B_max / Bt)
constexpr int YM_WORDS = 2;     // positives bitmask words per row (Bt <= 64)
constexpr int SW_MAX_BT = 64;

struct SweepArgs {
    int64_t L;
    int32_t d, k, B, Bt, T, nnz;
    int64_t nchunks;
    const void *X;
    void *W;
    const int32_t *I;
    float *bias, *m, *v, *bm, *bv, *dW, *dbias;
    const int32_t *tgt_b, *tgt_lab;
    float s;
    AdamParams adam;
    float *logits;
    float *loss_part;
    float *dx_part;
    int want_loss;
    int hinge;   // squared hinge instead of BCE
    int idx16;   // I holds uint16 indices
};

template <int KM>
__device__ __forceinline__ void load_row_idx(const int32_t *I, int64_t l, int k, int d, int (&idx)[KM],
                                             bool idx16) {
    if (idx16) {
        // 16-bit indices
        const uint16_t *I16 = reinterpret_cast<const uint16_t *>(I);
        if (k == KM && (KM % 8) == 0) {
            const uint4 *p = reinterpret_cast<const uint4 *>(I16 + l * KM);
#pragma unroll
            for (int q = 0; q < KM / 8; ++q) {
                const uint4 t = p[q];
                const uint32_t w[4] = {t.x, t.y, t.z, t.w};
#pragma unroll
                for (int h = 0; h < 4; ++h) {
                    idx[8 * q + 2 * h] = (int)(w[h] & 0xffffu);
                    idx[8 * q + 2 * h + 1] = (int)(w[h] >> 16);
                }
            }
        } else {
#pragma unroll
            for (int j = 0; j < KM; ++j) idx[j] = (j < k) ? (int)I16[l * k + j] : 0;
        }
    } else if (k == KM && (KM % 4) == 0) {
        const int4 *p = reinterpret_cast<const int4 *>(I + l * KM);
#pragma unroll
        for (int q = 0; q < KM / 4; ++q) {
            int4 t = p[q];
            idx[4 * q + 0] = t.x;
            idx[4 * q + 1] = t.y;
            idx[4 * q + 2] = t.z;
            idx[4 * q + 3] = t.w;
        }
    } else {
#pragma unroll
        for (int j = 0; j < KM; ++j) idx[j] = (j < k) ? I[l * k + j] : 0;
    }
    // Clamp so that a malformed index can never address outside the LDS tile.
#pragma unroll
    for (int j = 0; j < KM; ++j) idx[j] = min(max(idx[j], 0), d - 1);
}

template <int KM, int VT>
__device__ __forceinline__ void load_row_w(const void *Wv, int64_t l, int k, float (&w)[KM]) {
    if constexpr (VT == FFSL_BF16) {
        const uint16_t *W = static_cast<const uint16_t *>(Wv);
        if (k == KM && (KM % 8) == 0) {
            const uint4 *p = reinterpret_cast<const uint4 *>(W + l * KM);
#pragma unroll
            for (int q = 0; q < KM / 8; ++q) {
                uint4 t = p[q];
                uint32_t u[4] = {t.x, t.y, t.z, t.w};
#pragma unroll
                for (int h = 0; h < 4; ++h) {
                    w[8 * q + 2 * h + 0] = __uint_as_float(u[h] << 16);
                    w[8 * q + 2 * h + 1] = __uint_as_float(u[h] & 0xffff0000u);
                }
            }
        } else {
#pragma unroll
            for (int j = 0; j < KM; ++j) w[j] = (j < k) ? bf16_bits_to_f32(W[l * k + j]) : 0.f;
        }
    } else {
        const float *W = static_cast<const float *>(Wv);
        if (k == KM && (KM % 4) == 0) {
            const float4 *p = reinterpret_cast<const float4 *>(W + l * KM);
#pragma unroll
            for (int q = 0; q < KM / 4; ++q) {
                float4 t = p[q];
                w[4 * q + 0] = t.x;
                w[4 * q + 1] = t.y;
                w[4 * q + 2] = t.z;
                w[4 * q + 3] = t.w;
            }
        } else {
#pragma unroll
            for (int j = 0; j < KM; ++j) w[j] = (j < k) ? W[l * k + j] : 0.f;
        }
    }
}

__device__ __forceinline__ float adam_update(float p, float g, float &mm, float &vv,
                                             const AdamParams &ap, float decay) {
    p *= decay;
    mm = ap.b1 * mm + (1.f - ap.b1) * g;
    vv = ap.b2 * vv + (1.f - ap.b2) * g * g;
    const float mhat = mm / ap.bc1;
    const float vhat = vv / ap.bc2;
    return p - ap.lr * mhat / (sqrtf(vhat) + ap.eps);
}

template <int KM, int VT, int MODE>
__global__ void __launch_bounds__(SW_THREADS) k_sweep(const SweepArgs a) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    float *Xs = reinterpret_cast<float *>(smem_raw);
    float *dXs = Xs + (size_t)a.Bt * a.d;
    uint32_t *ym = reinterpret_cast<uint32_t *>(dXs + (MODE != SWEEP_FWD ? (size_t)a.Bt * a.d : 0));
    __shared__ float red[SW_THREADS];
    __shared__ uint8_t tflushed[SW_MAXT];

    using VTy = typename ValueT<VT>::T;
    const VTy *X = static_cast<const VTy *>(a.X);
    const int tid = threadIdx.x;
    const int d = a.d, k = a.k;
    float loss_acc = 0.f;
    int staged = -1;

    if (MODE != SWEEP_FWD) {
        for (int t = tid; t < SW_MAXT; t += SW_THREADS) tflushed[t] = 0;
        for (int e = tid; e < a.Bt * d; e += SW_THREADS) dXs[e] = 0.f;
    }

    // dX partial of this workgroup: [B][d]
    float *P = (MODE != SWEEP_FWD) ? a.dx_part + (size_t)blockIdx.x * a.B * d : nullptr;
    const float decay = 1.f - a.adam.lr * a.adam.wd;

    int ci = 0;
    for (int64_t chunk = blockIdx.x; chunk < a.nchunks; chunk += gridDim.x, ++ci) {
        const int64_t l0 = chunk * SW_THREADS;
        const int64_t l = l0 + tid;
        const bool valid = l < a.L;

        int idx[KM];
        float w[KM];
        float dw[KM];
        float bl = 0.f, db = 0.f;
        if (valid) {
            load_row_idx<KM>(a.I, l, k, d, idx, a.idx16 != 0);
            load_row_w<KM, VT>(a.W, l, k, w);
            if (a.bias) bl = a.bias[l];
        } else {
#pragma unroll
            for (int j = 0; j < KM; ++j) {
                idx[j] = 0;
                w[j] = 0.f;
            }
        }
#pragma unroll
        for (int j = 0; j < KM; ++j) dw[j] = 0.f;

        for (int tt = 0; tt < a.T; ++tt) {
            const int t = (ci & 1) ? (a.T - 1 - tt) : tt;
            const int b0 = t * a.Bt;
            const int bn = min(a.Bt, a.B - b0);
            __syncthreads();
            if (t != staged) {
                if (MODE != SWEEP_FWD && staged >= 0) {
                    const int sb0 = staged * a.Bt;
                    const int sbn = min(a.Bt, a.B - sb0);
                    const bool first = tflushed[staged] == 0;
                    for (int e = tid; e < sbn * d; e += SW_THREADS) {
                        const float val = dXs[e];
                        const size_t o = (size_t)sb0 * d + e;
                        P[o] = first ? val : P[o] + val;
                        dXs[e] = 0.f;
                    }
                    __syncthreads();
                    if (tid == 0) tflushed[staged] = 1;
                }
                for (int e = tid; e < bn * d; e += SW_THREADS)
                    Xs[e] = ValueT<VT>::load(X, (int64_t)b0 * d + e);
                staged = t;
            }
            for (int e = tid; e < SW_THREADS * YM_WORDS; e += SW_THREADS) ym[e] = 0u;
            __syncthreads();
            for (int e = tid; e < a.nnz; e += SW_THREADS) {
                const int32_t lab = a.tgt_lab[e];
                const int32_t b = a.tgt_b[e];
                if (lab >= l0 && lab < l0 + SW_THREADS && b >= b0 && b < b0 + bn) {
                    const int bb = b - b0;
                    atomicOr(&ym[(lab - l0) * YM_WORDS + (bb >> 5)], 1u << (bb & 31));
                }
            }
            __syncthreads();
            for (int bb = 0; bb < bn; ++bb) {
                float g = 0.f;
                if (valid) {
                    const float *xr = Xs + (size_t)bb * d;
                    float xg[KM];
                    float z = bl;
#pragma unroll
                    for (int j = 0; j < KM; ++j) {
                        if (j < k) {
                            xg[j] = xr[idx[j]];
                            z = fmaf(w[j], xg[j], z);
                        } else {
                            xg[j] = 0.f;
                        }
                    }
                    const float y = ((ym[tid * YM_WORDS + (bb >> 5)] >> (bb & 31)) & 1u) ? 1.f : 0.f;
                    // BCE with logits, or the squared hinge with yh = 2y - 1
                    const float yh = 2.f * y - 1.f;
                    const float hh = fmaxf(1.f - yh * z, 0.f);
                    const float e = a.hinge ? 0.f : expf(-fabsf(z));
                    if (MODE != SWEEP_BWD || a.want_loss)
                        loss_acc += a.hinge ? hh * hh : fmaxf(z, 0.f) - z * y + log1pf(e);
                    if (MODE == SWEEP_FWD && a.logits) a.logits[(int64_t)(b0 + bb) * a.L + l] = z;
                    if (MODE != SWEEP_FWD) {
                        const float r = 1.f / (1.f + e);
                        const float sig = z >= 0.f ? r : e * r;
                        g = a.hinge ? -2.f * a.s * yh * hh : a.s * (sig - y);
                        db += g;
#pragma unroll
                        for (int j = 0; j < KM; ++j)
                            if (j < k) dw[j] = fmaf(g, xg[j], dw[j]);
                    }
                }
                if (MODE != SWEEP_FWD) {
                    // dX: the waves add in turn (fixed order; see the header)
                    float *dxr = dXs + (size_t)bb * d;
                    for (int wv = 0; wv < SW_THREADS / 64; ++wv) {
                        if (valid && (tid >> 6) == wv) {
#pragma unroll
                            for (int j = 0; j < KM; ++j)
                                if (j < k) atomicAdd(&dxr[idx[j]], g * w[j]);
                        }
                        __syncthreads();
                    }
                }
            }
        }

        if (valid && MODE == SWEEP_BWD) {
#pragma unroll
            for (int j = 0; j < KM; ++j)
                if (j < k) a.dW[l * k + j] = dw[j];
            if (a.dbias) a.dbias[l] = db;
        }
        if (valid && MODE == SWEEP_FUSED) {
            VTy *W = static_cast<VTy *>(a.W);
#pragma unroll
            for (int j = 0; j < KM; ++j) {
                if (j < k) {
                    const int64_t o = l * k + j;
                    float mm = a.m[o], vv = a.v[o];
                    const float p = adam_update(w[j], dw[j], mm, vv, a.adam, decay);
                    a.m[o] = mm;
                    a.v[o] = vv;
                    ValueT<VT>::store(W, o, p);
                }
            }
            if (a.bias) {
                float mm = a.bm[l], vv = a.bv[l];
                a.bias[l] = adam_update(bl, db, mm, vv, a.adam, decay);
                a.bm[l] = mm;
                a.bv[l] = vv;
            }
        }
    }

    __syncthreads();
    if (MODE != SWEEP_FWD && staged >= 0) {
        const int sb0 = staged * a.Bt;
        const int sbn = min(a.Bt, a.B - sb0);
        const bool first = tflushed[staged] == 0;
        for (int e = tid; e < sbn * d; e += SW_THREADS) {
            const size_t o = (size_t)sb0 * d + e;
            P[o] = first ? dXs[e] : P[o] + dXs[e];
        }
    }
    red[tid] = loss_acc;
    __syncthreads();
    for (int s = SW_THREADS / 2; s > 0; s >>= 1) {
        if (tid < s) red[tid] += red[tid + s];
        __syncthreads();
    }
    if (tid == 0) a.loss_part[blockIdx.x] = red[0];
}

// sample index of every positive pair: tgt_b[e] = b for e in [off[b], off[b+1])
__global__ void k_targets_prep(const int32_t *off, int32_t B, int32_t nnz, int32_t *tgt_b) {
    const int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= B) return;
    const int e0 = max(0, min(off[b], nnz));
    const int e1 = max(e0, min(off[b + 1], nnz));
    for (int e = e0; e < e1; ++e) tgt_b[e] = b;
}

// loss (+)= s * sum of workgroup partials, in a fixed order (one workgroup of
// 256 threads)
__device__ __forceinline__ void loss_reduce_block(const float *part, int nparts, float s, float *out, int accum) {
    __shared__ float lred[256];
    float acc = 0.f;
    for (int p = threadIdx.x; p < nparts; p += 256) acc += part[p];
    lred[threadIdx.x] = acc;
    __syncthreads();
    for (int st = 128; st > 0; st >>= 1) {
        if ((int)threadIdx.x < st) lred[threadIdx.x] += lred[threadIdx.x + st];
        __syncthreads();
    }
    if (threadIdx.x == 0) out[0] = accum ? out[0] + s * lred[0] : s * lred[0];
}

// dX[e] (+)= sum over workgroup partials in workgroup order
__global__ void k_dx_reduce(const float *part, int nparts, int64_t n, float *out, int accum) {
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n;
         e += (int64_t)gridDim.x * blockDim.x) {
        float s = 0.f;
        for (int p = 0; p < nparts; ++p) s += part[(size_t)p * n + e];
        out[e] = accum ? out[e] + s : s;
    }
}

// The same sum for n divisible by 4: a workgroup owns 64 consecutive
// elements (16 float4 columns); its 16 lane groups take every 16th partial
// with independent 16-byte loads, and a fixed tree in LDS adds the groups.
// With lout set, one more workgroup past the dX ones reduces the loss
// partials (loss_reduce_block), so one launch finishes the step.
__global__ void __launch_bounds__(256) k_dx_reduce4(const float4 *part, int nparts, int64_t n4, float4 *out,
                                                    int accum, const float *lpart, int nl, float ls, float *lout,
                                                    int laccum) {
    if (lout && blockIdx.x == gridDim.x - 1) {
        loss_reduce_block(lpart, nl, ls, lout, laccum);
        return;
    }
    __shared__ float4 red[16][16];
    const int eg = threadIdx.x & 15, pg = threadIdx.x >> 4;
    const int64_t e = (int64_t)blockIdx.x * 16 + eg;
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    if (e < n4) {
        for (int p = pg; p < nparts; p += 16) {
            const float4 q = part[(size_t)p * n4 + e];
            s.x += q.x;
            s.y += q.y;
            s.z += q.z;
            s.w += q.w;
        }
    }
    red[pg][eg] = s;
    __syncthreads();
    if (pg == 0 && e < n4) {
        float4 t = red[0][eg];
        for (int g = 1; g < 16; ++g) {
            t.x += red[g][eg].x;
            t.y += red[g][eg].y;
            t.z += red[g][eg].z;
            t.w += red[g][eg].w;
        }
        if (accum) {
            const float4 o = out[e];
            t.x += o.x;
            t.y += o.y;
            t.z += o.z;
            t.w += o.w;
        }
        out[e] = t;
    }
}

// loss (+)= s * sum of workgroup partials, fixed order
__global__ void __launch_bounds__(256) k_loss_reduce(const float *part, int nparts, float s, float *out, int accum) {
    loss_reduce_block(part, nparts, s, out, accum);
}

template <int KM, int VT, int MODE>
int launch_mode(const SweepArgs &a, size_t shm, int grid, hipStream_t st) {
    auto kern = k_sweep<KM, VT, MODE>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
    if (e != hipSuccess) return fail(FFSL_EHIP, "hipFuncSetAttribute: %s", hipGetErrorString(e));
    hipLaunchKernelGGL(kern, dim3(grid), dim3(SW_THREADS), shm, st, a);
    return check_launch("sweep");
}

template <int KM, int VT>
int launch_km(int mode, const SweepArgs &a, size_t shm, int grid, hipStream_t st) {
    switch (mode) {
        case SWEEP_FWD: return launch_mode<KM, VT, SWEEP_FWD>(a, shm, grid, st);
        case SWEEP_BWD: return launch_mode<KM, VT, SWEEP_BWD>(a, shm, grid, st);
        default: return launch_mode<KM, VT, SWEEP_FUSED>(a, shm, grid, st);
    }
}

template <int VT>
int launch_vt(int mode, const SweepArgs &a, size_t shm, int grid, hipStream_t st) {
    if (a.k <= 8) return launch_km<8, VT>(mode, a, shm, grid, st);
    if (a.k <= 16) return launch_km<16, VT>(mode, a, shm, grid, st);
    if (a.k <= 32) return launch_km<32, VT>(mode, a, shm, grid, st);
    if (a.k <= 64) return launch_km<64, VT>(mode, a, shm, grid, st);
    return launch_km<128, VT>(mode, a, shm, grid, st);
}

}  // namespace

constexpr size_t LDS_BUDGET = 160 * 1024 - 4096;  // minus static arrays

int finish_sweep(const SweepCall &c, const float *loss_part, const float *dx_part, int nloss, int B, int d,
                 int ndx);

int launch_sweep(const SweepCall &c) {
    const Layer &ly = *c.layer;
    const int B = c.B, d = ly.d;
    const size_t per_b = (size_t)d * sizeof(float) * (c.mode == SWEEP_FWD ? 1 : 2);
    const size_t ym_bytes = SW_THREADS * YM_WORDS * sizeof(uint32_t);
    int Bt = (int)std::min<size_t>((LDS_BUDGET - ym_bytes) / per_b, (size_t)SW_MAX_BT);
    Bt = std::min(Bt, B);
    if (Bt < 1) return fail(FFSL_EUNSUPPORTED, "input width d=%d too large for the LDS tile", d);
    const int T = (B + Bt - 1) / Bt;
    if (T > SW_MAXT) return fail(FFSL_EUNSUPPORTED, "too many batch tiles (%d)", T);
    const size_t shm = (size_t)Bt * per_b + ym_bytes;

    const WsLayout wl = ws_layout(ly.L, d, ly.k, ly.vt, ly.B_max, ly.nnz_max, ly.max_parts);
    SweepArgs a{};
    a.L = ly.L;
    a.d = d;
    a.k = ly.k;
    a.B = B;
    a.Bt = Bt;
    a.T = T;
    a.nnz = c.nnz;
    a.nchunks = (ly.L + SW_THREADS - 1) / SW_THREADS;
    a.X = c.X;
    a.W = ly.W;
    a.I = ly.I;
    a.idx16 = ly.idx16;
    a.bias = ly.bias;
    a.m = ly.m;
    a.v = ly.v;
    a.bm = ly.bm;
    a.bv = ly.bv;
    a.dW = ly.dW;
    a.dbias = ly.dbias;
    a.tgt_b = reinterpret_cast<const int32_t *>(ly.ws + wl.tgt_b);
    a.tgt_lab = c.tgt_lab;
    a.s = c.s;
    a.adam = c.adam;
    a.logits = c.logits_out;
    a.loss_part = reinterpret_cast<float *>(ly.ws + wl.loss_part);
    a.dx_part = reinterpret_cast<float *>(ly.ws + wl.dx_part);
    a.want_loss = c.loss_out != nullptr;
    a.hinge = (c.flags & FFSL_LOSS_SQHINGE) ? 1 : 0;

    int grid = (int)std::min<int64_t>(a.nchunks, ly.max_parts);

    // the fused fast paths
    const bool use_wide = wl.has_xt && sweep_wide_eligible(ly, c.mode) && (B <= WD_PASS_B || wl.has_partial);
    const bool use_mx =
        !use_wide && wl.has_xt && sweep_mx_eligible(ly, B, c.mode) && (B <= MX_PASS_B || wl.has_partial);
    const bool fast = use_wide || use_mx;

    // the sample of every positive: the general path, and the fast paths when
    // the positives are too many for their sorted list in LDS
    if (c.nnz > 0 && (!fast || c.nnz > 1024)) {
        hipLaunchKernelGGL(k_targets_prep, dim3((B + 255) / 256), dim3(256), 0, c.stream, c.tgt_off, B,
                           c.nnz, const_cast<int32_t *>(a.tgt_b));
        int rc = check_launch("targets_prep");
        if (rc) return rc;
    }

    if (fast) {
        FastBufs fb{};
        fb.tgt_b = a.tgt_b;
        fb.keys = reinterpret_cast<const uint32_t *>(ly.ws + wl.keys);
        fb.xt = reinterpret_cast<const uint16_t *>(ly.ws + wl.xt);
        fb.loss_part = a.loss_part;
        fb.dx_part = a.dx_part;
        fb.dwp = reinterpret_cast<float *>(ly.ws + wl.dwp);
        fb.dbp = reinterpret_cast<float *>(ly.ws + wl.dbp);
        // the fan-in-32 path's list of rows left to SET on a row list, its
        // count cleared by the batch preparation
        fb.set_list = use_wide ? nullptr : reinterpret_cast<int32_t *>(ly.ws + wl.set_list);
        int rc = launch_batch_prep(static_cast<const uint16_t *>(c.X), B, d, c.tgt_off, c.tgt_lab, c.nnz, ly.L,
                                   use_wide ? WD_PASS_B : MX_PASS_B, reinterpret_cast<uint32_t *>(ly.ws + wl.keys),
                                   reinterpret_cast<uint16_t *>(ly.ws + wl.xt), c.set_n > 0 ? fb.set_list : nullptr,
                                   c.stream);
        if (rc) return rc;
        int passes = 1;
        rc = use_wide ? launch_sweep_wide(c, fb, &grid, &passes) : launch_sweep_mx(c, fb, &grid, &passes);
        if (rc) return rc;
        return finish_sweep(c, a.loss_part, a.dx_part, grid * passes, B, d, grid);
    }

    if (ly.ev_start) {
        hipError_t e = hipEventRecord(ly.ev_start, c.stream);
        if (e != hipSuccess) return fail(FFSL_EHIP, "hipEventRecord: %s", hipGetErrorString(e));
    }
    int rc = (ly.vt == FFSL_BF16) ? launch_vt<FFSL_BF16>(c.mode, a, shm, grid, c.stream)
                                  : launch_vt<FFSL_F32>(c.mode, a, shm, grid, c.stream);
    if (rc) return rc;
    if (ly.ev_stop) {
        hipError_t e = hipEventRecord(ly.ev_stop, c.stream);
        if (e != hipSuccess) return fail(FFSL_EHIP, "hipEventRecord: %s", hipGetErrorString(e));
    }
    return finish_sweep(c, a.loss_part, a.dx_part, grid, B, d, grid);
}

// loss and dX from the per-workgroup partials of a sweep: nloss loss partials,
// ndx dX partials of [B][d]
int finish_sweep(const SweepCall &c, const float *loss_part, const float *dx_part, int nloss, int B, int d,
                 int ndx) {
    int rc;
    const int laccum = (c.flags & FFSL_ACCUM_LOSS) ? 1 : 0;
    const bool want_dx = c.mode != SWEEP_FWD && c.dX_out;
    const int64_t n = (int64_t)B * d;
    const bool dx4 = want_dx && n % 4 == 0 && (reinterpret_cast<uintptr_t>(c.dX_out) & 15u) == 0;
    if (c.loss_out && !dx4) {
        hipLaunchKernelGGL(k_loss_reduce, dim3(1), dim3(256), 0, c.stream, loss_part, nloss, c.s, c.loss_out,
                           laccum);
        rc = check_launch("loss_reduce");
        if (rc) return rc;
    }
    if (want_dx) {
        const int accum = (c.flags & FFSL_ACCUM_DX) ? 1 : 0;
        if (dx4) {
            // the loss partials ride along in one extra workgroup
            const int64_t n4 = n / 4;
            const unsigned blocks = (unsigned)((n4 + 15) / 16) + (c.loss_out ? 1u : 0u);
            hipLaunchKernelGGL(k_dx_reduce4, dim3(blocks), dim3(256), 0, c.stream,
                               reinterpret_cast<const float4 *>(dx_part), ndx, n4,
                               reinterpret_cast<float4 *>(c.dX_out), accum, loss_part, nloss, c.s, c.loss_out,
                               laccum);
        } else {
            const int blocks = (int)std::min<int64_t>((n + 255) / 256, 4096);
            hipLaunchKernelGGL(k_dx_reduce, dim3(blocks), dim3(256), 0, c.stream, dx_part, ndx, n, c.dX_out,
                               accum);
        }
        rc = check_launch("dx_reduce");
        if (rc) return rc;
    }
    return FFSL_OK;
}

}  // namespace ffsl
