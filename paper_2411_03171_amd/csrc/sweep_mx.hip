// Fused training step of the fixed fan-in layer for bf16 values, fan-in 32,
// batches of up to 64 samples and input widths that are a multiple of 64
// (the gathered forward, BCE, dW, dbias, dX and Adam of Sec. 2.2, in one
// pass over the [L,k] arrays).
//
// Workgroup: 256 threads, one per CU, persistent over chunks of 16 label
// rows.  Sixteen lanes serve one row; lane u of a row owns batch rows
// b = 4u .. 4u+3.
//
//   LDS  Xs [d][64] bf16   the batch transposed (column i is 128 contiguous
//                          bytes), zero-padded past B
//        T  [d][16] bf16   the chunk's weights scattered densely by column
//        G  [64][16] bf16  the chunk's dlogits
//        Is, Ws           the chunk's index and weight rows
//
//   1. gather: for each slot, lane u reads the 8 bytes X[4u..4u+3, I[l,j]]
//      (16 lanes read one whole column, four columns per wave instruction,
//      which keeps LDS bank conflicts low);
//   2. forward: the b-pairs are repacked into slot pairs with v_perm and
//      reduced with v_dot2_f32_bf16 against the row's (W_j, W_j+1) pairs;
//   3. BCE loss and dlogits g for the lane's 4 batch rows;
//   4. dW partials over the lane's 4 rows with v_dot2 (g rounded to bf16),
//      then a reduce-scatter over the 16 lanes with DPP-fused adds.  Lane u
//      keeps slot r XOR K(u) in register r, K(u) = 2u0^6u1^12u2^24u3, which
//      makes every butterfly level one add with a mirror-pattern DPP source;
//      lane u ends with the full dW of slots K(u), K(u)+1;
//   5. Adam on those two slots, streaming W, m, v back to HBM;
//   6. dX: g and the old weights go to G and T, and the matrix cores add
//      G x T^T (64 x 16 by 16 x d) into a per-workgroup dX held in AGPRs for
//      the workgroup's whole life; it is written out once at the end.
#include "ffsl_internal.h"

namespace ffsl {

namespace {

constexpr int MX_THREADS = 256;
constexpr int MX_NLAB = 16;   // label rows per chunk
constexpr int MX_K = 32;      // fan-in of this path
constexpr int MX_NB = 64;     // padded batch
constexpr int MX_XS = 128;    // bytes per X column row in LDS

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

struct MxArgs {
    int64_t L;
    int32_t d, B, nnz;
    int64_t nchunks;
    const uint16_t *X;
    uint16_t *W;
    const int32_t *I;
    float *bias, *m, *v, *bm, *bv;
    const int32_t *tgt_b, *tgt_lab;
    float s;
    AdamParams adam;
    float *loss_part;
    float *dx_part;
    int want_loss;
};

__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), __builtin_bit_cast(bf16x2, b), c,
                                           false);
}

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
    bf16x2 p = {(__bf16)lo, (__bf16)hi};
    return __builtin_bit_cast(uint32_t, p);
}

// x + (value of register `y` in the DPP partner lane)
template <int CTRL>
__device__ __forceinline__ float add_dpp(float x, float y) {
    const int t = __builtin_amdgcn_update_dpp(0, __float_as_int(y), CTRL, 0xf, 0xf, false);
    return x + __int_as_float(t);
}

constexpr int DPP_ROW_MIRROR = 0x140;       // lane j <- 15 - j within 16
constexpr int DPP_ROW_HALF_MIRROR = 0x141;  // lane j <- 7 - j within 8
constexpr int DPP_QUAD_3210 = 0x1B;         // lane j <- j ^ 3 within 4
constexpr int DPP_QUAD_1032 = 0xB1;         // lane j <- j ^ 1 within 4

__device__ __forceinline__ int lane_key(int u) {
    return ((u & 1) ? 2 : 0) ^ ((u & 2) ? 6 : 0) ^ ((u & 4) ? 12 : 0) ^ ((u & 8) ? 24 : 0);
}

__device__ __forceinline__ float adam_step(float p, float g, float &mm, float &vv, const AdamParams &ap,
                                           float decay) {
    p *= decay;
    mm = ap.b1 * mm + (1.f - ap.b1) * g;
    vv = ap.b2 * vv + (1.f - ap.b2) * g * g;
    return p - ap.lr * (mm / ap.bc1) / (sqrtf(vv / ap.bc2) + ap.eps);
}

__global__ void __launch_bounds__(MX_THREADS, 1) k_sweep_mx(const MxArgs a) {
    extern __shared__ __align__(16) unsigned char lds[];
    const int d = a.d;
    unsigned char *Xs = lds;                                  // d * 128
    uint16_t *T = reinterpret_cast<uint16_t *>(lds + (size_t)d * MX_XS);   // d * 16
    uint16_t *G = T + (size_t)d * MX_NLAB;                    // 64 * 16
    int32_t *Is = reinterpret_cast<int32_t *>(G + MX_NB * MX_NLAB);       // 16 * 32
    uint32_t *Ws = reinterpret_cast<uint32_t *>(Is + MX_NLAB * MX_K);     // 16 * 16
    uint32_t *ym = Ws + MX_NLAB * (MX_K / 2);                 // 16 * 2
    float *red = reinterpret_cast<float *>(ym + MX_NLAB * 2); // 256

    const int tid = threadIdx.x;
    const int lab = tid >> 4, u = tid & 15;
    const int wave = tid >> 6, lane = tid & 63;
    const int K = lane_key(u);

    // stage X transposed (b fastest), zero past B; clear T
    {
        uint16_t *X16 = reinterpret_cast<uint16_t *>(Xs);
        for (int e = tid; e < d * MX_NB; e += MX_THREADS) {
            const int i = e >> 6, b = e & 63;
            X16[e] = b < a.B ? a.X[(size_t)b * d + i] : (uint16_t)0;
        }
        for (int e = tid; e < d * MX_NLAB / 2; e += MX_THREADS) reinterpret_cast<uint32_t *>(T)[e] = 0u;
    }

    // dX accumulators: 4 batch tiles x (d/64) column tiles of this wave
    const int ntiles = d / 64;  // column tiles of 16 per wave (d/4 columns per wave)
    f32x4 acc[4][12];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int nt = 0; nt < 12; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

    float loss_acc = 0.f;
    const float decay = 1.f - a.adam.lr * a.adam.wd;

    for (int64_t chunk = blockIdx.x; chunk < a.nchunks; chunk += gridDim.x) {
        const int64_t l0 = chunk * MX_NLAB;
        const int64_t l = l0 + lab;
        const bool valid = l < a.L;

        // stage the chunk's I and W rows; clear the positives mask
        {
            const int64_t base = l0 * MX_K;
            const int64_t lim = a.L * MX_K;
            const int e = 2 * tid;
            int2 iv = make_int2(0, 0);
            if (base + e + 1 < lim) iv = *reinterpret_cast<const int2 *>(a.I + base + e);
            *reinterpret_cast<int2 *>(Is + e) = iv;
            const int64_t wb = l0 * (MX_K / 2);
            uint32_t wv = 0u;
            if (wb + tid < a.L * (MX_K / 2)) wv = reinterpret_cast<const uint32_t *>(a.W)[wb + tid];
            Ws[tid] = wv;
            if (tid < MX_NLAB * 2) ym[tid] = 0u;
        }
        __syncthreads();
        for (int e = tid; e < a.nnz; e += MX_THREADS) {
            const int64_t ll = (int64_t)a.tgt_lab[e] - l0;
            const int b = a.tgt_b[e];
            if (ll >= 0 && ll < MX_NLAB && b >= 0 && b < MX_NB)
                atomicOr(&ym[ll * 2 + (b >> 5)], 1u << (b & 31));
        }
        __syncthreads();

        float g[4] = {0.f, 0.f, 0.f, 0.f};
        int32_t s0col = 0, s1col = 0;
        uint32_t wpair_own = 0u;
        if (valid) {
            // row data in the lane's slot order: register r <-> slot r ^ K
            int32_t idx[MX_K];
            uint32_t wp[MX_K / 2];
#pragma unroll
            for (int p = 0; p < MX_K / 2; ++p) {
                const int pp = p ^ (K >> 1);
                const int2 iv = *reinterpret_cast<const int2 *>(Is + lab * MX_K + 2 * pp);
                idx[2 * p] = min(max(iv.x, 0), d - 1);
                idx[2 * p + 1] = min(max(iv.y, 0), d - 1);
                wp[p] = Ws[lab * (MX_K / 2) + pp];
            }
            s0col = idx[0];
            s1col = idx[1];
            wpair_own = wp[0];
            // gather X[4u..4u+3, col] for every slot
            uint2 xg[MX_K];
#pragma unroll
            for (int r = 0; r < MX_K; ++r)
                xg[r] = *reinterpret_cast<const uint2 *>(Xs + (size_t)idx[r] * MX_XS + 8 * u);
            // forward: repack (b, b+1) pairs of two slots into slot pairs
            float z[4];
            const float bl = a.bias ? a.bias[l] : 0.f;
#pragma unroll
            for (int e = 0; e < 4; ++e) z[e] = 0.f;
#pragma unroll
            for (int p = 0; p < MX_K / 2; ++p) {
                const uint2 A = xg[2 * p], Bv = xg[2 * p + 1];
                z[0] = dot2(__builtin_amdgcn_perm(Bv.x, A.x, 0x05040100u), wp[p], z[0]);
                z[1] = dot2(__builtin_amdgcn_perm(Bv.x, A.x, 0x07060302u), wp[p], z[1]);
                z[2] = dot2(__builtin_amdgcn_perm(Bv.y, A.y, 0x05040100u), wp[p], z[2]);
                z[3] = dot2(__builtin_amdgcn_perm(Bv.y, A.y, 0x07060302u), wp[p], z[3]);
            }
            // BCE and dlogits for rows 4u..4u+3
            const uint32_t yw = ym[lab * 2 + (u >> 3)] >> ((4 * u) & 31);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int b = 4 * u + e;
                const float zz = z[e] + bl;
                const float y = ((yw >> e) & 1u) ? 1.f : 0.f;
                const float ex = __expf(-fabsf(zz));
                const float r = __builtin_amdgcn_rcpf(1.f + ex);
                const float sig = zz >= 0.f ? r : ex * r;
                if (b < a.B) {
                    if (a.want_loss) loss_acc += fmaxf(zz, 0.f) - zz * y + __logf(1.f + ex);
                    g[e] = a.s * (sig - y);
                }
            }
            // dW partials over the lane's rows, slot order r ^ K
            const uint32_t g01 = pack_bf16(g[0], g[1]), g23 = pack_bf16(g[2], g[3]);
            float pw[MX_K];
#pragma unroll
            for (int r = 0; r < MX_K; ++r) pw[r] = dot2(xg[r].y, g23, dot2(xg[r].x, g01, 0.f));
            // reduce-scatter over the 16 lanes of the row
#pragma unroll
            for (int r = 0; r < 16; ++r) pw[r] = add_dpp<DPP_ROW_MIRROR>(pw[r], pw[16 + r]);
#pragma unroll
            for (int r = 0; r < 8; ++r) pw[r] = add_dpp<DPP_ROW_HALF_MIRROR>(pw[r], pw[8 + r]);
#pragma unroll
            for (int r = 0; r < 4; ++r) pw[r] = add_dpp<DPP_QUAD_3210>(pw[r], pw[4 + r]);
#pragma unroll
            for (int r = 0; r < 2; ++r) pw[r] = add_dpp<DPP_QUAD_1032>(pw[r], pw[2 + r]);
            // Adam on slots K, K+1
            {
                const int64_t o = l * MX_K + K;
                const float2 mm2 = *reinterpret_cast<const float2 *>(a.m + o);
                const float2 vv2 = *reinterpret_cast<const float2 *>(a.v + o);
                float m0 = mm2.x, m1 = mm2.y, v0 = vv2.x, v1 = vv2.y;
                const float w0 = __uint_as_float(wpair_own << 16);
                const float w1 = __uint_as_float(wpair_own & 0xffff0000u);
                const float n0 = adam_step(w0, pw[0], m0, v0, a.adam, decay);
                const float n1 = adam_step(w1, pw[1], m1, v1, a.adam, decay);
                *reinterpret_cast<float2 *>(a.m + o) = make_float2(m0, m1);
                *reinterpret_cast<float2 *>(a.v + o) = make_float2(v0, v1);
                const uint32_t packed = (uint32_t)f32_to_bf16_bits(n0) | ((uint32_t)f32_to_bf16_bits(n1) << 16);
                reinterpret_cast<uint32_t *>(a.W)[o >> 1] = packed;
            }
        }
        // bias: sum of g over the 64 rows, lane u == 0 updates
        {
            float sg = (g[0] + g[1]) + (g[2] + g[3]);
            sg = add_dpp<DPP_ROW_MIRROR>(sg, sg);
            sg = add_dpp<DPP_ROW_HALF_MIRROR>(sg, sg);
            sg = add_dpp<DPP_QUAD_3210>(sg, sg);
            sg = add_dpp<DPP_QUAD_1032>(sg, sg);
            if (valid && u == 0 && a.bias) {
                float mm = a.bm[l], vv = a.bv[l];
                a.bias[l] = adam_step(a.bias[l], sg, mm, vv, a.adam, decay);
                a.bm[l] = mm;
                a.bv[l] = vv;
            }
        }
        // dX inputs: g (zero for invalid rows / padded samples) and the old weights
#pragma unroll
        for (int e = 0; e < 4; ++e) G[(4 * u + e) * MX_NLAB + lab] = f32_to_bf16_bits(g[e]);
        if (valid) {
            T[(size_t)s0col * MX_NLAB + lab] = (uint16_t)(wpair_own & 0xffffu);
            T[(size_t)s1col * MX_NLAB + lab] = (uint16_t)(wpair_own >> 16);
        }
        __syncthreads();
        // dX += G (64 x 16) * T^T (16 x d) on the matrix cores; this wave owns
        // columns [wave*d/4, (wave+1)*d/4)
        {
            const int col = lane & 15, kq = lane >> 4;
            bf16x4 af[4];
#pragma unroll
            for (int mt = 0; mt < 4; ++mt)
                af[mt] = *reinterpret_cast<const bf16x4 *>(G + (16 * mt + col) * MX_NLAB + 4 * kq);
            const int cbase = wave * (d / 4);
#pragma unroll
            for (int nt = 0; nt < 12; ++nt) {
                if (nt < ntiles) {
                    const bf16x4 bfr =
                        *reinterpret_cast<const bf16x4 *>(T + (size_t)(cbase + 16 * nt + col) * MX_NLAB + 4 * kq);
#pragma unroll
                    for (int mt = 0; mt < 4; ++mt)
                        acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(af[mt], bfr, acc[mt][nt], 0, 0, 0);
                }
            }
        }
        __syncthreads();
        if (valid) {
            T[(size_t)s0col * MX_NLAB + lab] = 0;
            T[(size_t)s1col * MX_NLAB + lab] = 0;
        }
    }

    // write this workgroup's dX partial [B][d]
    {
        float *P = a.dx_part + (size_t)blockIdx.x * a.B * d;
        const int col = lane & 15, kq = lane >> 4;
        const int cbase = wave * (d / 4);
#pragma unroll
        for (int nt = 0; nt < 12; ++nt) {
            if (nt < ntiles) {
                const int i = cbase + 16 * nt + col;
#pragma unroll
                for (int mt = 0; mt < 4; ++mt)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int b = 16 * mt + 4 * kq + r;
                        if (b < a.B) P[(size_t)b * d + i] = acc[mt][nt][r];
                    }
            }
        }
    }
    red[tid] = loss_acc;
    __syncthreads();
    for (int st = MX_THREADS / 2; st > 0; st >>= 1) {
        if (tid < st) red[tid] += red[tid + st];
        __syncthreads();
    }
    if (tid == 0) a.loss_part[blockIdx.x] = red[0];
}

}  // namespace

bool sweep_mx_eligible(const Layer &ly, int B, int mode) {
    return mode == SWEEP_FUSED && ly.vt == FFSL_BF16 && ly.k == MX_K && B <= MX_NB && ly.d % 64 == 0 &&
           ly.d <= 768;
}

size_t sweep_mx_lds(int d) {
    return (size_t)d * MX_XS + (size_t)d * MX_NLAB * 2 + MX_NB * MX_NLAB * 2 + MX_NLAB * MX_K * 4 +
           MX_NLAB * (MX_K / 2) * 4 + MX_NLAB * 2 * 4 + MX_THREADS * 4;
}

int launch_sweep_mx(const SweepCall &c, const int32_t *tgt_b, float *loss_part, float *dx_part, int *grid_out) {
    const Layer &ly = *c.layer;
    MxArgs a{};
    a.L = ly.L;
    a.d = ly.d;
    a.B = c.B;
    a.nnz = c.nnz;
    a.nchunks = (ly.L + MX_NLAB - 1) / MX_NLAB;
    a.X = static_cast<const uint16_t *>(c.X);
    a.W = static_cast<uint16_t *>(ly.W);
    a.I = ly.I;
    a.bias = ly.bias;
    a.m = ly.m;
    a.v = ly.v;
    a.bm = ly.bm;
    a.bv = ly.bv;
    a.tgt_b = tgt_b;
    a.tgt_lab = c.tgt_lab;
    a.s = c.s;
    a.adam = c.adam;
    a.loss_part = loss_part;
    a.dx_part = dx_part;
    a.want_loss = c.loss_out != nullptr;
    const size_t shm = sweep_mx_lds(ly.d);
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(k_sweep_mx),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
    if (e != hipSuccess) return fail(FFSL_EHIP, "hipFuncSetAttribute: %s", hipGetErrorString(e));
    const int grid = (int)std::min<int64_t>(a.nchunks, std::min(ly.max_parts, ly.num_cu));
    if (ly.ev_start) {
        e = hipEventRecord(ly.ev_start, c.stream);
        if (e != hipSuccess) return fail(FFSL_EHIP, "hipEventRecord: %s", hipGetErrorString(e));
    }
    hipLaunchKernelGGL(k_sweep_mx, dim3(grid), dim3(MX_THREADS), shm, c.stream, a);
    int rc = check_launch("sweep_mx");
    if (rc) return rc;
    if (ly.ev_stop) {
        e = hipEventRecord(ly.ev_stop, c.stream);
        if (e != hipSuccess) return fail(FFSL_EHIP, "hipEventRecord: %s", hipGetErrorString(e));
    }
    *grid_out = grid;
    return FFSL_OK;
}

}  // namespace ffsl
