// Dense parts of the architecture around the sparse classifier (Sec. 2.3,
// Fig. 1 left): the wide intermediate layer H = GELU(X W1 + c) with its
// backward, and the auxiliary cluster classifier Za = X Wa + ca with its BCE
// loss and backward.  All products run on the matrix cores through one tiled
// GEMM (with a fused GELU epilogue for the intermediate layer):
//
//   C[M,N] = sum_k A(m,k) B(k,n),   A(m,k) = TA ? A[k*lda+m] : A[m*lda+k]
//                                   B(k,n) = TB ? B[n*ldb+k] : B[k*ldb+n]
//
// bf16 operands, fp32 accumulation.  A workgroup of 256 threads computes a
// 64 x 64 tile; each wave a 32 x 32 quarter with 2 x 2 v_mfma_f32_16x16x32_bf16
// per 32-deep slice.  K advances 128 at a time: both operands are staged into
// LDS K-contiguous (every fragment is one 16-byte LDS read whatever the source
// layout), and the next 128-deep tiles are loaded into registers while the
// matrix cores work on the current ones.  Long K (the dX products) is split
// over blockIdx.z into fp32 partials that a second kernel sums in a fixed
// order.  The auxiliary head's forward runs in one pass over K with its BCE
// in the epilogue: each workgroup marks its rows' cluster targets in LDS and
// writes the bf16 dlogits, its column sums of them and its loss sum.
#include <math.h>

#include <algorithm>

#include "ffsl_internal.h"

namespace ffsl {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int GT = 64;        // tile edge in M and N
constexpr int GK = 128;       // K per stage
constexpr int GKP = GK + 8;   // LDS row in elements (padded against bank conflicts)

enum Epi { EPI_STORE = 0, EPI_PARTIAL = 1, EPI_GELU = 2, EPI_BCE = 3 };

struct GemmArgs {
    const uint16_t *A;
    int64_t lda;
    const uint16_t *B;
    int64_t ldb;
    int M, N, K, kchunk;
    float *C;                 // STORE: C[m*N+n]; PARTIAL: C[(z*M+m)*N+n]; GELU: pre-activation
    const float *bias;        // GELU, BCE: per-column bias (nullable)
    uint16_t *H;              // GELU: bf16 activation; BCE: bf16 dlogits [M,N]
    // BCE (the auxiliary head, M = samples, N = clusters): targets as CSR
    // over the rows, label l counting for cluster l mod N when 0 <= l <
    // n_labels; dlogit g = sc (sigmoid(z) - y); per workgroup, the column
    // sums of g over its rows go to csum_part[blockIdx.y][n] and sc times its
    // loss sum to loss_part[blockIdx.y * gridDim.x + blockIdx.x]; the logits
    // to C when C is not null
    const int32_t *off, *lab;
    int64_t n_labels;
    float sc;
    float *csum_part, *loss_part;
};

// One operand's 64-row x 128-deep tile in flight: four 16-byte groups per
// thread.
struct Tile {
    uint4 q[4];
};

// Load a tile of one operand into registers.
//   KC = true : source stored row-major with k contiguous, src[r*ld + k];
//               thread t takes row (t>>4) + 16 p, k group (t&15)*8
//   KC = false: source stored with the rows contiguous,   src[k*ld + r];
//               thread t takes k (t>>3) + 32 p, row group (t&7)*8
// Out-of-range rows and k read as zero.  Callers guarantee that the contiguous
// extent (K for KC, the row count otherwise) is a multiple of 8 and that
// src and ld keep every 8-element group 16-byte aligned.
template <bool KC>
__device__ __forceinline__ void load_tile(Tile &t, const uint16_t *src, int64_t ld, int r0, int R, int k0,
                                          int kend, int tid) {
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        t.q[p] = make_uint4(0u, 0u, 0u, 0u);
        if (KC) {
            const int gr = r0 + (tid >> 4) + 16 * p, gk = k0 + (tid & 15) * 8;
            if (gr < R && gk < kend) t.q[p] = *reinterpret_cast<const uint4 *>(src + (int64_t)gr * ld + gk);
        } else {
            const int gk = k0 + (tid >> 3) + 32 * p, gr = r0 + (tid & 7) * 8;
            if (gk < kend && gr < R) t.q[p] = *reinterpret_cast<const uint4 *>(src + (int64_t)gk * ld + gr);
        }
    }
}

// Store a loaded tile into S[row][k] (K-contiguous).
template <bool KC>
__device__ __forceinline__ void store_tile(uint16_t (*S)[GKP], const Tile &t, int tid) {
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        if (KC) {
            *reinterpret_cast<uint4 *>(&S[(tid >> 4) + 16 * p][(tid & 15) * 8]) = t.q[p];
        } else {
            const int kr = (tid >> 3) + 32 * p, rc = (tid & 7) * 8;
            const uint32_t w[4] = {t.q[p].x, t.q[p].y, t.q[p].z, t.q[p].w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                S[rc + 2 * e][kr] = (uint16_t)(w[e] & 0xffffu);
                S[rc + 2 * e + 1][kr] = (uint16_t)(w[e] >> 16);
            }
        }
    }
}

__device__ __forceinline__ float gelu_cdf(float a) { return 0.5f * (1.f + erff(a * 0.70710678118654752f)); }

template <bool TA, bool TB, int EPI>
__global__ void __launch_bounds__(256) k_gemm(const GemmArgs g) {
    __shared__ __align__(16) uint16_t As[GT][GKP];
    __shared__ __align__(16) uint16_t Bs[GT][GKP];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1, col = lane & 15, kq = lane >> 4;
    const int m0 = blockIdx.y * GT, n0 = blockIdx.x * GT;
    const int kbeg = blockIdx.z * g.kchunk, kend = min(g.K, kbeg + g.kchunk);

    f32x4 acc[2][2];
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni) acc[mi][ni] = f32x4{0.f, 0.f, 0.f, 0.f};

    // BCE: bit j of ym[r] iff a positive of sample m0 + r falls in cluster n0 + j
    __shared__ unsigned long long ym[EPI == EPI_BCE ? GT : 1];
    if constexpr (EPI == EPI_BCE) {
        if (tid < GT) ym[tid] = 0ull;
        __syncthreads();
        const int r1 = min(g.M, m0 + GT);
        const int e0 = g.off[m0], e1 = g.off[r1];
        for (int e = e0 + tid; e < e1; e += 256) {
            const int l = g.lab[e];
            if (l < 0 || l >= g.n_labels) continue;
            const int cc = l % g.N - n0;
            if (cc < 0 || cc >= GT) continue;
            // the sample of entry e: the last row r with off[m0 + r] <= e
            int lo = 0, hi = r1 - m0 - 1;
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (g.off[m0 + mid] <= e) lo = mid;
                else hi = mid - 1;
            }
            atomicOr(&ym[lo], 1ull << cc);
        }
        __syncthreads();
    }

    Tile ta, tb;
    load_tile<!TA>(ta, g.A, g.lda, m0, g.M, kbeg, kend, tid);
    load_tile<TB>(tb, g.B, g.ldb, n0, g.N, kbeg, kend, tid);
    for (int k0 = kbeg; k0 < kend; k0 += GK) {
        store_tile<!TA>(As, ta, tid);
        store_tile<TB>(Bs, tb, tid);
        __syncthreads();
        if (k0 + GK < kend) {   // the next tiles load while this one computes
            load_tile<!TA>(ta, g.A, g.lda, m0, g.M, k0 + GK, kend, tid);
            load_tile<TB>(tb, g.B, g.ldb, n0, g.N, k0 + GK, kend, tid);
        }
#pragma unroll
        for (int ks = 0; ks < GK; ks += 32) {
            bf16x8 af[2], bv[2];
#pragma unroll
            for (int mi = 0; mi < 2; ++mi)
                af[mi] = *reinterpret_cast<const bf16x8 *>(&As[32 * wm + 16 * mi + col][ks + 8 * kq]);
#pragma unroll
            for (int ni = 0; ni < 2; ++ni)
                bv[ni] = *reinterpret_cast<const bf16x8 *>(&Bs[32 * wn + 16 * ni + col][ks + 8 * kq]);
#pragma unroll
            for (int mi = 0; mi < 2; ++mi)
#pragma unroll
                for (int ni = 0; ni < 2; ++ni)
                    acc[mi][ni] =
                        __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[mi], bv[ni], acc[mi][ni], 0, 0, 0);
        }
        __syncthreads();
    }

    if constexpr (EPI == EPI_BCE) {
        // z = acc + bias, its BCE term and dlogit; the column sums of g over
        // the tile's rows: each thread's rows, then the four lane groups of
        // a wave, then the two waves of a column half, in that order
        float csum[2] = {0.f, 0.f};
        float lsum = 0.f;
#pragma unroll
        for (int ni = 0; ni < 2; ++ni) {
            const int nl = 32 * wn + 16 * ni + col, n = n0 + nl;
            const float bn = (g.bias && n < g.N) ? g.bias[n] : 0.f;
#pragma unroll
            for (int mi = 0; mi < 2; ++mi)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int ml = 32 * wm + 16 * mi + 4 * kq + r, m = m0 + ml;
                    if (m >= g.M || n >= g.N) continue;
                    const float z = acc[mi][ni][r] + bn;
                    const float y = ((ym[ml] >> nl) & 1ull) ? 1.f : 0.f;
                    const float ex = expf(-fabsf(z));
                    lsum += fmaxf(z, 0.f) - z * y + log1pf(ex);
                    const float sig = z >= 0.f ? 1.f / (1.f + ex) : ex / (1.f + ex);
                    const float gg = g.sc * (sig - y);
                    const int64_t o = (int64_t)m * g.N + n;
                    g.H[o] = f32_to_bf16_bits(gg);
                    if (g.C) g.C[o] = z;
                    csum[ni] += gg;
                }
        }
        __shared__ float cred[2][GT];
        __shared__ float lred[4];
#pragma unroll
        for (int ni = 0; ni < 2; ++ni) {
            csum[ni] += __shfl_xor(csum[ni], 16);
            csum[ni] += __shfl_xor(csum[ni], 32);
            if (kq == 0) cred[wm][32 * wn + 16 * ni + col] = csum[ni];
        }
#pragma unroll
        for (int sh = 32; sh >= 1; sh >>= 1) lsum += __shfl_xor(lsum, sh);
        if (lane == 0) lred[wave] = lsum;
        __syncthreads();
        if (tid < GT && n0 + tid < g.N) g.csum_part[(int64_t)blockIdx.y * g.N + n0 + tid] = cred[0][tid] + cred[1][tid];
        if (tid == 0)
            g.loss_part[blockIdx.y * gridDim.x + blockIdx.x] = g.sc * ((lred[0] + lred[1]) + (lred[2] + lred[3]));
        return;
    }

    // accumulator element r of tile (mi, ni) is C[row 4*kq + r][column col]
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = m0 + 32 * wm + 16 * mi + 4 * kq + r;
                const int n = n0 + 32 * wn + 16 * ni + col;
                if (m >= g.M || n >= g.N) continue;
                const float x = acc[mi][ni][r];
                const int64_t o = (int64_t)m * g.N + n;
                if constexpr (EPI == EPI_STORE) {
                    g.C[o] = x;
                } else if constexpr (EPI == EPI_PARTIAL) {
                    g.C[(int64_t)blockIdx.z * g.M * g.N + o] = x;
                } else {
                    const float a = x + (g.bias ? g.bias[n] : 0.f);
                    g.C[o] = a;
                    g.H[o] = f32_to_bf16_bits(a * gelu_cdf(a));
                }
            }
}

// Column kernels: a workgroup owns 32 columns; its 8 row groups take every
// 8th row and a fixed tree in LDS adds the groups' sums.
__device__ __forceinline__ void column_sum_out(float (*red)[33], float sum, int c, int rg, int n, int N,
                                               float *out) {
    red[rg][c] = sum;
    __syncthreads();
    if (rg == 0 && n < N && out) {
        float t = red[0][c];
        for (int g = 1; g < 8; ++g) t += red[g][c];
        out[n] = t;
    }
}

// dA = dH * GELU'(A), GELU'(a) = Phi(a) + a phi(a); the bf16 copy feeds the
// two products, the fp32 column sums are dc.
__global__ void __launch_bounds__(256) k_gelu_bwd_cols(const float *A, const float *dH, int B, int N,
                                                       uint16_t *dA16, float *dc) {
    __shared__ float red[8][33];
    const int c = threadIdx.x & 31, rg = threadIdx.x >> 5;
    const int n = blockIdx.x * 32 + c;
    float sum = 0.f;
    if (n < N) {
        // eight rows' loads in flight at a time
        for (int b0 = rg; b0 < B; b0 += 64) {
            float av[8], hv[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int b = b0 + 8 * i;
                av[i] = b < B ? A[(int64_t)b * N + n] : 0.f;
                hv[i] = b < B ? dH[(int64_t)b * N + n] : 0.f;
            }
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int b = b0 + 8 * i;
                if (b < B) {
                    const float a = av[i];
                    const float pdf = 0.39894228040143268f * expf(-0.5f * a * a);
                    const float da = hv[i] * (gelu_cdf(a) + a * pdf);
                    dA16[(int64_t)b * N + n] = f32_to_bf16_bits(da);
                    sum += da;
                }
            }
        }
    }
    column_sum_out(red, sum, c, rg, n, N, dc);
}

// out[n] = sum_r part[r][n] over R row blocks, in order (out nullable); the
// last workgroup also adds the nl loss partials into *loss (nullable)
__global__ void __launch_bounds__(256) k_bce_finish(const float *part, int R, int N, float *out, const float *lpart,
                                                    int nl, float *loss, int accum) {
    const int n = blockIdx.x * blockDim.x + threadIdx.x;
    if (n < N && out) {
        float t = part[n];
        for (int r = 1; r < R; ++r) t += part[(int64_t)r * N + n];
        out[n] = t;
    }
    if (blockIdx.x == gridDim.x - 1 && loss) {
        __shared__ float red[256];
        float s = 0.f;
        for (int i = threadIdx.x; i < nl; i += 256) s += lpart[i];
        red[threadIdx.x] = s;
        __syncthreads();
        for (int st = 128; st > 0; st >>= 1) {
            if ((int)threadIdx.x < st) red[threadIdx.x] += red[threadIdx.x + st];
            __syncthreads();
        }
        if (threadIdx.x == 0) *loss = (accum ? *loss : 0.f) + red[0];
    }
}

// The intermediate layer's forward epilogue over split-K partials:
// A = c + sum_s P[s] (ascending s), H = bf16(GELU(A))
__global__ void __launch_bounds__(256) k_gelu_epi(const float *P, int S, int B, int N, const float *bias, float *A,
                                                  uint16_t *H) {
    const int64_t MN = (int64_t)B * N;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < MN; e += stride) {
        float a = P[e];
        for (int sp = 1; sp < S; ++sp) a += P[sp * MN + e];
        a += bias ? bias[e % N] : 0.f;
        A[e] = a;
        H[e] = f32_to_bf16_bits(a * gelu_cdf(a));
    }
}

// out[e] (+)= sum_z P[z][e], the split-K partials in ascending z
__global__ void __launch_bounds__(256) k_split_sum(const float *P, int S, int64_t MN, float *out, int accum) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < MN; e += stride) {
        float s = accum ? out[e] : 0.f;
        for (int z = 0; z < S; ++z) s += P[(int64_t)z * MN + e];
        out[e] = s;
    }
}

// *loss (+)= sum of n partials, one workgroup
__global__ void __launch_bounds__(256) k_sum_partials(const float *part, int n, float *loss, int accum) {
    __shared__ float red[256];
    float s = 0.f;
    for (int i = threadIdx.x; i < n; i += 256) s += part[i];
    red[threadIdx.x] = s;
    __syncthreads();
    for (int st = 128; st > 0; st >>= 1) {
        if ((int)threadIdx.x < st) red[threadIdx.x] += red[threadIdx.x + st];
        __syncthreads();
    }
    if (threadIdx.x == 0) *loss = (accum ? *loss : 0.f) + red[0];
}

template <bool TA, bool TB, int EPI>
int gemm(const GemmArgs &g, int splits, hipStream_t st) {
    dim3 grid((g.N + GT - 1) / GT, (g.M + GT - 1) / GT, splits);
    hipLaunchKernelGGL((k_gemm<TA, TB, EPI>), grid, dim3(256), 0, st, g);
    return check_launch("gemm");
}

size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }

// split count and K chunk of a long-K product: chunks of at least 256,
// at most 16 splits
void split_k(int K, int *splits, int *kchunk) {
    int s = std::max(1, std::min(16, K / 512));
    int kc = (K + s - 1) / s;
    kc = (kc + GK - 1) / GK * GK;
    s = (K + kc - 1) / kc;
    *splits = s;
    *kchunk = kc;
}

int blocks_for(int64_t n) { return (int)std::min<int64_t>((n + 255) / 256, 4096); }

// split count and K chunk of a forward product whose tiles alone would not
// fill the device: enough splits for about 1024 workgroups, chunks of at
// least 256
void split_fwd(int K, int tiles, int *splits, int *kchunk) {
    int s = std::max(1, std::min(K / 256, (1024 + tiles - 1) / tiles));
    int kc = (K + s - 1) / s;
    kc = (kc + GK - 1) / GK * GK;
    s = (K + kc - 1) / kc;
    *splits = s;
    *kchunk = kc;
}

}  // namespace

DenseWs dense_ws(int B_max, int din, int dout) {
    DenseWs w{};
    int S, kc;
    split_k(dout, &S, &kc);
    int Sf, kcf;
    split_fwd(din, ((dout + GT - 1) / GT) * ((B_max + GT - 1) / GT), &Sf, &kcf);
    size_t off = 0;
    w.fwd_part = off;
    off = al256(off + sizeof(float) * (size_t)Sf * B_max * dout);
    w.dA16 = off;
    off = al256(off + sizeof(uint16_t) * (size_t)B_max * dout);
    w.dx_part = off;
    off = al256(off + sizeof(float) * (size_t)S * B_max * din);
    w.total = off;
    return w;
}

AuxWs aux_ws(int B_max, int d, int C) {
    AuxWs w{};
    int S, kc;
    split_k(C, &S, &kc);
    size_t off = 0;
    w.dz16 = off;
    off = al256(off + sizeof(uint16_t) * (size_t)B_max * C);
    w.loss_part = off;
    off = al256(off + sizeof(float) * (size_t)((C + GT - 1) / GT) * ((B_max + GT - 1) / GT));
    w.csum_part = off;
    off = al256(off + sizeof(float) * (size_t)((B_max + GT - 1) / GT) * C);
    w.dx_part = off;
    off = al256(off + sizeof(float) * (size_t)S * B_max * d);
    w.total = off;
    return w;
}

int launch_dense_gelu_fwd(const uint16_t *X, int B, int din, int dout, const uint16_t *W1, const float *c,
                          float *A_out, uint16_t *H_out, char *ws, hipStream_t st) {
    GemmArgs g{};
    g.A = X;
    g.lda = din;
    g.B = W1;
    g.ldb = dout;
    g.M = B;
    g.N = dout;
    g.K = din;
    const int tiles = ((dout + GT - 1) / GT) * ((B + GT - 1) / GT);
    int S = 1, kc = din;
    if (ws) split_fwd(din, tiles, &S, &kc);
    if (S <= 1) {
        // one pass with the GELU epilogue in the product
        g.kchunk = (din + GK - 1) / GK * GK;
        g.C = A_out;
        g.bias = c;
        g.H = H_out;
        return gemm<false, false, EPI_GELU>(g, 1, st);
    }
    // split-K partials in the workspace, then the epilogue
    const DenseWs w = dense_ws(B, din, dout);
    float *P = reinterpret_cast<float *>(ws + w.fwd_part);
    g.kchunk = kc;
    g.C = P;
    int rc = gemm<false, false, EPI_PARTIAL>(g, S, st);
    if (rc) return rc;
    hipLaunchKernelGGL(k_gelu_epi, dim3(blocks_for((int64_t)B * dout)), dim3(256), 0, st, P, S, B, dout, c, A_out,
                       H_out);
    return check_launch("gelu_epi");
}

int launch_dense_gelu_bwd(const uint16_t *X, int B, int din, int dout, const uint16_t *W1, const float *A,
                          const float *dH, float *dW1, float *dc, float *dX, bool accum, char *ws,
                          hipStream_t st) {
    const DenseWs w = dense_ws(B, din, dout);
    uint16_t *dA16 = reinterpret_cast<uint16_t *>(ws + w.dA16);
    hipLaunchKernelGGL(k_gelu_bwd_cols, dim3((dout + 31) / 32), dim3(256), 0, st, A, dH, B, dout, dA16, dc);
    int rc = check_launch("gelu_bwd_cols");
    if (rc) return rc;
    // dW1[i,o] = sum_b X[b,i] dA[b,o]: A(m=i, k=b) = X[b*din+i] (TA), B(k=b, n=o) = dA[b*dout+o]
    GemmArgs g{};
    g.A = X;
    g.lda = din;
    g.B = dA16;
    g.ldb = dout;
    g.M = din;
    g.N = dout;
    g.K = B;
    g.kchunk = (B + GK - 1) / GK * GK;
    g.C = dW1;
    rc = gemm<true, false, EPI_STORE>(g, 1, st);
    if (rc || !dX) return rc;
    // dX[b,i] = sum_o dA[b,o] W1[i,o]: A(m=b, k=o) = dA[b*dout+o], B(k=o, n=i) = W1[i*dout+o] (TB)
    int S, kc;
    split_k(dout, &S, &kc);
    float *P = reinterpret_cast<float *>(ws + w.dx_part);
    GemmArgs h{};
    h.A = dA16;
    h.lda = dout;
    h.B = W1;
    h.ldb = dout;
    h.M = B;
    h.N = din;
    h.K = dout;
    h.kchunk = kc;
    h.C = P;
    rc = gemm<false, true, EPI_PARTIAL>(h, S, st);
    if (rc) return rc;
    const int64_t MN = (int64_t)B * din;
    hipLaunchKernelGGL(k_split_sum, dim3(blocks_for(MN)), dim3(256), 0, st, P, S, MN, dX, accum ? 1 : 0);
    return check_launch("split_sum");
}

int launch_aux_bce(const uint16_t *X, int B, int d, int C, int64_t n_labels, const uint16_t *Wa, const float *ca,
                   const int32_t *off, const int32_t *lab, int nnz, float s, float *loss, float *dWa, float *dca,
                   float *dX, float *Zout, bool accum_dx, bool accum_loss, char *ws, hipStream_t st) {
    const AuxWs w = aux_ws(B, d, C);
    uint16_t *dz16 = reinterpret_cast<uint16_t *>(ws + w.dz16);
    float *lp = reinterpret_cast<float *>(ws + w.loss_part);
    int rc;
    // Za = X Wa + ca in one pass over K, A(m=b, k=i) = X[b*d+i], B(k=i, n=c) = Wa[i*C+c],
    // with the BCE epilogue: the bf16 dlogits, their column sums per row block
    // of 64 and the loss per workgroup
    float *cp = reinterpret_cast<float *>(ws + w.csum_part);
    GemmArgs g{};
    g.A = X;
    g.lda = d;
    g.B = Wa;
    g.ldb = C;
    g.M = B;
    g.N = C;
    g.K = d;
    g.kchunk = (d + GK - 1) / GK * GK;
    g.C = Zout;
    g.bias = ca;
    g.H = dz16;
    g.off = off;
    g.lab = lab;
    g.n_labels = n_labels;
    g.sc = s;
    g.csum_part = cp;
    g.loss_part = lp;
    rc = gemm<false, false, EPI_BCE>(g, 1, st);
    if (rc) return rc;
    const int eblocks = (C + GT - 1) / GT, rblocks = (B + GT - 1) / GT;
    if (dca || loss) {
        hipLaunchKernelGGL(k_bce_finish, dim3((C + 255) / 256), dim3(256), 0, st, cp, rblocks, C, dca, lp,
                           eblocks * rblocks, loss, accum_loss ? 1 : 0);
        rc = check_launch("bce_finish");
        if (rc) return rc;
    }
    // dWa[i,c] = sum_b X[b,i] dZ[b,c]
    GemmArgs h{};
    h.A = X;
    h.lda = d;
    h.B = dz16;
    h.ldb = C;
    h.M = d;
    h.N = C;
    h.K = B;
    h.kchunk = (B + GK - 1) / GK * GK;
    h.C = dWa;
    rc = gemm<true, false, EPI_STORE>(h, 1, st);
    if (rc || !dX) return rc;
    // dXa[b,i] = sum_c dZ[b,c] Wa[i,c], added into dX when asked
    int S, kc;
    split_k(C, &S, &kc);
    float *P = reinterpret_cast<float *>(ws + w.dx_part);
    GemmArgs q{};
    q.A = dz16;
    q.lda = C;
    q.B = Wa;
    q.ldb = C;
    q.M = B;
    q.N = d;
    q.K = C;
    q.kchunk = kc;
    q.C = P;
    rc = gemm<false, true, EPI_PARTIAL>(q, S, st);
    if (rc) return rc;
    const int64_t MN = (int64_t)B * d;
    hipLaunchKernelGGL(k_split_sum, dim3(blocks_for(MN)), dim3(256), 0, st, P, S, MN, dX, accum_dx ? 1 : 0);
    return check_launch("split_sum");
}

}  // namespace ffsl
