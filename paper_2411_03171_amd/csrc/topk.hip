// Inference over the label space: the scores of a batch against every label
// row (the gathered forward of Sec. 2.2) and, per sample, the labels with the
// highest scores -- the prediction that Precision@k scores (appendix on
// evaluation metrics).  The scores never reach memory.
//
// k_topk_scan   One persistent workgroup per CU slot and batch tile.  The X
//               tile is staged in LDS as [d+1][BT] (column d is zero).  A
//               wave serves 4 label rows at a time, one per DPP row of 16
//               lanes; a lane serves SPL consecutive samples of the tile.  In
//               each round of 32 slots, lane u loads slots 2u and 2u+1 of its
//               row, and row_newbcast hands every slot pair to all 16 lanes of
//               the row, which gather their samples' X values from LDS.  Each
//               lane keeps, per sample, the KP best (score, label) keys it
//               has seen, sorted, in registers; a new key is inserted only
//               when it beats the last one (one wave-wide test per sample).
//               At the end the workgroup merges its 32 lists per sample into
//               one and writes it out.
// k_topk_merge  One workgroup per sample merges the lists of all
//               workgroups: K rounds of a block-wide maximum over the heads
//               of the sorted lists.  Writes labels, scores and relevance.
// k_patk        Precision@k averaged over the batch.
//
// Order of the result: descending score, equal scores by ascending label;
// NaN scores are never selected.  A (score, label) pair is one 64-bit key
// that orders exactly that way, so lists compare with one integer compare.

#include <mutex>

#include "ffsl_internal.h"
#include "sweep_dev.h"

// Scratch of the no-allocation inference call (ffsl_infer_topk_noalloc): the
// same workspace layout as ffsl_infer_topk's, in a file-scope device array
// that each GPU the library runs on holds until the process ends.  Host code
// never uses this name as an address: the device address comes from
// hipGetSymbolAddress, once per device (topk_scratch below).  Nothing in it
// needs to start at zero: the scan writes every list the merge reads, and the
// merge every relevance flag the P@k kernel reads.
// The array has external linkage (and default visibility): with internal
// linkage the device code object keeps it as a local symbol, which the
// runtime's symbol lookup cannot find.
__device__ __align__(256) __attribute__((visibility("default"))) unsigned char
    ffsl_topk_scratch[FFSL_TOPK_SCRATCH_BYTES];

namespace ffsl {

namespace {
constexpr int SCRATCH_MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void *g_scratch[SCRATCH_MAX_DEVICES];   // device address of `scratch` per device
}  // namespace

int topk_scratch(int device, char **ptr) {
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return fail(FFSL_EHIP, "hipGetDevice: %s", hipGetErrorString(e));
    if (cur != device)
        return fail(FFSL_EINVAL, "the layer lives on device %d but device %d is current", device, cur);
    if (device < 0 || device >= SCRATCH_MAX_DEVICES)
        return fail(FFSL_EUNSUPPORTED, "device %d: the no-allocation call supports devices 0..%d", device,
                    SCRATCH_MAX_DEVICES - 1);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[device]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(ffsl_topk_scratch));
        if (e != hipSuccess || !p)
            return fail(FFSL_EHIP, "hipGetSymbolAddress(ffsl_topk_scratch): %s", hipGetErrorString(e));
        g_scratch[device] = p;
    }
    *ptr = static_cast<char *>(g_scratch[device]);
    return FFSL_OK;
}
namespace {
using namespace fdev;

constexpr int TK_THREADS = 512;
constexpr int TK_WAVES = TK_THREADS / 64;
constexpr int TK_ROWS = 4;                     // label rows per wave per step
constexpr int TK_LISTS = TK_WAVES * TK_ROWS;   // lists per sample in a workgroup
constexpr int TK_MERGE_THREADS = 256;
constexpr int TK_AHEAD = 8;                    // steps of row data loaded ahead
constexpr int DPP_ROW_NEWBCAST = 0x150;        // + n: lane n of each DPP row to the whole row

struct TkArgs {
    const void *X;
    const void *W;
    const int32_t *I;
    const float *bias;
    int64_t L;
    int32_t B, d, k;
    int32_t nwg;       // workgroups per batch tile (gridDim.x)
    int32_t thr_off;   // LDS byte offset of the per-sample shared bounds, then
                       // of the best score of each of the 32 lists per sample
    int32_t K;         // labels wanted per sample
    int32_t idx16;     // I holds uint16 indices
    uint64_t *part;    // [B][nwg][KP] keys, sorted descending per list
};

// (score, label) as an integer ordered like (score descending, label
// ascending): the score's bits mapped to an order-preserving unsigned value
// (with -0 taken as +0) in the high word, the complemented label in the low
// word.  Key 0 marks an empty entry; no scored label maps to it.
__device__ __forceinline__ uint64_t score_key(float z, uint32_t l) {
    uint32_t u = __float_as_uint(z);
    u = u == 0x80000000u ? 0u : u;
    u ^= (u & 0x80000000u) ? 0xffffffffu : 0x80000000u;
    return ((uint64_t)u << 32) | (uint64_t)(~l);
}

// the score of a key (-inf for the empty key 0)
__device__ __forceinline__ float key_score(uint64_t key) {
    const uint32_t u = (uint32_t)(key >> 32);
    return u == 0u ? -INFINITY : __uint_as_float((u & 0x80000000u) ? (u ^ 0x80000000u) : ~u);
}

__device__ __forceinline__ int32_t key_label(uint64_t key) { return key ? (int32_t)(~(uint32_t)key) : -1; }

// Insert nk into the descending list kl, dropping the last entry; nk must
// beat kl[KP-1].
template <int KP>
__device__ __forceinline__ void list_insert(uint64_t (&kl)[KP], uint64_t nk) {
    bool lt[KP];
#pragma unroll
    for (int p = 0; p < KP; ++p) lt[p] = kl[p] < nk;
#pragma unroll
    for (int p = KP - 1; p > 0; --p) kl[p] = lt[p - 1] ? kl[p - 1] : (lt[p] ? nk : kl[p]);
    kl[0] = lt[0] ? nk : kl[0];
}

// Merge the sorted list src[0..KP) (in memory) into kl: entries are taken in
// order until one does not beat kl's last.
template <int KP, typename P>
__device__ __forceinline__ void list_merge(uint64_t (&kl)[KP], const P *src) {
    for (int p = 0; p < KP; ++p) {
        const uint64_t key = src[p];
        if (key <= kl[KP - 1]) break;
        list_insert(kl, key);
    }
}

template <int VT>
struct TkVal;
template <>
struct TkVal<FFSL_BF16> {
    using T = uint16_t;
    using Wp = uint32_t;   // the two weights of a slot pair, packed
};
template <>
struct TkVal<FFSL_F32> {
    using T = float;
    using Wp = float2;
};

// row data of one round for this lane as loaded: the columns of its two
// slots (d for a slot past k: column d of the tile is zero), the two weights
// and, in round 0, the row's bias.  Converted to LDS offsets only where used,
// so the loads of the next step stay in flight.
template <int VT>
struct TkRaw {
    int2 c;
    typename TkVal<VT>::Wp w;
    float bias;
};

template <int VT>
__device__ __forceinline__ void tk_load(const TkArgs &a, int64_t l0, int r, int g, int u, TkRaw<VT> &out) {
    using T = typename TkVal<VT>::T;
    const int64_t l = min(l0 + g, a.L - 1);
    const int s0 = 32 * r + 2 * u;
    const int64_t base = l * a.k;
    const T *W = static_cast<const T *>(a.W);
    if ((a.k & 1) == 0) {
        // even fan-in: the pair is two word loads (the same word twice with
        // 16-bit indices) and one load of the weights
        if (s0 < a.k) {
            const uint32_t ish = a.idx16 ? 1u : 2u;
            const char *ip = reinterpret_cast<const char *>(a.I) + ((size_t)(base + s0) << ish);
            out.c.x = *reinterpret_cast<const int32_t *>(ip);
            out.c.y = *reinterpret_cast<const int32_t *>(ip + (a.idx16 ? 0 : 4));
            out.w = *reinterpret_cast<const typename TkVal<VT>::Wp *>(W + base + s0);
        } else {
            out.c = a.idx16 ? make_int2(a.d | (a.d << 16), 0) : make_int2(a.d, a.d);
            if constexpr (VT == FFSL_BF16)
                out.w = 0u;
            else
                out.w = make_float2(0.f, 0.f);
        }
    } else {
        // odd fan-in: the two slots are loaded one by one and packed as an
        // even fan-in's pair would be
        const uint16_t *I16 = reinterpret_cast<const uint16_t *>(a.I);
        if (a.idx16) {
            const uint32_t c0 = s0 < a.k ? I16[base + s0] : (uint32_t)a.d;
            const uint32_t c1 = s0 + 1 < a.k ? I16[base + s0 + 1] : (uint32_t)a.d;
            out.c = make_int2((int)(c0 | (c1 << 16)), 0);
        } else {
            out.c.x = s0 < a.k ? a.I[base + s0] : a.d;
            out.c.y = s0 + 1 < a.k ? a.I[base + s0 + 1] : a.d;
        }
        if constexpr (VT == FFSL_BF16) {
            const uint32_t w0 = s0 < a.k ? W[base + s0] : 0u;
            const uint32_t w1 = s0 + 1 < a.k ? W[base + s0 + 1] : 0u;
            out.w = w0 | (w1 << 16);
        } else {
            out.w = make_float2(s0 < a.k ? W[base + s0] : 0.f, s0 + 1 < a.k ? W[base + s0 + 1] : 0.f);
        }
    }
    out.bias = (r == 0 && a.bias) ? a.bias[l] : 0.f;
}

// LDS offsets and weights of a round, ready for the broadcasts
template <int VT>
struct TkRound {
    int32_t o0, o1;
    typename TkVal<VT>::Wp w;
};

template <int VT, int SPL>
__device__ __forceinline__ TkRound<VT> tk_prep(const TkRaw<VT> &raw, int d, int idx16) {
    constexpr int COL = 16 * SPL * (int)sizeof(typename TkVal<VT>::T);   // bytes per LDS column
    // 16-bit indices: one word holds both slots
    const uint32_t r0 = idx16 ? ((uint32_t)raw.c.x & 0xffffu) : (uint32_t)raw.c.x;
    const uint32_t r1 = idx16 ? ((uint32_t)raw.c.x >> 16) : (uint32_t)raw.c.y;
    // indices outside [0,d) are clamped (the layer's precondition excludes
    // them); d itself is the zero column
    const uint32_t c0 = min(r0, (uint32_t)d), c1 = min(r1, (uint32_t)d);
    TkRound<VT> t;
    t.o0 = (int32_t)c0 * COL;
    t.o1 = (int32_t)c1 * COL;
    t.w = raw.w;
    return t;
}

template <int CTRL>
__device__ __forceinline__ int32_t bcast(int32_t x) {
    return __builtin_amdgcn_update_dpp(0, x, CTRL, 0xf, 0xf, true);
}

template <int VT, int SPL>
struct TkGather;
template <> struct TkGather<FFSL_BF16, 4> { using G = uint2; };
template <> struct TkGather<FFSL_BF16, 2> { using G = uint32_t; };
template <> struct TkGather<FFSL_BF16, 1> { using G = uint16_t; };
template <> struct TkGather<FFSL_F32, 4> { using G = float4; };
template <> struct TkGather<FFSL_F32, 2> { using G = float2; };
template <> struct TkGather<FFSL_F32, 1> { using G = float; };

// z[e] += w0 * xa[e] + w1 * xb[e] for the lane's samples
template <int VT, int SPL>
__device__ __forceinline__ void tk_fma(typename TkGather<VT, SPL>::G xa, typename TkGather<VT, SPL>::G xb,
                                       typename TkVal<VT>::Wp w, float (&z)[SPL]) {
    if constexpr (VT == FFSL_BF16) {
        if constexpr (SPL == 4) {
            z[0] = dot2(__builtin_amdgcn_perm(xb.x, xa.x, 0x05040100u), w, z[0]);
            z[1] = dot2(__builtin_amdgcn_perm(xb.x, xa.x, 0x07060302u), w, z[1]);
            z[2] = dot2(__builtin_amdgcn_perm(xb.y, xa.y, 0x05040100u), w, z[2]);
            z[3] = dot2(__builtin_amdgcn_perm(xb.y, xa.y, 0x07060302u), w, z[3]);
        } else if constexpr (SPL == 2) {
            z[0] = dot2(__builtin_amdgcn_perm(xb, xa, 0x05040100u), w, z[0]);
            z[1] = dot2(__builtin_amdgcn_perm(xb, xa, 0x07060302u), w, z[1]);
        } else {
            z[0] = dot2((uint32_t)xa | ((uint32_t)xb << 16), w, z[0]);
        }
    } else {
        const float *pa = reinterpret_cast<const float *>(&xa);
        const float *pb = reinterpret_cast<const float *>(&xb);
#pragma unroll
        for (int e = 0; e < SPL; ++e) z[e] = fmaf(w.y, pb[e], fmaf(w.x, pa[e], z[e]));
    }
}

template <int VT, int N>
__device__ __forceinline__ typename TkVal<VT>::Wp bcast_w(typename TkVal<VT>::Wp w) {
    if constexpr (VT == FFSL_BF16)
        return (uint32_t)bcast<DPP_ROW_NEWBCAST + N>((int32_t)w);
    else
        return make_float2(__int_as_float(bcast<DPP_ROW_NEWBCAST + N>(__float_as_int(w.x))),
                           __int_as_float(bcast<DPP_ROW_NEWBCAST + N>(__float_as_int(w.y))));
}

// slot pair N of the round (loaded by lane N of the row): gather this lane's
// samples of the two columns and accumulate
template <int VT, int SPL, int N>
__device__ __forceinline__ void tk_pair(const TkRound<VT> &c, int xl, float (&z)[SPL]) {
    using G = typename TkGather<VT, SPL>::G;
    extern __shared__ __align__(16) unsigned char tk_smem[];
    const G xa = *reinterpret_cast<const G *>(tk_smem + (xl + bcast<DPP_ROW_NEWBCAST + N>(c.o0)));
    const G xb = *reinterpret_cast<const G *>(tk_smem + (xl + bcast<DPP_ROW_NEWBCAST + N>(c.o1)));
    tk_fma<VT, SPL>(xa, xb, bcast_w<VT, N>(c.w), z);
}

// the round's slot pairs N .. npairs-1 of a partial round (npairs is uniform)
template <int VT, int SPL, int N = 0>
__device__ __forceinline__ void tk_round_part(const TkRound<VT> &c, int xl, int npairs,
                                              float (&z)[SPL]) {
    if constexpr (N < 16) {
        if (N < npairs) {
            tk_pair<VT, SPL, N>(c, xl, z);
            tk_round_part<VT, SPL, N + 1>(c, xl, npairs, z);
        }
    }
}

// all 16 slot pairs: every gather is issued first, so that they are all in
// flight together, then the products
template <int VT, int SPL, int N = 0>
__device__ __forceinline__ void tk_gather_all(const TkRound<VT> &c, int xl, typename TkGather<VT, SPL>::G (&xa)[16],
                                              typename TkGather<VT, SPL>::G (&xb)[16]) {
    if constexpr (N < 16) {
        using G = typename TkGather<VT, SPL>::G;
        extern __shared__ __align__(16) unsigned char tk_smem[];
        xa[N] = *reinterpret_cast<const G *>(tk_smem + (xl + bcast<DPP_ROW_NEWBCAST + N>(c.o0)));
        xb[N] = *reinterpret_cast<const G *>(tk_smem + (xl + bcast<DPP_ROW_NEWBCAST + N>(c.o1)));
        tk_gather_all<VT, SPL, N + 1>(c, xl, xa, xb);
    }
}

template <int VT, int SPL, int N = 0>
__device__ __forceinline__ void tk_fma_all(const TkRound<VT> &c, const typename TkGather<VT, SPL>::G (&xa)[16],
                                           const typename TkGather<VT, SPL>::G (&xb)[16], float (&z)[SPL]) {
    if constexpr (N < 16) {
        tk_fma<VT, SPL>(xa[N], xb[N], bcast_w<VT, N>(c.w), z);
        tk_fma_all<VT, SPL, N + 1>(c, xa, xb, z);
    }
}

template <int VT, int SPL>
__device__ __forceinline__ void tk_round_full(const TkRound<VT> &c, int xl, float (&z)[SPL]) {
    typename TkGather<VT, SPL>::G xa[16], xb[16];
    tk_gather_all<VT, SPL>(c, xl, xa, xb);
    tk_fma_all<VT, SPL>(c, xa, xb, z);
}

// Stage the batch tile transposed, Xs[c*BT + b], with a zero column d and
// zero samples past B, and clear the per-sample bounds and list bests.
//
// With SWZ (the transposing scan), the 8-byte pieces of samples 4p .. 4p+3
// of column c sit at piece p ^ tr_swz(c) of the column.
__device__ __forceinline__ int tr_swz(int c) { return (c >> 1) & 3; }

template <typename T, int BT, bool SWZ = false>
__device__ __forceinline__ void tk_stage(const TkArgs &a, int b0, int nb) {
    extern __shared__ __align__(16) unsigned char tk_smem[];
    const int tid = threadIdx.x, d = a.d;
    T *Xs = reinterpret_cast<T *>(tk_smem);
    const T *X = static_cast<const T *>(a.X) + (int64_t)b0 * d;
    if constexpr (SWZ && BT == 64 && sizeof(T) == 2) {
        if ((d & 7) == 0 && (reinterpret_cast<uintptr_t>(a.X) & 15) == 0) {
            // a wave takes 8 columns of its 64 samples: one 16-byte load per
            // lane (lane = sample) and eight 2-byte LDS writes, which fall
            // on distinct banks
            const int lane = tid & 63;
            for (int cc = tid >> 6; cc < d / 8; cc += TK_THREADS / 64) {
                uint4 v = make_uint4(0u, 0u, 0u, 0u);
                if (lane < nb) v = *reinterpret_cast<const uint4 *>(X + (int64_t)lane * d + 8 * cc);
                const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                for (int k = 0; k < 8; ++k) {
                    const int c = 8 * cc + k;
                    const int pos = (((lane >> 2) ^ tr_swz(c)) << 2) | (lane & 3);
                    Xs[c * BT + pos] = (T)(w[k >> 1] >> (16 * (k & 1)));
                }
            }
            if (tid < BT) Xs[d * BT + tid] = T(0);
            for (int i = tid; i < BT * (1 + TK_LISTS); i += TK_THREADS)
                reinterpret_cast<uint32_t *>(tk_smem + a.thr_off)[i] = 0u;
            __syncthreads();
            return;
        }
    }
    for (int b = 0; b < BT; ++b)
        for (int c = tid; c <= d; c += TK_THREADS) {
            const int pos = SWZ ? ((((b >> 2) ^ tr_swz(c)) << 2) | (b & 3)) : b;
            Xs[c * BT + pos] = (b < nb && c < d) ? X[(int64_t)b * d + c] : T(0);
        }
    for (int i = tid; i < BT * (1 + TK_LISTS); i += TK_THREADS)
        reinterpret_cast<uint32_t *>(tk_smem + a.thr_off)[i] = 0u;
    __syncthreads();
}

// Every wave turns the list bests of BT/8 samples into bounds: the K-th
// largest of a sample's 32 list bests (K distinct labels reach it).
template <int KP, int BT>
__device__ __forceinline__ void tk_list_bound(const uint32_t *lmax, uint32_t *shared_thr, int K, int wave,
                                              int lane) {
    if (lane < BT / TK_WAVES) {
        const int bt = wave * (BT / TK_WAVES) + lane;
        uint32_t best[KP];
#pragma unroll
        for (int p = 0; p < KP; ++p) best[p] = 0u;
        for (int i = 0; i < TK_LISTS; ++i) {
            uint32_t v = __hip_atomic_load(lmax + bt * TK_LISTS + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
#pragma unroll
            for (int p = 0; p < KP; ++p) {
                const uint32_t hi = max(best[p], v), lo = min(best[p], v);
                best[p] = hi;
                v = lo;
            }
        }
        uint32_t vk = 0u;
#pragma unroll
        for (int p = 0; p < KP; ++p) vk = p == K - 1 ? best[p] : vk;
        atomicMax(shared_thr + bt, vk);
    }
}

// The workgroup's 32 lists per sample, written to LDS as Ls[bt][list][KP],
// merged into one per sample and written to a.part.
template <int KP, int BT>
__device__ __forceinline__ void tk_merge_lists(const TkArgs &a, int b0, int nb) {
    extern __shared__ __align__(16) unsigned char tk_smem[];
    uint64_t *Ls = reinterpret_cast<uint64_t *>(tk_smem);
    __syncthreads();
    constexpr int TPS = TK_THREADS / BT;    // threads per sample
    constexpr int LPT = TK_LISTS / TPS;     // lists per thread in the first stage
    const int tid = threadIdx.x;
    const int bt = tid / TPS, sub = tid % TPS;
    uint64_t m[KP];
#pragma unroll
    for (int p = 0; p < KP; ++p) m[p] = 0;
    if constexpr (LPT > 0) {
        for (int i = 0; i < LPT; ++i) list_merge(m, Ls + ((size_t)bt * TK_LISTS + sub * LPT + i) * KP);
    }
    __syncthreads();
    uint64_t *Ms = Ls;   // [BT][TPS][KP]
#pragma unroll
    for (int p = 0; p < KP; ++p) Ms[((size_t)bt * TPS + sub) * KP + p] = m[p];
    __syncthreads();
    if (sub == 0 && bt < nb) {
        for (int i = 1; i < TPS; ++i) list_merge(m, Ms + ((size_t)bt * TPS + i) * KP);
        uint64_t *dst = a.part + ((size_t)(b0 + bt) * a.nwg + blockIdx.x) * KP;
#pragma unroll
        for (int p = 0; p < KP; ++p) dst[p] = m[p];
    }
}

template <int VT, int SPL, int KP>
__global__ __launch_bounds__(TK_THREADS) void k_topk_scan(TkArgs a) {
    using T = typename TkVal<VT>::T;
    extern __shared__ __align__(16) unsigned char tk_smem[];
    constexpr int BT = 16 * SPL;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, u = lane & 15;
    const int d = a.d;
    const int b0 = blockIdx.y * BT;
    const int nb = min(BT, a.B - b0);

    tk_stage<T, BT>(a, b0, nb);

    const int xl = u * SPL * (int)sizeof(T);   // LDS byte offset of this lane's samples of column 0
    // Per sample: the lane's sorted list, the score of its last entry once it
    // is full, and whether it is full.  Shared by the workgroup: per sample the
    // highest last-entry score of any full list (as an order-preserving
    // integer, 0 = none), a bound below which no label can still make the
    // sample's top KP; a score equal to it may, by its label, so it passes.
    uint64_t kl[SPL][KP];
    float thr[SPL], thr_sh[SPL];
    bool full[SPL];
#pragma unroll
    for (int e = 0; e < SPL; ++e) {
#pragma unroll
        for (int p = 0; p < KP; ++p) kl[e][p] = 0;
        thr[e] = -INFINITY;
        thr_sh[e] = -INFINITY;
        full[e] = false;
    }
    uint32_t *shared_thr = reinterpret_cast<uint32_t *>(tk_smem + a.thr_off);
    // lmax[bt * TK_LISTS + list]: best score of each list (0 = empty).  The
    // K-th largest of a sample's 32 list bests is also a bound: K distinct
    // labels reach it.
    uint32_t *lmax = shared_thr + BT;
    const int my_list = wave * TK_ROWS + g;

    const int rounds = (a.k + 31) >> 5;
    const int64_t stride = (int64_t)gridDim.x * TK_WAVES * TK_ROWS;
    int64_t l0 = ((int64_t)blockIdx.x * TK_WAVES + wave) * TK_ROWS;
    int r = 0;
    // ring of row data, TK_AHEAD steps of (row group, round) ahead
    TkRaw<VT> ring[TK_AHEAD];
    int64_t ll0 = l0;
    int lr = 0;
#pragma unroll
    for (int i = 0; i < TK_AHEAD; ++i) {
        if (ll0 < a.L) tk_load<VT>(a, ll0, lr, g, u, ring[i]);
        if (++lr == rounds) {
            lr = 0;
            ll0 += stride;
        }
    }
    float z[SPL];
#pragma unroll
    for (int e = 0; e < SPL; ++e) z[e] = 0.f;
    float zb = 0.f;
    bool more = l0 < a.L;
    int steps = 0;
    while (more) {
#pragma unroll
        for (int i = 0; i < TK_AHEAD; ++i) {
            if (more) {   // uniform
                const TkRaw<VT> cur = ring[i];
                if (ll0 < a.L) tk_load<VT>(a, ll0, lr, g, u, ring[i]);
                if (++lr == rounds) {
                    lr = 0;
                    ll0 += stride;
                }

                if (r == 0) zb = cur.bias;
                const TkRound<VT> rd = tk_prep<VT, SPL>(cur, d, a.idx16);
                const int npairs = min(16, (a.k - 32 * r + 1) >> 1);
                if (npairs == 16)
                    tk_round_full<VT, SPL>(rd, xl, z);
                else
                    tk_round_part<VT, SPL>(rd, xl, npairs, z);

                if (r == rounds - 1) {
                    const int64_t l = l0 + g;
                    const bool valid = l < a.L;
                    ++steps;
                    if ((steps & (steps - 1)) == 0 || (steps & 63) == 0)
                        tk_list_bound<KP, BT>(lmax, shared_thr, a.K, wave, lane);
                    if ((steps & 3) == 0) {
                        // refresh the workgroup's bounds for this lane's samples
#pragma unroll
                        for (int e = 0; e < SPL; ++e)
                            thr_sh[e] = key_score((uint64_t)__hip_atomic_load(shared_thr + u * SPL + e, __ATOMIC_RELAXED,
                                                                              __HIP_MEMORY_SCOPE_WORKGROUP)
                                                  << 32);
                    }
#pragma unroll
                    for (int e = 0; e < SPL; ++e) {
                        const float ze = z[e] + zb;
                        // this lane's rows come in ascending label order, so a
                        // score equal to its own last entry's loses the tie;
                        // NaN never enters
                        const bool hit = valid & (u * SPL + e < nb) & ((ze > thr[e]) | (!full[e] & (ze == ze))) &
                                         (ze >= thr_sh[e]);
                        if (__builtin_amdgcn_ballot_w64(hit) != 0) {
                            if (hit) {
                                list_insert(kl[e], score_key(ze, (uint32_t)l));
                                lmax[(u * SPL + e) * TK_LISTS + my_list] = (uint32_t)(kl[e][0] >> 32);
                                full[e] = kl[e][KP - 1] != 0;
                                if (full[e]) {
                                    thr[e] = key_score(kl[e][KP - 1]);
                                    atomicMax(shared_thr + u * SPL + e, (uint32_t)(kl[e][KP - 1] >> 32));
                                }
                            }
                        }
                        z[e] = 0.f;
                    }
                }
                if (++r == rounds) {
                    r = 0;
                    l0 += stride;
                }
                more = l0 < a.L;
            }
        }
    }

    // merge the workgroup's 32 lists per sample into one
    __syncthreads();   // the X tile is no longer read
    uint64_t *Ls = reinterpret_cast<uint64_t *>(tk_smem);
#pragma unroll
    for (int e = 0; e < SPL; ++e) {
        const int bt = u * SPL + e;
        uint64_t *dst = Ls + ((size_t)bt * TK_LISTS + wave * TK_ROWS + g) * KP;
#pragma unroll
        for (int p = 0; p < KP; ++p) dst[p] = kl[e][p];
    }
    tk_merge_lists<KP, BT>(a, b0, nb);
}

// ---------------------------------------------------------------------------
// k_topk_tr: the scan for bf16 values and fan-in 32 with transposing LDS
// gathers (ds_read_b64_tr_b16).  The tile is the same [d+1][64] X tile, a
// wave again serves 4 label rows per step, one per DPP row of 16 lanes, and a
// lane keeps the lists of 4 samples; only the gather differs.
//
// ds_read_b64_tr_b16 reads 8 bytes per lane at the lane's own address and
// hands them out transposed within each group of 16 lanes: lane 4m + t of
// the group receives element t of the 8 bytes read by lanes m, m+4, m+8 and
// m+12, in that order.  So when lane m + 4j reads samples 16m + 4p .. +3 of
// the column of slot 4sq + j, lane 4m + t receives sample 16m + 4p + t of the
// four slots 4sq .. 4sq+3: a slot-major quad that v_dot2 takes against the
// row's weight pairs as stored, with no repacking.  Per row a lane issues 32
// such reads (8 slot quads x 4 sample pieces p) and 64 dot2.
//
// Bank conflicts.  In the wave's row group g the sample pieces are visited
// in the order p = e ^ g (e = 0..3), so the four groups of one read touch
// different pieces.  Within a group, the 16 lanes read 4 pieces of each of 4
// random columns; a column's bank half follows its parity, so two columns of
// the same parity would land on the same banks.  The tile therefore keeps
// piece p of column c at p ^ ((c >> 1) & 3): columns then collide only when
// they agree in their three low bits.
//
// The rows' indices and weights are read straight from HBM with range-checked
// buffer loads, TR_AHEAD steps ahead (a ring in registers: 3 steps, 2 for
// lists of 8, which hold 64 registers): lane m + 4j loads the 8 indices of
// slots 4sq + j it gathers for (immediate offsets, no address arithmetic), and
// every lane of a row its 16 weight pairs.

struct TrRow {
    uint32_t c[8];    // columns of slots 4sq + j (sq = 0..7) as stored
    uint32_t w[16];   // the row's weights, pairs (4sq, 4sq+1) and (4sq+2, 4sq+3)
    float bias;
};

template <bool IDX16>
__device__ __forceinline__ void tr_load(Rsrc rI, Rsrc rW, Rsrc rB, uint32_t l, int j, TrRow &r) {
    if constexpr (IDX16) {
        const uint32_t base = l * 64u + 2u * (uint32_t)j;
#pragma unroll
        for (int sq = 0; sq < 8; ++sq) r.c[sq] = __builtin_amdgcn_raw_buffer_load_b16(rI, base + 8u * sq, 0, 0);
    } else {
        const uint32_t base = l * 128u + 4u * (uint32_t)j;
#pragma unroll
        for (int sq = 0; sq < 8; ++sq) r.c[sq] = ld32(rI, base + 16u * sq);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const auto v = __builtin_amdgcn_raw_buffer_load_b128(rW, l * 64u + 16u * i, 0, 0);
        r.w[4 * i] = v[0];
        r.w[4 * i + 1] = v[1];
        r.w[4 * i + 2] = v[2];
        r.w[4 * i + 3] = v[3];
    }
    r.bias = ldf(rB, l * 4u);
}

typedef short tr_v4s __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint2 tr_read(uint32_t off) {
    extern __shared__ __align__(16) unsigned char tk_smem[];
    const tr_v4s v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) tr_v4s *)((__attribute__((address_space(3))) unsigned char *)tk_smem +
                                                      off));
    return __builtin_bit_cast(uint2, v);
}

template <int KP, bool IDX16>
__global__ __launch_bounds__(TK_THREADS) void k_topk_tr(TkArgs a) {
    extern __shared__ __align__(16) unsigned char tk_smem[];
    constexpr int TR_AHEAD = KP >= 8 ? 2 : 3;
    constexpr int BT = 64, NS = 4;   // tile, samples per lane
    constexpr uint32_t COL = BT * 2; // bytes per LDS column
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, q = lane & 15;
    const int d = a.d;
    const int b0 = blockIdx.y * BT;
    const int nb = min(BT, a.B - b0);
    tk_stage<uint16_t, BT, true>(a, b0, nb);

    // as a gather source, lane q reads sample block ms of slot js of each quad;
    // as a receiver it holds samples 16*(q >> 2) + 4p + (q & 3)
    const int ms = q & 3, js = q >> 2;
    int smp[NS];   // the sample of accumulator e (piece p = e ^ g)
    uint32_t poff[NS];
#pragma unroll
    for (int e = 0; e < NS; ++e) {
        smp[e] = 16 * (q >> 2) + 4 * (e ^ g) + (q & 3);
        poff[e] = 32u * ms + 8u * (e ^ g);
    }

    uint64_t kl[NS][KP];
    float thr[NS], thr_sh[NS];
    bool full[NS];
#pragma unroll
    for (int e = 0; e < NS; ++e) {
#pragma unroll
        for (int p = 0; p < KP; ++p) kl[e][p] = 0;
        thr[e] = -INFINITY;
        thr_sh[e] = smp[e] < nb ? -INFINITY : INFINITY;
        full[e] = false;
    }
    uint32_t *shared_thr = reinterpret_cast<uint32_t *>(tk_smem + a.thr_off);
    uint32_t *lmax = shared_thr + BT;
    const int my_list = wave * TK_ROWS + g;

    const Rsrc rI = make_rsrc(a.I, (uint32_t)a.L * (IDX16 ? 64u : 128u));
    const Rsrc rW = make_rsrc(a.W, (uint32_t)a.L * 64u);
    const Rsrc rB = make_rsrc(a.bias, a.bias ? (uint32_t)a.L * 4u : 0u);
    const uint32_t L = (uint32_t)a.L;
    const uint32_t stride = gridDim.x * (uint32_t)TK_LISTS;
    uint32_t l0 = (blockIdx.x * TK_WAVES + wave) * TK_ROWS;   // the wave's row group this step
    TrRow ring[TR_AHEAD];
#pragma unroll
    for (int i = 0; i < TR_AHEAD; ++i) tr_load<IDX16>(rI, rW, rB, l0 + i * stride + g, js, ring[i]);
    int steps = 0;
    const int kk = a.K - 1;   // the entry whose score bounds this lane's list (K <= KP)

    // column byte offsets of a ring entry (an index outside [0, d) reads the
    // zero column d) and their piece swizzles
    auto cols = [&](const TrRow &r, uint32_t(&cb)[8], uint32_t(&cx)[8]) __attribute__((always_inline)) {
#pragma unroll
        for (int sq = 0; sq < 8; ++sq) {
            const uint32_t c = min(r.c[sq], (uint32_t)d);
            cb[sq] = c * COL;
            cx[sq] = 8u * (uint32_t)tr_swz((int)c);
        }
    };
    // the 16 transposing reads of slot quads 4h .. 4h+3
    auto issue = [&](const uint32_t(&cb)[8], const uint32_t(&cx)[8], int h, uint2(&xr)[4][NS])
        __attribute__((always_inline)) {
#pragma unroll
        for (int s4 = 0; s4 < 4; ++s4)
#pragma unroll
            for (int e = 0; e < NS; ++e) xr[s4][e] = tr_read(cb[4 * h + s4] + (poff[e] ^ cx[4 * h + s4]));
    };
    // their 32 products, the four samples' chains interleaved
    auto mac = [&](const uint2(&xr)[4][NS], const TrRow &r, int h, float(&z)[NS]) __attribute__((always_inline)) {
#pragma unroll
        for (int s4 = 0; s4 < 4; ++s4) {
            const int sq = 4 * h + s4;
#pragma unroll
            for (int e = 0; e < NS; ++e) z[e] = dot2(xr[s4][e].x, r.w[2 * sq], z[e]);
#pragma unroll
            for (int e = 0; e < NS; ++e) z[e] = dot2(xr[s4][e].y, r.w[2 * sq + 1], z[e]);
        }
    };

    // Software pipeline by half steps: the reads of the next half are in
    // flight while the products of the current one run.  TR_AHEAD steps per
    // iteration with no branch around the loads, so that each ring entry is
    // reloaded in place right after its last use; a step past the wave's last
    // row group reads zeros (range-checked loads) and selects nothing.
    uint32_t cb[8], cx[8];
    uint2 xa[4][NS], xb[4][NS];
    cols(ring[0], cb, cx);
    issue(cb, cx, 0, xa);
    while (l0 < L) {
#pragma unroll
        for (int i = 0; i < TR_AHEAD; ++i) {
            {
                const TrRow &cur = ring[i];
                issue(cb, cx, 1, xb);
                __builtin_amdgcn_sched_barrier(0);
                float z[NS];
#pragma unroll
                for (int e = 0; e < NS; ++e) z[e] = 0.f;
                mac(xa, cur, 0, z);
                cols(ring[(i + 1) % TR_AHEAD], cb, cx);
                issue(cb, cx, 0, xa);
                __builtin_amdgcn_sched_barrier(0);
                mac(xb, cur, 1, z);

                const uint32_t l = l0 + i * stride + g;
                const bool valid = l < L;
                ++steps;
                if ((steps & (steps - 1)) == 0 || (steps & 63) == 0)
                    tk_list_bound<KP, BT>(lmax, shared_thr, a.K, wave, lane);
                if ((steps & 3) == 0) {
#pragma unroll
                    for (int e = 0; e < NS; ++e)
                        if (smp[e] < nb)
                            thr_sh[e] = key_score((uint64_t)__hip_atomic_load(shared_thr + smp[e], __ATOMIC_RELAXED,
                                                                              __HIP_MEMORY_SCOPE_WORKGROUP)
                                                  << 32);
                }
                // Admission: this lane's rows come in ascending label order,
                // so a score equal to its own K-th entry's loses the tie.
                // Only the lane's best K can reach the sample's top K, so the
                // K-th entry bounds the list (the entries after it are kept
                // but no longer admit).  thr_sh is never NaN, so a NaN score
                // fails the first compare; a sample past B has thr_sh = +inf.
                float ze[NS];
                bool hit[NS];
                bool any = false;
#pragma unroll
                for (int e = 0; e < NS; ++e) {
                    ze[e] = z[e] + cur.bias;
                    hit[e] = valid & (ze[e] >= thr_sh[e]) & ((ze[e] > thr[e]) | !full[e]);
                    any |= hit[e];
                }
                if (__builtin_amdgcn_ballot_w64(any) != 0) {
#pragma unroll
                    for (int e = 0; e < NS; ++e) {
                        if (hit[e]) {
                            list_insert(kl[e], score_key(ze[e], l));
                            lmax[smp[e] * TK_LISTS + my_list] = (uint32_t)(kl[e][0] >> 32);
                            uint64_t kth = kl[e][KP - 1];
                            if (kk != KP - 1) {
#pragma unroll
                                for (int p = 0; p < KP - 1; ++p) kth = p == kk ? kl[e][p] : kth;
                            }
                            full[e] = kth != 0;
                            if (full[e]) {
                                thr[e] = key_score(kth);
                                atomicMax(shared_thr + smp[e], (uint32_t)(kth >> 32));
                            }
                        }
                    }
                }
            }
            tr_load<IDX16>(rI, rW, rB, l0 + (i + TR_AHEAD) * stride + g, js, ring[i]);
        }
        l0 += TR_AHEAD * stride;
    }

    // merge the workgroup's 32 lists per sample into one
    __syncthreads();   // the X tile is no longer read
    uint64_t *Ls = reinterpret_cast<uint64_t *>(tk_smem);
#pragma unroll
    for (int e = 0; e < NS; ++e) {
        uint64_t *dst = Ls + ((size_t)smp[e] * TK_LISTS + my_list) * KP;
#pragma unroll
        for (int p = 0; p < KP; ++p) dst[p] = kl[e][p];
    }
    tk_merge_lists<KP, BT>(a, b0, nb);
}

// block-wide maximum of one key per thread (TK_MERGE_THREADS threads)
__device__ __forceinline__ uint64_t block_max_key(uint64_t x, uint64_t *red) {
#pragma unroll
    for (int s = 32; s >= 1; s >>= 1) {
        const uint32_t lo = __shfl_xor((uint32_t)x, s, 64);
        const uint32_t hi = __shfl_xor((uint32_t)(x >> 32), s, 64);
        const uint64_t y = ((uint64_t)hi << 32) | lo;
        x = y > x ? y : x;
    }
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) red[wave] = x;
    __syncthreads();
    uint64_t mx = red[0];
#pragma unroll
    for (int w = 1; w < TK_MERGE_THREADS / 64; ++w) mx = red[w] > mx ? red[w] : mx;
    __syncthreads();
    return mx;
}

template <int KP>
__global__ __launch_bounds__(TK_MERGE_THREADS) void k_topk_merge(const uint64_t *part, int nwg, int K,
                                                                  int32_t *top_lab, float *top_sc,
                                                                  const int32_t *off, const int32_t *lab,
                                                                  uint8_t *rel) {
    __shared__ uint64_t red[TK_MERGE_THREADS / 64];
    __shared__ uint64_t win[16];
    const int b = blockIdx.x, tid = threadIdx.x;
    const uint64_t *pb = part + (size_t)b * nwg * KP;
    uint64_t kl[KP];
#pragma unroll
    for (int p = 0; p < KP; ++p) kl[p] = 0;
    if (tid < nwg) {
#pragma unroll
        for (int p = 0; p < KP; ++p) kl[p] = pb[(size_t)tid * KP + p];
    }
    for (int i = tid + TK_MERGE_THREADS; i < nwg; i += TK_MERGE_THREADS) list_merge(kl, pb + (size_t)i * KP);
    // K rounds: the best head wins and its list moves up by one
    for (int j = 0; j < K; ++j) {
        const uint64_t w = block_max_key(kl[0], red);
        if (w != 0 && kl[0] == w) {
#pragma unroll
            for (int p = 0; p < KP - 1; ++p) kl[p] = kl[p + 1];
            kl[KP - 1] = 0;
        }
        if (tid == 0) win[j] = w;
    }
    __syncthreads();
    if (tid < K) {
        const uint64_t w = win[tid];
        const int32_t l = key_label(w);
        top_lab[(size_t)b * K + tid] = l;
        if (top_sc) top_sc[(size_t)b * K + tid] = w ? key_score(w) : -INFINITY;
        if (rel) {
            uint8_t hit = 0;
            if (l >= 0)
                for (int e = off[b]; e < off[b + 1]; ++e)
                    if (lab[e] == l) {
                        hit = 1;
                        break;
                    }
            rel[(size_t)b * K + tid] = hit;
        }
    }
}

// out[j] = mean over samples of (1/(j+1)) * (relevant among the first j+1)
constexpr int TK_PATK_THREADS = 256;
__global__ __launch_bounds__(TK_PATK_THREADS) void k_patk(const uint8_t *rel, int B, int K, float *out) {
    __shared__ int32_t part[16][TK_PATK_THREADS];
    const int t = threadIdx.x;
    int32_t acc[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) acc[j] = 0;
    for (int b = t; b < B; b += TK_PATK_THREADS) {
        int32_t h = 0;
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            if (j < K) h += rel[(size_t)b * K + j];
            acc[j] += h;
        }
    }
#pragma unroll
    for (int j = 0; j < 16; ++j) part[j][t] = acc[j];
    __syncthreads();
    for (int s = TK_PATK_THREADS / 2; s > 0; s >>= 1) {
        if (t < s)
#pragma unroll
            for (int j = 0; j < 16; ++j) part[j][t] += part[j][t + s];
        __syncthreads();
    }
    if (t < K) out[t] = (float)((double)part[t][0] / ((double)(t + 1) * (double)B));
}

template <int VT, int SPL, int KP>
const void *scan_kernel() {
    if constexpr (SPL * KP <= (VT == FFSL_BF16 ? 32 : 16))
        return reinterpret_cast<const void *>(&k_topk_scan<VT, SPL, KP>);
    else
        return nullptr;
}

template <int VT, int SPL>
const void *pick_kp(int kp) {
    return kp == 1 ? scan_kernel<VT, SPL, 1>() : kp == 4 ? scan_kernel<VT, SPL, 4>()
         : kp == 8 ? scan_kernel<VT, SPL, 8>() : scan_kernel<VT, SPL, 16>();
}

template <int VT>
const void *pick_spl(int spl, int kp) {
    return spl == 4 ? pick_kp<VT, 4>(kp) : spl == 2 ? pick_kp<VT, 2>(kp) : pick_kp<VT, 1>(kp);
}

// the transposing scan keeps lists of exactly 1, 3 or 5 entries for the
// usual P@1, P@3 and P@5 (an insert costs one compare and select per entry),
// and of 8 otherwise
int tr_kp(int topk) { return topk == 1 ? 1 : topk <= 3 ? 3 : topk <= 5 ? 5 : 8; }

template <bool IDX16>
const void *tr_kernel_i(int kp) {
    return kp == 1 ? reinterpret_cast<const void *>(&k_topk_tr<1, IDX16>)
         : kp == 3 ? reinterpret_cast<const void *>(&k_topk_tr<3, IDX16>)
         : kp == 5 ? reinterpret_cast<const void *>(&k_topk_tr<5, IDX16>)
                   : reinterpret_cast<const void *>(&k_topk_tr<8, IDX16>);
}

const void *tr_kernel(int kp, bool idx16) { return idx16 ? tr_kernel_i<true>(kp) : tr_kernel_i<false>(kp); }

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

}  // namespace

bool topk_shape(const Layer &ly, int B, int topk, TopkPlan *p) {
    if (topk < 1 || topk > FFSL_MAX_TOPK || B < 1 || B > FFSL_MAX_B) return false;
    if (ly.L >= ((int64_t)1 << 31)) return false;
    const int elt = ly.vt == FFSL_BF16 ? 2 : 4;
    p->kp = topk == 1 ? 1 : topk <= 4 ? 4 : topk <= 8 ? 8 : 16;
    // list registers per lane: spl * kp keys (fp32 lanes also hold wider gathers)
    const int max_keys = ly.vt == FFSL_BF16 ? 32 : 16;
    int spl = 4;
    while (spl > 1 &&
           ((size_t)(ly.d + 1) * 16 * spl * elt > TOPK_XS_MAX || spl * p->kp > max_keys || 16 * (spl / 2) >= B))
        spl /= 2;
    if ((size_t)(ly.d + 1) * 16 * spl * elt > TOPK_XS_MAX) return false;
    p->spl = spl;
    p->bt = 16 * spl;
    p->tiles = (B + p->bt - 1) / p->bt;
    p->thr_off = (int)align256((size_t)(ly.d + 1) * p->bt * elt);
    p->lds = std::max((size_t)p->thr_off + sizeof(uint32_t) * p->bt * (1 + TK_LISTS),
                      (size_t)TK_THREADS * spl * p->kp * 8);
    p->scan = ly.vt == FFSL_BF16 ? pick_spl<FFSL_BF16>(spl, p->kp) : pick_spl<FFSL_F32>(spl, p->kp);
    if (ly.vt == FFSL_BF16 && ly.k == 32 && spl == 4 && p->kp <= 8 && ly.L < ((int64_t)1 << 25)) {
        p->kp = tr_kp(topk);
        p->lds = std::max((size_t)p->thr_off + sizeof(uint32_t) * p->bt * (1 + TK_LISTS),
                          (size_t)TK_THREADS * spl * p->kp * 8);
        p->scan = tr_kernel(p->kp, ly.idx16 != 0);
    }
    if (!p->scan) return false;
    p->nwg = 0;
    p->part = 0;
    p->rel = align256(sizeof(uint64_t) * (size_t)B * (size_t)ly.num_cu * TOPK_MAX_WG_PER_CU * p->kp);
    p->total = p->rel + align256((size_t)B * topk);
    return true;
}

int topk_grid(const Layer &ly, TopkPlan *p) {
    hipError_t e = hipFuncSetAttribute(p->scan, hipFuncAttributeMaxDynamicSharedMemorySize, (int)p->lds);
    if (e != hipSuccess) return fail(FFSL_EHIP, "hipFuncSetAttribute: %s", hipGetErrorString(e));
    int occ = 0;
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, p->scan, TK_THREADS, p->lds);
    if (e != hipSuccess) return fail(FFSL_EHIP, "hipOccupancyMaxActiveBlocksPerMultiprocessor: %s",
                                     hipGetErrorString(e));
    occ = std::max(1, std::min(occ, TOPK_MAX_WG_PER_CU));
    const int64_t need = (ly.L + TK_LISTS - 1) / TK_LISTS;
    p->nwg = (int)std::max<int64_t>(1, std::min<int64_t>((int64_t)ly.num_cu * occ, need));
    return FFSL_OK;
}

int launch_topk(const Layer &ly, const void *X, int B, int topk, int32_t *top_lab, float *top_sc,
                const int32_t *off, const int32_t *lab, float *p_at_k, char *ws, const TopkPlan &p,
                hipStream_t st) {
    TkArgs a{};
    a.X = X;
    a.W = ly.W;
    a.I = ly.I;
    a.idx16 = ly.idx16;
    a.bias = ly.bias;
    a.L = ly.L;
    a.B = B;
    a.d = ly.d;
    a.k = ly.k;
    a.nwg = p.nwg;
    a.thr_off = p.thr_off;
    a.K = topk;
    a.part = reinterpret_cast<uint64_t *>(ws + p.part);
    uint8_t *rel = p_at_k ? reinterpret_cast<uint8_t *>(ws + p.rel) : nullptr;
    hipLaunchKernelGGL(reinterpret_cast<void (*)(TkArgs)>(const_cast<void *>(p.scan)), dim3(p.nwg, p.tiles),
                       dim3(TK_THREADS), p.lds, st, a);
    int rc = check_launch("k_topk_scan");
    if (rc) return rc;
    switch (p.kp) {
    case 1: hipLaunchKernelGGL(k_topk_merge<1>, dim3(B), dim3(TK_MERGE_THREADS), 0, st, a.part, p.nwg, topk,
                               top_lab, top_sc, off, lab, rel); break;
    case 3: hipLaunchKernelGGL(k_topk_merge<3>, dim3(B), dim3(TK_MERGE_THREADS), 0, st, a.part, p.nwg, topk,
                               top_lab, top_sc, off, lab, rel); break;
    case 4: hipLaunchKernelGGL(k_topk_merge<4>, dim3(B), dim3(TK_MERGE_THREADS), 0, st, a.part, p.nwg, topk,
                               top_lab, top_sc, off, lab, rel); break;
    case 5: hipLaunchKernelGGL(k_topk_merge<5>, dim3(B), dim3(TK_MERGE_THREADS), 0, st, a.part, p.nwg, topk,
                               top_lab, top_sc, off, lab, rel); break;
    case 8: hipLaunchKernelGGL(k_topk_merge<8>, dim3(B), dim3(TK_MERGE_THREADS), 0, st, a.part, p.nwg, topk,
                               top_lab, top_sc, off, lab, rel); break;
    default: hipLaunchKernelGGL(k_topk_merge<16>, dim3(B), dim3(TK_MERGE_THREADS), 0, st, a.part, p.nwg, topk,
                                top_lab, top_sc, off, lab, rel); break;
    }
    rc = check_launch("k_topk_merge");
    if (rc || !p_at_k) return rc;
    hipLaunchKernelGGL(k_patk, dim3(1), dim3(TK_PATK_THREADS), 0, st, rel, B, topk, p_at_k);
    return check_launch("k_patk");
}

}  // namespace ffsl
