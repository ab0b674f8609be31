// SET prune-and-regrow of the fixed fan-in layer (Sec. 2.1 of the paper:
// magnitude pruning, random regrowth of as many inactive weights; the
// hyperparameter appendix: random growth with zero initialisation), applied
// row by row so every row keeps exactly k weights (Sec. 2.2).
//
// A workgroup owns R consecutive label rows, one row per lane.  It first
// copies the R rows of I and W into LDS with coalesced 16-byte loads (the
// rows are contiguous in HBM), padded by one word per row so that lane t
// reading its own row hits bank t.  Each lane then:
//   - builds its keys (|W| bits, slot) and selects the n smallest with n
//     passes of "smallest key above the previous one" (keys are unique
//     because the slot is part of the key);
//   - marks the row's columns in a private bitmap in LDS laid out
//     [word][lane], so lanes never share a bank;
//   - draws candidates from Philox4x64-10 (Salmon et al., SC'11) keyed by the
//     seed and counted by (row, round, block), accepting a candidate whose
//     bitmap bit is clear and then marking it;
//   - writes the accepted columns to the pruned slots in ascending slot
//     order, with W = +0 and m = v = 0; all other slots are left untouched.
// Rows whose tiles would leave one small workgroup per CU (a fan-in of 64, a
// width of 2048, fp32 weights at d = 768) run k_set_reg instead, which holds
// each row in one lane's registers; see set_launch_km.
#include <algorithm>
#include <type_traits>

#include "sweep_dev.h"

namespace ffsl {

namespace {

constexpr int SET_MAX_ROWS = 256;
constexpr int SET_REG_ROWS = 256;  // rows (= lanes) per workgroup of k_set_reg
constexpr int SET_REG_ACC = 4;     // accepted columns k_set_reg keeps in registers
using fdev::philox4x64_10;
using fdev::SET_KEY_HI;

struct SetArgs {
    int64_t L;
    int32_t d, k, n, words;  // words = ceil(d/32) bitmap words per row
    int32_t R;               // rows (= threads) per workgroup
    void *W;
    int32_t *I;
    float *m, *v;
    uint8_t *mask;
    int32_t *exhausted;
    uint64_t seed, round;
    int64_t cap;
    // threshold mode: prune every slot with |W| < tau (tau_bits = fp32 bits of
    // tau >= 0; NaN weights are never below), so the count varies by row
    int32_t threshold;
    uint32_t tau_bits;
    int32_t idx16;   // I holds uint16 indices
};

// LDS layout (32-bit words): bitmap [words][R], Itile [R][k+1], Wtile [R][kw+1]
// where kw = k (fp32 W) or ceil(k/2) (bf16 W, two per word).
template <int VT>
__host__ __device__ inline int w_words(int k) {
    return VT == FFSL_BF16 ? (k + 1) / 2 : k;
}

template <int KM, int VT>
__global__ void __launch_bounds__(SET_MAX_ROWS) k_set(const SetArgs a) {
    extern __shared__ uint32_t lds[];
    const int R = a.R;
    const int k = a.k, d = a.d;
    const int kw = w_words<VT>(k);
    uint32_t *bitmap = lds;
    uint32_t *Itile = bitmap + (size_t)a.words * R;
    uint32_t *Wtile = Itile + (size_t)R * (k + 1);

    const int tid = threadIdx.x;
    const int64_t l0 = (int64_t)blockIdx.x * R;
    const int rows = (int)min<int64_t>(R, a.L - l0);

    // stage I and W rows (contiguous in HBM) into padded LDS rows
    {
        const uint32_t *Ig = reinterpret_cast<const uint32_t *>(a.I) + l0 * k;
        const int nI = rows * k;
        if (a.idx16) {
            const uint16_t *Ig16 = reinterpret_cast<const uint16_t *>(a.I) + l0 * k;
            if ((k & 7) == 0) {
                const uint4 *Ig4 = reinterpret_cast<const uint4 *>(Ig16);
                for (int e8 = tid; e8 < nI / 8; e8 += R) {
                    const uint4 q = Ig4[e8];
                    const int e = 8 * e8, r = e / k, j = e - r * k;
                    uint32_t *dst = Itile + r * (k + 1) + j;
                    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
                    for (int h = 0; h < 4; ++h) {
                        dst[2 * h] = w[h] & 0xffffu;
                        dst[2 * h + 1] = w[h] >> 16;
                    }
                }
            } else {
                for (int e = tid; e < nI; e += R) {
                    const int r = e / k, j = e - r * k;
                    Itile[r * (k + 1) + j] = Ig16[e];
                }
            }
        } else if ((k & 3) == 0) {
            const uint4 *Ig4 = reinterpret_cast<const uint4 *>(Ig);
            for (int e4 = tid; e4 < nI / 4; e4 += R) {
                const uint4 q = Ig4[e4];
                const int e = 4 * e4, r = e / k, j = e - r * k;
                uint32_t *dst = Itile + r * (k + 1) + j;
                dst[0] = q.x;
                dst[1] = q.y;
                dst[2] = q.z;
                dst[3] = q.w;
            }
        } else {
            for (int e = tid; e < nI; e += R) {
                const int r = e / k, j = e - r * k;
                Itile[r * (k + 1) + j] = Ig[e];
            }
        }
        if constexpr (VT == FFSL_BF16) {
            const uint16_t *Wg = static_cast<const uint16_t *>(a.W) + l0 * k;
            uint16_t *Wt = reinterpret_cast<uint16_t *>(Wtile);
            if ((k & 7) == 0) {
                const uint4 *Wg4 = reinterpret_cast<const uint4 *>(Wg);
                for (int e8 = tid; e8 < nI / 8; e8 += R) {
                    const uint4 q = Wg4[e8];
                    const int e = 8 * e8, r = e / k, j = e - r * k;
                    uint32_t *dst = Wtile + r * (kw + 1) + j / 2;
                    dst[0] = q.x;
                    dst[1] = q.y;
                    dst[2] = q.z;
                    dst[3] = q.w;
                }
            } else {
                for (int e = tid; e < nI; e += R) {
                    const int r = e / k, j = e - r * k;
                    Wt[2 * (r * (kw + 1)) + j] = Wg[e];
                }
            }
        } else {
            const uint32_t *Wg = static_cast<const uint32_t *>(a.W) + l0 * k;
            for (int e = tid; e < nI; e += R) {
                const int r = e / k, j = e - r * k;
                Wtile[r * (kw + 1) + j] = Wg[e];
            }
        }
    }
    __syncthreads();
    if (tid >= rows) return;  // no block-level synchronisation below
    const int64_t l = l0 + tid;

    int idx[KM];
    uint32_t key[KM];
#pragma unroll
    for (int j = 0; j < KM; ++j) {
        if (j < k) {
            idx[j] = (int)Itile[tid * (k + 1) + j];
            if constexpr (VT == FFSL_BF16) {
                const uint32_t pair = Wtile[tid * (kw + 1) + j / 2];
                key[j] = ((j & 1) ? (pair >> 16) : pair) & 0x7fffu;
            } else {
                key[j] = Wtile[tid * (kw + 1) + j] & 0x7fffffffu;
            }
        }
    }

    uint64_t pruned_lo = 0, pruned_hi = 0;  // slot bitmask, KM <= 128
    int n = a.n;
    if (a.threshold) {
        // |W| < tau compared as fp32 bit patterns of non-negative values
        n = 0;
#pragma unroll
        for (int j = 0; j < KM; ++j) {
            if (j < k) {
                const uint32_t mag = VT == FFSL_BF16 ? key[j] << 16 : key[j];
                if (mag < a.tau_bits) {
                    if (j < 64) pruned_lo |= 1ull << j;
                    else pruned_hi |= 1ull << (j - 64);
                    ++n;
                }
            }
        }
    } else if (n <= 4) {
        // the n smallest of the unique keys (|W| bits, slot) held in sorted
        // order by an insertion network of depth 4 over all k slots
        // bf16 keys (15 bits) and the slot fit one 32-bit word
        using KeyT = typename std::conditional<VT == FFSL_BF16, uint32_t, uint64_t>::type;
        const KeyT top = (KeyT)~(KeyT)0;
        KeyT s0 = top, s1 = top, s2 = top, s3 = top;
#pragma unroll
        for (int j = 0; j < KM; ++j) {
            if (j < k) {
                KeyT x = ((KeyT)key[j] << 7) | (KeyT)j;
                KeyT t = min(s0, x);
                x = max(s0, x);
                s0 = t;
                t = min(s1, x);
                x = max(s1, x);
                s1 = t;
                t = min(s2, x);
                x = max(s2, x);
                s2 = t;
                s3 = min(s3, x);
            }
        }
        const KeyT sel[4] = {s0, s1, s2, s3};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            if (q < n) {
                const int bj = (int)(sel[q] & 127u);
                if (bj < 64) pruned_lo |= 1ull << bj;
                else pruned_hi |= 1ull << (bj - 64);
            }
        }
    }
    // n > 4: pass s finds the smallest pair strictly above the pair found by
    // pass s-1.
    uint32_t pk = 0;
    int pj = -1;
    for (int s = 0; s < (a.threshold || n <= 4 ? 0 : n); ++s) {
        uint32_t bk = 0xffffffffu;
        int bj = KM;
#pragma unroll
        for (int j = 0; j < KM; ++j) {
            if (j < k) {
                const bool above = key[j] > pk || (key[j] == pk && j > pj);
                const bool better = key[j] < bk || (key[j] == bk && j < bj);
                if (above && better) {
                    bk = key[j];
                    bj = j;
                }
            }
        }
        pk = bk;
        pj = bj;
        if (bj < 64) pruned_lo |= 1ull << bj;
        else pruned_hi |= 1ull << (bj - 64);
    }

    // bitmap of columns held before pruning
    for (int q = 0; q < a.words; ++q) bitmap[q * R + tid] = 0u;
#pragma unroll
    for (int j = 0; j < KM; ++j) {
        if (j < k) {
            const int c = min(max(idx[j], 0), d - 1);
            bitmap[(c >> 5) * R + tid] |= 1u << (c & 31);
        }
    }

    // draws.  The row's staged indices are in idx[] now, so its LDS row holds
    // the accepted columns, each at the pruned slot it fills (pruned slots in
    // ascending order); nothing reaches memory unless the row finds all n.
    uint32_t *myrow = Itile + tid * (k + 1);
    uint64_t fill_lo = pruned_lo, fill_hi = pruned_hi;   // pruned slots still empty
    int got = 0;
    uint64_t w0 = 0, w1 = 0, w2 = 0, w3 = 0;
    for (int64_t att = 0; att < a.cap && got < n; ++att) {
        const int wsel = (int)(att & 3);
        if (wsel == 0) {
            w0 = (uint64_t)l;
            w1 = a.round;
            w2 = (uint64_t)(att >> 2);
            w3 = 0;
            philox4x64_10(w0, w1, w2, w3, a.seed, SET_KEY_HI);
        }
        const uint64_t word = wsel == 0 ? w0 : wsel == 1 ? w1 : wsel == 2 ? w2 : w3;
        const int c = (int)__umul64hi(word, (uint64_t)d);
        uint32_t &bw = bitmap[(c >> 5) * R + tid];
        const uint32_t bit = 1u << (c & 31);
        if (!(bw & bit)) {
            bw |= bit;
            const int j = fill_lo ? __builtin_ctzll(fill_lo) : 64 + __builtin_ctzll(fill_hi);
            if (fill_lo)
                fill_lo &= fill_lo - 1;
            else
                fill_hi &= fill_hi - 1;
            myrow[j] = (uint32_t)c;
            ++got;
        }
    }
    if (got < n) {
        if (a.exhausted) atomicAdd(a.exhausted, 1);
        if (a.mask)
            for (int j = 0; j < k; ++j) a.mask[l * k + j] = 0;
        return;
    }

    // write the pruned slots
    for (uint64_t wl = pruned_lo, wh = pruned_hi; wl | wh;) {
        const int j = wl ? __builtin_ctzll(wl) : 64 + __builtin_ctzll(wh);
        if (wl)
            wl &= wl - 1;
        else
            wh &= wh - 1;
        const int32_t c = (int32_t)myrow[j];
        const int64_t o = l * k + j;
        if (a.idx16)
            reinterpret_cast<uint16_t *>(a.I)[o] = (uint16_t)c;
        else
            a.I[o] = c;
        if constexpr (VT == FFSL_BF16)
            static_cast<uint16_t *>(a.W)[o] = 0;
        else
            static_cast<float *>(a.W)[o] = 0.f;
        a.m[o] = 0.f;
        a.v[o] = 0.f;
    }
    if (a.mask) {
        // k bytes per row, packed 4 per word when the row is word aligned
        if ((k & 3) == 0) {
            uint32_t *mrow = reinterpret_cast<uint32_t *>(a.mask + l * k);
#pragma unroll
            for (int j4 = 0; j4 < KM / 4; ++j4) {
                if (4 * j4 < k) {
                    uint32_t wv = 0;
#pragma unroll
                    for (int h = 0; h < 4; ++h) {
                        const int j = 4 * j4 + h;
                        const uint32_t pr =
                            j < 64 ? (uint32_t)((pruned_lo >> j) & 1ull) : (uint32_t)((pruned_hi >> (j - 64)) & 1ull);
                        wv |= pr << (8 * h);
                    }
                    mrow[j4] = wv;
                }
            }
        } else {
            for (int j = 0; j < k; ++j) {
                const bool pr = j < 64 ? ((pruned_lo >> j) & 1ull) : ((pruned_hi >> (j - 64)) & 1ull);
                a.mask[l * k + j] = pr ? 1 : 0;
            }
        }
    }
}

// The same update with one lane per row and no LDS tiles: the lane loads
// its row of I and W straight into registers (16-byte loads where the row
// allows), tests each candidate by comparing it with the row's columns before
// pruning (out-of-range indices taken as their clamped column, as the bitmap
// of k_set takes them) and with the columns accepted so far (the first
// SET_REG_ACC in registers, later ones in a per-lane LDS list), and writes
// the pruned slots as k_set does.  The draws, the selection and therefore
// every result are those of k_set.
template <int KM, int VT>
__device__ __forceinline__ void set_reg_row(const SetArgs &a, int64_t l, uint32_t *acc_lds, int tid) {
    const int k = a.k, d = a.d;

    // the row: indices (slots past k hold a value no candidate equals) and
    // keys |W| (bf16: 15 bits, fp32: 31 bits)
    uint32_t idx[KM], key[KM];
#pragma unroll
    for (int j = 0; j < KM; ++j) {
        idx[j] = 0xffffffffu;
        key[j] = 0u;
    }
    if (a.idx16) {
        const uint16_t *Ir = reinterpret_cast<const uint16_t *>(a.I) + l * k;
        if ((k & 7) == 0) {
#pragma unroll
            for (int u = 0; u < KM / 8; ++u) {
                if (8 * u < k) {
                    const uint4 q = reinterpret_cast<const uint4 *>(Ir)[u];
                    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
                    for (int h = 0; h < 4; ++h) {
                        idx[8 * u + 2 * h] = w[h] & 0xffffu;
                        idx[8 * u + 2 * h + 1] = w[h] >> 16;
                    }
                }
            }
        } else {
#pragma unroll
            for (int j = 0; j < KM; ++j)
                if (j < k) idx[j] = Ir[j];
        }
    } else {
        const uint32_t *Ir = reinterpret_cast<const uint32_t *>(a.I) + l * k;
        if ((k & 3) == 0) {
#pragma unroll
            for (int u = 0; u < KM / 4; ++u) {
                if (4 * u < k) {
                    const uint4 q = reinterpret_cast<const uint4 *>(Ir)[u];
                    idx[4 * u] = q.x;
                    idx[4 * u + 1] = q.y;
                    idx[4 * u + 2] = q.z;
                    idx[4 * u + 3] = q.w;
                }
            }
        } else {
#pragma unroll
            for (int j = 0; j < KM; ++j)
                if (j < k) idx[j] = Ir[j];
        }
    }
    if constexpr (VT == FFSL_BF16) {
        const uint16_t *Wr = static_cast<const uint16_t *>(a.W) + l * k;
        if ((k & 7) == 0) {
#pragma unroll
            for (int u = 0; u < KM / 8; ++u) {
                if (8 * u < k) {
                    const uint4 q = reinterpret_cast<const uint4 *>(Wr)[u];
                    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
                    for (int h = 0; h < 4; ++h) {
                        key[8 * u + 2 * h] = w[h] & 0x7fffu;
                        key[8 * u + 2 * h + 1] = (w[h] >> 16) & 0x7fffu;
                    }
                }
            }
        } else {
#pragma unroll
            for (int j = 0; j < KM; ++j)
                if (j < k) key[j] = Wr[j] & 0x7fffu;
        }
    } else {
        const uint32_t *Wr = static_cast<const uint32_t *>(a.W) + l * k;
        if ((k & 3) == 0) {
#pragma unroll
            for (int u = 0; u < KM / 4; ++u) {
                if (4 * u < k) {
                    const uint4 q = reinterpret_cast<const uint4 *>(Wr)[u];
                    key[4 * u] = q.x & 0x7fffffffu;
                    key[4 * u + 1] = q.y & 0x7fffffffu;
                    key[4 * u + 2] = q.z & 0x7fffffffu;
                    key[4 * u + 3] = q.w & 0x7fffffffu;
                }
            }
        } else {
#pragma unroll
            for (int j = 0; j < KM; ++j)
                if (j < k) key[j] = Wr[j] & 0x7fffffffu;
        }
    }
    // a column outside [0, d) counts as the nearest column in range
#pragma unroll
    for (int j = 0; j < KM; ++j)
        if (j < k) idx[j] = (uint32_t)min(max((int)idx[j], 0), d - 1);

    uint64_t pruned_lo = 0, pruned_hi = 0;  // slot bitmask, KM <= 128
    int n = a.n;
    if (a.threshold) {
        // |W| < tau compared as fp32 bit patterns of non-negative values
        n = 0;
#pragma unroll
        for (int j = 0; j < KM; ++j) {
            if (j < k) {
                const uint32_t mag = VT == FFSL_BF16 ? key[j] << 16 : key[j];
                if (mag < a.tau_bits) {
                    if (j < 64) pruned_lo |= 1ull << j;
                    else pruned_hi |= 1ull << (j - 64);
                    ++n;
                }
            }
        }
    } else if (n <= 4) {
        // the n smallest of the unique keys (|W| bits, slot) held in sorted
        // order by an insertion network of depth 4 over all k slots
        // bf16 keys (15 bits) and the slot fit one 32-bit word
        using KeyT = typename std::conditional<VT == FFSL_BF16, uint32_t, uint64_t>::type;
        const KeyT top = (KeyT)~(KeyT)0;
        KeyT s0 = top, s1 = top, s2 = top, s3 = top;
#pragma unroll
        for (int j = 0; j < KM; ++j) {
            if (j < k) {
                KeyT x = ((KeyT)key[j] << 7) | (KeyT)j;
                KeyT t = min(s0, x);
                x = max(s0, x);
                s0 = t;
                t = min(s1, x);
                x = max(s1, x);
                s1 = t;
                t = min(s2, x);
                x = max(s2, x);
                s2 = t;
                s3 = min(s3, x);
            }
        }
        const KeyT sel[4] = {s0, s1, s2, s3};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            if (q < n) {
                const int bj = (int)(sel[q] & 127u);
                if (bj < 64) pruned_lo |= 1ull << bj;
                else pruned_hi |= 1ull << (bj - 64);
            }
        }
    }
    // n > 4: pass s finds the smallest pair strictly above the pair found by
    // pass s-1.
    uint32_t pk = 0;
    int pj = -1;
    for (int s = 0; s < (a.threshold || n <= 4 ? 0 : n); ++s) {
        uint32_t bk = 0xffffffffu;
        int bj = KM;
#pragma unroll
        for (int j = 0; j < KM; ++j) {
            if (j < k) {
                const bool above = key[j] > pk || (key[j] == pk && j > pj);
                const bool better = key[j] < bk || (key[j] == bk && j < bj);
                if (above && better) {
                    bk = key[j];
                    bj = j;
                }
            }
        }
        pk = bk;
        pj = bj;
        if (bj < 64) pruned_lo |= 1ull << bj;
        else pruned_hi |= 1ull << (bj - 64);
    }

    // draws: the q-th accepted column fills the q-th pruned slot in
    // ascending slot order; nothing reaches memory unless the row finds all n
    uint32_t c0 = 0xffffffffu, c1 = 0xffffffffu, c2 = 0xffffffffu, c3 = 0xffffffffu;
    int got = 0;
    uint64_t w0 = 0, w1 = 0, w2 = 0, w3 = 0;
    for (int64_t att = 0; att < a.cap && got < n; ++att) {
        const int wsel = (int)(att & 3);
        if (wsel == 0) {
            w0 = (uint64_t)l;
            w1 = a.round;
            w2 = (uint64_t)(att >> 2);
            w3 = 0;
            philox4x64_10(w0, w1, w2, w3, a.seed, SET_KEY_HI);
        }
        const uint64_t word = wsel == 0 ? w0 : wsel == 1 ? w1 : wsel == 2 ? w2 : w3;
        const uint32_t c = (uint32_t)__umul64hi(word, (uint64_t)d);
        bool held = c == c0 || c == c1 || c == c2 || c == c3;
#pragma unroll
        for (int j = 0; j < KM; ++j) held = held || idx[j] == c;
        for (int q = SET_REG_ACC; q < got; ++q) held = held || acc_lds[(q - SET_REG_ACC) * SET_REG_ROWS + tid] == c;
        if (!held) {
            c0 = got == 0 ? c : c0;
            c1 = got == 1 ? c : c1;
            c2 = got == 2 ? c : c2;
            c3 = got == 3 ? c : c3;
            if (got >= SET_REG_ACC) acc_lds[(got - SET_REG_ACC) * SET_REG_ROWS + tid] = c;
            ++got;
        }
    }
    if (got < n) {
        if (a.exhausted) atomicAdd(a.exhausted, 1);
        if (a.mask)
            for (int j = 0; j < k; ++j) a.mask[l * k + j] = 0;
        return;
    }

    // write the pruned slots
    int q = 0;
    for (uint64_t wl = pruned_lo, wh = pruned_hi; wl | wh; ++q) {
        const int j = wl ? __builtin_ctzll(wl) : 64 + __builtin_ctzll(wh);
        if (wl)
            wl &= wl - 1;
        else
            wh &= wh - 1;
        const int32_t c = (int32_t)(q == 0   ? c0
                                    : q == 1 ? c1
                                    : q == 2 ? c2
                                    : q == 3 ? c3
                                             : acc_lds[(q - SET_REG_ACC) * SET_REG_ROWS + tid]);
        const int64_t o = l * k + j;
        if (a.idx16)
            reinterpret_cast<uint16_t *>(a.I)[o] = (uint16_t)c;
        else
            a.I[o] = c;
        if constexpr (VT == FFSL_BF16)
            static_cast<uint16_t *>(a.W)[o] = 0;
        else
            static_cast<float *>(a.W)[o] = 0.f;
        a.m[o] = 0.f;
        a.v[o] = 0.f;
    }
    if (a.mask) {
        // k bytes per row, packed 4 per word when the row is word aligned
        if ((k & 3) == 0) {
            uint32_t *mrow = reinterpret_cast<uint32_t *>(a.mask + l * k);
#pragma unroll
            for (int j4 = 0; j4 < KM / 4; ++j4) {
                if (4 * j4 < k) {
                    uint32_t wv = 0;
#pragma unroll
                    for (int h = 0; h < 4; ++h) {
                        const int j = 4 * j4 + h;
                        const uint32_t pr =
                            j < 64 ? (uint32_t)((pruned_lo >> j) & 1ull) : (uint32_t)((pruned_hi >> (j - 64)) & 1ull);
                        wv |= pr << (8 * h);
                    }
                    mrow[j4] = wv;
                }
            }
        } else {
            for (int j = 0; j < k; ++j) {
                const bool pr = j < 64 ? ((pruned_lo >> j) & 1ull) : ((pruned_hi >> (j - 64)) & 1ull);
                a.mask[l * k + j] = pr ? 1 : 0;
            }
        }
    }
}


// acc_lds: accepted columns beyond the first SET_REG_ACC of each row,
// [q][lane]; the rows need no block-level synchronisation
template <int KM, int VT>
__global__ void __launch_bounds__(SET_REG_ROWS) k_set_reg(const SetArgs a) {
    extern __shared__ uint32_t acc_lds[];
    const int64_t l = (int64_t)blockIdx.x * SET_REG_ROWS + threadIdx.x;
    if (l < a.L) set_reg_row<KM, VT>(a, l, acc_lds, threadIdx.x);
}

// SET on the rows of a list (list[0] = their count, the rows from list[1]):
// the rows whose first four regrowth draws the fused step+SET sweep could
// not use; each row's result is the one k_set_reg gives it
template <int KM, int VT>
__global__ void __launch_bounds__(SET_REG_ROWS) k_set_reg_list(const SetArgs a, const int32_t *list) {
    extern __shared__ uint32_t acc_lds[];
    const int64_t n = list[0];
    for (int64_t i = (int64_t)blockIdx.x * SET_REG_ROWS + threadIdx.x; i < n; i += (int64_t)gridDim.x * SET_REG_ROWS)
        set_reg_row<KM, VT>(a, list[1 + i], acc_lds, threadIdx.x);
}

template <int KM>
__global__ void __launch_bounds__(256) k_validate(const int32_t *I, int64_t L, int k, int d, int32_t *bad,
                                                  int idx16) {
    const int64_t l = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (l >= L) return;
    int idx[KM];
    bool ok = true;
#pragma unroll
    for (int j = 0; j < KM; ++j) {
        if (j < k) {
            idx[j] = idx16 ? (int)reinterpret_cast<const uint16_t *>(I)[l * k + j] : I[l * k + j];
            ok = ok && idx[j] >= 0 && idx[j] < d;
        }
    }
#pragma unroll
    for (int j = 0; j < KM; ++j)
#pragma unroll
        for (int q = j + 1; q < KM; ++q)
            if (q < k && idx[j] == idx[q]) ok = false;
    if (!ok) atomicAdd(bad, 1);
}

template <int VT>
size_t set_lds_bytes(int words, int R, int k) {
    return sizeof(uint32_t) * ((size_t)words * R + (size_t)R * (k + 1) + (size_t)R * (w_words<VT>(k) + 1));
}

// Rows whose tiles leave room for two 256-row workgroups per CU run the
// LDS-tiled k_set; wider rows (a larger fan-in or input width, where the tiles
// would leave one small workgroup per CU) run k_set_reg, which holds each row
// in one lane's registers.
template <int KM, int VT>
int set_launch_reg(const SetArgs &a, hipStream_t st) {
    constexpr size_t LDS_MAX = 160 * 1024;
    // rows that may accept more columns than the registers hold list the rest in LDS
    const int nmax = a.threshold ? a.k : a.n;
    const size_t shm = sizeof(uint32_t) * (size_t)max(nmax - SET_REG_ACC, 0) * SET_REG_ROWS;
    if (shm > LDS_MAX) return fail(FFSL_EUNSUPPORTED, "SET: too many pruned slots per row (%d)", nmax);
    auto kern = k_set_reg<KM, VT>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
    if (e != hipSuccess) return fail(FFSL_EHIP, "hipFuncSetAttribute: %s", hipGetErrorString(e));
    const int64_t blocks = (a.L + SET_REG_ROWS - 1) / SET_REG_ROWS;
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(SET_REG_ROWS), shm, st, a);
    return check_launch("set_update");
}

template <int KM, int VT>
int set_launch_km(SetArgs a, hipStream_t st) {
    constexpr size_t LDS_MAX = 160 * 1024;
    if (KM <= 64 && set_lds_bytes<VT>(a.words, SET_MAX_ROWS, a.k) > LDS_MAX / 2) return set_launch_reg<KM, VT>(a, st);
    int R = SET_MAX_ROWS;
    while (R > 64 && set_lds_bytes<VT>(a.words, R, a.k) > LDS_MAX) R /= 2;
    const size_t shm = set_lds_bytes<VT>(a.words, R, a.k);
    if (shm > LDS_MAX) return fail(FFSL_EUNSUPPORTED, "SET tile does not fit LDS (d=%d, k=%d)", a.d, a.k);
    a.R = R;
    auto kern = k_set<KM, VT>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
    if (e != hipSuccess) return fail(FFSL_EHIP, "hipFuncSetAttribute: %s", hipGetErrorString(e));
    const int64_t blocks = (a.L + R - 1) / R;
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(R), shm, st, a);
    return check_launch("set_update");
}

template <int VT>
int set_launch_vt(const SetArgs &a, hipStream_t st) {
    if (a.k <= 8) return set_launch_km<8, VT>(a, st);
    if (a.k <= 16) return set_launch_km<16, VT>(a, st);
    if (a.k <= 32) return set_launch_km<32, VT>(a, st);
    if (a.k <= 64) return set_launch_km<64, VT>(a, st);
    return set_launch_km<128, VT>(a, st);
}

}  // namespace

int launch_set(const Layer &ly, int32_t n, uint64_t seed, uint64_t round, uint8_t *mask,
               int32_t *exhausted, hipStream_t st, bool threshold, float tau) {
    SetArgs a{};
    a.threshold = threshold ? 1 : 0;
    a.tau_bits = threshold ? __builtin_bit_cast(uint32_t, tau) : 0u;
    a.L = ly.L;
    a.d = ly.d;
    a.k = ly.k;
    a.n = n;
    a.words = (ly.d + 31) / 32;
    a.W = ly.W;
    a.I = ly.I;
    a.idx16 = ly.idx16;
    a.m = ly.m;
    a.v = ly.v;
    a.mask = mask;
    a.exhausted = exhausted;
    a.seed = seed;
    a.round = round;
    a.cap = 64 * (int64_t)ly.k + 4096;
    return ly.vt == FFSL_BF16 ? set_launch_vt<FFSL_BF16>(a, st) : set_launch_vt<FFSL_F32>(a, st);
}

int launch_set_rows(const Layer &ly, int32_t n, uint64_t seed, uint64_t round, uint8_t *mask, int32_t *exhausted,
                    const int32_t *list, hipStream_t st) {
    if (ly.k > 64) return fail(FFSL_EUNSUPPORTED, "SET on a row list: fan-in %d", ly.k);
    SetArgs a{};
    a.L = ly.L;
    a.d = ly.d;
    a.k = ly.k;
    a.n = n;
    a.words = (ly.d + 31) / 32;
    a.W = ly.W;
    a.I = ly.I;
    a.idx16 = ly.idx16;
    a.m = ly.m;
    a.v = ly.v;
    a.mask = mask;
    a.exhausted = exhausted;
    a.seed = seed;
    a.round = round;
    a.cap = 64 * (int64_t)ly.k + 4096;
    const size_t shm = sizeof(uint32_t) * (size_t)max(n - SET_REG_ACC, 0) * SET_REG_ROWS;
    const void *kern;
    if (ly.vt == FFSL_BF16)
        kern = ly.k <= 32 ? reinterpret_cast<const void *>(&k_set_reg_list<32, FFSL_BF16>)
                          : reinterpret_cast<const void *>(&k_set_reg_list<64, FFSL_BF16>);
    else
        kern = ly.k <= 32 ? reinterpret_cast<const void *>(&k_set_reg_list<32, FFSL_F32>)
                          : reinterpret_cast<const void *>(&k_set_reg_list<64, FFSL_F32>);
    hipError_t e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
    if (e != hipSuccess) return fail(FFSL_EHIP, "hipFuncSetAttribute: %s", hipGetErrorString(e));
    // a few workgroups per CU cover the rare deferred rows; with none the
    // workgroups exit at once
    const int blocks = (int)std::min<int64_t>((ly.L + SET_REG_ROWS - 1) / SET_REG_ROWS, (int64_t)ly.num_cu * 4);
    hipLaunchKernelGGL(reinterpret_cast<void (*)(SetArgs, const int32_t *)>(const_cast<void *>(kern)), dim3(blocks),
                       dim3(SET_REG_ROWS), shm, st, a, list);
    return check_launch("set_update (deferred rows)");
}

int launch_validate(const Layer &ly, int32_t *bad, hipStream_t st) {
    const int64_t blocks = (ly.L + 255) / 256;
    if (ly.k <= 16)
        hipLaunchKernelGGL(k_validate<16>, dim3((unsigned)blocks), dim3(256), 0, st, ly.I, ly.L, ly.k, ly.d, bad, ly.idx16);
    else if (ly.k <= 32)
        hipLaunchKernelGGL(k_validate<32>, dim3((unsigned)blocks), dim3(256), 0, st, ly.I, ly.L, ly.k, ly.d, bad, ly.idx16);
    else if (ly.k <= 64)
        hipLaunchKernelGGL(k_validate<64>, dim3((unsigned)blocks), dim3(256), 0, st, ly.I, ly.L, ly.k, ly.d, bad, ly.idx16);
    else
        hipLaunchKernelGGL(k_validate<128>, dim3((unsigned)blocks), dim3(256), 0, st, ly.I, ly.L, ly.k, ly.d, bad, ly.idx16);
    return check_launch("validate_indices");
}

}  // namespace ffsl
