// Device helpers shared by the fused fast sweeps (sweep_mx.hip, sweep_wide.hip)
// and SET (set.hip): range-checked raw buffer access, bf16 dot products,
// DPP-fused adds, the slot key of the 16-lane dW reduce-scatter, the Adam
// update and the Philox generator of the regrowth draws.
#pragma once

#include "ffsl_internal.h"

namespace ffsl {
namespace fdev {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// what a batch pass does with the dW it has summed over its samples
enum PassMode {
    PASS_ONLY = 0,    // the whole batch: Adam
    PASS_FIRST = 1,   // first of several passes: store the partial dW
    PASS_LAST = 2,    // last pass: add the carried partial, then Adam
    PASS_MIDDLE = 3,  // add the carried partial and store it again
};

typedef __amdgpu_buffer_rsrc_t Rsrc;

// raw buffer resource over [p, p + nbytes): out-of-range loads read 0 and
// out-of-range stores are dropped
__device__ __forceinline__ Rsrc make_rsrc(const void *p, uint32_t nbytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, (int)nbytes, 0x00020000);
}

__device__ __forceinline__ uint32_t ld32(Rsrc r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
}
__device__ __forceinline__ float ldf(Rsrc r, uint32_t off) { return __uint_as_float(ld32(r, off)); }
__device__ __forceinline__ float2 ldf2(Rsrc r, uint32_t off) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
    return make_float2(__uint_as_float(v[0]), __uint_as_float(v[1]));
}
__device__ __forceinline__ void st32(Rsrc r, uint32_t off, uint32_t x) {
    __builtin_amdgcn_raw_buffer_store_b32(x, r, off, 0, 0);
}
__device__ __forceinline__ void stf(Rsrc r, uint32_t off, float x) { st32(r, off, __float_as_uint(x)); }
__device__ __forceinline__ void stf2(Rsrc r, uint32_t off, float2 x) {
    typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
    const u32x2 v = {__float_as_uint(x.x), __float_as_uint(x.y)};
    __builtin_amdgcn_raw_buffer_store_b64(v, r, off, 0, 0);
}

// a lane's two index words as loaded -> its two column indices: with 16-bit
// indices both words hold the one word of the two slots
__device__ __forceinline__ uint2 idx_pair(uint2 raw, int idx16) {
    return idx16 ? make_uint2(raw.x & 0xffffu, raw.x >> 16) : raw;
}

__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), __builtin_bit_cast(bf16x2, b), c,
                                           false);
}

// a.b with no accumulator (the three-operand form takes an inline zero)
__device__ __forceinline__ float dot2z(uint32_t a, uint32_t b) {
    float r;
    asm("v_dot2_f32_bf16 %0, %1, %2, 0" : "=v"(r) : "v"(a), "v"(b));
    return r;
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
constexpr int DPP_ROW_ROR8 = 0x128;        // lane j <- j ^ 8 within 16 (rotation by 8)

// Slot key of lane j of a 16-lane group in the dW reduce-scatter over 32
// slots: the lane keeps slot r ^ (lane_key(j) with bit 1 cleared) in register
// r, so the first three butterfly levels are one add each with a
// mirror-pattern DPP source and the lane reads its slots four at a time.
__device__ __forceinline__ int lane_key(int j) {
    return ((j & 1) ? 2 : 0) ^ ((j & 2) ? 6 : 0) ^ ((j & 4) ? 12 : 0) ^ ((j & 8) ? 24 : 0);
}

// Reduce-scatter of pw[0..31] (slot r ^ Kp in register r) over the 16 lanes
// of a DPP row.  Lane j ends with the sums of slots Kown(j), Kown(j) + 1 in
// the returned pair, Kown(j) = Kp(j) + 2 (j & 1).  At the last level lanes j
// and j^1 hold the same four slots; both add and each keeps two.
__device__ __forceinline__ float2 reduce_scatter16(float (&pw)[32], bool odd) {
#pragma unroll
    for (int r = 0; r < 16; ++r) pw[r] = add_dpp<DPP_ROW_MIRROR>(pw[r], pw[16 + r]);
#pragma unroll
    for (int r = 0; r < 8; ++r) pw[r] = add_dpp<DPP_ROW_HALF_MIRROR>(pw[r], pw[8 + r]);
#pragma unroll
    for (int r = 0; r < 4; ++r) pw[r] = add_dpp<DPP_QUAD_3210>(pw[r], pw[4 + r]);
#pragma unroll
    for (int r = 0; r < 4; ++r) pw[r] = add_dpp<DPP_QUAD_1032>(pw[r], pw[r]);
    return odd ? make_float2(pw[2], pw[3]) : make_float2(pw[0], pw[1]);
}

// sum of x over the 16 lanes of a DPP row, in every lane
__device__ __forceinline__ float sum16(float x) {
    x = add_dpp<DPP_ROW_MIRROR>(x, x);
    x = add_dpp<DPP_ROW_HALF_MIRROR>(x, x);
    x = add_dpp<DPP_QUAD_3210>(x, x);
    return add_dpp<DPP_QUAD_1032>(x, x);
}

// Lanes j of DPP rows 2r and 2r+1 of a wave: the first gets x of the second
// plus its own x, the second gets y of the first plus its own y
// (v_permlane16_swap exchanges x of the odd row with y of the even row).
__device__ __forceinline__ float cross_rows_add(float x, float y) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(y), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// LDS written by some lanes of a wave and read by others of the same wave:
// the wave's LDS operations run in order, so only the compiler is held back
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Ascending sort of a 512-thread workgroup's keys into tg (room for 1024
// words).  Thread t brings the keys of elements t and t + 512 (k0, k1; empty
// elements hold 0xffffffff), n of them in all, n <= 1024.  A bitonic network
// over N = max(64, next power of two >= n) elements: a stage whose partners
// lie within a wave (distance < 64) exchanges registers through a lane
// shuffle, with no barrier; the few stages across waves go through tg between
// two barriers; the one stage at distance 512 (N = 1024) swaps a thread's own
// pair.  On return tg[0 .. N) holds the keys in ascending order, visible to
// the whole workgroup.
__device__ __forceinline__ uint32_t bitonic_pick(uint32_t x, uint32_t y, int i, int j, int k) {
    return (((i & j) == 0) == ((i & k) == 0)) ? min(x, y) : max(x, y);
}
__device__ __forceinline__ void sort_keys512(uint32_t *tg, uint32_t k0, uint32_t k1, int n, int tid) {
    int N = 64;
    while (N < n) N <<= 1;
    const bool two = N > 512;
    const bool own = tid < N;   // whole waves: N is a multiple of 64
    for (int k = 2; k <= N; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            if (j >= 512) {
                // N = 1024, k = 1024: element tid is the lower of its own pair
                const uint32_t lo = min(k0, k1), hi = max(k0, k1);
                k0 = lo;
                k1 = hi;
            } else if (j >= 64) {
                __syncthreads();   // the previous exchange's reads are done
                if (own) tg[tid] = k0;
                if (two) tg[tid + 512] = k1;
                __syncthreads();
                if (own) k0 = bitonic_pick(k0, tg[tid ^ j], tid, j, k);
                if (two) k1 = bitonic_pick(k1, tg[(tid + 512) ^ j], tid + 512, j, k);
            } else {
                if (own) k0 = bitonic_pick(k0, (uint32_t)__shfl_xor((int)k0, j), tid, j, k);
                if (two) k1 = bitonic_pick(k1, (uint32_t)__shfl_xor((int)k1, j), tid + 512, j, k);
            }
        }
    }
    __syncthreads();
    if (own) tg[tid] = k0;
    if (two) tg[tid + 512] = k1;
    __syncthreads();
}

// Adam with the bias corrections folded into reciprocals; fp32 throughout.
// Every fused multiply-add is written out, so each kernel that inlines this
// rounds the same way (contraction left to the compiler may fuse a*b + c*d
// either way round).
__device__ __forceinline__ float adam_step(float p, float g, float &mm, float &vv, float b1, float b2,
                                           float inv_bc1, float inv_bc2, float lr, float eps, float decay) {
    p *= decay;
    mm = fmaf(b1, mm, (1.f - b1) * g);
    vv = fmaf(b2, vv, ((1.f - b2) * g) * g);
    const float den = __builtin_amdgcn_sqrtf(vv * inv_bc2) + eps;
    return fmaf(-((lr * inv_bc1) * mm), __builtin_amdgcn_rcpf(den), p);
}

// Regrowth draws of SET: Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC'11)
// keyed by (seed, SET_KEY_HI) and counted by (row, set_round, attempt / 4, 0).
constexpr uint64_t SET_KEY_HI = 0x5345545F52454752ull;  // "SET_REGR"

// Philox4x64-10 round structure: two 64x64->128 multiplies per round, the
// high halves mixed with the other counter words and the round key, the key
// advanced by the Weyl increments (golden ratio, sqrt(3)-1) between rounds.
__device__ __forceinline__ void philox4x64_10(uint64_t &c0, uint64_t &c1, uint64_t &c2,
                                              uint64_t &c3, uint64_t k0, uint64_t k1) {
    const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
    const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint64_t lo0 = M0 * c0, hi0 = __umul64hi(M0, c0);
        const uint64_t lo1 = M1 * c2, hi1 = __umul64hi(M1, c2);
        const uint64_t n0 = hi1 ^ c1 ^ k0;
        const uint64_t n2 = hi0 ^ c3 ^ k1;
        c0 = n0;
        c1 = lo1;
        c2 = n2;
        c3 = lo0;
        k0 += W0;
        k1 += W1;
    }
}

}  // namespace fdev
}  // namespace ffsl
