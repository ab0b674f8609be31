// Batch preparation for the fused fast sweeps (sweep_mx.hip, sweep_wide.hip),
// run once per call before their batch passes.  Every workgroup of a sweep
// pass needs the same two things before its first chunk: the pass's positives
// sorted by label (to find each chunk's targets with a forward-only cursor)
// and the pass's samples transposed into the LDS tile layout X^T [d][PB]
// (column i = the PB samples' values, so that one gather reads several samples
// of a column).  Built here once, they are copied by each workgroup with
// 16-byte loads instead of being rebuilt by all of them.
//
//   workgroups [0, nsort)   pass p = blockIdx.x: keys (label << SB | sample
//                           within the pass), ascending, in keys[p][0 .. 1024),
//                           padded with 0xffffffff (a key that matches no row);
//                           a label outside [0,L) becomes that padding key
//   the others              XT[p][i][b] = X[p*PB + b][i], zero past B
//   workgroup 0 also clears zero_word when given (the deferred-row count of a
//   fused step+SET sweep)
#include "sweep_dev.h"

namespace ffsl {

namespace {

using namespace fdev;

constexpr int BP_THREADS = 512;
constexpr int BP_KEYS = 1024;   // positives the sweeps keep in LDS

struct BatchPrepArgs {
    const uint16_t *X;      // [B][d] bf16
    const int32_t *off;     // [B+1] CSR offsets of the positives
    const int32_t *lab;     // [nnz] their labels
    int32_t B, d, nnz, passes, nsort;
    int64_t L;
    uint32_t *keys;         // [passes][BP_KEYS]
    uint16_t *xt;           // [passes][d][PB]
    int32_t *zero_word;     // set to 0 when given
};

template <int PB>
__global__ void __launch_bounds__(BP_THREADS) k_batch_prep(const BatchPrepArgs a) {
    constexpr int SB = PB == 64 ? 6 : 4;   // sample bits of a key
    static_assert((1 << SB) == PB, "pass width");
    const int tid = threadIdx.x;
    if (blockIdx.x == 0 && tid == 0 && a.zero_word) *a.zero_word = 0;
    if ((int)blockIdx.x < a.nsort) {
        __shared__ uint32_t tg[BP_KEYS];
        __shared__ int32_t smp[BP_KEYS];
        const int p = blockIdx.x;
        const int b0 = p * PB, Bp = min(PB, a.B - b0);
        // the thread's two labels and the offsets of its samples b = tid,
        // tid + 512 (B <= 1024), all loaded before the first barrier
        const int32_t lb0 = tid < a.nnz ? a.lab[tid] : -1;
        const int32_t lb1 = tid + BP_THREADS < a.nnz ? a.lab[tid + BP_THREADS] : -1;
        int er[2][2] = {{0, 0}, {0, 0}};
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int b = tid + h * BP_THREADS;
            if (b < a.B) {
                er[h][0] = max(0, min(a.off[b], a.nnz));
                er[h][1] = max(er[h][0], min(a.off[b + 1], a.nnz));
            }
        }
        for (int e = tid; e < BP_KEYS; e += BP_THREADS) smp[e] = -1;
        __syncthreads();
        // the sample of each positive pair, e in [off[b], off[b+1])
#pragma unroll
        for (int h = 0; h < 2; ++h)
            for (int e = er[h][0]; e < er[h][1]; ++e) smp[e] = tid + h * BP_THREADS;
        __syncthreads();
        auto key_of = [&](int e, int32_t lb) -> uint32_t {
            if (e >= a.nnz) return 0xffffffffu;
            const int32_t sb = smp[e] - b0;
            return lb >= 0 && (int64_t)lb < a.L && sb >= 0 && sb < Bp ? ((uint32_t)lb << SB) | (uint32_t)sb
                                                                       : 0xffffffffu;
        };
        static_assert(BP_THREADS == 512, "sort_keys512 takes a 512-thread workgroup");
        sort_keys512(tg, key_of(tid, lb0), key_of(tid + BP_THREADS, lb1), a.nnz, tid);
        int N = 64;
        while (N < a.nnz) N <<= 1;   // tg[0 .. N) is sorted
        uint32_t *out = a.keys + (size_t)p * BP_KEYS;
        out[tid] = tid < N ? tg[tid] : 0xffffffffu;
        out[tid + BP_THREADS] = tid + BP_THREADS < N ? tg[tid + BP_THREADS] : 0xffffffffu;
        return;
    }
    // transpose: unit un = (p * Q + q) * d + i writes XT[p][i][8q .. 8q+7];
    // consecutive lanes take consecutive columns, so each of the eight 2-byte
    // loads of a unit is coalesced over the wave
    constexpr int Q = PB / 8;
    const int64_t nunits = (int64_t)a.passes * Q * a.d;
    const int64_t stride = (int64_t)(gridDim.x - a.nsort) * BP_THREADS;
    for (int64_t un = (int64_t)(blockIdx.x - a.nsort) * BP_THREADS + tid; un < nunits; un += stride) {
        const int i = (int)(un % a.d);
        const int pq = (int)(un / a.d);
        const int p = pq / Q, q = pq % Q;
        uint32_t w[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int b = p * PB + 8 * q + 2 * r;
            const uint32_t lo = b < a.B ? a.X[(size_t)b * a.d + i] : 0u;
            const uint32_t hi = b + 1 < a.B ? a.X[(size_t)(b + 1) * a.d + i] : 0u;
            w[r] = lo | (hi << 16);
        }
        reinterpret_cast<uint4 *>(a.xt)[((size_t)p * a.d + i) * Q + q] = make_uint4(w[0], w[1], w[2], w[3]);
    }
}

}  // namespace

int launch_batch_prep(const uint16_t *X, int32_t B, int32_t d, const int32_t *off, const int32_t *lab,
                      int32_t nnz, int64_t L, int pass_b, uint32_t *keys, uint16_t *xt, int32_t *zero_word,
                      hipStream_t st) {
    if (B < 1 || B > 2 * BP_THREADS) return fail(FFSL_EINVAL, "batch prep: B = %d outside [1, %d]", B, 2 * BP_THREADS);
    BatchPrepArgs a{};
    a.X = X;
    a.off = off;
    a.lab = lab;
    a.B = B;
    a.d = d;
    a.nnz = nnz;
    a.L = L;
    a.passes = (B + pass_b - 1) / pass_b;
    // with more positives than the sweeps keep in LDS they scan the CSR arrays
    a.nsort = nnz <= BP_KEYS ? a.passes : 0;
    a.keys = keys;
    a.xt = xt;
    a.zero_word = zero_word;
    const int64_t units = (int64_t)a.passes * (pass_b / 8) * d;
    const int tgrid = (int)std::min<int64_t>((units + BP_THREADS - 1) / BP_THREADS, 1024);
    const dim3 grid(a.nsort + tgrid);
    if (pass_b == 64)
        hipLaunchKernelGGL(k_batch_prep<64>, grid, dim3(BP_THREADS), 0, st, a);
    else if (pass_b == 16)
        hipLaunchKernelGGL(k_batch_prep<16>, grid, dim3(BP_THREADS), 0, st, a);
    else
        return fail(FFSL_EUNSUPPORTED, "batch prep: pass width %d", pass_b);
    return check_launch("batch_prep");
}

}  // namespace ffsl
