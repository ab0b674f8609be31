// Fused training step of the fixed fan-in layer for bf16 values, fan-in 32 and
// input widths that are a multiple of 128 up to 768 (the gathered forward,
// BCE, dW, dbias, dX and Adam of Sec. 2.2, in one pass over the [L,k] arrays
// per 64 samples of the batch; see launch_sweep_mx for larger batches).
//
// Workgroup: 512 threads (8 waves, two per SIMD), one per CU, persistent over
// chunks of 32 label rows.  Sixteen lanes serve one row; lane u of a row owns
// batch rows b = 4u .. 4u+3.
//
//   LDS  Xs [d][64] bf16   the batch transposed (column i is 128 contiguous
//                          bytes), zero-padded past B
//        T  [d][32] bf16   the chunk's weights scattered densely by column
//        G  [64][32] bf16  the chunk's dlogits (both with XOR-swizzled 16-byte
//                          chunks, see swz)
//        Is, Ws            the chunk's index rows (as byte offsets into Xs)
//                          and weight rows
//        tg                the batch's positives as sorted (label, sample) keys;
//                          with more positives than fit, ym [32][2] u32 (in the
//                          same place) holds the chunk's targets built by a scan
//
//   1. gather: for each slot, lane u reads the 8 bytes X[4u..4u+3, I[l,j]]
//      (16 lanes read one whole column, four columns per wave instruction,
//      which keeps LDS bank conflicts low);
//   2. forward: the b-pairs are repacked into slot pairs with v_perm and
//      reduced with v_dot2_f32_bf16 against the row's (W_j, W_j+1) pairs;
//   3. BCE loss and dlogits g for the lane's 4 batch rows;
//   4. dW partials over the lane's 4 rows with v_dot2 (g rounded to bf16),
//      then a reduce-scatter over the 16 lanes with DPP-fused adds.  Lane u
//      keeps slot r XOR Kp(u) in register r, Kp(u) = (2u0^6u1^12u2^24u3) with
//      bit 1 cleared, which makes the first three butterfly levels one add
//      each with a mirror-pattern DPP source and lets the lane read its row's
//      indices four at a time; at the last level lanes u and u^1 hold the
//      same four slots, both add, and each keeps two: lane u ends with the
//      full dW of slots Kp(u) + 2u0 and the next one;
//   5. Adam on those two slots, streaming W, m, v back to HBM;
//   6. dX: g and the old weights go to G and T, and the matrix cores add
//      G x T^T (64 x 32 by 32 x d) into a per-workgroup dX held in registers for
//      the workgroup's whole life; it is written out once at the end.
// The next chunk's index and weight rows are loaded into registers while the
// current chunk computes; the matrix-core work of a chunk overlaps the VALU
// work of the next.  All HBM
// accesses of the chunk loop are range-checked buffer operations: a row past
// L reads zeros and its writes are dropped by the hardware, so the loop has no
// data-dependent branches and the compiler can keep exact counts of
// outstanding memory operations (a branch around a store makes it drain them
// all).
#include "sweep_dev.h"

namespace ffsl {

namespace {

constexpr int MX_THREADS = 512;
constexpr int MX_NLAB = 32;     // label rows per chunk
constexpr int MX_K = 32;        // fan-in of this path
constexpr int MX_NB = 64;       // padded batch
constexpr int MX_XS = 128;      // bytes per X column row in LDS
constexpr int MX_TG_MAX = 1024; // positives kept in LDS

using namespace fdev;

struct MxArgs {
    int64_t L;
    int32_t d, B, nnz;
    int64_t nchunks;
    const uint16_t *XT;     // this pass's samples transposed, [d][64] (batch prep)
    const uint32_t *keys;   // this pass's sorted positives, [1024] (nnz <= 1024)
    uint16_t *W;
    const int32_t *I;
    float *bias, *m, *v, *bm, *bv;
    const int32_t *tgt_b, *tgt_lab;
    float s;
    AdamParams adam;
    float *loss_part;
    float *dx_part;
    // array sizes in bytes: the range of each buffer resource, and the offset
    // that the chunk loop uses for an access that must not happen
    uint32_t nb_W, nb_I, nb_m, nb_b;
    int32_t idx16;   // I holds uint16 indices
    // batch pass: samples b0 .. b0+B-1 of Btot; dW / dbias carried between
    // passes in dwp [L][32], dbp [L]
    int32_t b0, Btot;
    float *dwp, *dbp;
    int32_t hinge;   // squared hinge instead of BCE
    // SET fused into the pass that applies Adam (see the SETF kernels)
    int32_t set_n;
    uint64_t set_seed, set_round;
    uint8_t *set_mask;
    int32_t *set_list;   // rows left to SET on a row list: count, then the rows
    uint32_t nb_mask;
};

// pass roles (see launch_sweep_mx)
constexpr int MX_ONLY = PASS_ONLY, MX_FIRST = PASS_FIRST, MX_LAST = PASS_LAST, MX_MIDDLE = PASS_MIDDLE;

struct Rsrcs {
    Rsrc XT, K, W, I, m, v, b, bm, bv, dwp, dbp, mk;
};

constexpr int MX_SET_NMAX = 4;   // pruned slots per row the fused SET handles (its four draws ahead)
constexpr int MX_SET_AHEAD = 8;  // chunks whose first candidates a wave draws at once

// minimum of x over the 16 lanes of a DPP row, in every lane
__device__ __forceinline__ uint32_t min16(uint32_t x) {
    x = min(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, DPP_ROW_MIRROR, 0xf, 0xf, false));
    x = min(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, DPP_ROW_HALF_MIRROR, 0xf, 0xf, false));
    x = min(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, DPP_QUAD_3210, 0xf, 0xf, false));
    return min(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, DPP_QUAD_1032, 0xf, 0xf, false));
}

// G and T rows hold 32 bf16 (64 bytes = four 16-byte chunks).  The matrix-
// core fragments read one chunk from each of 16 consecutive rows; stored
// plainly, rows r and r+4 would hit the same banks.  Chunk q of row r is
// therefore kept at chunk q ^ ((r >> 2) & 3); element e of row r sits at:
__device__ __forceinline__ int swz(int r, int e) {
    return r * MX_NLAB + ((((e >> 3) ^ (r >> 2)) & 3) << 3) + (e & 7);
}

struct Prefetch {
    uint2 iv;          // the lane's two index words as loaded (see idx_pair)
    uint32_t wv;       // one weight word of the chunk's W rows
    float2 m, v;       // moments of the lane's two slots (slot, slot + 1) of its row
    float b;           // its bias
};

// the chunk's rows and optimiser state (the moments only for a pass that
// applies Adam), loaded a chunk ahead of their use; a chunk or row past the
// end reads zeros
template <bool MOMENTS>
__device__ __forceinline__ void prefetch(const MxArgs &a, const Rsrcs &R, int64_t chunk, int tid, int lab, int u,
                                         int slot, Prefetch &p) {
    const int64_t l0 = chunk * MX_NLAB;
    const bool live = chunk < a.nchunks;
    // two word loads either way (no load reaches past the array): with 16-bit
    // indices both read the one word that holds the lane's two slots
    const uint32_t ish = a.idx16 ? 1u : 2u;   // log2 of the index bytes
    const uint32_t oi = live ? ((uint32_t)(l0 * MX_K) << ish) + (2u << ish) * tid : a.nb_I;
    const uint32_t w0 = ld32(R.I, oi), w1 = ld32(R.I, a.idx16 ? oi : oi + 4u);
    p.iv = make_uint2(w0, w1);   // decoded where used (idx_pair), so the loads stay in flight
    const uint32_t ow = live ? (uint32_t)(l0 * MX_K * 2) + 4u * tid : a.nb_W;
    p.wv = ld32(R.W, ow);
    const int64_t l = l0 + lab;
    const bool ok = live && l < a.L;
    const uint32_t om = ok ? (uint32_t)(l * MX_K + slot) * 4u : a.nb_m;
    if constexpr (MOMENTS) {
        p.m = ldf2(R.m, om);
        p.v = ldf2(R.v, om);
    } else {
        p.m = p.v = make_float2(0.f, 0.f);
    }
    p.b = ldf(R.b, ok ? (uint32_t)l * 4u : a.nb_b);
}

// NT = column tiles of 16 per wave: d = 128 * NT (a compile-time width keeps
// the dX accumulators in fixed registers)
// SETF: this pass applies Adam and then SET prune-and-regrow to every row
// (only with MODE MX_ONLY or MX_LAST)
template <int NT, int MODE, bool SETF>
__global__ void __launch_bounds__(MX_THREADS, 1) k_sweep_mx(const MxArgs a) {
    constexpr bool ADAM = MODE == MX_ONLY || MODE == MX_LAST;      // updates W, m, v, bias
    constexpr bool CARRY_IN = MODE == MX_LAST || MODE == MX_MIDDLE;
    extern __shared__ __align__(16) unsigned char lds[];
    constexpr int d = 128 * NT;
    unsigned char *Xs = lds;                                                // d * 128
    uint16_t *T = reinterpret_cast<uint16_t *>(lds + (size_t)d * MX_XS);    // d * 32
    uint16_t *G = T + (size_t)d * MX_NLAB;                                  // 64 * 32
    int32_t *Is = reinterpret_cast<int32_t *>(G + MX_NB * MX_NLAB);        // 32 * 32
    uint32_t *Ws = reinterpret_cast<uint32_t *>(Is + MX_NLAB * MX_K);      // 32 * 16
    uint32_t *tg = Ws + MX_NLAB * (MX_K / 2);                              // MX_TG_MAX
    uint32_t *ym = tg;   // [32][2]: only when the positives do not fit in tg
    // SETF: the first four regrowth candidates of each wave's rows of the next
    // MX_SET_AHEAD chunks, [wave][chunk][row][4] u16
    uint16_t *Pc = reinterpret_cast<uint16_t *>(tg + MX_TG_MAX);

    const int tid = threadIdx.x;
    const int lab = tid >> 4, u = tid & 15;
    const int wave = tid >> 6, lane = tid & 63;
    // register r of a lane holds slot r ^ Kp; Kp = lane_key with bit 1 cleared,
    // so the lane reads its row's slots four at a time (two pairs).  The lane
    // ends the dW reduce-scatter with the slots Kown, Kown + 1.
    const int Kp = lane_key(u) & ~2;
    const int Kown = Kp + 2 * (u & 1);
    const int nnz = a.nnz;
    const bool tg_lds = nnz <= MX_TG_MAX;

    Rsrcs R;
    R.XT = make_rsrc(a.XT, (uint32_t)d * MX_XS);
    R.K = make_rsrc(a.keys, tg_lds ? MX_TG_MAX * 4u : 0u);
    R.W = make_rsrc(a.W, a.nb_W);
    R.I = make_rsrc(a.I, a.nb_I);
    R.m = make_rsrc(a.m, a.nb_m);
    R.v = make_rsrc(a.v, a.nb_m);
    R.b = make_rsrc(a.bias, a.nb_b);
    R.bm = make_rsrc(a.bm, a.nb_b);
    R.bv = make_rsrc(a.bv, a.nb_b);
    R.dwp = make_rsrc(a.dwp, MODE == MX_ONLY ? 0u : a.nb_m);
    R.dbp = make_rsrc(a.dbp, MODE == MX_ONLY ? 0u : a.nb_b);
    R.mk = make_rsrc(a.set_mask, SETF ? a.nb_mask : 0u);

    Prefetch pa, pb;
    prefetch<ADAM>(a, R, blockIdx.x, tid, lab, u, Kown, pa);

    // stage the pass's X tile (transposed and zero-padded past B by the batch
    // prep) with 16-byte copies, its sorted positives, and clear T.  The
    // positives are keys (label << 6 | sample), ascending (a label outside
    // [0,L) is the largest key and is never matched).  Chunks of one
    // workgroup come in ascending order, so a cursor that only moves forward
    // finds each chunk's positives.
    {
#pragma unroll
        for (int it = 0; it < d / 64; ++it) {
            const uint32_t o = (uint32_t)(tid + it * MX_THREADS) * 16u;
            const auto q = __builtin_amdgcn_raw_buffer_load_b128(R.XT, o, 0, 0);
            *reinterpret_cast<uint4 *>(Xs + o) = make_uint4(q[0], q[1], q[2], q[3]);
        }
        if (tg_lds) {
            tg[tid] = ld32(R.K, 4u * tid);
            tg[tid + MX_THREADS] = ld32(R.K, 4u * (tid + MX_THREADS));
        }
        for (int e = tid; e < d * MX_NLAB / 2; e += MX_THREADS) reinterpret_cast<uint32_t *>(T)[e] = 0u;
    }
    __syncthreads();

    // dX accumulators: 4 batch tiles x NT column tiles of 16 per wave (8 waves)
    const int cbase = wave * (d / 8);
    f32x4 acc[4][NT];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

    float loss_acc = 0.f;
    const float decay = 1.f - a.adam.lr * a.adam.wd;
    const float inv_bc1 = 1.f / a.adam.bc1, inv_bc2 = 1.f / a.adam.bc2;
    const float b1 = a.adam.b1, b2 = a.adam.b2, lr = a.adam.lr, eps = a.adam.eps;
    int pos = 0;              // first sorted key not below the current chunk
    uint32_t head = 0xffffffffu;   // tg[pos] (uniform), or the largest key past the end
    if (tg_lds && nnz > 0) head = __builtin_amdgcn_readfirstlane(tg[0]);
    int32_t c0 = 0, c1 = 0;   // T columns written by this lane in the previous chunk

    // One chunk: `cur` holds its rows and optimiser state, `nxt` receives the
    // next chunk's.
    auto step = [&](int64_t chunk, const Prefetch &cur, Prefetch &nxt) {
        const int64_t l0 = chunk * MX_NLAB;
        const uint32_t l0u = (uint32_t)l0;   // L < 2^25: label offsets fit in 32 bits
        // this workgroup's chunk count so far
        const int ci = (int)((chunk - blockIdx.x) / gridDim.x);
        if constexpr (SETF) {
            // Every MX_SET_AHEAD chunks a wave draws the first Philox block of
            // its rows in the next MX_SET_AHEAD chunks, one row per lane (each
            // row's 16 lanes would otherwise all draw the same block), and
            // keeps the four candidate columns.
            if ((ci & (MX_SET_AHEAD - 1)) == 0 && lane < 4 * MX_SET_AHEAD) {
                const int64_t lr = (chunk + (int64_t)(lane >> 2) * gridDim.x) * MX_NLAB + 4 * wave + (lane & 3);
                uint64_t p0 = (uint64_t)lr, p1 = a.set_round, p2 = 0, p3 = 0;
                philox4x64_10(p0, p1, p2, p3, a.set_seed, SET_KEY_HI);
                typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));
                const u16x4 cw = {(uint16_t)__umul64hi(p0, (uint64_t)d), (uint16_t)__umul64hi(p1, (uint64_t)d),
                                  (uint16_t)__umul64hi(p2, (uint64_t)d), (uint16_t)__umul64hi(p3, (uint64_t)d)};
                *reinterpret_cast<u16x4 *>(Pc + (wave * 4 * MX_SET_AHEAD + lane) * 4) = cw;
            }
        }

        // stage this chunk's rows: indices become clamped byte offsets of X columns
        {
            const uint2 ip = idx_pair(cur.iv, a.idx16);
            const int i0 = min(max((int)ip.x, 0), d - 1), i1 = min(max((int)ip.y, 0), d - 1);
            *reinterpret_cast<int2 *>(Is + 2 * tid) = make_int2(i0 * MX_XS, i1 * MX_XS);
            Ws[tid] = cur.wv;
            if (!tg_lds && tid < MX_NLAB * 2) ym[tid] = 0u;
        }
        prefetch<ADAM>(a, R, chunk + gridDim.x, tid, lab, u, Kown, nxt);
        // The gathers read only X and the index rows this wave's own lanes
        // staged above, so they need no barrier: issued here, their LDS
        // latency runs on while the wave waits at the barrier below.
        wave_lds_sync();
        const int pc0 = c0, pc1 = c1;   // T columns written in the previous chunk
        int rl = lab;            // the row of the chunk this lane serves
        int k4 = Kp >> 2;        // quad order of this lane
        // opaque per chunk, so the per-slot LDS addresses are formed where
        // they are used instead of being held in registers across chunks
        asm volatile("" : "+v"(rl), "+v"(k4));
        // row data in the lane's slot order: register r <-> slot r ^ K (a row
        // past L has zero offsets and weights)
        uint32_t wp[MX_K / 2];
        uint2 xg[MX_K];
        const bool odd = (u & 1) != 0;
        uint32_t wpair_own = 0u;
#pragma unroll
        for (int q = 0; q < MX_K / 4; ++q) {
            const int qq = q ^ k4;   // registers 4q..4q+3 hold slots 4qq..4qq+3
            const int4 iv = *reinterpret_cast<const int4 *>(Is + rl * MX_K + 4 * qq);
            const uint2 wv = *reinterpret_cast<const uint2 *>(Ws + rl * (MX_K / 2) + 2 * qq);
            if (q == 0) {   // the lane's own slots are registers 2*odd, 2*odd + 1
                c0 = (odd ? iv.z : iv.x) / MX_XS;
                c1 = (odd ? iv.w : iv.y) / MX_XS;
                wpair_own = odd ? wv.y : wv.x;
            }
            xg[4 * q] = *reinterpret_cast<const uint2 *>(Xs + iv.x + 8 * u);
            xg[4 * q + 1] = *reinterpret_cast<const uint2 *>(Xs + iv.y + 8 * u);
            xg[4 * q + 2] = *reinterpret_cast<const uint2 *>(Xs + iv.z + 8 * u);
            xg[4 * q + 3] = *reinterpret_cast<const uint2 *>(Xs + iv.w + 8 * u);
            wp[2 * q] = wv.x;
            wp[2 * q + 1] = wv.y;
        }
        __syncthreads();
        // Every wave has read the previous chunk's G and T fragments before the
        // barrier above, so this lane's T entries of that chunk can be cleared;
        // the entries of one row are only ever touched by the wave that owns
        // the row, in program order.
        T[swz(pc0, lab)] = 0;
        T[swz(pc1, lab)] = 0;

        // targets of this lane's row as a 64-bit sample mask
        uint64_t yrow = 0;
        if (tg_lds) {
            // a chunk without positives costs one compare of the cached head key;
            // the cursor only moves past keys of chunks already behind
            while ((head >> 6) < l0u) {
                ++pos;
                head = pos < nnz ? __builtin_amdgcn_readfirstlane(tg[pos]) : 0xffffffffu;
            }
            if ((head >> 6) - l0u < (uint32_t)MX_NLAB) {
                for (int e = pos; e < nnz; ++e) {
                    const uint32_t key = tg[e];
                    const uint32_t ll = (key >> 6) - l0u;
                    if (ll >= (uint32_t)MX_NLAB) break;
                    if (ll == (uint32_t)lab) yrow |= 1ull << (key & 63u);
                }
            }
        } else {
            for (int e = tid; e < nnz; e += MX_THREADS) {
                const uint32_t ll = (uint32_t)a.tgt_lab[e] - l0u;
                const uint32_t b = (uint32_t)(a.tgt_b[e] - a.b0);
                if (ll < MX_NLAB && b < (uint32_t)a.B) atomicOr(&ym[ll * 2 + (b >> 5)], 1u << (b & 31));
            }
            __syncthreads();
            yrow = (uint64_t)ym[lab * 2] | ((uint64_t)ym[lab * 2 + 1] << 32);
        }

        {
            const int64_t l = l0 + rl;
            const bool valid = l < a.L;
            // the bias moments, used on lane u = 0 at the end of the row's work
            const uint32_t obm = valid && u == 0 ? (uint32_t)l * 4u : a.nb_b;
            float bmcur = 0.f, bvcur = 0.f;
            if constexpr (ADAM) {
                bmcur = ldf(R.bm, obm);
                bvcur = ldf(R.bv, obm);
            }
            // dW and dbias of this row summed over the earlier batch passes
            const uint32_t odw = valid ? (uint32_t)(l * MX_K + Kown) * 4u : a.nb_m;
            float2 dprev = make_float2(0.f, 0.f);
            float dbprev = 0.f;
            if constexpr (CARRY_IN) {
                dprev = ldf2(R.dwp, odw);
                dbprev = ldf(R.dbp, obm);
            }

            // forward: repack (b, b+1) pairs of two slots into slot pairs
            float z[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int p = 0; p < MX_K / 2; ++p) {
                const uint2 A = xg[2 * p], Bv = xg[2 * p + 1];
                z[0] = dot2(__builtin_amdgcn_perm(Bv.x, A.x, 0x05040100u), wp[p], z[0]);
                z[1] = dot2(__builtin_amdgcn_perm(Bv.x, A.x, 0x07060302u), wp[p], z[1]);
                z[2] = dot2(__builtin_amdgcn_perm(Bv.y, A.y, 0x05040100u), wp[p], z[2]);
                z[3] = dot2(__builtin_amdgcn_perm(Bv.y, A.y, 0x07060302u), wp[p], z[3]);
            }
            // BCE and dlogits for rows 4u..4u+3; zero for padded samples and
            // rows past L
            const uint32_t yw = (uint32_t)(yrow >> (4 * u));
            float g[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const bool live = valid && 4 * u + e < a.B;
                const float zz = z[e] + cur.b;
                const float y = ((yw >> e) & 1u) ? 1.f : 0.f;
                if (a.hinge) {
                    // squared hinge with yh = 2y - 1
                    const float yh = 2.f * y - 1.f;
                    const float hh = fmaxf(1.f - yh * zz, 0.f);
                    loss_acc += live ? hh * hh : 0.f;
                    g[e] = live ? -2.f * a.s * yh * hh : 0.f;
                } else {
                    // exp(-|z|) in (0, 1] and log(1 + exp(-|z|)) with the
                    // hardware base-2 exp and log (their arguments need no
                    // range reduction)
                    const float ex = __builtin_amdgcn_exp2f(-fabsf(zz) * 1.4426950408889634f);
                    const float opx = 1.f + ex;
                    const float r = __builtin_amdgcn_rcpf(opx);
                    const float sig = zz >= 0.f ? r : ex * r;
                    loss_acc += live ? fmaxf(zz, 0.f) - zz * y + __builtin_amdgcn_logf(opx) * 0.6931471805599453f
                                     : 0.f;
                    g[e] = live ? a.s * (sig - y) : 0.f;
                }
            }
            // dW partials over the lane's rows, slot order r ^ Kp
            const uint32_t g01 = pack_bf16(g[0], g[1]), g23 = pack_bf16(g[2], g[3]);
            // a wave whose dlogits are all zero (a hinge loss past its margin
            // everywhere, Sec. 2.2) has zero dW: its products are skipped
            float dw0 = dprev.x, dw1 = dprev.y;
            if (__builtin_amdgcn_ballot_w64((g01 | g23) != 0u) != 0) {
                float pw[MX_K];
#pragma unroll
                for (int r = 0; r < MX_K; ++r) pw[r] = dot2(xg[r].y, g23, dot2z(xg[r].x, g01));
                // reduce-scatter over the 16 lanes of the row
                const float2 dws = reduce_scatter16(pw, odd);
                dw0 += dws.x;
                dw1 += dws.y;
            }
            if constexpr (!ADAM) stf2(R.dwp, odw, make_float2(dw0, dw1));
            // Adam on slots Kown, Kown+1
            if constexpr (ADAM) {
                float m0 = cur.m.x, m1 = cur.m.y, v0 = cur.v.x, v1 = cur.v.y;
                const float w0 = __uint_as_float(wpair_own << 16);
                const float w1 = __uint_as_float(wpair_own & 0xffff0000u);
                const float n0 = adam_step(w0, dw0, m0, v0, b1, b2, inv_bc1, inv_bc2, lr, eps, decay);
                const float n1 = adam_step(w1, dw1, m1, v1, b1, b2, inv_bc1, inv_bc2, lr, eps, decay);
                const uint32_t o = (uint32_t)(l * MX_K + Kown);
                uint32_t wnew = pack_bf16(n0, n1);
                if constexpr (SETF) {
                    // SET on the updated row (Sec. 2.1): the n slots with the
                    // smallest keys (|W| bits, slot) of the stored bf16 weights.
                    // Every lane of the row finds the same slots: n rounds of a
                    // row-wide minimum, the owner of each minimum dropping it.
                    const uint32_t k0 = ((wnew & 0x7fffu) << 5) | (uint32_t)Kown;
                    const uint32_t k1 = (((wnew >> 16) & 0x7fffu) << 5) | (uint32_t)(Kown + 1);
                    uint32_t klo = min(k0, k1), khi = max(k0, k1);
                    uint32_t sel = 0;   // the row's pruned slots
                    for (int q = 0; q < a.set_n; ++q) {
                        const uint32_t mn = min16(klo);
                        sel |= 1u << (mn & 31u);
                        if (klo == mn) {
                            klo = khi;
                            khi = 0xffffffffu;
                        }
                    }
                    // Regrowth: attempt t takes word t mod 4 of Philox4x64-10 at
                    // counter (row, round, t / 4, 0); a column the row held
                    // before pruning or one already accepted is drawn again.
                    // Lane j of the row keeps the j-th accepted column, so one
                    // ballot over the row's lanes answers both questions.
                    int acol = -1;
                    int got = 0;
                    const int rsh = 16 * (lab & 3);   // this row's lanes in a wave-wide ballot
                    auto offer = [&](int c) {
                        const uint64_t held = __builtin_amdgcn_ballot_w64(c == c0 || c == c1 || c == acol);
                        if (((held >> rsh) & 0xffffull) == 0) {
                            if (u == got) acol = c;
                            ++got;
                        }
                    };
                    // attempts 0-3: the candidates drawn ahead
                    {
                        typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));
                        const u16x4 cw = *reinterpret_cast<const u16x4 *>(
                            Pc + (wave * 4 * MX_SET_AHEAD + 4 * (ci & (MX_SET_AHEAD - 1)) + (lab & 3)) * 4);
#pragma unroll
                        for (int q = 0; q < 4; ++q)
                            if (got < a.set_n) offer((int)cw[q]);
                    }
                    // A row that met a held column among its first four draws
                    // is left as the plain step leaves it and goes on a list
                    // that SET then processes row by row (later draws are
                    // rare, and drawing them here costs every row registers)
                    if (got < a.set_n) {
                        sel = 0;
                        if (valid && u == 0) a.set_list[1 + atomicAdd(a.set_list, 1)] = (int32_t)l;
                    }
                    // pruned slots restart at zero
                    if ((sel >> Kown) & 1u) {
                        wnew &= 0xffff0000u;
                        m0 = v0 = 0.f;
                    }
                    if ((sel >> (Kown + 1)) & 1u) {
                        wnew &= 0x0000ffffu;
                        m1 = v1 = 0.f;
                    }
                    // the row's index words (this lane's load: slots 2u, 2u+1),
                    // rewritten whole: the regrown columns fill the pruned
                    // slots in ascending slot order, the others keep their bits
                    const int s0 = 2 * u, s1 = 2 * u + 1;
                    const int r0 = __builtin_popcount(sel & ((1u << s0) - 1u));
                    const int r1 = r0 + (int)((sel >> s0) & 1u);
                    const int rowlane = lane & ~15;   // lane 0 of this row in the wave
                    const uint32_t n0c = (uint32_t)__builtin_amdgcn_ds_bpermute(4 * (rowlane + min(r0, 15)), acol);
                    const uint32_t n1c = (uint32_t)__builtin_amdgcn_ds_bpermute(4 * (rowlane + min(r1, 15)), acol);
                    const uint2 ip = idx_pair(cur.iv, a.idx16);
                    const uint32_t iw0 = ((sel >> s0) & 1u) ? n0c : ip.x;
                    const uint32_t iw1 = ((sel >> s1) & 1u) ? n1c : ip.y;
                    if (a.idx16) {
                        st32(R.I, valid ? (uint32_t)(l * MX_K + s0) * 2u : a.nb_I, (iw0 & 0xffffu) | (iw1 << 16));
                    } else {
                        typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
                        const u32x2 iw = {iw0, iw1};
                        const uint32_t oi = valid ? (uint32_t)(l * MX_K + s0) * 4u : a.nb_I;
                        __builtin_amdgcn_raw_buffer_store_b64(iw, R.I, oi, 0, 0);
                    }
                    const uint16_t mk = (uint16_t)(((sel >> s0) & 1u) | (((sel >> s1) & 1u) << 8));
                    __builtin_amdgcn_raw_buffer_store_b16(mk, R.mk, valid ? (uint32_t)(l * MX_K + s0) : a.nb_mask, 0, 0);
                }
                stf2(R.m, valid ? 4u * o : a.nb_m, make_float2(m0, m1));
                stf2(R.v, valid ? 4u * o : a.nb_m, make_float2(v0, v1));
                st32(R.W, valid ? 2u * o : a.nb_W, wnew);
            }
            // bias: sum of g over the 64 rows, lane u == 0 updates
            {
                float sg = (g[0] + g[1]) + (g[2] + g[3]);
                sg = add_dpp<DPP_ROW_MIRROR>(sg, sg);
                sg = add_dpp<DPP_ROW_HALF_MIRROR>(sg, sg);
                sg = add_dpp<DPP_QUAD_3210>(sg, sg);
                sg = add_dpp<DPP_QUAD_1032>(sg, sg) + dbprev;
                if constexpr (ADAM) {
                    float mm = bmcur, vv = bvcur;
                    const float nb = adam_step(cur.b, sg, mm, vv, b1, b2, inv_bc1, inv_bc2, lr, eps, decay);
                    stf(R.b, obm, nb);
                    stf(R.bm, obm, mm);
                    stf(R.bv, obm, vv);
                } else {
                    stf(R.dbp, obm, sg);
                }
            }
            // dX inputs: g and the old weights (a row past L writes zeros at column 0)
#pragma unroll
            for (int e = 0; e < 4; ++e)
                G[swz(4 * u + e, rl)] = (uint16_t)((e < 2 ? g01 : g23) >> (16 * (e & 1)));
            T[swz(c0, rl)] = (uint16_t)(wpair_own & 0xffffu);
            T[swz(c1, rl)] = (uint16_t)(wpair_own >> 16);
        }
        __syncthreads();
        // dX += G (64 x 32) * T^T (32 x d) on the matrix cores; this wave owns
        // columns [wave*d/8, (wave+1)*d/8).  The MFMAs run on while the next
        // chunk starts; its first barrier orders the fragment reads before any
        // rewrite of G or T.
        {
            const int col = lane & 15, kq = lane >> 4;
            bf16x8 af[4];
#pragma unroll
            for (int mt = 0; mt < 4; ++mt)
                af[mt] = *reinterpret_cast<const bf16x8 *>(G + swz(16 * mt + col, 8 * kq));
            bf16x8 bfr[NT];
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
                bfr[nt] = *reinterpret_cast<const bf16x8 *>(T + swz(cbase + 16 * nt + col, 8 * kq));
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
#pragma unroll
                for (int mt = 0; mt < 4; ++mt)
                    acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[mt], bfr[nt], acc[mt][nt], 0, 0, 0);
        }
    };

    if constexpr (SETF) {
        // one chunk per iteration, the next chunk's registers copied at the
        // end of the step (its loads have landed by then): with SET's state
        // the two-chunk body below exceeds the registers and spills, this one
        // does not
        for (int64_t chunk = blockIdx.x; chunk < a.nchunks; chunk += gridDim.x) {
            step(chunk, pa, pb);
            pa = pb;
        }
    } else {
        // two chunks per iteration, so the prefetch buffers swap roles instead
        // of being copied (a copy would wait for the loads in flight)
        for (int64_t chunk = blockIdx.x; chunk < a.nchunks; chunk += 2 * (int64_t)gridDim.x) {
            step(chunk, pa, pb);
            if (chunk + gridDim.x >= a.nchunks) break;
            step(chunk + gridDim.x, pb, pa);
        }
    }

    // write this workgroup's dX partial [B][d]
    {
        float *P = a.dx_part + ((size_t)blockIdx.x * a.Btot + a.b0) * d;
        const int col = lane & 15, kq = lane >> 4;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
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
    // loss: workgroup tree reduction in the (now unused) G tile
    float *red = reinterpret_cast<float *>(G);
    __syncthreads();
    red[tid] = loss_acc;
    __syncthreads();
    for (int st = MX_THREADS / 2; st > 0; st >>= 1) {
        if (tid < st) red[tid] += red[tid + st];
        __syncthreads();
    }
    if (tid == 0) a.loss_part[blockIdx.x] = red[0];
}

constexpr int MX_NT_MAX = 6;    // widest input: 768 columns

typedef void (*MxKernel)(const MxArgs);
template <int NT>
struct MxModes {
    static constexpr MxKernel k[4] = {k_sweep_mx<NT, MX_ONLY, false>, k_sweep_mx<NT, MX_FIRST, false>,
                                      k_sweep_mx<NT, MX_LAST, false>, k_sweep_mx<NT, MX_MIDDLE, false>};
    // the passes that apply Adam, with SET fused
    static constexpr MxKernel kset[4] = {k_sweep_mx<NT, MX_ONLY, true>, nullptr, k_sweep_mx<NT, MX_LAST, true>,
                                         nullptr};
};
MxKernel mx_kernel(int nt, int mode, bool setf) {
    switch (nt) {
    case 1: return setf ? MxModes<1>::kset[mode] : MxModes<1>::k[mode];
    case 2: return setf ? MxModes<2>::kset[mode] : MxModes<2>::k[mode];
    case 3: return setf ? MxModes<3>::kset[mode] : MxModes<3>::k[mode];
    case 4: return setf ? MxModes<4>::kset[mode] : MxModes<4>::k[mode];
    case 5: return setf ? MxModes<5>::kset[mode] : MxModes<5>::k[mode];
    default: return setf ? MxModes<6>::kset[mode] : MxModes<6>::k[mode];
    }
}

size_t sweep_mx_lds(int d, bool setf = false) {
    return (size_t)d * MX_XS + (size_t)d * MX_NLAB * 2 + MX_NB * MX_NLAB * 2 + MX_NLAB * MX_K * 4 +
           MX_NLAB * (MX_K / 2) * 4 + MX_TG_MAX * 4 + (setf ? (MX_THREADS / 64) * 4 * MX_SET_AHEAD * 8 : 0);
}

}  // namespace

bool sweep_mx_eligible(const Layer &ly, int B, int mode) {
    static_assert(MX_K == 32 && MX_NT_MAX * 128 == 768, "the shape predicate mx_shape");
    return mode == SWEEP_FUSED && ly.vt == FFSL_BF16 && mx_shape(ly.L, ly.d, ly.k) && B <= FFSL_MAX_B &&
           sweep_mx_lds(ly.d) <= 160 * 1024;
}

// With c.set_n in [1, MX_SET_NMAX] the pass that applies Adam also applies
// SET to every row (the SETF kernels).
// Batches of up to 64 samples take one pass.  A larger batch is split into
// passes of 64 samples: every pass accumulates its samples' dX rows and loss,
// the first stores its dW / dbias in the carry buffers, middle passes add to
// them, and the last adds its share and applies Adam.  W, the moments and the
// bias change only in the last pass, so every pass sees the step's old state.
int launch_sweep_mx(const SweepCall &c, const FastBufs &fb, int *grid_out, int *passes_out) {
    const Layer &ly = *c.layer;
    MxArgs a{};
    a.L = ly.L;
    a.d = ly.d;
    a.nnz = c.nnz;
    a.nchunks = (ly.L + MX_NLAB - 1) / MX_NLAB;
    a.W = static_cast<uint16_t *>(ly.W);
    a.I = ly.I;
    a.bias = ly.bias;
    a.m = ly.m;
    a.v = ly.v;
    a.bm = ly.bm;
    a.bv = ly.bv;
    a.tgt_b = fb.tgt_b;
    a.tgt_lab = c.tgt_lab;
    a.s = c.s;
    a.adam = c.adam;
    a.dx_part = fb.dx_part;
    a.dwp = fb.dwp;
    a.dbp = fb.dbp;
    a.Btot = c.B;
    a.hinge = (c.flags & FFSL_LOSS_SQHINGE) ? 1 : 0;
    const bool setf = c.set_n >= 1 && c.set_n <= MX_SET_NMAX && sweep_mx_lds(ly.d, true) <= 160 * 1024;
    a.set_n = c.set_n;
    a.set_seed = c.set_seed;
    a.set_round = c.set_round;
    a.set_mask = c.set_mask;
    a.set_list = fb.set_list;
    a.nb_mask = c.set_mask ? (uint32_t)(ly.L * MX_K) : 0u;
    a.nb_W = (uint32_t)(ly.L * MX_K * 2);
    a.idx16 = ly.idx16;
    a.nb_I = (uint32_t)(ly.L * MX_K * (ly.idx16 ? 2 : 4));
    a.nb_m = (uint32_t)(ly.L * MX_K * 4);
    a.nb_b = ly.bias ? (uint32_t)(ly.L * 4) : 0u;
    const int grid = (int)std::min<int64_t>(a.nchunks, std::min(ly.max_parts, ly.num_cu));
    const int passes = (c.B + MX_NB - 1) / MX_NB;
    if (ly.ev_start) {
        hipError_t e = hipEventRecord(ly.ev_start, c.stream);
        if (e != hipSuccess) return fail(FFSL_EHIP, "hipEventRecord: %s", hipGetErrorString(e));
    }
    for (int p = 0; p < passes; ++p) {
        const int mode = passes == 1 ? MX_ONLY : p == 0 ? MX_FIRST : p == passes - 1 ? MX_LAST : MX_MIDDLE;
        a.b0 = p * MX_NB;
        a.B = std::min(MX_NB, c.B - a.b0);
        a.XT = fb.xt + (size_t)p * ly.d * MX_NB;
        a.keys = fb.keys + (size_t)p * MX_TG_MAX;
        a.loss_part = fb.loss_part + (size_t)p * grid;
        const bool kset = setf && (mode == MX_ONLY || mode == MX_LAST);
        const MxKernel kern = mx_kernel(ly.d / 128, mode, kset);
        const size_t shm = sweep_mx_lds(ly.d, kset);
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
        if (e != hipSuccess) return fail(FFSL_EHIP, "hipFuncSetAttribute: %s", hipGetErrorString(e));
        hipLaunchKernelGGL(kern, dim3(grid), dim3(MX_THREADS), shm, c.stream, a);
        int rc = check_launch("sweep_mx");
        if (rc) return rc;
    }
    if (ly.ev_stop) {
        hipError_t e = hipEventRecord(ly.ev_stop, c.stream);
        if (e != hipSuccess) return fail(FFSL_EHIP, "hipEventRecord: %s", hipGetErrorString(e));
    }
    if (setf) {
        // the rows whose first four draws did not suffice
        int rc = launch_set_rows(ly, c.set_n, c.set_seed, c.set_round, c.set_mask, c.set_exhausted, fb.set_list,
                                 c.stream);
        if (rc) return rc;
    }
    *grid_out = grid;
    *passes_out = passes;
    if (setf && c.set_fused) *c.set_fused = true;
    return FFSL_OK;
}

}  // namespace ffsl
