// Fused training step of the fixed fan-in layer for bf16 values, fan-in 64 and
// wide inputs (d a multiple of 128 up to 2048, the intermediate-layer width):
// the gathered forward, BCE, dW, dbias, dX and Adam of Sec. 2.2.
//
// At d = 2048 neither X for 64 samples (256 KB) nor a 32-row weight tile for
// the dX product (128 KB) fits next to the other in the 160 KB of LDS, and a
// dX accumulator of 64 samples (512 KB) exceeds the register file.  The batch
// therefore runs in passes of 16 samples (see launch_sweep_wide), each one
// sweep over the [L,k] arrays:
//
// Workgroup: 512 threads (8 waves), one per CU, persistent over chunks of 16
// label rows.  Thirty-two lanes serve one row: lane u handles the four
// samples 4q .. 4q+3 of the pass, q = u >> 3, and the eight slots
// 8g .. 8g+7 of the row, g = u & 7.
//
//   LDS  Xs [d][16] bf16   the pass's samples transposed (column i is 32
//                          contiguous bytes), zero-padded past the pass
//        T  [d][16] bf16   the chunk's weights scattered densely by column
//        G  [16][16] bf16  the chunk's dlogits (both with the 8-byte quarters
//                          of a row rotated every 4 rows, see qswz)
//        Is, Ws            the chunk's index rows (as byte offsets into Xs)
//                          and weight rows; each wave stages its own two rows
//        tg                the pass's positives as sorted (label, sample) keys
//
//   1. gather: for each of its 8 slots the lane reads the 8 bytes
//      X[4q .. 4q+3, I[l,j]]; the sample pairs are repacked into slot pairs
//      with v_perm and reduced with v_dot2 against the row's weight pairs,
//      and the eight slot groups' partial scores meet in an 8-lane DPP sum;
//   2. BCE loss and dlogit g: lane u computes sample 4q + (u & 3) and the
//      quad's four values reach every lane of it by DPP broadcast;
//   3. dW: two v_dot2 per slot over the lane's four samples (g rounded to
//      bf16), then a reduce-scatter over the four quads: one
//      v_permlane16_swap level and one DPP level (register i holds slot
//      i ^ 2(q & 1) of the group; the lane keeps slots 2q, 2q+1);
//   4. Adam on those two slots, streaming W, m, v back to HBM;
//   5. dX: g and the old weights go to G and T, and the matrix cores add
//      G x T^T (16 x 16 by 16 x d) into a per-workgroup dX in registers (each
//      wave owns the 16-column tiles w, w+8, ...), written out at the end.
// All HBM accesses of the chunk loop are range-checked buffer operations: a
// row past L reads zeros and its writes are dropped.
#include <utility>

#include "sweep_dev.h"

namespace ffsl {

namespace {

using namespace fdev;

constexpr int WD_THREADS = 512;
constexpr int WD_NLAB = 16;      // label rows per chunk
constexpr int WD_K = 64;         // fan-in of this path
constexpr int WD_NB = 16;        // samples per pass
constexpr int WD_XS = 32;        // bytes per X column row in LDS
constexpr int WD_TG_MAX = 1024;  // positives kept in LDS
constexpr int WD_NT_MAX = 16;    // widest input: 2048 columns

typedef short s16x4 __attribute__((ext_vector_type(4)));

struct WdArgs {
    int64_t L;
    int32_t d, B, nnz;
    int64_t nchunks;
    const uint16_t *XT;     // this pass's samples transposed, [d][16] (batch prep)
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
    // passes in dwp [L][64], dbp [L]
    int32_t b0, Btot;
    float *dwp, *dbp;
    int32_t hinge;   // squared hinge instead of BCE
};

struct Rsrcs {
    Rsrc XT, K, W, I, m, v, b, bm, bv, dwp, dbp;
};

// G and T rows hold 16 bf16 (32 bytes = four 8-byte quarters).  A matrix-core
// fragment reads one quarter from each of 16 consecutive rows; stored plainly,
// rows r, r+4, ... would share banks.  Quarter q of row r is kept at quarter
// q ^ ((r >> 2) & 3); element e of row r sits at:
__device__ __forceinline__ int qswz(int r, int e) {
    return r * 16 + ((((e >> 2) ^ (r >> 2)) & 3) << 2) + (e & 3);
}

struct Prefetch {
    uint2 iv;          // the lane's two index words as loaded (see idx_pair)
    uint32_t wv;       // one weight word of the chunk's W rows
    float2 m, v;       // moments of the lane's two slots of its row
    float b;           // its bias
};

// the chunk's rows and optimiser state (the moments only for a pass that
// applies Adam), loaded a chunk ahead of their use; a chunk or row past the
// end reads zeros.  Lane tid loads words of row tid / 32 only: a row its wave
// serves.
template <bool MOMENTS>
__device__ __forceinline__ void prefetch(const WdArgs &a, const Rsrcs &R, int64_t chunk, int tid, int lab,
                                         int slot, Prefetch &p) {
    const int64_t l0 = chunk * WD_NLAB;
    const bool live = chunk < a.nchunks;
    // two word loads either way (no load reaches past the array): with 16-bit
    // indices both read the one word that holds the lane's two slots
    const uint32_t ish = a.idx16 ? 1u : 2u;   // log2 of the index bytes
    const uint32_t oi = live ? ((uint32_t)(l0 * WD_K) << ish) + (2u << ish) * tid : a.nb_I;
    const uint32_t w0 = ld32(R.I, oi), w1 = ld32(R.I, a.idx16 ? oi : oi + 4u);
    p.iv = make_uint2(w0, w1);   // decoded where used (idx_pair), so the loads stay in flight
    p.wv = ld32(R.W, live ? (uint32_t)(l0 * WD_K * 2) + 4u * tid : a.nb_W);
    const int64_t l = l0 + lab;
    const bool ok = live && l < a.L;
    const uint32_t om = ok ? (uint32_t)(l * WD_K + slot) * 4u : a.nb_m;
    if constexpr (MOMENTS) {
        p.m = ldf2(R.m, om);
        p.v = ldf2(R.v, om);
    } else {
        p.m = p.v = make_float2(0.f, 0.f);
    }
    p.b = ldf(R.b, ok ? (uint32_t)l * 4u : a.nb_b);
}

// NT = d / 128: the d / 16 column tiles of 16 are dealt to the 8 waves, NT each
template <int NT, int MODE>
__global__ void __launch_bounds__(WD_THREADS, 1) k_sweep_wide(const WdArgs a) {
    constexpr bool ADAM = MODE == PASS_ONLY || MODE == PASS_LAST;      // updates W, m, v, bias
    constexpr bool CARRY_IN = MODE == PASS_LAST || MODE == PASS_MIDDLE;
    constexpr int d = 128 * NT;
    extern __shared__ __align__(16) unsigned char lds[];
    unsigned char *Xs = lds;                                                  // d * 32
    uint16_t *T = reinterpret_cast<uint16_t *>(lds + (size_t)d * WD_XS);      // d * 16
    uint16_t *G = T + (size_t)d * WD_NLAB;                                    // 16 * 16
    int32_t *Is = reinterpret_cast<int32_t *>(G + WD_NB * WD_NLAB);          // 16 * 64
    uint16_t *Ws = reinterpret_cast<uint16_t *>(Is + WD_NLAB * WD_K);        // 16 * 64
    uint32_t *tg = reinterpret_cast<uint32_t *>(Ws + WD_NLAB * WD_K);        // WD_TG_MAX

    const int tid = threadIdx.x;
    const int lab = tid >> 5, u = tid & 31;
    const int qd = u >> 3, grp = u & 7;         // sample quad of the pass, slot group of the row
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
    // the reduce-scatter over the quads leaves the lane with slots 2 qd,
    // 2 qd + 1 of its group
    const int myslot = 8 * grp + 2 * qd;
    const int sj = grp & 3;                     // the sample of its quad whose dlogit the lane computes
    const int nnz = a.nnz;
    const bool tg_lds = nnz <= WD_TG_MAX;
    uint32_t *ymw = tg + 2 * wave;   // scan path: this wave's two rows' masks

    Rsrcs R;
    R.XT = make_rsrc(a.XT, (uint32_t)d * WD_XS);
    R.K = make_rsrc(a.keys, tg_lds ? WD_TG_MAX * 4u : 0u);
    R.W = make_rsrc(a.W, a.nb_W);
    R.I = make_rsrc(a.I, a.nb_I);
    R.m = make_rsrc(a.m, a.nb_m);
    R.v = make_rsrc(a.v, a.nb_m);
    R.b = make_rsrc(a.bias, a.nb_b);
    R.bm = make_rsrc(a.bm, a.nb_b);
    R.bv = make_rsrc(a.bv, a.nb_b);
    R.dwp = make_rsrc(a.dwp, MODE == PASS_ONLY ? 0u : a.nb_m);
    R.dbp = make_rsrc(a.dbp, MODE == PASS_ONLY ? 0u : a.nb_b);

    Prefetch pa, pb;
    prefetch<ADAM>(a, R, blockIdx.x, tid, lab, myslot, pa);

    // stage the pass's X tile (transposed and zero-padded past B by the batch
    // prep) with 16-byte copies, its sorted positives, and clear T and G.  The
    // positives are keys (label << 4 | sample), ascending (a label outside
    // [0,L) is the largest key and is never matched).  Chunks of one
    // workgroup come in ascending order, so a cursor that only moves forward
    // finds each chunk's positives.
    {
#pragma unroll
        for (int e = tid; e < d * WD_XS / 16; e += WD_THREADS) {
            const auto q = __builtin_amdgcn_raw_buffer_load_b128(R.XT, 16u * e, 0, 0);
            *reinterpret_cast<uint4 *>(Xs + 16 * e) = make_uint4(q[0], q[1], q[2], q[3]);
        }
        if (tg_lds) {
            tg[tid] = ld32(R.K, 4u * tid);
            tg[tid + WD_THREADS] = ld32(R.K, 4u * (tid + WD_THREADS));
        }
        uint32_t *TG = reinterpret_cast<uint32_t *>(T);
        for (int e = tid; e < (d * WD_NLAB + WD_NB * WD_NLAB) / 2; e += WD_THREADS) TG[e] = 0u;
    }
    __syncthreads();

    // dX accumulators: the 16 samples x NT column tiles of 16 of this wave
    f32x4 acc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};

    float loss_acc = 0.f;
    const float decay = 1.f - a.adam.lr * a.adam.wd;
    const float inv_bc1 = 1.f / a.adam.bc1, inv_bc2 = 1.f / a.adam.bc2;
    const float b1 = a.adam.b1, b2 = a.adam.b2, lr = a.adam.lr, eps = a.adam.eps;
    int pos = 0;              // first sorted key not below the current chunk
    uint32_t head = 0xffffffffu;   // tg[pos] (uniform), or the largest key past the end
    if (tg_lds && nnz > 0) head = __builtin_amdgcn_readfirstlane(tg[0]);
    int32_t c0 = 0, c1 = 0;   // T columns written by this lane in the previous chunk
    const int kk = lab;       // the row within the chunk

    // One chunk: `cur` holds its rows and optimiser state, `nxt` receives the
    // next chunk's.
    auto step = [&](int64_t chunk, const Prefetch &cur, Prefetch &nxt) {
        const int64_t l0 = chunk * WD_NLAB;
        const uint32_t l0u = (uint32_t)l0;   // L < 2^24: label offsets fit in 32 bits

        // stage this wave's rows: indices become clamped byte offsets of X columns
        {
            const uint2 ip = idx_pair(cur.iv, a.idx16);
            const int i0 = min(max((int)ip.x, 0), d - 1), i1 = min(max((int)ip.y, 0), d - 1);
            *reinterpret_cast<int2 *>(Is + 2 * tid) = make_int2(i0 * WD_XS, i1 * WD_XS);
            reinterpret_cast<uint32_t *>(Ws)[tid] = cur.wv;
        }
        prefetch<ADAM>(a, R, chunk + gridDim.x, tid, lab, myslot, nxt);

        // targets of this lane's row as a 16-bit sample mask
        uint32_t yrow = 0;
        if (tg_lds) {
            while ((head >> 4) < l0u) {
                ++pos;
                head = pos < nnz ? __builtin_amdgcn_readfirstlane(tg[pos]) : 0xffffffffu;
            }
            if ((head >> 4) - l0u < (uint32_t)WD_NLAB) {
                for (int e = pos; e < nnz; ++e) {
                    const uint32_t key = tg[e];
                    const uint32_t ll = (key >> 4) - l0u;
                    if (ll >= (uint32_t)WD_NLAB) break;
                    if (ll == (uint32_t)lab) yrow |= 1u << (key & 15u);
                }
            }
            wave_lds_sync();
        } else {
            // each wave scans the whole target list for its two rows
            if (lane < 2) ymw[lane] = 0u;
            wave_lds_sync();
            const uint32_t r0 = l0u + 2u * (uint32_t)wave;
            for (int e = lane; e < nnz; e += 64) {
                const uint32_t ll = (uint32_t)a.tgt_lab[e] - r0;
                const uint32_t b = (uint32_t)(a.tgt_b[e] - a.b0);
                if (ll < 2u && b < (uint32_t)a.B) atomicOr(&ymw[ll], 1u << b);
            }
            wave_lds_sync();
            yrow = ymw[lab & 1];
        }
        int rl = lab;            // the row of the chunk this lane serves
        int kq = qd & 1;         // pair order of this lane's registers
        // opaque per chunk, so the per-slot LDS addresses are formed where
        // they are used instead of being held in registers across chunks
        asm volatile("" : "+v"(rl), "+v"(kq));
        const int64_t l = l0 + rl;
        const bool valid = l < a.L;
        const uint32_t obm = valid && u == 0 ? (uint32_t)l * 4u : a.nb_b;
        float bmcur = 0.f, bvcur = 0.f;
        if constexpr (ADAM) {
            bmcur = ldf(R.bm, obm);
            bvcur = ldf(R.bv, obm);
        }
        const uint32_t odw = valid ? (uint32_t)(l * WD_K + myslot) * 4u : a.nb_m;
        float2 dprev = make_float2(0.f, 0.f);
        float dbprev = 0.f;
        if constexpr (CARRY_IN) {
            dprev = ldf2(R.dwp, odw);
            dbprev = ldf(R.dbp, obm);
        }

        // gather the lane's 8 slots for its 4 samples: registers 2p, 2p+1
        // hold slots 2(p ^ kq), 2(p ^ kq) + 1 of the group, each as the
        // samples' bf16 pairs (4q, 4q+1 | 4q+2, 4q+3)
        const int32_t *Ig = Is + rl * WD_K + 8 * grp;
        const uint4 wq = *reinterpret_cast<const uint4 *>(reinterpret_cast<const uint32_t *>(Ws) +
                                                          rl * (WD_K / 2) + 4 * grp);
        const unsigned char *Xq = Xs + 8 * qd;
        uint2 xv[8];
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            const int2 io = *reinterpret_cast<const int2 *>(Ig + 2 * (p ^ kq));
            xv[2 * p] = *reinterpret_cast<const uint2 *>(Xq + io.x);
            xv[2 * p + 1] = *reinterpret_cast<const uint2 *>(Xq + io.y);
        }
        // the lane's own slots 2 qd, 2 qd + 1: their columns and weight pair
        const int2 co = *reinterpret_cast<const int2 *>(Ig + 2 * qd);
        const int32_t c0n = co.x / WD_XS, c1n = co.y / WD_XS;
        const uint32_t wown = qd == 0 ? wq.x : qd == 1 ? wq.y : qd == 2 ? wq.z : wq.w;
        // forward: the weight pairs in register order
        const uint32_t wp[4] = {kq ? wq.y : wq.x, kq ? wq.x : wq.y, kq ? wq.w : wq.z, kq ? wq.z : wq.w};
        float z[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            const uint2 A = xv[2 * p], Bv = xv[2 * p + 1];
            z[0] = dot2(__builtin_amdgcn_perm(Bv.x, A.x, 0x05040100u), wp[p], z[0]);
            z[1] = dot2(__builtin_amdgcn_perm(Bv.x, A.x, 0x07060302u), wp[p], z[1]);
            z[2] = dot2(__builtin_amdgcn_perm(Bv.y, A.y, 0x05040100u), wp[p], z[2]);
            z[3] = dot2(__builtin_amdgcn_perm(Bv.y, A.y, 0x07060302u), wp[p], z[3]);
        }
        // the eight slot groups (lanes of one half DPP row) add up their scores
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            float t = add_dpp<DPP_ROW_HALF_MIRROR>(z[e], z[e]);
            t = add_dpp<DPP_QUAD_3210>(t, t);
            z[e] = add_dpp<DPP_QUAD_1032>(t, t);
        }
        // BCE and dlogit of (row, sample 4 qd + sj); zero for padded samples
        // and rows past L; the loss is counted once, by the lanes with g < 4
        const int bj = 4 * qd + sj;
        const float zz = (sj == 0 ? z[0] : sj == 1 ? z[1] : sj == 2 ? z[2] : z[3]) + cur.b;
        const bool live = valid && bj < a.B;
        const float y = ((yrow >> bj) & 1u) ? 1.f : 0.f;
        float gj;
        if (a.hinge) {
            // squared hinge with yh = 2y - 1
            const float yh = 2.f * y - 1.f;
            const float hh = fmaxf(1.f - yh * zz, 0.f);
            loss_acc += live && grp < 4 ? hh * hh : 0.f;
            gj = live ? -2.f * a.s * yh * hh : 0.f;
        } else {
            const float ex = __builtin_amdgcn_exp2f(-fabsf(zz) * 1.4426950408889634f);
            const float opx = 1.f + ex;
            const float rr = __builtin_amdgcn_rcpf(opx);
            const float sig = zz >= 0.f ? rr : ex * rr;
            loss_acc += live && grp < 4
                            ? fmaxf(zz, 0.f) - zz * y + __builtin_amdgcn_logf(opx) * 0.6931471805599453f
                            : 0.f;
            gj = live ? a.s * (sig - y) : 0.f;
        }
        // every lane of a quad gets the dlogits of its four samples (lane i of
        // each group of four computed sample 4 qd + i)
        const int gji = __float_as_int(gj);
        const float g[4] = {__int_as_float(__builtin_amdgcn_update_dpp(0, gji, 0x00, 0xf, 0xf, false)),
                            __int_as_float(__builtin_amdgcn_update_dpp(0, gji, 0x55, 0xf, 0xf, false)),
                            __int_as_float(__builtin_amdgcn_update_dpp(0, gji, 0xAA, 0xf, 0xf, false)),
                            __int_as_float(__builtin_amdgcn_update_dpp(0, gji, 0xFF, 0xf, 0xf, false))};
        // dW partials of the lane's slots over its samples, register order
        const uint32_t g01 = pack_bf16(g[0], g[1]), g23 = pack_bf16(g[2], g[3]);
        // a wave whose dlogits are all zero (a hinge loss past its margin
        // everywhere, Sec. 2.2) has zero dW: its products are skipped
        float dw0 = dprev.x, dw1 = dprev.y;
        if (__builtin_amdgcn_ballot_w64((g01 | g23) != 0u) != 0) {
            float pw[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) pw[i] = dot2(xv[i].y, g23, dot2z(xv[i].x, g01));
            // reduce-scatter over the four quads: quads qd and qd ^ 2 sit in
            // the two DPP rows of the row's 32 lanes, quads qd and qd ^ 1 8
            // lanes apart in one DPP row
            float r4[4];
#pragma unroll
            for (int t = 0; t < 4; ++t) r4[t] = cross_rows_add(pw[t], pw[4 + t]);
            dw0 += add_dpp<DPP_ROW_ROR8>(r4[0], r4[2]);
            dw1 += add_dpp<DPP_ROW_ROR8>(r4[1], r4[3]);
        }
        if constexpr (!ADAM) stf2(R.dwp, odw, make_float2(dw0, dw1));
        if constexpr (ADAM) {
            float m0 = cur.m.x, m1 = cur.m.y, v0 = cur.v.x, v1 = cur.v.y;
            const float w0 = __uint_as_float(wown << 16);
            const float w1 = __uint_as_float(wown & 0xffff0000u);
            const float n0 = adam_step(w0, dw0, m0, v0, b1, b2, inv_bc1, inv_bc2, lr, eps, decay);
            const float n1 = adam_step(w1, dw1, m1, v1, b1, b2, inv_bc1, inv_bc2, lr, eps, decay);
            const uint32_t o = (uint32_t)(l * WD_K + myslot);
            stf2(R.m, valid ? 4u * o : a.nb_m, make_float2(m0, m1));
            stf2(R.v, valid ? 4u * o : a.nb_m, make_float2(v0, v1));
            st32(R.W, valid ? 2u * o : a.nb_W, pack_bf16(n0, n1));
        }
        // bias: sum of g over the pass's samples (the quad's four, then the
        // four quads), lane u == 0 updates
        {
            float sg = (g[0] + g[1]) + (g[2] + g[3]);
            sg = cross_rows_add(sg, sg);
            sg = add_dpp<DPP_ROW_ROR8>(sg, sg) + dbprev;
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
        // Every wave has read the previous chunk's G and T fragments before
        // this barrier, so this lane's T entries of that chunk can be cleared;
        // the entries of one row are only ever touched by the wave that owns
        // the row, in program order.
        __syncthreads();
        T[qswz(c0, kk)] = 0;
        T[qswz(c1, kk)] = 0;
        // dX inputs: g and the old weights (a row past L writes zeros at column 0)
        if (grp < 4) G[qswz(bj, kk)] = (uint16_t)(pack_bf16(gj, 0.f) & 0xffffu);
        T[qswz(c0n, kk)] = (uint16_t)(wown & 0xffffu);
        T[qswz(c1n, kk)] = (uint16_t)(wown >> 16);
        c0 = c0n;
        c1 = c1n;
        __syncthreads();
        // dX += G (16 x 16) * T^T (16 x d) on the matrix cores for this wave's
        // column tiles; the next chunk's barrier orders these fragment reads
        // before any rewrite of G or T
        {
            const int col = lane & 15, kq = lane >> 4;
            const s16x4 af = *reinterpret_cast<const s16x4 *>(G + qswz(col, 4 * kq));
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const s16x4 bfr = *reinterpret_cast<const s16x4 *>(T + qswz(16 * (wave + 8 * t) + col, 4 * kq));
                acc[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(af, bfr, acc[t], 0, 0, 0);
            }
        }
    };

    // two chunks per iteration, so the prefetch buffers swap roles instead of
    // being copied (a copy would wait for the loads in flight)
    for (int64_t chunk = blockIdx.x; chunk < a.nchunks; chunk += 2 * (int64_t)gridDim.x) {
        step(chunk, pa, pb);
        if (chunk + gridDim.x >= a.nchunks) break;
        step(chunk + gridDim.x, pb, pa);
    }

    // write this workgroup's dX partial [B][d] (its rows of the pass)
    {
        float *P = a.dx_part + ((size_t)blockIdx.x * a.Btot + a.b0) * d;
        const int col = lane & 15, kq = lane >> 4;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int i = 16 * (wave + 8 * t) + col;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int b = 4 * kq + r;
                if (b < a.B) P[(size_t)b * d + i] = acc[t][r];
            }
        }
    }
    // loss: workgroup tree reduction in the (now unused) T tile
    float *red = reinterpret_cast<float *>(T);
    __syncthreads();
    red[tid] = loss_acc;
    __syncthreads();
    for (int st = WD_THREADS / 2; st > 0; st >>= 1) {
        if (tid < st) red[tid] += red[tid + st];
        __syncthreads();
    }
    if (tid == 0) a.loss_part[blockIdx.x] = red[0];
}

typedef void (*WdKernel)(const WdArgs);
template <int NT>
struct WdModes {
    static constexpr WdKernel k[4] = {k_sweep_wide<NT, PASS_ONLY>, k_sweep_wide<NT, PASS_FIRST>,
                                      k_sweep_wide<NT, PASS_LAST>, k_sweep_wide<NT, PASS_MIDDLE>};
};
template <int... NTs>
WdKernel wd_pick(int nt, int mode, std::integer_sequence<int, NTs...>) {
    WdKernel r = nullptr;
    ((nt == NTs + 1 ? (r = WdModes<NTs + 1>::k[mode], 0) : 0), ...);
    return r;
}
WdKernel wd_kernel(int nt, int mode) { return wd_pick(nt, mode, std::make_integer_sequence<int, WD_NT_MAX>{}); }

size_t sweep_wide_lds(int d) {
    return (size_t)d * WD_XS + (size_t)d * WD_NLAB * 2 + WD_NB * WD_NLAB * 2 + WD_NLAB * WD_K * 4 +
           WD_NLAB * WD_K * 2 + WD_TG_MAX * 4;
}

}  // namespace

bool sweep_wide_eligible(const Layer &ly, int mode) {
    static_assert(WD_NB == WD_PASS_B, "pass width");
    return mode == SWEEP_FUSED && ly.vt == FFSL_BF16 && wide_shape(ly.L, ly.d, ly.k) && ly.k == WD_K &&
           ly.d <= 128 * WD_NT_MAX && sweep_wide_lds(ly.d) <= 160 * 1024;
}

// The batch runs in passes of 16 samples: every pass accumulates its samples'
// dX rows and loss, the first stores its dW / dbias in the carry buffers,
// middle passes add to them, and the last adds its share and applies Adam.
// W, the moments and the bias change only in the last pass, so every pass
// sees the step's old state.
int launch_sweep_wide(const SweepCall &c, const FastBufs &fb, int *grid_out, int *passes_out) {
    const Layer &ly = *c.layer;
    WdArgs a{};
    a.L = ly.L;
    a.d = ly.d;
    a.nnz = c.nnz;
    a.nchunks = (ly.L + WD_NLAB - 1) / WD_NLAB;
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
    a.nb_W = (uint32_t)(ly.L * WD_K * 2);
    a.idx16 = ly.idx16;
    a.nb_I = (uint32_t)(ly.L * WD_K * (ly.idx16 ? 2 : 4));
    a.nb_m = (uint32_t)(ly.L * WD_K * 4);
    a.nb_b = ly.bias ? (uint32_t)(ly.L * 4) : 0u;
    const size_t shm = sweep_wide_lds(ly.d);
    const int grid = (int)std::min<int64_t>(a.nchunks, std::min(ly.max_parts, ly.num_cu));
    const int passes = (c.B + WD_NB - 1) / WD_NB;
    if (ly.ev_start) {
        hipError_t e = hipEventRecord(ly.ev_start, c.stream);
        if (e != hipSuccess) return fail(FFSL_EHIP, "hipEventRecord: %s", hipGetErrorString(e));
    }
    for (int p = 0; p < passes; ++p) {
        const int mode = passes == 1 ? PASS_ONLY : p == 0 ? PASS_FIRST : p == passes - 1 ? PASS_LAST : PASS_MIDDLE;
        a.b0 = p * WD_NB;
        a.B = std::min(WD_NB, c.B - a.b0);
        a.XT = fb.xt + (size_t)p * ly.d * WD_NB;
        a.keys = fb.keys + (size_t)p * WD_TG_MAX;
        a.loss_part = fb.loss_part + (size_t)p * grid;
        const WdKernel kern = wd_kernel(ly.d / 128, mode);
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
        if (e != hipSuccess) return fail(FFSL_EHIP, "hipFuncSetAttribute: %s", hipGetErrorString(e));
        hipLaunchKernelGGL(kern, dim3(grid), dim3(WD_THREADS), shm, c.stream, a);
        int rc = check_launch("sweep_wide");
        if (rc) return rc;
    }
    if (ly.ev_stop) {
        hipError_t e = hipEventRecord(ly.ev_stop, c.stream);
        if (e != hipSuccess) return fail(FFSL_EHIP, "hipEventRecord: %s", hipGetErrorString(e));
    }
    *grid_out = grid;
    *passes_out = passes;
    return FFSL_OK;
}

}  // namespace ffsl
