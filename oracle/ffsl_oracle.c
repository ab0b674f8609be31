/*
 * ffsl_oracle.c -- plain, slow CPU oracle for the fixed fan-in sparse
 * classification layer of "Navigating Extremes: Dynamic Sparsity in Large
 * Output Spaces" (Ullah, Schultheis, Lasby, Ioannou, Babbar; NeurIPS 2024).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may call, link or
 * load this file: only the test-suite, the smoke check and the CPU-baseline
 * leg of the benchmark use it.  It shares no code, header, table or constant
 * generator with the HIP library; it is written directly from the paper and
 * from the textbook definitions named at each function.
 *
 * Conventions
 *   - Every floating-point value is held and accumulated in double.  Callers
 *     widen fp32/bf16 inputs to double exactly before calling.
 *   - Reductions run in ascending index order, exactly as the sums are
 *     written below; there is no blocking, fusion or reordering.
 *   - Row-major layouts: X[b*d+i], W[l*k+j], I[l*k+j], z[b*L+l].
 *
 * Parity status of each function (what pins it in tests/test_oracle_*.py):
 *   forward / backward   dense masked matmul + autograd + finite differences
 *   bce                  closed form + torch BCE-with-logits
 *   sqhinge              hand-computed values, finite differences, symmetry
 *   adam                 torch.optim.Adam / AdamW
 *   round_bf16           torch float32 -> bfloat16 conversion
 *   philox4x64_10        numpy.random.Philox (a library implementation)
 *   set_update           stable argsort, brute force, invariants; the draw
 *                        stream itself is our own contract (see set_update)
 *   set_update_threshold a plain-Python restatement; reduces to the fraction
 *                        mode when tau selects exactly n slots; extremes
 *   topk, precision_at_k numpy lexsort on tied / NaN / -inf scores, a
 *                        set-based P@k count, a hand-computed case
 *   gelu / dense / aux   closed forms + torch autograd
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define EXPORT __attribute__((visibility("default")))

/* ------------------------------------------------------------------------ */
/* Gathered forward (Sec. 2.1 one-vs-all classifier; Sec. 2.2 fixed fan-in,
 * ELLPACK storage without padding): every label row l holds exactly k weights
 * W[l,j] at input columns I[l,j], so its score for sample b is
 *     z[b,l] = bias[l] + sum_{j<k} W[l,j] * X[b, I[l,j]].                    */
EXPORT void ffslref_forward(int64_t B, int64_t d, int64_t L, int64_t k,
                            const double *X, const double *W, const int32_t *I,
                            const double *bias, double *z)
{
    (void)d;
    for (int64_t b = 0; b < B; ++b) {
        for (int64_t l = 0; l < L; ++l) {
            double acc = 0.0;
            for (int64_t j = 0; j < k; ++j)
                acc += W[l * k + j] * X[b * d + I[l * k + j]];
            z[b * L + l] = (bias ? bias[l] : 0.0) + acc;
        }
    }
}

/* Multi-hot targets (Sec. 2.1: P_b is the set of relevant labels of sample b),
 * given in CSR form: the labels of sample b are lab[off[b] .. off[b+1]).
 * y[b,l] = 1 iff l is in P_b; repeated labels count once.                    */
EXPORT void ffslref_targets_dense(int64_t B, int64_t L, const int64_t *off,
                                  const int32_t *lab, uint8_t *y)
{
    memset(y, 0, (size_t)(B * L));
    for (int64_t b = 0; b < B; ++b)
        for (int64_t e = off[b]; e < off[b + 1]; ++e)
            if (lab[e] >= 0 && lab[e] < L)   /* labels outside [0,L) are ignored */
                y[b * L + lab[e]] = 1;
}

/* Binary cross-entropy with logits (the loss used for LF-AmazonTitles-131K,
 * Appendix "Hyperparameter Settings"), summed over labels and samples and
 * scaled by s (s = 1/B averages over the batch):
 *     loss = s * sum_n [ max(z,0) - z*y + log(1 + exp(-|z|)) ]
 *     g_n  = d loss / d z_n = s * (sigmoid(z_n) - y_n).
 * The max/log1p form is the textbook overflow-free rewriting of
 * -y log sigmoid(z) - (1-y) log(1 - sigmoid(z)).                            */
EXPORT double ffslref_bce(int64_t n, const double *z, const uint8_t *y, double s,
                          double *g)
{
    double loss = 0.0;
    for (int64_t t = 0; t < n; ++t) {
        double zz = z[t];
        double yy = y[t] ? 1.0 : 0.0;
        loss += (zz > 0.0 ? zz : 0.0) - zz * yy + log1p(exp(-fabs(zz)));
        if (g) {
            double sig = 1.0 / (1.0 + exp(-zz));
            g[t] = s * (sig - yy);
        }
    }
    return s * loss;
}

/* Squared hinge loss (the loss of every dataset but LF-AmazonTitles-131K,
 * Appendix "Hyperparameter Settings"; the paper names it without a formula,
 * so we take the textbook one), with signed targets yh = 2y - 1, summed and
 * scaled by s:
 *     loss = s * sum_n max(0, 1 - yh_n z_n)^2
 *     g_n  = d loss / d z_n = -2 s yh_n max(0, 1 - yh_n z_n).
 * g_n is exactly 0 wherever yh_n z_n >= 1: the activation sparsity that Sec.
 * 2.2 counts on for the backward pass.                                      */
EXPORT double ffslref_sqhinge(int64_t n, const double *z, const uint8_t *y, double s,
                              double *g)
{
    double loss = 0.0;
    for (int64_t t = 0; t < n; ++t) {
        double yh = y[t] ? 1.0 : -1.0;
        double h = 1.0 - yh * z[t];
        if (h < 0.0) h = 0.0;
        loss += h * h;
        if (g) g[t] = -2.0 * s * yh * h;
    }
    return s * loss;
}

/* Both backward products of the sparse layer (Sec. 2.2: the weight gradient
 * needs the transposed product), for upstream gradient g[b,l] = dloss/dz:
 *     dW[l,j]  = sum_b g[b,l] * X[b, I[l,j]]
 *     dbias[l] = sum_b g[b,l]
 *     dX[b,i]  = sum_l sum_j [I[l,j] == i] * g[b,l] * W[l,j].
 * dbias and dX are optional (NULL skips them).                               */
EXPORT void ffslref_backward(int64_t B, int64_t d, int64_t L, int64_t k,
                             const double *X, const double *W, const int32_t *I,
                             const double *g, double *dW, double *dbias,
                             double *dX)
{
    for (int64_t l = 0; l < L; ++l) {
        for (int64_t j = 0; j < k; ++j) {
            double acc = 0.0;
            for (int64_t b = 0; b < B; ++b)
                acc += g[b * L + l] * X[b * d + I[l * k + j]];
            dW[l * k + j] = acc;
        }
        if (dbias) {
            double acc = 0.0;
            for (int64_t b = 0; b < B; ++b)
                acc += g[b * L + l];
            dbias[l] = acc;
        }
    }
    if (dX) {
        for (int64_t b = 0; b < B; ++b) {
            for (int64_t i = 0; i < d; ++i)
                dX[b * d + i] = 0.0;
            for (int64_t l = 0; l < L; ++l)
                for (int64_t j = 0; j < k; ++j)
                    dX[b * d + I[l * k + j]] += g[b * L + l] * W[l * k + j];
        }
    }
}

/* Adam (Kingma & Ba, 2015, Algorithm 1) with optional decoupled weight decay
 * (AdamW, Loshchilov & Hutter, 2019), the optimizer of the classifier in
 * Appendix "Hyperparameter Settings".  t is the step number after this
 * update (1 for the first step).  For each element:
 *     p <- p * (1 - lr*wd)                       (only if wd != 0)
 *     m <- b1*m + (1-b1)*grad
 *     v <- b2*v + (1-b2)*grad^2
 *     p <- p - lr * (m / (1-b1^t)) / (sqrt(v / (1-b2^t)) + eps).            */
EXPORT void ffslref_adam(int64_t n, double *p, double *m, double *v,
                         const double *grad, int64_t t, double lr, double b1,
                         double b2, double eps, double wd)
{
    double c1 = 1.0 - pow(b1, (double)t);
    double c2 = 1.0 - pow(b2, (double)t);
    for (int64_t e = 0; e < n; ++e) {
        if (wd != 0.0)
            p[e] = p[e] * (1.0 - lr * wd);
        m[e] = b1 * m[e] + (1.0 - b1) * grad[e];
        v[e] = b2 * v[e] + (1.0 - b2) * grad[e] * grad[e];
        double mhat = m[e] / c1;
        double vhat = v[e] / c2;
        p[e] = p[e] - lr * mhat / (sqrt(vhat) + eps);
    }
}

/* Round a double to the nearest bfloat16 value (8 significant bits, the
 * exponent range of fp32), ties to even.  Returns the bf16 bit pattern.
 * Written from the definition: scale the significand to [128,256), round to
 * an integer with ties-to-even, rescale; below 2^-126 the quantum is fixed
 * at 2^-133 (subnormals).  Used to model a weight that is stored in bf16.    */
static uint16_t bits_from_float(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    return (uint16_t)(u >> 16);
}

EXPORT uint16_t ffslref_round_bf16(double x)
{
    if (isnan(x))
        return 0x7fc0;
    double ax = fabs(x);
    double r;
    if (ax == 0.0) {
        r = 0.0;
    } else if (ax < ldexp(1.0, -126)) {
        r = nearbyint(ldexp(ax, 133));
        r = ldexp(r, -133);
    } else {
        int e;
        double mant = frexp(ax, &e); /* ax = mant * 2^e, mant in [0.5,1) */
        double q = nearbyint(ldexp(mant, 8));
        r = ldexp(q, e - 8);
    }
    /* largest finite bf16 is (2 - 2^-7) * 2^127; anything that rounds above
     * it overflows to infinity */
    float f;
    if (r > ldexp(2.0 - ldexp(1.0, -7), 127))
        f = INFINITY;
    else
        f = (float)r; /* exact: r has at most 8 significant bits */
    if (x < 0 || (x == 0 && signbit(x)))
        f = -f;
    return bits_from_float(f);
}

EXPORT void ffslref_round_bf16_array(int64_t n, const double *x, uint16_t *out)
{
    for (int64_t e = 0; e < n; ++e)
        out[e] = ffslref_round_bf16(x[e]);
}

/* ------------------------------------------------------------------------ */
/* Philox4x64-10: the counter-based generator of Salmon, Moraes, Dror and
 * Shaw, "Parallel Random Numbers: As Easy as 1, 2, 3" (SC'11).  Each of the
 * ten rounds multiplies two counter words by the Philox multipliers, keeping
 * the 128-bit products' high and low halves, and mixes them with the other
 * two words and the round key:
 *     (hi0,lo0) = M0*c0,  (hi1,lo1) = M1*c2
 *     c <- (hi1 ^ c1 ^ k0,  lo1,  hi0 ^ c3 ^ k1,  lo0)
 * and the key is advanced by the Weyl increments between rounds.  The
 * multipliers and increments are the ones the SC'11 paper gives for 4x64.   */
#define PHILOX_M0 0xD2E7470EE14C6C93ULL
#define PHILOX_M1 0xCA5A826395121157ULL
#define PHILOX_W0 0x9E3779B97F4A7C15ULL /* golden ratio */
#define PHILOX_W1 0xBB67AE8584CAA73BULL /* sqrt(3) - 1 */

EXPORT void ffslref_philox4x64_10(const uint64_t ctr[4], const uint64_t key[2],
                                  uint64_t out[4])
{
    uint64_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint64_t k0 = key[0], k1 = key[1];
    for (int r = 0; r < 10; ++r) {
        if (r > 0) {
            k0 += PHILOX_W0;
            k1 += PHILOX_W1;
        }
        unsigned __int128 p0 = (unsigned __int128)PHILOX_M0 * c0;
        unsigned __int128 p1 = (unsigned __int128)PHILOX_M1 * c2;
        uint64_t hi0 = (uint64_t)(p0 >> 64), lo0 = (uint64_t)p0;
        uint64_t hi1 = (uint64_t)(p1 >> 64), lo1 = (uint64_t)p1;
        uint64_t n0 = hi1 ^ c1 ^ k0;
        uint64_t n2 = hi0 ^ c3 ^ k1;
        c0 = n0;
        c1 = lo1;
        c2 = n2;
        c3 = lo0;
    }
    out[0] = c0;
    out[1] = c1;
    out[2] = c2;
    out[3] = c3;
}

/* ------------------------------------------------------------------------ */
/* SET prune-and-regrow (Sec. 2.1: every Delta-T steps a fraction of the
 * active weights is pruned and as many inactive weights are regrown; the
 * pruning criterion is magnitude, regrowth is random, Mocanu et al. 2018;
 * Appendix "Hyperparameter Settings": random growth with zero
 * initialisation).  Applied to each label row independently so that the
 * fan-in stays exactly k (Sec. 2.2).
 *
 * Readings where the paper is silent (each listed in the design notes):
 *   n      = floor(frac*k) weights per row (computed as floor(frac*k + 1e-9)).
 *   order  = key (|W| bit pattern, slot): |W| is the stored value's bit
 *            pattern with the sign cleared (bf16: & 0x7fff, fp32:
 *            & 0x7fffffff), so -0 ties +0 and NaN ranks above +inf; equal
 *            magnitudes prune the smaller slot first.  The n smallest keys
 *            are pruned; P lists their slots in ascending slot order.
 *   inactive = every column not held by the row before pruning, unless
 *            allow_regrow_pruned is set, in which case the just-pruned
 *            columns are eligible again.
 *   draws  = attempt a = 0,1,2,... reads 64-bit word (a mod 4) of
 *            Philox4x64-10(counter = (l, set_round, a/4, 0),
 *                          key = (seed, 0x5345545F52454752 "SET_REGR")),
 *            maps it to a column c = floor(word * d / 2^64), and accepts c
 *            if it is inactive and not yet accepted in this row.  The
 *            accepted columns fill the slots of P in ascending slot order.
 *   cap    = after 64*k + 4096 attempts without n acceptances the row is
 *            left unchanged and counted as exhausted.
 *   zero init = a regrown slot gets W = +0 (bits 0), m = v = 0, mask = 1.
 * The survivors' bits are untouched and the row is not re-sorted.
 *
 * The arrays hold rows row0 .. row0+L-1 of the layer (row0 = 0 for the
 * whole layer); the draw counter uses the layer's row number row0 + l.
 * W is given as bit patterns: wbits = 16 (bf16, uint16_t*) or 32 (fp32,
 * uint32_t*).  m, v, mask may be NULL.  Returns the number of exhausted rows,
 * or -1 for invalid arguments (n > d - k while the pruned columns are not
 * eligible leaves fewer than n inactive columns).                            */
#define SET_KEY_HI 0x5345545F52454752ULL

EXPORT int64_t ffslref_set_prune_count(int64_t k, double frac)
{
    return (int64_t)floor(frac * (double)k + 1e-9);
}

/* The magnitude of stored weight j of row l as a real number. */
static double set_magnitude(int wbits, const void *Wbits, int64_t o)
{
    if (wbits == 16) {
        const uint32_t u = (uint32_t)(((const uint16_t *)Wbits)[o] & 0x7fffu) << 16;
        float f;
        memcpy(&f, &u, 4);
        return (double)f;
    }
    const uint32_t u = ((const uint32_t *)Wbits)[o] & 0x7fffffffu;
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
}

/* SET over rows, in one of two prune modes (Sec. 2.1; the appendix table of
 * DST settings lists both):
 *   fraction   the n = floor(frac*k) smallest keys (|W| bits, slot) of every row
 *   threshold  the slots of a row with |W| < tau (NaN is never below), so n
 *              varies by row
 * then the same regrowth for the n pruned slots of each row. */
static int64_t set_update_rows(int64_t L, int64_t d, int64_t k, int wbits, void *Wbits,
                               int32_t *I, float *m, float *v, uint8_t *mask, int threshold,
                               double frac, double tau, uint64_t seed, uint64_t set_round,
                               int allow_regrow_pruned, uint64_t row0)
{
    const int64_t nf = ffslref_set_prune_count(k, frac);
    if (wbits != 16 && wbits != 32)
        return -1;
    if (!threshold && (nf < 0 || nf > k || (!allow_regrow_pruned && nf > d - k)))
        return -1;
    if (threshold && !(tau >= 0.0))
        return -1;
    if (mask)
        memset(mask, 0, (size_t)(L * k));
    if (!threshold && nf == 0)
        return 0;

    uint64_t *keys = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)k);
    int64_t *pruned = (int64_t *)malloc(sizeof(int64_t) * (size_t)k);
    int32_t *accepted = (int32_t *)malloc(sizeof(int32_t) * (size_t)k);
    uint8_t *taken = (uint8_t *)malloc((size_t)k);
    int64_t exhausted = 0;
    const int64_t cap = 64 * k + 4096;

    for (int64_t l = 0; l < L; ++l) {
        memset(taken, 0, (size_t)k);
        int64_t n = 0;
        if (threshold) {
            for (int64_t j = 0; j < k; ++j)
                if (set_magnitude(wbits, Wbits, l * k + j) < tau) {
                    taken[j] = 1;
                    ++n;
                }
        } else {
            /* keys of the row */
            for (int64_t j = 0; j < k; ++j) {
                uint64_t mag;
                if (wbits == 16)
                    mag = ((uint16_t *)Wbits)[l * k + j] & 0x7fffu;
                else
                    mag = ((uint32_t *)Wbits)[l * k + j] & 0x7fffffffu;
                keys[j] = mag;
            }
            /* select the n smallest (mag, slot) by repeated minimum search */
            n = nf;
            for (int64_t s = 0; s < n; ++s) {
                int64_t best = -1;
                for (int64_t j = 0; j < k; ++j) {
                    if (taken[j])
                        continue;
                    if (best < 0 || keys[j] < keys[best])
                        best = j; /* strict <: the smaller slot wins ties */
                }
                taken[best] = 1;
            }
        }
        if (n == 0)
            continue;
        int64_t np = 0;
        for (int64_t j = 0; j < k; ++j)
            if (taken[j])
                pruned[np++] = j; /* ascending slot order */

        /* draw n new columns */
        int64_t got = 0;
        for (int64_t a = 0; a < cap && got < n; ++a) {
            uint64_t ctr[4] = {row0 + (uint64_t)l, set_round, (uint64_t)(a / 4), 0};
            uint64_t key[2] = {seed, SET_KEY_HI};
            uint64_t out[4];
            ffslref_philox4x64_10(ctr, key, out);
            uint64_t word = out[a % 4];
            int32_t c = (int32_t)(((unsigned __int128)word * (uint64_t)d) >> 64);
            int ok = 1;
            for (int64_t j = 0; j < k && ok; ++j) {
                if (I[l * k + j] != c)
                    continue;
                /* c is held by slot j before pruning */
                if (!(allow_regrow_pruned && taken[j]))
                    ok = 0;
            }
            for (int64_t q = 0; q < got && ok; ++q)
                if (accepted[q] == c)
                    ok = 0;
            if (ok)
                accepted[got++] = c;
        }
        if (got < n) {
            ++exhausted;
            continue;
        }
        for (int64_t q = 0; q < n; ++q) {
            int64_t p = pruned[q];
            I[l * k + p] = accepted[q];
            if (wbits == 16)
                ((uint16_t *)Wbits)[l * k + p] = 0;
            else
                ((uint32_t *)Wbits)[l * k + p] = 0;
            if (m)
                m[l * k + p] = 0.0f;
            if (v)
                v[l * k + p] = 0.0f;
            if (mask)
                mask[l * k + p] = 1;
        }
    }
    free(keys);
    free(pruned);
    free(accepted);
    free(taken);
    return exhausted;
}

EXPORT int64_t ffslref_set_update(int64_t L, int64_t d, int64_t k, int wbits,
                                  void *Wbits, int32_t *I, float *m, float *v,
                                  uint8_t *mask, double frac, uint64_t seed,
                                  uint64_t set_round, int allow_regrow_pruned,
                                  uint64_t row0)
{
    return set_update_rows(L, d, k, wbits, Wbits, I, m, v, mask, 0, frac, 0.0, seed, set_round,
                           allow_regrow_pruned, row0);
}

/* SET in threshold mode: every slot with |W| < tau is pruned and as many
 * columns are regrown in its row (the appendix's "rewire threshold"). */
EXPORT int64_t ffslref_set_update_threshold(int64_t L, int64_t d, int64_t k, int wbits,
                                            void *Wbits, int32_t *I, float *m, float *v,
                                            uint8_t *mask, double tau, uint64_t seed,
                                            uint64_t set_round, int allow_regrow_pruned,
                                            uint64_t row0)
{
    return set_update_rows(L, d, k, wbits, Wbits, I, m, v, mask, 1, 0.0, tau, seed, set_round,
                           allow_regrow_pruned, row0);
}

/* ------------------------------------------------------------------------ */
/* Dense parts of the architectures in Fig. 1 (left).
 *
 * Intermediate layer (Sec. 1 and Sec. 2.3: a dense layer wider than the
 * embedding, placed before the sparse classifier; the activation is not
 * named in the paper, GELU is our reading):
 *     A[b,o] = c[o] + sum_i X[b,i] * W1[i,o]        (W1 is [din, dout])
 *     H[b,o] = GELU(A[b,o]) = A * Phi(A),  Phi(a) = (1 + erf(a/sqrt 2)) / 2.
 * Backward for upstream dH:
 *     dA[b,o]  = dH[b,o] * (Phi(A) + A * phi(A)),   phi(a) = exp(-a^2/2)/sqrt(2 pi)
 *     dW1[i,o] = sum_b X[b,i] * dA[b,o]
 *     dc[o]    = sum_b dA[b,o]
 *     dX[b,i]  = sum_o dA[b,o] * W1[i,o].                                    */
static double gelu_cdf(double a) { return 0.5 * (1.0 + erf(a / sqrt(2.0))); }
static double gelu_pdf(double a) { return exp(-0.5 * a * a) / sqrt(2.0 * M_PI); }

EXPORT void ffslref_dense_gelu_fwd(int64_t B, int64_t din, int64_t dout,
                                   const double *X, const double *W1,
                                   const double *c, double *A, double *H)
{
    for (int64_t b = 0; b < B; ++b)
        for (int64_t o = 0; o < dout; ++o) {
            double acc = 0.0;
            for (int64_t i = 0; i < din; ++i)
                acc += X[b * din + i] * W1[i * dout + o];
            double a = (c ? c[o] : 0.0) + acc;
            if (A)
                A[b * dout + o] = a;
            H[b * dout + o] = a * gelu_cdf(a);
        }
}

EXPORT void ffslref_dense_gelu_bwd(int64_t B, int64_t din, int64_t dout,
                                   const double *X, const double *W1,
                                   const double *A, const double *dH,
                                   double *dW1, double *dc, double *dX)
{
    double *dA = (double *)malloc(sizeof(double) * (size_t)(B * dout));
    for (int64_t b = 0; b < B; ++b)
        for (int64_t o = 0; o < dout; ++o) {
            double a = A[b * dout + o];
            dA[b * dout + o] = dH[b * dout + o] * (gelu_cdf(a) + a * gelu_pdf(a));
        }
    for (int64_t i = 0; i < din; ++i)
        for (int64_t o = 0; o < dout; ++o) {
            double acc = 0.0;
            for (int64_t b = 0; b < B; ++b)
                acc += X[b * din + i] * dA[b * dout + o];
            dW1[i * dout + o] = acc;
        }
    if (dc)
        for (int64_t o = 0; o < dout; ++o) {
            double acc = 0.0;
            for (int64_t b = 0; b < B; ++b)
                acc += dA[b * dout + o];
            dc[o] = acc;
        }
    if (dX)
        for (int64_t b = 0; b < B; ++b)
            for (int64_t i = 0; i < din; ++i) {
                double acc = 0.0;
                for (int64_t o = 0; o < dout; ++o)
                    acc += dA[b * dout + o] * W1[i * dout + o];
                dX[b * din + i] = acc;
            }
    free(dA);
}

/* Auxiliary meta-classifier (Sec. 2.3: a dense classifier over clusters of
 * labels whose loss is added to the main loss; Appendix on random clusters:
 * a random label-to-cluster assignment works as well as k-means, so the
 * fixed map cluster(l) = l mod C is used).  The cluster targets are the
 * multi-hot set of clusters that hold at least one positive label:
 *     Za[b,c]  = ca[c] + sum_i X[b,i] * Wa[i,c]          (Wa is [d, C])
 *     ya[b,c]  = 1 iff some l in P_b has l mod C == c
 *     loss_a   = BCE-with-logits(Za, ya) summed, times s
 * A label outside [0, L) is not a label of the layer and has no cluster: it
 * is ignored, exactly as the sparse head's targets ignore it.
 *     dZa      = s * (sigmoid(Za) - ya)
 *     dWa[i,c] = sum_b X[b,i] dZa[b,c];  dca[c] = sum_b dZa[b,c]
 *     dXa[b,i] = sum_c dZa[b,c] Wa[i,c].
 * Returns loss_a.  ca, dca may be NULL.                                      */
EXPORT double ffslref_aux_bce(int64_t B, int64_t d, int64_t C, int64_t L, const double *X,
                              const double *Wa, const double *ca,
                              const int64_t *off, const int32_t *lab, double s,
                              double *Za, double *dWa, double *dca, double *dXa)
{
    uint8_t *ya = (uint8_t *)calloc((size_t)(B * C), 1);
    double *dZ = (double *)malloc(sizeof(double) * (size_t)(B * C));
    for (int64_t b = 0; b < B; ++b)
        for (int64_t e = off[b]; e < off[b + 1]; ++e)
            if (lab[e] >= 0 && lab[e] < L)   /* labels outside [0,L) are ignored */
                ya[b * C + (lab[e] % C)] = 1;
    for (int64_t b = 0; b < B; ++b)
        for (int64_t c = 0; c < C; ++c) {
            double acc = 0.0;
            for (int64_t i = 0; i < d; ++i)
                acc += X[b * d + i] * Wa[i * C + c];
            Za[b * C + c] = (ca ? ca[c] : 0.0) + acc;
        }
    double loss = ffslref_bce(B * C, Za, ya, s, dZ);
    for (int64_t i = 0; i < d; ++i)
        for (int64_t c = 0; c < C; ++c) {
            double acc = 0.0;
            for (int64_t b = 0; b < B; ++b)
                acc += X[b * d + i] * dZ[b * C + c];
            dWa[i * C + c] = acc;
        }
    if (dca)
        for (int64_t c = 0; c < C; ++c) {
            double acc = 0.0;
            for (int64_t b = 0; b < B; ++b)
                acc += dZ[b * C + c];
            dca[c] = acc;
        }
    for (int64_t b = 0; b < B; ++b)
        for (int64_t i = 0; i < d; ++i) {
            double acc = 0.0;
            for (int64_t c = 0; c < C; ++c)
                acc += dZ[b * C + c] * Wa[i * C + c];
            dXa[b * d + i] = acc;
        }
    free(ya);
    free(dZ);
    return loss;
}

/* ------------------------------------------------------------------------
 * Inference: the top-k labels of each sample and Precision@k (appendix on
 * evaluation metrics: P@k of a sample is the fraction of its k best-scored
 * labels that are relevant).
 *
 * Order: descending score, equal scores by ascending label.  Labels whose
 * score is NaN are never selected; when fewer than K labels can be
 * selected the remaining entries are label -1 with score -inf.
 * Plain selection: the j-th entry is the best label that comes after the
 * (j-1)-th in this order, found by one pass over the row.               */
EXPORT void ffslref_topk(int64_t B, int64_t L, const double *z, int64_t K,
                         int32_t *top_lab, double *top_z)
{
    for (int64_t b = 0; b < B; ++b) {
        const double *zr = z + b * L;
        int64_t prev = -1;
        double prev_z = 0.0;
        for (int64_t j = 0; j < K; ++j) {
            int64_t best = -1;
            double best_z = 0.0;
            for (int64_t l = 0; l < L; ++l) {
                const double v = zr[l];
                if (v != v)
                    continue;
                /* only labels after the previous pick in the order */
                if (prev >= 0 && !(v < prev_z || (v == prev_z && l > prev)))
                    continue;
                if (best < 0 || v > best_z || (v == best_z && l < best)) {
                    best = l;
                    best_z = v;
                }
            }
            top_lab[b * K + j] = (int32_t)best;
            top_z[b * K + j] = best < 0 ? -INFINITY : best_z;
            if (best < 0) {
                /* nothing left: the rest of the row stays empty */
                for (int64_t r = j + 1; r < K; ++r) {
                    top_lab[b * K + r] = -1;
                    top_z[b * K + r] = -INFINITY;
                }
                break;
            }
            prev = best;
            prev_z = best_z;
        }
    }
}

/* Precision@k for k = 1..K, averaged over the B samples:
 *     out[k-1] = (1/B) sum_b (1/k) sum_{j<k} y[b, top_lab[b,j]]
 * y[b,l] = 1 iff l is among the labels lab[off[b] .. off[b+1]) (repeats
 * count once); an empty entry (label -1) is never relevant.            */
EXPORT void ffslref_precision_at_k(int64_t B, int64_t K, const int32_t *top_lab,
                                   const int64_t *off, const int32_t *lab, double *out)
{
    for (int64_t k = 0; k < K; ++k)
        out[k] = 0.0;
    for (int64_t b = 0; b < B; ++b) {
        int64_t hits = 0;
        for (int64_t j = 0; j < K; ++j) {
            const int32_t t = top_lab[b * K + j];
            int rel = 0;
            for (int64_t e = off[b]; e < off[b + 1] && t >= 0; ++e)
                if (lab[e] == t) {
                    rel = 1;
                    break;
                }
            hits += rel;
            out[j] += (double)hits / (double)(j + 1);
        }
    }
    for (int64_t k = 0; k < K; ++k)
        out[k] /= (double)B;
}
