/*
 * Test infrastructure: a C driver that calls every function of the CPU oracle
 * (oracle/ffsl_oracle.c) on small inputs, including the edge cases the tests
 * pin (NULL optional outputs, labels outside [0,L), NaN and infinite values,
 * ties, exhausted SET rows, rows offset by row0, topk past the selectable
 * labels).  tests/test_oracle_sanitize.py builds it together with the oracle
 * under AddressSanitizer and UndefinedBehaviorSanitizer and runs it: any
 * out-of-bounds access, use after free, leak or undefined operation aborts
 * the run.  It prints one checksum line so the optimiser keeps every call.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

void ffslref_forward(int64_t, int64_t, int64_t, int64_t, const double *, const double *, const int32_t *,
                     const double *, double *);
void ffslref_targets_dense(int64_t, int64_t, const int64_t *, const int32_t *, uint8_t *);
double ffslref_bce(int64_t, const double *, const uint8_t *, double, double *);
double ffslref_sqhinge(int64_t, const double *, const uint8_t *, double, double *);
void ffslref_backward(int64_t, int64_t, int64_t, int64_t, const double *, const double *, const int32_t *,
                      const double *, double *, double *, double *);
void ffslref_adam(int64_t, double *, double *, double *, const double *, int64_t, double, double, double, double,
                  double);
uint16_t ffslref_round_bf16(double);
void ffslref_round_bf16_array(int64_t, const double *, uint16_t *);
void ffslref_philox4x64_10(const uint64_t *, const uint64_t *, uint64_t *);
int64_t ffslref_set_prune_count(int64_t, double);
int64_t ffslref_set_update(int64_t, int64_t, int64_t, int, void *, int32_t *, float *, float *, uint8_t *, double,
                           uint64_t, uint64_t, int, uint64_t);
int64_t ffslref_set_update_threshold(int64_t, int64_t, int64_t, int, void *, int32_t *, float *, float *, uint8_t *,
                                     double, uint64_t, uint64_t, int, uint64_t);
void ffslref_dense_gelu_fwd(int64_t, int64_t, int64_t, const double *, const double *, const double *, double *,
                            double *);
void ffslref_dense_gelu_bwd(int64_t, int64_t, int64_t, const double *, const double *, const double *,
                            const double *, double *, double *, double *);
double ffslref_aux_bce(int64_t, int64_t, int64_t, int64_t, const double *, const double *, const double *,
                       const int64_t *, const int32_t *, double, double *, double *, double *, double *);
void ffslref_topk(int64_t, int64_t, const double *, int64_t, int32_t *, double *);
void ffslref_precision_at_k(int64_t, int64_t, const int32_t *, const int64_t *, const int32_t *, double *);

static uint64_t rs = 0x9E3779B97F4A7C15ull;
static double urand(void)   /* xorshift64*, uniform in [0,1) */
{
    rs ^= rs >> 12;
    rs ^= rs << 25;
    rs ^= rs >> 27;
    return (double)((rs * 0x2545F4914F6CDD1Dull) >> 11) / 9007199254740992.0;
}

static double acc;   /* checksum of finite outputs */
static void sum(const double *x, int64_t n)
{
    for (int64_t i = 0; i < n; ++i)
        if (isfinite(x[i]))
            acc += x[i];
}

/* k distinct columns in [0,d) per row */
static void rows_of_indices(int32_t *I, int64_t L, int64_t k, int64_t d)
{
    for (int64_t l = 0; l < L; ++l)
        for (int64_t j = 0; j < k; ++j) {
            for (;;) {
                int32_t c = (int32_t)(urand() * (double)d);
                int dup = 0;
                for (int64_t q = 0; q < j; ++q)
                    dup |= I[l * k + q] == c;
                if (!dup) {
                    I[l * k + j] = c;
                    break;
                }
            }
        }
}

static void layer(void)
{
    enum { B = 3, d = 9, L = 7, k = 4 };
    double X[B * d], W[L * k], bias[L], z[B * L], g[B * L], dW[L * k], db[L], dX[B * d];
    int32_t I[L * k];
    for (int i = 0; i < B * d; ++i) X[i] = urand() - 0.5;
    for (int i = 0; i < L * k; ++i) W[i] = urand() - 0.5;
    for (int i = 0; i < L; ++i) bias[i] = urand();
    rows_of_indices(I, L, k, d);
    /* labels outside [0,L) and a repeat */
    int64_t off[B + 1] = {0, 3, 3, 6};
    int32_t lab[6] = {2, -1, 2, L, 6, 1 << 30};
    uint8_t y[B * L];
    ffslref_forward(B, d, L, k, X, W, I, bias, z);
    ffslref_forward(B, d, L, k, X, W, I, NULL, z);
    ffslref_targets_dense(B, L, off, lab, y);
    acc += ffslref_bce(B * L, z, y, 1.0 / B, g);
    acc += ffslref_bce(B * L, z, y, 1.0 / B, NULL);
    acc += ffslref_sqhinge(B * L, z, y, 1.0 / B, g);
    acc += ffslref_sqhinge(B * L, z, y, 1.0 / B, NULL);
    /* extreme scores */
    double ze[6] = {0.0, 100.0, -100.0, INFINITY, -INFINITY, NAN}, ge[6];
    uint8_t ye[6] = {0, 1, 0, 1, 0, 1};
    acc += isfinite(ffslref_bce(6, ze, ye, 1.0, ge)) ? 1.0 : 0.0;
    ffslref_bce(B * L, z, y, 1.0 / B, g);
    ffslref_backward(B, d, L, k, X, W, I, g, dW, db, dX);
    ffslref_backward(B, d, L, k, X, W, I, g, dW, NULL, NULL);
    sum(dW, L * k);
    sum(dX, B * d);
    double m[L * k], v[L * k];
    memset(m, 0, sizeof m);
    memset(v, 0, sizeof v);
    ffslref_adam(L * k, W, m, v, dW, 1, 1e-3, 0.9, 0.999, 1e-8, 0.0);
    ffslref_adam(L * k, W, m, v, dW, 2, 1e-3, 0.9, 0.999, 1e-8, 1e-4);
    sum(W, L * k);
}

static void bf16_and_philox(void)
{
    double x[10] = {0.0, -0.0, 1.0, -1.5, 1e-40, -1e-45, 3.4e38, INFINITY, NAN, 1.00390625};
    uint16_t b[10];
    ffslref_round_bf16_array(10, x, b);
    for (int i = 0; i < 10; ++i) acc += b[i];
    acc += ffslref_round_bf16(1e300);
    uint64_t ctr[4] = {1, 2, 3, 4}, key[2] = {5, 6}, out[4];
    ffslref_philox4x64_10(ctr, key, out);
    acc += (double)(out[0] >> 40);
}

static void set_rounds(void)
{
    enum { L = 40, k = 8, d = 24 };
    uint16_t W16[L * k];
    uint32_t W32[L * k];
    int32_t I[L * k];
    float m[L * k], v[L * k];
    uint8_t mask[L * k];
    for (int wbits = 16; wbits <= 32; wbits += 16) {
        for (int round = 0; round < 3; ++round) {
            rows_of_indices(I, L, k, d);
            for (int i = 0; i < L * k; ++i) {
                float f = (float)((int)(urand() * 7.0) - 3) * 0.125f;   /* ties, +-0 */
                if (i % 17 == 0) f = NAN;
                uint32_t u;
                memcpy(&u, &f, 4);
                W32[i] = u;
                W16[i] = (uint16_t)(u >> 16);
                m[i] = (float)urand();
                v[i] = (float)urand();
            }
            void *Wp = wbits == 16 ? (void *)W16 : (void *)W32;
            acc += (double)ffslref_set_update(L, d, k, wbits, Wp, I, m, v, mask, 0.3, 7, round, round == 1, 100);
            acc += (double)ffslref_set_update(L, d, k, wbits, Wp, I, NULL, NULL, NULL, 0.25, 7, round, 0, 0);
            acc += (double)ffslref_set_update_threshold(L, d, k, wbits, Wp, I, m, v, mask, 0.2, 9, round, 0, 3);
            acc += (double)ffslref_set_update_threshold(L, d, k, wbits, Wp, I, m, v, mask, INFINITY, 9, round, 0,
                                                        3);
            /* every column taken: the rows run out of draws */
            acc += (double)ffslref_set_update_threshold(L, k, k, wbits, Wp, I, m, v, mask, 1e9, 1, round, 0, 0);
        }
    }
    acc += (double)ffslref_set_update(L, d, k, 7, W16, I, m, v, mask, 0.3, 7, 0, 0, 0);   /* bad width: -1 */
    acc += (double)ffslref_set_update(L, k + 1, k, 16, W16, I, m, v, mask, 0.5, 7, 0, 0, 0); /* n > d-k: -1 */
    acc += (double)ffslref_set_prune_count(k, 0.3);
}

static void dense_and_inference(void)
{
    enum { B = 4, din = 5, dout = 6, C = 3, L = 11, K = 4 };
    double X[B * din], W1[din * dout], c[dout], A[B * dout], H[B * dout], dH[B * dout];
    double dW1[din * dout], dc[dout], dX[B * din];
    for (int i = 0; i < B * din; ++i) X[i] = urand() - 0.5;
    for (int i = 0; i < din * dout; ++i) W1[i] = urand() - 0.5;
    for (int i = 0; i < dout; ++i) c[i] = urand();
    for (int i = 0; i < B * dout; ++i) dH[i] = urand() - 0.5;
    ffslref_dense_gelu_fwd(B, din, dout, X, W1, c, A, H);
    ffslref_dense_gelu_fwd(B, din, dout, X, W1, NULL, NULL, H);
    ffslref_dense_gelu_bwd(B, din, dout, X, W1, A, dH, dW1, dc, dX);
    ffslref_dense_gelu_bwd(B, din, dout, X, W1, A, dH, dW1, NULL, NULL);
    sum(dW1, din * dout);
    double Wa[din * C], ca[C], Za[B * C], dWa[din * C], dca[C], dXa[B * din];
    for (int i = 0; i < din * C; ++i) Wa[i] = urand() - 0.5;
    for (int i = 0; i < C; ++i) ca[i] = urand();
    int64_t off[B + 1] = {0, 2, 2, 5, 6};
    int32_t lab[6] = {1, L, -3, 4, 10, 11};
    acc += ffslref_aux_bce(B, din, C, L, X, Wa, ca, off, lab, 0.25, Za, dWa, dca, dXa);
    acc += ffslref_aux_bce(B, din, C, L, X, Wa, NULL, off, lab, 0.25, Za, dWa, NULL, dXa);
    sum(dXa, B * din);
    /* scores with ties, NaN and -inf; K above the selectable count in row 3 */
    double z[B * L];
    for (int i = 0; i < B * L; ++i) z[i] = (double)((int)(urand() * 4.0));
    z[1] = NAN;
    z[5] = -INFINITY;
    for (int l = 0; l < L; ++l) z[3 * L + l] = l < 2 ? 1.0 : NAN;
    int32_t top[B * K];
    double tz[B * K], p[K];
    ffslref_topk(B, L, z, K, top, tz);
    ffslref_precision_at_k(B, K, top, off, lab, p);
    sum(p, K);
    for (int i = 0; i < B * K; ++i) acc += top[i];
}

int main(void)
{
    for (int rep = 0; rep < 3; ++rep) {
        layer();
        bf16_and_philox();
        set_rounds();
        dense_and_inference();
    }
    printf("oracle sanitize driver ok %.6e\n", acc);
    return 0;
}
