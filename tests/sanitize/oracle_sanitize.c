/*
 * Runs every entry point of oracle/oracle.c on small random patterns (empty
 * rows, repeated entries, N = 1, feature sizes 1..8) and on malformed ones,
 * built with AddressSanitizer and UndefinedBehaviorSanitizer by
 * tests/test_sanitize_oracle.py: any out-of-bounds access, leak, overflow or
 * other undefined behaviour in the oracle aborts the run.  The forward is
 * also compared with a dense masked softmax computed here, so the run checks
 * results as well as memory.  Prints "ok" and returns 0 on success.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int oracle_check_csr(int32_t N, const int32_t *row_ptr, const int32_t *col_idx);
int oracle_3s_f64d(int32_t N, const int32_t *row_ptr, const int32_t *col_idx, int32_t d,
                   const double *Q, const double *K, const double *V, double scale,
                   double *O, double *lse, double *P, int32_t nthreads);
int oracle_3s_f64(int32_t N, const int32_t *row_ptr, const int32_t *col_idx, int32_t d,
                  const uint16_t *Q, const uint16_t *K, const uint16_t *V, double scale,
                  double *O, double *lse, double *P, int32_t nthreads);
int oracle_3s_bwd_f64d(int32_t N, const int32_t *row_ptr, const int32_t *col_idx, int32_t d,
                       const double *Q, const double *K, const double *V, const double *G,
                       double scale, double *dQ, double *dK, double *dV);
int oracle_3s_bwd_f64(int32_t N, const int32_t *row_ptr, const int32_t *col_idx, int32_t d,
                      const uint16_t *Q, const uint16_t *K, const uint16_t *V,
                      const uint16_t *G, double scale, double *dQ, double *dK, double *dV);
int oracle_3s_f64_rows(int32_t N, const int32_t *row_ptr, const int32_t *col_idx, int32_t d,
                       const uint16_t *Q, const uint16_t *K, const uint16_t *V, double scale,
                       int32_t r0, int32_t r1, double *O, int32_t nthreads);
int32_t oracle_num_windows(int32_t N);
int oracle_bsb_sizes(int32_t N, const int32_t *row_ptr, const int32_t *col_idx, int32_t *u,
                     int32_t *nb);
int oracle_bsb_build(int32_t N, const int32_t *row_ptr, const int32_t *col_idx,
                     int32_t *blk_off, int32_t *cols, uint32_t *mask);
double oracle_half_to_double(uint16_t h);
double oracle_bf16_to_double(uint16_t h);
double oracle_e4m3_to_double(uint8_t b);
void oracle_widen_bf16(int64_t count, const uint16_t *h, double *out);
void oracle_widen_e4m3(int64_t count, const uint8_t *b, double *out);

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static uint32_t next_u32(void)
{
    /* xorshift64* */
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    return (uint32_t)((rng_state * 0x2545F4914F6CDD1Dull) >> 32);
}
static int32_t uniform(int32_t n) { return (int32_t)(next_u32() % (uint32_t)n); }
static double unit(void) { return (double)next_u32() / 4294967296.0 * 2.0 - 1.0; }

#define CHECK(c)                                                   \
    do {                                                           \
        if (!(c)) {                                                \
            fprintf(stderr, "check failed: %s (line %d)\n", #c, __LINE__); \
            exit(1);                                               \
        }                                                          \
    } while (0)

/* One random pattern: returns row_ptr (N+1) and col_idx via pointers. */
static void random_pattern(int32_t N, int32_t **rp_out, int32_t **ci_out)
{
    int32_t *rp = malloc(sizeof(int32_t) * (N + 1));
    int32_t cap = N * 12 + 1;
    int32_t *ci = malloc(sizeof(int32_t) * cap);
    rp[0] = 0;
    for (int32_t i = 0; i < N; ++i) {
        int32_t deg = uniform(4) == 0 ? 0 : 1 + uniform(N < 8 ? N : 8);
        for (int32_t k = 0; k < deg; ++k) ci[rp[i] + k] = uniform(N);
        if (deg > 1 && uniform(2)) ci[rp[i] + deg - 1] = ci[rp[i]];   /* a repeat */
        rp[i + 1] = rp[i] + deg;
    }
    *rp_out = rp;
    *ci_out = ci;
}

/* Dense masked softmax of row i (distinct columns), written into o[d]. */
static void dense_row(int32_t N, const int32_t *rp, const int32_t *ci, int32_t d,
                      const double *Q, const double *K, const double *V, double scale,
                      int32_t i, double *o)
{
    char *in = calloc(N, 1);
    for (int32_t e = rp[i]; e < rp[i + 1]; ++e) in[ci[e]] = 1;
    double m = -INFINITY, l = 0.0;
    for (int32_t j = 0; j < N; ++j) {
        if (!in[j]) continue;
        double s = 0.0;
        for (int32_t k = 0; k < d; ++k) s += Q[i * d + k] * K[j * d + k];
        if (scale * s > m) m = scale * s;
    }
    for (int32_t k = 0; k < d; ++k) o[k] = 0.0;
    for (int32_t j = 0; j < N; ++j) {
        if (!in[j]) continue;
        double s = 0.0;
        for (int32_t k = 0; k < d; ++k) s += Q[i * d + k] * K[j * d + k];
        l += exp(scale * s - m);
    }
    for (int32_t j = 0; j < N; ++j) {
        if (!in[j]) continue;
        double s = 0.0;
        for (int32_t k = 0; k < d; ++k) s += Q[i * d + k] * K[j * d + k];
        const double p = exp(scale * s - m) / l;
        for (int32_t k = 0; k < d; ++k) o[k] += p * V[j * d + k];
    }
    free(in);
}

int main(void)
{
    /* decoders over every code */
    for (uint32_t h = 0; h < 65536; ++h) {
        (void)oracle_half_to_double((uint16_t)h);
        (void)oracle_bf16_to_double((uint16_t)h);
    }
    for (uint32_t b = 0; b < 256; ++b) (void)oracle_e4m3_to_double((uint8_t)b);
    {
        uint16_t hb[7] = {0, 1, 0x3f80, 0x7f80, 0x8000, 0xffff, 0x0080};
        uint8_t eb[5] = {0, 1, 0x7e, 0x7f, 0xff};
        double out[7];
        oracle_widen_bf16(7, hb, out);
        oracle_widen_e4m3(5, eb, out);
        oracle_widen_bf16(0, hb, out);
    }
    /* malformed patterns are refused before any row is read */
    {
        int32_t rp[4] = {1, 2, 2, 3}, ci[3] = {0, 1, 2};
        CHECK(oracle_check_csr(3, rp, ci) != 0);
        int32_t rp2[4] = {0, 2, 1, 3};
        CHECK(oracle_check_csr(3, rp2, ci) != 0);
        int32_t rp3[4] = {0, 1, 2, 3}, ci3[3] = {0, 3, 1};
        CHECK(oracle_check_csr(3, rp3, ci3) != 0);
        int32_t ci4[3] = {0, -1, 1};
        CHECK(oracle_check_csr(3, rp3, ci4) != 0);
        double x[3] = {0, 0, 0}, o[3];
        CHECK(oracle_3s_f64d(3, rp3, ci3, 1, x, x, x, 1.0, o, NULL, NULL, 1) != 0);
        CHECK(oracle_3s_f64d(-1, rp3, ci3, 1, x, x, x, 1.0, o, NULL, NULL, 1) != 0);
    }
    for (int trial = 0; trial < 60; ++trial) {
        const int32_t N = trial == 0 ? 1 : 1 + uniform(70);
        const int32_t d = 1 + uniform(8);
        int32_t *rp, *ci;
        random_pattern(N, &rp, &ci);
        CHECK(oracle_check_csr(N, rp, ci) == 0);
        const int64_t nd = (int64_t)N * d, nnz = rp[N];
        double *Q = malloc(sizeof(double) * nd), *K = malloc(sizeof(double) * nd);
        double *V = malloc(sizeof(double) * nd), *G = malloc(sizeof(double) * nd);
        uint16_t *Qh = malloc(2 * nd), *Kh = malloc(2 * nd), *Vh = malloc(2 * nd),
                 *Gh = malloc(2 * nd);
        for (int64_t k = 0; k < nd; ++k) {
            Q[k] = unit();
            K[k] = unit();
            V[k] = unit();
            G[k] = unit();
            Qh[k] = (uint16_t)(0x3000 + uniform(0x0800));   /* finite halves */
            Kh[k] = (uint16_t)(0x3000 + uniform(0x0800)) | (uniform(2) << 15);
            Vh[k] = (uint16_t)(0x3000 + uniform(0x0800)) | (uniform(2) << 15);
            Gh[k] = (uint16_t)(0x3000 + uniform(0x0800));
        }
        double *O = malloc(sizeof(double) * nd), *lse = malloc(sizeof(double) * N);
        double *P = malloc(sizeof(double) * (nnz > 0 ? nnz : 1));
        double *row = malloc(sizeof(double) * d);
        CHECK(oracle_3s_f64d(N, rp, ci, d, Q, K, V, 0.7, O, lse, P, 2) == 0);
        for (int32_t i = 0; i < N; ++i) {
            dense_row(N, rp, ci, d, Q, K, V, 0.7, i, row);
            for (int32_t k = 0; k < d; ++k) CHECK(fabs(row[k] - O[i * d + k]) < 1e-12);
        }
        CHECK(oracle_3s_f64(N, rp, ci, d, Qh, Kh, Vh, 0.3, O, lse, P, 0) == 0);
        const int32_t r0 = uniform(N), r1 = r0 + uniform(N - r0 + 1);
        CHECK(oracle_3s_f64_rows(N, rp, ci, d, Qh, Kh, Vh, 0.3, r0, r1, O, 1) == 0);
        double *dQ = malloc(sizeof(double) * nd), *dK = malloc(sizeof(double) * nd),
               *dV = malloc(sizeof(double) * nd);
        CHECK(oracle_3s_bwd_f64d(N, rp, ci, d, Q, K, V, G, 0.7, dQ, dK, dV) == 0);
        CHECK(oracle_3s_bwd_f64(N, rp, ci, d, Qh, Kh, Vh, Gh, 0.3, dQ, dK, dV) == 0);
        /* BSB layout: every set bit decodes to an entry of the pattern and
           every entry sets a bit */
        const int32_t T = oracle_num_windows(N);
        int32_t *u = malloc(sizeof(int32_t) * T), *nb = malloc(sizeof(int32_t) * T);
        CHECK(oracle_bsb_sizes(N, rp, ci, u, nb) == 0);
        int64_t B = 0;
        for (int32_t w = 0; w < T; ++w) B += nb[w];
        int32_t *blk_off = malloc(sizeof(int32_t) * (T + 1));
        /* exact sizes (one element for an empty layout) */
        int32_t *cols = malloc(sizeof(int32_t) * (B > 0 ? 16 * B : 1));
        uint32_t *mask = malloc(sizeof(uint32_t) * (B > 0 ? 8 * B : 1));
        CHECK(oracle_bsb_build(N, rp, ci, blk_off, cols, mask) == 0);
        CHECK(blk_off[T] == B);
        int64_t bits = 0;
        for (int32_t w = 0; w < T; ++w)
            for (int64_t b = blk_off[w]; b < blk_off[w + 1]; ++b)
                for (int32_t r = 0; r < 16; ++r)
                    for (int32_t c = 0; c < 16; ++c) {
                        const int32_t k = 4 * (r + 16 * (c / 4)) + c % 4;
                        if (!((mask[8 * b + k / 32] >> (k % 32)) & 1u)) continue;
                        ++bits;
                        const int32_t row_i = 16 * w + r, col = cols[16 * b + c];
                        CHECK(row_i < N && col >= 0);
                        int found = 0;
                        for (int32_t e = rp[row_i]; e < rp[row_i + 1]; ++e)
                            found |= ci[e] == col;
                        CHECK(found);
                    }
        int64_t distinct = 0;
        for (int32_t i = 0; i < N; ++i)
            for (int32_t e = rp[i]; e < rp[i + 1]; ++e) {
                int first = 1;
                for (int32_t f = rp[i]; f < e; ++f) first &= ci[f] != ci[e];
                distinct += first;
            }
        CHECK(bits == distinct);
        free(u); free(nb); free(blk_off); free(cols); free(mask);
        free(dQ); free(dK); free(dV);
        free(O); free(lse); free(P); free(row);
        free(Q); free(K); free(V); free(G); free(Qh); free(Kh); free(Vh); free(Gh);
        free(rp); free(ci);
    }
    printf("ok\n");
    return 0;
}
