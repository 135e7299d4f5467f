/*
 * Fused-3S reference oracle: plain, slow, obviously correct fp64 CPU code.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or
 * call this file; only the tests, the package smoke check and the bench's
 * CPU-baseline leg do.  It shares no code, header, table or helper with the
 * HIP library (it has its own binary16 decoder, its own sort, its own CSR
 * walk).
 *
 * What it computes (paper: Section 2.1, Eq. 1 and its three-step
 * decomposition; Section 3.5, Eq. 7; Algorithm 1's Ensure clause):
 *
 *     O = softmax_rows( mask_A( scale * Q K^T ) ) V
 *
 * read as a MASKED softmax: for row i only the columns j with A[i][j] != 0
 * take part, every other column is excluded (not a zero score).  A is binary,
 * so a column listed twice in a CSR row counts once.  A row with no
 * neighbour produces O[i,:] = 0 (the paper divides by l = 0 there; we take
 * the limit of an empty sum).
 *
 * Second part: the Binary Sparse Block (BSB) layout of Section 3.1 (row
 * windows of r = 16 rows, all-zero columns removed per window, the compacted
 * window cut into 16x16 blocks, one bitmap per block), together with the
 * reordered work list of Section 3.2 ("row window reordering": windows in
 * decreasing order of block count).  These are integer definitions; the GPU
 * plan must reproduce them bit for bit.
 *
 * Parity status of each function is stated in its comment; all are pinned by
 * the CPU test-suite against closed forms, library routines and brute force.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ---------------------------------------------------------------------- */
/* IEEE 754 binary16 -> double, written from the format definition:        */
/* 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits.                 */
/* Every binary16 value is exactly representable as a double.              */
/* ---------------------------------------------------------------------- */
static double half_bits_to_double(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int expo = (h >> 10) & 0x1f;
    int frac = h & 0x3ff;
    double v;
    if (expo == 0) {
        v = ldexp((double)frac, -24);            /* subnormal: frac * 2^-24 */
    } else if (expo == 31) {
        v = frac ? NAN : INFINITY;
    } else {
        v = ldexp((double)(frac + 1024), expo - 25); /* (1 + f/1024) 2^(e-15) */
    }
    return sign ? -v : v;
}

double oracle_half_to_double(uint16_t h) { return half_bits_to_double(h); }

/* ---------------------------------------------------------------------- */
/* bfloat16 -> double, from the format definition: 1 sign bit, 8 exponent  */
/* bits (bias 127, as binary32), 7 fraction bits.  Exact in double.        */
/* ---------------------------------------------------------------------- */
static double bf16_bits_to_double(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int expo = (h >> 7) & 0xff;
    int frac = h & 0x7f;
    double v;
    if (expo == 0) {
        v = ldexp((double)frac, -133);           /* subnormal: frac * 2^-133 */
    } else if (expo == 255) {
        v = frac ? NAN : INFINITY;
    } else {
        v = ldexp((double)(frac + 128), expo - 134); /* (1 + f/128) 2^(e-127) */
    }
    return sign ? -v : v;
}

double oracle_bf16_to_double(uint16_t h) { return bf16_bits_to_double(h); }

/* count bfloat16 bit patterns -> fp64 (exact). */
void oracle_widen_bf16(int64_t count, const uint16_t *h, double *out)
{
    for (int64_t k = 0; k < count; ++k) out[k] = bf16_bits_to_double(h[k]);
}

/* ---------------------------------------------------------------------- */
/* OCP 8-bit float e4m3 -> double, from the format definition: 1 sign bit, */
/* 4 exponent bits (bias 7), 3 fraction bits; no infinities, the all-ones  */
/* exponent with all-ones fraction is NaN.  Exact in double.               */
/* ---------------------------------------------------------------------- */
static double e4m3_bits_to_double(uint8_t b)
{
    int sign = (b >> 7) & 1;
    int expo = (b >> 3) & 0xf;
    int frac = b & 0x7;
    double v;
    if (expo == 0) {
        v = ldexp((double)frac, -9);             /* subnormal: frac * 2^-9 */
    } else if (expo == 15 && frac == 7) {
        v = NAN;
    } else {
        v = ldexp((double)(frac + 8), expo - 10); /* (1 + f/8) 2^(e-7) */
    }
    return sign ? -v : v;
}

double oracle_e4m3_to_double(uint8_t b) { return e4m3_bits_to_double(b); }

/* count e4m3 bytes -> fp64 (exact). */
void oracle_widen_e4m3(int64_t count, const uint8_t *b, double *out)
{
    for (int64_t k = 0; k < count; ++k) out[k] = e4m3_bits_to_double(b[k]);
}

/* Decoding table: entry h is half_bits_to_double(h) (filled once). */
static double g_half_table[65536];
static int g_half_table_ready = 0;

static void fill_half_table(void)
{
    if (g_half_table_ready) return;
    for (int h = 0; h < 65536; ++h) g_half_table[h] = half_bits_to_double((uint16_t)h);
    g_half_table_ready = 1;
}

#define H2D(h) (g_half_table[(h)])

static int cmp_int32(const void *a, const void *b)
{
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    return (x > y) - (x < y);
}

/* CSR sanity: row_ptr[0] == 0, non-decreasing, every column in [0, N). */
int oracle_check_csr(int32_t N, const int32_t *row_ptr, const int32_t *col_idx)
{
    if (N < 0) return -1;
    if (row_ptr[0] != 0) return -2;
    for (int32_t i = 0; i < N; ++i)
        if (row_ptr[i + 1] < row_ptr[i]) return -3;
    for (int64_t k = 0; k < row_ptr[N]; ++k)
        if (col_idx[k] < 0 || col_idx[k] >= N) return -4;
    return 0;
}

/*
 * The 3S operator, fp64 throughout, on fp64 inputs (the binary16 entry point
 * below widens its inputs exactly and calls this one).
 *
 * Q, K, V: N x d row-major.  O: N x d output.
 * lse (may be NULL): per row m + log(l), -inf for an empty row.
 * P   (may be NULL): per CSR entry k, the probability of its column, written
 *     at the FIRST occurrence of that column in the row; 0 at repeats.
 * nthreads <= 0 means "OpenMP default".
 * Returns 0, or a negative code when the CSR is malformed.
 *
 * Steps per row i, in the order of the definition (Eq. 1, Eq. 7):
 *   1. Nb(i) = distinct columns of row i
 *   2. s_j   = scale * sum_k Q[i,k] K[j,k]           (SDDMM on the pattern)
 *   3. m     = max_j s_j                              (max-stabilised softmax)
 *   4. e_j   = exp(s_j - m),  l = sum_j e_j,  P_ij = e_j / l
 *   5. O[i,:] = sum_j P_ij V[j,:]                     (SpMM)
 */
int oracle_3s_f64d(int32_t N, const int32_t *row_ptr, const int32_t *col_idx,
                   int32_t d, const double *Q, const double *K, const double *V,
                   double scale, double *O, double *lse, double *P, int32_t nthreads)
{
    int rc = oracle_check_csr(N, row_ptr, col_idx);
    if (rc) return rc;
    if (d <= 0) return -5;
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 64) reduction(| : bad)
    for (int32_t i = 0; i < N; ++i) {
        int64_t beg = row_ptr[i], end = row_ptr[i + 1];
        int64_t n = end - beg;
        double *o = O + (int64_t)i * d;
        for (int32_t k = 0; k < d; ++k) o[k] = 0.0;
        if (P)
            for (int64_t k = beg; k < end; ++k) P[k] = 0.0;
        if (n == 0) {
            if (lse) lse[i] = -INFINITY;
            continue;
        }
        /* 1. distinct neighbours */
        int32_t *nb = (int32_t *)malloc(sizeof(int32_t) * n);
        double *s = (double *)malloc(sizeof(double) * n);
        if (!nb || !s) { free(nb); free(s); bad = 1; continue; }
        memcpy(nb, col_idx + beg, sizeof(int32_t) * n);
        qsort(nb, n, sizeof(int32_t), cmp_int32);
        int64_t u = 0;
        for (int64_t k = 0; k < n; ++k)
            if (k == 0 || nb[k] != nb[k - 1]) nb[u++] = nb[k];
        /* 2. scores */
        for (int64_t a = 0; a < u; ++a) {
            const double *q = Q + (int64_t)i * d;
            const double *kr = K + (int64_t)nb[a] * d;
            double acc = 0.0;
            for (int32_t k = 0; k < d; ++k) acc += q[k] * kr[k];
            s[a] = scale * acc;
        }
        /* 3. row max */
        double m = s[0];
        for (int64_t a = 1; a < u; ++a)
            if (s[a] > m) m = s[a];
        /* 4. exponentials and their sum */
        double l = 0.0;
        for (int64_t a = 0; a < u; ++a) {
            s[a] = exp(s[a] - m);
            l += s[a];
        }
        /* 5. weighted sum of neighbour V rows */
        for (int64_t a = 0; a < u; ++a) {
            double p = s[a] / l;
            const double *vr = V + (int64_t)nb[a] * d;
            for (int32_t k = 0; k < d; ++k) o[k] += p * vr[k];
            if (P) {
                for (int64_t k = beg; k < end; ++k)
                    if (col_idx[k] == nb[a]) { P[k] = p; break; }
            }
        }
        if (lse) lse[i] = m + log(l);
        free(nb);
        free(s);
    }
    return bad ? -6 : 0;
}

/* N x d binary16 bit patterns -> fp64 (exact). */
static double *widen(const uint16_t *h, int64_t count)
{
    double *out = (double *)malloc(sizeof(double) * (count > 0 ? count : 1));
    if (!out) return NULL;
    for (int64_t k = 0; k < count; ++k) out[k] = H2D(h[k]);
    return out;
}

/* The 3S operator on binary16 inputs (see oracle_3s_f64d). */
int oracle_3s_f64(int32_t N, const int32_t *row_ptr, const int32_t *col_idx,
                  int32_t d, const uint16_t *Q, const uint16_t *K,
                  const uint16_t *V, double scale, double *O, double *lse,
                  double *P, int32_t nthreads)
{
    if (d <= 0 || N < 0) return -5;
    fill_half_table();
    int64_t count = (int64_t)N * d;
    double *q = widen(Q, count), *k = widen(K, count), *v = widen(V, count);
    int rc = -6;
    if (q && k && v)
        rc = oracle_3s_f64d(N, row_ptr, col_idx, d, q, k, v, scale, O, lse, P, nthreads);
    free(q);
    free(k);
    free(v);
    return rc;
}

/*
 * Gradients of the 3S operator (the backward pass the paper names as the
 * next step), fp64, on fp64 inputs.  With P_ij the probabilities of the
 * forward (masked, Eq. 1 / Eq. 7) and G = dL/dO:
 *   dV_j   = sum_i P_ij G_i                      (i over rows holding column j)
 *   dP_ij  = G_i . V_j
 *   D_i    = sum_j P_ij dP_ij  (= G_i . O_i)
 *   dS_ij  = P_ij (dP_ij - D_i)                  (softmax Jacobian)
 *   dQ_i   = scale * sum_j dS_ij K_j
 *   dK_j   = scale * sum_i dS_ij Q_i
 * Rows are visited in order and the column sums are accumulated in that
 * order (sequential; no threads).  Empty rows contribute nothing.
 */
int oracle_3s_bwd_f64d(int32_t N, const int32_t *row_ptr, const int32_t *col_idx,
                       int32_t d, const double *Q, const double *K, const double *V,
                       const double *G, double scale, double *dQ, double *dK,
                       double *dV)
{
    int rc = oracle_check_csr(N, row_ptr, col_idx);
    if (rc) return rc;
    if (d <= 0) return -5;
    int64_t count = (int64_t)N * d;
    for (int64_t k = 0; k < count; ++k) dQ[k] = dK[k] = dV[k] = 0.0;
    int64_t maxn = 0;
    for (int32_t i = 0; i < N; ++i)
        if (row_ptr[i + 1] - row_ptr[i] > maxn) maxn = row_ptr[i + 1] - row_ptr[i];
    int32_t *nb = (int32_t *)malloc(sizeof(int32_t) * (maxn > 0 ? maxn : 1));
    double *p = (double *)malloc(sizeof(double) * (maxn > 0 ? maxn : 1));
    double *dp = (double *)malloc(sizeof(double) * (maxn > 0 ? maxn : 1));
    if (!nb || !p || !dp) { free(nb); free(p); free(dp); return -6; }
    for (int32_t i = 0; i < N; ++i) {
        int64_t beg = row_ptr[i], n = row_ptr[i + 1] - beg;
        if (n == 0) continue;
        memcpy(nb, col_idx + beg, sizeof(int32_t) * n);
        qsort(nb, n, sizeof(int32_t), cmp_int32);
        int64_t u = 0;
        for (int64_t k = 0; k < n; ++k)
            if (k == 0 || nb[k] != nb[k - 1]) nb[u++] = nb[k];
        const double *q = Q + (int64_t)i * d, *g = G + (int64_t)i * d;
        /* forward probabilities of row i */
        double m = -INFINITY;
        for (int64_t a = 0; a < u; ++a) {
            const double *kr = K + (int64_t)nb[a] * d;
            double acc = 0.0;
            for (int32_t k = 0; k < d; ++k) acc += q[k] * kr[k];
            p[a] = scale * acc;
            if (p[a] > m) m = p[a];
        }
        double l = 0.0;
        for (int64_t a = 0; a < u; ++a) {
            p[a] = exp(p[a] - m);
            l += p[a];
        }
        for (int64_t a = 0; a < u; ++a) p[a] /= l;
        /* dP and D */
        double D = 0.0;
        for (int64_t a = 0; a < u; ++a) {
            const double *vr = V + (int64_t)nb[a] * d;
            double acc = 0.0;
            for (int32_t k = 0; k < d; ++k) acc += g[k] * vr[k];
            dp[a] = acc;
            D += p[a] * acc;
        }
        /* accumulate */
        for (int64_t a = 0; a < u; ++a) {
            const int64_t j = nb[a];
            const double ds = p[a] * (dp[a] - D);
            const double *kr = K + j * d;
            double *dq = dQ + (int64_t)i * d, *dk = dK + j * d, *dv = dV + j * d;
            for (int32_t k = 0; k < d; ++k) {
                dq[k] += scale * ds * kr[k];
                dk[k] += scale * ds * q[k];
                dv[k] += p[a] * g[k];
            }
        }
    }
    free(nb);
    free(p);
    free(dp);
    return 0;
}

/* Gradients on binary16 inputs (G = dL/dO given as binary16 too). */
int oracle_3s_bwd_f64(int32_t N, const int32_t *row_ptr, const int32_t *col_idx,
                      int32_t d, const uint16_t *Q, const uint16_t *K,
                      const uint16_t *V, const uint16_t *G, double scale, double *dQ,
                      double *dK, double *dV)
{
    if (d <= 0 || N < 0) return -5;
    fill_half_table();
    int64_t count = (int64_t)N * d;
    double *q = widen(Q, count), *k = widen(K, count), *v = widen(V, count),
           *g = widen(G, count);
    int rc = -6;
    if (q && k && v && g)
        rc = oracle_3s_bwd_f64d(N, row_ptr, col_idx, d, q, k, v, g, scale, dQ, dK, dV);
    free(q);
    free(k);
    free(v);
    free(g);
    return rc;
}

/* Same as oracle_3s_f64 on the row range [r0, r1) only (bounded samples). */
int oracle_3s_f64_rows(int32_t N, const int32_t *row_ptr, const int32_t *col_idx,
                       int32_t d, const uint16_t *Q, const uint16_t *K,
                       const uint16_t *V, double scale, int32_t r0, int32_t r1,
                       double *O_rows, int32_t nthreads)
{
    if (r0 < 0 || r1 > N || r0 > r1) return -7;
    /* Build a CSR view of rows [r0, r1) whose column space is still [0, N);
     * Q rows are taken from the same range so the sub-problem is the exact
     * restriction of the full operator to those rows. */
    int32_t n = r1 - r0;
    int32_t *rp = (int32_t *)malloc(sizeof(int32_t) * ((size_t)N + 1));
    if (!rp) return -6;
    /* rows outside the range are empty in this view */
    int64_t base = row_ptr[r0];
    for (int32_t i = 0; i <= N; ++i) {
        int32_t src = i < r0 ? r0 : (i > r1 ? r1 : i);
        rp[i] = (int32_t)(row_ptr[src] - base);
    }
    double *Ofull = (double *)calloc((size_t)N * d, sizeof(double));
    if (!Ofull) { free(rp); return -6; }
    int rc = oracle_3s_f64(N, rp, col_idx + base, d, Q, K, V, scale, Ofull,
                           NULL, NULL, nthreads);
    if (rc == 0) memcpy(O_rows, Ofull + (int64_t)r0 * d, sizeof(double) * (size_t)n * d);
    free(rp);
    free(Ofull);
    return rc;
}

/* ---------------------------------------------------------------------- */
/* Binary Sparse Block layout (Section 3.1), r = 16 rows per window,       */
/* c = 16 columns per block.                                                */
/* ---------------------------------------------------------------------- */
#define RW 16
#define BC 16

/* Number of row windows, ceil(N / r) (Algorithm 1: T_r). */
int32_t oracle_num_windows(int32_t N) { return (N + RW - 1) / RW; }

/*
 * Row windows given by their first rows: window w covers the rows
 * [win_row[w], win_row[w+1]), between 1 and 16 of them, in increasing order
 * from win_row[0] = 0.  The fixed windows of Algorithm 1 are
 * win_row[w] = 16 w (the last one clipped at N); windows aligned to the
 * graphs of a batch (the component-aware layout Section 4.2 leaves to
 * future work) give other starts.  Returns 0, or -2 if win_row breaks
 * these rules.
 */
static int check_windows(int32_t T, const int32_t *win_row)
{
    if (T < 0 || win_row[0] != 0) return -2;
    for (int32_t w = 0; w < T; ++w) {
        int32_t n = win_row[w + 1] - win_row[w];
        if (n < 1 || n > RW) return -2;
    }
    return 0;
}

/*
 * Step 2 of the construction: per window w, the sorted distinct columns that
 * hold at least one non-zero (all-zero columns removed).  Writes u[w] (count)
 * and nb[w] = ceil(u[w] / 16) (step 3: number of blocks).  Returns 0.
 */
int oracle_bsb_sizes_rows(int32_t T, const int32_t *win_row, const int32_t *row_ptr,
                          const int32_t *col_idx, int32_t *u, int32_t *nb)
{
    if (check_windows(T, win_row)) return -2;
    for (int32_t w = 0; w < T; ++w) {
        int32_t r0 = win_row[w], r1 = win_row[w + 1];
        int64_t beg = row_ptr[r0], end = row_ptr[r1], n = end - beg;
        int64_t cnt = 0;
        if (n > 0) {
            int32_t *c = (int32_t *)malloc(sizeof(int32_t) * n);
            if (!c) return -6;
            memcpy(c, col_idx + beg, sizeof(int32_t) * n);
            qsort(c, n, sizeof(int32_t), cmp_int32);
            for (int64_t k = 0; k < n; ++k)
                if (k == 0 || c[k] != c[k - 1]) ++cnt;
            free(c);
        }
        u[w] = (int32_t)cnt;
        nb[w] = (int32_t)((cnt + BC - 1) / BC);
    }
    return 0;
}

/*
 * Steps 2-4 of the construction, written into caller-sized arrays:
 *   blk_off[T+1]  exclusive prefix of blocks per window (the paper's tro)
 *   cols[16*B]    compacted -> original column of each block slot (the
 *                 gather list the paper calls sptd), -1 in padding slots
 *   mask[8*B]     one 256-bit bitmap per 16x16 block.
 * Bit convention (a storage choice; it does not change which bits are set):
 * the non-zero at window row r (0..15, counted from the window's first row)
 * and block column c (0..15) is bit
 *     k = 4 * (r + 16 * (c / 4)) + (c % 4)
 * of the block, i.e. bit (k % 32) of 32-bit word (k / 32).
 */
int oracle_bsb_build_rows(int32_t T, const int32_t *win_row, const int32_t *row_ptr,
                          const int32_t *col_idx, int32_t *blk_off, int32_t *cols,
                          uint32_t *mask)
{
    if (check_windows(T, win_row)) return -2;
    int32_t *u = (int32_t *)malloc(sizeof(int32_t) * (T > 0 ? T : 1));
    int32_t *nb = (int32_t *)malloc(sizeof(int32_t) * (T > 0 ? T : 1));
    if (!u || !nb) { free(u); free(nb); return -6; }
    int rc = oracle_bsb_sizes_rows(T, win_row, row_ptr, col_idx, u, nb);
    if (rc) { free(u); free(nb); return rc; }
    blk_off[0] = 0;
    for (int32_t w = 0; w < T; ++w) blk_off[w + 1] = blk_off[w] + nb[w];
    int64_t B = blk_off[T];
    for (int64_t k = 0; k < BC * B; ++k) cols[k] = -1;
    for (int64_t k = 0; k < 8 * B; ++k) mask[k] = 0;
    for (int32_t w = 0; w < T; ++w) {
        int32_t r0 = win_row[w], r1 = win_row[w + 1];
        int64_t beg = row_ptr[r0], end = row_ptr[r1], n = end - beg;
        if (n == 0) continue;
        int32_t *c = (int32_t *)malloc(sizeof(int32_t) * n);
        if (!c) { free(u); free(nb); return -6; }
        memcpy(c, col_idx + beg, sizeof(int32_t) * n);
        qsort(c, n, sizeof(int32_t), cmp_int32);
        int64_t cnt = 0;
        for (int64_t k = 0; k < n; ++k)
            if (k == 0 || c[k] != c[k - 1]) c[cnt++] = c[k];
        int32_t *slot = cols + (int64_t)BC * blk_off[w];
        for (int64_t k = 0; k < cnt; ++k) slot[k] = c[k];
        for (int32_t r = r0; r < r1; ++r) {
            for (int64_t e = row_ptr[r]; e < row_ptr[r + 1]; ++e) {
                /* compacted position of the column in the sorted list */
                const int32_t *hit = (const int32_t *)bsearch(
                    &col_idx[e], c, cnt, sizeof(int32_t), cmp_int32);
                int64_t p = hit - c;
                int64_t blk = blk_off[w] + p / BC;
                int32_t cc = (int32_t)(p % BC), rr = r - r0;
                int32_t bit = 4 * (rr + 16 * (cc / 4)) + (cc % 4);
                mask[8 * blk + bit / 32] |= 1u << (bit % 32);
            }
        }
        free(c);
    }
    free(u);
    free(nb);
    return 0;
}

/* The fixed windows of Algorithm 1: rows [16 w, min(16 w + 16, N)). */
static int32_t *fixed_windows(int32_t N)
{
    int32_t T = oracle_num_windows(N);
    int32_t *win_row = (int32_t *)malloc(sizeof(int32_t) * (T + 1));
    if (!win_row) return NULL;
    for (int32_t w = 0; w < T; ++w) win_row[w] = w * RW;
    win_row[T] = N;
    return win_row;
}

int oracle_bsb_sizes(int32_t N, const int32_t *row_ptr, const int32_t *col_idx,
                     int32_t *u, int32_t *nb)
{
    int32_t *win_row = fixed_windows(N);
    if (!win_row) return -6;
    int rc = oracle_bsb_sizes_rows(oracle_num_windows(N), win_row, row_ptr, col_idx, u, nb);
    free(win_row);
    return rc;
}

int oracle_bsb_build(int32_t N, const int32_t *row_ptr, const int32_t *col_idx,
                     int32_t *blk_off, int32_t *cols, uint32_t *mask)
{
    int32_t *win_row = fixed_windows(N);
    if (!win_row) return -6;
    int rc = oracle_bsb_build_rows(oracle_num_windows(N), win_row, row_ptr, col_idx,
                                   blk_off, cols, mask);
    free(win_row);
    return rc;
}
