/*
 * Fastmax fp64 CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow, obviously-correct implementation of the Fastmax attention of
 * "FAST: Factorizable Attention for Speeding up Transformers" (Gerami, Hoover,
 * Dulepet, Duraiswami, arXiv 2402.07901).  Only the test-suite, the smoke
 * check and the bench's CPU-baseline leg may load this library; the product
 * path (the HIP library) never does, and the two share no code.
 *
 * Everything is float64.  Layout of every tensor: [B, H, N, D] contiguous,
 * D fastest; per-row scalars (G) are [B, H, N].
 *
 * Readings of the paper used here (each is justified in the project notes):
 *  - f_p(s) = sum_{l=0..p} s^l / l!, so f_2 = 1 + s + s^2/2 (Sec. 2.2, Eq.
 *    "taylor"); the factorised equations of Sec. 2.4 print the quadratic term
 *    without its 1/2, the definition in Sec. 2.2 has it, and the definition wins.
 *  - Standardisation (Sec. 2.2, Eqs. 6-7) is over the D channels of one token,
 *    with the population standard deviation and no epsilon.
 *  - No temperature by default: the score is q^.k^ itself (Sec. 2.2), unlike
 *    softmax's 1/sqrt(D) (Sec. 2.1).  Every routine takes a score scale tau
 *    (weights f_p(tau q^.k^)); tau = 1 is the paper's definition, tau = 1/D
 *    the unit-norm variant (q^ and k^ divided by sqrt(D), so |tau s| <= 1 as
 *    the bound of Sec. 2.3 assumes and f_1 >= 0, Eq. "valid").
 *  - Causal mask is inclusive: row i sums over n <= i (Sec. 2.1 tril, Sec. 2.4
 *    causal F and G).
 *  - The "I" in the matrix forms of F and G (Sec. 2.4) is the all-ones matrix:
 *    the element forms beside them carry "1 +" for every (i, n).
 *
 * Parity pins: every function here is checked by tests/test_oracle.py against
 * hand-derived golden values (tests/golden/), closed forms, invariants, a
 * library matmul of the explicit attention matrix, finite differences and
 * PyTorch fp64 autograd.  No function is left unpinned.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <omp.h>

/* ------------------------------------------------------------------------ */
/* Sec. 2.2, Eq. (6)-(7): q~ = q - mean(q); q^ = q~ / STD(q~), per token.     */
/* ------------------------------------------------------------------------ */
static void standardize_row(const double *x, long D, double *xh, double *mu_out,
                            double *sig_out)
{
    double mu = 0.0;
    for (long d = 0; d < D; ++d) mu += x[d];
    mu /= (double)D;
    double var = 0.0;
    for (long d = 0; d < D; ++d) {
        double c = x[d] - mu;
        var += c * c;
    }
    var /= (double)D;                 /* population variance */
    double sig = sqrt(var);
    for (long d = 0; d < D; ++d) xh[d] = (x[d] - mu) / sig;
    if (mu_out) *mu_out = mu;
    if (sig_out) *sig_out = sig;
}

/* Sec. 2.2, Eq. "taylor": f(x) = sum_{l=0}^{p} x^l / l!. */
static double f_taylor(double s, int p)
{
    double term = 1.0, acc = 1.0;
    for (int l = 1; l <= p; ++l) {
        term *= s / (double)l;
        acc += term;
    }
    return acc;
}

/* Derivative of f_taylor: sum_{l=1}^{p} x^{l-1}/(l-1)!, i.e. f_{p-1}. */
static double df_taylor(double s, int p)
{
    return p >= 1 ? f_taylor(s, p - 1) : 0.0;
}

static void standardize_all(const double *x, long rows, long D, double *xh,
                            double *mu, double *sig)
{
#pragma omp parallel for schedule(static)
    for (long r = 0; r < rows; ++r)
        standardize_row(x + r * D, D, xh + r * D, mu ? mu + r : NULL,
                        sig ? sig + r : NULL);
}

int fmo_num_threads(void) { return omp_get_max_threads(); }

/* Exposed for tests: standardise `rows` token rows of width D. */
void fmo_standardize(const double *x, long rows, long D, double *xh, double *mu,
                     double *sig)
{
    standardize_all(x, rows, D, xh, mu, sig);
}

/* ------------------------------------------------------------------------ */
/* The explicit attention matrix of one head (Sec. 2.2, a_ij and Eq. "valid";  */
/* masked with tril when causal, Sec. 2.1).  A is N x N, row-major.           */
/* ------------------------------------------------------------------------ */
void fmo_attention_matrix(const double *q, const double *k, long N, long D,
                          int p, int causal, double tau, double *A)
{
    double *qh = malloc(sizeof(double) * N * D);
    double *kh = malloc(sizeof(double) * N * D);
    standardize_all(q, N, D, qh, NULL, NULL);
    standardize_all(k, N, D, kh, NULL, NULL);
#pragma omp parallel for schedule(static)
    for (long i = 0; i < N; ++i) {
        double *row = A + i * N;
        double g = 0.0;
        for (long n = 0; n < N; ++n) {
            double w = 0.0;
            if (!causal || n <= i) {
                double s = 0.0;
                for (long d = 0; d < D; ++d) s += qh[i * D + d] * kh[n * D + d];
                w = f_taylor(tau * s, p);
            }
            row[n] = w;
            g += w;
        }
        for (long n = 0; n < N; ++n) row[n] /= g;
    }
    free(qh);
    free(kh);
}

/* ------------------------------------------------------------------------ */
/* Brute force, one row: o_i = sum_n f(s_in) v_n / sum_n f(s_in)              */
/* (Sec. 2.2, Eq. "tobeexpanded"; causal range n <= i, Sec. 2.4).             */
/* qh_i: standardised query row; kh, v: the head's N x D blocks.              */
/* ------------------------------------------------------------------------ */
static void brute_row(const double *qh_i, const double *kh, const double *v,
                      long i, long N, long D, int p, int causal, double tau,
                      double *o, double *g_out, double *gabs_out)
{
    long nend = causal ? i + 1 : N;
    double g = 0.0, gabs = 0.0;
    for (long d = 0; d < D; ++d) o[d] = 0.0;
    for (long n = 0; n < nend; ++n) {
        double s = 0.0;
        for (long d = 0; d < D; ++d) s += qh_i[d] * kh[n * D + d];
        double w = f_taylor(tau * s, p);
        g += w;
        gabs += fabs(w);
        for (long d = 0; d < D; ++d) o[d] += w * v[n * D + d];
    }
    for (long d = 0; d < D; ++d) o[d] /= g;
    if (g_out) *g_out = g;
    if (gabs_out) *gabs_out = gabs;
}

/* Full brute-force forward, O(N^2 D) per head.  g (row sums G_i) and gabs
 * (sum_n |w_in|, the scale of the cancellation in G for p = 1) may be NULL. */
void fmo_fwd_brute(const double *q, const double *k, const double *v, long B,
                   long H, long N, long D, int p, int causal, double tau,
                   double *out, double *g, double *gabs)
{
    long rows = B * H * N;
    double *qh = malloc(sizeof(double) * rows * D);
    double *kh = malloc(sizeof(double) * rows * D);
    standardize_all(q, rows, D, qh, NULL, NULL);
    standardize_all(k, rows, D, kh, NULL, NULL);
#pragma omp parallel for schedule(dynamic, 16)
    for (long r = 0; r < rows; ++r) {
        long head = r / N, i = r % N;
        brute_row(qh + r * D, kh + head * N * D, v + head * N * D, i, N, D, p,
                  causal, tau, out + r * D, g ? g + r : NULL,
                  gabs ? gabs + r : NULL);
    }
    free(qh);
    free(kh);
}

/* Brute force on a sample of rows.  rows[] holds flat indices b*H*N + h*N + i;
 * out_rows is [nrows, D]; g_rows and gabs_rows are [nrows] (may be NULL). */
void fmo_fwd_rows(const double *q, const double *k, const double *v, long B,
                  long H, long N, long D, int p, int causal, double tau, long nrows,
                  const int64_t *rows, double *out_rows, double *g_rows,
                  double *gabs_rows)
{
    (void)B;
    (void)H;
#pragma omp parallel for schedule(dynamic, 1)
    for (long t = 0; t < nrows; ++t) {
        long r = (long)rows[t];
        long head = r / N, i = r % N;
        long nend = causal ? i + 1 : N;
        double *qh = malloc(sizeof(double) * D);
        double *kh = malloc(sizeof(double) * nend * D);
        standardize_row(q + r * D, D, qh, NULL, NULL);
        for (long n = 0; n < nend; ++n)
            standardize_row(k + (head * N + n) * D, D, kh + n * D, NULL, NULL);
        brute_row(qh, kh, v + head * N * D, i, N, D, p, causal, tau,
                  out_rows + t * D, g_rows ? g_rows + t : NULL,
                  gabs_rows ? gabs_rows + t : NULL);
        free(qh);
        free(kh);
    }
}

/* ------------------------------------------------------------------------ */
/* Factorised forward (Sec. 2.4).  Moments, with j the value column and m, l  */
/* channels (Eqs. "x", "y"):                                                  */
/*   x1_j = sum_n v_nj,  x2_jm = sum_n k_nm v_nj,  x3_jml = sum_n k_nm k_nl v_nj */
/*   y1 = sum_n 1,       y2_m = sum_n k_nm,       y3_ml = sum_n k_nm k_nl      */
/* Query side (Eqs. "f", "g" after reordering, with f_2's 1/2 restored):      */
/*   f_ij = x1_j + sum_m q_im x2_jm + 1/2 sum_{m,l} q_im q_il x3_jml          */
/*   g_i  = y1   + sum_m q_im y2_m  + 1/2 sum_{m,l} q_im q_il y3_ml           */
/*   o_ij = f_ij / g_i  (Eq. "bigo").                                         */
/* Causal: the moments are running sums over n <= i, updated token by token  */
/* (Eqs. "xcausal", "ycausal") and read after adding token i.                 */
/* The quadratic moments are kept as full D x D (not symmetric-packed), as    */
/* the paper writes them.                                                     */
/* ------------------------------------------------------------------------ */
typedef struct {
    long D;
    double *x1, *x2, *x3; /* [D], [D][D], [D][D][D] */
    double y1, *y2, *y3;  /* scalar, [D], [D][D]     */
} moments_t;

static void moments_init(moments_t *M, long D)
{
    M->D = D;
    M->x1 = calloc(D, sizeof(double));
    M->x2 = calloc(D * D, sizeof(double));
    M->x3 = calloc(D * D * D, sizeof(double));
    M->y1 = 0.0;
    M->y2 = calloc(D, sizeof(double));
    M->y3 = calloc(D * D, sizeof(double));
}

static void moments_free(moments_t *M)
{
    free(M->x1);
    free(M->x2);
    free(M->x3);
    free(M->y2);
    free(M->y3);
}

/* Add token n's contribution: k = k^_n (standardised), v = v_n. */
static void moments_add(moments_t *M, const double *k, const double *v, int p)
{
    long D = M->D;
    M->y1 += 1.0;
    for (long m = 0; m < D; ++m) M->y2[m] += k[m];
    if (p >= 2)
        for (long m = 0; m < D; ++m)
            for (long l = 0; l < D; ++l) M->y3[m * D + l] += k[m] * k[l];
    for (long j = 0; j < D; ++j) {
        double vj = v[j];
        M->x1[j] += vj;
        for (long m = 0; m < D; ++m) M->x2[j * D + m] += k[m] * vj;
        if (p >= 2)
            for (long m = 0; m < D; ++m) {
                double kmv = k[m] * vj;
                double *x3jm = M->x3 + (j * D + m) * D;
                for (long l = 0; l < D; ++l) x3jm[l] += kmv * k[l];
            }
    }
}

/* Contract the moments with a standardised query row; writes o (D) and g.
 * With the score scale tau, f(tau s) = 1 + tau s + tau^2 s^2 / 2, so the
 * linear moments enter with tau and the quadratic ones with tau^2 / 2. */
static void moments_query(const moments_t *M, const double *q, int p,
                          double tau, double *o, double *g_out)
{
    long D = M->D;
    double lin = 0.0;
    for (long m = 0; m < D; ++m) lin += q[m] * M->y2[m];
    double g = M->y1 + tau * lin;
    if (p >= 2) {
        double quad = 0.0;
        for (long m = 0; m < D; ++m)
            for (long l = 0; l < D; ++l) quad += q[m] * q[l] * M->y3[m * D + l];
        g += 0.5 * tau * tau * quad;
    }
    for (long j = 0; j < D; ++j) {
        double fl = 0.0;
        for (long m = 0; m < D; ++m) fl += q[m] * M->x2[j * D + m];
        double f = M->x1[j] + tau * fl;
        if (p >= 2) {
            double quad = 0.0;
            for (long m = 0; m < D; ++m) {
                const double *x3jm = M->x3 + (j * D + m) * D;
                double inner = 0.0;
                for (long l = 0; l < D; ++l) inner += q[l] * x3jm[l];
                quad += q[m] * inner;
            }
            f += 0.5 * tau * tau * quad;
        }
        o[j] = f / g;
    }
    if (g_out) *g_out = g;
}

void fmo_fwd_fact(const double *q, const double *k, const double *v, long B,
                  long H, long N, long D, int p, int causal, double tau,
                  double *out, double *g)
{
    long heads = B * H;
#pragma omp parallel for schedule(dynamic, 1)
    for (long hd = 0; hd < heads; ++hd) {
        const double *qb = q + hd * N * D, *kb = k + hd * N * D,
                     *vb = v + hd * N * D;
        double *ob = out + hd * N * D;
        double *gb = g ? g + hd * N : NULL;
        double *qh = malloc(sizeof(double) * D);
        double *kh = malloc(sizeof(double) * D);
        moments_t M;
        moments_init(&M, D);
        if (!causal) {
            for (long n = 0; n < N; ++n) {
                standardize_row(kb + n * D, D, kh, NULL, NULL);
                moments_add(&M, kh, vb + n * D, p);
            }
            for (long i = 0; i < N; ++i) {
                standardize_row(qb + i * D, D, qh, NULL, NULL);
                moments_query(&M, qh, p, tau, ob + i * D, gb ? gb + i : NULL);
            }
        } else {
            for (long i = 0; i < N; ++i) {
                standardize_row(kb + i * D, D, kh, NULL, NULL);
                moments_add(&M, kh, vb + i * D, p);
                standardize_row(qb + i * D, D, qh, NULL, NULL);
                moments_query(&M, qh, p, tau, ob + i * D, gb ? gb + i : NULL);
            }
        }
        moments_free(&M);
        free(qh);
        free(kh);
    }
}

/* ------------------------------------------------------------------------ */
/* Brute-force backward, O(N^2 D) per head.                                  */
/*                                                                           */
/* Score derivative (Sec. 2.3, Eq. "bound", with the index typos read as     */
/* a_in / a_il):  d o_ij / d s_il = f'(s_il) / G_i * (v_lj - o_ij), and       */
/* d o_ij / d v_lj = a_il.  With the score scale tau the weight is            */
/* f(tau s_il), whose derivative in s_il is tau f'(tau s_il).  With upstream  */
/* dO:                                                                        */
/*   ds_il  = sum_j dO_ij tau f'(tau s_il)/G_i (v_lj - o_ij)                   */
/*   dv_l   = sum_i a_il dO_i                                                 */
/*   dq^_i  = sum_l ds_il k^_l,   dk^_l = sum_i ds_il q^_i                     */
/* then back through Eqs. (6)-(7):                                            */
/*   dx = (dx^ - mean(dx^) - x^ * mean(dx^ . x^)) / sigma.                     */
/* Rows of the causal problem only see l <= i.                                */
/* ------------------------------------------------------------------------ */
static void std_backward_row(const double *xh, const double *dxh, double sig,
                             long D, double *dx)
{
    double m1 = 0.0, m2 = 0.0;
    for (long d = 0; d < D; ++d) {
        m1 += dxh[d];
        m2 += dxh[d] * xh[d];
    }
    m1 /= (double)D;
    m2 /= (double)D;
    for (long d = 0; d < D; ++d) dx[d] = (dxh[d] - m1 - xh[d] * m2) / sig;
}

/* o_used (nullable, [B,H,N,D]) is the forward output the gradient is taken
 * at: NULL means the exact O computed here; a caller may pass that O rounded
 * to its storage precision (the stored output a bf16 backward consumes). */
void fmo_bwd_brute(const double *q, const double *k, const double *v,
                   const double *dout, const double *o_used, long B, long H,
                   long N, long D, int p, int causal, double tau, double *dq,
                   double *dk, double *dv)
{
    long heads = B * H;
    for (long hd = 0; hd < heads; ++hd) {
        const double *qb = q + hd * N * D, *kb = k + hd * N * D,
                     *vb = v + hd * N * D, *dob = dout + hd * N * D;
        double *qh = malloc(sizeof(double) * N * D);
        double *kh = malloc(sizeof(double) * N * D);
        double *qs = malloc(sizeof(double) * N), *ks = malloc(sizeof(double) * N);
        double *o = malloc(sizeof(double) * N * D);
        double *G = malloc(sizeof(double) * N);
        double *dqh = malloc(sizeof(double) * N * D);
        double *dkh = malloc(sizeof(double) * N * D);
        standardize_all(qb, N, D, qh, NULL, qs);
        standardize_all(kb, N, D, kh, NULL, ks);
        /* forward, per row */
#pragma omp parallel for schedule(dynamic, 8)
        for (long i = 0; i < N; ++i)
            brute_row(qh + i * D, kh, vb, i, N, D, p, causal, tau, o + i * D, G + i,
                      NULL);
        if (o_used)
            memcpy(o, o_used + hd * N * D, sizeof(double) * N * D);
        /* dq^_i: row i, sums over its allowed columns l */
#pragma omp parallel for schedule(dynamic, 8)
        for (long i = 0; i < N; ++i) {
            long lend = causal ? i + 1 : N;
            double *acc = dqh + i * D;
            for (long d = 0; d < D; ++d) acc[d] = 0.0;
            for (long l = 0; l < lend; ++l) {
                double s = 0.0;
                for (long d = 0; d < D; ++d) s += qh[i * D + d] * kh[l * D + d];
                double coef = tau * df_taylor(tau * s, p) / G[i];
                double ds = 0.0;
                for (long j = 0; j < D; ++j)
                    ds += dob[i * D + j] * coef * (vb[l * D + j] - o[i * D + j]);
                for (long d = 0; d < D; ++d) acc[d] += ds * kh[l * D + d];
            }
        }
        /* dk^_l and dv_l: column l, sums over rows i that see it */
#pragma omp parallel for schedule(dynamic, 8)
        for (long l = 0; l < N; ++l) {
            long istart = causal ? l : 0;
            double *acck = dkh + l * D;
            double *accv = dv + (hd * N + l) * D;
            for (long d = 0; d < D; ++d) acck[d] = accv[d] = 0.0;
            for (long i = istart; i < N; ++i) {
                double s = 0.0;
                for (long d = 0; d < D; ++d) s += qh[i * D + d] * kh[l * D + d];
                double a = f_taylor(tau * s, p) / G[i];
                double coef = tau * df_taylor(tau * s, p) / G[i];
                double ds = 0.0;
                for (long j = 0; j < D; ++j)
                    ds += dob[i * D + j] * coef * (vb[l * D + j] - o[i * D + j]);
                for (long d = 0; d < D; ++d) {
                    acck[d] += ds * qh[i * D + d];
                    accv[d] += a * dob[i * D + d];
                }
            }
        }
#pragma omp parallel for schedule(static)
        for (long r = 0; r < N; ++r) {
            std_backward_row(qh + r * D, dqh + r * D, qs[r], D,
                             dq + (hd * N + r) * D);
            std_backward_row(kh + r * D, dkh + r * D, ks[r], D,
                             dk + (hd * N + r) * D);
        }
        free(qh);
        free(kh);
        free(qs);
        free(ks);
        free(o);
        free(G);
        free(dqh);
        free(dkh);
    }
}

/* ------------------------------------------------------------------------ */
/* "Quadratic" dropout on the factorised terms (Sec. 2.4, the dropout        */
/* paragraph, and Fig. 2).  For p = 2 every key token n carries a keep bit   */
/* b_nt for each of its quadratic features, the D(D+1)/2 distinct products  */
/* k^_nm k^_nl (m <= l), numbered m-major: t(m, l) = m D - m(m-1)/2 + l - m. */
/* A kept feature is scaled by 1/(1 - rate), a dropped one is zero; the      */
/* masked feature enters both x^(3) and y^(3) (it is one embedding), so the  */
/* weight of the pair (i, n) is                                              */
/*   w_in = 1 + tau s_in + sum_{m<=l} c_ml tau^2 q^_im q^_il k^_nm k^_nl b~, */
/* c_mm = 1/2, c_ml = 1 (m < l), b~ = b_nt / (1 - rate).  With every bit set */
/* and rate 0 this is f_2(tau s_in).                                         */
/* Bits: for head hd and token n a row of NW = ceil(D(D+1)/2 / 32) uint32    */
/* words at bits + (hd N + n) NW; feature t is bit t % 32 of word t / 32.    */
/* ------------------------------------------------------------------------ */
static long pair_index(long D, long m, long l)
{
    return m * D - m * (m - 1) / 2 + (l - m);
}

long fmo_mask_words(long D) { return (D * (D + 1) / 2 + 31) / 32; }

/* Philox4x32-10, the counter-based generator of Salmon, Moraes, Dror and
 * Shaw, "Parallel Random Numbers: As Easy as 1, 2, 3" (SC 2011): ten rounds
 * of two 32x32->64 multiplications on a 4-word counter, the 2-word key
 * advanced by the Weyl constants between rounds. */
void fmo_philox4x32_10(const uint32_t *ctr, const uint32_t *key, uint32_t *out)
{
    uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k0 += 0x9E3779B9u;
            k1 += 0xBB67AE85u;
        }
        uint64_t p0 = (uint64_t)0xD2511F53u * c0;
        uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
        uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0;
        uint32_t n1 = (uint32_t)p1;
        uint32_t n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
        uint32_t n3 = (uint32_t)p0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* Keep bits drawn with Philox4x32-10: key = (seed low word, seed high word),
 * counter = (n, t / 4, hd, 0), feature t uses output word t % 4 and is dropped
 * iff that word is below floor(rate 2^32). */
void fmo_dropout_mask(long B, long H, long N, long D, double rate, uint64_t seed,
                      uint32_t *bits)
{
    long heads = B * H, npair = D * (D + 1) / 2, nw = fmo_mask_words(D);
    double t32 = floor(rate * 4294967296.0);
    uint32_t thr = t32 >= 4294967295.0 ? 0xFFFFFFFFu : (uint32_t)t32;
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
#pragma omp parallel for schedule(static)
    for (long r = 0; r < heads * N; ++r) {
        long hd = r / N, n = r % N;
        uint32_t *row = bits + r * nw;
        for (long w = 0; w < nw; ++w) row[w] = 0u;
        for (long t = 0; t < npair; ++t) {
            uint32_t ctr[4] = {(uint32_t)n, (uint32_t)(t / 4), (uint32_t)hd, 0u}, o[4];
            fmo_philox4x32_10(ctr, key, o);
            if (o[t % 4] >= thr) row[t / 32] |= 1u << (t % 32);
        }
    }
}

static double keep_mult(const uint32_t *row, long t, double inv_keep)
{
    return (row[t / 32] >> (t % 32)) & 1u ? inv_keep : 0.0;
}

/* w_in of the definition above for standardised rows qh_i (already times
 * tau) and kh_n with the keep row of token n. */
static double drop_weight(const double *qt, const double *kn, const uint32_t *row,
                          long D, double inv_keep)
{
    double s = 0.0, quad = 0.0;
    for (long m = 0; m < D; ++m) {
        s += qt[m] * kn[m];
        for (long l = m; l < D; ++l) {
            double c = (l == m) ? 0.5 : 1.0;
            quad += c * qt[m] * qt[l] * kn[m] * kn[l] *
                    keep_mult(row, pair_index(D, m, l), inv_keep);
        }
    }
    return 1.0 + s + quad;
}

/* Brute force with the masked weights: O_i = sum_n w_in v_n / sum_n w_in. */
void fmo_fwd_drop_brute(const double *q, const double *k, const double *v,
                        const uint32_t *bits, long B, long H, long N, long D,
                        int causal, double tau, double rate, double *out,
                        double *g)
{
    long heads = B * H, nw = fmo_mask_words(D);
    double inv_keep = 1.0 / (1.0 - rate);
    for (long hd = 0; hd < heads; ++hd) {
        double *qh = malloc(sizeof(double) * N * D);
        double *kh = malloc(sizeof(double) * N * D);
        standardize_all(q + hd * N * D, N, D, qh, NULL, NULL);
        standardize_all(k + hd * N * D, N, D, kh, NULL, NULL);
        for (long r = 0; r < N * D; ++r) qh[r] *= tau;
        const double *vb = v + hd * N * D;
#pragma omp parallel for schedule(dynamic, 4)
        for (long i = 0; i < N; ++i) {
            double *o = out + (hd * N + i) * D;
            for (long j = 0; j < D; ++j) o[j] = 0.0;
            double G = 0.0;
            long nend = causal ? i + 1 : N;
            for (long n = 0; n < nend; ++n) {
                double w = drop_weight(qh + i * D, kh + n * D,
                                       bits + (hd * N + n) * nw, D, inv_keep);
                G += w;
                for (long j = 0; j < D; ++j) o[j] += w * vb[n * D + j];
            }
            for (long j = 0; j < D; ++j) o[j] /= G;
            if (g) g[hd * N + i] = G;
        }
        free(qh);
        free(kh);
    }
}

/* The same by the factorised moments of Sec. 2.4 with the masked quadratic
 * embedding: X1 = sum v'_n, X2[m] = sum k^_nm v'_n, X3[t(m,l)] = sum b~_nt
 * k^_nm k^_nl v'_n over n (all n, or n <= i as a running prefix), v' = [v|1];
 * F_i, G_i = X1 + sum_m tau q^_im X2[m] + sum_{m<=l} c_ml tau^2 q^_im q^_il X3[t]. */
void fmo_fwd_drop_fact(const double *q, const double *k, const double *v,
                       const uint32_t *bits, long B, long H, long N, long D,
                       int causal, double tau, double rate, double *out,
                       double *g)
{
    long heads = B * H, nw = fmo_mask_words(D), npair = D * (D + 1) / 2;
    long D1 = D + 1;
    double inv_keep = 1.0 / (1.0 - rate);
#pragma omp parallel for schedule(dynamic, 1)
    for (long hd = 0; hd < heads; ++hd) {
        double *qh = malloc(sizeof(double) * N * D);
        double *kh = malloc(sizeof(double) * N * D);
        double *X1 = calloc(D1, sizeof(double));
        double *X2 = calloc(D * D1, sizeof(double));
        double *X3 = calloc(npair * D1, sizeof(double));
        double *vp = malloc(sizeof(double) * D1);
        for (long r = 0; r < N; ++r) {
            standardize_row(q + (hd * N + r) * D, D, qh + r * D, NULL, NULL);
            standardize_row(k + (hd * N + r) * D, D, kh + r * D, NULL, NULL);
        }
        const double *vb = v + hd * N * D;
        /* adds token n to the moments */
        #define DROP_ADD(n)                                                       \
            do {                                                                  \
                const double *kn = kh + (n) * D;                                  \
                const uint32_t *row = bits + (hd * N + (n)) * nw;                 \
                for (long j = 0; j < D; ++j) vp[j] = vb[(n) * D + j];             \
                vp[D] = 1.0;                                                      \
                for (long j = 0; j < D1; ++j) X1[j] += vp[j];                     \
                for (long m = 0; m < D; ++m)                                      \
                    for (long j = 0; j < D1; ++j) X2[m * D1 + j] += kn[m] * vp[j]; \
                for (long m = 0; m < D; ++m)                                      \
                    for (long l = m; l < D; ++l) {                                \
                        long t = pair_index(D, m, l);                             \
                        double e = kn[m] * kn[l] * keep_mult(row, t, inv_keep);   \
                        for (long j = 0; j < D1; ++j) X3[t * D1 + j] += e * vp[j]; \
                    }                                                             \
            } while (0)
        if (!causal)
            for (long n = 0; n < N; ++n) DROP_ADD(n);
        for (long i = 0; i < N; ++i) {
            if (causal) DROP_ADD(i);
            const double *qi = qh + i * D;
            double *o = out + (hd * N + i) * D;
            double F[D1];
            for (long j = 0; j < D1; ++j) {
                double acc = X1[j];
                for (long m = 0; m < D; ++m) acc += tau * qi[m] * X2[m * D1 + j];
                for (long m = 0; m < D; ++m)
                    for (long l = m; l < D; ++l) {
                        double c = (l == m) ? 0.5 : 1.0;
                        acc += c * tau * tau * qi[m] * qi[l] *
                               X3[pair_index(D, m, l) * D1 + j];
                    }
                F[j] = acc;
            }
            for (long j = 0; j < D; ++j) o[j] = F[j] / F[D];
            if (g) g[hd * N + i] = F[D];
        }
        #undef DROP_ADD
        free(qh); free(kh); free(X1); free(X2); free(X3); free(vp);
    }
}

/* Gradients of the masked forward (the mask is a constant).  With
 * q~ = tau q^, z_l = q~_l k^_nl and h_a = 1 + sum_l z_l b~_{n,t(a,l)}:
 *   dw_in/dq~_ia = k^_na h_a,  dw_in/dk^_na = q~_ia h_a,
 * and, as in the unmasked case, dO_i/dw_in = (v_n - O_i) / G_i, so
 *   dq~_i = sum_n (dO_i.(v_n - O_i)/G_i) k^_n (.) h,  dq^ = tau dq~,
 *   dk^_n = sum_i (dO_i.(v_n - O_i)/G_i) q~_i (.) h,  dv_n = sum_i w_in dO_i/G_i,
 * then back through Eqs. (6)-(7).  o_used as in fmo_bwd_brute. */
void fmo_bwd_drop_brute(const double *q, const double *k, const double *v,
                        const double *dout, const double *o_used,
                        const uint32_t *bits, long B, long H, long N, long D,
                        int causal, double tau, double rate, double *dq,
                        double *dk, double *dv)
{
    long heads = B * H, nw = fmo_mask_words(D);
    double inv_keep = 1.0 / (1.0 - rate);
    for (long hd = 0; hd < heads; ++hd) {
        const double *vb = v + hd * N * D, *dob = dout + hd * N * D;
        double *qh = malloc(sizeof(double) * N * D);
        double *kh = malloc(sizeof(double) * N * D);
        double *qs = malloc(sizeof(double) * N), *ks = malloc(sizeof(double) * N);
        double *o = malloc(sizeof(double) * N * D);
        double *G = malloc(sizeof(double) * N);
        double *dqt = calloc(N * D, sizeof(double));
        double *dkh = calloc(N * D, sizeof(double));
        double *dvh = calloc(N * D, sizeof(double));
        standardize_all(q + hd * N * D, N, D, qh, NULL, qs);
        standardize_all(k + hd * N * D, N, D, kh, NULL, ks);
        double *qt = malloc(sizeof(double) * N * D);
        for (long r = 0; r < N * D; ++r) qt[r] = tau * qh[r];
        const uint32_t *hb = bits + hd * N * nw;
        /* forward at the same mask */
        for (long i = 0; i < N; ++i) {
            double Gi = 0.0;
            for (long j = 0; j < D; ++j) o[i * D + j] = 0.0;
            long nend = causal ? i + 1 : N;
            for (long n = 0; n < nend; ++n) {
                double w = drop_weight(qt + i * D, kh + n * D, hb + n * nw, D, inv_keep);
                Gi += w;
                for (long j = 0; j < D; ++j) o[i * D + j] += w * vb[n * D + j];
            }
            for (long j = 0; j < D; ++j) o[i * D + j] /= Gi;
            G[i] = Gi;
        }
        if (o_used) memcpy(o, o_used + hd * N * D, sizeof(double) * N * D);
        /* dq~: row i over the keys it sees; dk^, dv: key n over the rows
         * that see it (each loop parallel over the index it owns) */
#pragma omp parallel for schedule(dynamic, 4)
        for (long i = 0; i < N; ++i) {
            double h[D];
            long nend = causal ? i + 1 : N;
            for (long n = 0; n < nend; ++n) {
                const uint32_t *row = hb + n * nw;
                const double *qi = qt + i * D, *kn = kh + n * D;
                double dw = 0.0;
                for (long j = 0; j < D; ++j) dw += dob[i * D + j] * (vb[n * D + j] - o[i * D + j]);
                dw /= G[i];
                for (long a = 0; a < D; ++a) {
                    double acc = 1.0;
                    for (long l = 0; l < D; ++l) {
                        long t = a <= l ? pair_index(D, a, l) : pair_index(D, l, a);
                        acc += qi[l] * kn[l] * keep_mult(row, t, inv_keep);
                    }
                    h[a] = acc;
                }
                for (long a = 0; a < D; ++a) dqt[i * D + a] += dw * kn[a] * h[a];
            }
        }
#pragma omp parallel for schedule(dynamic, 4)
        for (long n = 0; n < N; ++n) {
            double h[D];
            long istart = causal ? n : 0;
            const uint32_t *row = hb + n * nw;
            for (long i = istart; i < N; ++i) {
                const double *qi = qt + i * D, *kn = kh + n * D;
                double dw = 0.0;
                for (long j = 0; j < D; ++j) dw += dob[i * D + j] * (vb[n * D + j] - o[i * D + j]);
                dw /= G[i];
                double w = drop_weight(qi, kn, row, D, inv_keep);
                for (long a = 0; a < D; ++a) {
                    double acc = 1.0;
                    for (long l = 0; l < D; ++l) {
                        long t = a <= l ? pair_index(D, a, l) : pair_index(D, l, a);
                        acc += qi[l] * kn[l] * keep_mult(row, t, inv_keep);
                    }
                    h[a] = acc;
                }
                for (long a = 0; a < D; ++a) {
                    dkh[n * D + a] += dw * qi[a] * h[a];
                    dvh[n * D + a] += w * dob[i * D + a] / G[i];
                }
            }
        }
#pragma omp parallel for schedule(static)
        for (long r = 0; r < N; ++r) {
            double dqh[D];
            for (long a = 0; a < D; ++a) dqh[a] = tau * dqt[r * D + a];
            std_backward_row(qh + r * D, dqh, qs[r], D, dq + (hd * N + r) * D);
            std_backward_row(kh + r * D, dkh + r * D, ks[r], D, dk + (hd * N + r) * D);
            for (long a = 0; a < D; ++a) dv[(hd * N + r) * D + a] = dvh[r * D + a];
        }
        free(qh); free(kh); free(qs); free(ks); free(o); free(G);
        free(dqt); free(dkh); free(dvh); free(qt);
    }
}
