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
