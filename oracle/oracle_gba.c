/*
 * oracle_gba.c -- CPU reference for the fused matmul + bias + ReLU.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path links, loads or
 * calls this file: only the tests, the smoke check and the benchmark's CPU
 * baseline leg do.  It shares no code, header or constant with the HIP
 * library.
 *
 * What it computes (Problem Statement section, Listing 1 and the expression
 * tree described there: the root of the pointwise statement is ReLU, its
 * child is the add of the matmul result and the bias):
 *
 *     pre(i,j) = sum_{k=0..K-1} A(i,k) * B(k,j)  +  bias(j)
 *     out(i,j) = act == RELU ? (pre > 0 ? pre : 0) : pre
 *
 * evaluated in IEEE binary64 with k ascending, the bias added last, and no
 * rounding to fp16 anywhere.  (The one exception is the fp16-accumulation
 * reading offered by oracle_fused_rows_f64 with acc16 = 1, described above
 * product_row_acc16: one running sum through both products, rounded to
 * binary16 at the end of every aligned 32-deep group of each product.)  Inputs are fp16 bit patterns decoded by the
 * routine below (sign, 5-bit exponent, 10-bit fraction, subnormals).  The
 * product of two fp16 values is exact in binary64 (11 + 11 significant bits),
 * so the only rounding is in the running sum.
 *
 * Operand storage (row- or column-major A and B, Background section and the
 * four layout specialisations of the Matmul Compute Decomposition section):
 *     A(i,k) = layout_a == ROW ? A[i*lda + k] : A[k*lda + i]
 *     B(k,j) = layout_b == ROW ? B[k*ldb + j] : B[j*ldb + k]
 * The output is written row-major as doubles: out[r*ldo + j].
 *
 * Readings of points the paper leaves open: bias is a length-N vector
 * broadcast over rows (NULL = no bias); leading dimensions have BLAS meaning.
 *
 * Build: plain C11, no -ffast-math, -ffp-contract=off (no fused multiply-add,
 * so every product is rounded exactly as written).
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { OR_ROW = 0, OR_COL = 1 };
enum { OR_ACT_NONE = 0, OR_ACT_RELU = 1 };

/* IEEE 754 binary16 -> binary64, written out from the format definition. */
double oracle_f16_to_f64(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int expo = (h >> 10) & 0x1f;
    int frac = h & 0x3ff;
    double v;
    if (expo == 0)              /* zero or subnormal: frac * 2^-24 */
        v = ldexp((double)frac, -24);
    else if (expo == 31)        /* infinity or NaN */
        v = frac ? NAN : INFINITY;
    else                        /* normal: (1 + frac/1024) * 2^(expo-15) */
        v = ldexp((double)(1024 + frac), expo - 25);
    return sign ? -v : v;
}

/*
 * Round a binary64 value to the nearest binary16 value, ties to even
 * (IEEE 754 roundTiesToEven), returned as a binary64.  Written from the
 * format: a value in [2^(e-1), 2^e) has quantum 2^(e-11) in binary16; below
 * 2^-14 (subnormals) the quantum is 2^-24.  Magnitudes of 65520 and above
 * (halfway past the largest finite value 65504) become infinities.
 */
double oracle_round_f16(double x)
{
    if (isnan(x) || x == 0.0)
        return x;
    double ax = fabs(x);
    if (ax >= 65520.0)
        return copysign(INFINITY, x);
    int e;
    frexp(ax, &e);                       /* ax = m * 2^e, m in [0.5, 1) */
    int q = e - 11;
    if (q < -24)
        q = -24;
    double r = rint(ldexp(ax, -q));      /* exact scaling; rint rounds ties to even */
    return copysign(ldexp(r, q), x);
}

typedef struct {
    int layout_a;
    int64_t M, N, K;
    const uint16_t *A;
    int64_t lda;
    const double *Bd;        /* decoded logical B, K x N row-major */
    const double *biasd;     /* decoded bias or NULL */
    int act;
    const int64_t *rows;     /* rows to evaluate (NULL = 0..M-1) */
    int64_t nrows;
    double *out;
    int64_t ldo;
    int nthreads, tid;
} job_t;

static double a_elem(const job_t *J, int64_t i, int64_t k)
{
    uint16_t h = J->layout_a == OR_ROW ? J->A[i * J->lda + k] : J->A[k * J->lda + i];
    return oracle_f16_to_f64(h);
}

/* One output row: the i-k-j loop, k ascending, then bias, then activation. */
static void row_worker(const job_t *J, int64_t r, double *acc)
{
    int64_t i = J->rows ? J->rows[r] : r;
    for (int64_t j = 0; j < J->N; ++j)
        acc[j] = 0.0;
    for (int64_t k = 0; k < J->K; ++k) {
        double a = a_elem(J, i, k);
        const double *brow = J->Bd + k * J->N;
        for (int64_t j = 0; j < J->N; ++j)
            acc[j] = acc[j] + a * brow[j];
    }
    double *o = J->out + r * J->ldo;
    for (int64_t j = 0; j < J->N; ++j) {
        double pre = acc[j] + (J->biasd ? J->biasd[j] : 0.0);
        o[j] = (J->act == OR_ACT_RELU) ? (pre > 0.0 ? pre : 0.0) : pre;
    }
}

static void *thread_main(void *arg)
{
    job_t *J = (job_t *)arg;
    double *acc = (double *)malloc((size_t)(J->N > 0 ? J->N : 1) * sizeof(double));
    if (!acc)
        return (void *)1;
    for (int64_t r = J->tid; r < J->nrows; r += J->nthreads)
        row_worker(J, r, acc);
    free(acc);
    return NULL;
}

/*
 * Evaluate out for the listed rows (rows == NULL: every row 0..M-1, nrows
 * must equal M).  out has nrows rows of stride ldo.  Returns 0 on success,
 * 1 on bad arguments, 2 on allocation or thread failure.
 */
int oracle_gemm_bias_act_rows_f64(int layout_a, int layout_b,
                                  int64_t M, int64_t N, int64_t K,
                                  const uint16_t *A, int64_t lda,
                                  const uint16_t *B, int64_t ldb,
                                  const uint16_t *bias, int act,
                                  const int64_t *rows, int64_t nrows,
                                  double *out, int64_t ldo, int nthreads)
{
    if (M < 0 || N < 0 || K < 0 || nrows < 0 || ldo < N)
        return 1;
    if ((layout_a != OR_ROW && layout_a != OR_COL) || (layout_b != OR_ROW && layout_b != OR_COL))
        return 1;
    if (act != OR_ACT_NONE && act != OR_ACT_RELU)
        return 1;
    if (M > 0 && K > 0 && lda < (layout_a == OR_ROW ? K : M))
        return 1;
    if (N > 0 && K > 0 && ldb < (layout_b == OR_ROW ? N : K))
        return 1;
    if (!rows && nrows != M)
        return 1;
    for (int64_t r = 0; rows && r < nrows; ++r)
        if (rows[r] < 0 || rows[r] >= M)
            return 1;
    if (nrows == 0 || N == 0)
        return 0;
    if (nthreads < 1)
        nthreads = 1;

    /* fp64 copy of the logical K x N matrix B, and of the bias. */
    double *Bd = (double *)malloc((size_t)(K > 0 ? K : 1) * (size_t)N * sizeof(double));
    double *biasd = bias ? (double *)malloc((size_t)N * sizeof(double)) : NULL;
    if (!Bd || (bias && !biasd)) {
        free(Bd);
        free(biasd);
        return 2;
    }
    for (int64_t k = 0; k < K; ++k)
        for (int64_t j = 0; j < N; ++j) {
            uint16_t h = layout_b == OR_ROW ? B[k * ldb + j] : B[j * ldb + k];
            Bd[k * N + j] = oracle_f16_to_f64(h);
        }
    for (int64_t j = 0; bias && j < N; ++j)
        biasd[j] = oracle_f16_to_f64(bias[j]);

    if (nthreads > nrows)
        nthreads = (int)nrows;
    job_t *jobs = (job_t *)calloc((size_t)nthreads, sizeof(job_t));
    pthread_t *th = (pthread_t *)calloc((size_t)nthreads, sizeof(pthread_t));
    int rc = 0;
    if (!jobs || !th) {
        rc = 2;
        goto done;
    }
    for (int t = 0; t < nthreads; ++t) {
        job_t J = {layout_a, M, N, K, A, lda, Bd, biasd, act, rows, nrows, out, ldo, nthreads, t};
        jobs[t] = J;
    }
    int started = 0;
    for (int t = 1; t < nthreads; ++t) {
        if (pthread_create(&th[t], NULL, thread_main, &jobs[t]) != 0) {
            rc = 2;
            break;
        }
        started = t;
    }
    if (thread_main(&jobs[0]) != NULL)
        rc = 2;
    for (int t = 1; t <= started; ++t) {
        void *ret = NULL;
        pthread_join(th[t], &ret);
        if (ret != NULL)
            rc = 2;
    }
done:
    free(jobs);
    free(th);
    free(Bd);
    free(biasd);
    return rc;
}

/* Every row: out is M x N with stride ldo. */
int oracle_gemm_bias_act_f64(int layout_a, int layout_b,
                             int64_t M, int64_t N, int64_t K,
                             const uint16_t *A, int64_t lda,
                             const uint16_t *B, int64_t ldb,
                             const uint16_t *bias, int act,
                             double *out, int64_t ldo, int nthreads)
{
    return oracle_gemm_bias_act_rows_f64(layout_a, layout_b, M, N, K, A, lda, B, ldb, bias, act,
                                         NULL, M, out, ldo, nthreads);
}

/*
 * Oracle for the other idioms of the paper's scope (Introduction: matmul
 * with a pointwise prologue, with a pointwise epilogue, and matmuls of the
 * same output shape feeding a pointwise op; pointwise ops add, subtract,
 * ReLU, Sigmoid, Tanh):
 *   - prologue (Listing 4): the product uses relu(X(i,k)) for its left
 *     operand X; here it is applied to the left operand of every product;
 *   - a second product (Listing 5, Sum of Matmuls): R = P.Q with its own
 *     reduction length K2 (the two products need only agree in output
 *     shape), combined with C = A.B by add or subtract;
 *   - a bias of shape N (broadcast over rows) or M x N, added or subtracted;
 *   - activation none, ReLU, Sigmoid or Tanh.
 * For 0<=i<M, 0<=j<N, in binary64 with k ascending:
 *
 *     C(i,j)   = sum_{k<K}  pro(A(i,k)) * B(k,j)
 *     R(i,j)   = sum_{k<K2} pro(P(i,k)) * Q(k,j)          (second != 0)
 *     Z(i,j)   = second > 0 ? C + R : second < 0 ? C - R : C
 *     pre(i,j) = bias_sign > 0 ? Z + bias(i,j) : Z - bias(i,j)
 *     out(i,j) = act(pre)
 *
 * pro(x) = pro_relu ? (x > 0 ? x : 0) : x.  bias(i,j) = bias[j] for
 * bias_kind 1, bias[i*ldbias + j] for bias_kind 2; bias_kind 0 means no
 * bias term.  act: 0 identity, 1 ReLU (x > 0 ? x : 0), 2 Sigmoid
 * 1 / (1 + exp(-x)), 3 Tanh (the C library's tanh).  P and Q are stored in
 * the layouts of A and B.
 */
enum { OR_ACT_SIGMOID = 2, OR_ACT_TANH = 3 };
enum { OR_BIAS_NONE = 0, OR_BIAS_ROW = 1, OR_BIAS_FULL = 2 };

typedef struct {
    int layout_a;
    int64_t N, K, K2;
    const uint16_t *A, *P;
    int64_t lda, ldp;
    const double *Bd, *Qd;    /* decoded logical B (K x N) and Q (K2 x N), row-major */
    int pro_relu, second, acc16;
    int bias_kind, bias_sign;
    const uint16_t *bias;
    int64_t ldbias;
    int act;
    const int64_t *rows;
    int64_t nrows;
    double *out;
    int64_t ldo;
    int nthreads, tid;
} fjob_t;

/* Left operand element X(i,k) of a product, after the prologue. */
static double left_elem(int layout, const uint16_t *X, int64_t ld, int64_t i, int64_t k, int pro_relu)
{
    double v = oracle_f16_to_f64(layout == OR_ROW ? X[i * ld + k] : X[k * ld + i]);
    if (pro_relu)
        v = v > 0.0 ? v : 0.0;
    return v;
}

static double activation(int act, double x)
{
    switch (act) {
    case OR_ACT_RELU: return x > 0.0 ? x : 0.0;
    case OR_ACT_SIGMOID: return 1.0 / (1.0 + exp(-x));
    case OR_ACT_TANH: return tanh(x);
    default: return x;
    }
}

/* sum_{k<K} pro(X(i,k)) * Yd[k][j] into s[0..N-1], k ascending. */
static void product_row(const fjob_t *J, const uint16_t *X, int64_t ldx, const double *Yd, int64_t K,
                        int64_t i, double *s)
{
    for (int64_t j = 0; j < J->N; ++j)
        s[j] = 0.0;
    for (int64_t k = 0; k < K; ++k) {
        double x = left_elem(J->layout_a, X, ldx, i, k, J->pro_relu);
        const double *yrow = Yd + k * J->N;
        for (int64_t j = 0; j < J->N; ++j)
            s[j] = s[j] + x * yrow[j];
    }
}

/*
 * fp16 accumulation (the reading of the fp16-accumulation mode): one running
 * sum per output, rounded to binary16 at the end of every aligned group of
 * 32 reduction indices of a product (k = 32c .. 32c+31, the last group
 * possibly partial); inside a group the products are summed exactly enough
 * (binary64) that only the group-end rounding matters.  sign = +1 adds the
 * product's terms, -1 subtracts them; s carries the running sum in and out.
 */
static void product_row_acc16(const fjob_t *J, const uint16_t *X, int64_t ldx, const double *Yd,
                              int64_t K, int64_t i, double *s, double sign)
{
    for (int64_t k = 0; k < K; ++k) {
        double x = sign * left_elem(J->layout_a, X, ldx, i, k, J->pro_relu);
        const double *yrow = Yd + k * J->N;
        for (int64_t j = 0; j < J->N; ++j)
            s[j] = s[j] + x * yrow[j];
        if (k % 32 == 31 || k == K - 1)
            for (int64_t j = 0; j < J->N; ++j)
                s[j] = oracle_round_f16(s[j]);
    }
}

static void *fused_thread(void *arg)
{
    fjob_t *J = (fjob_t *)arg;
    size_t n = (size_t)(J->N > 0 ? J->N : 1);
    double *c = (double *)malloc(n * sizeof(double));
    double *r = (double *)malloc(n * sizeof(double));
    if (!c || !r) {
        free(c);
        free(r);
        return (void *)1;
    }
    for (int64_t q = J->tid; q < J->nrows; q += J->nthreads) {
        int64_t i = J->rows ? J->rows[q] : q;
        if (J->acc16) {
            /* one running sum over both products; R is then already in c */
            for (int64_t j = 0; j < J->N; ++j) {
                c[j] = 0.0;
                r[j] = 0.0;
            }
            product_row_acc16(J, J->A, J->lda, J->Bd, J->K, i, c, 1.0);
            if (J->second != 0)
                product_row_acc16(J, J->P, J->ldp, J->Qd, J->K2, i, c, J->second > 0 ? 1.0 : -1.0);
        } else {
            product_row(J, J->A, J->lda, J->Bd, J->K, i, c);
            if (J->second != 0)
                product_row(J, J->P, J->ldp, J->Qd, J->K2, i, r);
        }
        double *o = J->out + q * J->ldo;
        for (int64_t j = 0; j < J->N; ++j) {
            double z = J->acc16 ? c[j] : (J->second > 0 ? c[j] + r[j] : (J->second < 0 ? c[j] - r[j] : c[j]));
            double pre = z;
            if (J->bias_kind != OR_BIAS_NONE) {
                double b = oracle_f16_to_f64(J->bias_kind == OR_BIAS_ROW ? J->bias[j]
                                                                         : J->bias[i * J->ldbias + j]);
                pre = J->bias_sign > 0 ? z + b : z - b;
            }
            o[j] = activation(J->act, pre);
        }
    }
    free(c);
    free(r);
    return NULL;
}

static double *decode_right(int layout_b, int64_t K, int64_t N, const uint16_t *B, int64_t ldb)
{
    double *d = (double *)malloc((size_t)(K > 0 ? K : 1) * (size_t)(N > 0 ? N : 1) * sizeof(double));
    if (!d)
        return NULL;
    for (int64_t k = 0; k < K; ++k)
        for (int64_t j = 0; j < N; ++j)
            d[k * N + j] = oracle_f16_to_f64(layout_b == OR_ROW ? B[k * ldb + j] : B[j * ldb + k]);
    return d;
}

/*
 * second: 0 one product, +1 add R, -1 subtract R.  bias_sign: +1 add,
 * -1 subtract.  acc16: 0 binary64 sums (the definition), 1 the fp16
 * accumulation described above product_row_acc16.  rows == NULL: every row
 * (nrows must equal M).  Returns 0 on success, 1 on bad arguments, 2 on
 * allocation or thread failure.
 */
int oracle_fused_rows_f64(int layout_a, int layout_b, int64_t M, int64_t N, int64_t K,
                          const uint16_t *A, int64_t lda, const uint16_t *B, int64_t ldb,
                          int pro_relu, int second, int64_t K2, const uint16_t *P, int64_t ldp,
                          const uint16_t *Q, int64_t ldq, int bias_kind, int bias_sign,
                          const uint16_t *bias, int64_t ldbias, int act, int acc16,
                          const int64_t *rows, int64_t nrows, double *out, int64_t ldo, int nthreads)
{
    if (M < 0 || N < 0 || K < 0 || nrows < 0 || ldo < N)
        return 1;
    if ((layout_a != OR_ROW && layout_a != OR_COL) || (layout_b != OR_ROW && layout_b != OR_COL))
        return 1;
    if (act < OR_ACT_NONE || act > OR_ACT_TANH || bias_kind < OR_BIAS_NONE || bias_kind > OR_BIAS_FULL)
        return 1;
    if (second < -1 || second > 1 || (bias_sign != 1 && bias_sign != -1) || (acc16 != 0 && acc16 != 1))
        return 1;
    if ((bias_kind != OR_BIAS_NONE && !bias) || (bias_kind == OR_BIAS_FULL && ldbias < N))
        return 1;
    if (M > 0 && K > 0 && (!A || lda < (layout_a == OR_ROW ? K : M)))
        return 1;
    if (N > 0 && K > 0 && (!B || ldb < (layout_b == OR_ROW ? N : K)))
        return 1;
    if (second != 0) {
        if (K2 < 0)
            return 1;
        if (M > 0 && K2 > 0 && (!P || ldp < (layout_a == OR_ROW ? K2 : M)))
            return 1;
        if (N > 0 && K2 > 0 && (!Q || ldq < (layout_b == OR_ROW ? N : K2)))
            return 1;
    } else {
        K2 = 0;
    }
    if (!rows && nrows != M)
        return 1;
    for (int64_t q = 0; rows && q < nrows; ++q)
        if (rows[q] < 0 || rows[q] >= M)
            return 1;
    if (nrows == 0 || N == 0)
        return 0;
    if (nthreads < 1)
        nthreads = 1;
    if (nthreads > nrows)
        nthreads = (int)nrows;

    double *Bd = decode_right(layout_b, K, N, B, ldb);
    double *Qd = second != 0 ? decode_right(layout_b, K2, N, Q, ldq) : NULL;
    fjob_t *jobs = (fjob_t *)calloc((size_t)nthreads, sizeof(fjob_t));
    pthread_t *th = (pthread_t *)calloc((size_t)nthreads, sizeof(pthread_t));
    int rc = 0;
    if (!Bd || (second != 0 && !Qd) || !jobs || !th) {
        rc = 2;
        goto done;
    }
    for (int t = 0; t < nthreads; ++t) {
        fjob_t J = {layout_a, N, K, K2, A, P, lda, ldp, Bd, Qd, pro_relu, second, acc16, bias_kind,
                    bias_sign, bias, ldbias, act, rows, nrows, out, ldo, nthreads, t};
        jobs[t] = J;
    }
    int started = 0;
    for (int t = 1; t < nthreads; ++t) {
        if (pthread_create(&th[t], NULL, fused_thread, &jobs[t]) != 0) {
            rc = 2;
            break;
        }
        started = t;
    }
    if (fused_thread(&jobs[0]) != NULL)
        rc = 2;
    for (int t = 1; t <= started; ++t) {
        void *ret = NULL;
        pthread_join(th[t], &ret);
        if (ret != NULL)
            rc = 2;
    }
done:
    free(jobs);
    free(th);
    free(Bd);
    free(Qd);
    return rc;
}
