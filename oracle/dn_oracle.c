/*
 * dn_oracle.c -- fp64 CPU oracle for deferred normalization.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, obviously correct
 * definition that the GPU path is checked against.  Only the test suite, the
 * package smoke check and the benchmark's CPU-baseline leg may load it; the
 * product path never does.  It shares no code, header, table or helper with
 * the HIP library.
 *
 * Paper: "LLM Inference Acceleration via Efficient Operation Fusion"
 * (Salmani & Soloveychik, arXiv 2502.17728).
 *
 * What is computed (the conventional, un-fused sub-graphs; the fused forms of
 * the paper are algebraically equal to these, Sec. II):
 *   - LayerNorm statistics, Eq. (1): mean and the biased (1/n) variance.
 *   - LayerNorm output,     Eq. (2): y = (x - mean)/sqrt(var + eps) * gamma + beta.
 *   - Linear layer,         Eq. (4): out = y F (+ bias), F stored as W[K][N].
 *   - RMSNorm,              Eq. (6): y = x / sqrt(x x^T / n + eps) * gamma (+ beta),
 *                           and RMSNorm followed by the linear layer.
 *   - The Llama MLP input stage that the same subsubsection fuses: RMSNorm,
 *     the gate and up projections, and h = SiLU(y Wg) * (y Wu) with
 *     SiLU(z) = z / (1 + exp(-z)).
 *   - Attention from Q, K: the scores s_ij = scale * q_i . k_j formed here,
 *     then Eq. (7) on them (the same softmax and value product).
 *   - Softmax then values,  Eq. (7) with the footnote's max subtraction:
 *       m = max_j x_j, e_j = exp(x_j - m), y_j = e_j / sum_i e_i, out = y V.
 *
 * Arithmetic is IEEE fp64 throughout, summation in natural index order, no
 * blocking, no reordering.  Rows are independent; a row range is handed to
 * each POSIX thread, which changes no arithmetic.
 *
 * Readings where the paper is silent (listed with the rest in the design notes):
 *   - eps is an argument (Eq. (2) names it without a value) and sits inside
 *     the square root as printed.
 *   - The variance is the biased one of Eq. (1): divide by n, two passes.
 *   - RMSNorm (Eq. (6)) prints no eps; it is an argument here, inside the
 *     root like LayerNorm's, and eps = 0 is the printed form.  Eq. (6) has no
 *     shift; an optional beta is added after gamma, as for LayerNorm.
 *   - Causal masking keeps key j for query i iff j <= i.  Keys outside the
 *     mask are ignored, not read as values.
 *   - A row whose kept scores are all -inf yields NaN (0/0), as the plain
 *     definition does.
 *
 * Error behaviour: every entry point returns 0 on success and -1 on a
 * NULL pointer or a non-positive size; it never allocates device memory and
 * holds no global state.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include "dn_oracle.h"

/* ------------------------------------------------------------------------ */
/* Row-parallel driver: splits [0, rows) into contiguous ranges.             */

typedef void (*row_fn)(void* ctx, int64_t r0, int64_t r1);

typedef struct {
    row_fn fn;
    void* ctx;
    int64_t r0, r1;
} row_job;

static void* row_job_main(void* p) {
    row_job* j = (row_job*)p;
    j->fn(j->ctx, j->r0, j->r1);
    return NULL;
}

static void run_rows(row_fn fn, void* ctx, int64_t rows, int nthreads) {
    if (nthreads < 1) nthreads = 1;
    if ((int64_t)nthreads > rows) nthreads = (int)rows;
    if (nthreads <= 1) {
        fn(ctx, 0, rows);
        return;
    }
    pthread_t* tid = (pthread_t*)calloc((size_t)nthreads, sizeof(pthread_t));
    row_job* jobs = (row_job*)calloc((size_t)nthreads, sizeof(row_job));
    int* started = (int*)calloc((size_t)nthreads, sizeof(int));
    int64_t per = rows / nthreads, extra = rows % nthreads, r = 0;
    for (int t = 0; t < nthreads; ++t) {
        int64_t n = per + (t < extra ? 1 : 0);
        jobs[t].fn = fn;
        jobs[t].ctx = ctx;
        jobs[t].r0 = r;
        jobs[t].r1 = r + n;
        r += n;
        started[t] = pthread_create(&tid[t], NULL, row_job_main, &jobs[t]) == 0;
        if (!started[t]) fn(ctx, jobs[t].r0, jobs[t].r1); /* run inline */
    }
    for (int t = 0; t < nthreads; ++t)
        if (started[t]) pthread_join(tid[t], NULL);
    free(started);
    free(jobs);
    free(tid);
}

/* ------------------------------------------------------------------------ */
/* LayerNorm, Eq. (1) and Eq. (2), one row.                                  */

static void layernorm_row(const double* x, int64_t K, const double* gamma,
                          const double* beta, double eps, double* y) {
    /* Eq. (1): mean */
    double sum = 0.0;
    for (int64_t k = 0; k < K; ++k) sum += x[k];
    double mean = sum / (double)K;
    /* Eq. (1): variance, (x - mean 1)(x - mean 1)^T / n */
    double ss = 0.0;
    for (int64_t k = 0; k < K; ++k) {
        double d = x[k] - mean;
        ss += d * d;
    }
    double var = ss / (double)K;
    /* Eq. (2): normalize, then the affine gamma, beta */
    double denom = sqrt(var + eps);
    for (int64_t k = 0; k < K; ++k) {
        double v = (x[k] - mean) / denom * gamma[k];
        y[k] = beta ? v + beta[k] : v;
    }
}

typedef struct {
    const double *x, *gamma, *beta;
    int64_t K;
    double eps;
    double* y;
} ln_ctx;

static void ln_rows(void* p, int64_t r0, int64_t r1) {
    ln_ctx* c = (ln_ctx*)p;
    for (int64_t m = r0; m < r1; ++m)
        layernorm_row(c->x + m * c->K, c->K, c->gamma, c->beta, c->eps, c->y + m * c->K);
}

int oracle_layernorm(const double* x, const double* gamma, const double* beta,
                     int64_t M, int64_t K, double eps, double* y, int nthreads) {
    if (!x || !gamma || !y || M < 1 || K < 1) return -1;
    ln_ctx c = {x, gamma, beta, K, eps, y};
    run_rows(ln_rows, &c, M, nthreads);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Linear layer, the product y F of Eq. (4), one row.                        */
/* out[n] = bias[n] + sum_k y[k] W[k][n], k ascending for every n.           */

static void linear_row(const double* y, const double* W, const double* bias,
                       int64_t K, int64_t N, double* out) {
    for (int64_t n = 0; n < N; ++n) out[n] = 0.0;
    for (int64_t k = 0; k < K; ++k) {
        const double yk = y[k];
        const double* wk = W + k * N;
        for (int64_t n = 0; n < N; ++n) out[n] += yk * wk[n];
    }
    if (bias)
        for (int64_t n = 0; n < N; ++n) out[n] += bias[n];
}

typedef struct {
    const double *a, *W, *bias;
    int64_t M, K, N;
    double* out;
} lin_ctx;

/* Rows of the batched product are numbered b*M + m; batch b uses W + b*K*N. */
static void lin_rows(void* p, int64_t r0, int64_t r1) {
    lin_ctx* c = (lin_ctx*)p;
    for (int64_t r = r0; r < r1; ++r) {
        int64_t b = r / c->M;
        linear_row(c->a + r * c->K, c->W + b * c->K * c->N, c->bias, c->K, c->N,
                   c->out + r * c->N);
    }
}

int oracle_linear(const double* a, const double* W, const double* bias,
                  int64_t batch, int64_t M, int64_t K, int64_t N, double* out,
                  int nthreads) {
    if (!a || !W || !out || batch < 1 || M < 1 || K < 1 || N < 1) return -1;
    lin_ctx c = {a, W, bias, M, K, N, out};
    run_rows(lin_rows, &c, batch * M, nthreads);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Conventional LayerNorm followed by the linear layer, Eq. (4).             */

typedef struct {
    const double *x, *gamma, *beta, *W, *bias;
    int64_t K, N;
    double eps;
    double* out;
} lnlin_ctx;

static void lnlin_rows(void* p, int64_t r0, int64_t r1) {
    lnlin_ctx* c = (lnlin_ctx*)p;
    double* y = (double*)malloc((size_t)c->K * sizeof(double));
    if (!y) return;
    for (int64_t m = r0; m < r1; ++m) {
        layernorm_row(c->x + m * c->K, c->K, c->gamma, c->beta, c->eps, y);
        linear_row(y, c->W, c->bias, c->K, c->N, c->out + m * c->N);
    }
    free(y);
}

int oracle_ln_linear(const double* x, const double* gamma, const double* beta,
                     const double* W, const double* bias, int64_t M, int64_t K,
                     int64_t N, double eps, double* out, int nthreads) {
    if (!x || !gamma || !W || !out || M < 1 || K < 1 || N < 1) return -1;
    lnlin_ctx c = {x, gamma, beta, W, bias, K, N, eps, out};
    run_rows(lnlin_rows, &c, M, nthreads);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* RMSNorm, Eq. (6), one row: the root mean square replaces the standard     */
/* deviation and no mean is subtracted.                                      */

static void rmsnorm_row(const double* x, int64_t K, const double* gamma,
                        const double* beta, double eps, double* y) {
    double ss = 0.0;
    for (int64_t k = 0; k < K; ++k) ss += x[k] * x[k];
    double denom = sqrt(ss / (double)K + eps);
    for (int64_t k = 0; k < K; ++k) {
        double v = x[k] / denom * gamma[k];
        y[k] = beta ? v + beta[k] : v;
    }
}

static void rms_rows(void* p, int64_t r0, int64_t r1) {
    ln_ctx* c = (ln_ctx*)p;
    for (int64_t m = r0; m < r1; ++m)
        rmsnorm_row(c->x + m * c->K, c->K, c->gamma, c->beta, c->eps, c->y + m * c->K);
}

int oracle_rmsnorm(const double* x, const double* gamma, const double* beta,
                   int64_t M, int64_t K, double eps, double* y, int nthreads) {
    if (!x || !gamma || !y || M < 1 || K < 1) return -1;
    ln_ctx c = {x, gamma, beta, K, eps, y};
    run_rows(rms_rows, &c, M, nthreads);
    return 0;
}

/* RMSNorm followed by the linear layer: the product of Eq. (4) on Eq. (6)'s y. */
static void rmslin_rows(void* p, int64_t r0, int64_t r1) {
    lnlin_ctx* c = (lnlin_ctx*)p;
    double* y = (double*)malloc((size_t)c->K * sizeof(double));
    if (!y) return;
    for (int64_t m = r0; m < r1; ++m) {
        rmsnorm_row(c->x + m * c->K, c->K, c->gamma, c->beta, c->eps, y);
        linear_row(y, c->W, c->bias, c->K, c->N, c->out + m * c->N);
    }
    free(y);
}

int oracle_rms_linear(const double* x, const double* gamma, const double* beta,
                      const double* W, const double* bias, int64_t M, int64_t K,
                      int64_t N, double eps, double* out, int nthreads) {
    if (!x || !gamma || !W || !out || M < 1 || K < 1 || N < 1) return -1;
    lnlin_ctx c = {x, gamma, beta, W, bias, K, N, eps, out};
    run_rows(rmslin_rows, &c, M, nthreads);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* RMSNorm, then the gated MLP input stage of a Llama block: the gate and up */
/* projections of y, combined as SiLU(gate) * up (element-wise).             */

static double silu(double z) { return z / (1.0 + exp(-z)); }

typedef struct {
    const double *x, *gamma, *Wg, *Wu;
    int64_t K, N;
    double eps;
    double* h;
} swiglu_ctx;

static void swiglu_rows(void* p, int64_t r0, int64_t r1) {
    swiglu_ctx* c = (swiglu_ctx*)p;
    double* y = (double*)malloc((size_t)c->K * sizeof(double));
    double* g = (double*)malloc((size_t)c->N * sizeof(double));
    double* u = (double*)malloc((size_t)c->N * sizeof(double));
    if (y && g && u) {
        for (int64_t m = r0; m < r1; ++m) {
            rmsnorm_row(c->x + m * c->K, c->K, c->gamma, NULL, c->eps, y);
            linear_row(y, c->Wg, NULL, c->K, c->N, g);
            linear_row(y, c->Wu, NULL, c->K, c->N, u);
            double* h = c->h + m * c->N;
            for (int64_t n = 0; n < c->N; ++n) h[n] = silu(g[n]) * u[n];
        }
    }
    free(u);
    free(g);
    free(y);
}

int oracle_rms_swiglu(const double* x, const double* gamma, const double* Wg,
                      const double* Wu, int64_t M, int64_t K, int64_t N, double eps,
                      double* h, int nthreads) {
    if (!x || !gamma || !Wg || !Wu || !h || M < 1 || K < 1 || N < 1) return -1;
    swiglu_ctx c = {x, gamma, Wg, Wu, K, N, eps, h};
    run_rows(swiglu_rows, &c, M, nthreads);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Softmax, Eq. (7) with the footnote's maximum subtraction, one row.        */
/* Keys kept: all of them, or j <= qpos when qpos >= 0 (causal).             */

static int64_t kept_keys(int64_t Lk, int64_t qpos) {
    if (qpos < 0) return Lk;
    return qpos + 1 < Lk ? qpos + 1 : Lk;
}

static void softmax_row(const double* s, int64_t Lk, int64_t qpos, double* p) {
    int64_t J = kept_keys(Lk, qpos);
    double m = -INFINITY;
    for (int64_t j = 0; j < J; ++j) {
        if (isnan(s[j])) { /* a NaN score makes the whole row NaN */
            m = s[j];
            break;
        }
        if (s[j] > m) m = s[j];
    }
    double l = 0.0;
    for (int64_t j = 0; j < J; ++j) {
        p[j] = exp(s[j] - m);
        l += p[j];
    }
    for (int64_t j = 0; j < J; ++j) p[j] = p[j] / l;
    for (int64_t j = J; j < Lk; ++j) p[j] = 0.0;
}

typedef struct {
    const double* S;
    const int64_t* qpos;
    int64_t Lk;
    double* P;
} sm_ctx;

static void sm_rows(void* p, int64_t r0, int64_t r1) {
    sm_ctx* c = (sm_ctx*)p;
    for (int64_t r = r0; r < r1; ++r)
        softmax_row(c->S + r * c->Lk, c->Lk, c->qpos ? c->qpos[r] : -1, c->P + r * c->Lk);
}

int oracle_softmax(const double* S, const int64_t* qpos, int64_t R, int64_t Lk,
                   double* P, int nthreads) {
    if (!S || !P || R < 1 || Lk < 1) return -1;
    sm_ctx c = {S, qpos, Lk, P};
    run_rows(sm_rows, &c, R, nthreads);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Conventional Softmax followed by the values, Eq. (7).                     */
/* Row r uses the value matrix V[head[r]] of shape [Lk][d].                  */

typedef struct {
    const double *S, *V;
    const int64_t *head, *qpos;
    int64_t Lk, d;
    double* out;
} smpv_ctx;

static void smpv_rows(void* p, int64_t r0, int64_t r1) {
    smpv_ctx* c = (smpv_ctx*)p;
    double* prob = (double*)malloc((size_t)c->Lk * sizeof(double));
    if (!prob) return;
    for (int64_t r = r0; r < r1; ++r) {
        int64_t q = c->qpos ? c->qpos[r] : -1;
        softmax_row(c->S + r * c->Lk, c->Lk, q, prob);
        const double* V = c->V + (c->head ? c->head[r] : 0) * c->Lk * c->d;
        double* o = c->out + r * c->d;
        for (int64_t t = 0; t < c->d; ++t) o[t] = 0.0;
        int64_t J = kept_keys(c->Lk, q);
        for (int64_t j = 0; j < J; ++j)
            for (int64_t t = 0; t < c->d; ++t) o[t] += prob[j] * V[j * c->d + t];
    }
    free(prob);
}

int oracle_softmax_pv(const double* S, const double* V, const int64_t* head,
                      const int64_t* qpos, int64_t R, int64_t Lk, int64_t d,
                      double* out, int nthreads) {
    if (!S || !V || !out || R < 1 || Lk < 1 || d < 1) return -1;
    smpv_ctx c = {S, V, head, qpos, Lk, d, out};
    run_rows(smpv_rows, &c, R, nthreads);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Attention: the scores of row r against head h's keys, scale * q . k_j,    */
/* then the softmax and value product of Eq. (7).                            */

typedef struct {
    const double *Q, *K, *V;
    const int64_t *head, *qpos;
    int64_t Lk, d;
    double scale;
    double* out;
} attn_ctx;

static void attn_rows(void* p, int64_t r0, int64_t r1) {
    attn_ctx* c = (attn_ctx*)p;
    double* s = (double*)malloc((size_t)c->Lk * sizeof(double));
    double* prob = (double*)malloc((size_t)c->Lk * sizeof(double));
    if (s && prob) {
        for (int64_t r = r0; r < r1; ++r) {
            const int64_t h = c->head ? c->head[r] : 0;
            const int64_t q = c->qpos ? c->qpos[r] : -1;
            const double* qr = c->Q + r * c->d;
            const double* K = c->K + h * c->Lk * c->d;
            const double* V = c->V + h * c->Lk * c->d;
            const int64_t J = kept_keys(c->Lk, q);
            for (int64_t j = 0; j < c->Lk; ++j) {
                double dot = 0.0;
                if (j < J)
                    for (int64_t t = 0; t < c->d; ++t) dot += qr[t] * K[j * c->d + t];
                s[j] = c->scale * dot;
            }
            softmax_row(s, c->Lk, q, prob);
            double* o = c->out + r * c->d;
            for (int64_t t = 0; t < c->d; ++t) o[t] = 0.0;
            for (int64_t j = 0; j < J; ++j)
                for (int64_t t = 0; t < c->d; ++t) o[t] += prob[j] * V[j * c->d + t];
        }
    }
    free(prob);
    free(s);
}

int oracle_attention(const double* Q, const double* K, const double* V, const int64_t* head,
                     const int64_t* qpos, int64_t R, int64_t Lk, int64_t d, double scale,
                     double* out, int nthreads) {
    if (!Q || !K || !V || !out || R < 1 || Lk < 1 || d < 1) return -1;
    attn_ctx c = {Q, K, V, head, qpos, Lk, d, scale, out};
    run_rows(attn_rows, &c, R, nthreads);
    return 0;
}
