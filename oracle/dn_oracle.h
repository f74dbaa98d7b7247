/*
 * dn_oracle.h -- fp64 CPU oracle for deferred normalization (arXiv 2502.17728).
 * TEST INFRASTRUCTURE ONLY: used by the tests, the smoke check and the
 * benchmark's CPU-baseline leg, never by the product path.
 *
 * All arrays are host fp64, row-major, contiguous, owned by the caller.
 * Functions return 0 on success, -1 on a NULL required pointer or a size < 1.
 * nthreads < 1 means 1.
 */
#ifndef DN_ORACLE_H
#define DN_ORACLE_H
#include <stdint.h>
#ifdef __cplusplus
extern "C" {
#endif

/* Eq. (1)-(2): y[M][K] = LayerNorm(x) * gamma + beta (beta may be NULL). */
int oracle_layernorm(const double* x, const double* gamma, const double* beta,
                     int64_t M, int64_t K, double eps, double* y, int nthreads);

/* Eq. (4) product: out[b][M][N] = a[b][M][K] . W[b][K][N] + bias[N] (bias may be NULL). */
int oracle_linear(const double* a, const double* W, const double* bias,
                  int64_t batch, int64_t M, int64_t K, int64_t N, double* out,
                  int nthreads);

/* Eq. (4): out[M][N] = LayerNorm(x[M][K]) . W[K][N] + bias[N]. */
int oracle_ln_linear(const double* x, const double* gamma, const double* beta,
                     const double* W, const double* bias, int64_t M, int64_t K,
                     int64_t N, double eps, double* out, int nthreads);

/* Eq. (6): y[M][K] = x / sqrt(mean(x^2) + eps) * gamma + beta (beta may be NULL;
   eps = 0 is the printed form). */
int oracle_rmsnorm(const double* x, const double* gamma, const double* beta,
                   int64_t M, int64_t K, double eps, double* y, int nthreads);

/* out[M][N] = RMSNorm(x[M][K]) . W[K][N] + bias[N]. */
int oracle_rms_linear(const double* x, const double* gamma, const double* beta,
                      const double* W, const double* bias, int64_t M, int64_t K,
                      int64_t N, double eps, double* out, int nthreads);

/* Llama MLP input stage (the subsubsection on RMSNorm in Llama models):
   y = RMSNorm(x[M][K]) (Eq. (6)), h[M][N] = SiLU(y . Wg) * (y . Wu) element-wise,
   SiLU(z) = z / (1 + exp(-z)); Wg, Wu are [K][N]. */
int oracle_rms_swiglu(const double* x, const double* gamma, const double* Wg,
                      const double* Wu, int64_t M, int64_t K, int64_t N, double eps,
                      double* h, int nthreads);

/* Eq. (7) softmax of R rows of length Lk.  qpos[r] >= 0 keeps keys j <= qpos[r]
   (causal) and writes 0 beyond; qpos NULL or qpos[r] < 0 keeps every key. */
int oracle_softmax(const double* S, const int64_t* qpos, int64_t R, int64_t Lk,
                   double* P, int nthreads);

/* Eq. (7): out[R][d] = softmax(S[R][Lk]) . V[head[r]][Lk][d]
   (head NULL means head 0 for every row; qpos as for oracle_softmax). */
int oracle_softmax_pv(const double* S, const double* V, const int64_t* head,
                      const int64_t* qpos, int64_t R, int64_t Lk, int64_t d,
                      double* out, int nthreads);

/* Attention: out[R][d] = softmax(scale * Q[r] . K[head[r]]^T) . V[head[r]] with
   Q[R][d] (one query row per r), K, V[H][Lk][d]; head and qpos as for
   oracle_softmax_pv (qpos[r] >= 0: keys j <= qpos[r] only). */
int oracle_attention(const double* Q, const double* K, const double* V, const int64_t* head,
                     const int64_t* qpos, int64_t R, int64_t Lk, int64_t d, double scale,
                     double* out, int nthreads);

#ifdef __cplusplus
}
#endif
#endif
