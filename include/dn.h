/*
 * dn.h -- C ABI of the deferred-normalization library (libdn.so), gfx950.
 *
 * Method: "LLM Inference Acceleration via Efficient Operation Fusion"
 * (Salmani & Soloveychik, arXiv 2502.17728).  A LayerNorm or a Softmax that
 * feeds a matrix product is split into an element-wise part, which becomes
 * the product's operand, and a per-row collective part (the LayerNorm
 * mean/variance, the softmax denominator), which is reduced concurrently and
 * applied once after the product (Sec. II, Fig. 1; Eq. (5) and Eq. (8)).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Tensor pointers are DEVICE pointers (hipMalloc'd or equivalent), row-major
 *   and contiguous, 16-byte aligned.  The caller owns all memory; the library
 *   allocates nothing.  Two library-owned device arrays exist on each GPU the
 *   library runs on, held until the process ends: the 1 MiB mailbox in which
 *   the workgroups of one LayerNorm/RMSNorm product exchange their shares of
 *   the row moments (every entry stamped with its call's number, so no call
 *   ever uses another's; see ln_linear_deferred), and the partials array of
 *   attention_decode_deferred_noalloc.  No other state outlives a call.
 * - Every call validates its arguments on the host BEFORE any HIP call; an
 *   invalid call returns a status and enqueues nothing.  A valid call only
 *   enqueues kernels on `stream` (NULL = the default stream) and returns; it
 *   never synchronizes.  Buffers must stay alive until that work completes.
 *   Calls on different streams are independent (reentrant).
 * - Element types: DN_F32 (IEEE fp32) or DN_BF16 (bfloat16).  All accumulation
 *   is fp32; outputs are rounded once, to nearest even, to the input type.
 * - NaN/Inf inputs are not errors: they propagate as in the plain definition.
 * - Sizes are int64 element counts; K and N (and d) must be multiples of 8.
 * - Output ranges must not overlap input ranges (checked: DN_ERR_INVALID_ARG).
 */
#ifndef DN_H
#define DN_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DN_API __attribute__((visibility("default")))

typedef enum { DN_F32 = 0, DN_BF16 = 1 } dn_dtype;

typedef enum {
    DN_OK = 0,
    DN_ERR_INVALID_ARG = 1, /* NULL pointer, size < 1, bad eps, overlap, bad descriptor   */
    DN_ERR_UNSUPPORTED = 2, /* valid request outside what the kernels implement            */
    DN_ERR_MISALIGNED = 3,  /* a tensor pointer is not 16-byte aligned                     */
    DN_ERR_HIP = 4          /* the HIP runtime reported an error when launching            */
} dn_status;

/* Human-readable name of a status code (static string; never NULL). */
DN_API const char* dn_status_string(int status);

/* Library version, (major << 16) | minor. */
DN_API int dn_version(void);

/* ======================================================================= */
/* LayerNorm -> Linear, deferred (Sec. II-A, Eq. (1), (2), (4), (5))        */
/* ======================================================================= */

/*
 * Static weights prepared once (the paper computes the static factors of
 * Eq. (5) "at compile time", Sec. II-A; here once per weight set, off the
 * per-token path).  From W[K][N] (the paper's F, n x m), gamma[K], beta[K]
 * and an optional bias[N], ln_linear_prepare writes into `packed`:
 *   Wt'[N][K] = (Diag(gamma) W)^T  rounded once to `dtype` (K contiguous),
 *   c[N]      = sum_k W'[k][n]     over the ROUNDED W' (fp32),
 *   b[N]      = sum_k beta[k] W[k][n] + bias[n]     (fp32; beta F of Eq. (5)).
 * `packed` must be ln_linear_packed_bytes(K, N, dtype) bytes, 256-byte
 * aligned, device memory; `*w_out` is filled on the host and is what
 * ln_linear_deferred takes.  beta and bias may be NULL (treated as zero).
 * Layout of W'^T in `packed` (version 2): 16-row x 64-byte fragment chunks
 * (16 output features x 32 bf16 or 16 fp32 of K), in chunk order
 * [ceil(N/16)][ceil(K/kchunk)][64 lanes][16 B], zero padded; lane l of a
 * chunk holds feature 16*nb + (l & 15) at K offset kchunk*kc + (l >> 4)*(16 B).
 */
typedef struct {
    int64_t K, N;           /* normalized dim, output features                */
    int32_t dtype;          /* dn_dtype of W' and of x/out                    */
    int32_t layout_version; /* DN_LN_LAYOUT_VERSION when produced by prepare   */
    void* packed;           /* device buffer holding Wt', c, b                */
} ln_linear_weights;

#define DN_LN_LAYOUT_VERSION 2

/* Bytes of the packed buffer for (K, N, dtype); 0 if the request is invalid. */
DN_API size_t ln_linear_packed_bytes(int64_t K, int64_t N, int dtype);

DN_API dn_status ln_linear_prepare(const void* W, const void* gamma, const void* beta,
                            const void* bias, int64_t K, int64_t N, int dtype,
                            void* packed, size_t packed_bytes,
                            ln_linear_weights* w_out, hipStream_t stream);

/*
 * out[M][N] = LayerNorm(x[M][K]) . W + bias, computed the deferred way:
 * the MFMA product acc = x . W' runs on the un-normalized x while the row
 * statistics (sum x, sum x^2) are reduced in the same workgroup, and the
 * epilogue applies  out = rstd * (acc - mean * c) + b  once (Eq. (5) with the
 * centering (I - E/n) applied as  x(I - E/n)W' = xW' - mean 1 W').
 * mean and the biased variance follow Eq. (1); rstd = 1/sqrt(var + eps) as
 * in Eq. (2).  eps must be finite and >= 0.  x and out have w->dtype.
 * On the large-tile kernels (more than 128 rows, K % 64 == 0) the
 * workgroups that share a 256-row block split the reduction of its moments
 * and exchange the sums through the library's mailbox; a workgroup that does
 * not find a peer's sums within 200 us (a peer not resident on a busy GPU)
 * reduces all its rows itself, so the result never depends on scheduling.
 * (DN_MOMENT_WAIT_TICKS in the environment overrides the wait, in 10 ns
 * ticks; 0 makes every workgroup reduce its rows itself.)  A launch recorded
 * under stream capture (a HIP graph) uses no mailbox: each workgroup reduces
 * the moments of its rows alongside its first tile, so every replay of the
 * graph normalizes with its own inputs' statistics.  A row holding
 * NaN or +-inf gives an all-NaN output row; with eps = 0 a row whose fp32
 * one-pass variance is exactly 0 (a constant row whose squares sum exactly)
 * gives NaN, as (x - mean) / 0 does.  |x| >= 2^64 (fp32 overflow of x^2) is
 * outside the supported range.
 */
DN_API dn_status ln_linear_deferred(const void* x, const ln_linear_weights* w, int64_t M,
                             float eps, void* out, hipStream_t stream);

/*
 * out[M][N] = RMSNorm(x[M][K]) . W + bias (Sec. II-A, RMSNorm in Llama
 * models, Eq. (6)), the deferred way: acc = x . W' on the MFMA with the row
 * sum of squares reduced concurrently, then  out = rstd * acc + b  with
 * rstd = 1/sqrt(sum_k x^2 / K + eps).  Eq. (6) subtracts no mean, so c is not
 * used.  Eq. (6) prints no eps: eps is an argument inside the root, finite
 * and >= 0, and eps = 0 is the printed form (an all-zero row then gives NaN).
 * w comes from ln_linear_prepare with the RMSNorm gamma; Eq. (6) has no
 * shift, so pass beta = NULL there (a non-NULL beta adds beta W to every
 * row, as it does for LayerNorm).  Same argument rules, layout, ownership
 * and status codes as ln_linear_deferred.
 */
DN_API dn_status rms_linear_deferred(const void* x, const ln_linear_weights* w, int64_t M,
                              float eps, void* out, hipStream_t stream);

/*
 * Post-LN placement (Sec. II-A: the residual branch taken right after the
 * normalization instead of before it).  There the normalized rows y are needed
 * twice -- as the input of the next linear layer and as the residual -- so the
 * call returns both: out[M][N] = y . W + bias the deferred way (exactly as
 * ln_linear_deferred / rms_linear_deferred, the product never waiting for the
 * statistics), and y[M][K] = (x - mean) rstd gamma + beta (RMS: x rstd gamma)
 * applied afterwards from the statistics the product's kernel reduced, which
 * it exports to stats[2 M] (fp32 (mean, rstd) pairs; RMS: mean = 0).  gamma
 * (and beta, nullable, LayerNorm only) are the [K] vectors that were folded
 * into w, in w->dtype.  stats and y: caller-owned device memory, 16-byte
 * aligned, overlapping no other argument.  Status codes as ln_linear_deferred;
 * DN_ERR_UNSUPPORTED also when y is too large for one launch.
 */
DN_API dn_status ln_linear_deferred_post(const void* x, const ln_linear_weights* w, int64_t M, float eps,
                                  const void* gamma, const void* beta, float* stats, void* y,
                                  void* out, hipStream_t stream);

DN_API dn_status rms_linear_deferred_post(const void* x, const ln_linear_weights* w, int64_t M, float eps,
                                   const void* gamma, float* stats, void* y, void* out,
                                   hipStream_t stream);

/* ----------------------------------------------------------------------- */
/* Ablations of the LayerNorm -> Linear fusion                              */
/* ----------------------------------------------------------------------- */

/*
 * Eq. (5) taken literally: the centering (I - E/n) of Eq. (3) folded into
 * the static weight, W'' = (I - E/n) Diag(gamma) W, i.e. gamma_k W[k][n]
 * minus its column mean (fp64, unrounded), rounded once to dtype; c is set
 * to 0 so ln_linear_deferred computes out = rstd * (x . W'') + b, the
 * epilogue of Eq. (5) with no mean term.  Same arguments, layout and status
 * codes as ln_linear_prepare; the result is used with ln_linear_deferred.
 * Equal to the mean * c epilogue in exact arithmetic; in floating point the
 * rounded W'' columns no longer sum to exactly 0, so rows with a large
 * |mean| / std lose about |mean| / std * 2^-9 of relative accuracy (bf16).
 */
DN_API dn_status ln_linear_prepare_centered(const void* W, const void* gamma, const void* beta,
                                     const void* bias, int64_t K, int64_t N, int dtype,
                                     void* packed, size_t packed_bytes,
                                     ln_linear_weights* w_out, hipStream_t stream);

/*
 * Serial (not concurrent) statistics: a pre-pass kernel computes each row's
 * mean and 1/sqrt(var + eps) (two passes over the row, Eq. (1)-(2)) into
 * stats[2 M] (fp32 pairs; caller-owned device memory, 16-byte aligned, not
 * overlapping x, out or the weights), then the product runs with the same
 * deferred epilogue, reading them instead of reducing the moments
 * concurrently.  It isolates what concurrency buys over a stats pre-pass.
 * K must also fit the row kernel (<= 16384 bf16 / 8192 fp32) else
 * DN_ERR_UNSUPPORTED.  Otherwise as ln_linear_deferred.
 */
DN_API dn_status ln_linear_serial(const void* x, const ln_linear_weights* w, int64_t M, float eps,
                           float* stats, void* out, hipStream_t stream);

/*
 * Fused without deferral (ablation of Eq. (5)): the same statistics pre-pass
 * as ln_linear_serial into stats[2 M], then one kernel that normalizes each x
 * fragment as it is loaded, xh = (x - mean) / sqrt(var + eps) rounded to the
 * GEMM dtype, and runs xh . W' + b (W' = Diag(gamma) W and b = beta W + bias
 * from ln_linear_prepare, so this is y F of Eq. (4) with y formed in
 * registers).  The normalization sits on the product's input path instead of
 * after it, which isolates what deferral buys over plain fusion.  bf16 only,
 * and only where the 256 x 256 kernel applies (M > 128, K % 64 == 0,
 * K and N < 2^22; it runs there even when ln_linear_deferred would take
 * 128 x 128 tiles); other shapes give DN_ERR_UNSUPPORTED.  Otherwise as
 * ln_linear_serial.
 */
DN_API dn_status ln_linear_norm_on_load(const void* x, const ln_linear_weights* w, int64_t M, float eps,
                                 float* stats, void* out, hipStream_t stream);

/* ======================================================================= */
/* RMSNorm -> gated MLP input (SwiGLU), deferred                            */
/* ======================================================================= */

/*
 * The Llama MLP input stage (Sec. II-A, subsubsection on RMSNorm in Llama
 * models, which fuses the up-projection and gating): y = RMSNorm(x) (Eq. (6)),
 * h = SiLU(y Wg) * (y Wu) element-wise, SiLU(z) = z / (1 + e^-z).
 * Deferred: both products run on the MFMA over the un-normalized x, each x
 * fragment feeding the gate and the up columns, with sum x^2 reduced
 * concurrently; the epilogue applies rstd to both products (before the SiLU,
 * which is not homogeneous, so the deferral ends there) and writes h once.
 *
 * swiglu_prepare folds gamma into both [K][N] weights and packs them into one
 * buffer of swiglu_packed_bytes(K, N, dtype) bytes (256-byte aligned device
 * memory): Wg' and Wu' in the fragment-chunk layout of ln_linear_prepare,
 * interleaved by 16-feature blocks (block 2j = gate features 16j.., block
 * 2j+1 = up features 16j..), with c and b (zero: no shift, no bias) in the
 * same interleaved order.  *w_out gets N (the output features) and
 * layout_version DN_SWIGLU_LAYOUT_VERSION; only rms_swiglu_deferred takes it.
 * rms_swiglu_deferred writes h[M][N] in w->dtype; eps as for
 * rms_linear_deferred.  Status codes and alignment rules as for the
 * LayerNorm -> Linear calls.
 */
#define DN_SWIGLU_LAYOUT_VERSION 0x102

DN_API size_t swiglu_packed_bytes(int64_t K, int64_t N, int dtype);

DN_API dn_status swiglu_prepare(const void* W_gate, const void* W_up, const void* gamma,
                         int64_t K, int64_t N, int dtype, void* packed, size_t packed_bytes,
                         ln_linear_weights* w_out, hipStream_t stream);

DN_API dn_status rms_swiglu_deferred(const void* x, const ln_linear_weights* w, int64_t M,
                              float eps, void* h, hipStream_t stream);

/* ======================================================================= */
/* Softmax -> P.V, deferred (Sec. II-B, Eq. (7), (8) and its footnote)      */
/* ======================================================================= */

/*
 * out[BH][Lq][d] = softmax(S[BH][Lq][Lk]) . V[BH][Lk][d] per head, computed
 * the deferred way: the MFMA consumes the un-normalized numerators
 * exp(s - m) (rounded to bf16), the row max m (footnote of Eq. (7)) is kept
 * online per key tile, the row sum l is accumulated concurrently, and the
 * epilogue divides once: out = acc / l (Eq. (8)).
 * causal = 1 keeps key j for query i iff j <= i (requires Lq == Lk); the
 * stored values at j > i are ignored (tiles wholly above the diagonal are
 * never read; inside diagonal tiles they are masked).  causal = 0 uses every
 * key.  A row whose kept scores are all -inf gives NaN.  dtype must be
 * DN_BF16; d must be 64 or 128; Lk a multiple of 8, Lq * Lk <= 2^31 and
 * Lk * d * 2 < 2^32 (else DN_ERR_UNSUPPORTED).
 */
DN_API dn_status softmax_pv_deferred(const void* S, const void* V, int64_t BH, int64_t Lq,
                              int64_t Lk, int64_t d, int causal, int dtype, void* out,
                              hipStream_t stream);

/*
 * The same deferred Softmax -> P.V with the scores formed in the kernel:
 * out[BH][Lq][d] = softmax(scale * Q K^T) . V per head, Q[BH][Lq][d],
 * K, V[BH][Lk][d] (Sec. II-B carried one operation earlier, so that S never
 * exists in memory: Eq. (8)'s numerators exp(s - m) come straight from the
 * Q.K^T product on the matrix core, the row max is kept online, the row sum
 * reduced alongside, and out = acc / l once).  causal = 1 keeps key j for
 * query i iff j <= i (Lq == Lk).  scale must be finite and > 0.  dtype must
 * be DN_BF16; d 64 or 128; Lq * d * 2 and Lk * d * 2 < 2^31 per head (else
 * DN_ERR_UNSUPPORTED).  A row whose scores are all -inf cannot occur (finite
 * inputs); NaN inputs propagate.
 */
DN_API dn_status attention_deferred(const void* Q, const void* K, const void* V, int64_t BH,
                             int64_t Lq, int64_t Lk, int64_t d, int causal, float scale,
                             int dtype, void* out, hipStream_t stream);

/*
 * attention_deferred with grouped-query attention (as in the Llama 3 models
 * the paper evaluates): K, V hold BH_kv heads [BH_kv][Lk][d], and Q, out
 * hold BH_kv * group query heads [BH_kv * group][Lq][d]; query head h reads
 * key/value head h / group (the group's query heads are consecutive).  Each
 * query head is computed exactly as by attention_deferred.  group >= 1;
 * other rules and status codes as attention_deferred.
 */
DN_API dn_status attention_gqa_deferred(const void* Q, const void* K, const void* V, int64_t BH_kv,
                                 int64_t group, int64_t Lq, int64_t Lk, int64_t d, int causal,
                                 float scale, int dtype, void* out, hipStream_t stream);

/*
 * Decode-shaped attention: Lq <= 16 query rows per head against all Lk keys
 * (the key/value cache holds exactly the visible keys, so no mask).  The keys
 * are cut into ranges, one workgroup each, that leave their un-normalized
 * partial sums (acc, l and the reference max m, fp32) in `workspace`; one
 * merge kernel then combines them, m = max m_g, out = sum 2^(m_g - m) acc_g /
 * sum 2^(m_g - m) l_g -- the deferred division of Eq. (8) once more, across
 * key ranges.  workspace: caller-owned device memory of
 * attention_decode_workspace_bytes(BH, Lq, Lk, d) bytes, 16-byte aligned, not
 * overlapping the other arguments; its contents are scratch.  Q[BH][Lq][d],
 * K, V[BH][Lk][d], out[BH][Lq][d]; other rules as attention_deferred
 * (DN_ERR_UNSUPPORTED for Lq > 16).  Grouped-query attention (g query heads
 * sharing each key/value head, the g heads consecutive): pass Q and out as
 * [BH][g * Lq][d] -- the same memory as [BH * g][Lq][d] -- with Lq := g * Lq
 * (<= 16), so each key/value tile read from HBM serves all g heads at once.
 * With enough heads to fill the chip the
 * keys are not split and one pass writes out directly (the workspace is then
 * not touched).  attention_decode_workspace_bytes
 * returns 0 for an invalid request.
 */
DN_API size_t attention_decode_workspace_bytes(int64_t BH, int64_t Lq, int64_t Lk, int64_t d);

DN_API dn_status attention_decode_deferred(const void* Q, const void* K, const void* V, int64_t BH,
                                    int64_t Lq, int64_t Lk, int64_t d, float scale, int dtype,
                                    void* workspace, size_t workspace_bytes, void* out,
                                    hipStream_t stream);

/*
 * For callers that cannot allocate (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): attention_decode_deferred
 * with no workspace argument.  The key-range partials go to a 12 MiB device
 * array that the library holds on each GPU it runs on until the process ends;
 * no call allocates or frees memory.  Every request attention_decode_deferred
 * accepts fits it (the partials stay below 4.25 MiB at d = 64 and 4.125 MiB
 * at d = 128); a request that would not gives DN_ERR_UNSUPPORTED.  The array
 * keeps the last call's partials, which every call overwrites before it reads
 * them; calls that overlap on one GPU (concurrent streams) share it and race.
 * Arguments, layout, grouped-query use and status codes as
 * attention_decode_deferred; the output is bitwise the same.
 */
DN_API dn_status attention_decode_deferred_noalloc(const void* Q, const void* K, const void* V, int64_t BH,
                                            int64_t Lq, int64_t Lk, int64_t d, float scale, int dtype,
                                            void* out, hipStream_t stream);

/* ======================================================================= */
/* Unfused comparators: the conventional sub-graph of Fig. 1(a)             */
/* ======================================================================= */

/* y[M][K] = (x - mean)/sqrt(var + eps) * gamma + beta, Eq. (1)-(2).  beta may be NULL. */
DN_API dn_status layernorm(const void* x, const void* gamma, const void* beta, int64_t M,
                    int64_t K, float eps, int dtype, void* y, hipStream_t stream);

/* y[M][K] = x / sqrt(sum_k x^2 / K + eps) * gamma, Eq. (6) (eps as for
   rms_linear_deferred).  Same rules and status codes as layernorm. */
DN_API dn_status rmsnorm(const void* x, const void* gamma, int64_t M, int64_t K, float eps,
                  int dtype, void* y, hipStream_t stream);

/* h[i] = SiLU(g[i]) * u[i] for count elements (count a multiple of 8); the
   conventional last step of the gated MLP input.  h must not overlap g or u. */
DN_API dn_status silu_mul(const void* g, const void* u, int64_t count, int dtype, void* h,
                   hipStream_t stream);

/*
 * P[BH][Lq][Lk] = softmax of each row of S (Eq. (7) with the max subtraction).
 * causal = 0: every key.  causal = 1: keys j <= i, and P = 0 for j > i (dense,
 * the conventional output).  causal = 2: keys j <= i, and only the aligned
 * 8-element groups that contain some j <= i are written (entries j > i inside
 * such a group are 0; the rest of the upper triangle is left untouched); this
 * is the input gemm(a_causal = 1) expects.  causal != 0 requires Lq == Lk.
 * dtype must be DN_BF16; Lk <= 16384.
 */
DN_API dn_status softmax(const void* S, int64_t BH, int64_t Lq, int64_t Lk, int causal,
                  int dtype, void* P, hipStream_t stream);

/*
 * C[batch][M][N] = A[batch][M][K] . B (+ bias[N]), fp32 accumulation.
 * b_layout = 0: B is [batch][K][N] (row-major, N contiguous).
 * b_layout = 1: B is given transposed, [batch][N][K] (K contiguous).
 * b_layout = 2: B is the packed buffer ln_linear_prepare wrote for (K, N,
 *               dtype) -- with gamma = 1 it holds W itself; its c and b parts
 *               are ignored.  batch must be 1.  This is the weight layout and
 *               main loop ln_linear_deferred uses, so the two paths differ
 *               only by the fusion.
 * a_causal = 1: A is lower-triangular by contract (A[i][j] treated as 0 for
 *               j > i, never read beyond the diagonal tile); requires M == K,
 *               bf16 and b_layout 0 or 1.
 * bias may be NULL.
 */
DN_API dn_status gemm(const void* A, const void* B, const void* bias, int64_t batch, int64_t M,
               int64_t K, int64_t N, int b_layout, int a_causal, int dtype, void* C,
               hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* DN_H */
