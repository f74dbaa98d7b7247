// abi.cpp -- the C ABI of libdn (declared in include/dn.h): argument
// validation on the host, then dispatch to the kernel launchers.  No entry
// point touches the HIP runtime before its arguments have been validated.
#include <math.h>
#include <stdint.h>

#include "dn.h"
#include "dn_launch.hpp"

namespace {

constexpr int kVersion = (0 << 16) | 1;

bool valid_dtype(int dt) { return dt == DN_F32 || dt == DN_BF16; }
size_t esize(int dt) { return dt == DN_F32 ? 4 : 2; }
bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

// bytes = a * b * c without overflow (all >= 1); false on overflow.
bool bytes_of(int64_t a, int64_t b, int64_t c, size_t* out) {
    int64_t ab, abc;
    if (__builtin_mul_overflow(a, b, &ab) || __builtin_mul_overflow(ab, c, &abc)) return false;
    *out = (size_t)abc;
    return true;
}

// [p, p+n) and [q, q+m) intersect (NULL ranges never do).
bool overlaps(const void* p, size_t n, const void* q, size_t m) {
    if (!p || !q || n == 0 || m == 0) return false;
    const uintptr_t a = reinterpret_cast<uintptr_t>(p), b = reinterpret_cast<uintptr_t>(q);
    return a < b + m && b < a + n;
}

dn_status from_hip(hipError_t e) { return e == hipSuccess ? DN_OK : DN_ERR_HIP; }

constexpr int64_t kMaxGridX = 0x7fffffff;
constexpr int64_t kMaxBatch = 65535;

}  // namespace

extern "C" {

DN_API const char* dn_status_string(int status) {
    switch (status) {
        case DN_OK: return "DN_OK";
        case DN_ERR_INVALID_ARG: return "DN_ERR_INVALID_ARG";
        case DN_ERR_UNSUPPORTED: return "DN_ERR_UNSUPPORTED";
        case DN_ERR_MISALIGNED: return "DN_ERR_MISALIGNED";
        case DN_ERR_HIP: return "DN_ERR_HIP";
        default: return "DN_ERR_UNKNOWN";
    }
}

DN_API int dn_version(void) { return kVersion; }

DN_API size_t ln_linear_packed_bytes(int64_t K, int64_t N, int dtype) {
    size_t wt;
    if (K < 1 || N < 1 || !valid_dtype(dtype) || !bytes_of(K, N, (int64_t)esize(dtype), &wt)) return 0;
    return dn::packed_layout(K, N, dtype).total;
}

static dn_status prepare_ln(const void* W, const void* gamma, const void* beta, const void* bias, int64_t K,
                            int64_t N, int dtype, int center, void* packed, size_t packed_bytes,
                            ln_linear_weights* w_out, hipStream_t stream) {
    if (!W || !gamma || !packed || !w_out || K < 1 || N < 1 || !valid_dtype(dtype)) return DN_ERR_INVALID_ARG;
    const size_t need = ln_linear_packed_bytes(K, N, dtype);
    if (need == 0 || packed_bytes < need) return DN_ERR_INVALID_ARG;
    if (K % 8 || N % 8) return DN_ERR_UNSUPPORTED;
    if (!aligned(W, 16) || !aligned(gamma, 16) || !aligned(beta, 16) || !aligned(bias, 16) || !aligned(packed, 256))
        return DN_ERR_MISALIGNED;
    const size_t es = esize(dtype);
    if (overlaps(packed, need, W, (size_t)K * N * es) || overlaps(packed, need, gamma, K * es) ||
        overlaps(packed, need, beta, K * es) || overlaps(packed, need, bias, N * es))
        return DN_ERR_INVALID_ARG;
    if ((N + 63) / 64 > kMaxGridX || (K + 63) / 64 > kMaxBatch) return DN_ERR_UNSUPPORTED;
    const dn_status st = from_hip(dn::launch_ln_prepare(W, gamma, beta, bias, K, N, dtype, center, packed, stream));
    if (st == DN_OK) {
        w_out->K = K;
        w_out->N = N;
        w_out->dtype = dtype;
        w_out->layout_version = DN_LN_LAYOUT_VERSION;
        w_out->packed = packed;
    }
    return st;
}

DN_API dn_status ln_linear_prepare(const void* W, const void* gamma, const void* beta, const void* bias,
                                   int64_t K, int64_t N, int dtype, void* packed, size_t packed_bytes,
                                   ln_linear_weights* w_out, hipStream_t stream) {
    return prepare_ln(W, gamma, beta, bias, K, N, dtype, 0, packed, packed_bytes, w_out, stream);
}

DN_API dn_status ln_linear_prepare_centered(const void* W, const void* gamma, const void* beta, const void* bias,
                                            int64_t K, int64_t N, int dtype, void* packed, size_t packed_bytes,
                                            ln_linear_weights* w_out, hipStream_t stream) {
    return prepare_ln(W, gamma, beta, bias, K, N, dtype, 1, packed, packed_bytes, w_out, stream);
}

static dn_status deferred_linear(const void* x, const ln_linear_weights* w, int64_t M, float eps, int rms,
                                 float* stats, void* out, hipStream_t stream, bool on_load = false,
                                 float* stats_out = nullptr) {
    if (!x || !w || !out || !w->packed || M < 1) return DN_ERR_INVALID_ARG;
    if (w->layout_version != DN_LN_LAYOUT_VERSION || w->K < 1 || w->N < 1 || !valid_dtype(w->dtype))
        return DN_ERR_INVALID_ARG;
    if (!isfinite(eps) || eps < 0.f) return DN_ERR_INVALID_ARG;
    const int64_t K = w->K, N = w->N;
    const int dt = w->dtype;
    size_t xb, ob;
    if (!bytes_of(M, K, (int64_t)esize(dt), &xb) || !bytes_of(M, N, (int64_t)esize(dt), &ob))
        return DN_ERR_INVALID_ARG;
    if (K % 8 || N % 8) return DN_ERR_UNSUPPORTED;
    if (!aligned(x, 16) || !aligned(out, 16) || !aligned(w->packed, 256)) return DN_ERR_MISALIGNED;
    const size_t pb = ln_linear_packed_bytes(K, N, dt);
    if (overlaps(out, ob, x, xb) || overlaps(out, ob, w->packed, pb)) return DN_ERR_INVALID_ARG;
    if (((M + 15) / 16) * ((N + 15) / 16) > kMaxGridX) return DN_ERR_UNSUPPORTED;
    if (on_load && !dn::ln_on_load_supported(M, K, N, dt)) return DN_ERR_UNSUPPORTED;
    if (stats) {
        if (!aligned(stats, 16)) return DN_ERR_MISALIGNED;
        const size_t sb = (size_t)M * 8;
        if (overlaps(stats, sb, x, xb) || overlaps(stats, sb, out, ob) || overlaps(stats, sb, w->packed, pb))
            return DN_ERR_INVALID_ARG;
        if (K > (dt == DN_F32 ? dn::kMaxRowElemsF32 : dn::kMaxRowElemsBf16) || (M + 3) / 4 > kMaxGridX)
            return DN_ERR_UNSUPPORTED;
        const dn_status st = from_hip(dn::launch_row_stats(x, M, K, eps, dt, stats, stream));
        if (st != DN_OK) return st;
    }
    if (on_load) return from_hip(dn::launch_ln_linear_on_load(x, w->packed, M, K, N, stats, out, stream));
    return from_hip(dn::launch_ln_linear_deferred(x, w->packed, M, K, N, dt, eps, rms, stats, out, stream,
                                                  stats_out));
}

DN_API dn_status ln_linear_deferred(const void* x, const ln_linear_weights* w, int64_t M, float eps, void* out,
                                    hipStream_t stream) {
    return deferred_linear(x, w, M, eps, 0, nullptr, out, stream);
}

DN_API dn_status ln_linear_serial(const void* x, const ln_linear_weights* w, int64_t M, float eps, float* stats,
                                  void* out, hipStream_t stream) {
    if (!stats) return DN_ERR_INVALID_ARG;
    return deferred_linear(x, w, M, eps, 0, stats, out, stream);
}

DN_API dn_status ln_linear_norm_on_load(const void* x, const ln_linear_weights* w, int64_t M, float eps,
                                        float* stats, void* out, hipStream_t stream) {
    if (!stats) return DN_ERR_INVALID_ARG;
    return deferred_linear(x, w, M, eps, 0, stats, out, stream, true);
}

// Post-LN placement: the deferred product plus the normalized rows themselves
// (the residual branch), from the statistics the product's kernel reduced.
static dn_status post_linear(const void* x, const ln_linear_weights* w, int64_t M, float eps, int rms,
                             const void* gamma, const void* beta, float* stats, void* y, void* out,
                             hipStream_t stream) {
    if (!x || !w || !gamma || !stats || !y || !out || M < 1) return DN_ERR_INVALID_ARG;
    if (w->layout_version != DN_LN_LAYOUT_VERSION || w->K < 1 || w->N < 1 || !valid_dtype(w->dtype))
        return DN_ERR_INVALID_ARG;
    const int64_t K = w->K;
    const size_t es = esize(w->dtype);
    size_t xb, sb, ob;
    if (!bytes_of(M, K, (int64_t)es, &xb) || !bytes_of(M, 2, 4, &sb) || !bytes_of(M, w->N, (int64_t)es, &ob))
        return DN_ERR_INVALID_ARG;
    if (K % 8) return DN_ERR_UNSUPPORTED;
    if (!aligned(gamma, 16) || !aligned(beta, 16) || !aligned(stats, 16) || !aligned(y, 16))
        return DN_ERR_MISALIGNED;
    const size_t pb = ln_linear_packed_bytes(K, w->N, w->dtype);
    if (overlaps(y, xb, x, xb) || overlaps(y, xb, out, ob) || overlaps(y, xb, stats, sb) ||
        overlaps(y, xb, w->packed, pb) || overlaps(y, xb, gamma, K * es) || overlaps(y, xb, beta, K * es) ||
        overlaps(stats, sb, x, xb) || overlaps(stats, sb, out, ob) || overlaps(stats, sb, w->packed, pb) ||
        overlaps(stats, sb, gamma, K * es) || overlaps(stats, sb, beta, K * es))
        return DN_ERR_INVALID_ARG;
    if ((M * K / (w->dtype == DN_F32 ? 4 : 8) + 255) / 256 > kMaxGridX) return DN_ERR_UNSUPPORTED;
    // the product with its concurrent statistics (validated as ln_linear_deferred), exporting them
    const dn_status st = deferred_linear(x, w, M, eps, rms, nullptr, out, stream, false, stats);
    if (st != DN_OK) return st;
    return from_hip(dn::launch_apply_norm(x, stats, gamma, rms ? nullptr : beta, M, K, w->dtype, y, stream));
}

DN_API dn_status ln_linear_deferred_post(const void* x, const ln_linear_weights* w, int64_t M, float eps,
                                         const void* gamma, const void* beta, float* stats, void* y, void* out,
                                         hipStream_t stream) {
    return post_linear(x, w, M, eps, 0, gamma, beta, stats, y, out, stream);
}

DN_API dn_status rms_linear_deferred_post(const void* x, const ln_linear_weights* w, int64_t M, float eps,
                                          const void* gamma, float* stats, void* y, void* out, hipStream_t stream) {
    return post_linear(x, w, M, eps, 1, gamma, nullptr, stats, y, out, stream);
}

DN_API dn_status rms_linear_deferred(const void* x, const ln_linear_weights* w, int64_t M, float eps, void* out,
                                     hipStream_t stream) {
    return deferred_linear(x, w, M, eps, 1, nullptr, out, stream);
}

DN_API size_t swiglu_packed_bytes(int64_t K, int64_t N, int dtype) {
    size_t wt;
    if (K < 1 || N < 1 || !valid_dtype(dtype) || !bytes_of(K, 2 * N + 32, (int64_t)esize(dtype), &wt)) return 0;
    return dn::swiglu_layout(K, N, dtype).total;
}

DN_API dn_status swiglu_prepare(const void* W_gate, const void* W_up, const void* gamma, int64_t K, int64_t N,
                                int dtype, void* packed, size_t packed_bytes, ln_linear_weights* w_out,
                                hipStream_t stream) {
    if (!W_gate || !W_up || !gamma || !packed || !w_out || K < 1 || N < 1 || !valid_dtype(dtype))
        return DN_ERR_INVALID_ARG;
    const size_t need = swiglu_packed_bytes(K, N, dtype);
    if (need == 0 || packed_bytes < need) return DN_ERR_INVALID_ARG;
    if (K % 8 || N % 8) return DN_ERR_UNSUPPORTED;
    if (!aligned(W_gate, 16) || !aligned(W_up, 16) || !aligned(gamma, 16) || !aligned(packed, 256))
        return DN_ERR_MISALIGNED;
    const size_t es = esize(dtype);
    if (overlaps(packed, need, W_gate, (size_t)K * N * es) || overlaps(packed, need, W_up, (size_t)K * N * es) ||
        overlaps(packed, need, gamma, K * es))
        return DN_ERR_INVALID_ARG;
    if ((2 * N + 255) / 256 > kMaxGridX || (K + 63) / 64 > kMaxBatch) return DN_ERR_UNSUPPORTED;
    const dn_status st = from_hip(dn::launch_swiglu_prepare(W_gate, W_up, gamma, K, N, dtype, packed, stream));
    if (st == DN_OK) {
        w_out->K = K;
        w_out->N = N;
        w_out->dtype = dtype;
        w_out->layout_version = DN_SWIGLU_LAYOUT_VERSION;
        w_out->packed = packed;
    }
    return st;
}

DN_API dn_status rms_swiglu_deferred(const void* x, const ln_linear_weights* w, int64_t M, float eps, void* h,
                                     hipStream_t stream) {
    if (!x || !w || !h || !w->packed || M < 1) return DN_ERR_INVALID_ARG;
    if (w->layout_version != DN_SWIGLU_LAYOUT_VERSION || w->K < 1 || w->N < 1 || !valid_dtype(w->dtype))
        return DN_ERR_INVALID_ARG;
    if (!isfinite(eps) || eps < 0.f) return DN_ERR_INVALID_ARG;
    const int64_t K = w->K, N = w->N;
    const int dt = w->dtype;
    size_t xb, ob;
    if (!bytes_of(M, K, (int64_t)esize(dt), &xb) || !bytes_of(M, N, (int64_t)esize(dt), &ob))
        return DN_ERR_INVALID_ARG;
    if (K % 8 || N % 8) return DN_ERR_UNSUPPORTED;
    if (!aligned(x, 16) || !aligned(h, 16) || !aligned(w->packed, 256)) return DN_ERR_MISALIGNED;
    const size_t pb = swiglu_packed_bytes(K, N, dt);
    if (overlaps(h, ob, x, xb) || overlaps(h, ob, w->packed, pb)) return DN_ERR_INVALID_ARG;
    if (((M + 15) / 16) * ((2 * N + 31) / 16) > kMaxGridX) return DN_ERR_UNSUPPORTED;
    return from_hip(dn::launch_swiglu_deferred(x, w->packed, M, K, N, dt, eps, 1, h, stream));
}

DN_API dn_status softmax_pv_deferred(const void* S, const void* V, int64_t BH, int64_t Lq, int64_t Lk, int64_t d,
                                     int causal, int dtype, void* out, hipStream_t stream) {
    if (!S || !V || !out || BH < 1 || Lq < 1 || Lk < 1 || d < 1 || !valid_dtype(dtype)) return DN_ERR_INVALID_ARG;
    if (causal != 0 && causal != 1) return DN_ERR_INVALID_ARG;
    if (causal && Lq != Lk) return DN_ERR_INVALID_ARG;
    size_t sb, vb, ob;
    int64_t bhlq;
    if (!bytes_of(BH, Lq, Lk * 2, &sb) || !bytes_of(BH, Lk, d * 2, &vb) || !bytes_of(BH, Lq, d * 2, &ob) ||
        __builtin_mul_overflow(BH, Lq, &bhlq))
        return DN_ERR_INVALID_ARG;
    if (dtype != DN_BF16 || (d != 64 && d != 128) || Lk % 8) return DN_ERR_UNSUPPORTED;
    if (Lq * Lk > (int64_t(1) << 31) || Lk * d * 2 >= (int64_t(1) << 32))
        return DN_ERR_UNSUPPORTED;  // one head's scores and values within 4 GiB
    if (!aligned(S, 16) || !aligned(V, 16) || !aligned(out, 16)) return DN_ERR_MISALIGNED;
    if (overlaps(out, ob, S, sb) || overlaps(out, ob, V, vb)) return DN_ERR_INVALID_ARG;
    if (BH * ((Lq + 255) / 256) > kMaxGridX) return DN_ERR_UNSUPPORTED;
    return from_hip(dn::launch_softmax_pv_deferred(S, V, BH, Lq, Lk, d, causal, out, stream));
}

// BH key/value heads, each read by `group` consecutive query heads (group = 1: one each).
static dn_status attention_grouped(const void* Q, const void* K, const void* V, int64_t BH, int64_t group,
                                   int64_t Lq, int64_t Lk, int64_t d, int causal, float scale, int dtype, void* out,
                                   hipStream_t stream) {
    if (!Q || !K || !V || !out || BH < 1 || group < 1 || Lq < 1 || Lk < 1 || d < 1 || !valid_dtype(dtype))
        return DN_ERR_INVALID_ARG;
    if (causal != 0 && causal != 1) return DN_ERR_INVALID_ARG;
    if (causal && Lq != Lk) return DN_ERR_INVALID_ARG;
    if (!isfinite(scale) || !(scale > 0.f)) return DN_ERR_INVALID_ARG;
    int64_t BHq;
    size_t qb, kb;
    if (__builtin_mul_overflow(BH, group, &BHq) || !bytes_of(BHq, Lq, d * 2, &qb) || !bytes_of(BH, Lk, d * 2, &kb))
        return DN_ERR_INVALID_ARG;
    const size_t ob = qb;
    if (dtype != DN_BF16 || (d != 64 && d != 128)) return DN_ERR_UNSUPPORTED;
    if (Lq * d * 2 >= (int64_t(1) << 31) || Lk * d * 2 >= (int64_t(1) << 31)) return DN_ERR_UNSUPPORTED;
    if (group > (int64_t(1) << 20)) return DN_ERR_UNSUPPORTED;
    if (!aligned(Q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(out, 16)) return DN_ERR_MISALIGNED;
    if (overlaps(out, ob, Q, qb) || overlaps(out, ob, K, kb) || overlaps(out, ob, V, kb)) return DN_ERR_INVALID_ARG;
    if (BHq * ((Lq + 255) / 256) > kMaxGridX) return DN_ERR_UNSUPPORTED;
    return from_hip(dn::launch_attention_deferred(Q, K, V, BHq, Lq, Lk, d, causal, scale, out, stream, (int)group));
}

DN_API dn_status attention_deferred(const void* Q, const void* K, const void* V, int64_t BH, int64_t Lq, int64_t Lk,
                                    int64_t d, int causal, float scale, int dtype, void* out, hipStream_t stream) {
    return attention_grouped(Q, K, V, BH, 1, Lq, Lk, d, causal, scale, dtype, out, stream);
}

DN_API dn_status attention_gqa_deferred(const void* Q, const void* K, const void* V, int64_t BH_kv, int64_t group,
                                        int64_t Lq, int64_t Lk, int64_t d, int causal, float scale, int dtype,
                                        void* out, hipStream_t stream) {
    return attention_grouped(Q, K, V, BH_kv, group, Lq, Lk, d, causal, scale, dtype, out, stream);
}

DN_API size_t attention_decode_workspace_bytes(int64_t BH, int64_t Lq, int64_t Lk, int64_t d) {
    size_t b;
    if (BH < 1 || Lq < 1 || Lq > 16 || Lk < 1 || (d != 64 && d != 128) || !bytes_of(BH, Lk, d * 2, &b))
        return 0;
    return dn::attention_decode_workspace_bytes(BH, Lq, Lk, d);
}

DN_API dn_status attention_decode_deferred(const void* Q, const void* K, const void* V, int64_t BH, int64_t Lq,
                                           int64_t Lk, int64_t d, float scale, int dtype, void* workspace,
                                           size_t workspace_bytes, void* out, hipStream_t stream) {
    if (!Q || !K || !V || !out || !workspace || BH < 1 || Lq < 1 || Lk < 1 || d < 1 || !valid_dtype(dtype))
        return DN_ERR_INVALID_ARG;
    if (!isfinite(scale) || !(scale > 0.f)) return DN_ERR_INVALID_ARG;
    size_t qb, kb;
    if (!bytes_of(BH, Lq, d * 2, &qb) || !bytes_of(BH, Lk, d * 2, &kb)) return DN_ERR_INVALID_ARG;
    if (dtype != DN_BF16 || (d != 64 && d != 128) || Lq > 16) return DN_ERR_UNSUPPORTED;
    if (Lk * d * 2 >= (int64_t(1) << 31)) return DN_ERR_UNSUPPORTED;
    const size_t need = attention_decode_workspace_bytes(BH, Lq, Lk, d);
    if (need == 0 || workspace_bytes < need) return DN_ERR_INVALID_ARG;
    if (!aligned(Q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(out, 16) || !aligned(workspace, 16))
        return DN_ERR_MISALIGNED;
    if (overlaps(out, qb, Q, qb) || overlaps(out, qb, K, kb) || overlaps(out, qb, V, kb) ||
        overlaps(workspace, need, Q, qb) || overlaps(workspace, need, K, kb) || overlaps(workspace, need, V, kb) ||
        overlaps(workspace, need, out, qb))
        return DN_ERR_INVALID_ARG;
    if (BH * 16 > kMaxGridX) return DN_ERR_UNSUPPORTED;  // grids: BH + 1280 splits, BH * Lq / 4 merges
    return from_hip(dn::launch_attention_decode(Q, K, V, BH, Lq, Lk, d, scale, workspace, out, stream));
}

DN_API dn_status attention_decode_deferred_noalloc(const void* Q, const void* K, const void* V, int64_t BH,
                                                   int64_t Lq, int64_t Lk, int64_t d, float scale, int dtype,
                                                   void* out, hipStream_t stream) {
    if (!Q || !K || !V || !out || BH < 1 || Lq < 1 || Lk < 1 || d < 1 || !valid_dtype(dtype))
        return DN_ERR_INVALID_ARG;
    if (!isfinite(scale) || !(scale > 0.f)) return DN_ERR_INVALID_ARG;
    size_t qb, kb;
    if (!bytes_of(BH, Lq, d * 2, &qb) || !bytes_of(BH, Lk, d * 2, &kb)) return DN_ERR_INVALID_ARG;
    if (dtype != DN_BF16 || (d != 64 && d != 128) || Lq > 16) return DN_ERR_UNSUPPORTED;
    if (Lk * d * 2 >= (int64_t(1) << 31)) return DN_ERR_UNSUPPORTED;
    if (!aligned(Q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(out, 16)) return DN_ERR_MISALIGNED;
    if (overlaps(out, qb, Q, qb) || overlaps(out, qb, K, kb) || overlaps(out, qb, V, kb)) return DN_ERR_INVALID_ARG;
    if (BH * 16 > kMaxGridX) return DN_ERR_UNSUPPORTED;
    if (dn::attention_decode_partials_bytes(BH, Lq, Lk, d) > dn::kDecodeScratchBytes) return DN_ERR_UNSUPPORTED;
    return from_hip(dn::launch_attention_decode_noalloc(Q, K, V, BH, Lq, Lk, d, scale, out, stream));
}

static dn_status row_norm(const void* x, const void* gamma, const void* beta, int64_t M, int64_t K, float eps,
                          int rms, int dtype, void* y, hipStream_t stream) {
    if (!x || !gamma || !y || M < 1 || K < 1 || !valid_dtype(dtype)) return DN_ERR_INVALID_ARG;
    if (!isfinite(eps) || eps < 0.f) return DN_ERR_INVALID_ARG;
    size_t xb;
    if (!bytes_of(M, K, (int64_t)esize(dtype), &xb)) return DN_ERR_INVALID_ARG;
    if (K % 8 || K > (dtype == DN_F32 ? dn::kMaxRowElemsF32 : dn::kMaxRowElemsBf16)) return DN_ERR_UNSUPPORTED;
    if (!aligned(x, 16) || !aligned(gamma, 16) || !aligned(beta, 16) || !aligned(y, 16)) return DN_ERR_MISALIGNED;
    const size_t es = esize(dtype);
    if (overlaps(y, xb, x, xb) || overlaps(y, xb, gamma, K * es) || overlaps(y, xb, beta, K * es))
        return DN_ERR_INVALID_ARG;
    if ((M + 3) / 4 > kMaxGridX) return DN_ERR_UNSUPPORTED;
    return from_hip(dn::launch_layernorm(x, gamma, beta, M, K, eps, rms, dtype, y, stream));
}

DN_API dn_status layernorm(const void* x, const void* gamma, const void* beta, int64_t M, int64_t K, float eps,
                           int dtype, void* y, hipStream_t stream) {
    return row_norm(x, gamma, beta, M, K, eps, 0, dtype, y, stream);
}

DN_API dn_status rmsnorm(const void* x, const void* gamma, int64_t M, int64_t K, float eps, int dtype, void* y,
                         hipStream_t stream) {
    return row_norm(x, gamma, nullptr, M, K, eps, 1, dtype, y, stream);
}

DN_API dn_status silu_mul(const void* g, const void* u, int64_t count, int dtype, void* h, hipStream_t stream) {
    if (!g || !u || !h || count < 1 || !valid_dtype(dtype)) return DN_ERR_INVALID_ARG;
    size_t b;
    if (!bytes_of(count, 1, (int64_t)esize(dtype), &b)) return DN_ERR_INVALID_ARG;
    if (count % 8) return DN_ERR_UNSUPPORTED;
    if (!aligned(g, 16) || !aligned(u, 16) || !aligned(h, 16)) return DN_ERR_MISALIGNED;
    if (overlaps(h, b, g, b) || overlaps(h, b, u, b)) return DN_ERR_INVALID_ARG;
    if ((count / 4 + 255) / 256 > kMaxGridX) return DN_ERR_UNSUPPORTED;
    return from_hip(dn::launch_silu_mul(g, u, count, dtype, h, stream));
}

DN_API dn_status softmax(const void* S, int64_t BH, int64_t Lq, int64_t Lk, int causal, int dtype, void* P,
                         hipStream_t stream) {
    if (!S || !P || BH < 1 || Lq < 1 || Lk < 1 || !valid_dtype(dtype)) return DN_ERR_INVALID_ARG;
    if (causal < 0 || causal > 2 || (causal && Lq != Lk)) return DN_ERR_INVALID_ARG;
    size_t sb;
    if (!bytes_of(BH, Lq, Lk * 2, &sb)) return DN_ERR_INVALID_ARG;
    if (dtype != DN_BF16 || Lk % 8 || Lk > dn::kMaxRowElemsBf16) return DN_ERR_UNSUPPORTED;
    if (!aligned(S, 16) || !aligned(P, 16)) return DN_ERR_MISALIGNED;
    if (overlaps(P, sb, S, sb)) return DN_ERR_INVALID_ARG;
    if ((BH * Lq + 3) / 4 > kMaxGridX) return DN_ERR_UNSUPPORTED;
    return from_hip(dn::launch_softmax(S, BH, Lq, Lk, causal, P, stream));
}

DN_API dn_status gemm(const void* A, const void* B, const void* bias, int64_t batch, int64_t M, int64_t K, int64_t N,
                      int b_layout, int a_causal, int dtype, void* C, hipStream_t stream) {
    if (!A || !B || !C || batch < 1 || M < 1 || K < 1 || N < 1 || !valid_dtype(dtype)) return DN_ERR_INVALID_ARG;
    if (b_layout < 0 || b_layout > 2 || (a_causal != 0 && a_causal != 1)) return DN_ERR_INVALID_ARG;
    if (a_causal && M != K) return DN_ERR_INVALID_ARG;
    if (b_layout == 2 && batch != 1) return DN_ERR_INVALID_ARG;
    const int64_t es = (int64_t)esize(dtype);
    size_t ab, bb, cb, t;
    if (!bytes_of(batch, M, K * es, &ab) || !bytes_of(batch, K, N * es, &bb) || !bytes_of(batch, M, N * es, &cb) ||
        !bytes_of(M, K, 1, &t) || !bytes_of(K, N, 1, &t))
        return DN_ERR_INVALID_ARG;
    if (b_layout == 2) bb = ln_linear_packed_bytes(K, N, dtype);
    if (K % 8 || N % 8) return DN_ERR_UNSUPPORTED;
    if (dtype == DN_F32 && (b_layout == 0 || a_causal)) return DN_ERR_UNSUPPORTED;
    if (a_causal && b_layout == 2) return DN_ERR_UNSUPPORTED;
    if (batch > kMaxBatch) return DN_ERR_UNSUPPORTED;
    if (!aligned(A, 16) || !aligned(B, b_layout == 2 ? 256 : 16) || !aligned(bias, 16) || !aligned(C, 16))
        return DN_ERR_MISALIGNED;
    if (overlaps(C, cb, A, ab) || overlaps(C, cb, B, bb) || overlaps(C, cb, bias, (size_t)(N * es)))
        return DN_ERR_INVALID_ARG;
    if (((M + 31) / 32) * ((N + 63) / 64) > kMaxGridX) return DN_ERR_UNSUPPORTED;
    return from_hip(dn::launch_gemm(A, B, bias, batch, M, K, N, b_layout, a_causal, dtype, C, stream));
}

}  // extern "C"
