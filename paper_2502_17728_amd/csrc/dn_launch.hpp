// dn_launch.hpp -- host-side launchers of the libdn kernels (internal; the
// public C ABI in include/dn.h validates arguments and then calls these).
// Every launcher only enqueues on `stream` and returns hipGetLastError().
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace dn {

// Byte offsets of the pieces of a prepared LN->Linear weight buffer.
struct PackedLayout {
    int64_t kchunks, nblocks;  // K_pad / kchunk, N_pad / 16
    size_t wt_off, wt_bytes;   // W'^T in fragment-chunk order, element type, zero padded
    size_t c_off, b_off;       // c[N], b[N] fp32
    size_t total;
};
PackedLayout packed_layout(int64_t K, int64_t N, int dtype);

// Layout of SwiGLU weights: the gate and up W' interleaved in 16-column blocks
// (block 2j = gate columns 16j.., block 2j+1 = up columns 16j..), c and b likewise.
PackedLayout swiglu_layout(int64_t K, int64_t N, int dtype);

hipError_t launch_swiglu_prepare(const void* Wg, const void* Wu, const void* gamma, int64_t K, int64_t N,
                                 int dtype, void* packed, hipStream_t s);

// out[M][N] = SiLU(gate) * up with gate, up the deferred-normalized products.
hipError_t launch_swiglu_deferred(const void* x, const void* packed, int64_t M, int64_t K, int64_t N,
                                  int dtype, float eps, int rms, void* out, hipStream_t s);

// h[M][N] = SiLU(g) * u element-wise (unfused comparator).
hipError_t launch_silu_mul(const void* g, const void* u, int64_t count, int dtype, void* h, hipStream_t s);

// center = 1: pack the literal Eq. (5) weight (I - E/n) Diag(gamma) W and set c = 0.
hipError_t launch_ln_prepare(const void* W, const void* gamma, const void* beta, const void* bias,
                             int64_t K, int64_t N, int dtype, int center, void* packed, hipStream_t s);

// rms = 1: RMSNorm statistics (Eq. (6)), the mean taken as zero.  row_stats (nullable):
// (mean, rstd) per row from a pre-pass, used instead of the concurrent moments.
// stats_out (nullable): the concurrently reduced (mean, rstd) of every row, exported.
hipError_t launch_ln_linear_deferred(const void* x, const void* packed, int64_t M, int64_t K,
                                     int64_t N, int dtype, float eps, int rms, const float* row_stats,
                                     void* out, hipStream_t s, float* stats_out = nullptr);

// y = (x - mean) rstd gamma + beta from per-row (mean, rstd); beta nullable.
hipError_t launch_apply_norm(const void* x, const float* stats, const void* gamma, const void* beta, int64_t M,
                             int64_t K, int dtype, void* y, hipStream_t s);

// Normalize-on-load ablation (bf16, large-tile shapes only): xh = (x - mean) rstd on the
// product's input path from pre-pass row_stats, out = xh . W' + b.
bool ln_on_load_supported(int64_t M, int64_t K, int64_t N, int dtype);
hipError_t launch_ln_linear_on_load(const void* x, const void* packed, int64_t M, int64_t K, int64_t N,
                                    const float* row_stats, void* out, hipStream_t s);

// stats[2 r], stats[2 r + 1] = mean, 1/sqrt(var + eps) of row r of x (two-pass, Eq. (1)-(2)).
hipError_t launch_row_stats(const void* x, int64_t M, int64_t K, float eps, int dtype, float* stats,
                            hipStream_t s);

hipError_t launch_gemm(const void* A, const void* B, const void* bias, int64_t batch, int64_t M,
                       int64_t K, int64_t N, int b_layout, int a_causal, int dtype, void* C,
                       hipStream_t s);

hipError_t launch_softmax_pv_deferred(const void* S, const void* V, int64_t BH, int64_t Lq,
                                      int64_t Lk, int64_t d, int causal, void* out, hipStream_t s);

// out[BH][Lq][d] = softmax(scale * Q K^T) V per query head, the scores formed in the kernel;
// query head h reads key/value head h / group (K, V hold BH / group heads).
hipError_t launch_attention_deferred(const void* Q, const void* K, const void* V, int64_t BH, int64_t Lq,
                                     int64_t Lk, int64_t d, int causal, float scale, void* out, hipStream_t s,
                                     int group = 1);

// Decode attention (Lq <= 16, all Lk keys visible): key ranges split over workgroups
// (partials in `workspace`, attention_decode_workspace_bytes of them), then one merge;
// a single pass straight to `out` when the heads alone fill the chip.
size_t attention_decode_workspace_bytes(int64_t BH, int64_t Lq, int64_t Lk, int64_t d);
hipError_t launch_attention_decode(const void* Q, const void* K, const void* V, int64_t BH, int64_t Lq, int64_t Lk,
                                   int64_t d, float scale, void* workspace, void* out, hipStream_t s);

// The same with the partials in a library-owned device array of kDecodeScratchBytes per GPU
// (no workspace argument, no allocation).  attention_decode_partials_bytes: the bytes of
// partials a call uses there (0 when the heads alone fill the chip and one pass suffices).
constexpr size_t kDecodeScratchBytes = size_t(12) << 20;
size_t attention_decode_partials_bytes(int64_t BH, int64_t Lq, int64_t Lk, int64_t d);
hipError_t launch_attention_decode_noalloc(const void* Q, const void* K, const void* V, int64_t BH, int64_t Lq,
                                           int64_t Lk, int64_t d, float scale, void* out, hipStream_t s);

hipError_t launch_layernorm(const void* x, const void* gamma, const void* beta, int64_t M,
                            int64_t K, float eps, int rms, int dtype, void* y, hipStream_t s);

hipError_t launch_softmax(const void* S, int64_t BH, int64_t Lq, int64_t Lk, int causal, void* P,
                          hipStream_t s);

// Largest K (elements per row) the row-wise unfused kernels keep in registers.
constexpr int64_t kMaxRowElemsBf16 = 16384;
constexpr int64_t kMaxRowElemsF32 = 8192;

}  // namespace dn
