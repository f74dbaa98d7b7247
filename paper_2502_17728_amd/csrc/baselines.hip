// baselines.hip -- the unfused comparators of Fig. 1(a): LayerNorm (Eq. (1)-(2))
// and Softmax (Eq. (7) with the max subtraction), each materializing its full
// output before the separate GEMM.  One wave per row; the row stays in
// registers, so each element is read once and written once.  Also the
// element-wise pieces around the deferred path: the statistics pre-pass of the
// serial ablation, SiLU * up, and the normalized output of the post-LN
// placement (applied from statistics the deferred kernel has already reduced).
#include "dn_device.hpp"
#include "dn_launch.hpp"

namespace dn {

constexpr float kLog2eB = 1.4426950408889634f;

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = __builtin_fmaxf(v, __shfl_xor(v, o));
    return v;
}

template <class T>
__device__ __forceinline__ void unpack16(const u32x4& w, float* f);
template <>
__device__ __forceinline__ void unpack16<__bf16>(const u32x4& w, float* f) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        f[2 * e] = bf_lo(w[e]);
        f[2 * e + 1] = bf_hi(w[e]);
    }
}
template <>
__device__ __forceinline__ void unpack16<float>(const u32x4& w, float* f) {
#pragma unroll
    for (int e = 0; e < 4; ++e) f[e] = __uint_as_float(w[e]);
}
template <class T>
__device__ __forceinline__ u32x4 pack16(const float* f);
template <>
__device__ __forceinline__ u32x4 pack16<__bf16>(const float* f) {
    return u32x4{pack_bf16(f[0], f[1]), pack_bf16(f[2], f[3]), pack_bf16(f[4], f[5]), pack_bf16(f[6], f[7])};
}
template <>
__device__ __forceinline__ u32x4 pack16<float>(const float* f) {
    return u32x4{__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]), __float_as_uint(f[3])};
}

// y = (x - mean) / sqrt(var + eps) * gamma + beta; lane chunk j covers elements
// [(j*64 + lane) * EPL, +EPL).  rms = 1: RMSNorm (Eq. (6)), the mean taken as 0,
// so var is the mean square.
template <class T, int NCH>
__global__ __launch_bounds__(256) void layernorm_kernel(const T* __restrict__ x, const T* __restrict__ gamma,
                                                        const T* __restrict__ beta, int64_t M, int64_t K, float eps,
                                                        int rms, T* __restrict__ y) {
    constexpr int EPL = elem<T>::per16;
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= M) return;
    const T* xr = x + row * K;
    float v[NCH][EPL];
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
        const int64_t k = (int64_t)(j * 64 + lane) * EPL;
        if (k < K) {
            unpack16<T>(ld16(xr + k), v[j]);
        } else {
#pragma unroll
            for (int e = 0; e < EPL; ++e) v[j][e] = 0.f;
        }
#pragma unroll
        for (int e = 0; e < EPL; ++e) s += v[j][e];
    }
    const float mean = rms ? 0.f : wave_sum(s) / (float)K;
    float ss = 0.f;
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
        const int64_t k = (int64_t)(j * 64 + lane) * EPL;
        if (k < K) {
#pragma unroll
            for (int e = 0; e < EPL; ++e) {
                const float dlt = v[j][e] - mean;
                ss = __builtin_fmaf(dlt, dlt, ss);
            }
        }
    }
    const float var = wave_sum(ss) / (float)K;
    const float rstd = 1.0f / __builtin_sqrtf(var + eps);
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
        const int64_t k = (int64_t)(j * 64 + lane) * EPL;
        if (k < K) {
            float g[EPL], b[EPL], o[EPL];
            unpack16<T>(ld16(gamma + k), g);
            if (beta) {
                unpack16<T>(ld16(beta + k), b);
            } else {
#pragma unroll
                for (int e = 0; e < EPL; ++e) b[e] = 0.f;
            }
#pragma unroll
            for (int e = 0; e < EPL; ++e) o[e] = __builtin_fmaf((v[j][e] - mean) * rstd, g[e], b[e]);
            *reinterpret_cast<u32x4*>(y + row * K + k) = pack16<T>(o);
        }
    }
}

// Row statistics only (the serial ablation's pre-pass): stats[2 row] = mean,
// stats[2 row + 1] = 1/sqrt(var + eps), two passes over the row kept in registers.
template <class T, int NCH>
__global__ __launch_bounds__(256) void row_stats_kernel(const T* __restrict__ x, int64_t M, int64_t K, float eps,
                                                        float* __restrict__ stats) {
    constexpr int EPL = elem<T>::per16;
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= M) return;
    const T* xr = x + row * K;
    float v[NCH][EPL];
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
        const int64_t k = (int64_t)(j * 64 + lane) * EPL;
        if (k < K) {
            unpack16<T>(ld16(xr + k), v[j]);
        } else {
#pragma unroll
            for (int e = 0; e < EPL; ++e) v[j][e] = 0.f;
        }
#pragma unroll
        for (int e = 0; e < EPL; ++e) s += v[j][e];
    }
    const float mean = wave_sum(s) / (float)K;
    float ss = 0.f;
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
        const int64_t k = (int64_t)(j * 64 + lane) * EPL;
        if (k < K) {
#pragma unroll
            for (int e = 0; e < EPL; ++e) {
                const float dlt = v[j][e] - mean;
                ss = __builtin_fmaf(dlt, dlt, ss);
            }
        }
    }
    const float var = wave_sum(ss) / (float)K;
    if (lane == 0) {
        stats[2 * row] = mean;
        stats[2 * row + 1] = 1.0f / __builtin_sqrtf(var + eps);
    }
}

template <class T>
static hipError_t dispatch_stats(const void* x, int64_t M, int64_t K, float eps, float* st, hipStream_t s) {
    const int64_t nch = (K + 64 * elem<T>::per16 - 1) / (64 * elem<T>::per16);
    const dim3 grid((unsigned)((M + 3) / 4));
    const T* xt = (const T*)x;
    if (nch <= 2) row_stats_kernel<T, 2><<<grid, 256, 0, s>>>(xt, M, K, eps, st);
    else if (nch <= 4) row_stats_kernel<T, 4><<<grid, 256, 0, s>>>(xt, M, K, eps, st);
    else if (nch <= 8) row_stats_kernel<T, 8><<<grid, 256, 0, s>>>(xt, M, K, eps, st);
    else if (nch <= 16) row_stats_kernel<T, 16><<<grid, 256, 0, s>>>(xt, M, K, eps, st);
    else row_stats_kernel<T, 32><<<grid, 256, 0, s>>>(xt, M, K, eps, st);
    return hipGetLastError();
}

hipError_t launch_row_stats(const void* x, int64_t M, int64_t K, float eps, int dtype, float* stats,
                            hipStream_t s) {
    if (dtype == 0) return dispatch_stats<float>(x, M, K, eps, stats, s);
    return dispatch_stats<__bf16>(x, M, K, eps, stats, s);
}

// P = softmax(S) row-wise (bf16).  causal: keys j <= i; mode 1 writes zeros for
// j > i, mode 2 writes only the 8-element groups that reach the diagonal.
template <int NCH>
__global__ __launch_bounds__(256) void softmax_kernel(const __bf16* __restrict__ S, int64_t rows, int64_t Lq,
                                                      int64_t Lk, int causal, __bf16* __restrict__ P) {
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= rows) return;
    const int64_t i = row % Lq;
    const int64_t kept = causal ? min(i + 1, Lk) : Lk;
    const __bf16* sr = S + row * Lk;
    __bf16* pr = P + row * Lk;
    float v[NCH][8];
    float m = -__builtin_inff();
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
        const int64_t k = (int64_t)(j * 64 + lane) * 8;
        if (k < kept) {
            unpack16<__bf16>(ld16(sr + k), v[j]);
#pragma unroll
            for (int e = 0; e < 8; ++e)
                if (k + e >= kept) v[j][e] = -__builtin_inff();
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) v[j][e] = -__builtin_inff();
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) m = __builtin_fmaxf(m, v[j][e]);
    }
    m = wave_max(m);
    const float nb = m == -__builtin_inff() ? 0.f : -m * kLog2eB;
    float l = 0.f;
#pragma unroll
    for (int j = 0; j < NCH; ++j)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            v[j][e] = __builtin_amdgcn_exp2f(__builtin_fmaf(v[j][e], kLog2eB, nb));
            l += v[j][e];
        }
    const float inv = 1.0f / wave_sum(l);
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
        const int64_t k = (int64_t)(j * 64 + lane) * 8;
        if (k >= Lk) continue;
        if (causal == 2 && k >= kept) continue;
        float o[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = v[j][e] * inv;
        *reinterpret_cast<u32x4*>(pr + k) = pack16<__bf16>(o);
    }
}

template <class T, int NCH>
static hipError_t run_ln(const void* x, const void* g, const void* b, int64_t M, int64_t K, float eps, int rms,
                         void* y, hipStream_t s) {
    layernorm_kernel<T, NCH><<<dim3((unsigned)((M + 3) / 4)), 256, 0, s>>>((const T*)x, (const T*)g, (const T*)b, M,
                                                                          K, eps, rms, (T*)y);
    return hipGetLastError();
}

template <class T>
static hipError_t dispatch_ln(const void* x, const void* g, const void* b, int64_t M, int64_t K, float eps,
                              int rms, void* y, hipStream_t s) {
    const int64_t per_chunk = 64 * elem<T>::per16;
    const int64_t nch = (K + per_chunk - 1) / per_chunk;
    if (nch <= 1) return run_ln<T, 1>(x, g, b, M, K, eps, rms, y, s);
    if (nch <= 2) return run_ln<T, 2>(x, g, b, M, K, eps, rms, y, s);
    if (nch <= 4) return run_ln<T, 4>(x, g, b, M, K, eps, rms, y, s);
    if (nch <= 8) return run_ln<T, 8>(x, g, b, M, K, eps, rms, y, s);
    if (nch <= 16) return run_ln<T, 16>(x, g, b, M, K, eps, rms, y, s);
    return run_ln<T, 32>(x, g, b, M, K, eps, rms, y, s);
}

hipError_t launch_layernorm(const void* x, const void* gamma, const void* beta, int64_t M, int64_t K, float eps,
                            int rms, int dtype, void* y, hipStream_t s) {
    if (dtype == 0) return dispatch_ln<float>(x, gamma, beta, M, K, eps, rms, y, s);
    return dispatch_ln<__bf16>(x, gamma, beta, M, K, eps, rms, y, s);
}

template <int NCH>
static hipError_t run_sm(const void* S, int64_t rows, int64_t Lq, int64_t Lk, int causal, void* P, hipStream_t s) {
    softmax_kernel<NCH><<<dim3((unsigned)((rows + 3) / 4)), 256, 0, s>>>((const __bf16*)S, rows, Lq, Lk, causal,
                                                                        (__bf16*)P);
    return hipGetLastError();
}

hipError_t launch_softmax(const void* S, int64_t BH, int64_t Lq, int64_t Lk, int causal, void* P, hipStream_t s) {
    const int64_t rows = BH * Lq;
    const int64_t nch = (Lk + 511) / 512;
    if (nch <= 1) return run_sm<1>(S, rows, Lq, Lk, causal, P, s);
    if (nch <= 2) return run_sm<2>(S, rows, Lq, Lk, causal, P, s);
    if (nch <= 4) return run_sm<4>(S, rows, Lq, Lk, causal, P, s);
    if (nch <= 8) return run_sm<8>(S, rows, Lq, Lk, causal, P, s);
    if (nch <= 16) return run_sm<16>(S, rows, Lq, Lk, causal, P, s);
    return run_sm<32>(S, rows, Lq, Lk, causal, P, s);
}

// h = SiLU(g) * u element-wise, SiLU(z) = z / (1 + e^-z); one 16-byte piece per lane.
template <class T>
__global__ __launch_bounds__(256) void silu_mul_kernel(const T* __restrict__ g, const T* __restrict__ u,
                                                       int64_t count, T* __restrict__ h) {
    constexpr int EPL = elem<T>::per16;
    const int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * EPL;
    if (i >= count) return;
    float a[EPL], b[EPL], o[EPL];
    unpack16<T>(ld16(g + i), a);
    unpack16<T>(ld16(u + i), b);
#pragma unroll
    for (int e = 0; e < EPL; ++e) o[e] = a[e] / (1.0f + __builtin_amdgcn_exp2f(-a[e] * kLog2eB)) * b[e];
    *reinterpret_cast<u32x4*>(h + i) = pack16<T>(o);
}

hipError_t launch_silu_mul(const void* g, const void* u, int64_t count, int dtype, void* h, hipStream_t s) {
    const int64_t epl = dtype == 0 ? 4 : 8;
    const dim3 grid((unsigned)((count / epl + 255) / 256));
    if (dtype == 0)
        silu_mul_kernel<float><<<grid, 256, 0, s>>>((const float*)g, (const float*)u, count, (float*)h);
    else
        silu_mul_kernel<__bf16><<<grid, 256, 0, s>>>((const __bf16*)g, (const __bf16*)u, count, (__bf16*)h);
    return hipGetLastError();
}

// y = (x - mean) rstd gamma + beta (beta nullable) from per-row (mean, rstd):
// Eq. (2) with the statistics already reduced, one 16-byte piece per lane.
template <class T>
__global__ __launch_bounds__(256) void apply_norm_kernel(const T* __restrict__ x, const float* __restrict__ stats,
                                                         const T* __restrict__ gamma, const T* __restrict__ beta,
                                                         int64_t M, int64_t K, T* __restrict__ y) {
    constexpr int EPL = elem<T>::per16;
    const int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * EPL;
    if (i >= M * K) return;
    const int64_t r = i / K, k = i - r * K;  // K % EPL == 0: a piece never straddles rows
    const float mean = stats[2 * r], rstd = stats[2 * r + 1];
    float v[EPL], g[EPL], b[EPL], o[EPL];
    unpack16<T>(ld16(x + i), v);
    unpack16<T>(ld16(gamma + k), g);
    if (beta) {
        unpack16<T>(ld16(beta + k), b);
    } else {
#pragma unroll
        for (int e = 0; e < EPL; ++e) b[e] = 0.f;
    }
#pragma unroll
    for (int e = 0; e < EPL; ++e) o[e] = __builtin_fmaf((v[e] - mean) * rstd, g[e], b[e]);
    *reinterpret_cast<u32x4*>(y + i) = pack16<T>(o);
}

hipError_t launch_apply_norm(const void* x, const float* stats, const void* gamma, const void* beta, int64_t M,
                             int64_t K, int dtype, void* y, hipStream_t s) {
    const int64_t epl = dtype == 0 ? 4 : 8;
    const dim3 grid((unsigned)((M * K / epl + 255) / 256));
    if (dtype == 0)
        apply_norm_kernel<float><<<grid, 256, 0, s>>>((const float*)x, stats, (const float*)gamma,
                                                      (const float*)beta, M, K, (float*)y);
    else
        apply_norm_kernel<__bf16><<<grid, 256, 0, s>>>((const __bf16*)x, stats, (const __bf16*)gamma,
                                                       (const __bf16*)beta, M, K, (__bf16*)y);
    return hipGetLastError();
}

}  // namespace dn
