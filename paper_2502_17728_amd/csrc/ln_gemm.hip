// ln_gemm.hip -- deferred LayerNorm -> Linear (Sec. II-A, Eq. (5)) and the
// plain GEMM comparator, sharing one MFMA main loop; plus the decode-shaped
// deferred kernel and the static-weight preparation.
//
// Deferred LayerNorm -> Linear.  With W' = Diag(gamma) W (static, folded once),
// Eq. (5) with the centering applied after the product reads
//     out[m][n] = rstd_m * (x_m . W'[:, n] - mean_m * c_n) + b_n,
//     c = 1^T W' (column sums of the rounded W'),  b = beta W + bias,
// because x (I - E/n) = x - mean_m 1.  The product acc = x . W' runs on MFMA
// over the raw x tiles; the same x fragments, already in registers for the
// MFMA, feed the row moments (sum x, sum x^2) on the VALU -- the paper's
// "collective sub-operation" running concurrently with the matmul -- and the
// epilogue applies the normalization once before the single rounded store.
#include "dn_device.hpp"
#include "dn_launch.hpp"

namespace dn {

enum class Epi { kLnDeferred, kGemm };

struct MainArgs {
    const void* A;  // [batch][M][K]
    const void* B;  // NK: [batch][N][K];  KN: [batch][K][N]
    void* C;        // [batch][M][N]
    int64_t M, K, N;
    int64_t sA, sB, sC;   // batch strides, elements
    const float* c_col;   // LN: c[N]
    const float* b_col;   // LN: b[N]
    float eps;            // LN
    const void* bias;     // GEMM: bias[N] in the element type, or null
    int a_causal;         // GEMM: A lower-triangular, skip k > row
};

// Wait until every global->LDS copy issued by this wave has landed.
__device__ __forceinline__ void wait_vm() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

template <class T, int BM, int BN, int WM, int WN, bool B_KN, Epi EPI>
__global__ __launch_bounds__(WM* WN* kWave) void main_loop_kernel(MainArgs p) {
    constexpr int NW = WM * WN;
    constexpr int EPL = elem<T>::per16;  // elements per lane per chunk
    constexpr int KC = elem<T>::kchunk;  // k per chunk
    constexpr int KB = 2;                // chunks per stage along k
    constexpr int BK = KC * KB;
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int FM = WTM / 16, FN = WTN / 16;
    constexpr int A_CH = (BM / 16) * KB, B_CH = (BN / 16) * KB;
    constexpr int STAGE = (A_CH + B_CH) * kChunkBytes;
    constexpr bool LN = EPI == Epi::kLnDeferred;
    static_assert(FM >= 1 && FN >= 1 && BM % (16 * WM) == 0 && BN % (16 * WN) == 0, "tile");
    static_assert(!B_KN || sizeof(T) == 2, "KN staging is bf16 only");
    static_assert(A_CH % NW == 0 && B_CH % NW == 0, "every wave issues the same number of chunk copies");
    static_assert(EPI != Epi::kLnDeferred || WN <= KB, "moments split: one k-chunk column per wave column");

    __shared__ __attribute__((aligned(1024))) char smem[2 * STAGE];
    __shared__ float red[LN ? 2 * WN * BM : 1];
    __shared__ float row_mean[LN ? BM : 1], row_rstd[LN ? BM : 1];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;
    const int64_t M = p.M, K = p.K, N = p.N;

    // ---- tile selection: XCD-contiguous logical ids, grouped along M
    const int tiles_m = (int)((M + BM - 1) / BM), tiles_n = (int)((N + BN - 1) / BN);
    const int t = xcd_contiguous(blockIdx.x, gridDim.x);
    constexpr int GM = 8;
    const int group = GM * tiles_n, gid = t / group, first = gid * GM;
    const int gsz = min(tiles_m - first, GM);
    int pm = first + (t % group) % gsz;
    const int pn = (t % group) / gsz;
    if (p.a_causal) pm = tiles_m - 1 - pm;  // longest k-ranges first
    const int64_t m0 = (int64_t)pm * BM, n0 = (int64_t)pn * BN;

    const T* A = reinterpret_cast<const T*>(p.A) + (int64_t)blockIdx.y * p.sA;
    const T* B = reinterpret_cast<const T*>(p.B) + (int64_t)blockIdx.y * p.sB;
    T* C = reinterpret_cast<T*>(p.C) + (int64_t)blockIdx.y * p.sC;

    const int64_t kend = p.a_causal ? min(K, m0 + BM) : K;
    const int nst = (int)((kend + BK - 1) / BK);

    // ---- global -> LDS staging
    auto issue_dma = [&](int s, int buf) {
        char* base = smem + buf * STAGE;
        const int64_t k0 = (int64_t)s * BK;
#pragma unroll
        for (int j = 0; j < A_CH / NW; ++j) {
            const int c = wave + j * NW;
            const int mb = c / KB, kb = c % KB;
            const int64_t row = min(m0 + mb * 16 + (lane & 15), M - 1);
            const int64_t kk = min(k0 + kb * KC + (lane >> 4) * EPL, K - EPL);
            g2lds16(A + row * K + kk, lds_ptr(base + c * kChunkBytes));
        }
        if constexpr (!B_KN) {
#pragma unroll
            for (int j = 0; j < B_CH / NW; ++j) {
                const int c = wave + j * NW;
                const int nb = c / KB, kb = c % KB;
                const int64_t row = min(n0 + nb * 16 + (lane & 15), N - 1);
                const int64_t kk = min(k0 + kb * KC + (lane >> 4) * EPL, K - EPL);
                g2lds16(B + row * K + kk, lds_ptr(base + (A_CH + c) * kChunkBytes));
            }
        }
    };

    // B in [K][N] layout: 8x8 blocks through registers, transposed into chunk order.
    constexpr int KN_BLOCKS = (BK / 8) * (BN / 8);
    constexpr int KN_PER_T = (KN_BLOCKS + NW * kWave - 1) / (NW * kWave);
    u32x4 knreg[B_KN ? KN_PER_T : 1][8];
    auto kn_load = [&](int s) {
        if constexpr (B_KN) {
            const int64_t k0 = (int64_t)s * BK;
#pragma unroll
            for (int j = 0; j < KN_PER_T; ++j) {
                const int blk = tid + j * NW * kWave;
                if (blk < KN_BLOCKS) {
                    const int kb8 = blk / (BN / 8), nb8 = blk % (BN / 8);
                    const int64_t n = n0 + nb8 * 8;
#pragma unroll
                    for (int r = 0; r < 8; ++r) {
                        const int64_t k = k0 + kb8 * 8 + r;
                        if (k < K && n < N)
                            knreg[j][r] = ld16(B + k * N + n);
                        else
                            knreg[j][r] = u32x4{0, 0, 0, 0};
                    }
                }
            }
        }
    };
    auto kn_store = [&](int buf) {
        if constexpr (B_KN) {
            char* base = smem + buf * STAGE + A_CH * kChunkBytes;
#pragma unroll
            for (int j = 0; j < KN_PER_T; ++j) {
                const int blk = tid + j * NW * kWave;
                if (blk < KN_BLOCKS) {
                    const int kb8 = blk / (BN / 8), nb8 = blk % (BN / 8);
                    u32x4 col[8];
                    transpose8x8_bf16(knreg[j], col);
                    const int k8 = kb8 * 8;
#pragma unroll
                    for (int c = 0; c < 8; ++c) {
                        const int n = nb8 * 8 + c;
                        const int chunk = (n >> 4) * KB + k8 / KC;
                        const int l2 = (n & 15) + 16 * ((k8 % KC) / 8);
                        *reinterpret_cast<DN_LDS u32x4*>(lds_ptr(base + chunk * kChunkBytes + l2 * 16)) = col[c];
                    }
                }
            }
        }
    };

    f32x4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    float s1[FM], s2[FM];
#pragma unroll
    for (int i = 0; i < FM; ++i) s1[i] = s2[i] = 0.f;

    issue_dma(0, 0);
    kn_load(0);
    kn_store(0);
    wait_vm();
    __syncthreads();

    for (int s = 0; s < nst; ++s) {
        const int buf = s & 1;
        const char* base = smem + buf * STAGE;
        u32x4 af[FM][KB], bfr[FN][KB];
#pragma unroll
        for (int fm = 0; fm < FM; ++fm)
#pragma unroll
            for (int kb = 0; kb < KB; ++kb)
                af[fm][kb] = lds_ld16(lds_ptr((char*)base + ((wm * FM + fm) * KB + kb) * kChunkBytes + lane * 16));
#pragma unroll
        for (int fn = 0; fn < FN; ++fn)
#pragma unroll
            for (int kb = 0; kb < KB; ++kb)
                bfr[fn][kb] = lds_ld16(
                    lds_ptr((char*)base + (A_CH + (wn * FN + fn) * KB + kb) * kChunkBytes + lane * 16));

        if (s + 1 < nst) {
            issue_dma(s + 1, buf ^ 1);
            kn_load(s + 1);
        }

        const int64_t k0 = (int64_t)s * BK;
        if (k0 + BK > K) {  // K tail: zero the lane-chunks past K (their loads were clamped)
#pragma unroll
            for (int kb = 0; kb < KB; ++kb) {
                if (k0 + kb * KC + (lane >> 4) * EPL >= K) {
#pragma unroll
                    for (int fm = 0; fm < FM; ++fm) af[fm][kb] = u32x4{0, 0, 0, 0};
#pragma unroll
                    for (int fn = 0; fn < FN; ++fn) bfr[fn][kb] = u32x4{0, 0, 0, 0};
                }
            }
        }
        if constexpr (!LN && sizeof(T) == 2) {
            if (p.a_causal && k0 + BK > m0) {  // stage reaches the diagonal: A[i][j] = 0 for j > i
#pragma unroll
                for (int fm = 0; fm < FM; ++fm) {
                    const int64_t row = m0 + (wm * FM + fm) * 16 + (lane & 15);
#pragma unroll
                    for (int kb = 0; kb < KB; ++kb) {
                        const int64_t kk = k0 + kb * KC + (lane >> 4) * EPL;
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            uint32_t w = af[fm][kb][e];
                            if (kk + 2 * e > row) w &= 0xffff0000u;
                            if (kk + 2 * e + 1 > row) w &= 0x0000ffffu;
                            af[fm][kb][e] = w;
                        }
                    }
                }
            }
        }

        if constexpr (LN) {  // row moments from the operand registers, each element once per workgroup
#pragma unroll
            for (int fm = 0; fm < FM; ++fm)
#pragma unroll
                for (int kb = 0; kb < KB; ++kb)
                    if (kb % WN == wn) chunk_moments<T>(af[fm][kb], s1[fm], s2[fm]);
        }

#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
            for (int fm = 0; fm < FM; ++fm)
#pragma unroll
                for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = mfma_chunk<T>(af[fm][kb], bfr[fn][kb], acc[fm][fn]);

        if (s + 1 < nst) kn_store(buf ^ 1);
        wait_vm();
        __syncthreads();
    }

    // ---- epilogue
    if constexpr (LN) {
#pragma unroll
        for (int fm = 0; fm < FM; ++fm) {
            const float a = sum_lane_groups(s1[fm]);
            const float b = sum_lane_groups(s2[fm]);
            if (lane < 16) {
                const int r = wm * WTM + fm * 16 + lane;
                red[(0 * WN + wn) * BM + r] = a;
                red[(1 * WN + wn) * BM + r] = b;
            }
        }
        __syncthreads();
        for (int r = tid; r < BM; r += NW * kWave) {
            float a = 0.f, b = 0.f;
#pragma unroll
            for (int w = 0; w < WN; ++w) {
                a += red[(0 * WN + w) * BM + r];
                b += red[(1 * WN + w) * BM + r];
            }
            const float mean = a / (float)K;
            const float var = __builtin_fmaxf(b / (float)K - mean * mean, 0.f);
            row_mean[r] = mean;
            row_rstd[r] = 1.0f / __builtin_sqrtf(var + p.eps);
        }
        __syncthreads();
    }

#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
        const int64_t n = n0 + wn * WTN + fn * 16 + (lane & 15);
        const int64_t nc = min(n, N - 1);
        float cn = 0.f, bn = 0.f;
        if constexpr (LN) {
            cn = p.c_col[nc];
            bn = p.b_col[nc];
        } else {
            if (p.bias) bn = to_f32<T>(reinterpret_cast<const T*>(p.bias)[nc]);
        }
#pragma unroll
        for (int fm = 0; fm < FM; ++fm) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int rl = wm * WTM + fm * 16 + 4 * (lane >> 4) + i;
                const int64_t r = m0 + rl;
                float v = acc[fm][fn][i];
                if constexpr (LN) {
                    v = __builtin_fmaf(-row_mean[rl], cn, v);
                    v = __builtin_fmaf(row_rstd[rl], v, bn);
                } else {
                    v += bn;
                }
                if (r < M && n < N) C[r * N + n] = from_f32<T>(v);
            }
        }
    }
}

// =============================================================================
// Decode-shaped deferred LN -> Linear: M <= 16 tokens, bf16.
// The work is streaming W' from HBM, so each workgroup owns 16 output columns
// and its four waves split K; one 16x16x32 MFMA per 32-k chunk multiplies the
// (zero-padded) x rows with W' read straight from HBM into operand registers.
// The row moments ride on the otherwise idle matrix core: with B = all-ones
// the product gives sum_k x[m][k] in every column, and with B = x itself the
// Gram matrix x x^T whose diagonal is sum_k x[m][k]^2.
// =============================================================================
constexpr int kDecUnroll = 8;

__global__ __launch_bounds__(256) void ln_decode_bf16_kernel(const __bf16* __restrict__ x,
                                                             const __bf16* __restrict__ Wt,
                                                             const float* __restrict__ c_col,
                                                             const float* __restrict__ b_col, int M,
                                                             int64_t K, int64_t N, float eps,
                                                             __bf16* __restrict__ out) {
    __shared__ f32x4 part[3][4][kWave];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t n0 = (int64_t)blockIdx.x * 16;
    const int row = lane & 15;
    const bool row_ok = row < M;
    const int64_t n = min(n0 + (lane & 15), N - 1);
    const __bf16* xr = x + (int64_t)(row_ok ? row : 0) * K;
    const __bf16* wr = Wt + n * K;

    const int64_t nchunks = (K + 31) / 32;
    const int64_t per = (nchunks + 3) / 4;
    const int64_t c_begin = wave * per, c_end = min(nchunks, c_begin + per);

    const u32x4 ones = {0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u};
    const u32x4 zero = {0, 0, 0, 0};
    f32x4 acc = {0.f, 0.f, 0.f, 0.f}, sx = acc, sxx = acc;

    int64_t c = c_begin;
    for (; c + kDecUnroll <= c_end; c += kDecUnroll) {
        u32x4 a[kDecUnroll], b[kDecUnroll];
#pragma unroll
        for (int u = 0; u < kDecUnroll; ++u) {
            const int64_t kk = (c + u) * 32 + (lane >> 4) * 8;
            const bool ok = kk < K;
            b[u] = ok ? ld16(wr + kk) : zero;
            a[u] = (ok && row_ok) ? ld16(xr + kk) : zero;
        }
#pragma unroll
        for (int u = 0; u < kDecUnroll; ++u) {
            acc = mfma_chunk<__bf16>(a[u], b[u], acc);
            sx = mfma_chunk<__bf16>(a[u], ones, sx);
            sxx = mfma_chunk<__bf16>(a[u], a[u], sxx);
        }
    }
    for (; c < c_end; ++c) {
        const int64_t kk = c * 32 + (lane >> 4) * 8;
        const bool ok = kk < K;
        const u32x4 b = ok ? ld16(wr + kk) : zero;
        const u32x4 a = (ok && row_ok) ? ld16(xr + kk) : zero;
        acc = mfma_chunk<__bf16>(a, b, acc);
        sx = mfma_chunk<__bf16>(a, ones, sx);
        sxx = mfma_chunk<__bf16>(a, a, sxx);
    }
    part[0][wave][lane] = acc;
    part[1][wave][lane] = sx;
    part[2][wave][lane] = sxx;
    __syncthreads();
    if (wave == 0) {
        f32x4 tot[3];
#pragma unroll
        for (int q = 0; q < 3; ++q) {
            tot[q] = part[q][0][lane];
#pragma unroll
            for (int w = 1; w < 4; ++w) tot[q] += part[q][w][lane];
        }
        // Gram diagonal (r, r) sits in lane r + 16*(r>>2), element r&3.  This lane's
        // rows are r = 4*(l>>4) + i, so the source lane is 20*(l>>4) + i.
        float diag[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) diag[i] = __shfl(tot[2][i], 20 * (lane >> 4) + i);
        const int64_t col = n0 + (lane & 15);
        const float cn = c_col[n], bn = b_col[n];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = 4 * (lane >> 4) + i;
            const float mean = tot[1][i] / (float)K;
            const float var = __builtin_fmaxf(diag[i] / (float)K - mean * mean, 0.f);
            const float rstd = 1.0f / __builtin_sqrtf(var + eps);
            float v = __builtin_fmaf(-mean, cn, tot[0][i]);
            v = __builtin_fmaf(rstd, v, bn);
            if (r < M && col < N) out[(int64_t)r * N + col] = (__bf16)v;
        }
    }
}

// =============================================================================
// Static-weight preparation (off the per-token path).
// =============================================================================
// c[n] = sum_k round(gamma_k W[k][n]),  b[n] = sum_k beta_k W[k][n] + bias[n]; fp64 sums.
template <class T>
__global__ __launch_bounds__(256) void prep_colsum_kernel(const T* __restrict__ W, const T* __restrict__ gamma,
                                                          const T* __restrict__ beta, const T* __restrict__ bias,
                                                          int64_t K, int64_t N, float* __restrict__ c_col,
                                                          float* __restrict__ b_col) {
    const int64_t n = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (n >= N) return;
    double cs = 0.0, bs = 0.0;
    for (int64_t k = 0; k < K; ++k) {
        const float w = to_f32<T>(W[k * N + n]);
        const float wp = to_f32<T>(from_f32<T>(to_f32<T>(gamma[k]) * w));
        cs += (double)wp;
        if (beta) bs += (double)to_f32<T>(beta[k]) * (double)w;
    }
    if (bias) bs += (double)to_f32<T>(bias[n]);
    c_col[n] = (float)cs;
    b_col[n] = (float)bs;
}

// Wt'[n][k] = round(gamma_k W[k][n]) through a 64x64 LDS tile.
template <class T>
__global__ __launch_bounds__(256) void prep_transpose_kernel(const T* __restrict__ W, const T* __restrict__ gamma,
                                                             int64_t K, int64_t N, T* __restrict__ Wt) {
    __shared__ float tile[64][65];
    const int64_t k0 = (int64_t)blockIdx.y * 64, n0 = (int64_t)blockIdx.x * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    for (int r = ty; r < 64; r += 4) {
        const int64_t k = k0 + r, n = n0 + tx;
        if (k < K && n < N) tile[r][tx] = to_f32<T>(gamma[k]) * to_f32<T>(W[k * N + n]);
    }
    __syncthreads();
    for (int r = ty; r < 64; r += 4) {
        const int64_t n = n0 + r, k = k0 + tx;
        if (k < K && n < N) Wt[n * K + k] = from_f32<T>(tile[tx][r]);
    }
}

// =============================================================================
// Host launchers
// =============================================================================
static size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

PackedLayout packed_layout(int64_t K, int64_t N, int dtype) {
    PackedLayout L;
    const size_t es = dtype == 0 ? 4 : 2;
    L.wt_off = 0;
    L.wt_bytes = (size_t)K * (size_t)N * es;
    L.c_off = align256(L.wt_bytes);
    L.b_off = L.c_off + align256((size_t)N * 4);
    L.total = L.b_off + align256((size_t)N * 4);
    return L;
}

template <class T>
static hipError_t prepare_t(const void* W, const void* gamma, const void* beta, const void* bias, int64_t K,
                            int64_t N, void* packed, hipStream_t s) {
    const PackedLayout L = packed_layout(K, N, sizeof(T) == 4 ? 0 : 1);
    char* base = reinterpret_cast<char*>(packed);
    dim3 g1((unsigned)((N + 255) / 256));
    prep_colsum_kernel<T><<<g1, 256, 0, s>>>((const T*)W, (const T*)gamma, (const T*)beta, (const T*)bias, K, N,
                                             (float*)(base + L.c_off), (float*)(base + L.b_off));
    dim3 g2((unsigned)((N + 63) / 64), (unsigned)((K + 63) / 64));
    prep_transpose_kernel<T><<<g2, 256, 0, s>>>((const T*)W, (const T*)gamma, K, N, (T*)(base + L.wt_off));
    return hipGetLastError();
}

hipError_t launch_ln_prepare(const void* W, const void* gamma, const void* beta, const void* bias, int64_t K,
                             int64_t N, int dtype, void* packed, hipStream_t s) {
    if (dtype == 0) return prepare_t<float>(W, gamma, beta, bias, K, N, packed, s);
    return prepare_t<__bf16>(W, gamma, beta, bias, K, N, packed, s);
}

template <class T, int BM, int BN, int WM, int WN, bool B_KN, Epi EPI>
static hipError_t run_main(const MainArgs& a, int64_t batch, hipStream_t s) {
    const int64_t tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
    dim3 grid((unsigned)tiles, (unsigned)batch);
    main_loop_kernel<T, BM, BN, WM, WN, B_KN, EPI><<<grid, WM * WN * kWave, 0, s>>>(a);
    return hipGetLastError();
}

hipError_t launch_ln_linear_deferred(const void* x, const void* packed, int64_t M, int64_t K, int64_t N,
                                     int dtype, float eps, void* out, hipStream_t s) {
    const PackedLayout L = packed_layout(K, N, dtype);
    const char* base = reinterpret_cast<const char*>(packed);
    if (dtype == 1 && M <= 16) {
        ln_decode_bf16_kernel<<<dim3((unsigned)((N + 15) / 16)), 256, 0, s>>>(
            (const __bf16*)x, (const __bf16*)(base + L.wt_off), (const float*)(base + L.c_off),
            (const float*)(base + L.b_off), (int)M, K, N, eps, (__bf16*)out);
        return hipGetLastError();
    }
    MainArgs a{};
    a.A = x;
    a.B = base + L.wt_off;
    a.C = out;
    a.M = M;
    a.K = K;
    a.N = N;
    a.c_col = (const float*)(base + L.c_off);
    a.b_col = (const float*)(base + L.b_off);
    a.eps = eps;
    if (dtype == 0) return run_main<float, 32, 64, 2, 2, false, Epi::kLnDeferred>(a, 1, s);
    return run_main<__bf16, 128, 128, 2, 2, false, Epi::kLnDeferred>(a, 1, s);
}

hipError_t launch_gemm(const void* A, const void* B, const void* bias, int64_t batch, int64_t M, int64_t K,
                       int64_t N, int b_layout, int a_causal, int dtype, void* C, hipStream_t s) {
    MainArgs a{};
    a.A = A;
    a.B = B;
    a.C = C;
    a.M = M;
    a.K = K;
    a.N = N;
    a.sA = M * K;
    a.sB = K * N;
    a.sC = M * N;
    a.bias = bias;
    a.a_causal = a_causal;
    if (dtype == 0) return run_main<float, 32, 64, 2, 2, false, Epi::kGemm>(a, batch, s);
    if (b_layout == 1) return run_main<__bf16, 128, 128, 2, 2, false, Epi::kGemm>(a, batch, s);
    return run_main<__bf16, 128, 128, 2, 2, true, Epi::kGemm>(a, batch, s);
}

}  // namespace dn
