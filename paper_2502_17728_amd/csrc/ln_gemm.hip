// ln_gemm.hip -- deferred LayerNorm -> Linear (Sec. II-A, Eq. (5)) and the
// plain GEMM comparator, sharing the same MFMA main loops; plus the
// decode-shaped deferred kernel and the static-weight preparation.
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
//
// Deferred RMSNorm -> Linear (Eq. (6)) is the same computation with the mean
// taken as zero: rstd_m = 1/sqrt(sum x^2 / K + eps) and no mean_m * c_n term,
// so every kernel here serves it through one flag (MainArgs::rms).
//
// Packed weight layout (written by the prepare kernels, read by every LN
// kernel and by gemm with b_layout = 2).  W'^T is cut into 16-row x 64-byte
// fragment chunks (16 output features x 32 bf16 / 16 fp32 of K), stored in
// chunk order [N_pad/16][K_pad/kchunk][64 lanes][16 B], zero padded.  One
// chunk is 1 KiB, contiguous, already in MFMA operand order: a wave copies it
// with one fully coalesced instruction, and a lane's 16 bytes are its operand.
#include <algorithm>
#include <atomic>
#include <cstdlib>
#include <mutex>
#include <type_traits>

#include "dn_device.hpp"
#include "dn_launch.hpp"

namespace dn {

// kLnDeferred: out = rstd (acc - mean c) + b.  kSwiGlu: the same for the gate
// and up columns, which the packed weights interleave in 16-column blocks (gate
// block j, then up block j), combined as h = SiLU(gate) * up.  kGemm: acc + bias.
// kLnOnLoad (ablation, no deferral): statistics from a pre-pass, each x fragment
// normalized as it is loaded, xh = (x - mean) rstd rounded to bf16, then out =
// xh . W' + b -- the plain fused LayerNorm -> Linear the deferred form replaces.
enum class Epi { kLnDeferred, kGemm, kSwiGlu, kLnOnLoad };
enum class BMode { kKN, kNK, kPacked };

struct MainArgs {
    const void* A;  // [batch][M][K]
    const void* B;  // kKN: [batch][K][N];  kNK: [batch][N][K];  kPacked: packed chunks
    void* C;        // [batch][M][N]
    int64_t M, K, N;
    int64_t sA, sB, sC;   // batch strides, elements
    int64_t kchunks;      // kPacked: K_pad / kchunk
    int64_t nblocks;      // kPacked: N_pad / 16
    const float* c_col;   // LN: c[N]
    const float* b_col;   // LN: b[N]
    float eps;            // LN
    int rms;              // LN: RMSNorm statistics (Eq. (6)): mean taken as 0
    int64_t n_out;        // kSwiGlu: output features (row stride of C); N counts packed columns
    const float* row_stats;  // LN, serial ablation: (mean, rstd) per row from a pre-pass, or null
    float* stats_out;        // LN: (mean, rstd) per row as reduced by the kernel, written once per row, or null
    const void* bias;     // GEMM: bias[N] in the element type, or null
    int a_causal;         // GEMM: A lower-triangular, skip k > row
    // LN, shared row moments (pipelined kernel): the workgroups that share a row block each
    // reduce a share of its rows and exchange them through mom_slots (2 words per row,
    // stamped with mom_call); null = every workgroup reduces all its rows itself
    unsigned long long* mom_slots;
    uint32_t mom_call;
    uint32_t mom_wait_ticks;  // bound of the wait for the peers' shares, s_memrealtime ticks (100 MHz)
};

// SiLU(z) = z / (1 + e^-z) with e^-z = 2^(-z log2 e) on the hardware exponential;
// below z ~ -88 that overflows to +inf and the quotient is -0, the limit.
constexpr float kLog2eF = 1.4426950408889634f;
__device__ __forceinline__ float silu(float z) { return z / (1.0f + __builtin_amdgcn_exp2f(-z * kLog2eF)); }

// ---------------------------------------------------------------------------- waits
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
    // gfx9 s_waitcnt: vmcnt[3:0] bits 3:0, vmcnt[5:4] bits 15:14, expcnt bits 6:4, lgkmcnt bits 11:8
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4)); }
__device__ __forceinline__ void wait_vm() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
__device__ __forceinline__ void block_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Address of packed chunk (nb, kc), lane `lane` (bytes from the packed base).
__device__ __forceinline__ int64_t packed_chunk(int64_t nb, int64_t kc, int64_t kchunks, int lane) {
    return ((nb * kchunks + kc) * kWave + lane) * 16;
}

// =============================================================================
// General main loop: 128x128 (bf16) or 32x64 (fp32) tiles.  Used for problems
// too small for the 256x256 kernel, for K not a multiple of 64, for fp32, for
// batched products and for B in [K][N] layout.
// NST = 2: two LDS stages, the copy of stage s+1 issued while stage s is read.
// NST > 2 (chunk copies only, NST >= 3): a ring of NST stages whose copies run
// NST-1 stages ahead, with each stage's fragments read while the previous
// stage's products run, for tiles whose per-stage matrix work is too short to
// cover the latency of a copy (the fp32 tiles: 16 fp32 MFMAs per wave and stage).
// =============================================================================
template <class T, int BM, int BN, int WM, int WN, BMode BMODE, Epi EPI, int NST = 2, int KBT = 2>
__global__ __launch_bounds__(WM* WN* kWave) void main_loop_kernel(MainArgs p) {
    constexpr int NW = WM * WN;
    constexpr int EPL = elem<T>::per16;  // elements per lane per chunk
    constexpr int KC = elem<T>::kchunk;  // k per chunk
    constexpr int KB = KBT;              // chunks per stage along k
    constexpr int BK = KC * KB;
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int FM = WTM / 16, FN = WTN / 16;
    constexpr int A_CH = (BM / 16) * KB, B_CH = (BN / 16) * KB;
    constexpr int STAGE = (A_CH + B_CH) * kChunkBytes;
    constexpr bool LN = EPI != Epi::kGemm;
    constexpr bool SW = EPI == Epi::kSwiGlu;
    constexpr bool B_KN = BMODE == BMode::kKN;
    static_assert(FM >= 1 && FN >= 1 && BM % (16 * WM) == 0 && BN % (16 * WN) == 0, "tile");
    static_assert(!B_KN || sizeof(T) == 2, "KN staging is bf16 only");
    static_assert(A_CH % NW == 0 && B_CH % NW == 0, "every wave issues the same number of chunk copies");
    static_assert(!LN || WN <= KB, "moments split: one k-chunk column per wave column");
    static_assert(!SW || FN % 2 == 0, "gate/up fragment pairs");
    static_assert(NST == 2 || (NST >= 3 && !B_KN), "the deep ring moves whole chunks only");

    __shared__ __attribute__((aligned(1024))) char smem[NST * STAGE];
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

    // ---- global -> LDS staging.  The deep ring issues its copies from inline
    // assembly (the compiler does not track them, so it adds no wait of its own
    // for all outstanding copies before the LDS reads of other stages) and counts
    // its waits by hand: every call issues exactly A_CH / NW + B_CH / NW copies.
    auto copy = [&](const void* g, char* l) {
        if constexpr (NST > 2)
            g2lds16_async(g, lds_addr32(l));
        else
            g2lds16(g, lds_ptr(l));
    };
    auto issue_dma = [&](int s, int buf) {
        char* base = smem + buf * STAGE;
        const int64_t k0 = (int64_t)s * BK;
#pragma unroll
        for (int j = 0; j < A_CH / NW; ++j) {
            const int c = wave + j * NW;
            const int mb = c / KB, kb = c % KB;
            const int64_t row = min(m0 + mb * 16 + (lane & 15), M - 1);
            const int64_t kk = min(k0 + kb * KC + (lane >> 4) * EPL, K - EPL);
            copy(A + row * K + kk, base + c * kChunkBytes);
        }
        if constexpr (BMODE == BMode::kNK) {
#pragma unroll
            for (int j = 0; j < B_CH / NW; ++j) {
                const int c = wave + j * NW;
                const int nb = c / KB, kb = c % KB;
                const int64_t row = min(n0 + nb * 16 + (lane & 15), N - 1);
                const int64_t kk = min(k0 + kb * KC + (lane >> 4) * EPL, K - EPL);
                copy(B + row * K + kk, base + (A_CH + c) * kChunkBytes);
            }
        }
        if constexpr (BMODE == BMode::kPacked) {
#pragma unroll
            for (int j = 0; j < B_CH / NW; ++j) {
                const int c = wave + j * NW;
                const int nb = c / KB, kb = c % KB;
                const int64_t gnb = min(n0 / 16 + nb, p.nblocks - 1);
                const int64_t gkc = min((int64_t)s * KB + kb, p.kchunks - 1);
                copy(reinterpret_cast<const char*>(p.B) + packed_chunk(gnb, gkc, p.kchunks, lane),
                     base + (A_CH + c) * kChunkBytes);
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

    constexpr int PER = (A_CH + (B_KN ? 0 : B_CH)) / NW;  // copies per wave per stage

    // Fragments of the stage in LDS slot `buf` (stage s: zero past K, causal mask), and the
    // stage's work on them: the row moments (each element once per workgroup) and the MFMAs.
    auto read_frags = [&](int buf, u32x4(&af)[FM][KB], u32x4(&bfr)[FN][KB]) {
        const char* base = smem + buf * STAGE;
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
    };
    // TAIL: the stage may reach past K (only the last one can).  MOM: 0 -- the moments of the
    // chunks whose index matches the wave column (each element once per workgroup); 1 -- of
    // every chunk (the deep ring gives them all to wave column 0); 2 -- none.
    auto compute = [&](int s, u32x4(&af)[FM][KB], u32x4(&bfr)[FN][KB], auto tail, auto mom) {
        const int64_t k0 = (int64_t)s * BK;
        if (decltype(tail)::value && k0 + BK > K) {  // K tail: zero the lane-chunks past K (their loads were clamped)
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
        constexpr int MOM = decltype(mom)::value;
        if constexpr (LN && MOM < 2) {  // row moments from the operand registers, each element once per workgroup
#pragma unroll
            for (int fm = 0; fm < FM; ++fm)
#pragma unroll
                for (int kb = 0; kb < KB; ++kb)
                    if (MOM == 1 || kb % WN == wn) chunk_moments<T>(af[fm][kb], s1[fm], s2[fm]);
        }
        if constexpr (sizeof(T) == 4) {
            // fp32: a chunk is four dependent 16x16x4 products on one accumulator; taking the
            // chunk's k-slices in the outer loop interleaves the FM x FN independent chains
#pragma unroll
            for (int kb = 0; kb < KB; ++kb)
#pragma unroll
                for (int j = 0; j < 4; ++j)
#pragma unroll
                    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
                        for (int fn = 0; fn < FN; ++fn)
                            acc[fm][fn] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                                __uint_as_float(af[fm][kb][j]), __uint_as_float(bfr[fn][kb][j]), acc[fm][fn], 0, 0, 0);
        } else {
#pragma unroll
            for (int kb = 0; kb < KB; ++kb)
#pragma unroll
                for (int fm = 0; fm < FM; ++fm)
#pragma unroll
                    for (int fn = 0; fn < FN; ++fn)
                        acc[fm][fn] = mfma_chunk<T>(af[fm][kb], bfr[fn][kb], acc[fm][fn]);
        }
    };

    if constexpr (NST > 2) {
        // Deep ring.  Stages 0 .. NST-2 are in flight before the loop; iteration s waits for
        // stage s+1, refills the slot of stage s-1 (read two iterations ago, consumed one ago)
        // and reads stage s+1's fragments while stage s's products run.  Stages past the last
        // re-copy the last one into slots that are never read, so every iteration issues the
        // same count of copies and the waits are exact.  Only the last stage can reach past K,
        // and the row moments go to wave column 0 alone (a uniform choice made once, outside
        // the loop), so the loop body has no branch: its products, fragment reads and moment
        // arithmetic form one block that the scheduler interleaves.
        auto deep = [&](auto mom) {
#pragma unroll
            for (int j = 0; j < NST - 1; ++j) issue_dma(min(j, nst - 1), j);
            wait_vmcnt<(NST - 2) * PER>();  // stage 0
            block_barrier();
            u32x4 af[2][FM][KB], bfr[2][FN][KB];
            read_frags(0, af[0], bfr[0]);
            auto body = [&](int ss, auto h, auto tail) {
                constexpr int H = decltype(h)::value;
                wait_vmcnt<(NST - 3) * PER>();  // this wave's copies of stage ss+1 have landed
                block_barrier();                // every wave's have
                issue_dma(min(ss + NST - 1, nst - 1), (ss + NST - 1) % NST);  // slot of stage ss-1
                if (!decltype(tail)::value || ss + 1 < nst) read_frags((ss + 1) % NST, af[H ^ 1], bfr[H ^ 1]);
                compute(ss, af[H], bfr[H], tail, mom);
            };
            using h0 = std::integral_constant<int, 0>;
            using h1 = std::integral_constant<int, 1>;
            int ss = 0;
            for (; ss + 2 <= nst - 1; ss += 2) {  // stages before the last: no tail, no exit test inside
                body(ss, h0{}, std::false_type{});
                body(ss + 1, h1{}, std::false_type{});
            }
            if (ss < nst - 1) {
                body(ss, h0{}, std::false_type{});
                body(ss + 1, h1{}, std::true_type{});
            } else {
                body(ss, h0{}, std::true_type{});
            }
            wait_vmcnt<0>();  // no copy into LDS may outlive the workgroup
        };
        if (LN && __builtin_amdgcn_readfirstlane(wn) == 0)
            deep(std::integral_constant<int, 1>{});
        else
            deep(std::integral_constant<int, 2>{});
    } else {
        issue_dma(0, 0);
        kn_load(0);
        kn_store(0);
        wait_vm();
        __syncthreads();
        for (int s = 0; s < nst; ++s) {
            const int buf = s & 1;
            u32x4 af[FM][KB], bfr[FN][KB];
            read_frags(buf, af, bfr);
            if (s + 1 < nst) {
                issue_dma(s + 1, buf ^ 1);
                kn_load(s + 1);
            }
            compute(s, af, bfr, std::true_type{}, std::integral_constant<int, 0>{});
            if (s + 1 < nst) kn_store(buf ^ 1);
            wait_vm();
            __syncthreads();
        }
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
            if (p.row_stats) {  // serial ablation: the pre-pass statistics replace the moments
                const int64_t rr = min(m0 + r, M - 1);
                row_mean[r] = p.row_stats[2 * rr];
                row_rstd[r] = p.row_stats[2 * rr + 1];
                continue;
            }
            float a = 0.f, b = 0.f;
#pragma unroll
            for (int w = 0; w < WN; ++w) {
                a += red[(0 * WN + w) * BM + r];
                b += red[(1 * WN + w) * BM + r];
            }
            const float mean = p.rms ? 0.f : a / (float)K;
            row_mean[r] = mean;
            row_rstd[r] = rstd_from_moments(b / (float)K, mean, p.eps);
            if (p.stats_out && pn == 0 && m0 + r < M) {  // one tile per row block exports them
                p.stats_out[2 * (m0 + r)] = mean;
                p.stats_out[2 * (m0 + r) + 1] = row_rstd[r];
            }
        }
        __syncthreads();
    }

    if constexpr (SW) {
        // fragment 2j holds gate columns, 2j+1 the up columns of the same outputs
        const int64_t nw = n0 + wn * WTN;  // packed column of the wave's first fragment (multiple of 32)
#pragma unroll
        for (int j = 0; j < FN / 2; ++j) {
            const int64_t ng = min(nw + 2 * j * 16 + (lane & 15), N - 1), nu = min(ng + 16, N - 1);
            const int64_t o = nw / 2 + j * 16 + (lane & 15);
            const float cg = p.c_col[ng], bg = p.b_col[ng], cu = p.c_col[nu], bu = p.b_col[nu];
#pragma unroll
            for (int fm = 0; fm < FM; ++fm) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int rl = wm * WTM + fm * 16 + 4 * (lane >> 4) + i;
                    const int64_t r = m0 + rl;
                    const float mu = row_mean[rl], rs = row_rstd[rl];
                    const float g = __builtin_fmaf(rs, __builtin_fmaf(-mu, cg, acc[fm][2 * j][i]), bg);
                    const float u = __builtin_fmaf(rs, __builtin_fmaf(-mu, cu, acc[fm][2 * j + 1][i]), bu);
                    if (r < M && o < p.n_out) C[r * p.n_out + o] = from_f32<T>(silu(g) * u);
                }
            }
        }
        return;
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
// Large-problem main loop (bf16, packed B, K % 64 == 0): 256x256 tiles, eight
// waves as 4 x 2, each wave 64 x 128 of the output.
//
// Copies.  The L2 -> CU path is limited by cache lines per instruction: a wave
// instruction touching 16 half lines moves about half of what one touching 8
// full lines does.  A (activations, row-major) is therefore copied as 8 rows
// x 128 bytes per instruction (BK = 64), and the packed B as one contiguous
// KiB.  A's 16-byte pieces land XOR-swizzled, piece p of tile row r at slot
// p ^ f(r) with f(r) = (r & 7) ^ ((r >> 3) & 1): any 8 or 16 consecutive rows
// read at one piece index hit distinct banks, so the fragment reads are
// conflict-free.
//
// Pipeline.  Two 64 KiB stages.  A stage is consumed in two halves (k 0-31,
// 32-63): the MFMAs of one half run while the next half's fragments are read
// from LDS.  The copy of stage s+2 is issued right after the barrier in the
// middle of stage s (when every wave has finished reading stage s), so it has
// a whole stage of MFMA time to land.
// =============================================================================
constexpr int kSgValu = 0x002, kSgMfma = 0x008, kSgDsRead = 0x100;
// cache-policy operand of the buffer stores: non-temporal
constexpr int kStoreStream = 2;

// xh = x r + nb for the 8 bf16 of a fragment chunk, rounded once to bf16.
__device__ __forceinline__ u32x4 normalize_chunk(const u32x4& a, float r, float nb) {
    const uint32_t w[4] = {a.x, a.y, a.z, a.w};
    uint32_t o[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
        o[j] = pack_bf16(__builtin_fmaf(bf_lo(w[j]), r, nb), __builtin_fmaf(bf_hi(w[j]), r, nb));
    return u32x4{o[0], o[1], o[2], o[3]};
}

__device__ __forceinline__ int a_swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

template <Epi EPI, int WM, int WN, int BM = 256, int BN = 256>
__global__ __launch_bounds__(WM* WN* kWave) void pipe_kernel(MainArgs p, int group) {
    constexpr int NW = WM * WN;
    static_assert(WN == 2, "the two wave columns split each row fragment's moments");
    constexpr int BK = 64;                        // bf16 elements per stage (128 B per row)
    constexpr int WTM = BM / WM, WTN = BN / WN;   // 64 x 128 per wave
    constexpr int FM = WTM / 16, FN = WTN / 16;   // 4 x 8 output fragments
    constexpr int A_BYTES = BM * 128;             // 32 KiB
    constexpr int STAGE = A_BYTES + BN / 16 * 2 * kChunkBytes;  // + 32 KiB of B chunks
    constexpr int A_INS = BM / 8 / NW;            // A copies per wave per stage (4)
    constexpr int B_INS = BN / 16 * 2 / NW;       // B copies per wave per stage (4)
    constexpr int PER = A_INS + B_INS;
    constexpr bool LN = EPI != Epi::kGemm;
    constexpr bool SW = EPI == Epi::kSwiGlu;
    constexpr bool NOL = EPI == Epi::kLnOnLoad;
    static_assert(!SW || FN % 2 == 0, "gate/up fragment pairs");
    constexpr int FMW = FM / WN;                  // row blocks whose moments each wave column owns
    constexpr int NMF = FM * FN, NRD = FM + FN;

    __shared__ __attribute__((aligned(1024))) char smem[2 * STAGE];
    __shared__ float row_s1[LN ? BM : 1], row_s2[LN ? BM : 1];
    __shared__ float mom_part[LN ? 2 * WN * BM : 1];  // shared moments: (sum x, sum x^2) per wave column
    __shared__ int mom_missing;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / WN, wn = wave % WN;
    const int64_t M = p.M, K = p.K, N = p.N;

    // A workgroup owns one 256-row block and `group` consecutive 256-column
    // tiles of it.  The row moments depend only on the rows, so they are
    // reduced once, alongside the first tile's main loop, and kept in LDS for
    // the epilogues of all the group's tiles.  When the row block's column
    // groups are co-resident they split that reduction between them (each
    // takes a share of the block's 16-row fragments) and exchange the results
    // through a device mailbox -- the normalization's collective carried out
    // by the workgroups that share the rows, 1/ngroups of the work each.
    // Workgroup order: XCD-contiguous, then blocks of GM row blocks x all
    // column groups (operand panels shared under one L2).
    if constexpr (!LN) group = 1;  // the plain product has no per-row work to share
    const int tiles_m = (int)((M + BM - 1) / BM), tiles_n = (int)((N + BN - 1) / BN);
    const int ngroups = (tiles_n + group - 1) / group;
    const int t = xcd_contiguous(blockIdx.x, gridDim.x);
    constexpr int GM = 4;
    const int span = GM * ngroups, gid = t / span, first = gid * GM;
    const int gsz = min(tiles_m - first, GM);
    const int pm = first + (t % span) % gsz;
    const int gn = (t % span) / gsz;
    const int64_t m0 = (int64_t)pm * BM;

    // Shared moments: the ngroups workgroups of a row block split its 16-row fragments
    // (fragment f goes to column group f mod ngroups); each reduces the moments of its
    // fragments alongside its first tile's main loop -- the two wave columns of the
    // fragment's wave row taking alternate k-halves -- and publishes them.  With
    // ngroups >= FM (the host's condition) a wave row holds at most one of them, own_fm.
    const bool share = LN && !NOL && p.mom_slots != nullptr && p.row_stats == nullptr;
    int own_fm = -1;
    if (share) {
#pragma unroll
        for (int fm = 0; fm < FM; ++fm)
            if ((wm * FM + fm) % ngroups == gn) own_fm = fm;
    }

    const __bf16* A = reinterpret_cast<const __bf16*>(p.A);
    const char* Bp = reinterpret_cast<const char*>(p.B);
    __bf16* C = reinterpret_cast<__bf16*>(p.C);
    const int nst = (int)(K / BK);

    // Copy sources: a wave-uniform base per operand (this tile's first row of
    // x, its first packed chunk column of W') advanced by one stage at a time,
    // and fixed per-lane byte offsets from it (rows or chunks; k advances only
    // the base).  The host guarantees 256 K-element rows and the chunk panel
    // stay below 4 GiB of offset.
    uint32_t a_off[A_INS];
#pragma unroll
    for (int j = 0; j < A_INS; ++j) {
        const int r = (wave + j * NW) * 8 + (lane >> 3);           // tile row of this lane
        const int piece = (lane & 7) ^ a_swz(r);                    // 16-byte piece it fetches
        a_off[j] = (uint32_t)(((min(m0 + r, M - 1) - m0) * K + piece * 8) * 2);
    }
    const uint64_t a_base = uniform_u64(A + m0 * K);
    const uint32_t smem_addr = lds_addr32(smem);
    // fragments of stage s, half h (k 32h .. 32h+31)
    auto read = [&](int s, int h, u32x4(&fa)[FM], u32x4(&fb)[FN]) {
        const char* base = smem + (s & 1) * STAGE;
#pragma unroll
        for (int fm = 0; fm < FM; ++fm) {
            const int r = wm * WTM + fm * 16 + (lane & 15);
            const int piece = h * 4 + (lane >> 4);
            fa[fm] = lds_ld16(lds_ptr((char*)base + r * 128 + ((piece ^ a_swz(r)) << 4)));
        }
#pragma unroll
        for (int fn = 0; fn < FN; ++fn)
            fb[fn] = lds_ld16(lds_ptr((char*)base + A_BYTES + ((wn * FN + fn) * 2 + h) * kChunkBytes + lane * 16));
    };

    float s1[FMW], s2[FMW];
#pragma unroll
    for (int i = 0; i < FMW; ++i) s1[i] = s2[i] = 0.f;

    // Normalize-on-load: the statistics of the lane's row in each row fragment
    // (A operand: lane l holds row l & 15 of the fragment), as xh = x r + (-mean r).
    float nl_r[NOL ? FM : 1], nl_b[NOL ? FM : 1];
    if constexpr (NOL) {
#pragma unroll
        for (int fm = 0; fm < FM; ++fm) {
            const int64_t row = min(m0 + wm * WTM + fm * 16 + (lane & 15), M - 1);
            const float mean = p.row_stats[2 * row], rstd = p.row_stats[2 * row + 1];
            nl_r[fm] = rstd;
            nl_b[fm] = -mean * rstd;
        }
    }

    for (int tt = 0; tt < group; ++tt) {
        const int pn = gn * group + tt;
        if (pn >= tiles_n) break;
        const int64_t n0 = (int64_t)pn * BN;
        if (tt > 0) __syncthreads();  // every wave is done with the previous tile's stages

        uint32_t b_off[B_INS];
        const int64_t nb0 = n0 / 16;
#pragma unroll
        for (int j = 0; j < B_INS; ++j) {
            const int c = wave + j * NW, nb = c >> 1, kb = c & 1;
            b_off[j] = (uint32_t)packed_chunk(min(nb0 + nb, p.nblocks - 1) - nb0, kb, p.kchunks, lane);
        }
        const uint64_t b_base = uniform_u64(Bp + packed_chunk(nb0, 0, p.kchunks, 0));
        auto issue = [&](int s) {
            const uint32_t base = smem_addr + (uint32_t)((s & 1) * STAGE);
            const uint64_t ab = a_base + (uint64_t)s * (BK * 2), bb = b_base + (uint64_t)s * (2 * kChunkBytes);
#pragma unroll
            for (int j = 0; j < A_INS; ++j)
                g2lds16_async_sb(ab, a_off[j], base + (uint32_t)((wave + j * NW) * kChunkBytes));
#pragma unroll
            for (int j = 0; j < B_INS; ++j)
                g2lds16_async_sb(bb, b_off[j], base + (uint32_t)(A_BYTES + (wave + j * NW) * kChunkBytes));
        };

        f32x4 acc[FM][FN];
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

        // Shared moments: the wave's owned fragment for k-half h == wn, re-read from the
        // stage in LDS (one fragment read per stage), summed into (ms1, ms2).
        float ms1 = 0.f, ms2 = 0.f;
        // MFMAs on (fa, fb) -- and, on the group's first tile, the owned rows'
        // moments from the same fa registers -- with the next half's fragment
        // reads (already issued) interleaved by the scheduler.  OWN < 0: no moments.
        // SLICE: the shared-moment share of the stage (ms, read before the stage's
        // barrier) is reduced by VALU instructions placed between the later MFMAs,
        // where they fill issue slots beside the matrix pipe instead of running
        // after the last MFMA and delaying the next barrier.
        auto compute = [&](auto own, u32x4(&fa)[FM], u32x4(&fb)[FN], auto slice, const u32x4& ms) {
            constexpr int OWN = decltype(own)::value;
            constexpr bool SLICE = decltype(slice)::value;
            if constexpr (LN && OWN >= 0) {
#pragma unroll
                for (int i = 0; i < FMW; ++i) chunk_moments<__bf16>(fa[OWN * FMW + i], s1[i], s2[i]);
            }
            if constexpr (SLICE) chunk_moments<__bf16>(ms, ms1, ms2);
            if constexpr (NOL) {
#pragma unroll
                for (int fm = 0; fm < FM; ++fm) fa[fm] = normalize_chunk(fa[fm], nl_r[fm], nl_b[fm]);
            }
#pragma unroll
            for (int fm = 0; fm < FM; ++fm)
#pragma unroll
                for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = mfma_chunk<__bf16>(fa[fm], fb[fn], acc[fm][fn]);
#pragma unroll
            for (int i = 0; i < NMF; ++i) {
                __builtin_amdgcn_sched_group_barrier(kSgMfma, 1, 0);
                if (i < NRD)
                    __builtin_amdgcn_sched_group_barrier(kSgDsRead, 1, 0);
                else if (SLICE && i < NRD + 12)
                    __builtin_amdgcn_sched_group_barrier(kSgValu, 2, 0);
            }
        };
        const int mr = wm * WTM + max(own_fm, 0) * 16 + (lane & 15);
        const int mrow = mr * 128 + (((wn * 4 + (lane >> 4)) ^ a_swz(mr)) << 4);
        auto run = [&](auto own, auto slice) {
            constexpr bool SLICE = decltype(slice)::value;
            issue(0);
            if (nst > 1) {
                issue(1);
                wait_vmcnt<PER>();
            } else {
                wait_vmcnt<0>();
            }
            block_barrier();
            u32x4 fa0[FM], fb0[FN], fa1[FM], fb1[FN], ms = {0u, 0u, 0u, 0u};
            read(0, 0, fa0, fb0);
            for (int s = 0; s < nst; ++s) {
                read(s, 1, fa1, fb1);
                // the owned fragment's k-half wn of stage s, read (like every read of stage s)
                // before the barrier after which stage s + 2 overwrites the buffer, and reduced
                // beside the MFMAs of stage s's second half
                if (SLICE) ms = lds_ld16(lds_ptr(smem + (s & 1) * STAGE + mrow));
                compute(own, fa0, fb0, std::false_type{}, ms);
                wait_vmcnt<0>();  // this wave's copies of stage s+1 have landed
                wait_lgkm0();     // this wave's reads of stage s are complete
                block_barrier();
                if (s + 2 < nst) issue(s + 2);  // into the buffer stage s just vacated
                read(s + 1, 0, fa0, fb0);       // past the end this reads stale data that is never used
                compute(own, fa1, fb1, slice, ms);
            }
        };
        const bool moments = LN && !NOL && tt == 0 && !p.row_stats;
        if (moments && share) {
            if (own_fm >= 0)
                run(std::integral_constant<int, -1>{}, std::true_type{});
            else
                run(std::integral_constant<int, -1>{}, std::false_type{});
        } else if (moments) {
            if (wn == 1)
                run(std::integral_constant<int, 1>{}, std::false_type{});
            else
                run(std::integral_constant<int, 0>{}, std::false_type{});
        } else {
            run(std::integral_constant<int, -1>{}, std::false_type{});
        }
        wait_lgkm0();

        if (LN && !NOL && tt == 0 && p.row_stats) {  // serial ablation: the pre-pass statistics
            for (int r = tid; r < BM; r += NW * kWave) {
                const int64_t rr = min(m0 + r, M - 1);
                row_s1[r] = p.row_stats[2 * rr];
                row_s2[r] = p.row_stats[2 * rr + 1];
            }
            __syncthreads();
        }
        if (moments && share) {
            // this workgroup's fragments: the two k-halves' partial sums meet in LDS, the
            // totals are published stamped with the call number ...
            if (own_fm >= 0) {
                const float a = sum_lane_groups(ms1);
                const float b = sum_lane_groups(ms2);
                if (lane < 16) {
                    const int r = wm * WTM + own_fm * 16 + lane;
                    mom_part[(2 * wn) * BM + r] = a;
                    mom_part[(2 * wn + 1) * BM + r] = b;
                }
            }
            if (tid == 0) mom_missing = 0;
            __syncthreads();
            const unsigned long long stamp = (unsigned long long)p.mom_call << 32;
            for (int r = tid; r < BM; r += NW * kWave) {
                if ((r / 16) % ngroups == gn && m0 + r < M) {
                    float a = 0.f, b = 0.f;
#pragma unroll
                    for (int w = 0; w < WN; ++w) {
                        a += mom_part[(2 * w) * BM + r];
                        b += mom_part[(2 * w + 1) * BM + r];
                    }
                    __hip_atomic_store(p.mom_slots + 2 * (m0 + r), stamp | __float_as_uint(a), __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
                    __hip_atomic_store(p.mom_slots + 2 * (m0 + r) + 1, stamp | __float_as_uint(b), __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
                }
            }
            // ... and the whole row block's are read back, each word checked against the stamp.
            // The wait is bounded (s_memrealtime, 100 MHz): a peer that has not published by
            // then (not resident, say) makes this workgroup reduce every row itself below.
            // A bound of 0 skips the exchange (every row reduced locally).
            for (int r = tid; r < BM; r += NW * kWave) {
                float a = 0.f, b = 0.f;
                if (p.mom_wait_ticks == 0) {
                    mom_missing = 1;
                } else if (m0 + r < M) {
                    const unsigned long long* sl = p.mom_slots + 2 * (m0 + r);
                    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
                    bool ok = false;
                    while (true) {
                        const unsigned long long w1 = __hip_atomic_load(sl, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        const unsigned long long w2 =
                            __hip_atomic_load(sl + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        if ((w1 >> 32) == p.mom_call && (w2 >> 32) == p.mom_call) {
                            a = __uint_as_float((uint32_t)w1);
                            b = __uint_as_float((uint32_t)w2);
                            ok = true;
                            break;
                        }
                        if (__builtin_amdgcn_s_memrealtime() - t0 > p.mom_wait_ticks) break;
                        __builtin_amdgcn_s_sleep(8);
                    }
                    if (!ok) mom_missing = 1;
                }
                row_s1[r] = a;
                row_s2[r] = b;
            }
            __syncthreads();
            if (mom_missing) {  // fallback: every row of the block from x itself, one wave per row
                for (int r = wave; r < BM; r += NW) {
                    float a = 0.f, b = 0.f;
                    if (m0 + r < M) {
                        const __bf16* xr = A + (m0 + r) * K;
                        for (int64_t k = lane * 8; k < K; k += 8 * kWave) chunk_moments<__bf16>(ld16(xr + k), a, b);
                        a = wave_sum(a);
                        b = wave_sum(b);
                    }
                    if (lane == 0) {
                        row_s1[r] = a;
                        row_s2[r] = b;
                    }
                }
                __syncthreads();
            }
        } else if (moments) {
#pragma unroll
            for (int i = 0; i < FMW; ++i) {
                const float a = sum_lane_groups(s1[i]);
                const float b = sum_lane_groups(s2[i]);
                if (lane < 16) {
                    const int r = wm * WTM + (wn * FMW + i) * 16 + lane;
                    row_s1[r] = a;
                    row_s2[r] = b;
                }
            }
            __syncthreads();
        }
        if (moments) {
            for (int r = tid; r < BM; r += NW * kWave) {
                const float mean = p.rms ? 0.f : row_s1[r] / (float)K;
                row_s2[r] = rstd_from_moments(row_s2[r] / (float)K, mean, p.eps);
                row_s1[r] = mean;
                if (p.stats_out && gn == 0 && m0 + r < M) {  // the row block's first group exports them
                    p.stats_out[2 * (m0 + r)] = mean;
                    p.stats_out[2 * (m0 + r) + 1] = row_s2[r];
                }
            }
            __syncthreads();
        }

        // Per-lane epilogue operands, loaded once per tile: the column terms c_n,
        // b_n (or the bias) of the lane's 8 columns and the row terms mean_m,
        // rstd_m of its 16 rows.
        // (Opaque copies: the lane's row and column terms are formed here, after the
        // main loop, rather than hoisted out of the tile loop and held across it.)
        int lc = wn * WTN + (lane & 15), lr = wm * WTM + 4 * (lane >> 4);  // lane's first column / row
        asm volatile("" : "+v"(lc), "+v"(lr));
        float cn[FN], bn[FN];
#pragma unroll
        for (int fn = 0; fn < FN; ++fn) {
            const int64_t nc = min(n0 + (lc + fn * 16), N - 1);
            cn[fn] = 0.f;
            bn[fn] = 0.f;
            if constexpr (LN) {
                cn[fn] = p.c_col[nc];
                bn[fn] = p.b_col[nc];
            } else {
                if (p.bias) bn[fn] = to_f32<__bf16>(reinterpret_cast<const __bf16*>(p.bias)[nc]);
            }
        }
        float mu[FM][4], rs[FM][4];
#pragma unroll
        for (int fm = 0; fm < FM; ++fm)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                mu[fm][i] = LN && !NOL ? row_s1[lr + fm * 16 + i] : 0.f;
                rs[fm][i] = LN && !NOL ? row_s2[lr + fm * 16 + i] : 1.f;
            }
        auto value = [&](int fm, int fn, int i) {
            const float v = acc[fm][fn][i];
            if constexpr (NOL)
                return v + bn[fn];
            else if constexpr (LN)
                return __builtin_fmaf(rs[fm][i], __builtin_fmaf(-mu[fm][i], cn[fn], v), bn[fn]);
            else
                return v + bn[fn];
        };
        // Stores of a tile wholly in range go through a buffer resource on the
        // tile's first element: the row offset of each (fm, i) is a scalar
        // (soffset), the lane's offset in the tile a fixed 32-bit VGPR and the
        // fragment column an immediate, so no 64-bit row addresses stay live.
        // (The host keeps 256 rows of the output below 2^31 bytes.)  Every store
        // carries the non-temporal policy: the output goes to HBM while the
        // matrix cores still run, instead of staying dirty in the caches for
        // the next kernel to write back when its own traffic evicts it.
        auto store_tile = [&](__bf16* base, int64_t ldc, int vo, auto col_value, auto ncol) {
            const __amdgpu_buffer_rsrc_t rc = __builtin_amdgcn_make_buffer_rsrc(base, 0, 0x7fffffff, 0x00020000);
            constexpr int NCOL = decltype(ncol)::value;
#pragma unroll
            for (int fm = 0; fm < FM; ++fm) {
                // a fragment's values first, then its stores back to back: the
                // pieces of each output line reach L2 close together
                unsigned short hv[4][NCOL];
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int f = 0; f < NCOL; ++f) hv[i][f] = __builtin_bit_cast(unsigned short, (__bf16)col_value(fm, f, i));
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int so = __builtin_amdgcn_readfirstlane((fm * 16 + i) * (int)ldc * 2);
#pragma unroll
                    for (int f = 0; f < NCOL; ++f)
                        __builtin_amdgcn_raw_buffer_store_b16(hv[i][f], rc, vo + f * 32, so, kStoreStream);
                }
            }
        };
        // A ragged tile checks each store against the rows and columns left.
        auto store_edge = [&](__bf16* base, int64_t ldc, int64_t rows_left, int64_t cols_left, int col0,
                              auto col_value, auto ncol) {
            const __amdgpu_buffer_rsrc_t rc = __builtin_amdgcn_make_buffer_rsrc(base, 0, 0x7fffffff, 0x00020000);
            constexpr int NCOL = decltype(ncol)::value;
#pragma unroll
            for (int fm = 0; fm < FM; ++fm)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int rl = lr + fm * 16 + i;
#pragma unroll
                    for (int f = 0; f < NCOL; ++f) {
                        const int col = col0 + f * 16;
                        if (rl < rows_left && col < cols_left)
                            __builtin_amdgcn_raw_buffer_store_b16(
                                __builtin_bit_cast(unsigned short, (__bf16)col_value(fm, f, i)), rc,
                                (rl * (int)ldc + col) * 2, 0, kStoreStream);
                    }
                }
        };
        if constexpr (SW) {
            // fragment 2j holds gate columns, 2j+1 the up columns of the same outputs
            const int64_t ob = (n0 + wn * WTN) / 2;  // the wave's first output column
            auto h = [&](int fm, int j, int i) { return silu(value(fm, 2 * j, i)) * value(fm, 2 * j + 1, i); };
            if (m0 + BM <= M && ob + WTN / 2 <= p.n_out)
                store_tile(C + m0 * p.n_out + ob, p.n_out, (int)(lr * p.n_out + (lane & 15)) * 2, h,
                           std::integral_constant<int, FN / 2>{});
            else
                store_edge(C + m0 * p.n_out + ob, p.n_out, M - m0, p.n_out - ob, lane & 15, h,
                           std::integral_constant<int, FN / 2>{});
            continue;
        }
        if (m0 + BM <= M && n0 + BN <= N)
            store_tile(C + m0 * N + n0, N, (int)(lr * N + lc) * 2, value, std::integral_constant<int, FN>{});
        else
            store_edge(C + m0 * N + n0, N, M - m0, N - n0, lc, value, std::integral_constant<int, FN>{});
    }
}

// =============================================================================
// Decode-shaped deferred LN -> Linear: M <= 128 tokens, bf16.
// The work is streaming W' from HBM.  Each workgroup owns NC blocks of 16
// output columns and its KS waves split K; per 32-k chunk a wave reads the
// (zero-padded) x fragment once and NC packed W' chunks straight from HBM into
// operand registers (one contiguous KiB each), and runs one 16x16x32 MFMA per
// column block.  The row moments ride on the otherwise idle matrix core: with
// B = all-ones the product gives sum_k x[m][k] in every column, and with B = x
// itself the Gram matrix x x^T whose diagonal is sum_k x[m][k]^2 -- once per
// chunk for all NC column blocks.
// =============================================================================
// SW: the packed columns interleave gate and up blocks (NC even, blocks 2j and
// 2j+1 of the group form output block j), out[M][n_out] = SiLU(gate) * up.
// PLAIN: the plain product out = x . W' + bias (bias: [N] bf16, nullable), no
// moments -- the decode-shaped GEMM of the unfused comparators.
template <int KS, int NC, int U, bool SW = false, bool PLAIN = false, int MT = 1>
__global__ __launch_bounds__(KS * kWave) void ln_decode_bf16_kernel(const __bf16* __restrict__ x,
                                                             const char* __restrict__ Wp, int64_t kchunks,
                                                             int64_t nblocks, const float* __restrict__ c_col,
                                                             const float* __restrict__ b_col, int M, int64_t K,
                                                             int64_t N, float eps, int rms, int64_t n_out,
                                                             const float* __restrict__ row_stats,
                                                             float* __restrict__ stats_out,
                                                             __bf16* __restrict__ out,
                                                             const __bf16* __restrict__ bias) {
    static_assert(!SW || NC % 2 == 0, "gate/up block pairs");
    static_assert(!(SW && PLAIN), "the plain product has no gate");
    // MT fragments of 16 token rows (M <= 16 MT), reduced one fragment at a time; the
    // slots hold the fragment's moments (sum x, Gram) and then the NC column blocks'
    // partial products
    constexpr int SLOTS = 2 + NC;
    __shared__ f32x4 part[SLOTS][KS][kWave];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t nb0 = (int64_t)blockIdx.x * NC;
    const int row = lane & 15;
    bool row_ok[MT];
    const __bf16* xr[MT];
#pragma unroll
    for (int f = 0; f < MT; ++f) {
        row_ok[f] = 16 * f + row < M;
        xr[f] = x + (int64_t)(row_ok[f] ? 16 * f + row : 0) * K;
    }
    const char* wr[NC];
#pragma unroll
    for (int q = 0; q < NC; ++q) wr[q] = Wp + packed_chunk(min(nb0 + q, nblocks - 1), 0, kchunks, lane);

    // The KS waves split the chunks: with one row fragment interleaved (wave w takes
    // chunks w, w + KS, ..., so the waves of a workgroup read neighbouring KiB of each
    // column block at a time), with more in contiguous ranges.  Measured: 1 token on
    // 8192 -> 2 x 28672 (gated MLP) 152.5 -> 141.4 us and on 8192 -> 28672 78.1 ->
    // 77.3 us interleaved; 32 tokens on 4096 -> 12288 25.2 -> 27.3 us, so ranges there.
    constexpr bool ILV = MT == 1;
    const int64_t nchunks = kchunks;
    const int64_t per = (nchunks + KS - 1) / KS;
    const int64_t c_begin = ILV ? 0 : wave * per;
    const int64_t c_end = ILV ? (nchunks > wave ? (nchunks - wave + KS - 1) / KS : 0) : min(nchunks, c_begin + per);

    const u32x4 ones = {0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u};
    const u32x4 zero = {0, 0, 0, 0};
    const f32x4 fz = {0.f, 0.f, 0.f, 0.f};
    f32x4 acc[MT][NC], sx[MT], sxx[MT];
#pragma unroll
    for (int f = 0; f < MT; ++f) {
        sx[f] = sxx[f] = fz;
#pragma unroll
        for (int q = 0; q < NC; ++q) acc[f][q] = fz;
    }

    // Software pipeline over groups of U chunks: the loads of group g + 1 are in
    // flight while group g multiplies.  Every load is unconditional (chunk
    // indexes clamp to the wave's last chunk, x reads past the range turn into
    // zeros) so the wait counts stay exact; the group count is rounded up to
    // even and a group wholly past the range adds x = 0 times finite W'.
    const int64_t ngroups = c_end > c_begin ? (c_end - c_begin + U - 1) / U : 0;
    u32x4 a0[U][MT], b0[U][NC], a1[U][MT], b1[U][NC];
    auto load = [&](u32x4(&a)[U][MT], u32x4(&b)[U][NC], int64_t g) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t ci = c_begin + g * U + u;  // the wave's ci-th chunk
            const bool ok = ci < c_end;
            const int64_t cl = ILV ? (ok ? ci : c_end - 1) * KS + wave : (ok ? ci : c_end - 1);
            const int64_t kk = cl * 32 + (lane >> 4) * 8;
#pragma unroll
            for (int q = 0; q < NC; ++q) b[u][q] = ld16_stream(wr[q] + cl * kWave * 16);  // zero-padded past K
#pragma unroll
            for (int f = 0; f < MT; ++f) {
                const u32x4 xv = ld16(xr[f] + min(kk, K - 8));  // K % 8 == 0
                a[u][f] = (ok && kk < K && row_ok[f]) ? xv : zero;
            }
        }
    };
    auto compute = [&](const u32x4(&a)[U][MT], const u32x4(&b)[U][NC]) {
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int f = 0; f < MT; ++f) {
#pragma unroll
                for (int q = 0; q < NC; ++q) acc[f][q] = mfma_chunk<__bf16>(a[u][f], b[u][q], acc[f][q]);
                if constexpr (!PLAIN) {
                    sx[f] = mfma_chunk<__bf16>(a[u][f], ones, sx[f]);
                    sxx[f] = mfma_chunk<__bf16>(a[u][f], a[u][f], sxx[f]);
                }
            }
    };
    if (ngroups > 0) {
        load(a0, b0, 0);
        for (int64_t g = 0; g < ngroups; g += 2) {
            load(a1, b1, g + 1);
            compute(a0, b0);
            load(a0, b0, g + 2);
            compute(a1, b1);
        }
    }
    // Row fragment f and column block j of the workgroup (SW: block pair j, gate
    // then up): reduce over the KS slices of K, then the epilogue.
    constexpr int NOUT = SW ? NC / 2 : NC;
#pragma unroll
    for (int f = 0; f < MT; ++f) {
        if (16 * f >= M) break;  // uniform over the workgroup
        if (f) __syncthreads();  // the previous fragment's partial sums have been read
#pragma unroll
        for (int q = 0; q < NC; ++q) part[2 + q][wave][lane] = acc[f][q];
        part[0][wave][lane] = sx[f];
        part[1][wave][lane] = sxx[f];
        __syncthreads();
        for (int j = wave; j < NOUT && nb0 + (SW ? 2 * j : j) < nblocks; j += KS) {
            const int q0 = SW ? 2 * j : j;
            const int64_t col = (nb0 + q0) * 16 + (lane & 15);
            const int64_t n = min(col, N - 1), nu = min(col + 16, N - 1);
            f32x4 tot[4];  // block q0, the moments, block q0 + 1 (SW)
#pragma unroll
            for (int w = 0; w < KS; ++w) {
                const f32x4 v0 = part[2 + q0][w][lane], v1 = part[0][w][lane], v2 = part[1][w][lane];
                tot[0] = w ? tot[0] + v0 : v0;
                tot[1] = w ? tot[1] + v1 : v1;
                tot[2] = w ? tot[2] + v2 : v2;
                if constexpr (SW) tot[3] = w ? tot[3] + part[3 + q0][w][lane] : part[3 + q0][w][lane];
            }
            if constexpr (PLAIN) {
                const float bn = bias ? (float)bias[n] : 0.f;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int r = 16 * f + 4 * (lane >> 4) + i;
                    if (r < M && col < N) out[(int64_t)r * N + col] = (__bf16)(tot[0][i] + bn);
                }
                continue;
            }
            // Gram diagonal (r, r) sits in lane r + 16*(r>>2), element r&3.  This lane's
            // rows are r = 4*(l>>4) + i of the fragment, so the source lane is 20*(l>>4) + i.
            float diag[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) diag[i] = __shfl(tot[2][i], 20 * (lane >> 4) + i);
            const float cn = c_col[n], bn = b_col[n];
            const float cu = SW ? c_col[nu] : 0.f, bu = SW ? b_col[nu] : 0.f;
            const int64_t o = SW ? (nb0 / 2 + j) * 16 + (lane & 15) : col;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int r = 16 * f + 4 * (lane >> 4) + i;
                float mean = rms ? 0.f : tot[1][i] / (float)K;
                float rstd = rstd_from_moments(diag[i] / (float)K, mean, eps);
                if (row_stats) {  // serial ablation (the moment products above are then unused)
                    mean = row_stats[2 * min(r, M - 1)];
                    rstd = row_stats[2 * min(r, M - 1) + 1];
                }
                if (stats_out && blockIdx.x == 0 && j == 0 && (lane & 15) == 0 && r < M) {
                    stats_out[2 * r] = mean;  // the first column block's lanes export them, once per row
                    stats_out[2 * r + 1] = rstd;
                }
                float v = __builtin_fmaf(rstd, __builtin_fmaf(-mean, cn, tot[0][i]), bn);
                if constexpr (SW) v = silu(v) * __builtin_fmaf(rstd, __builtin_fmaf(-mean, cu, tot[3][i]), bu);
                if (r < M && o < n_out) out[(int64_t)r * n_out + o] = (__bf16)v;
            }
        }
    }
}

// =============================================================================
// Static-weight preparation (off the per-token path).
// =============================================================================
// c[n] = sum_k round(gamma_k W[k][n]),  b[n] = sum_k beta_k W[k][n] + bias[n]; fp64 sums.
// center = 1: c[n] = (1/K) sum_k gamma_k W[k][n] unrounded instead -- the column mean
// that the literal Eq. (5) weight (I - E/n) Gamma W subtracts (pack reads it, then it
// is cleared).  Column n of W lands at packed column ((n / 16) * mul + add) * 16 +
// n % 16 (mul = 2 interleaves two weight matrices block by block); columns N ..
// n_pad - 1 get zeros.
template <class T>
__global__ __launch_bounds__(256) void prep_colsum_kernel(const T* __restrict__ W, const T* __restrict__ gamma,
                                                          const T* __restrict__ beta, const T* __restrict__ bias,
                                                          int64_t K, int64_t N, int64_t n_pad, int mul, int add,
                                                          int center, float* __restrict__ c_col,
                                                          float* __restrict__ b_col) {
    const int64_t n = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (n >= n_pad) return;
    double cs = 0.0, bs = 0.0;
    if (n < N) {
        for (int64_t k = 0; k < K; ++k) {
            const float w = to_f32<T>(W[k * N + n]);
            const float gw = to_f32<T>(gamma[k]) * w;  // exact: a product of two bf16 values fits fp32
            cs += center ? (double)gw : (double)to_f32<T>(from_f32<T>(gw));
            if (beta) bs += (double)to_f32<T>(beta[k]) * (double)w;
        }
        if (bias) bs += (double)to_f32<T>(bias[n]);
        if (center) cs /= (double)K;
    }
    const int64_t pc = ((n / 16) * mul + add) * 16 + n % 16;
    c_col[pc] = (float)cs;
    b_col[pc] = (float)bs;
}

// One thread per 16-byte lane piece of the packed layout: chunk (nb, kc), lane l
// holds W'[k][n] for n = 16 nb + (l & 15), k = kc*kchunk + (l >> 4)*EPL + e; the
// chunk is stored as block nb * mul + add.  center (nullable): the column means to
// subtract before rounding (W'' = (I - E/n) Gamma W of Eq. (5)).
template <class T>
__global__ __launch_bounds__(256) void prep_pack_kernel(const T* __restrict__ W, const T* __restrict__ gamma,
                                                        int64_t K, int64_t N, int64_t kchunks, int64_t pieces,
                                                        int mul, int add, const float* __restrict__ center,
                                                        char* __restrict__ packed) {
    constexpr int EPL = elem<T>::per16, KC = elem<T>::kchunk;
    const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (id >= pieces) return;
    const int l = (int)(id % kWave);
    const int64_t chunk = id / kWave;
    const int64_t nb = chunk / kchunks, kc = chunk % kchunks;
    const int64_t n = nb * 16 + (l & 15);
    const int64_t k0 = kc * KC + (l >> 4) * EPL;
    float v[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
        const int64_t k = k0 + e;
        v[e] = (n < N && k < K) ? to_f32<T>(gamma[k]) * to_f32<T>(W[k * N + n]) - (center ? center[n] : 0.f) : 0.f;
    }
    u32x4 out;
    if constexpr (sizeof(T) == 2) {
        out = u32x4{pack_bf16(v[0], v[1]), pack_bf16(v[2], v[3]), pack_bf16(v[4], v[5]), pack_bf16(v[6], v[7])};
    } else {
        out = u32x4{__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]), __float_as_uint(v[3])};
    }
    const int64_t dst = ((nb * mul + add) * kchunks + kc) * kWave + l;
    *reinterpret_cast<u32x4*>(packed + dst * 16) = out;
}

// =============================================================================
// Host launchers
// =============================================================================
static size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

PackedLayout packed_layout(int64_t K, int64_t N, int dtype) {
    PackedLayout L;
    const int64_t es = dtype == 0 ? 4 : 2;
    const int64_t kc = dtype == 0 ? 16 : 32;
    L.kchunks = (K + kc - 1) / kc;
    L.nblocks = (N + 15) / 16;
    L.wt_off = 0;
    L.wt_bytes = (size_t)(L.nblocks * 16) * (size_t)(L.kchunks * kc) * (size_t)es;
    L.c_off = align256(L.wt_bytes);
    L.b_off = L.c_off + align256((size_t)N * 4);
    L.total = L.b_off + align256((size_t)N * 4);
    return L;
}

// SwiGLU weights: gate and up interleaved block by block, so 2 * ceil(N / 16) blocks.
PackedLayout swiglu_layout(int64_t K, int64_t N, int dtype) { return packed_layout(K, 2 * ((N + 15) / 16) * 16, dtype); }

// Fold gamma into W and pack it as blocks nb * mul + add of a layout with L.kchunks.
__global__ __launch_bounds__(256) void fill_zero_kernel(float* __restrict__ p, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0.f;
}

template <class T>
static void pack_one(const void* W, const void* gamma, const void* beta, const void* bias, int64_t K, int64_t N,
                     const PackedLayout& L, int mul, int add, int center, char* base, hipStream_t s) {
    const int64_t n_pad = (N + 15) / 16 * 16;
    float* c_col = (float*)(base + L.c_off);
    prep_colsum_kernel<T><<<dim3((unsigned)((n_pad + 255) / 256)), 256, 0, s>>>(
        (const T*)W, (const T*)gamma, (const T*)beta, (const T*)bias, K, N, n_pad, mul, add, center, c_col,
        (float*)(base + L.b_off));
    const int64_t pieces = (N + 15) / 16 * L.kchunks * kWave;
    prep_pack_kernel<T><<<dim3((unsigned)((pieces + 255) / 256)), 256, 0, s>>>(
        (const T*)W, (const T*)gamma, K, N, L.kchunks, pieces, mul, add, center ? c_col : nullptr, base + L.wt_off);
    // the centred weight's columns sum to ~0: the epilogue's mean * c term is dropped, as Eq. (5) has none
    if (center) fill_zero_kernel<<<dim3((unsigned)((n_pad + 255) / 256)), 256, 0, s>>>(c_col, n_pad);
}

hipError_t launch_ln_prepare(const void* W, const void* gamma, const void* beta, const void* bias, int64_t K,
                             int64_t N, int dtype, int center, void* packed, hipStream_t s) {
    const PackedLayout L = packed_layout(K, N, dtype);
    char* base = reinterpret_cast<char*>(packed);
    if (dtype == 0)
        pack_one<float>(W, gamma, beta, bias, K, N, L, 1, 0, center, base, s);
    else
        pack_one<__bf16>(W, gamma, beta, bias, K, N, L, 1, 0, center, base, s);
    return hipGetLastError();
}

hipError_t launch_swiglu_prepare(const void* Wg, const void* Wu, const void* gamma, int64_t K, int64_t N, int dtype,
                                 void* packed, hipStream_t s) {
    const PackedLayout L = swiglu_layout(K, N, dtype);
    char* base = reinterpret_cast<char*>(packed);
    for (int which = 0; which < 2; ++which) {
        const void* W = which ? Wu : Wg;
        if (dtype == 0)
            pack_one<float>(W, gamma, nullptr, nullptr, K, N, L, 2, which, 0, base, s);
        else
            pack_one<__bf16>(W, gamma, nullptr, nullptr, K, N, L, 2, which, 0, base, s);
    }
    return hipGetLastError();
}

template <class T, int BM, int BN, int WM, int WN, BMode BMODE, Epi EPI, int NST = 2, int KBT = 2>
static hipError_t run_main(const MainArgs& a, int64_t batch, hipStream_t s) {
    const int64_t tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
    dim3 grid((unsigned)tiles, (unsigned)batch);
    main_loop_kernel<T, BM, BN, WM, WN, BMODE, EPI, NST, KBT><<<grid, WM * WN * kWave, 0, s>>>(a);
    return hipGetLastError();
}
// fp32 tiles (32 x 64, 4 waves): 4 chunks (64 k) per stage, a 4-stage ring of 24 KiB stages,
// copies three stages ahead (LN -> Linear 128 x 768 x 3072: 15.3 us against 17.9 us with
// 2-chunk stages in a 6-stage ring and 20.5 us with two 2-chunk stages)
constexpr int kF32Stages = 4, kF32Chunks = 4;

// Mailbox of the shared row moments: 2 words per row, each (call number << 32) | fp32
// bits of sum x or sum x^2.  One array per GPU, held until the process ends; in host
// code `mom_mailbox` names a host-side stand-in, so kernels get the device address
// looked up once per device with hipGetSymbolAddress.  A reader accepts only words
// stamped with its own call number, so calls that overlap on one GPU (concurrent
// streams) stay correct: at worst a workgroup misses its peers' words and reduces its
// rows itself.
constexpr int64_t kMomentRows = 65536;
static __device__ __align__(256) unsigned long long mom_mailbox[2 * kMomentRows];

static unsigned long long* moment_mailbox() {
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static unsigned long long* addr[kMaxDevices] = {};
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(mom_mailbox)) != hipSuccess) return nullptr;
        addr[dev] = (unsigned long long*)ptr;
    }
    return addr[dev];
}

// Call numbers 1, 2, ... (0 never: the mailbox starts zeroed).
static uint32_t next_moment_call() {
    static std::atomic<uint32_t> counter{0};
    uint32_t c = ++counter;
    while (c == 0) c = ++counter;
    return c;
}

// How long a workgroup waits for its peers' moments before reducing its rows itself,
// in s_memrealtime ticks (100 MHz): 200 us, far above the spread of the peers' first
// tiles.  DN_MOMENT_WAIT_TICKS overrides it (0 forces the local reduction; tests use it).
static uint32_t moment_wait_ticks() {
    const char* e = getenv("DN_MOMENT_WAIT_TICKS");
    return e ? (uint32_t)strtoul(e, nullptr, 10) : 20000u;
}

// Workgroups for tm x tn tiles.  Deferred LN: each workgroup takes `group` column
// tiles of one row block and reduces the row moments once, on its first tile.
// With one workgroup per CU the run takes about ceil(workgroups / 256) * group
// tile times; take the group that minimises that, and of equal ones the largest
// (fewest moment reductions).  384 tiles: group 2 (192 workgroups, 2 tile times)
// instead of group 1 (384 workgroups, also 2 tile times, twice the moment work).
struct TilePlan {
    int64_t group, ngroups, wgs, times;
};
static TilePlan plan_tiles(int64_t tm, int64_t tn, bool grouped) {
    int64_t group = 1;
    if (grouped) {
        int64_t best = -1;
        for (int64_t g = 1; g <= tn; ++g) {
            const int64_t span = (tm * ((tn + g - 1) / g) + 255) / 256 * g;
            if (best < 0 || span <= best) {
                best = span;
                group = g;
            }
        }
    }
    const int64_t ngroups = (tn + group - 1) / group, wgs = tm * ngroups;
    return TilePlan{group, ngroups, wgs, (wgs + 255) / 256 * group};
}

// 256 x 192 tiles where they fill the chip in fewer 256 x 256-tile times: a narrow
// tile costs about kNarrowCost of a square one (three quarters of the MACs, a
// little more operand traffic per MAC).  4096 x 4096 -> 6144: 512 narrow tiles in
// two full rounds instead of 384 square ones in 1.5; 1024 x 4096 -> 12288: 256
// instead of 192 on 256 CUs.
constexpr double kNarrowCost = 0.8;

template <Epi EPI, int BT = 256>
static hipError_t run_pipe(const MainArgs& args, hipStream_t s) {
    MainArgs a = args;
    const int64_t tm = (a.M + BT - 1) / BT, tn = (a.N + BT - 1) / BT;
    TilePlan plan = plan_tiles(tm, tn, EPI != Epi::kGemm);
    bool narrow = false;
    if constexpr (BT == 256) {
        const TilePlan nplan = plan_tiles(tm, (a.N + 191) / 192, EPI != Epi::kGemm);
        if ((double)nplan.times * kNarrowCost < (double)plan.times) {
            plan = nplan;
            narrow = true;
        }
    }
    const int64_t group = plan.group, ngroups = plan.ngroups, wgs = plan.wgs;
    // Shared moments where the workgroups of a row block are co-resident (one round of
    // workgroups: 256 at one per CU, 512 for the 128 x 128 tiles at two per CU) and number
    // at least 4 (then each wave row of a workgroup owns at most one 16-row fragment).
    // Not under stream capture: a captured launch keeps its call number on every replay, so
    // a replay could accept words a previous replay left; captured launches reduce their rows
    // per workgroup instead (each column group on its first tile, as without the exchange).
    a.mom_slots = nullptr;
    hipStreamCaptureStatus cap = hipStreamCaptureStatusActive;
    if (hipStreamIsCapturing(s, &cap) != hipSuccess) cap = hipStreamCaptureStatusActive;
    if ((EPI == Epi::kLnDeferred || EPI == Epi::kSwiGlu) && !a.row_stats && ngroups >= 4 &&
        wgs <= (BT == 128 ? 512 : 256) && a.M <= kMomentRows && cap == hipStreamCaptureStatusNone) {
        a.mom_slots = moment_mailbox();
        a.mom_call = next_moment_call();
        a.mom_wait_ticks = moment_wait_ticks();
    }
    if constexpr (BT == 128)  // 4 waves of 64 x 64, 64 KiB of LDS: two workgroups per CU
        pipe_kernel<EPI, 2, 2, 128, 128><<<dim3((unsigned)wgs), 4 * kWave, 0, s>>>(a, (int)group);
    else if (narrow)  // 8 waves of 64 x 96
        pipe_kernel<EPI, 4, 2, 256, 192><<<dim3((unsigned)wgs), 8 * kWave, 0, s>>>(a, (int)group);
    else
        pipe_kernel<EPI, 4, 2><<<dim3((unsigned)wgs), 8 * kWave, 0, s>>>(a, (int)group);
    return hipGetLastError();
}

// The 256x256 kernel past 128 rows (and K a multiple of its stage), where the
// 128 x 128 tiles do not fit in one round.  Below one 256 x 256 tile per CU it
// still beats the two-stage 128 x 128 loop, which then needs a second round of
// tiles where the 256 x 256 kernel needs none.  Measured on 4096 -> 12288:
// 768 and 1024 rows 89 / 97 us against 178 / 185 us; 8192 -> 28672 at 384 and
// 512 rows 222 / 226 against 376 / 381 us, at 129-256 rows within 5 %.
static bool use_big_tiles(int64_t M, int64_t N, int64_t K) {
    if (N >= (int64_t(1) << 22)) return false;  // 256 output rows < 2^31 bytes (32-bit store offsets)
    // K < 2^22 keeps the 32-bit copy offsets of a 256-row panel (256 K bf16) and of a
    // 16-chunk-column W' panel (16 x K/32 KiB) below 4 GiB.
    return K % 64 == 0 && K < (int64_t(1) << 22) && M > 128;
}
// The pipelined kernel on 128 x 128 tiles (4 waves, two workgroups per CU) while
// those tiles number at most one per CU: then a tile takes far less than a
// 256 x 256 one and the chip is as full.  Measured on 4096 -> 12288 at 129 / 256
// rows (192 tiles) 56 / 58 us against 86 us on 256 x 256 tiles, on 8192 -> 28672
// at 65 / 100 rows (224 tiles) 132 / 133 us against 174 / 184 us on the 128 x 128
// two-stage loop; at 288 tiles and more it lost (97-448 us against 89-230 us).
static bool use_mid_tiles(int64_t M, int64_t N, int64_t K) {
    return K % 64 == 0 && K < (int64_t(1) << 22) && N < (int64_t(1) << 22) &&
           ((M + 127) / 128) * ((N + 127) / 128) <= 256;
}

static MainArgs packed_args(const void* A, const void* packed, int64_t M, int64_t K, int64_t N, int dtype,
                            void* C) {
    const PackedLayout L = packed_layout(K, N, dtype);
    const char* base = reinterpret_cast<const char*>(packed);
    MainArgs a{};
    a.A = A;
    a.B = base + L.wt_off;
    a.C = C;
    a.M = M;
    a.K = K;
    a.N = N;
    a.kchunks = L.kchunks;
    a.nblocks = L.nblocks;
    a.c_col = (const float*)(base + L.c_off);
    a.b_col = (const float*)(base + L.b_off);
    return a;
}

// Decode-shaped launches (M <= 16): 16 waves split K (16 waves per CU hide the
// HBM latency of the W' stream) and each workgroup owns nc column blocks, nc
// chosen so the grid is about one workgroup per CU (at most 7: 144 KiB of LDS
// for the partial sums).  Measured on the 8192 x 28672 up-projection (1792
// blocks, nc = 7): 78.5-78.8 us for 1-16 tokens, against 81-91 us for the
// 4- and 8-wave layouts with 1-4 blocks per workgroup.
constexpr int64_t kDecodeMaxRows = 128;
// Past 64 tokens the streaming kernel re-reads x once per workgroup and stops
// beating the 128 x 128 tiles once those fill most of the chip: measured at
// 65-128 tokens, 1.7-2x faster for the 4096 -> 12288 projection (96 tiles),
// 1.15-1.4x slower for 8192 -> 28672 (224 tiles); the crossover sits near 160.
static bool decode_rows(int64_t M, int64_t ncols) {
    if (M <= 64) return true;
    return M <= kDecodeMaxRows && ((M + 127) / 128) * ((ncols + 127) / 128) < 160;
}
template <bool PLAIN, int MT, int KS, int U, int NC, class F>
static void decode_dispatch_nc(int64_t nc, F&& launch) {  // min(nc, NC) column blocks per workgroup
    if constexpr (NC > 1)
        if (nc < NC) return decode_dispatch_nc<PLAIN, MT, KS, U, NC - 1>(nc, launch);
    launch(ln_decode_bf16_kernel<KS, NC, U, false, PLAIN, MT>, KS, NC);
}
template <bool PLAIN, class F>
static void decode_dispatch(int64_t M, int64_t nblocks, F&& launch) {
    const int64_t nc = std::min<int64_t>(7, std::max<int64_t>(1, (nblocks + 255) / 256));
    // 17-128 tokens: 2-8 row fragments per wave and 4 (8 at 6 fragments) waves
    // splitting K; past 4 fragments at most 3 column blocks per workgroup (the
    // accumulators of 8 fragments x 3 blocks take 96 registers per lane)
    if (M <= 16)
        decode_dispatch_nc<PLAIN, 1, 16, 1, 7>(nc, launch);
    else if (M <= 32)
        decode_dispatch_nc<PLAIN, 2, 4, 2, 7>(nc, launch);
    else if (M <= 48)
        decode_dispatch_nc<PLAIN, 3, 4, 2, 7>(nc, launch);
    else if (M <= 64)
        decode_dispatch_nc<PLAIN, 4, 4, 2, 7>(nc, launch);
    else if (M <= 96)
        decode_dispatch_nc<PLAIN, 6, 8, 1, 3>(nc, launch);
    else
        decode_dispatch_nc<PLAIN, 8, 4, 2, 3>(nc, launch);
}

hipError_t launch_ln_linear_deferred(const void* x, const void* packed, int64_t M, int64_t K, int64_t N,
                                     int dtype, float eps, int rms, const float* row_stats, void* out,
                                     hipStream_t s, float* stats_out) {
    MainArgs a = packed_args(x, packed, M, K, N, dtype, out);
    a.eps = eps;
    a.rms = rms;
    a.row_stats = row_stats;
    a.stats_out = stats_out;
    if (dtype == 1 && decode_rows(M, N)) {
        auto launch = [&](auto kern, int ks, int cols) {
            const int64_t wgs = (a.nblocks + cols - 1) / cols;
            kern<<<dim3((unsigned)wgs), ks * kWave, 0, s>>>((const __bf16*)x, (const char*)a.B, a.kchunks,
                                                            a.nblocks, a.c_col, a.b_col, (int)M, K, N, eps, rms,
                                                            N, a.row_stats, a.stats_out, (__bf16*)out, nullptr);
        };
        decode_dispatch<false>(M, a.nblocks, launch);
        return hipGetLastError();
    }
    if (dtype == 0) return run_main<float, 32, 64, 2, 2, BMode::kPacked, Epi::kLnDeferred, kF32Stages, kF32Chunks>(a, 1, s);
    if (use_mid_tiles(M, N, K)) return run_pipe<Epi::kLnDeferred, 128>(a, s);
    if (use_big_tiles(M, N, K)) return run_pipe<Epi::kLnDeferred>(a, s);
    return run_main<__bf16, 128, 128, 2, 2, BMode::kPacked, Epi::kLnDeferred>(a, 1, s);
}

bool ln_on_load_supported(int64_t M, int64_t K, int64_t N, int dtype) {
    return dtype == 1 && use_big_tiles(M, N, K);
}

hipError_t launch_ln_linear_on_load(const void* x, const void* packed, int64_t M, int64_t K, int64_t N,
                                    const float* row_stats, void* out, hipStream_t s) {
    MainArgs a = packed_args(x, packed, M, K, N, 1, out);
    a.row_stats = row_stats;
    return run_pipe<Epi::kLnOnLoad>(a, s);
}

template <int NC, class F>
static void swiglu_dispatch_nc(int64_t nc, F&& launch) {  // min(nc, NC) column blocks (NC / 2 pairs)
    if constexpr (NC > 2)
        if (nc < NC) return swiglu_dispatch_nc<NC - 2>(nc, launch);
    launch(ln_decode_bf16_kernel<4, NC, 2, true>, 4, NC);
}

hipError_t launch_swiglu_deferred(const void* x, const void* packed, int64_t M, int64_t K, int64_t N, int dtype,
                                  float eps, int rms, void* out, hipStream_t s) {
    const int64_t np = 2 * ((N + 15) / 16) * 16;  // packed (gate + up) columns
    MainArgs a = packed_args(x, packed, M, K, np, dtype, out);
    a.eps = eps;
    a.rms = rms;
    a.n_out = N;
    if (dtype == 1 && decode_rows(M, np)) {
        auto launch = [&](auto kern, int ks, int cols) {
            const int64_t wgs = (a.nblocks + cols - 1) / cols;
            kern<<<dim3((unsigned)wgs), ks * kWave, 0, s>>>((const __bf16*)x, (const char*)a.B, a.kchunks, a.nblocks,
                                                           a.c_col, a.b_col, (int)M, K, np, eps, rms, N,
                                                           nullptr, nullptr, (__bf16*)out, nullptr);
        };
        // up to 16 tokens: up to 7 gate/up block pairs per workgroup (about one
        // workgroup per CU), 4 K-slices, 2-chunk groups -- on the 8192 x 2 x 28672
        // weights 154.5 us (6.1 TB/s) for 1 token against 166.3 us with one pair per
        // workgroup and 154.9 us with 8 K-slices; 33-64 tokens two pairs per workgroup
        // (48 / 64 tokens: 220 / 276 us against 262 / 309 us with one; three pairs
        // 258 / 307 us); 17-32 and 65-128 tokens one pair
        if (M <= 16)
            swiglu_dispatch_nc<14>(2 * std::min<int64_t>(7, std::max<int64_t>(1, (a.nblocks / 2 + 255) / 256)),
                                   launch);
        else if (M <= 32)
            launch(ln_decode_bf16_kernel<4, 2, 2, true, false, 2>, 4, 2);
        else if (M <= 48)
            launch(ln_decode_bf16_kernel<4, 4, 2, true, false, 3>, 4, 4);
        else if (M <= 64)
            launch(ln_decode_bf16_kernel<4, 4, 2, true, false, 4>, 4, 4);
        else if (M <= 96)
            launch(ln_decode_bf16_kernel<4, 2, 2, true, false, 6>, 4, 2);
        else
            launch(ln_decode_bf16_kernel<4, 2, 2, true, false, 8>, 4, 2);
        return hipGetLastError();
    }
    if (dtype == 0) return run_main<float, 32, 64, 2, 2, BMode::kPacked, Epi::kSwiGlu, kF32Stages, kF32Chunks>(a, 1, s);
    if (use_mid_tiles(M, np, K)) return run_pipe<Epi::kSwiGlu, 128>(a, s);
    if (use_big_tiles(M, np, K)) return run_pipe<Epi::kSwiGlu>(a, s);
    return run_main<__bf16, 128, 128, 2, 2, BMode::kPacked, Epi::kSwiGlu>(a, 1, s);
}

hipError_t launch_gemm(const void* A, const void* B, const void* bias, int64_t batch, int64_t M, int64_t K,
                       int64_t N, int b_layout, int a_causal, int dtype, void* C, hipStream_t s) {
    MainArgs a{};
    if (b_layout == 2) {
        a = packed_args(A, B, M, K, N, dtype, C);
    } else {
        a.A = A;
        a.B = B;
        a.C = C;
        a.M = M;
        a.K = K;
        a.N = N;
        a.sA = M * K;
        a.sB = K * N;
        a.sC = M * N;
    }
    a.bias = bias;
    a.a_causal = a_causal;
    if (b_layout == 2) {
        if (dtype == 1 && decode_rows(M, N)) {
            // decode shapes: the streaming kernel of the deferred path without its moments,
            // in the same layouts (so the unfused comparison is like for like)
            auto launch = [&](auto kern, int ks, int cols) {
                const int64_t wgs = (a.nblocks + cols - 1) / cols;
                kern<<<dim3((unsigned)wgs), ks * kWave, 0, s>>>((const __bf16*)A, (const char*)a.B, a.kchunks,
                                                                a.nblocks, nullptr, nullptr, (int)M, K, N, 0.f, 0,
                                                                N, nullptr, nullptr, (__bf16*)C,
                                                                (const __bf16*)bias);
            };
            decode_dispatch<true>(M, a.nblocks, launch);
            return hipGetLastError();
        }
        if (dtype == 0) return run_main<float, 32, 64, 2, 2, BMode::kPacked, Epi::kGemm, kF32Stages, kF32Chunks>(a, 1, s);
        if (use_mid_tiles(M, N, K)) return run_pipe<Epi::kGemm, 128>(a, s);
        if (use_big_tiles(M, N, K)) return run_pipe<Epi::kGemm>(a, s);
        return run_main<__bf16, 128, 128, 2, 2, BMode::kPacked, Epi::kGemm>(a, 1, s);
    }
    if (dtype == 0) return run_main<float, 32, 64, 2, 2, BMode::kNK, Epi::kGemm, kF32Stages, kF32Chunks>(a, batch, s);
    if (b_layout == 1) return run_main<__bf16, 128, 128, 2, 2, BMode::kNK, Epi::kGemm>(a, batch, s);
    return run_main<__bf16, 128, 128, 2, 2, BMode::kKN, Epi::kGemm>(a, batch, s);
}

}  // namespace dn
