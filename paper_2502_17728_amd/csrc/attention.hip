// attention.hip -- deferred Softmax -> P.V with the scores formed in the
// kernel from Q and K (Eq. (8) carried past the paper's operation boundary):
//
//   out_i = (1 / l_i) * sum_j exp(s_ij - m_i) V_j,   s_ij = scale * q_i . k_j,
//
// the numerators feeding the matrix core un-normalized, the row maximum kept
// online and the row sum reduced alongside, one division in the epilogue.  S
// never exists in memory, so the work is the two products on the MFMA instead
// of a stream of scores from HBM.
//
// Orientation.  Both products are taken transposed so that every lane keeps
// one query: S^T = K . Q^T (A = K fragments from LDS, B = the wave's Q
// fragments, held in registers for the whole kernel) and out^T = V^T . P~^T
// (A = V^T from LDS, B = the numerators).  A 16x16 S^T block leaves lane
// (i, G) (i = lane & 15, G = lane >> 4) the scores of query i against keys
// 4G .. 4G+3 of the block.  Two adjacent blocks therefore give the lane 8
// scores -- keys 4G..4G+3 and 16+4G..16+4G+3 of a 32-key chunk -- which is
// exactly one B-operand fragment of the P~ . V product once the keys of that
// product are taken in the same order; the V^T fragments are read with that
// key order, so no score ever moves between lanes.  The maximum over a
// query's keys needs one exchange across the four lane groups; the row sum is
// one more MFMA per chunk with A = all ones.
//
// Data movement.  One workgroup owns NW x QW x 16 queries of one head and walks
// the keys in steps of BKV (128).  K and V tiles ([BKV keys][d], row-major) share an
// NS-slot ring in LDS filled by global->LDS copies of whole KiB (one barrier
// per step); 16-byte pieces are XOR-swizzled per key row so that the K
// fragment reads (16 rows at one piece) and the transposing V^T reads
// (ds_read_b64_tr_b16) are free of bank conflicts.  Causal: key steps wholly
// above the workgroup's queries are never read; a wave skips the products of
// steps wholly above its own queries; keys above the diagonal inside a step
// are masked to -inf before the exponentials.
//
// Decode (a few new queries against a long key/value cache).  One workgroup
// per head would leave most CUs idle, so the keys of each head are cut into
// ranges, one single-wave workgroup each, sized so that the grid is one
// resident round; every range leaves (acc, l, m) in fp32 and a merge kernel
// combines them with weights 2^(m_g - m) -- the deferred division of Eq. (8)
// postponed once more, past the reduction over key ranges.
#include <algorithm>
#include <mutex>

#include "dn_device.hpp"
#include "dn_launch.hpp"

namespace dn {
namespace fa {
constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4)); }
template <int N>
__device__ __forceinline__ void wait_vmcnt_asm() {
    static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
__device__ __forceinline__ void block_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}
// K rows: the A-operand read takes 16 consecutive rows at one 16-byte piece.
// 256-byte rows span all 64 banks, so each of the 16 rows gets its own slot;
// 128-byte rows alternate bank halves, and the 8 rows of a half get 8 slots.
template <int D>
__device__ __forceinline__ int k_swz(int r) {
    if constexpr (D == 128) return r & 15;
    return (r & 7) ^ ((r >> 3) & 1);
}
// V rows: the transposing read is serviced 32 lanes at a time and, in the key
// order above, covers 8 consecutive key rows; the swizzle (an even piece count,
// so 32-byte blocks stay whole) gives each of them its own 32-byte bank window.
template <int D>
__device__ __forceinline__ int v_swz(int r) {
    if constexpr (D == 128) return 2 * (r & 3) + 8 * ((r >> 2) & 1);
    return 4 * ((r >> 1) & 1) + 2 * ((r >> 2) & 1);
}
typedef short v4s_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint2 lds_tr16(const char* p) {
    v4s_t r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((DN_LDS v4s_t*)(DN_LDS char*)p);
    return __builtin_bit_cast(uint2, r);
}
}  // namespace fa

// STREAM: every key/value row is read by one workgroup only (decode), so the copies
// carry the non-temporal hint; prefill workgroups share them through L2.
template <int D, int NW, int QW, int NS, int BKV, bool STREAM = false>
__global__ __launch_bounds__(NW * 64) void attention_kernel(const __bf16* __restrict__ Q,
                                                            const __bf16* __restrict__ K,
                                                            const __bf16* __restrict__ V, int64_t Lq,
                                                            int64_t Lk, int causal, float sl2, int nqb,
                                                            int nsplit, int64_t kchunk, float* __restrict__ part,
                                                            __bf16* __restrict__ out, int group) {
    using namespace fa;
    constexpr int BQ = NW * QW * 16;   // queries per workgroup
    constexpr int NKB = BKV / 16;      // 16-key S^T blocks per step
    constexpr int NKC = BKV / 32;      // 32-key chunks of the P.V product per step
    constexpr int ROW = D * 2;         // bytes per K or V row
    constexpr int TILE = BKV * ROW;    // one K (or V) tile
    constexpr int SLOT = 2 * TILE;     // ring slot: K tile, then V tile
    constexpr int T_INS = TILE / kChunkBytes / NW;  // copies per wave per tile
    constexpr int KV_INS = 2 * T_INS;
    constexpr int PPR = ROW / 16;      // 16-byte pieces per row
    constexpr int RPI = kChunkBytes / ROW;  // rows per copy instruction
    constexpr int DB = D / 16, DC = D / 32;
    static_assert(TILE % (kChunkBytes * NW) == 0, "tiles split evenly over the waves");
    static_assert(NS >= 2 && (NS - 2) * KV_INS < 64, "ring depth: the copies in flight fit vmcnt");

    __shared__ __attribute__((aligned(1024))) char smem[NS * SLOT];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    // logical id: XCD-contiguous; each XCD walks whole heads, longest query blocks first.
    // Split mode (part != null): the keys are cut into nsplit ranges of kchunk, one per
    // workgroup, each leaving its un-normalized partial sums for the merge kernel.
    const int t0 = xcd_contiguous(blockIdx.x, gridDim.x);
    const int sp = t0 % nsplit, t = t0 / nsplit;
    const int h = t / nqb;
    const int qb = causal ? (nqb - 1 - t % nqb) : (t % nqb);
    const int64_t q0 = (int64_t)qb * BQ;
    const int64_t kv_end = causal ? min(Lk, q0 + BQ) : Lk;
    const int64_t k_lo = (int64_t)sp * kchunk;                  // this workgroup's keys: [k_lo, k_hi)
    const int64_t k_hi = min(kv_end, k_lo + kchunk);
    const int nsteps = (int)((k_hi - k_lo + BKV - 1) / BKV);

    const __bf16* Qh = Q + (int64_t)h * Lq * D;
    // grouped-query attention: query head h reads key/value head h / group
    const __bf16* Kh = K + (int64_t)(h / group) * Lk * D;
    const __bf16* Vh = V + (int64_t)(h / group) * Lk * D;
    __bf16* Oh = out + (int64_t)h * Lq * D;

    const int64_t qw0 = q0 + wave * QW * 16;  // first query of this wave
    const int G = lane >> 4, i = lane & 15;
    int64_t qrow[QW];
#pragma unroll
    for (int f = 0; f < QW; ++f) qrow[f] = qw0 + f * 16 + i;

    // Q^T fragments (B operand of S^T): lane (i, G) holds query 16f + i, d 32c + 8G .. +8
    u32x4 qf[QW][DC];
#pragma unroll
    for (int f = 0; f < QW; ++f) {
        const int64_t qr = qrow[f] < Lq ? qrow[f] : Lq - 1;
#pragma unroll
        for (int c = 0; c < DC; ++c) qf[f][c] = ld16(Qh + qr * D + 32 * c + 8 * G);
    }
    // Q is in registers before the key loop: each fragment is an operand of an empty
    // statement here, so the compiler places its waits for these loads before the
    // loop.  Left to find the first use inside it, it kept waits there on every
    // step, and at run time those also drained the copies issued for the next step.
#pragma unroll
    for (int f = 0; f < QW; ++f)
#pragma unroll
        for (int c = 0; c < DC; ++c) asm volatile("" : "+v"(qf[f][c]));
    wait_vmcnt_asm<0>();  // before the hand-counted copies below start

    // ---- K/V ring.  Copy instruction j of a wave covers tile rows
    // RPI * (wave + j * NW) .. + RPI; lane l fetches piece (l % PPR) ^ swz(row),
    // so logical piece p of a row lands in slot p ^ swz(row).  Keys past Lk
    // clamp onto the last row (their scores are masked); byte offsets from the
    // head's base fit 32 bits (Lk * d * 2 < 2^32).
    uint32_t c_row[T_INS], k_p16[T_INS], v_p16[T_INS];
#pragma unroll
    for (int j = 0; j < T_INS; ++j) {
        const int r = (wave + j * NW) * RPI + lane / PPR;
        c_row[j] = (uint32_t)r;
        k_p16[j] = (uint32_t)(((lane % PPR) ^ k_swz<D>(r)) * 16);
        v_p16[j] = (uint32_t)(((lane % PPR) ^ v_swz<D>(r)) * 16);
    }
    const uint64_t k_base = uniform_u64(Kh), v_base = uniform_u64(Vh);
    const uint32_t last = (uint32_t)(Lk - 1);
    const uint32_t smem_addr = lds_addr32(smem);
    auto issue_kv = [&](int step) {
        const uint32_t base = smem_addr + (uint32_t)((step % NS) * SLOT);
        const uint32_t k0 = (uint32_t)k_lo + (uint32_t)step * BKV;
#pragma unroll
        for (int j = 0; j < T_INS; ++j) {
            const uint32_t key = k0 + c_row[j] < last ? k0 + c_row[j] : last;  // a select, no branch
            const uint32_t dst = base + (uint32_t)((wave + j * NW) * kChunkBytes);
            if constexpr (STREAM) {
                g2lds16_stream_sb(k_base, key * (uint32_t)ROW + k_p16[j], dst);
                g2lds16_stream_sb(v_base, key * (uint32_t)ROW + v_p16[j], dst + TILE);
            } else {
                g2lds16_async_sb(k_base, key * (uint32_t)ROW + k_p16[j], dst);
                g2lds16_async_sb(v_base, key * (uint32_t)ROW + v_p16[j], dst + TILE);
            }
        }
    };

    // Lane-constant LDS offsets.  K: row 16 kb + i, logical piece 4c + G (the
    // swizzle depends on the row only through i).  V^T: two transposing reads
    // per 16-wide d block, the first covering keys 4G .. 4G+3 of the chunk, the
    // second keys 16+4G .. 16+4G+3 (within a 16-lane group, lane j, slot t gets
    // element j & 3 of the 8 bytes lane 4t + (j >> 2) reads, so lane (i, G)
    // reads row 4G + (i >> 2), d 4 (i & 3) .. +3 of the block).
    int k_rd[DC];
#pragma unroll
    for (int c = 0; c < DC; ++c) k_rd[c] = i * ROW + (((4 * c + G) ^ k_swz<D>(i)) << 4);
    const int vr = 4 * G + (i >> 2);
    const int vsw2 = v_swz<D>(vr) >> 1;  // swizzle of the 32-byte d block
    int v_off[DB];
#pragma unroll
    for (int b = 0; b < DB; ++b) v_off[b] = vr * ROW + (i & 3) * 8 + 32 * (b ^ vsw2);

    f32x4 acc[QW][DB], accl[QW];
#pragma unroll
    for (int f = 0; f < QW; ++f) {
#pragma unroll
        for (int b = 0; b < DB; ++b) acc[f][b] = f32x4{0.f, 0.f, 0.f, 0.f};
        accl[f] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    const u32x4 ones = {0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u};

    // Reference maximum per query in scaled log2 units, raised only when a step
    // exceeds it by more than 8 (numerators stay below 256; the rescale of the
    // partial sums, an exact identity, is rare).
    float mref[QW];
#pragma unroll
    for (int f = 0; f < QW; ++f) mref[f] = -__builtin_inff();

    const int qw0i = (int)qw0, kv_endi = (int)k_hi;  // positions fit 32 bits (checked by the host)
    const int qlast = qw0i + QW * 16 - 1;              // this wave's last query

    // scores S^T of one step: 4 blocks of 16 keys per query fragment
    auto scores = [&](int step, f32x4(&st)[QW][NKB]) {
        const char* kb = smem + (step % NS) * SLOT;
#pragma unroll
        for (int f = 0; f < QW; ++f)
#pragma unroll
            for (int b4 = 0; b4 < NKB; ++b4) st[f][b4] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int b4 = 0; b4 < NKB; ++b4)
#pragma unroll
            for (int c = 0; c < DC; ++c) {
                const u32x4 kf = lds_ld16(lds_ptr((char*)kb + b4 * 16 * ROW + k_rd[c]));
#pragma unroll
                for (int f = 0; f < QW; ++f) st[f][b4] = mfma_chunk<__bf16>(kf, qf[f][c], st[f][b4]);
            }
    };
    // numerators of one step (keys past the diagonal or past Lk masked first),
    // with the reference max raised where needed; returns whether any lane raised it
    auto numerators = [&](int step, f32x4(&st)[QW][NKB], u32x4(&pf)[QW][NKC], float(&alpha)[QW]) {
        const int k0 = (int)k_lo + step * BKV;
        if ((causal && k0 + BKV - 1 > qw0i) || k0 + BKV > kv_endi) {
#pragma unroll
            for (int f = 0; f < QW; ++f) {
                const int lim = causal ? min((int)qrow[f], kv_endi - 1) : kv_endi - 1;
#pragma unroll
                for (int b4 = 0; b4 < NKB; ++b4) {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (k0 + 16 * b4 + 4 * G + e > lim) st[f][b4][e] = -__builtin_inff();
                    // one block's compare masks at a time: issued all at once they
                    // took 64 SGPRs and pushed loop-long scalars into VGPR lanes
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
        }
        bool raised = false;
#pragma unroll
        for (int f = 0; f < QW; ++f) {
            float tmax = st[f][0][0];
#pragma unroll
            for (int b4 = 0; b4 < NKB; ++b4)
#pragma unroll
                for (int e = 0; e < 4; ++e) tmax = __builtin_fmaxf(tmax, st[f][b4][e]);
            const float tmax2 = max_lane_groups(tmax) * sl2;
            const bool raise = tmax2 > mref[f] + 8.0f;
            const float mnew = raise ? tmax2 : mref[f];
            alpha[f] = __builtin_amdgcn_exp2f(raise ? mref[f] - mnew : 0.f);
            mref[f] = mnew;
            raised |= raise;
            const float nb = mnew == -__builtin_inff() ? 0.f : -mnew;
            float p[NKB][4];
#pragma unroll
            for (int b4 = 0; b4 < NKB; ++b4)
#pragma unroll
                for (int e = 0; e < 4; ++e) p[b4][e] = __builtin_amdgcn_exp2f(__builtin_fmaf(st[f][b4][e], sl2, nb));
#pragma unroll
            for (int kc = 0; kc < NKC; ++kc)
                pf[f][kc] = u32x4{pack_bf16(p[2 * kc][0], p[2 * kc][1]), pack_bf16(p[2 * kc][2], p[2 * kc][3]),
                                  pack_bf16(p[2 * kc + 1][0], p[2 * kc + 1][1]),
                                  pack_bf16(p[2 * kc + 1][2], p[2 * kc + 1][3])};
        }
        return raised;
    };
    // out^T += V^T . P~^T, keys of chunk kc in the order of the numerators
    auto products = [&](int step, const u32x4(&pf)[QW][NKC]) {
        const char* vb = smem + (step % NS) * SLOT + TILE;
#pragma unroll
        for (int kc = 0; kc < NKC; ++kc) {
            u32x4 vf[DB];
#pragma unroll
            for (int b = 0; b < DB; ++b) {
                const uint2 lo = lds_tr16(vb + v_off[b] + (kc * 32) * ROW);
                const uint2 hi = lds_tr16(vb + v_off[b] + (kc * 32 + 16) * ROW);
                vf[b] = u32x4{lo.x, lo.y, hi.x, hi.y};
            }
#pragma unroll
            for (int b = 0; b < DB; ++b)
#pragma unroll
                for (int f = 0; f < QW; ++f) acc[f][b] = mfma_chunk<__bf16>(vf[b], pf[f][kc], acc[f][b]);
#pragma unroll
            for (int f = 0; f < QW; ++f) accl[f] = mfma_chunk<__bf16>(ones, pf[f][kc], accl[f]);
        }
    };
    auto rescale = [&](bool raised, const float(&alpha)[QW]) {
        if (__any(raised)) {
#pragma unroll
            for (int f = 0; f < QW; ++f) {
#pragma unroll
                for (int b = 0; b < DB; ++b) acc[f][b] *= alpha[f];
                accl[f] *= alpha[f];
            }
        }
    };
    auto active = [&](int step) { return step < nsteps && !(causal && (int)k_lo + step * BKV > qlast); };

    for (int s = 0; s < NS - 1; ++s) issue_kv(s);
    for (int s = 0; s < nsteps; ++s) {
        wait_vmcnt_asm<(NS - 2) * KV_INS>();  // this wave's copies of step s have landed
        wait_lgkm0();                         // its LDS reads of step s-1 are done
        block_barrier();                      // ... and every wave's
        issue_kv(s + NS - 1);                 // into the slot step s-1 vacated
        if (!active(s)) continue;             // wholly above this wave's queries
        f32x4 st[QW][NKB];
        scores(s, st);
        u32x4 pf[QW][NKC];
        float alpha[QW];
        const bool raised = numerators(s, st, pf, alpha);
        rescale(raised, alpha);
        products(s, pf);
    }
    wait_vmcnt_asm<0>();  // no copy into LDS may outlive the workgroup

    if (part) {
        // split mode: the partial (acc[d], l, m, 2 pad) of each query row, fp32, for the merge
#pragma unroll
        for (int f = 0; f < QW; ++f) {
            if (qrow[f] >= Lq) continue;
            float* pr = part + (((int64_t)h * Lq + qrow[f]) * nsplit + sp) * (D + 4);  // 16-byte rows
#pragma unroll
            for (int b = 0; b < DB; ++b)
                *reinterpret_cast<f32x4*>(pr + b * 16 + 4 * G) = acc[f][b];
            if (G == 0) {
                pr[D] = accl[f][0];
                pr[D + 1] = mref[f];
            }
        }
        return;
    }

    // ---- epilogue: the single deferred division, one rounding to bf16
#pragma unroll
    for (int f = 0; f < QW; ++f) {
        if (qrow[f] >= Lq) continue;
        const float inv = 1.0f / accl[f][0];
        __bf16* orow = Oh + qrow[f] * D + 4 * G;
#pragma unroll
        for (int b = 0; b < DB; ++b) {
            uint2 v;
            v.x = pack_bf16(acc[f][b][0] * inv, acc[f][b][1] * inv);
            v.y = pack_bf16(acc[f][b][2] * inv, acc[f][b][3] * inv);
            *reinterpret_cast<uint2*>(orow + b * 16) = v;
        }
    }
}

template <int D, int NW, int QW, int NS, int BKV>
static hipError_t run_attention(const void* Q, const void* K, const void* V, int64_t BH, int64_t Lq, int64_t Lk,
                                int causal, float scale, void* out, hipStream_t s, int group) {
    constexpr int BQ = NW * QW * 16;
    const int nqb = (int)((Lq + BQ - 1) / BQ);
    attention_kernel<D, NW, QW, NS, BKV><<<dim3((unsigned)(BH * nqb)), NW * 64, 0, s>>>(
        (const __bf16*)Q, (const __bf16*)K, (const __bf16*)V, Lq, Lk, causal, scale * fa::kLog2e, nqb, 1, Lk,
        nullptr, (__bf16*)out, group);
    return hipGetLastError();
}

// Merge of the split partials (the log-sum-exp combination of Eq. (8) over key
// ranges): m = max_g m_g, out = sum_g 2^(m_g - m) acc_g / sum_g 2^(m_g - m) l_g,
// one wave per query row.
template <int D>
__global__ __launch_bounds__(256) void attention_merge_kernel(const float* __restrict__ part, int nsplit,
                                                              int64_t rows, __bf16* __restrict__ out) {
    constexpr int PER = D / 64;
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= rows) return;
    const float* pr = part + row * nsplit * (D + 4);
    float m = -__builtin_inff();
    for (int g = 0; g < nsplit; ++g) m = __builtin_fmaxf(m, pr[g * (D + 4) + D + 1]);
    float l = 0.f, acc[PER];
#pragma unroll
    for (int j = 0; j < PER; ++j) acc[j] = 0.f;
    for (int g = 0; g < nsplit; ++g) {
        const float* pg = pr + g * (D + 4);
        const float w = __builtin_amdgcn_exp2f(pg[D + 1] - m);
        l = __builtin_fmaf(w, pg[D], l);
#pragma unroll
        for (int j = 0; j < PER; ++j) acc[j] = __builtin_fmaf(w, pg[lane + 64 * j], acc[j]);
    }
    const float inv = 1.0f / l;
#pragma unroll
    for (int j = 0; j < PER; ++j) out[row * D + lane + 64 * j] = (__bf16)(acc[j] * inv);
}

// Decode kernel: one wave of 16 query slots per workgroup (Lq <= 16), 128-key steps, a
// ring of 2 slots (the next step's copies in flight while one is computed): 1024 d
// bytes of LDS.  Measured on 256 heads x 8192 keys, d = 128, per call:
// 157 us, against 164 us for 3 slots of 64 keys, 167 us for 2 of 64 and 173 us for
// 4 of 32 -- fewer, larger copies in flight per workgroup stream best.
constexpr int kDecNS = 2, kDecBKV = 128;
constexpr int64_t kCUs = 256, kLdsPerCU = 160 * 1024;
inline int64_t decode_lds_bytes(int64_t d) { return (int64_t)kDecNS * 2 * kDecBKV * d * 2; }

// Decode split: as many workgroups as fit on the chip at once (LDS-bound: 1 per CU at
// d = 128, 2 at d = 64), spread over the heads; each split a whole number of steps.
// One resident round beats 2 and 4 rounds (their tails).
static void attention_decode_split(int64_t BH, int64_t Lk, int64_t d, int* nsplit, int64_t* kchunk) {
    const int64_t wgs = kCUs * (kLdsPerCU / decode_lds_bytes(d));
    const int64_t steps = (Lk + kDecBKV - 1) / kDecBKV;
    const int64_t want = std::max<int64_t>(1, std::min<int64_t>(steps, (wgs + BH - 1) / BH));
    const int64_t per = (steps + want - 1) / want;  // steps per split
    *kchunk = per * kDecBKV;
    *nsplit = (int)((Lk + *kchunk - 1) / *kchunk);
}

template <int D>
static hipError_t run_attention_decode(const void* Q, const void* K, const void* V, int64_t BH, int64_t Lq,
                                       int64_t Lk, float scale, float* part, void* out, hipStream_t s) {
    int nsplit;
    int64_t kchunk;
    attention_decode_split(BH, Lk, D, &nsplit, &kchunk);
    if (nsplit == 1) {  // enough heads to fill the chip: one pass, the division in the kernel's epilogue
        attention_kernel<D, 1, 1, kDecNS, kDecBKV, true><<<dim3((unsigned)BH), 64, 0, s>>>(
            (const __bf16*)Q, (const __bf16*)K, (const __bf16*)V, Lq, Lk, 0, scale * fa::kLog2e, 1, 1, Lk,
            nullptr, (__bf16*)out, 1);
        return hipGetLastError();
    }
    attention_kernel<D, 1, 1, kDecNS, kDecBKV, true><<<dim3((unsigned)(BH * nsplit)), 64, 0, s>>>(
        (const __bf16*)Q, (const __bf16*)K, (const __bf16*)V, Lq, Lk, 0, scale * fa::kLog2e, 1, nsplit, kchunk,
        part, nullptr, 1);
    const int64_t rows = BH * Lq;
    attention_merge_kernel<D><<<dim3((unsigned)((rows + 3) / 4)), 256, 0, s>>>(part, nsplit, rows, (__bf16*)out);
    return hipGetLastError();
}

size_t attention_decode_workspace_bytes(int64_t BH, int64_t Lq, int64_t Lk, int64_t d) {
    int nsplit;
    int64_t kchunk;
    attention_decode_split(BH, Lk, d, &nsplit, &kchunk);
    return (size_t)BH * (size_t)Lq * (size_t)nsplit * (size_t)(d + 4) * sizeof(float);
}

hipError_t launch_attention_decode(const void* Q, const void* K, const void* V, int64_t BH, int64_t Lq, int64_t Lk,
                                   int64_t d, float scale, void* workspace, void* out, hipStream_t s) {
    if (d == 64) return run_attention_decode<64>(Q, K, V, BH, Lq, Lk, scale, (float*)workspace, out, s);
    return run_attention_decode<128>(Q, K, V, BH, Lq, Lk, scale, (float*)workspace, out, s);
}

// ---------------------------------------------------------------------------
// Allocation-free decode: the per-split partials go to a file-scope device array
// instead of a caller workspace.  Every valid call fits it: with nsplit > 1 the
// heads number fewer than the resident workgroups W (512 at d = 64, 256 at
// d = 128), so BH * nsplit < 2 W and the partials take less than
// 2 W * 16 * (d + 4) * 4 bytes -- 4.25 MiB at d = 64, 4.125 MiB at d = 128.
// In host code `scratch` names a host-side stand-in; its device address (one
// copy per GPU) is looked up once per device with hipGetSymbolAddress and only
// that address is passed to kernels.
static __device__ __align__(256) float scratch[kDecodeScratchBytes / sizeof(float)];

static hipError_t decode_scratch_address(void** out) {
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static void* addr[kMaxDevices] = {};
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));  // on the current device
        if (e != hipSuccess) return e;
        addr[dev] = p;
    }
    *out = addr[dev];
    return hipSuccess;
}

size_t attention_decode_partials_bytes(int64_t BH, int64_t Lq, int64_t Lk, int64_t d) {
    int nsplit;
    int64_t kchunk;
    attention_decode_split(BH, Lk, d, &nsplit, &kchunk);
    return nsplit == 1 ? 0 : (size_t)BH * (size_t)Lq * (size_t)nsplit * (size_t)(d + 4) * sizeof(float);
}

hipError_t launch_attention_decode_noalloc(const void* Q, const void* K, const void* V, int64_t BH, int64_t Lq,
                                           int64_t Lk, int64_t d, float scale, void* out, hipStream_t s) {
    void* part = nullptr;
    if (attention_decode_partials_bytes(BH, Lq, Lk, d) > 0) {
        const hipError_t e = decode_scratch_address(&part);
        if (e != hipSuccess) return e;
    }
    return launch_attention_decode(Q, K, V, BH, Lq, Lk, d, scale, part, out, s);
}

hipError_t launch_attention_deferred(const void* Q, const void* K, const void* V, int64_t BH, int64_t Lq,
                                     int64_t Lk, int64_t d, int causal, float scale, void* out, hipStream_t s,
                                     int group) {
    // 8 waves x 2 query fragments (256 queries per workgroup), two ring slots of 128 keys
    // (128 KiB of LDS at d = 128): measured fastest against 64-key steps, 3 slots, 1 or 3
    // fragments, and 4 waves on the causal 32 x 8192 x 8192, d = 128.  BH counts query heads.
    if (d == 64) return run_attention<64, 8, 2, 2, 128>(Q, K, V, BH, Lq, Lk, causal, scale, out, s, group);
    return run_attention<128, 8, 2, 2, 128>(Q, K, V, BH, Lq, Lk, causal, scale, out, s, group);
}

}  // namespace dn
