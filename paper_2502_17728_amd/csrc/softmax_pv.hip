// softmax_pv.hip -- deferred Softmax -> P.V (Sec. II-B, Eq. (8)).
//
// out_i = (1 / l_i) * sum_j exp(s_ij - m_i) V_j,   l_i = sum_j exp(s_ij - m_i),
// with m_i the row maximum (footnote of Eq. (7)).  The matrix core consumes the
// un-normalized numerators; the collective part (max and sum over the row) is
// reduced alongside, and the single division happens in the epilogue.
//
// Keys are streamed in steps of 64.  Because S is materialized, the maximum is
// kept online as a reference value m: when a step's scores exceed it enough
// to matter, m moves to m' and the partial products and the partial sum are
// scaled by exp(m - m') -- Eq. (8) applied to the row prefix, which leaves the
// result unchanged in exact arithmetic.  Any reference works (the footnote's
// shift invariance); it only has to keep the numerators in range.
//
// Orientation.  The kernel computes out^T = V^T . P~^T with V^T as the MFMA A
// operand and the numerator fragment P~ as the B operand, so lane l owns query
// (l & 15) both in its P~ fragment and in its accumulator columns: the rescale
// and the final 1/l are lane-local.  The row sum is one more MFMA per chunk
// with A = all ones, which sums exactly the bf16-rounded numerators the
// product used and keeps the VALU -- the second bottleneck after HBM -- free of
// the additions.
//
// Data movement.  One workgroup owns NW x 32 queries of one head (NW waves of 32).
// Per step it copies the S tile (BQ rows x 128 bytes, 8 rows of full cache
// lines per wave instruction) and the V tile (64 keys x d, contiguous in
// memory, one KiB per instruction) into an NS-deep LDS ring with global->LDS
// copies issued NS-1 steps ahead.  S pieces are XOR-swizzled (rows of
// one fragment read hit distinct banks).  V stays in its row-major [key][d]
// layout, pieces XOR-swizzled per key row, and the V^T operand -- eight
// consecutive keys of one d per lane -- is read with two transposing LDS reads
// (ds_read_b64_tr_b16: within a 16-lane group, lane j, slot t receives element
// j & 3 of the 8 bytes read by lane 4t + (j >> 2)).
#include <type_traits>

#include "dn_device.hpp"
#include "dn_launch.hpp"

namespace dn {

constexpr float kLog2e = 1.4426950408889634f;

namespace sm {
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4)); }
__device__ __forceinline__ void block_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}
// v_max3_f32 directly: fmaxf on values assembled from bit operations gets an
// extra canonicalizing max per operand from the compiler.  Its operands are
// bf16 widenings (shifts and masks), never transcendental results.
__device__ __forceinline__ float max3f(float a, float b, float c) {
    float d;
    asm("v_max3_f32 %0, %1, %2, %3" : "=v"(d) : "v"(a), "v"(b), "v"(c));
    return d;
}
// Scale a 4-float accumulator in place (tied operands keep it in its registers).
// alpha is the result of v_exp_f32; a transcendental result needs one wait
// state before a non-transcendental VALU reads it, and the compiler's hazard
// pass does not insert it in front of inline assembly -- hence the s_nop.
__device__ __forceinline__ void scale_inplace(f32x4& a, float alpha) {
    asm volatile("s_nop 0\n\tv_mul_f32 %0, %0, %4\n\tv_mul_f32 %1, %1, %4\n\tv_mul_f32 %2, %2, %4\n\tv_mul_f32 %3, %3, %4"
                 : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(a[3])
                 : "v"(alpha));
}
__device__ __forceinline__ int s_swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }  // 128-byte S rows
// V pieces: the transposing read is serviced 32 lanes at a time, covering 8 key
// rows (4 per 16-lane group, two groups 8 rows apart); the swizzle gives each
// of those rows its own 32-byte bank window.  256-byte rows (d = 128): 8
// windows per row; 128-byte rows (d = 64): rows alternate bank halves, so 4
// windows per half.
template <int D>
__device__ __forceinline__ int v_swz(int r) {
    if constexpr (D == 128) return 2 * (r & 3) + 8 * ((r >> 3) & 1);
    return 4 * ((r >> 1) & 1) + 2 * ((r >> 3) & 1);
}
typedef short v4s_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint2 lds_tr16(const char* p) {
    v4s_t r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((DN_LDS v4s_t*)(DN_LDS char*)p);
    return __builtin_bit_cast(uint2, r);
}
}  // namespace sm

template <int D, int NW, int NS>
__global__ __launch_bounds__(NW * 64) void softmax_pv_kernel(const __bf16* __restrict__ S,
                                                         const __bf16* __restrict__ V, int BH,
                                                         int64_t Lq, int64_t Lk, int causal, int nqb,
                                                         __bf16* __restrict__ out) {
    using namespace sm;
    constexpr int QW = 2;                  // 16-query fragments per wave
    constexpr int BQ = NW * QW * 16;       // queries per workgroup
    constexpr int BKV = 64;                // keys per step
    constexpr int S_BYTES = BQ * BKV * 2;
    constexpr int VROW = D * 2;            // bytes per V row
    constexpr int V_BYTES = BKV * VROW;
    constexpr int STAGE = S_BYTES + V_BYTES;
    constexpr int S_INS = BQ / 8 / NW;     // S copies per wave per step
    constexpr int V_INS = V_BYTES / kChunkBytes / NW;
    constexpr int PER = S_INS + V_INS;
    constexpr int VPR = VROW / 16;         // 16-byte pieces per V row
    constexpr int VRPI = kChunkBytes / VROW;  // V rows per copy instruction
    constexpr int DB = D / 16;
    static_assert(V_BYTES % (kChunkBytes * NW) == 0, "V tile split evenly over the waves");
    static_assert(NS == 2 || NS == 3, "ring depth");

    __shared__ __attribute__((aligned(1024))) char smem[NS * STAGE];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    // logical id: XCD-contiguous; each XCD walks whole heads, longest query blocks first
    const int t = xcd_contiguous(blockIdx.x, gridDim.x);
    const int h = t / nqb;
    const int qb = causal ? (nqb - 1 - t % nqb) : (t % nqb);
    const int64_t q0 = (int64_t)qb * BQ;
    const int64_t kv_end = causal ? min(Lk, q0 + BQ) : Lk;
    const int nsteps = (int)((kv_end + BKV - 1) / BKV);

    const __bf16* Sh = S + (int64_t)h * Lq * Lk;
    const __bf16* Vh = V + (int64_t)h * Lk * D;
    __bf16* Oh = out + (int64_t)h * Lq * D;

    const int64_t qw0 = q0 + wave * QW * 16;  // first query of this wave
    int64_t qrow[QW];
#pragma unroll
    for (int f = 0; f < QW; ++f) qrow[f] = qw0 + f * 16 + (lane & 15);

    // ---- copy sources.  S: instruction i covers tile rows 8i..8i+7; V: piece i covers rows VRPI*i..
    const __bf16* s_row[S_INS];
    int s_piece[S_INS];
#pragma unroll
    for (int j = 0; j < S_INS; ++j) {
        const int r = (wave + j * NW) * 8 + (lane >> 3);
        s_piece[j] = (lane & 7) ^ s_swz(r);
        s_row[j] = Sh + min(q0 + r, Lq - 1) * Lk;
    }
    int v_row[V_INS], v_piece[V_INS];
#pragma unroll
    for (int j = 0; j < V_INS; ++j) {
        const int r = (wave + j * NW) * VRPI + lane / VPR;
        v_row[j] = r;
        v_piece[j] = (lane % VPR) ^ v_swz<D>(r);
    }
    const uint32_t smem_addr = lds_addr32(smem);
    auto issue = [&](int step) {
        const uint32_t base = smem_addr + (uint32_t)((step % NS) * STAGE);
        const int64_t k0 = (int64_t)step * BKV;
        const bool tail = k0 + BKV > Lk;  // only the last step of a ragged key range needs clamping
#pragma unroll
        for (int j = 0; j < S_INS; ++j) {
            const int64_t key = tail ? min(k0 + s_piece[j] * 8, Lk - 8) : k0 + s_piece[j] * 8;
            g2lds16_async(s_row[j] + key, base + (uint32_t)((wave + j * NW) * kChunkBytes));
        }
#pragma unroll
        for (int j = 0; j < V_INS; ++j) {
            const int64_t key = tail ? min(k0 + v_row[j], Lk - 1) : k0 + v_row[j];
            g2lds16_async(Vh + key * D + v_piece[j] * 8, base + (uint32_t)(S_BYTES + (wave + j * NW) * kChunkBytes));
        }
    };

    f32x4 acc[QW][DB], accl[QW];
#pragma unroll
    for (int f = 0; f < QW; ++f) {
#pragma unroll
        for (int b = 0; b < DB; ++b) acc[f][b] = f32x4{0.f, 0.f, 0.f, 0.f};
        accl[f] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    const u32x4 ones = {0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u};

#pragma unroll
    for (int st = 0; st < NS - 1; ++st)
        if (st < nsteps) issue(st);

    // Lane-constant LDS offsets.  The S swizzle depends only on the row's low 4
    // bits (lane & 15); the V swizzle only on bits of (8G + (i >> 2)), which the
    // chunk (kc) and half (hh) offsets leave unchanged.  The per-step parts are
    // uniform and fold into the instructions' immediate offsets.
    const int G = lane >> 4, i = lane & 15;
    int s_off[2];
#pragma unroll
    for (int kc = 0; kc < 2; ++kc)
        s_off[kc] = (wave * QW * 16 + i) * 128 + (((kc * 4 + G) ^ s_swz(i)) << 4);
    const int vsw2 = v_swz<D>(8 * G + (i >> 2)) >> 1;  // even swizzle, applied to the 32-byte d block
    int v_off[DB];
#pragma unroll
    for (int b = 0; b < DB; ++b)
        v_off[b] = (8 * G + (i >> 2)) * VROW + ((i & 3) >> 1) * 16 + (i & 1) * 8 + 32 * (b ^ vsw2);

    // Reference maximum per query, in log2 units.  It is raised only when a tile
    // exceeds it by more than 8, so the numerators exp2(s log2e - mref) stay
    // below 256 (exact as well in bf16 and fp32) and the rescale of the partial
    // products -- an exact identity -- is rare.
    float mref[QW];
#pragma unroll
    for (int f = 0; f < QW; ++f) mref[f] = -__builtin_inff();

    for (int step = 0; step < nsteps; ++step) {
        // this wave's copies of this step have landed (later steps may still be in flight)
        if (NS > 2 && step + 1 < nsteps)
            wait_vmcnt<(NS > 2 ? PER : 0)>();
        else
            wait_vmcnt<0>();
        wait_lgkm0();  // this wave's reads of the previous step are complete
        block_barrier();
        if (step + NS - 1 < nsteps) issue(step + NS - 1);  // into the buffer the previous step vacated

        const int64_t k0 = (int64_t)step * BKV;
        // this wave has work unless every key of the step lies above all of its queries
        if (causal && k0 > qw0 + QW * 16 - 1) continue;
        const char* sb = smem + (step % NS) * STAGE;
        const char* vb = sb + S_BYTES;

        u32x4 sraw[QW][2];
#pragma unroll
        for (int f = 0; f < QW; ++f)
#pragma unroll
            for (int kc = 0; kc < 2; ++kc) sraw[f][kc] = lds_ld16(lds_ptr((char*)sb + s_off[kc] + f * 16 * 128));
        // V^T fragments (A operand) of key chunk kc: two transposing reads of 4 keys per d block
        auto read_v = [&](int kc, u32x4(&vf)[DB]) {
#pragma unroll
            for (int b = 0; b < DB; ++b) {
                const uint2 lo = lds_tr16(vb + v_off[b] + (kc * 32) * VROW);
                const uint2 hi = lds_tr16(vb + v_off[b] + (kc * 32 + 4) * VROW);
                vf[b] = u32x4{lo.x, lo.y, hi.x, hi.y};
            }
        };
        u32x4 vf0[DB], vf1[DB];
        read_v(0, vf0);  // in flight during the softmax arithmetic below
        __builtin_amdgcn_sched_barrier(0);

        const bool edge = (causal && k0 + BKV - 1 > qw0) || k0 + BKV > kv_end;
        u32x4 pf[QW][2];
#pragma unroll
        for (int f = 0; f < QW; ++f) {
            float sv[2][8];
#pragma unroll
            for (int kc = 0; kc < 2; ++kc) {
                const uint32_t w[4] = {sraw[f][kc].x, sraw[f][kc].y, sraw[f][kc].z, sraw[f][kc].w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    sv[kc][2 * e] = bf_lo(w[e]);
                    sv[kc][2 * e + 1] = bf_hi(w[e]);
                }
            }
            if (edge) {  // keys beyond the row (causal) or beyond Lk are not part of it
                const int64_t last = causal ? (qrow[f] < kv_end - 1 ? qrow[f] : kv_end - 1) : kv_end - 1;
                const int64_t rel = last - k0;  // last kept key, relative to the step
                const int lim = rel < 0 ? -1 : (rel > BKV ? BKV : (int)rel);
#pragma unroll
                for (int kc = 0; kc < 2; ++kc)
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (kc * 32 + G * 8 + e > lim) sv[kc][e] = -__builtin_inff();
            }
            // balanced max tree over the lane's 16 scores, then across the 4 lanes of the query
            const float m0 = max3f(sv[0][0], sv[0][1], sv[0][2]), m1 = max3f(sv[0][3], sv[0][4], sv[0][5]);
            const float m2 = max3f(sv[0][6], sv[0][7], sv[1][0]), m3 = max3f(sv[1][1], sv[1][2], sv[1][3]);
            const float m4 = max3f(sv[1][4], sv[1][5], sv[1][6]);
            const float tmax = max3f(max3f(m0, m1, m2), max3f(m3, m4, sv[1][7]), m0);
            const float tmax2 = max_lane_groups(tmax) * kLog2e;
            const bool raise = tmax2 > mref[f] + 8.0f;
            if (__any(raise)) {
                const float mnew = raise ? tmax2 : mref[f];
                const float alpha = __builtin_amdgcn_exp2f(mref[f] - mnew);  // 1 if unchanged, 0 from -inf
#pragma unroll
                for (int b = 0; b < DB; ++b) scale_inplace(acc[f][b], alpha);
                scale_inplace(accl[f], alpha);
                mref[f] = mnew;
            }
            const float nb = mref[f] == -__builtin_inff() ? 0.f : -mref[f];
#pragma unroll
            for (int kc = 0; kc < 2; ++kc)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[kc][2 * e], kLog2e, nb));
                    const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[kc][2 * e + 1], kLog2e, nb));
                    pf[f][kc][e] = pack_bf16(p0, p1);
                }
        }
        __builtin_amdgcn_sched_barrier(0);
        read_v(1, vf1);  // in flight during chunk 0's products
#pragma unroll
        for (int b = 0; b < DB; ++b)
#pragma unroll
            for (int f = 0; f < QW; ++f) acc[f][b] = mfma_chunk<__bf16>(vf0[b], pf[f][0], acc[f][b]);
#pragma unroll
        for (int f = 0; f < QW; ++f) accl[f] = mfma_chunk<__bf16>(ones, pf[f][0], accl[f]);
#pragma unroll
        for (int b = 0; b < DB; ++b)
#pragma unroll
            for (int f = 0; f < QW; ++f) acc[f][b] = mfma_chunk<__bf16>(vf1[b], pf[f][1], acc[f][b]);
#pragma unroll
        for (int f = 0; f < QW; ++f) accl[f] = mfma_chunk<__bf16>(ones, pf[f][1], accl[f]);
    }
    wait_vmcnt<0>();

    // ---- epilogue: the single deferred division, one rounding to bf16
#pragma unroll
    for (int f = 0; f < QW; ++f) {
        if (qrow[f] >= Lq) continue;
        const float inv = 1.0f / accl[f][0];
        __bf16* orow = Oh + qrow[f] * D + 4 * (lane >> 4);
#pragma unroll
        for (int b = 0; b < DB; ++b) {
            uint2 v;
            v.x = pack_bf16(acc[f][b][0] * inv, acc[f][b][1] * inv);
            v.y = pack_bf16(acc[f][b][2] * inv, acc[f][b][3] * inv);
            *reinterpret_cast<uint2*>(orow + b * 16) = v;
        }
    }
}

template <int D, int NW, int NS>
static hipError_t run_softmax_pv(const void* S, const void* V, int64_t BH, int64_t Lq, int64_t Lk, int causal,
                                 void* out, hipStream_t s) {
    constexpr int BQ = NW * 32;
    const int nqb = (int)((Lq + BQ - 1) / BQ);
    dim3 grid((unsigned)(BH * nqb));
    softmax_pv_kernel<D, NW, NS><<<grid, NW * 64, 0, s>>>((const __bf16*)S, (const __bf16*)V, (int)BH, Lq, Lk, causal,
                                                          nqb, (__bf16*)out);
    return hipGetLastError();
}

// 8 waves x 32 queries and a two-stage ring: 80 KiB (d = 64) or 96 KiB (d = 128)
// of LDS, one workgroup per CU; measured faster than 4 waves or three stages
// on the causal 32 x 8192 x 128 workload.
constexpr int kSmWaves = 8, kSmStages = 2;

hipError_t launch_softmax_pv_deferred(const void* S, const void* V, int64_t BH, int64_t Lq, int64_t Lk, int64_t d,
                                      int causal, void* out, hipStream_t s) {
    if (d == 64) return run_softmax_pv<64, kSmWaves, kSmStages>(S, V, BH, Lq, Lk, causal, out, s);
    return run_softmax_pv<128, kSmWaves, kSmStages>(S, V, BH, Lq, Lk, causal, out, s);
}

}  // namespace dn
