// softmax_pv.hip -- deferred Softmax -> P.V (Sec. II-B, Eq. (8)).
//
// out_i = (1 / l_i) * sum_j exp(s_ij - m_i) V_j,   l_i = sum_j exp(s_ij - m_i),
// with m_i the row maximum (footnote of Eq. (7)).  The matrix core consumes the
// un-normalized numerators; the collective part (max and sum over the row) is
// reduced alongside, and the single division happens in the epilogue.
//
// Keys are streamed in steps of 64.  Because S is materialized, the maximum is
// kept online: when a step raises a row's running max from m to m', the
// partial products and the partial sum are scaled by exp(m - m') -- Eq. (8)
// applied to the row prefix, which leaves the result unchanged in exact
// arithmetic.
//
// Orientation.  The kernel computes out^T = V^T . P~^T with V^T as the MFMA A
// operand and the numerator fragment P~ as the B operand, so lane l owns query
// (l & 15) both in its P~ fragment and in its accumulator columns: the rescale
// and the final 1/l are lane-local.  The row sum is one more MFMA per chunk
// with A = all ones, which sums exactly the bf16-rounded numerators the
// product used and keeps the VALU -- the second bottleneck after HBM -- free of
// the additions.
//
// Data movement.  One workgroup owns 256 queries of one head (8 waves x 32).
// Per step it copies the S tile (256 rows x 128 bytes, 8 rows of full cache
// lines per wave instruction) and the V tile (64 keys x d, contiguous in
// memory, one KiB per instruction) into a three-deep LDS ring with
// global->LDS copies issued two steps ahead, so about 64 KiB of S per CU is in
// flight while the current step computes.  S pieces are XOR-swizzled (rows of
// one fragment read hit distinct banks).  V stays in its row-major [key][d]
// layout, pieces swizzled by 2*(key & 3), and the V^T operand -- eight
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
__device__ __forceinline__ int s_swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }  // 128-byte S rows
__device__ __forceinline__ int v_swz(int r) { return 2 * (r & 3); }              // V rows
typedef short v4s_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint2 lds_tr16(const char* p) {
    v4s_t r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((DN_LDS v4s_t*)(DN_LDS char*)p);
    return __builtin_bit_cast(uint2, r);
}
}  // namespace sm

template <int D>
__global__ __launch_bounds__(512) void softmax_pv_kernel(const __bf16* __restrict__ S,
                                                         const __bf16* __restrict__ V, int BH,
                                                         int64_t Lq, int64_t Lk, int causal, int nqb,
                                                         __bf16* __restrict__ out) {
    using namespace sm;
    constexpr int NW = 8, QW = 2;          // waves, 16-query fragments per wave
    constexpr int BQ = NW * QW * 16;       // 256 queries per workgroup
    constexpr int BKV = 64;                // keys per step
    constexpr int NS = 3;                  // LDS ring depth
    constexpr int S_BYTES = BQ * BKV * 2;  // 32 KiB
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
        v_piece[j] = (lane % VPR) ^ v_swz(r);
    }
    const uint32_t smem_addr = lds_addr32(smem);
    auto issue = [&](int step) {
        const uint32_t base = smem_addr + (uint32_t)((step % NS) * STAGE);
        const int64_t k0 = (int64_t)step * BKV;
#pragma unroll
        for (int j = 0; j < S_INS; ++j) {
            const int64_t key = min(k0 + s_piece[j] * 8, Lk - 8);
            g2lds16_async(s_row[j] + key, base + (uint32_t)((wave + j * NW) * kChunkBytes));
        }
#pragma unroll
        for (int j = 0; j < V_INS; ++j) {
            const int64_t key = min(k0 + v_row[j], Lk - 1);
            g2lds16_async(Vh + key * D + v_piece[j] * 8, base + (uint32_t)(S_BYTES + (wave + j * NW) * kChunkBytes));
        }
    };

    f32x4 acc[QW][DB], accl[QW];
    float mrun[QW];
#pragma unroll
    for (int f = 0; f < QW; ++f) {
#pragma unroll
        for (int b = 0; b < DB; ++b) acc[f][b] = f32x4{0.f, 0.f, 0.f, 0.f};
        accl[f] = f32x4{0.f, 0.f, 0.f, 0.f};
        mrun[f] = -__builtin_inff();
    }
    const u32x4 ones = {0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u};

    issue(0);
    if (nsteps > 1) issue(1);

    for (int step = 0; step < nsteps; ++step) {
        if (step + 1 < nsteps)
            wait_vmcnt<PER>();  // this wave's copies of this step have landed
        else
            wait_vmcnt<0>();
        wait_lgkm0();  // this wave's reads of the previous step are complete
        block_barrier();
        if (step + 2 < nsteps) issue(step + 2);  // into the buffer the previous step vacated

        const int64_t k0 = (int64_t)step * BKV;
        // this wave has work unless every key of the step lies above all of its queries
        if (causal && k0 > qw0 + QW * 16 - 1) continue;
        const char* sb = smem + (step % NS) * STAGE;
        const char* vb = sb + S_BYTES;

        u32x4 sraw[QW][2];
#pragma unroll
        for (int f = 0; f < QW; ++f)
#pragma unroll
            for (int kc = 0; kc < 2; ++kc) {
                const int r = wave * QW * 16 + f * 16 + (lane & 15);
                const int piece = kc * 4 + (lane >> 4);
                sraw[f][kc] = lds_ld16(lds_ptr((char*)sb + r * 128 + ((piece ^ s_swz(r)) << 4)));
            }
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
                const int64_t lim = causal ? min(qrow[f], kv_end - 1) : kv_end - 1;
#pragma unroll
                for (int kc = 0; kc < 2; ++kc)
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (k0 + kc * 32 + (lane >> 4) * 8 + e > lim) sv[kc][e] = -__builtin_inff();
            }
            float tmax = -__builtin_inff();
#pragma unroll
            for (int kc = 0; kc < 2; ++kc)
#pragma unroll
                for (int e = 0; e < 8; e += 2) tmax = __builtin_fmaxf(tmax, __builtin_fmaxf(sv[kc][e], sv[kc][e + 1]));
            tmax = max_lane_groups(tmax);
            const float mnew = __builtin_fmaxf(mrun[f], tmax);
            const float alpha = mnew == mrun[f] ? 1.0f : __builtin_amdgcn_exp2f((mrun[f] - mnew) * kLog2e);
            if (__any(alpha != 1.0f)) {
#pragma unroll
                for (int b = 0; b < DB; ++b) acc[f][b] *= alpha;
                accl[f] *= alpha;
            }
            mrun[f] = mnew;
            const float nb = mnew == -__builtin_inff() ? 0.f : -mnew * kLog2e;
#pragma unroll
            for (int kc = 0; kc < 2; ++kc)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[kc][2 * e], kLog2e, nb));
                    const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[kc][2 * e + 1], kLog2e, nb));
                    pf[f][kc][e] = pack_bf16(p0, p1);
                }
        }
        // V^T fragments (A operand) per key chunk: two transposing reads of 4 keys per d block
        const int G = lane >> 4, i = lane & 15;
#pragma unroll
        for (int kc = 0; kc < 2; ++kc) {
#pragma unroll
            for (int b = 0; b < DB; ++b) {
                uint2 half[2];
#pragma unroll
                for (int hh = 0; hh < 2; ++hh) {
                    const int r = kc * 32 + 8 * G + 4 * hh + (i >> 2);
                    const int piece = 2 * b + ((i & 3) >> 1);
                    half[hh] = lds_tr16(vb + r * VROW + ((piece ^ v_swz(r)) << 4) + (i & 1) * 8);
                }
                const u32x4 vf = {half[0].x, half[0].y, half[1].x, half[1].y};
#pragma unroll
                for (int f = 0; f < QW; ++f) acc[f][b] = mfma_chunk<__bf16>(vf, pf[f][kc], acc[f][b]);
            }
#pragma unroll
            for (int f = 0; f < QW; ++f) accl[f] = mfma_chunk<__bf16>(ones, pf[f][kc], accl[f]);
        }
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

template <int D>
static hipError_t run_softmax_pv(const void* S, const void* V, int64_t BH, int64_t Lq, int64_t Lk, int causal,
                                 void* out, hipStream_t s) {
    constexpr int BQ = 256;
    const int nqb = (int)((Lq + BQ - 1) / BQ);
    dim3 grid((unsigned)(BH * nqb));
    softmax_pv_kernel<D><<<grid, 512, 0, s>>>((const __bf16*)S, (const __bf16*)V, (int)BH, Lq, Lk, causal, nqb,
                                             (__bf16*)out);
    return hipGetLastError();
}

hipError_t launch_softmax_pv_deferred(const void* S, const void* V, int64_t BH, int64_t Lq, int64_t Lk, int64_t d,
                                      int causal, void* out, hipStream_t s) {
    if (d == 64) return run_softmax_pv<64>(S, V, BH, Lq, Lk, causal, out, s);
    return run_softmax_pv<128>(S, V, BH, Lq, Lk, causal, out, s);
}

}  // namespace dn
