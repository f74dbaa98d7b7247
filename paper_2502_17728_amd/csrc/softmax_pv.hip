// softmax_pv.hip -- deferred Softmax -> P.V (Sec. II-B, Eq. (8)).
//
// out_i = (1 / l_i) * sum_j exp(s_ij - m_i) V_j,   l_i = sum_j exp(s_ij - m_i),
// with m_i the row maximum (footnote of Eq. (7)).  The matrix core consumes the
// un-normalized numerators; the collective part (max and sum over the row) is
// reduced alongside, and the single division happens in the epilogue.
//
// Keys are streamed in steps of 128.  Because S is materialized, the maximum
// is kept online: when a step raises a row's running max from m to m', the
// partial products and the partial sum are scaled by exp(m - m') -- Eq. (8)
// applied to the row prefix, which leaves the result unchanged in exact
// arithmetic.
//
// Orientation.  The kernel computes out^T = V^T . P~^T with V^T as the MFMA A
// operand (from LDS) and the numerator fragment P~ as the B operand (straight
// from HBM into registers).  Lane l then owns query (l & 15) both in its P~
// fragment and in its accumulator columns, so the rescale and the final 1/l
// are lane-local.  The row sum is one more MFMA per chunk with A = all ones,
// which sums exactly the bf16-rounded numerators the product used and keeps
// the VALU (the second bottleneck after HBM) free of the additions.
#include "dn_device.hpp"
#include "dn_launch.hpp"

namespace dn {

constexpr float kLog2e = 1.4426950408889634f;

template <int D, int QW>
__global__ __launch_bounds__(256) void softmax_pv_kernel(const __bf16* __restrict__ S,
                                                         const __bf16* __restrict__ V, int BH,
                                                         int64_t Lq, int64_t Lk, int causal, int nqb,
                                                         __bf16* __restrict__ out) {
    constexpr int NW = 4;
    constexpr int BQ = NW * QW * 16;   // queries per workgroup
    constexpr int BKV = 128;           // keys per step
    constexpr int KCH = BKV / 32;      // 32-key chunks per step
    constexpr int DB = D / 16;         // 16-row blocks of V^T
    constexpr int VST = DB * KCH * kChunkBytes;
    constexpr int VBLK = (BKV / 8) * (D / 8);  // 8x8 blocks of a V tile
    static_assert(VBLK <= NW * kWave, "one V block per thread at most");

    __shared__ __attribute__((aligned(1024))) char vs[2][VST];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
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

    // ---- V tile staging: 8 keys x 8 dims per thread, transposed into chunk order
    u32x4 vreg[8];
    const int vb = tid;
    const int vk8 = (vb / (D / 8)) * 8, vd8 = (vb % (D / 8)) * 8;
    auto v_load = [&](int step) {
        if (vb < VBLK) {
#pragma unroll
            for (int r = 0; r < 8; ++r) {
                const int64_t key = (int64_t)step * BKV + vk8 + r;
                vreg[r] = key < kv_end ? ld16(Vh + key * D + vd8) : u32x4{0, 0, 0, 0};
            }
        }
    };
    auto v_store = [&](int buf) {
        if (vb < VBLK) {
            u32x4 col[8];
            transpose8x8_bf16(vreg, col);
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                const int d = vd8 + c;
                const int chunk = (d >> 4) * KCH + vk8 / 32;
                const int l2 = (d & 15) + 16 * ((vk8 % 32) / 8);
                *reinterpret_cast<DN_LDS u32x4*>(lds_ptr(&vs[buf][chunk * kChunkBytes + l2 * 16])) = col[c];
            }
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

    v_load(0);
    v_store(0);
    __syncthreads();

    for (int step = 0; step < nsteps; ++step) {
        const int buf = step & 1;
        const int64_t k0 = (int64_t)step * BKV;
        // this wave has work in the step unless every key lies above all of its queries
        const bool active = !causal || k0 <= qw0 + QW * 16 - 1;

        u32x4 sraw[QW][KCH];
        if (active) {
#pragma unroll
            for (int f = 0; f < QW; ++f) {
                const int64_t q = min(qrow[f], Lq - 1);
#pragma unroll
                for (int kc = 0; kc < KCH; ++kc) {
                    const int64_t key = k0 + kc * 32 + (lane >> 4) * 8;
                    const bool need = key < kv_end && (!causal || key <= qrow[f]);
                    sraw[f][kc] = need ? ld16(Sh + q * Lk + key) : u32x4{0, 0, 0, 0};
                }
            }
        }
        if (step + 1 < nsteps) v_load(step + 1);

        if (active) {
            const bool edge = (causal && k0 + BKV - 1 > qw0) || k0 + BKV > kv_end;
            u32x4 pf[QW][KCH];
#pragma unroll
            for (int f = 0; f < QW; ++f) {
                float sv[KCH][8];
#pragma unroll
                for (int kc = 0; kc < KCH; ++kc)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        sv[kc][2 * e] = bf_lo(sraw[f][kc][e]);
                        sv[kc][2 * e + 1] = bf_hi(sraw[f][kc][e]);
                    }
                if (edge) {  // keys beyond the row (causal) or beyond Lk are not part of it
                    const int64_t lim = causal ? min(qrow[f], kv_end - 1) : kv_end - 1;
#pragma unroll
                    for (int kc = 0; kc < KCH; ++kc)
#pragma unroll
                        for (int e = 0; e < 8; ++e)
                            if (k0 + kc * 32 + (lane >> 4) * 8 + e > lim) sv[kc][e] = -__builtin_inff();
                }
                float tmax = -__builtin_inff();
#pragma unroll
                for (int kc = 0; kc < KCH; ++kc)
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
                for (int kc = 0; kc < KCH; ++kc)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[kc][2 * e], kLog2e, nb));
                        const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[kc][2 * e + 1], kLog2e, nb));
                        pf[f][kc][e] = pack_bf16(p0, p1);
                    }
            }
#pragma unroll
            for (int kc = 0; kc < KCH; ++kc) {
#pragma unroll
                for (int b = 0; b < DB; ++b) {
                    const u32x4 a = lds_ld16(lds_ptr(&vs[buf][(b * KCH + kc) * kChunkBytes + lane * 16]));
#pragma unroll
                    for (int f = 0; f < QW; ++f) acc[f][b] = mfma_chunk<__bf16>(a, pf[f][kc], acc[f][b]);
                }
#pragma unroll
                for (int f = 0; f < QW; ++f) accl[f] = mfma_chunk<__bf16>(ones, pf[f][kc], accl[f]);
            }
        }
        if (step + 1 < nsteps) v_store(buf ^ 1);
        __syncthreads();
    }

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

template <int D, int QW>
static hipError_t run_softmax_pv(const void* S, const void* V, int64_t BH, int64_t Lq, int64_t Lk, int causal,
                                 void* out, hipStream_t s) {
    constexpr int BQ = 4 * QW * 16;
    const int nqb = (int)((Lq + BQ - 1) / BQ);
    dim3 grid((unsigned)(BH * nqb));
    softmax_pv_kernel<D, QW><<<grid, 256, 0, s>>>((const __bf16*)S, (const __bf16*)V, (int)BH, Lq, Lk, causal, nqb,
                                                  (__bf16*)out);
    return hipGetLastError();
}

hipError_t launch_softmax_pv_deferred(const void* S, const void* V, int64_t BH, int64_t Lq, int64_t Lk, int64_t d,
                                      int causal, void* out, hipStream_t s) {
    if (d == 64) return run_softmax_pv<64, 2>(S, V, BH, Lq, Lk, causal, out, s);
    return run_softmax_pv<128, 2>(S, V, BH, Lq, Lk, causal, out, s);
}

}  // namespace dn
