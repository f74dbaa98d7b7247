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
// Data movement.  One workgroup owns NW x QW x 16 queries of one head (NW
// waves, QW 16-query fragments each) and walks the keys in steps of 64.
// Scores are private to a wave, so each wave streams its own rows into a
// ring of PF LDS slots that only it reads: global->LDS copies of whole
// 128-byte lines (8 rows per instruction), 16-byte pieces XOR-swizzled so that
// the fragment reads are bank-conflict free, and no barrier; S is read once, so
// its copies carry the non-temporal hint and leave L2 to V.  V is shared by
// all waves and goes through an NS-slot ring with one barrier per step; it
// stays in its row-major [key][d] layout, pieces XOR-swizzled per key row, and
// the V^T operand -- eight consecutive keys of one d per lane -- is read with
// two transposing LDS reads (ds_read_b64_tr_b16: within a 16-lane group, lane
// j, slot t receives element j & 3 of the 8 bytes read by lane 4t + (j >> 2)).
// Every copy is issued from inline assembly and waited on with hand-counted
// vmcnt values.
//
// Schedule.  Iteration s issues the products of step s (numerators computed in
// iteration s-1) and computes the numerators of step s+1: independent work,
// which the compiler interleaves, so the exponentials of one step run beside
// the matrix instructions of the previous one (only the rare rise of a
// reference maximum branches off).
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
// vmcnt wait that also orders the compiler's memory operations: every memory
// operation of the main loop is issued from inline assembly, so every wait on
// them is written by hand.
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
// v_max3_f32 directly: fmaxf on values assembled from bit operations gets an
// extra canonicalizing max per operand from the compiler.  Its operands are
// bf16 widenings (shifts and masks), never transcendental results.
__device__ __forceinline__ float max3f(float a, float b, float c) {
    float d;
    asm("v_max3_f32 %0, %1, %2, %3" : "=v"(d) : "v"(a), "v"(b), "v"(c));
    return d;
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

// KSP > 1 (non-causal only): the workgroup's NW waves are KSP groups of NW / KSP query
// waves; group g walks the g-th of KSP equal runs of key steps, and the groups' partial
// sums are merged in LDS at the end (Eq. (8) over key ranges, each with its own reference
// maximum) -- for grids too small to fill the chip, where the steps one wave walks in
// sequence set the time.
template <int D, int NW, int QW, int NS, int PF, int KSP = 1>
__global__ __launch_bounds__(NW * 64) void softmax_pv_kernel(const __bf16* __restrict__ S,
                                                         const __bf16* __restrict__ V, int BH,
                                                         int64_t Lq, int64_t Lk, int causal, int nqb,
                                                         __bf16* __restrict__ out) {
    using namespace sm;
    constexpr int NQW = NW / KSP;          // waves per key group (one per 16 x QW queries)
    constexpr int BQ = NQW * QW * 16;      // queries per workgroup (QW 16-query fragments per wave)
    constexpr int BKV = 64;                // keys per step
    constexpr int VROW = D * 2;            // bytes per V row
    constexpr int V_BYTES = BKV * VROW;    // one V ring slot
    constexpr int V_INS = V_BYTES / kChunkBytes / NQW;  // V copies per wave per step
    constexpr int WROWS = QW * 16;         // score rows per wave
    constexpr int S_SLOT = WROWS * BKV * 2;  // one step of a wave's scores
    constexpr int S_LD = WROWS / 8;        // S copies per wave per step (8 rows x 128 B each)
    constexpr int VPR = VROW / 16;         // 16-byte pieces per V row
    constexpr int VRPI = kChunkBytes / VROW;  // V rows per copy instruction
    constexpr int DB = D / 16;
    static_assert(V_BYTES % (kChunkBytes * NQW) == 0, "V tile split evenly over the waves");
    static_assert(KSP >= 1 && NW % KSP == 0, "key groups of equal size");
    static_assert(NS >= 2 && NS <= 4 && PF >= 2 && PF >= NS - 2 && PF <= NS, "ring depths the counts assume");
    // Memory-op order per iteration j: [top] V copies of step j+NS-1, [middle] S copies of step
    // j+1+PF.  At the top of iteration s the wave needs S(s+1) and V(s); the ops issued after each:
    constexpr int AFTER_S = (PF - 1) * (V_INS + S_LD);
    constexpr int AFTER_V = S_LD + (NS - 2) * (V_INS + S_LD);
    constexpr int WAIT_N = AFTER_S < AFTER_V ? AFTER_S : AFTER_V;
    constexpr int AHEAD = PF + 1 > NS - 1 ? PF + 1 : NS - 1;  // prologue length

    __shared__ __attribute__((aligned(1024))) char smem[KSP * NS * V_BYTES + NW * PF * S_SLOT];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    // logical id: XCD-contiguous; each XCD walks whole heads, longest query blocks first
    const int t = xcd_contiguous(blockIdx.x, gridDim.x);
    const int h = t / nqb;
    const int qb = causal ? (nqb - 1 - t % nqb) : (t % nqb);
    const int64_t q0 = (int64_t)qb * BQ;
    const int64_t kv_end = causal ? min(Lk, q0 + BQ) : Lk;
    // key group: waves kg * NQW .. kg * NQW + NQW - 1 walk global steps gs0 .. gs0 + nsteps - 1;
    // keys from kv_end_g on are masked for the group (the last group: kv_end)
    const int qg = KSP == 1 ? wave : wave % NQW, kg = KSP == 1 ? 0 : wave / NQW;
    const int nsteps = (int)((((kv_end + BKV - 1) / BKV) + KSP - 1) / KSP);
    const int gs0 = kg * nsteps;
    const int64_t kv_end_g = min(kv_end, (int64_t)(gs0 + nsteps) * BKV);

    const __bf16* Sh = S + (int64_t)h * Lq * Lk;
    const __bf16* Vh = V + (int64_t)h * Lk * D;
    __bf16* Oh = out + (int64_t)h * Lq * D;

    const int64_t qw0 = q0 + qg * WROWS;  // first query of this wave
    const int G = lane >> 4, i = lane & 15;
    int64_t qrow[QW];
#pragma unroll
    for (int f = 0; f < QW; ++f) qrow[f] = qw0 + f * 16 + i;
    const uint32_t smem_addr = lds_addr32(smem);

    // ---- S: each score row belongs to one wave, so it goes through a ring
    // private to that wave (PF steps deep) and needs no barrier.  Copies move
    // whole 128-byte lines (8 rows per instruction); lane l fetches piece
    // (l & 7) ^ s_swz(row) of row 8j + (l >> 3), so piece c of a row sits in
    // 16-byte slot c ^ s_swz(row), which makes the fragment reads below
    // bank-conflict free.  Offsets from the head's base fit 32 bits
    // (Lq * Lk <= 2^31).  Keys past the last one this wave needs (causal
    // diagonal, Lk, or steps past the end) are clamped onto its last 8-key
    // group, lines it has just read: every step issues the same copies (the
    // wait counts rely on it) and skipped work costs no memory traffic.
    const int64_t kend_w = causal ? min(kv_end, qw0 + WROWS) : kv_end;  // exclusive, multiple of 8
    const uint64_t s_base = uniform_u64(Sh);
    uint32_t s_row[S_LD], s_p8[S_LD], s_off[S_LD];
#pragma unroll
    for (int j = 0; j < S_LD; ++j) {
        const int r = 8 * j + (lane >> 3);
        const int64_t q = qw0 + r < Lq ? qw0 + r : Lq - 1;
        s_row[j] = (uint32_t)(q * Lk * 2);
        s_p8[j] = (uint32_t)(((lane & 7) ^ s_swz(r)) * 8);
        s_off[j] = s_row[j] + 2 * s_p8[j];
    }
    const uint32_t s_lds = smem_addr + (uint32_t)(KSP * NS * V_BYTES + wave * PF * S_SLOT);
    const uint32_t klast = (uint32_t)(kend_w - 8);  // the wave's last 8-key group
    // FAST: no key of the step is clamped (the caller's loop guarantees it), so the step's
    // offset goes into the scalar base and the lanes' offsets stay fixed
    auto issue_s = [&](int step, auto fast) {
        const uint32_t dst = s_lds + (uint32_t)((step % PF) * S_SLOT);
        const uint32_t k0 = (uint32_t)(gs0 + step) * BKV;
        if constexpr (decltype(fast)::value) {
#pragma unroll
            for (int j = 0; j < S_LD; ++j) g2lds16_stream_sb(s_base + 2u * k0, s_off[j], dst + j * kChunkBytes);
        } else {
#pragma unroll
            for (int j = 0; j < S_LD; ++j) {
                const uint32_t key = k0 + s_p8[j] < klast ? k0 + s_p8[j] : klast;  // a select, no branch
                g2lds16_stream_sb(s_base, s_row[j] + key * 2u, dst + j * kChunkBytes);
            }
        }
    };
    // fragment reads: lane (i, G) takes row 16f + i, piece 4kc + G (8 keys), the B-operand order
    int s_rd[2];
#pragma unroll
    for (int kc = 0; kc < 2; ++kc) s_rd[kc] = i * 128 + (((4 * kc + G) ^ s_swz(i)) << 4);
    const char* s_ring = smem + KSP * NS * V_BYTES + wave * PF * S_SLOT;
    auto read_s = [&](int slot, u32x4(&r)[QW][2]) {
        const char* b = s_ring + slot * S_SLOT;
#pragma unroll
        for (int f = 0; f < QW; ++f)
#pragma unroll
            for (int kc = 0; kc < 2; ++kc) r[f][kc] = lds_ld16(lds_ptr((char*)b + f * 16 * 128 + s_rd[kc]));
    };

    // ---- V: shared by every wave, so it goes through an NS-deep ring with a
    // barrier per step (copy instruction j covers key rows VRPI*(wave + j*NW) ..).
    // Byte offsets from the head's base: 32 bits (Lk * d * 2 < 2^32).
    uint32_t v_row[V_INS], v_p16[V_INS];
#pragma unroll
    for (int j = 0; j < V_INS; ++j) {
        const int r = (qg + j * NQW) * VRPI + lane / VPR;
        v_row[j] = (uint32_t)r;
        v_p16[j] = (uint32_t)(((lane % VPR) ^ v_swz<D>(r)) * 16);
    }
    const uint64_t v_base = uniform_u64(Vh);
    const uint32_t vlast = (uint32_t)(Lk - 1);
    uint32_t vc_off[V_INS];
#pragma unroll
    for (int j = 0; j < V_INS; ++j) vc_off[j] = v_row[j] * (uint32_t)VROW + v_p16[j];
    auto issue_v = [&](int step, auto fast) {  // FAST: every row of the step exists
        const uint32_t base = smem_addr + (uint32_t)((kg * NS + step % NS) * V_BYTES);
        const uint32_t k0 = (uint32_t)(gs0 + step) * BKV;
        if constexpr (decltype(fast)::value) {
#pragma unroll
            for (int j = 0; j < V_INS; ++j)
                g2lds16_async_sb(v_base + (uint64_t)k0 * VROW, vc_off[j], base + (uint32_t)((qg + j * NQW) * kChunkBytes));
        } else {
#pragma unroll
            for (int j = 0; j < V_INS; ++j) {
                const uint32_t key = k0 + v_row[j] < vlast ? k0 + v_row[j] : vlast;  // rows past Lk clamp onto the last
                g2lds16_async_sb(v_base, key * (uint32_t)VROW + v_p16[j],
                                 base + (uint32_t)((qg + j * NQW) * kChunkBytes));
            }
        }
    };

    f32x4 acc[QW][DB], accl[QW];
#pragma unroll
    for (int f = 0; f < QW; ++f) {
#pragma unroll
        for (int b = 0; b < DB; ++b) acc[f][b] = f32x4{0.f, 0.f, 0.f, 0.f};
        accl[f] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    u32x4 ones = {0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u};
    // opaque to the compiler, which would otherwise rebuild the constant in every iteration
    asm volatile("" : "+v"(ones));

    // Lane-constant LDS offsets of the V^T fragments.  The V swizzle depends
    // only on bits of (8G + (i >> 2)), which the chunk (kc) and half offsets
    // leave unchanged; the per-step parts are uniform.
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

    // Numerators of one step: bf16 exp2(s log2e - mref) in the B-operand order,
    // with the reference raised where the step's maximum requires it; alpha is
    // the factor the partial sums must take to follow (1 where unchanged).
    // Masked keys arrive as -inf scores (mask_scores) and yield zeros.
    auto numerators = [&](const u32x4(&sc)[QW][2], u32x4(&pfo)[QW][2], float(&alpha)[QW]) {
        bool raised = false;
        float sv[QW][2][8], tmax[QW];
        bool want = false;  // some lane's own scores would raise its query's reference
#pragma unroll
        for (int f = 0; f < QW; ++f) {
#pragma unroll
            for (int kc = 0; kc < 2; ++kc) {
                const uint32_t w[4] = {sc[f][kc].x, sc[f][kc].y, sc[f][kc].z, sc[f][kc].w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    sv[f][kc][2 * e] = bf_lo(w[e]);
                    sv[f][kc][2 * e + 1] = bf_hi(w[e]);
                }
            }
            const float m0 = max3f(sv[f][0][0], sv[f][0][1], sv[f][0][2]), m1 = max3f(sv[f][0][3], sv[f][0][4], sv[f][0][5]);
            const float m2 = max3f(sv[f][0][6], sv[f][0][7], sv[f][1][0]), m3 = max3f(sv[f][1][1], sv[f][1][2], sv[f][1][3]);
            const float m4 = max3f(sv[f][1][4], sv[f][1][5], sv[f][1][6]);
            tmax[f] = max3f(max3f(m0, m1, m2), max3f(m3, m4, sv[f][1][7]), m0);
            want |= tmax[f] * kLog2e > mref[f] + 8.0f;
        }
        // The reference rises when the query's maximum over its 4 lanes exceeds it by more
        // than 8; that holds exactly when one of the lanes' own maxima does (scaling by
        // log2e keeps the order), so the cross-lane maximum is formed only in the rare
        // steps where some lane of the wave asks for it.
        if (__any(want)) {
#pragma unroll
            for (int f = 0; f < QW; ++f) {
                const float tmax2 = max_lane_groups(tmax[f]) * kLog2e;
                const bool raise = tmax2 > mref[f] + 8.0f;
                const float mnew = raise ? tmax2 : mref[f];
                alpha[f] = __builtin_amdgcn_exp2f(raise ? mref[f] - mnew : 0.f);
                mref[f] = mnew;
                raised |= raise;
            }
        } else {
#pragma unroll
            for (int f = 0; f < QW; ++f) alpha[f] = 1.f;
        }
#pragma unroll
        for (int f = 0; f < QW; ++f) {
            const float nb = mref[f] == -__builtin_inff() ? 0.f : -mref[f];
#pragma unroll
            for (int kc = 0; kc < 2; ++kc)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[f][kc][2 * e], kLog2e, nb));
                    const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[f][kc][2 * e + 1], kLog2e, nb));
                    pfo[f][kc][e] = pack_bf16(p0, p1);
                }
        }
        return raised;
    };
    // Keys beyond the row (causal) or beyond Lk are not part of it: their raw
    // bf16 scores are replaced by -inf (0xff80), two per word.  A step wholly
    // above a wave's queries, or past the last step, is masked entirely.
    auto mask_scores = [&](int step, u32x4(&sc)[QW][2]) {
        const int64_t k0 = (int64_t)(gs0 + step) * BKV;
#pragma unroll
        for (int f = 0; f < QW; ++f) {
            const int64_t last = causal ? (qrow[f] < kv_end - 1 ? qrow[f] : kv_end - 1) : kv_end_g - 1;
            const int64_t rel = last - k0;  // last kept key, relative to the step
            const int lim = rel < 0 ? -1 : (rel > BKV ? BKV : (int)rel);
#pragma unroll
            for (int kc = 0; kc < 2; ++kc)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int k = kc * 32 + G * 8 + 2 * e;  // key of the low half
                    const uint32_t m = (k > lim ? 0x0000ffffu : 0u) | (k + 1 > lim ? 0xffff0000u : 0u);
                    sc[f][kc][e] = (sc[f][kc][e] & ~m) | (0xff80ff80u & m);
                }
        }
    };
    const int qw0i = (int)qw0, kv_endi = (int)kv_end_g;  // positions fit 32 bits (Lq * Lk <= 2^31)
    auto is_edge = [&](int step) {
        const int k0 = (gs0 + step) * BKV;
        return (causal && k0 + BKV - 1 > qw0i) || k0 + BKV > kv_endi;
    };

    // Prologue: the copies of iterations -AHEAD .. -1 in the steady-state
    // order (iteration j issues, at its top, the V copies of step j+NS-1 and,
    // after its numerators, the S copies of step j+1+PF), with the numerators
    // of step 0 computed in iteration -1.
#pragma unroll
    for (int j = -AHEAD; j < -1; ++j) {
        if (j + NS - 1 >= 0) issue_v(j + NS - 1, std::false_type{});
        if (j + 1 + PF >= 0) issue_s(j + 1 + PF, std::false_type{});
    }
    issue_v(NS - 2, std::false_type{});
    wait_vmcnt_asm<(PF - 1) * S_LD>();  // S(0) is complete once only the later S copies may remain
    u32x4 pf[QW][2];
    float alpha[QW];
    bool raised;
    {
        u32x4 sc[QW][2];
        read_s(0, sc);
        if (is_edge(0)) mask_scores(0, sc);
        numerators(sc, pf, alpha);
    }
    raised = false;  // the partial sums are still zero: nothing to rescale
    issue_s(PF, std::false_type{});  // into the slot step 0 vacated

    // Iteration s: the products of step s (V(s) from the ring, numerators
    // computed one iteration earlier) and, independent of them, the numerators
    // of step s+1 -- one basic block, so the scheduler interleaves the matrix
    // instructions with the exponentials.  When step s's numerators raised the
    // reference, the partial sums follow it first (a rare branch ahead of the
    // block).
    // two numerator buffers used in turn: the loop is unrolled by two so that
    // neither is ever copied
    u32x4 pf2[QW][2];
    // FAST: the copies this iteration issues need no clamping and step s+1 is not an edge
    // step (both follow from the bound of the loop that passes it, see below).  PAR = s % 2:
    // the loops run iterations in pairs from step 0, so with two-slot rings the slots each
    // iteration reads are known at compile time and their offsets go into the LDS reads'
    // immediate fields.
    auto iteration = [&](int s, u32x4(&pcur)[QW][2], u32x4(&pnext)[QW][2], auto fast, auto par) {
        constexpr bool FAST = decltype(fast)::value;
        constexpr int PAR = decltype(par)::value;
        const int vslot = NS == 2 ? PAR : s % NS;               // V(s)
        const int sslot = PF == 2 ? PAR ^ 1 : (s + 1) % PF;     // S(s+1)
        wait_vmcnt_asm<WAIT_N>();  // S(s+1) and this wave's V copies of step s are complete
        wait_lgkm0();              // this wave's LDS reads of step s-1 are complete
        block_barrier();
        issue_v(s + NS - 1, fast);  // into the slot step s-1 vacated
        if (__any(raised)) {
#pragma unroll
            for (int f = 0; f < QW; ++f) {
#pragma unroll
                for (int b = 0; b < DB; ++b) acc[f][b] *= alpha[f];
                accl[f] *= alpha[f];
            }
        }
        u32x4 sc[QW][2];
        read_s(sslot, sc);
        if (!FAST && is_edge(s + 1)) mask_scores(s + 1, sc);
        const char* vb = smem + (kg * NS + vslot) * V_BYTES;  // this key group's V ring
        // V^T fragments of key chunk kc (A operand): two transposing reads of 4 keys per d block
        auto read_v = [&](int kc, u32x4(&vf)[DB]) {
#pragma unroll
            for (int b = 0; b < DB; ++b) {
                const uint2 lo = lds_tr16(vb + v_off[b] + (kc * 32) * VROW);
                const uint2 hi = lds_tr16(vb + v_off[b] + (kc * 32 + 4) * VROW);
                vf[b] = u32x4{lo.x, lo.y, hi.x, hi.y};
            }
        };
        auto products = [&](int kc, const u32x4(&vf)[DB]) {
#pragma unroll
            for (int b = 0; b < DB; ++b)
#pragma unroll
                for (int f = 0; f < QW; ++f) acc[f][b] = mfma_chunk<__bf16>(vf[b], pcur[f][kc], acc[f][b]);
#pragma unroll
            for (int f = 0; f < QW; ++f) accl[f] = mfma_chunk<__bf16>(ones, pcur[f][kc], accl[f]);
        };
        {
            u32x4 vf[DB];
            read_v(0, vf);
            raised = numerators(sc, pnext, alpha);
            issue_s(s + 1 + PF, fast);  // the slot of S(s+1) has been read
            products(0, vf);
        }
        {
            u32x4 vf[DB];
            read_v(1, vf);
            products(1, vf);
        }
        // The next step's numerators are consumed in the next iteration, which the loop's
        // exit test may skip; without these uses the compiler sinks their exponentials past
        // that test, out of this block and away from the products they should run beside.
#pragma unroll
        for (int f = 0; f < QW; ++f) {
#pragma unroll
            for (int kc = 0; kc < 2; ++kc) asm volatile("" ::"v"(pnext[f][kc]));
            asm volatile("" ::"v"(alpha[f]));
        }
    };
    // Iterations s < fast_end (local steps; global step = gs0 + local) issue only unclamped
    // copies and mask nothing: the S copy of step s+1+PF lies wholly before the wave's last
    // 8-key group, (s+1+PF+1)·64 - 8 <= klast, the V copy of step s+NS-1 wholly inside the
    // keys, (s+NS)·64 - 1 <= vlast, and step s+1 is no edge step: (s+1)·64 + 63 <= the wave's
    // first query (causal) and (s+2)·64 <= kv_end_g.
    const int64_t a_s = (int64_t)klast + 8 - BKV, a_v = (int64_t)vlast + 1 - BKV;
    const int64_t a_e = min(causal ? (int64_t)qw0i - (BKV - 1) : (int64_t)kv_endi, (int64_t)kv_endi - BKV);
    int fast_end = nsteps;
    fast_end = a_s < 0 ? 0 : min(fast_end, (int)(a_s / BKV) - PF - gs0);
    fast_end = a_v < 0 ? 0 : min(fast_end, (int)(a_v / BKV) - NS + 2 - gs0);
    fast_end = a_e < 0 ? 0 : min(fast_end, (int)(a_e / BKV) - gs0);
    fast_end = __builtin_amdgcn_readfirstlane(max(fast_end, 0));
    int s = 0;
    using even = std::integral_constant<int, 0>;
    using odd = std::integral_constant<int, 1>;
    for (; s + 1 < fast_end; s += 2) {  // both iterations of the pair run: no exit test between them
        iteration(s, pf, pf2, std::true_type{}, even{});
        iteration(s + 1, pf2, pf, std::true_type{}, odd{});
    }
    for (; s < nsteps; s += 2) {
        iteration(s, pf, pf2, std::false_type{}, even{});
        if (s + 1 < nsteps) iteration(s + 1, pf2, pf, std::false_type{}, odd{});
    }
    wait_vmcnt_asm<0>();  // no copy into LDS may outlive the workgroup

    if constexpr (KSP > 1) {
        // Merge of the key groups (KSP = 2): group 1 leaves its partial products, its row sum
        // and its reference maximum in LDS (the rings are idle now), group 0 rescales both to
        // the larger reference, out = (acc0 2^(m0-m) + acc1 2^(m1-m)) / (l0 2^(m0-m) + l1 2^(m1-m)).
        // A group without any unmasked key has m = -inf and contributes nothing.
        static_assert(KSP == 2, "two key groups");
        constexpr int NF = QW * (DB * 4 + 2);  // floats per lane
        float* xch = reinterpret_cast<float*>(smem) + (qg * kWave + lane) * NF;
        wait_lgkm0();
        block_barrier();  // every wave is done with the rings
        if (kg == 1) {
#pragma unroll
            for (int f = 0; f < QW; ++f) {
#pragma unroll
                for (int b = 0; b < DB; ++b)
#pragma unroll
                    for (int e = 0; e < 4; ++e) xch[f * (DB * 4 + 2) + b * 4 + e] = acc[f][b][e];
                xch[f * (DB * 4 + 2) + DB * 4] = accl[f][0];
                xch[f * (DB * 4 + 2) + DB * 4 + 1] = mref[f];
            }
        }
        __syncthreads();
        if (kg == 1) return;
#pragma unroll
        for (int f = 0; f < QW; ++f) {
            const float m1 = xch[f * (DB * 4 + 2) + DB * 4 + 1], l1 = xch[f * (DB * 4 + 2) + DB * 4];
            const float m = mref[f] > m1 ? mref[f] : m1;
            const float a0 = mref[f] == -__builtin_inff() ? 0.f : __builtin_amdgcn_exp2f(mref[f] - m);
            const float a1 = m1 == -__builtin_inff() ? 0.f : __builtin_amdgcn_exp2f(m1 - m);
#pragma unroll
            for (int b = 0; b < DB; ++b)
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    acc[f][b][e] = __builtin_fmaf(acc[f][b][e], a0, xch[f * (DB * 4 + 2) + b * 4 + e] * a1);
            accl[f][0] = __builtin_fmaf(accl[f][0], a0, l1 * a1);
        }
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

template <int D, int NW, int QW, int NS, int PF, int KSP = 1>
static hipError_t run_softmax_pv(const void* S, const void* V, int64_t BH, int64_t Lq, int64_t Lk, int causal,
                                 void* out, hipStream_t s) {
    constexpr int BQ = NW / KSP * QW * 16;
    const int nqb = (int)((Lq + BQ - 1) / BQ);
    dim3 grid((unsigned)(BH * nqb));
    softmax_pv_kernel<D, NW, QW, NS, PF, KSP><<<grid, NW * 64, 0, s>>>((const __bf16*)S, (const __bf16*)V, (int)BH,
                                                                       Lq, Lk, causal, nqb, (__bf16*)out);
    return hipGetLastError();
}

// 8 waves x 2 fragments (256 queries per workgroup), two V slots and two S
// slots per wave: 80 KiB (d = 64) or 96 KiB (d = 128) of LDS.  Deeper rings
// measured no faster on the causal 32 x 8192 x 8192, d = 128 workload.
constexpr int kSmWaves = 8, kSmFrags = 2, kSmStages = 2, kSmPrefetch = 2;
// Where 256-query blocks would give fewer workgroups than the chip has CUs
// (12 heads x 512 queries: 24), the work is latency-bound: 2 waves x 1
// fragment (32 queries per workgroup) spread it over 8x more workgroups, with
// rings 4 (d = 64, 48 KiB) or 3 (d = 128, 60 KiB) steps deep.
constexpr int64_t kSmCUs = 256;

hipError_t launch_softmax_pv_deferred(const void* S, const void* V, int64_t BH, int64_t Lq, int64_t Lk, int64_t d,
                                      int causal, void* out, hipStream_t s) {
    const bool small = BH * ((Lq + 255) / 256) < kSmCUs;
    // small and non-causal with more than one key step: two key groups per workgroup, each
    // walking half the steps with 2-deep rings, merged in LDS (12 x 512 x 512, d64, graph
    // replays: 6.8 us unsplit, 5.4 us split; 3- and 4-deep rings 5.7-6.0 us, one query wave
    // per group 6.3-6.5 us)
    const bool split = small && !causal && Lk > 64;
    if (d == 64) {
        if (split) return run_softmax_pv<64, 4, 1, 2, 2, 2>(S, V, BH, Lq, Lk, causal, out, s);
        if (small) return run_softmax_pv<64, 2, 1, 4, 4>(S, V, BH, Lq, Lk, causal, out, s);
        return run_softmax_pv<64, kSmWaves, kSmFrags, kSmStages, kSmPrefetch>(S, V, BH, Lq, Lk, causal, out, s);
    }
    if (split) return run_softmax_pv<128, 4, 1, 2, 2, 2>(S, V, BH, Lq, Lk, causal, out, s);
    if (small) return run_softmax_pv<128, 2, 1, 3, 3>(S, V, BH, Lq, Lk, causal, out, s);
    return run_softmax_pv<128, kSmWaves, kSmFrags, kSmStages, kSmPrefetch>(S, V, BH, Lq, Lk, causal, out, s);
}

}  // namespace dn
