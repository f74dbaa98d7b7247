// dn_device.hpp -- device helpers shared by the gfx950 kernels of libdn.
//
// MFMA operand layout used throughout (v_mfma_f32_16x16x32_bf16 and, for fp32,
// four v_mfma_f32_16x16x4_f32): a "fragment chunk" is 16 rows x 64 bytes of
// the K dimension (32 bf16 or 16 fp32).  Lane l holds row (l & 15) and the 16
// contiguous bytes starting at K byte offset 16 * (l >> 4).  Both operands of
// a product use the same chunk layout, so every lane's k-slots agree.  The
// 16x16 fp32 result is held as: lane l, element i  ->  row 4*(l >> 4) + i,
// column (l & 15).  A chunk occupies 1 KiB of LDS with lane l at byte 16*l,
// which is exactly where a wave-wide global_load_lds_dwordx4 deposits lane l's
// 16 bytes, and makes every fragment read a conflict-free ds_read_b128.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dn {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

#define DN_LDS __attribute__((address_space(3)))

constexpr int kWave = 64;
constexpr int kChunkBytes = 1024;  // one 16-row x 64-byte fragment chunk

// ----------------------------------------------------------------- element traits
template <class T>
struct elem;
template <>
struct elem<__bf16> {
    static constexpr int per16 = 8;   // elements in 16 bytes
    static constexpr int kchunk = 32; // K elements in one fragment chunk
};
template <>
struct elem<float> {
    static constexpr int per16 = 4;
    static constexpr int kchunk = 16;
};

// ----------------------------------------------------------------- bf16 <-> fp32
__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Round two fp32 to bf16 (nearest even) and pack (lo = a).  One v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
    bf16x2_t v = {(__bf16)a, (__bf16)b};
    return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ __bf16 to_bf16(float a) { return (__bf16)a; }

template <class T>
__device__ __forceinline__ T from_f32(float v);
template <>
__device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <>
__device__ __forceinline__ __bf16 from_f32<__bf16>(float v) { return (__bf16)v; }

template <class T>
__device__ __forceinline__ float to_f32(T v);
template <>
__device__ __forceinline__ float to_f32<float>(float v) { return v; }
template <>
__device__ __forceinline__ float to_f32<__bf16>(__bf16 v) { return (float)v; }

// ----------------------------------------------------------------- MFMA on one chunk
// acc += A_chunk(16 x kchunk) . B_chunk(16 x kchunk)^T for one 16x16 output tile.
template <class T>
__device__ __forceinline__ f32x4 mfma_chunk(const u32x4& a, const u32x4& b, f32x4 acc);

template <>
__device__ __forceinline__ f32x4 mfma_chunk<__bf16>(const u32x4& a, const u32x4& b, f32x4 acc) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                   __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
}

template <>
__device__ __forceinline__ f32x4 mfma_chunk<float>(const u32x4& a, const u32x4& b, f32x4 acc) {
    // lane group g = l>>4 holds k = 4g..4g+3 of the chunk; slot j of the
    // 16x16x4 instruction takes element j, so the four calls cover all 16 k.
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
    return acc;
}

// ----------------------------------------------------------------- row sums of a chunk
// Adds the lane's 16 bytes of one row into (s1 = sum x, s2 = sum x^2), fp32.
template <class T>
__device__ __forceinline__ void chunk_moments(const u32x4& a, float& s1, float& s2);

template <>
__device__ __forceinline__ void chunk_moments<__bf16>(const u32x4& a, float& s1, float& s2) {
    // Widened to fp32 (exact) and accumulated with FMAs.  Measured faster inside
    // the MFMA loop than v_dot2c_f32_bf16, whose accumulate chains stall the
    // in-order issue of the wave's next matrix instruction.  The words are
    // copied out first: reading the vector element a[j] straight into a
    // bit_cast was compiled as a read of element 0 for every j.
    const uint32_t w[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const float lo = bf_lo(w[j]), hi = bf_hi(w[j]);
        s1 += lo + hi;
        s2 = __builtin_fmaf(lo, lo, __builtin_fmaf(hi, hi, s2));
    }
}

template <>
__device__ __forceinline__ void chunk_moments<float>(const u32x4& a, float& s1, float& s2) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        float v = __uint_as_float(a[j]);
        s1 += v;
        s2 = __builtin_fmaf(v, v, s2);
    }
}

// ----------------------------------------------------------------- memory helpers
// One wave-wide direct global->LDS copy: lane l's 16 bytes at `g` land at lds_base + 16*l.
__device__ __forceinline__ void g2lds16(const void* g, DN_LDS void* lds_base) {
    __builtin_amdgcn_global_load_lds(g, lds_base, 16, 0, 0);
}

// The same copy issued through inline asm.  The compiler then does not track
// it, so it cannot add its own conservative "s_waitcnt vmcnt(0)" before later
// LDS reads of other buffers; the caller owns every wait for these copies
// (explicit vmcnt counts).  m0 is written here and used by nothing else in the
// kernels that call this.  `lds_addr` must be wave-uniform.
__device__ __forceinline__ void g2lds16_async(const void* g, uint32_t lds_addr) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
                 :
                 : "s"(__builtin_amdgcn_readfirstlane(lds_addr)), "v"(g)
                 : "memory", "m0");
}

// Scalar-base form: the wave-uniform 64-bit base sits in SGPRs and each lane
// supplies only a 32-bit byte offset, which saves two VGPRs and a 64-bit add
// per copy stream.  `offset` must be below 2^32.
__device__ __forceinline__ uint64_t uniform_u64(const void* p) {
    const uint64_t v = (uint64_t)(uintptr_t)p;
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
    return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ void g2lds16_async_sb(uint64_t sbase, uint32_t offset, uint32_t lds_addr) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2"
                 :
                 : "s"(__builtin_amdgcn_readfirstlane(lds_addr)), "v"(offset), "s"(sbase)
                 : "memory", "m0");
}

// Streaming form, for bytes one launch reads exactly once (a score matrix, a decode
// key/value cache): the non-temporal hint keeps them from evicting lines that other
// workgroups re-read from L2.  Not for data shared between workgroups.
__device__ __forceinline__ void g2lds16_stream_sb(uint64_t sbase, uint32_t offset, uint32_t lds_addr) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2 nt"
                 :
                 : "s"(__builtin_amdgcn_readfirstlane(lds_addr)), "v"(offset), "s"(sbase)
                 : "memory", "m0");
}

__device__ __forceinline__ uint32_t lds_addr32(const void* p) {
    return (uint32_t)(uintptr_t)(const DN_LDS void*)p;
}

__device__ __forceinline__ u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
// register load with the non-temporal hint (read-once streams, as above)
__device__ __forceinline__ u32x4 ld16_stream(const void* p) {
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

__device__ __forceinline__ u32x4 lds_ld16(const DN_LDS void* p) {
    return *reinterpret_cast<const DN_LDS u32x4*>(p);
}

__device__ __forceinline__ DN_LDS char* lds_ptr(char* p) { return (DN_LDS char*)(p); }

// ----------------------------------------------------------------- cross-lane
// Sum / max over the four lanes that share (l & 15): l, l^16, l^32, l^48.
// v_permlane{16,32}_swap with both operands = v leaves lane l holding the pair
// {v[l], v[l ^ 16]} (resp. l ^ 32), so one VALU op per level, no LDS traffic.
// v_max_f32 directly (fmaxf on bit-cast values gets canonicalizing maxes added).
// The compiler's hazard pass does not guard inline assembly that consumes a
// just-written VGPR, so the s_nop supplies the wait state a permlane-swap or
// transcendental result may need.
__device__ __forceinline__ float vmax2(float a, float b) {
    float d;
    asm("s_nop 0\n\tv_max_f32 %0, %1, %2" : "=v"(d) : "v"(a), "v"(b));
    return d;
}
__device__ __forceinline__ float xor16_pair_op(float v, bool is_max) {
    const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    const float a = __uint_as_float(p[0]), b = __uint_as_float(p[1]);
    return is_max ? vmax2(a, b) : a + b;
}
__device__ __forceinline__ float xor32_pair_op(float v, bool is_max) {
    const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    const float a = __uint_as_float(p[0]), b = __uint_as_float(p[1]);
    return is_max ? vmax2(a, b) : a + b;
}
// Sum over all 64 lanes (every lane gets the total).
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
    return v;
}
__device__ __forceinline__ float sum_lane_groups(float v) { return xor32_pair_op(xor16_pair_op(v, false), false); }
__device__ __forceinline__ float max_lane_groups(float v) { return xor32_pair_op(xor16_pair_op(v, true), true); }

// ----------------------------------------------------------------- row statistics
// rstd = 1/sqrt(var + eps) from one-pass moments, var = E[x^2] - mean^2 (Eq. (1)-(2);
// RMSNorm, Eq. (6): mean = 0).  Rounding can take the difference slightly below
// zero, so it is clamped at 0 -- but only when it is a number: a row holding NaN
// or +-inf has NaN moments (inf - inf), and its statistics stay NaN so that every
// output of the row is NaN, as the plain definition gives.  A zero variance with
// eps = 0 makes the definition (x - mean) / 0 = 0/0 for every element: NaN as well.
__device__ __forceinline__ float rstd_from_moments(float mean_sq, float mean, float eps) {
    const float d = mean_sq - mean * mean;
    const float var = d > 0.f ? d : (d == d ? 0.f : d);
    const float r = 1.0f / __builtin_sqrtf(var + eps);
    return r == __builtin_inff() ? __builtin_nanf("") : r;
}

// ----------------------------------------------------------------- 8x8 bf16 transpose
// in[r] holds 8 bf16 (columns 0..7) of row r; out[c] gets column c (rows 0..7).
__device__ __forceinline__ void transpose8x8_bf16(const u32x4 in[8], u32x4 out[8]) {
#pragma unroll
    for (int c = 0; c < 8; ++c) {
        const int w = c >> 1;
        // v_perm_b32(hi_src, lo_src, sel): bytes 0-3 come from lo_src, 4-7 from hi_src
        const uint32_t sel = (c & 1) ? 0x07060302u : 0x05040100u;
#pragma unroll
        for (int j = 0; j < 4; ++j)
            out[c][j] = __builtin_amdgcn_perm(in[2 * j + 1][w], in[2 * j][w], sel);
    }
}

// ----------------------------------------------------------------- workgroup -> tile order
// Consecutive workgroup ids are dispatched round-robin over the 8 XCDs.  This
// bijection gives each XCD a contiguous range of logical tile ids, so tiles
// that share operand rows run under the same L2.
__device__ __forceinline__ int xcd_contiguous(int bid, int nblk) {
    const int q = nblk >> 3, r = nblk & 7;
    const int x = bid & 7, local = bid >> 3;
    return x * q + (x < r ? x : r) + local;
}

}  // namespace dn
