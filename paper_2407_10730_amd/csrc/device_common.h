// device_common.h -- device helpers shared by the GEMM kernels of the conv2d library.
#pragma once

#include "conv2d_internal.h"

namespace cv {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

#define OOB_OFF 0x80000000u
#define RSRC_WORD3 0x00020000

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, RSRC_WORD3);
}

__device__ __forceinline__ float ld_f32(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}
__device__ __forceinline__ uint16_t ld_u16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0);
}
__device__ __forceinline__ void st_f32(__amdgpu_buffer_rsrc_t r, uint32_t off, float v) {
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), r, off, 0, 0);
}
__device__ __forceinline__ void st_u16(__amdgpu_buffer_rsrc_t r, uint32_t off, uint16_t v) {
    __builtin_amdgcn_raw_buffer_store_b16(v, r, off, 0, 0);
}

// fp32 -> bf16 bits, round to nearest even (inputs are finite).
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __builtin_bit_cast(uint32_t, f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

template <typename TOut>
__device__ __forceinline__ void store_out(__amdgpu_buffer_rsrc_t r, uint32_t elem_off_valid, bool ok,
                                          float v);
template <>
__device__ __forceinline__ void store_out<float>(__amdgpu_buffer_rsrc_t r, uint32_t e, bool ok, float v) {
    st_f32(r, ok ? e * 4u : OOB_OFF, v);
}
template <>
__device__ __forceinline__ void store_out<uint16_t>(__amdgpu_buffer_rsrc_t r, uint32_t e, bool ok,
                                                    float v) {
    st_u16(r, ok ? e * 2u : OOB_OFF, f32_to_bf16_rne(v));
}

// Four consecutive output elements starting at element e (e a multiple of 4): one 16-byte
// (fp32) or 8-byte (bf16, round to nearest even) store.
template <typename TOut>
__device__ __forceinline__ void store_out4(__amdgpu_buffer_rsrc_t r, uint32_t e, bool ok, float a, float b, float c,
                                           float d);
template <>
__device__ __forceinline__ void store_out4<float>(__amdgpu_buffer_rsrc_t r, uint32_t e, bool ok, float a, float b,
                                                  float c, float d) {
    __builtin_amdgcn_raw_buffer_store_b128(u32x4{__builtin_bit_cast(uint32_t, a), __builtin_bit_cast(uint32_t, b),
                                                 __builtin_bit_cast(uint32_t, c), __builtin_bit_cast(uint32_t, d)},
                                           r, ok ? e * 4u : OOB_OFF, 0, 0);
}
template <>
__device__ __forceinline__ void store_out4<uint16_t>(__amdgpu_buffer_rsrc_t r, uint32_t e, bool ok, float a, float b,
                                                     float c, float d) {
    __builtin_amdgcn_raw_buffer_store_b64(
        u32x2{(uint32_t)f32_to_bf16_rne(a) | ((uint32_t)f32_to_bf16_rne(b) << 16),
              (uint32_t)f32_to_bf16_rne(c) | ((uint32_t)f32_to_bf16_rne(d) << 16)},
        r, ok ? e * 2u : OOB_OFF, 0, 0);
}

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Two consecutive output elements starting at element e (e even): one 8-byte (fp32) or
// 4-byte (bf16: the hardware's packed conversion, round to nearest even) store.
template <typename TOut>
__device__ __forceinline__ void store_out2(__amdgpu_buffer_rsrc_t r, uint32_t e, bool ok, float lo, float hi);
template <>
__device__ __forceinline__ void store_out2<float>(__amdgpu_buffer_rsrc_t r, uint32_t e, bool ok, float lo, float hi) {
    __builtin_amdgcn_raw_buffer_store_b64(u32x2{__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi)}, r,
                                          ok ? e * 4u : OOB_OFF, 0, 0);
}
template <>
__device__ __forceinline__ void store_out2<uint16_t>(__amdgpu_buffer_rsrc_t r, uint32_t e, bool ok, float lo,
                                                     float hi) {
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2)),
                                          r, ok ? e * 2u : OOB_OFF, 0, 0);
}

// The value of lane l ^ 1 (a DPP quad permutation, no LDS).
__device__ __forceinline__ float swap_adjacent_lanes(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0xB1, 0xF, 0xF, false));
}

// n / d for 0 <= n < 2^31 with the divisor's multiplier and shift (FastDiv).
__device__ __forceinline__ uint32_t fdiv(uint32_t n, FastDiv f) { return (__umulhi(n, f.m) + n) >> f.s; }

// Linear block id -> tile id such that consecutive tile ids land on the same
// XCD (workgroups are handed to the 8 XCDs round-robin), so the M tiles of one
// pixel tile and neighbouring pixel tiles share an L2.
__device__ __forceinline__ int xcd_remap(int bid, int nb) {
    const int per = nb >> 3, rem = nb & 7;
    const int xcd = bid & 7, slot = bid >> 3;
    return xcd < rem ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
}

// Per-column state of the implicit gather: window origin and base offset.
struct ColState {
    int64_t base;  // element offset of x[n, gi*Cg, hi0, wi0] (may be "negative" in padding)
    int32_t hi0, wi0;
};

__device__ __forceinline__ ColState col_state(const GemmArgs& A, int p, int gi) {
    ColState s;
    if (p < A.P) {
        const int n = p / A.HoWo;
        const int hw = p - n * A.HoWo;
        const int ho = hw / A.Wo;
        const int wo = hw - ho * A.Wo;
        s.hi0 = ho * A.sh - A.ph;
        s.wi0 = wo * A.sw - A.pw;
        s.base = (int64_t)n * A.x_nstride + (int64_t)gi * A.b_gstride + (int64_t)s.hi0 * A.W + s.wi0;
    } else {
        s.hi0 = KTAB_DEAD;
        s.wi0 = 0;
        s.base = 0;
    }
    return s;
}

// Byte offset of B[kr][col] for the implicit gather (or OOB_OFF for a zero tap).
template <int ESIZE>
__device__ __forceinline__ uint32_t implicit_off(const GemmArgs& A, const ColState& cs, const KTabEntry& e) {
    const int hi = cs.hi0 + e.roff;
    const int wi = cs.wi0 + e.soff;
    const bool ok = ((unsigned)hi < (unsigned)A.H) & ((unsigned)wi < (unsigned)A.W);
    return ok ? (uint32_t)((cs.base + e.coff) * ESIZE) : OOB_OFF;
}

// Scalar (wave-uniform) read of one table entry.
__device__ __forceinline__ KTabEntry ktab_at(const KTabEntry* t, int kr) {
    kr = __builtin_amdgcn_readfirstlane(kr);
    return t[kr];
}

}  // namespace cv
