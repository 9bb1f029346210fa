// bdlm_device.h -- device helpers shared by the gfx950 kernels of libbdlm:
// vector types, bf16 hi/lo splitting, MFMA wrappers, unconditional chunk loads and
// the LDS image layout of the B and C operands.  Internal; included by the .hip
// sources only.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bdlm.h"

namespace bdlm {
namespace {

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kP = BDLM_HEADDIM;  // 64 head-dim columns per head
constexpr float kLog2e = 1.4426950408889634f;


// ---------------------------------------------------------------- bf16 helpers
__device__ __forceinline__ short bf16_bits(float v) {
    return __builtin_bit_cast(short, static_cast<__bf16>(v));  // round to nearest even
}
__device__ __forceinline__ float bf16_to_f32(short s) {
    return __uint_as_float(static_cast<uint32_t>(static_cast<uint16_t>(s)) << 16);
}
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Two floats to two bf16 (round to nearest even), a in the low half, b in the high
// half: a two-wide conversion compiles to one packed v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t cvt_pk_bf16(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{a, b}, bf16x2));
}

// v = hi + lo + O(2^-16 |v|), both parts rounded to nearest even
__device__ __forceinline__ void split4(f32x4 v, s16x4 &hi, s16x4 &lo) {
    const uint32_t h01 = cvt_pk_bf16(v[0], v[1]), h23 = cvt_pk_bf16(v[2], v[3]);
    const float r0 = v[0] - __uint_as_float(h01 << 16);
    const float r1 = v[1] - __uint_as_float(h01 & 0xffff0000u);
    const float r2 = v[2] - __uint_as_float(h23 << 16);
    const float r3 = v[3] - __uint_as_float(h23 & 0xffff0000u);
    hi = __builtin_bit_cast(s16x4, uint2{h01, h23});
    lo = __builtin_bit_cast(s16x4, uint2{cvt_pk_bf16(r0, r1), cvt_pk_bf16(r2, r3)});
}

// v = hi + mid + lo + O(2^-26 |v|): three bf16 terms, each the rounded remainder of the
// previous ones (the remainders v - hi and v - hi - mid are exact in fp32).  Operands of
// state updates whose results are carried over many blocks use three terms: the
// two-term residual (2^-18 per input) adds up across the tokens a state remembers.
__device__ __forceinline__ void split4x3(f32x4 v, s16x4 &hi, s16x4 &mid, s16x4 &lo) {
    split4(v, hi, mid);
    f32x4 r;
#pragma unroll
    for (int i = 0; i < 4; ++i) r[i] = (v[i] - bf16_to_f32(hi[i])) - bf16_to_f32(mid[i]);
    lo = __builtin_bit_cast(s16x4, uint2{cvt_pk_bf16(r[0], r[1]), cvt_pk_bf16(r[2], r[3])});
}

// Materialise v here: later code depends on this point, so the compiler can neither
// sink the computation of v below it nor hoist its uses above it.
__device__ __forceinline__ void pin(float &v) { asm volatile("" : "+v"(v)); }

// Activation storage.
template <bool F32> struct Act;
template <> struct Act<false> {
    using T = uint16_t;
    static __device__ __forceinline__ float val(T v) {
        return __uint_as_float(static_cast<uint32_t>(v) << 16);
    }
};
template <> struct Act<true> {
    using T = float;
    static __device__ __forceinline__ float val(T v) { return v; }
};

// ---------------------------------------------------------------- MFMA helpers
__device__ __forceinline__ f32x4 mma_k32(s16x4 a0, s16x4 a1, s16x4 b0, s16x4 b1, f32x4 c) {
    const s16x8 a = __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
    const s16x8 b = __builtin_shufflevector(b0, b1, 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma_k16(s16x4 a, s16x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
}
// c += sum over Q quads of A_q B_q (16 contraction indices per quad).  An accumulator is
// never handed from one MFMA shape to another: a dependent 16-deep MFMA issued right after
// the 32-deep one that produced its accumulator input has read part of that input before
// it was written (two of the four rows, measured).  So an odd last quad after pairs runs
// as a 32-deep MFMA with a zero upper half.
template <int Q>
__device__ __forceinline__ f32x4 mma_quads(const s16x4 (&a)[Q], const s16x4 (&b)[Q], f32x4 c) {
#pragma unroll
    for (int q = 0; q + 1 < Q; q += 2) c = mma_k32(a[q], a[q + 1], b[q], b[q + 1], c);
    if constexpr (Q == 1) {
        c = mma_k16(a[0], b[0], c);
    } else if constexpr (Q & 1) {
        constexpr s16x4 z = {0, 0, 0, 0};
        c = mma_k32(a[Q - 1], z, b[Q - 1], z, c);
    }
    return c;
}

__device__ __forceinline__ float shfl(float v, int src) { return __shfl(v, src, 64); }

// Inclusive sum over the 64 lanes of a wave on DPP, without LDS: shifts by 1, 2, 4, 8
// within each row of 16 lanes (lanes shifted in from outside the row read 0), then
// row 0's total into row 1 (and row 2's into row 3), then the total of rows 0-1 into
// rows 2-3.
template <int CTRL, int ROW_MASK, bool BOUND_ZERO>
__device__ __forceinline__ float dpp(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, ROW_MASK, 0xf,
                                                      BOUND_ZERO));
}
__device__ __forceinline__ float wave_inclusive_sum(float v) {
    v += dpp<0x111, 0xf, true>(v);   // row_shr:1
    v += dpp<0x112, 0xf, true>(v);   // row_shr:2
    v += dpp<0x114, 0xf, true>(v);   // row_shr:4
    v += dpp<0x118, 0xf, true>(v);   // row_shr:8
    v += dpp<0x142, 0xa, false>(v);  // row_bcast:15 into rows 1 and 3
    v += dpp<0x143, 0xc, false>(v);  // row_bcast:31 into rows 2 and 3
    return v;
}

// Rows past the end of the block read this zero chunk instead of activations: the
// load address is selected, never the loaded value, so every load stays an
// unconditional instruction that can be issued ahead of any wait.
__device__ const uint4 kZeroChunk = {0u, 0u, 0u, 0u};

// Global-address-space views, so selected pointers still compile to global loads.
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) const u32x4 g_u4;
template <typename T>
__device__ __forceinline__ const g_u4 *gchunk(const T *p) {
    return (const g_u4 *)(p);
}
__device__ __forceinline__ const g_u4 *gzero() { return (const g_u4 *)(&kZeroChunk); }

__device__ __forceinline__ s16x4 as_s16x4(uint2 v) { return __builtin_bit_cast(s16x4, v); }
__device__ __forceinline__ uint2 as_u2(s16x4 v) { return __builtin_bit_cast(uint2, v); }

// LDS image of B or C: the quad that lane (col, grp) of an MFMA operand holds for
// token tile mt and dstate quad q (rows 16mt + col, columns 16q + 4grp .. +3).
// The column-in-tile is XOR-swizzled with the index of the 16-byte global chunk
// the quad came from, so a wave writing one row's chunks and a wave reading one
// quad per lane both touch 16 distinct bank pairs per 16 lanes.
template <int QN, bool F32>
__device__ __forceinline__ int img_idx(int mt, int q, int grp, int col) {
    const int chunk = F32 ? (4 * q + grp) : (2 * q + (grp >> 1));
    return (mt * QN + q) * 64 + grp * 16 + (col ^ (chunk & 15));
}

}  // namespace
}  // namespace bdlm
