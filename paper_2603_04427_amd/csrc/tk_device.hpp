// Device helpers shared by the gfx950 kernels: bf16 unpacking and packing,
// OCP E4M3 decoding through the hardware converter, and wavefront reductions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tk {

typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(8 * sizeof(short)))) short bf16x8;
typedef __attribute__((__vector_size__(2 * sizeof(float)))) float f32x2;

// bf16 pair packed in one dword -> two floats (exact).
__device__ __forceinline__ float bf16lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Two floats -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    typedef float f32x2_t __attribute__((ext_vector_type(2)));
    const f32x2_t x = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(x, bf16x2_t));
}

// sum of a packed bf16 pair, accumulated in fp32 (v_dot2c_f32_bf16 against (1, 1))
__device__ __forceinline__ float add_bf16_pair(uint32_t pair, float acc) {
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    const uint32_t ones = 0x3f803f80u;
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, pair),
                                           __builtin_bit_cast(bf16x2_t, ones), acc, false);
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// acc + a.lo * b.lo + a.hi * b.hi for packed bf16 pairs (v_dot2c_f32_bf16; the
// products are exact in fp32).
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float acc) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a), __builtin_bit_cast(bf16x2_t, b), acc,
                                           false);
}

// Two OCP E4M3 codes (byte pair 0-1 or 2-3 of w) -> packed bf16 pair, exact.
template <bool HI>
__device__ __forceinline__ uint32_t e4m3x2_bf16(uint32_t w) {
    return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, HI));
}

// Byte permute: pairs of 16-bit halves from two dwords.
__device__ __forceinline__ uint32_t lo_halves(uint32_t a, uint32_t b) {  // (a.lo, b.lo)
    return __builtin_amdgcn_perm(b, a, 0x05040100u);
}
__device__ __forceinline__ uint32_t hi_halves(uint32_t a, uint32_t b) {  // (a.hi, b.hi)
    return __builtin_amdgcn_perm(b, a, 0x07060302u);
}

// Four OCP E4M3 codes in one dword -> four floats (exact), gfx950 converter.
__device__ __forceinline__ void e4m3x4(uint32_t w, float& a, float& b, float& c, float& d) {
    f32x2 lo = __builtin_amdgcn_cvt_pk_f32_fp8(w, false);
    f32x2 hi = __builtin_amdgcn_cvt_pk_f32_fp8(w, true);
    a = lo[0];
    b = lo[1];
    c = hi[0];
    d = hi[1];
}

__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// ---------------------------------------------------------------- cross-lane
// DPP lane permutations inside a row of 16 lanes.
template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, true));
}
constexpr int kQuadXor1 = 0xB1;    // quad_perm [1,0,3,2]
constexpr int kQuadXor2 = 0x4E;    // quad_perm [2,3,0,1]
constexpr int kRowHalfMirror = 0x141;
constexpr int kRowMirror = 0x140;

// Exchange across 16- and 32-lane halves (gfx950 v_permlane16_swap /
// v_permlane32_swap with both operands the same value): r[0] + r[1] is the sum of
// the lane's value and its partner's (lane ^ 16, resp. lane ^ 32).
__device__ __forceinline__ float xor16_sum(float x) {
    auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float xor32_sum(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
// Maximum of two floats, NaN-propagating: one v_maximum_f32 (or a third operand
// of v_maximum3_f32) on gfx950, with no canonicalising copies of its inputs,
// which fmaxf's NaN-ignoring rule needs for values of unknown origin (matrix
// accumulators, lane exchanges). Equal to fmaxf whenever neither input is NaN.
__device__ __forceinline__ float max_f(float a, float b) { return __builtin_elementwise_maximum(a, b); }
__device__ __forceinline__ float xor16_max(float x) {
    auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return max_f(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xor32_max(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return max_f(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Sum / max over aligned groups of N lanes (N a power of two <= 64); every lane
// of the group receives the result.
template <int N>
__device__ __forceinline__ float group_sum(float x) {
    if constexpr (N >= 2) x += dpp<kQuadXor1>(x);
    if constexpr (N >= 4) x += dpp<kQuadXor2>(x);
    if constexpr (N >= 8) x += dpp<kRowHalfMirror>(x);
    if constexpr (N >= 16) x += dpp<kRowMirror>(x);
    if constexpr (N >= 32) x = xor16_sum(x);
    if constexpr (N >= 64) x = xor32_sum(x);
    return x;
}

template <int N>
__device__ __forceinline__ float group_max(float x) {
    if constexpr (N >= 2) x = max_f(x, dpp<kQuadXor1>(x));
    if constexpr (N >= 4) x = max_f(x, dpp<kQuadXor2>(x));
    if constexpr (N >= 8) x = max_f(x, dpp<kRowHalfMirror>(x));
    if constexpr (N >= 16) x = max_f(x, dpp<kRowMirror>(x));
    if constexpr (N >= 32) x = xor16_max(x);
    if constexpr (N >= 64) x = xor32_max(x);
    return x;
}

// Max / sum across lanes with the same (lane % STRIDE), STRIDE a power of two:
// row rotations (DPP row_ror by multiples of STRIDE keep the residue class)
// inside each 16-lane row, then the 16- and 32-lane half swaps.
template <int STRIDE>
__device__ __forceinline__ float strided_max(float x) {
    if constexpr (STRIDE <= 1) x = max_f(x, dpp<0x121>(x));
    if constexpr (STRIDE <= 2) x = max_f(x, dpp<0x122>(x));
    if constexpr (STRIDE <= 4) x = max_f(x, dpp<0x124>(x));
    if constexpr (STRIDE <= 8) x = max_f(x, dpp<0x128>(x));
    if constexpr (STRIDE <= 16) x = xor16_max(x);
    if constexpr (STRIDE <= 32) x = xor32_max(x);
    return x;
}
template <int STRIDE>
__device__ __forceinline__ float strided_sum(float x) {
    if constexpr (STRIDE <= 1) x += dpp<0x121>(x);
    if constexpr (STRIDE <= 2) x += dpp<0x122>(x);
    if constexpr (STRIDE <= 4) x += dpp<0x124>(x);
    if constexpr (STRIDE <= 8) x += dpp<0x128>(x);
    if constexpr (STRIDE <= 16) x = xor16_sum(x);
    if constexpr (STRIDE <= 32) x = xor32_sum(x);
    return x;
}

// Make this wave's LDS writes visible to its other lanes before they read.
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Global->LDS copy of 16 bytes per lane (global_load_lds_dwordx4: lane i writes
// LDS bytes lds + 16 i .. + 15 from base + off). It is issued as inline assembly
// on purpose: for the compiler's own form of this copy, every later transposing
// LDS read waits for all copies in flight, including the next tile's copy into
// the other buffer, which would stall each tile halfway. The copies are awaited
// explicitly (wait_loads) before the barrier that publishes a tile. M0, which
// holds the LDS destination, is restored afterwards.
__device__ __forceinline__ void copy16_to_lds(const char* base, uint32_t off, const uint16_t* lds) {
    const uint32_t la = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)lds;
    uint32_t saved;
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %3\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %1, %2\n\t"
        "s_nop 0\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "v"(off), "s"(base), "s"(la)
        : "memory");
}

// Global->LDS copy of 4 bytes per lane (global_load_lds_dword: lane i writes LDS
// bytes lds + 4 i .. + 3 from base + off), issued and awaited like copy16_to_lds.
__device__ __forceinline__ void copy4_to_lds(const char* base, uint32_t off, const void* lds) {
    const uint32_t la = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)lds;
    uint32_t saved;
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %3\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dword %1, %2\n\t"
        "s_nop 0\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "v"(off), "s"(base), "s"(la)
        : "memory");
}

// All of this wave's vector memory operations (the tile copies) have completed.
__device__ __forceinline__ void wait_loads() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

}  // namespace tk
