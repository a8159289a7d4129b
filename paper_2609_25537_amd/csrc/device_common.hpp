// Device-side helpers shared by the CMC kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cmc {

constexpr int kWave = 64;

// ---------------------------------------------------------------- bf16

// bf16 is the upper half of an fp32 pattern; a 32-bit word holds element 2i
// in its low half and element 2i+1 in its high half.
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Widen one 16-byte vector of K/V elements to fp32.
template <typename T> struct Vec16;

template <> struct Vec16<float> {
    static constexpr int N = 4;
    __device__ __forceinline__ static void widen(const uint4 &v, float (&f)[4]) {
        f[0] = __uint_as_float(v.x);
        f[1] = __uint_as_float(v.y);
        f[2] = __uint_as_float(v.z);
        f[3] = __uint_as_float(v.w);
    }
};

template <> struct Vec16<uint16_t> {
    static constexpr int N = 8;
    __device__ __forceinline__ static void widen(const uint4 &v, float (&f)[8]) {
        f[0] = bf16_lo(v.x); f[1] = bf16_hi(v.x);
        f[2] = bf16_lo(v.y); f[3] = bf16_hi(v.y);
        f[4] = bf16_lo(v.z); f[5] = bf16_hi(v.z);
        f[6] = bf16_lo(v.w); f[7] = bf16_hi(v.w);
    }
};

// ------------------------------------------------------- lane exchange
//
// Exchanging v with lane (lane ^ M): masks 1 and 2 are DPP
// quad permutes, 7 and 15 the DPP half-row / row mirrors, 8 a row rotate by
// 8; 16 and 32 are the gfx950 row swaps v_permlane16_swap /
// v_permlane32_swap (VALU, no LDS round trip, so independent reductions
// interleave).  A butterfly over masks {1, 2, 7, 15, 16, 32} (linearly
// independent bit patterns) reduces a group of 2^n lanes with every lane
// ending on the bitwise same value, because each step combines symmetric
// pairs.

template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL,
                                                                0xF, 0xF, false));
}
// The same exchange for a sum: with 0 as the value a lane outside the row
// would read (none does: every pattern used stays inside a 16-lane row), the
// compiler folds the exchange into the add (one v_add_f32 with a DPP
// operand per step instead of a move and an add).
template <int CTRL>
__device__ __forceinline__ float dpp_sum_operand(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL,
                                                                   0xF, 0xF, true));
}

struct OpSum {
    __device__ __forceinline__ static float f(float a, float b) { return a + b; }
    template <int CTRL>
    __device__ __forceinline__ static float partner(float v) { return dpp_sum_operand<CTRL>(v); }
};
struct OpMax {
    __device__ __forceinline__ static float f(float a, float b) { return fmaxf(a, b); }
    template <int CTRL>
    __device__ __forceinline__ static float partner(float v) { return dpp_mov<CTRL>(v); }
};

// The max over aligned 16-lane groups on order-preserving integer keys (a
// float's bits with the magnitude bits flipped when the sign is set, so the
// signed integer order is the float order, -0 below +0): the exchange folds
// into v_max_i32 (one instruction per step), where fmaxf needs a move and
// two NaN-quieting maxima besides.  Same result as lane_reduce<OpMax, 1, 16>
// for inputs without NaN.
__device__ __forceinline__ int f32_order_key(float x) {
    const int b = __float_as_int(x);
    return b ^ (int)((unsigned)(b >> 31) >> 1);
}
__device__ __forceinline__ float lane_max16(float v) {
    int k = f32_order_key(v);
    k = max(k, __builtin_amdgcn_update_dpp(0, k, 0xB1, 0xF, 0xF, true));   // ^1
    k = max(k, __builtin_amdgcn_update_dpp(0, k, 0x4E, 0xF, 0xF, true));   // ^2
    k = max(k, __builtin_amdgcn_update_dpp(0, k, 0x141, 0xF, 0xF, true));  // ^7
    k = max(k, __builtin_amdgcn_update_dpp(0, k, 0x140, 0xF, 0xF, true));  // ^15
    return __int_as_float(k ^ (int)((unsigned)(k >> 31) >> 1));
}

// f(v, v of lane ^ 16) and f(v, v of lane ^ 32).  Each swap returns the pair
// {v, partner's v} in a lane-dependent order; the combine ops are
// commutative, so the result is the same bits in either order.
template <typename Op>
__device__ __forceinline__ float combine_xor16(float v) {
    const unsigned u = __float_as_uint(v);
    const auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    return Op::f(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
template <typename Op>
__device__ __forceinline__ float combine_xor32(float v) {
    const unsigned u = __float_as_uint(v);
    const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
    return Op::f(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Combine v over the lane-index bits selected by [LO, HI) (powers of two):
// lane_reduce<Op, 1, 16> reduces within aligned 16-lane groups,
// lane_reduce<Op, 16, 64> across the four 16-lane rows, etc.
template <typename Op, int LO, int HI>
__device__ __forceinline__ float lane_reduce(float v) {
    if constexpr (LO <= 1 && HI > 1) v = Op::f(v, Op::template partner<0xB1>(v));     // ^1
    if constexpr (LO <= 2 && HI > 2) v = Op::f(v, Op::template partner<0x4E>(v));     // ^2
    if constexpr (LO <= 4 && HI > 4) {
        if constexpr (LO <= 1) v = Op::f(v, Op::template partner<0x141>(v));           // ^7 (after ^1,^2)
        else v = Op::f(v, __shfl_xor(v, 4));
    }
    if constexpr (LO <= 8 && HI > 8) {
        if constexpr (LO <= 1) v = Op::f(v, Op::template partner<0x140>(v));           // ^15 (after ^1,^2,^7)
        else v = Op::f(v, Op::template partner<0x128>(v));                             // ^8 (row rotate 8)
    }
    if constexpr (LO <= 16 && HI > 16) v = combine_xor16<Op>(v);
    if constexpr (LO <= 32 && HI > 32) v = combine_xor32<Op>(v);
    return v;
}

}  // namespace cmc
