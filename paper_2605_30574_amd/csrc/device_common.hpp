// device_common.hpp -- constants and device helpers shared by the splice
// library's kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "plan.hpp"
#include "splice_attn.h"

namespace splice_dev {


constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
using splice::kMaxSlots;
using splice::kRowBlock;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

constexpr int cmax(int x, int y) { return x > y ? x : y; }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                           __builtin_bit_cast(bf16x2_t, b), c, false);
}

// Sum over the LPK consecutive lanes of a row group (LPK in {4, 8, 16}), every
// lane of the group ending with the same bits.  DPP: quad_perm [1,0,3,2],
// quad_perm [2,3,0,1], row_half_mirror, row_mirror.
template <int LPK>
__device__ __forceinline__ float group_sum(float x) {
    // update_dpp with old = 0 lets the compiler fold each move into v_add_f32_dpp
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0xB1, 0xF, 0xF, false));
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x4E, 0xF, 0xF, false));
    if constexpr (LPK >= 8)
        x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x141, 0xF, 0xF, false));
    if constexpr (LPK >= 16)
        x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x140, 0xF, 0xF, false));
    return x;
}

// x + (x of the lane r places further on in its 16-lane DPP row), r in {4, 8}.
template <int R>
__device__ __forceinline__ float add_row_ror(float x) {
    return x + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x120 + R, 0xF, 0xF, false));
}

// 2^x with v_exp_f32 (results below 2^-126 flush to zero: negligible weights).
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ bool bit_set(const uint32_t *mask, int c) {
    return (mask[c >> 5] >> (c & 31)) & 1u;
}

// Compile-time loop: f(std::integral_constant<int, I>) for I in [B, E), so
// register arrays are only ever indexed by constants.
template <int B, int E, class F>
__device__ __forceinline__ void static_for(F &&f) {
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        static_for<B + 1, E>(f);
    }
}

// Lazy rescaling: a running maximum is only raised when a score exceeds it
// by more than this many powers of two, so weights stay <= 2^kSlack and the
// rescale of the accumulators is rare.  The result is exact either way: a
// partial result only needs its (m, l, o) to share one reference m.
constexpr float kSlack = 8.f;

// Select one of two row bases by a flag that may differ between lanes.  The
// choice is made on a 64-bit offset in registers: written as a choice between
// two kernel-argument fields, it can compile to a load from the argument
// segment whose wait also waits for every row load already in flight.
__device__ __forceinline__ const char *pick_base(bool second, const char *first_base,
                                                 const char *second_base) {
    const uintptr_t delta = (uintptr_t)second_base - (uintptr_t)first_base;
    return first_base + (second ? delta : (uintptr_t)0);
}

}  // namespace splice_dev
