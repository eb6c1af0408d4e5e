// RoPE at read time, shared by the prefill and decode kernels (App. B: the cache holds
// unrotated vectors and the kernel rotates what it reads, so a pair the window prunes is
// neither read nor rotated).  Rotate-half convention: pair r of a d-vector is dims r and
// r + d/2, turned by position * theta_r.  A fragment is the 8 elements of half hh of pairs
// 8c .. 8c + 7 (16 bytes), as the matrix-instruction operands hold them.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace atf {
namespace rope {

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// The angle of pair r at position pos, in revolutions: the high word of the fraction of
// pos * rho_r (rho_r = theta_r / (2 pi) in 0.64 fixed point), exact for every position
// below 2^32 up to the last bit of rho_r.
__device__ __forceinline__ float revolutions(uint32_t pos, uint2 rho) {
    return float(pos * rho.x + __umulhi(pos, rho.y)) * 2.3283064365386963e-10f;  // 2^-32
}

// Rotate one element pair given cos and sin of its angle: half 0 holds the first
// components x_r, half 1 the second x_{r + d/2}; x'_r = x_r cos - x_{r+d/2} sin and
// x'_{r+d/2} = x_{r+d/2} cos + x_r sin, in fp32.
__device__ __forceinline__ float turn(float own, float other, float sgn, float cs, float sn) {
    return __builtin_fmaf(own, cs, sgn * other * sn);
}

// Rotate one fragment (`own`, half hh) given the other half of the same pairs (`other`)
// and the cosines and sines of the 8 pairs' angles; rounded to bf16.
__device__ __forceinline__ u32x4_t rotate_cs(u32x4_t own, u32x4_t other, int hh, const float* cs8,
                                             const float* sn8) {
    const float sgn = hh ? 1.f : -1.f;
    u32x4_t r;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        const float o0 = __uint_as_float(own[t] << 16), o1 = __uint_as_float(own[t] & 0xFFFF0000u);
        const float x0 = __uint_as_float(other[t] << 16), x1 = __uint_as_float(other[t] & 0xFFFF0000u);
        bf16x2_t two;
        two[0] = (__bf16)turn(o0, x0, sgn, cs8[2 * t], sn8[2 * t]);
        two[1] = (__bf16)turn(o1, x1, sgn, cs8[2 * t + 1], sn8[2 * t + 1]);
        r[t] = __builtin_bit_cast(uint32_t, two);
    }
    return r;
}

// The same for a vector at position pos, its angles evaluated directly (v_cos_f32 /
// v_sin_f32 take their argument in revolutions).
__device__ __forceinline__ u32x4_t rotate(u32x4_t own, u32x4_t other, int hh, uint32_t pos,
                                          const uint32_t* rho_hi8, const uint32_t* rho_lo8) {
    float cs8[8], sn8[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const float u = revolutions(pos, make_uint2(rho_hi8[e], rho_lo8[e]));
        cs8[e] = __builtin_amdgcn_cosf(u);
        sn8[e] = __builtin_amdgcn_sinf(u);
    }
    return rotate_cs(own, other, hh, cs8, sn8);
}

// The other half of a fragment: lane l gets the registers of lane l ^ 32 (the same
// token or row, the other 8 dims of each pair).  Every lane of the wave must execute it.
__device__ __forceinline__ u32x4_t other_half(u32x4_t x, int hh) {
    u32x4_t r;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        // lanes 32..63 of the first copy trade places with lanes 0..31 of the second
        const auto sw = __builtin_amdgcn_permlane32_swap(x[t], x[t], false, false);
        r[t] = hh ? sw[0] : sw[1];
    }
    return r;
}

}  // namespace rope
}  // namespace atf
