// es_device.hpp -- device-side random stream of the library (gfx950).
//
// The search distribution of the evosax report (arXiv 2212.04180, Sec. 2.1)
// is an isotropic Gaussian N(m, sigma^2 I); the report samples it with JAX's
// splittable keys (Listing 1) and names no generator.  This library draws it
// from Philox-4x32-10 (Salmon et al., SC'11), a counter-based generator: any
// block of four words is a pure function of (key, counter), so the same
// perturbation is regenerated in the evaluate kernel and again in the tell
// kernel and never written to memory.
//
// Stream layout: key = (lo32(seed + r), hi32(seed + r)) for run r; counter =
// (block = d/4, row, t, domain).  Domains: NOISE (row = antithetic pair,
// t = generation), INIT (initial mean), PROBLEM (shift vector / teacher),
// EVAL (MLP inputs of generation t).
//
// Normals: Box-Muller on word pairs, u = ((w >> 8) + 1) 2^-24 in (0, 1] for
// the radius and th = (w >> 8) 2^-24 in [0, 1) for the angle.  The angle goes
// straight into v_sin_f32 / v_cos_f32, which take their argument in
// revolutions, and the radius uses v_log_f32 (log2) and v_sqrt_f32.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace esmi {

enum : uint32_t { DOM_NOISE = 0, DOM_INIT = 1, DOM_PROBLEM = 2, DOM_EVAL = 3 };

// 32x32 -> 64-bit product as one v_mad_u64_u32.  Left to itself the compiler
// sometimes splits a product into v_mul_lo_u32 + v_mul_hi_u32, which costs
// twice the issue slots.
__device__ __forceinline__ uint64_t mul_wide(uint32_t a, uint32_t b)
{
    uint64_t r;
    asm("v_mad_u64_u32 %0, vcc, %1, %2, 0" : "=v"(r) : "v"(a), "s"(b) : "vcc");
    return r;
}

// Which counter word varies across the lanes of a wavefront; the others are
// uniform (the generation t and the domain always are).
enum PhiloxLanes { LANES_BLOCK_AND_ROW = 0, LANES_ROW = 1, LANES_BLOCK = 2 };

// Philox-4x32-10.  Each round forms two 32x32->64 products and folds the high
// halves with the other words and the round key through one three-input xor
// (v_bitop3_b32, truth table 0x96).  The key is uniform across a wavefront,
// so the key schedule lives in scalar registers.  In the first rounds some
// words only depend on uniform inputs (the generation, the domain, and the
// block or the row when it is the same across the wavefront): those products
// and xors are written as plain integer arithmetic, which the compiler runs
// on the scalar unit, and every lane-varying product is one v_mad_u64_u32.
//
// Uniformity of the counter words at the start of round i for lane layout V:
// bit k set = word k is the same across the wavefront.
template <int V>
struct PhiloxUniform {
    static constexpr unsigned at(int i)
    {
        // round 0: the block (word 0) varies unless V == LANES_ROW, the row
        // (word 1) unless V == LANES_BLOCK; t and the domain never vary
        unsigned u = (V == LANES_ROW ? 1u : 0u) | (V == LANES_BLOCK ? 2u : 0u) | 4u | 8u;
        for (int r = 0; r < i; ++r) {
            const bool p0 = u & 1u, p1 = u & 4u;             // products of words 0 and 2
            const bool n0 = p1 && (u & 2u), n2 = p0 && (u & 8u);
            u = (n0 ? 1u : 0u) | (p1 ? 2u : 0u) | (n2 ? 4u : 0u) | (p0 ? 8u : 0u);
        }
        return u;
    }
};

template <int V = LANES_BLOCK_AND_ROW>
__device__ __forceinline__ uint4 philox4x32_10(uint32_t k0, uint32_t k1, uint32_t c0, uint32_t c1,
                                               uint32_t c2, uint32_t c3)
{
#pragma unroll
    for (int i = 0; i < 10; ++i) {
        const unsigned u = PhiloxUniform<V>::at(i);
        const bool u0 = u & 1u, u1 = u & 2u, u2 = u & 4u, u3 = u & 8u;
        const uint64_t p0 = u0 ? (uint64_t)0xD2511F53u * c0 : mul_wide(c0, 0xD2511F53u);
        const uint64_t p1 = u2 ? (uint64_t)0xCD9E8D57u * c2 : mul_wide(c2, 0xCD9E8D57u);
        const uint32_t h1 = (uint32_t)(p1 >> 32), h0 = (uint32_t)(p0 >> 32);
        const uint32_t n0 = u2 && u1 ? h1 ^ c1 ^ k0 : __builtin_amdgcn_bitop3_b32(h1, c1, k0, 0x96);
        const uint32_t n2 = u0 && u3 ? h0 ^ c3 ^ k1 : __builtin_amdgcn_bitop3_b32(h0, c3, k1, 0x96);
        c1 = (uint32_t)p1;
        c3 = (uint32_t)p0;
        c0 = n0;
        c2 = n2;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    return make_uint4(c0, c1, c2, c3);
}

// Box-Muller radius sqrt(-2 ln u) = sqrt(-2 ln2 * log2 u), u in (0, 1].
// u = ((w >> 8) + 1) 2^-24 is formed as one fma of the integer w >> 8 (exact
// in fp32, below 2^24): the exact product plus 2^-24 is at most 1 and a
// multiple of 2^-24, so the fma rounds nothing and no integer add is needed.
__device__ __forceinline__ float bm_radius(uint32_t w)
{
    const float u = __builtin_fmaf((float)(w >> 8), 0x1p-24f, 0x1p-24f);
    return __builtin_amdgcn_sqrtf(-1.38629436111989061883f * __builtin_amdgcn_logf(u));
}

// Angle in revolutions, exact.
__device__ __forceinline__ float bm_turns(uint32_t w) { return (float)(w >> 8) * 0x1p-24f; }

// Four standard normals from one Philox block.
__device__ __forceinline__ void box_muller4(uint4 w, float e[4])
{
    const float r0 = bm_radius(w.x), a0 = bm_turns(w.y);
    const float r1 = bm_radius(w.z), a1 = bm_turns(w.w);
    e[0] = r0 * __builtin_amdgcn_cosf(a0);
    e[1] = r0 * __builtin_amdgcn_sinf(a0);
    e[2] = r1 * __builtin_amdgcn_cosf(a1);
    e[3] = r1 * __builtin_amdgcn_sinf(a1);
}

__device__ __forceinline__ void normals4(uint64_t key, uint32_t block, uint32_t row, uint32_t t,
                                         uint32_t domain, float e[4])
{
    box_muller4(philox4x32_10((uint32_t)key, (uint32_t)(key >> 32), block, row, t, domain), e);
}

// cos(2 pi x) for any finite x: v_cos_f32 takes revolutions and is accurate
// for small arguments, so the integer part is removed first.  cos is even, so
// the turns are taken of |x| (a free source modifier) and one v_fract_f32
// (|x| - floor |x|, exact for a non-negative argument) does the reduction, one
// instruction fewer than x - rint x; f(m + s) and f(m - s) stay equal bit for
// bit, as the antithetic pairs of a symmetric problem must.
__device__ __forceinline__ float cos_2pi(float x)
{
    return __builtin_amdgcn_cosf(__builtin_amdgcn_fractf(__builtin_fabsf(x)));
}

// Order-preserving map of a fitness to an unsigned key: minimisation order,
// maximise = 1 negates, NaN sorts as +inf, -0 equals +0.
__device__ __forceinline__ uint32_t order_key(float f, int maximize)
{
    float k = maximize ? -f : f;
    if (k != k) k = __builtin_inff();
    if (k == 0.0f) k = 0.0f;
    const uint32_t u = __float_as_uint(k);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

}  // namespace esmi
