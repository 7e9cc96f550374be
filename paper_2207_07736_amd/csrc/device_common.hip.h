// device_common.hip.h -- RNG, uniform mapping and the cart-pole step, as gfx950
// device functions used by every simulator kernel.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rlsim_dev {

// ---------------------------------------------------------------------------
// Kernel-side constants.  Computed once on the host from rlsim_cfg, each by one
// fp32 operation (see make_dev_params in rlsim.hip).
// ---------------------------------------------------------------------------
struct DevParams {
    float gravity, force_mag, tau, half_length;   // tau here is the iteration length tau / C
    uint32_t iters;       // compute factor C: Euler iterations per simulation step
    float pole_ml;        // masspole * half_length
    float inv_total;      // 1 / (masscart + masspole)
    float m_over_M;       // masspole * inv_total
    float ml_over_M;      // pole_ml * inv_total
    float thr_x, thr_th;  // +inf when termination is disabled
    uint32_t max_steps;   // 0 = no time limit
    float reset_lo, reset_width;   // width = reset_high - reset_low
    float reset_width_u24;         // width * 2^-24 (exact; see uniform24_to)
    uint32_t key0, key1;  // Philox key: low and high word of the seed
    uint32_t env0;        // global id of the handle's environment 0 (RNG counters use global ids)
};

// Counter stream ids (third counter word).
enum : uint32_t { STREAM_RESET = 0u, STREAM_ACTION = 1u, STREAM_PARAMS = 2u, STREAM_POLICY = 3u };

// Philox4x32-10 (Salmon et al., SC'11) on counter (c0, c1, c2, c3) and key
// (k0, k1).  c1, c2, c3 and the key are wave-uniform in every caller, so the
// first round's second product and the whole key schedule land on the scalar
// unit.
__device__ __forceinline__ uint4 philox(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t k0, uint32_t k1,
                                        uint32_t c3 = 0u)
{
    // Recompute the key schedule at every call (scalar adds) rather than let
    // it be hoisted into twenty loop-invariant scalars that spill to VGPR lanes.
    asm volatile("" : "+s"(k0), "+s"(k1));
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        // full 64-bit products: one v_mad_u64_u32 gives both halves
        const uint64_t p0 = (uint64_t)0xD2511F53u * c0;
        const uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
        // three-input XOR in one v_bitop3_b32 (truth table 0x96)
        const uint32_t n0 = __builtin_amdgcn_bitop3_b32((uint32_t)(p1 >> 32), c1, k0, 0x96);
        const uint32_t n2 = __builtin_amdgcn_bitop3_b32((uint32_t)(p0 >> 32), c3, k1, 0x96);
        c0 = n0;
        c1 = (uint32_t)p1;
        c2 = n2;
        c3 = (uint32_t)p0;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    return make_uint4(c0, c1, c2, c3);
}

// Top 24 bits of r as a float in [0, 1 - 2^-24] (exact), then lo + u * width
// with a single rounding.
__device__ __forceinline__ float u24(uint32_t r) { return (float)(r >> 8) * 0x1.0p-24f; }
__device__ __forceinline__ float uniform01_to(uint32_t r, float lo, float width)
{
    return __builtin_fmaf(u24(r), width, lo);
}
// The same value with the 2^-24 scale moved onto the width: (m 2^-24) w and
// m (w 2^-24) are the same real number when w 2^-24 is exact, and the FMA
// rounds it once either way.  width_u24 must equal width * 2^-24 exactly.
__device__ __forceinline__ float uniform24_to(uint32_t r, float lo, float width_u24)
{
    return __builtin_fmaf((float)(r >> 8), width_u24, lo);
}

// Series sin / cos of degree 9 / 8, Horner form, one rounding per operation.
// Accurate to < 1 ulp for |th| <= 12 degrees (every pre-step angle of a live
// episode) and to 2.5e-8 + 2 ulp on |th| <= pi/4.
__device__ __forceinline__ void sincos_series(float th, float& s, float& c)
{
    const float s3 = (float)(-1.0 / 6.0), s5 = (float)(1.0 / 120.0);
    const float s7 = (float)(-1.0 / 5040.0), s9 = (float)(1.0 / 362880.0);
    const float c2 = -0.5f, c4 = (float)(1.0 / 24.0);
    const float c6 = (float)(-1.0 / 720.0), c8 = (float)(1.0 / 40320.0);
    const float z = th * th;
    float qs = __builtin_fmaf(s9, z, s7);
    qs = __builtin_fmaf(qs, z, s5);
    qs = __builtin_fmaf(qs, z, s3);
    s = __builtin_fmaf(th * z, qs, th);
    float qc = __builtin_fmaf(c8, z, c6);
    qc = __builtin_fmaf(qc, z, c4);
    qc = __builtin_fmaf(qc, z, c2);
    c = __builtin_fmaf(z, qc, 1.0f);
}

// sin / cos at any angle.  |th| <= fp32(pi/4) (every angle of a live
// cart-pole episode): the series itself.  Otherwise reduce by quadrants first:
// k = rint(th * fp32(2/pi)), r = th - k pi/2 with pi/2 = hi + lo in two FMAs
// (th - k hi is exact: both are multiples of 2^-24 and |th - k hi| < 2), and
// k mod 4 = k - 4 floor(k / 4) (exact in fp32) picks and signs the series
// values.  A non-finite th gives NaN.  The rare reduction sits in a branch, so
// a wave whose lanes all hold small angles skips it.
__device__ __forceinline__ void sincos_full(float th, float& s, float& c)
{
    const float quarter_pi = 0x1.921fb6p-1f;        // fp32(pi/4)
    if (__builtin_fabsf(th) <= quarter_pi) {
        sincos_series(th, s, c);
    } else {
        const float two_over_pi = 0x1.45f306p-1f;   // fp32(2/pi)
        const float half_pi_hi = 0x1.921fb6p+0f;    // fp32(pi/2)
        const float half_pi_lo = -0x1.777a5cp-25f;  // fp32(pi/2 - half_pi_hi)
        const float k = __builtin_rintf(th * two_over_pi);
        float r = __builtin_fmaf(-k, half_pi_hi, th);
        r = __builtin_fmaf(-k, half_pi_lo, r);
        const float quadrant = k - 4.0f * __builtin_floorf(k * 0.25f);
        float sr, cr;
        sincos_series(r, sr, cr);
        const bool odd = quadrant == 1.0f || quadrant == 3.0f;
        const float a = odd ? cr : sr, b = odd ? sr : cr;      // sin, cos up to sign
        s = (quadrant == 2.0f || quadrant == 3.0f) ? -a : a;
        c = (quadrant == 1.0f || quadrant == 2.0f) ? -b : b;
    }
}

// One explicit-Euler step of the frictionless cart with a uniform rod:
//   thacc = (g sin - cos * temp) / (l (4/3 - m cos^2 / M)),
//   temp  = (F + m l thd^2 sin) / M,   xacc = temp - (m l / M) thacc cos,
// positions advanced with the old velocities.  act 1 pushes towards +x.
struct CartState { float x, xd, th, thd; };

__device__ __forceinline__ CartState cartpole_step(const DevParams& p, const CartState& s, uint32_t act)
{
    const float force = act ? p.force_mag : -p.force_mag;
    float sn, cs;
    sincos_full(s.th, sn, cs);
    const float ml_thd2 = p.pole_ml * (s.thd * s.thd);
    const float temp = __builtin_fmaf(ml_thd2, sn, force) * p.inv_total;
    const float num = __builtin_fmaf(-cs, temp, p.gravity * sn);
    const float den = p.half_length * __builtin_fmaf(-p.m_over_M, cs * cs, 4.0f / 3.0f);
    const float thacc = num / den;                       // IEEE division
    const float xacc = __builtin_fmaf(-(p.ml_over_M * thacc), cs, temp);
    CartState o;
    o.x = __builtin_fmaf(p.tau, s.xd, s.x);
    o.xd = __builtin_fmaf(p.tau, xacc, s.xd);
    o.th = __builtin_fmaf(p.tau, s.thd, s.th);
    o.thd = __builtin_fmaf(p.tau, thacc, s.thd);
    return o;
}

// Strict thresholds; NaN compares false.  Disabled termination is encoded as
// infinite thresholds, under which every comparison is false.
// |v| > t is the same predicate as (v < -t or v > t) for every v and t,
// including signed zeros, infinities, NaN and negative t.
__device__ __forceinline__ bool crossed(const DevParams& p, const CartState& s)
{
    return (__builtin_fabsf(s.x) > p.thr_x) || (__builtin_fabsf(s.th) > p.thr_th);
}

// Byte offset addressing: base + 32-bit unsigned offset lets the compiler use a
// scalar base register plus a per-lane 32-bit offset (n_envs <= 2^30).
template <class T>
__device__ __forceinline__ T* at(T* base, uint32_t byte_off)
{
    return reinterpret_cast<T*>(reinterpret_cast<char*>(base) + byte_off);
}
template <class T>
__device__ __forceinline__ const T* at(const T* base, uint32_t byte_off)
{
    return reinterpret_cast<const T*>(reinterpret_cast<const char*>(base) + byte_off);
}

// Sum over the 64 lanes of a wave (every lane gets the total).
__device__ __forceinline__ uint32_t wave_sum(uint32_t v)
{
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += (uint32_t)__shfl_xor((int)v, off, 64);
    return v;
}

}  // namespace rlsim_dev
