// math_probe.hip.h -- rlsim_probe_policy_math of include/rlsim_probe.h: the
// policy kernel's elementwise functions (tanh_fast, policy_p0, log_pi, the very
// device functions the kernel calls) evaluated at every fp32 value of a bit
// range and compared with double-precision evaluations of their definitions.
// Part of the probe library's single translation unit (store_probe.hip).
#pragma once

#include "rlsim_probe.h"
#include "k_policy.hip.h"

namespace rlsim_dev {

constexpr uint32_t kMathPerThread = 256;

__device__ __forceinline__ double ref_log_pi(double d, uint32_t act)
{
    const double z = act ? -d : d;            // log pi(a) = -softplus(l_other - l_a)
    return -(fmax(z, 0.0) + log1p(exp(-fabs(z))));
}

__device__ __forceinline__ float wave_max(float v)
{
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m, 64));
    return v;
}

__global__ __launch_bounds__(256) void k_math_probe(uint32_t lo, uint64_t count, uint32_t* out)
{
    float e_tanh = 0.0f, e_p0 = 0.0f, e_lp = 0.0f;
    const uint64_t first = ((uint64_t)blockIdx.x * 256u + threadIdx.x) * kMathPerThread;
    for (uint32_t j = 0; j < kMathPerThread; ++j) {
        const uint64_t i = first + j;
        if (i >= count) break;
        const float x = __uint_as_float((uint32_t)(lo + i));
        if (!__builtin_isfinite(x)) continue;
        const double xd = (double)x;
        e_tanh = fmaxf(e_tanh, __double2float_ru(fabs((double)tanh_fast(x) - tanh(xd))));
        e_p0 = fmaxf(e_p0, __double2float_ru(fabs((double)policy_p0(x) - 1.0 / (1.0 + exp(xd)))));
        for (uint32_t a = 0; a < 2u; ++a) {
            const double r = ref_log_pi(xd, a);
            e_lp = fmaxf(e_lp, __double2float_ru(fabs((double)log_pi(x, a) - r) / (1.0 + fabs(r))));
        }
    }
    e_tanh = wave_max(e_tanh);
    e_p0 = wave_max(e_p0);
    e_lp = wave_max(e_lp);
    if ((threadIdx.x & 63u) == 0u) {
        // non-negative floats order as their bit patterns
        atomicMax(out + 0, __float_as_uint(e_tanh));
        atomicMax(out + 1, __float_as_uint(e_p0));
        atomicMax(out + 2, __float_as_uint(e_lp));
    }
}

}  // namespace rlsim_dev

extern "C" int rlsim_probe_policy_math(uint32_t lo_bits, uint64_t count, uint32_t* out_max, void* stream)
{
    if (count == 0u || (uint64_t)lo_bits + count > (1ull << 32) || !out_max || (uintptr_t)out_max % 4u != 0u)
        return -1;
    const uint64_t per_block = 256ull * rlsim_dev::kMathPerThread;
    const dim3 grid((uint32_t)((count + per_block - 1u) / per_block)), block(256);
    hipLaunchKernelGGL(rlsim_dev::k_math_probe, grid, block, 0, (hipStream_t)stream, lo_bits, count, out_max);
    return hipGetLastError() == hipSuccess ? 0 : -3;
}
