// store_probe.hip -- the probe library of include/rlsim_probe.h.  Here the
// store-only probe: the fused kernel's trajectory stores (same planes, same
// per-lane offsets laundered through an empty asm, same scalar row bases, same
// workgroup mapping) with the simulation taken out.  The policy-math error
// probe is math_probe.hip.h, included at the end (one translation unit: the
// kernel headers define kernels).
#include <hip/hip_runtime.h>

#include "rlsim_probe.h"
#include "k_cartpole.hip.h"

namespace rlsim_dev {

__global__ __launch_bounds__(kBlock) void k_store_probe(uint32_t n, uint32_t K, float* obs, uint8_t* act,
                                                        float* rew, uint8_t* done)
{
    const uint32_t env = xcd_block() * kBlock + threadIdx.x;
    if (env >= n) return;
    const size_t plane = n;
    uint32_t off4 = env * 4u, off1a = env, off1d = env;
    float v = (float)(env & 0xFFFFu);
    uint32_t bits = env;
#pragma unroll 1
    for (uint32_t k = 0; k < K; ++k) {
        asm volatile("" : "+v"(off4), "+v"(off1a), "+v"(off1d));
        *at(obs, off4) = v;
        *at(obs + plane, off4) = v + 1.0f;
        *at(obs + 2 * plane, off4) = v + 2.0f;
        *at(obs + 3 * plane, off4) = v + 3.0f;
        *at(act, off1a) = (uint8_t)(bits & 1u);
        *at(rew, off4) = 1.0f;
        *at(done, off1d) = (uint8_t)((env ^ k) & 3u);
        v += 1.0f;
        bits += 1u;
        obs += 4 * plane;
        act += plane;
        rew += plane;
        done += plane;
    }
}

}  // namespace rlsim_dev

extern "C" int rlsim_probe_store(uint32_t n, uint32_t K, float* obs, uint8_t* action, float* reward, uint8_t* done,
                                 void* stream)
{
    if (n == 0u || n > (1u << 30) || K == 0u || K >= (1u << 23)) return -1;
    if (!obs || !action || !reward || !done) return -1;
    if (((uintptr_t)obs | (uintptr_t)reward) % 4u != 0u) return -1;
    const dim3 grid((n + rlsim_dev::kBlock - 1u) / rlsim_dev::kBlock), block(rlsim_dev::kBlock);
    hipLaunchKernelGGL(rlsim_dev::k_store_probe, grid, block, 0, (hipStream_t)stream, n, K, obs, action, reward, done);
    return hipGetLastError() == hipSuccess ? 0 : -3;
}

#include "math_probe.hip.h"
