// store_probe.hip -- the probe library of include/rlsim_probe.h.  Here the
// store-only probe: the trajectory bytes of the fused kernel (same planes,
// scalar row bases with per-lane offsets, same workgroup mapping) with the
// simulation taken out.  Each step's seven stores issue back to back, byte
// planes first: of the orders measured for these planes this one writes
// fastest (about 6 % faster than the same stores with other instructions
// between them), so the probe's time is the ceiling for the layout.  The
// policy-math error probe (math_probe.hip.h), the read/write stream probe
// (stream_probe.hip.h) and the instruction-rate probes (issue_probe.hip.h) are
// included at the end (one translation unit: the kernel headers define
// kernels).
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
    const uint32_t off4 = env * 4u, off1 = env;
    float v = (float)(env & 0xFFFFu);
    uint32_t bits = env;
#pragma unroll 1
    for (uint32_t k = 0; k < K; ++k) {
        const float v1 = v + 1.0f, v2 = v + 2.0f, v3 = v + 3.0f;
        const uint8_t a = (uint8_t)(bits & 1u), d = (uint8_t)((env ^ k) & 3u);
        float* o1 = obs + plane;
        float* o2 = obs + 2 * plane;
        float* o3 = obs + 3 * plane;
        *at(act, off1) = a;
        *at(done, off1) = d;
        *at(obs, off4) = v;
        *at(o1, off4) = v1;
        *at(o2, off4) = v2;
        *at(o3, off4) = v3;
        *at(rew, off4) = 1.0f;
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

#include "fill_probe.hip.h"
#include "issue_probe.hip.h"
#include "math_probe.hip.h"
#include "stream_probe.hip.h"
