// fill_probe.hip.h -- rlsim_probe_fill of include/rlsim_probe.h: plain fills
// of one contiguous buffer in different kernel shapes, from one float4 store
// per thread over a grid of many small workgroups to a long loop of stores per
// thread over a workgroup-contiguous chunk (the trajectory's per-workgroup
// volume is 256 x 275 float4).  Part of the probe library's single translation
// unit (store_probe.hip).
#pragma once

#include "rlsim_probe.h"

namespace rlsim_dev {

// Workgroup b writes float4 indices b 256 per + t + 256 j, j < per.
__global__ __launch_bounds__(256) void k_fill_probe(float4* p, uint64_t n4, uint32_t per)
{
    const uint64_t base = (uint64_t)blockIdx.x * per * 256u + threadIdx.x;
    for (uint32_t j = 0; j < per; ++j) {
        const uint64_t i = base + 256u * (uint64_t)j;
        if (i < n4) {
            const float v = (float)(uint32_t)(i & 0xFFFFFu);
            p[i] = float4{v, v + 1.0f, v + 2.0f, v + 3.0f};
        }
    }
}

}  // namespace rlsim_dev

extern "C" int rlsim_probe_fill(uint64_t n4, uint32_t per_thread, float* dst, void* stream)
{
    if (n4 == 0u || per_thread == 0u || per_thread > (1u << 20) || !dst || (uintptr_t)dst % 16u != 0u) return -1;
    const uint64_t per_block = 256u * (uint64_t)per_thread;
    const uint64_t blocks = (n4 + per_block - 1u) / per_block;
    if (blocks >= (1ull << 31)) return -1;
    hipLaunchKernelGGL(rlsim_dev::k_fill_probe, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream,
                       reinterpret_cast<float4*>(dst), n4, per_thread);
    return hipGetLastError() == hipSuccess ? 0 : -3;
}
