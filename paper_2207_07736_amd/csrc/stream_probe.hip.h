// stream_probe.hip.h -- rlsim_probe_stream of include/rlsim_probe.h: a plain
// float4 stream with the traffic mix of one unfused step of the wide padding
// state (read s, a and b, write s: 12 bytes read and 4 written per word), the
// ceiling that the K = 1 wide launches are compared with.  Part of the probe
// library's single translation unit (store_probe.hip).
#pragma once

#include "rlsim_probe.h"

namespace rlsim_dev {

__global__ __launch_bounds__(256) void k_stream_probe(float4* s, const float4* a, const float4* b, uint64_t n4)
{
    const uint64_t stride = (uint64_t)gridDim.x * 256u;
    for (uint64_t i = (uint64_t)blockIdx.x * 256u + threadIdx.x; i < n4; i += stride) {
        float4 x = s[i];
        const float4 p = a[i], q = b[i];
        x.x = __builtin_fmaf(p.x, x.x, q.x);
        x.y = __builtin_fmaf(p.y, x.y, q.y);
        x.z = __builtin_fmaf(p.z, x.z, q.z);
        x.w = __builtin_fmaf(p.w, x.w, q.w);
        s[i] = x;
    }
}

}  // namespace rlsim_dev

extern "C" int rlsim_probe_stream(uint64_t n4, float* s, const float* a, const float* b, void* stream)
{
    if (n4 == 0u || !s || !a || !b) return -1;
    if (((uintptr_t)s | (uintptr_t)a | (uintptr_t)b) % 16u != 0u) return -1;
    const uint64_t blocks = (n4 + 255u) / 256u;
    const dim3 grid((unsigned)(blocks < 65536u ? blocks : 65536u)), block(256);
    hipLaunchKernelGGL(rlsim_dev::k_stream_probe, grid, block, 0, (hipStream_t)stream, reinterpret_cast<float4*>(s),
                       reinterpret_cast<const float4*>(a), reinterpret_cast<const float4*>(b), n4);
    return hipGetLastError() == hipSuccess ? 0 : -3;
}
