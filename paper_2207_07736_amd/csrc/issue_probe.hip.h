// issue_probe.hip.h -- rlsim_probe_issue of include/rlsim_probe.h: the
// instruction rates the kernels' bounds rest on, measured on this device by
// kernels that do nothing else.  Each lane runs eight (MFMA: four)
// independent dependency chains of one instruction kind, so the time is set by
// issue throughput, not latency, once a SIMD holds enough waves.  Every chain
// ends in a value with a closed form, written out so that the work is kept and
// a test can check it.  Part of the probe library's single translation unit
// (store_probe.hip).
#pragma once

#include "rlsim_probe.h"
#include "k_cartpole.hip.h"

namespace rlsim_dev {

enum : uint32_t {
    ISSUE_FMA = 0,         // v_fma_f32 x <- x * 1 + 1           (x0 + iters)
    ISSUE_SELECT_FMA = 1,  // t <- u ? b : -0; s <- fma(a, s, t)  (the per-lane padding update)
    ISSUE_EXP = 2,         // v_exp_f32 x <- 2^-x                  (converges to x = 2^-x)
    ISSUE_RCP = 3,         // v_rcp_f32 x <- 1 / x                 (x0 after an even count)
    ISSUE_MFMA = 4,        // v_mfma_f32_32x32x2_f32 C += A B, A = B = 1 (2 iters per element)
    ISSUE_MIXED = 5,       // even waves of a workgroup run ISSUE_MFMA, odd waves ISSUE_FMA
    ISSUE_MUL = 6,         // v_mul_f32 x <- x * 1                 (x0)
    ISSUE_KINDS = 7
};

__device__ __forceinline__ float issue_fma(uint32_t iters, uint32_t lane)
{
    float x[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = (float)(lane + (uint32_t)j);
    const float one = 1.0f;
#pragma unroll 1
    for (uint32_t i = 0; i < iters; ++i) {
#pragma unroll
        for (int j = 0; j < 8; ++j) asm volatile("v_fma_f32 %0, %0, %1, %1" : "+v"(x[j]) : "v"(one));
    }
    float sum = 0.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j) sum += x[j];
    return sum;
}

__device__ __forceinline__ float issue_mul(uint32_t iters, uint32_t lane)
{
    float x[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = (float)(lane + (uint32_t)j);
    const float one = 1.0f;
#pragma unroll 1
    for (uint32_t i = 0; i < iters; ++i) {
#pragma unroll
        for (int j = 0; j < 8; ++j) asm volatile("v_mul_f32 %0, %0, %1" : "+v"(x[j]) : "v"(one));
    }
    float sum = 0.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j) sum += x[j];
    return sum;
}

__device__ __forceinline__ float issue_select_fma(uint32_t iters, uint32_t lane)
{
    float s[8], a[8], b[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        s[j] = (float)j;
        a[j] = 1.0f;
        b[j] = 1.0f;
        asm volatile("" : "+v"(a[j]), "+v"(b[j]));        // opaque: no folding into an add
    }
    const float mz = -0.0f;
#pragma unroll 1
    for (uint32_t i = 0; i < iters; ++i) {
        // this lane's action bit at step i, as the lane mask a select reads
        const uint64_t u = __builtin_amdgcn_ballot_w64(((lane + i) & 1u) != 0u);
        float t[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) asm volatile("v_cndmask_b32_e64 %0, %1, %2, %3" : "=v"(t[j]) : "v"(mz), "v"(b[j]), "s"(u));
#pragma unroll
        for (int j = 0; j < 8; ++j) asm volatile("v_fma_f32 %0, %1, %0, %2" : "+v"(s[j]) : "v"(a[j]), "v"(t[j]));
    }
    float sum = 0.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j) sum += s[j];
    return sum;
}

__device__ __forceinline__ float issue_exp(uint32_t iters, uint32_t lane)
{
    float x[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = 0.125f * (float)j + 0.001f * (float)(lane & 7u);
#pragma unroll 1
    for (uint32_t i = 0; i < iters; ++i) {
#pragma unroll
        for (int j = 0; j < 8; ++j) x[j] = __builtin_amdgcn_exp2f(-x[j]);
    }
    float sum = 0.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j) sum += x[j];
    return sum;
}

__device__ __forceinline__ float issue_rcp(uint32_t iters, uint32_t)
{
    float x[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = (float)(1u << j);
#pragma unroll 1
    for (uint32_t i = 0; i < iters; ++i) {
#pragma unroll
        for (int j = 0; j < 8; ++j) x[j] = __builtin_amdgcn_rcpf(x[j]);
    }
    float sum = 0.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j) sum += x[j];
    return sum;
}

typedef float issue_f16x __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float issue_mfma(uint32_t iters, uint32_t)
{
    issue_f16x c0 = {}, c1 = {}, c2 = {}, c3 = {};
    float a = 1.0f, b = 1.0f;
    asm volatile("" : "+v"(a), "+v"(b));
#pragma unroll 1
    for (uint32_t i = 0; i < iters; ++i) {
        c0 = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c0, 0, 0, 0);
        c1 = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c1, 0, 0, 0);
        c2 = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c2, 0, 0, 0);
        c3 = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c3, 0, 0, 0);
    }
    return c0[0] + c1[5] + c2[10] + c3[15];
}

// One kernel per kind, so that each gets only the registers its own chains
// need (the FMA kind fits eight waves per SIMD).  Mixed: wave w of workgroup
// b runs the MFMA chains when b + w is even and 16 times as many FMA
// iterations otherwise (about as long), so both kinds share every SIMD however
// the waves are placed.
template <uint32_t KIND>
__global__ __launch_bounds__(256) void k_issue_probe(uint32_t iters, float* out)
{
    const uint32_t lane = threadIdx.x % 64u, wave = threadIdx.x / 64u;
    float v;
    if (KIND == ISSUE_FMA) v = issue_fma(iters, lane);
    else if (KIND == ISSUE_SELECT_FMA) v = issue_select_fma(iters, lane);
    else if (KIND == ISSUE_EXP) v = issue_exp(iters, lane);
    else if (KIND == ISSUE_RCP) v = issue_rcp(iters, lane);
    else if (KIND == ISSUE_MFMA) v = issue_mfma(iters, lane);
    else if (KIND == ISSUE_MUL) v = issue_mul(iters, lane);
    else v = ((blockIdx.x + wave) & 1u) ? issue_fma(16u * iters, lane) : issue_mfma(iters, lane);
    out[(size_t)blockIdx.x * 256u + threadIdx.x] = v;
}

}  // namespace rlsim_dev

extern "C" int rlsim_probe_issue(uint32_t kind, uint32_t blocks, uint32_t iters, float* out, void* stream)
{
    if (kind >= rlsim_dev::ISSUE_KINDS || blocks == 0u || blocks > (1u << 20) || iters == 0u || iters > (1u << 22) ||
        (kind == rlsim_dev::ISSUE_MIXED && iters > (1u << 19)) || !out || (uintptr_t)out % 4u != 0u)
        return -1;
    const dim3 grid(blocks), block(256);
    hipStream_t s = (hipStream_t)stream;
    switch (kind) {
    case rlsim_dev::ISSUE_FMA: hipLaunchKernelGGL(rlsim_dev::k_issue_probe<rlsim_dev::ISSUE_FMA>, grid, block, 0, s, iters, out); break;
    case rlsim_dev::ISSUE_SELECT_FMA:
        hipLaunchKernelGGL(rlsim_dev::k_issue_probe<rlsim_dev::ISSUE_SELECT_FMA>, grid, block, 0, s, iters, out);
        break;
    case rlsim_dev::ISSUE_EXP: hipLaunchKernelGGL(rlsim_dev::k_issue_probe<rlsim_dev::ISSUE_EXP>, grid, block, 0, s, iters, out); break;
    case rlsim_dev::ISSUE_RCP: hipLaunchKernelGGL(rlsim_dev::k_issue_probe<rlsim_dev::ISSUE_RCP>, grid, block, 0, s, iters, out); break;
    case rlsim_dev::ISSUE_MFMA: hipLaunchKernelGGL(rlsim_dev::k_issue_probe<rlsim_dev::ISSUE_MFMA>, grid, block, 0, s, iters, out); break;
    case rlsim_dev::ISSUE_MUL: hipLaunchKernelGGL(rlsim_dev::k_issue_probe<rlsim_dev::ISSUE_MUL>, grid, block, 0, s, iters, out); break;
    default: hipLaunchKernelGGL(rlsim_dev::k_issue_probe<rlsim_dev::ISSUE_MIXED>, grid, block, 0, s, iters, out); break;
    }
    return hipGetLastError() == hipSuccess ? 0 : -3;
}
