// issue_probe.hip.h -- rlsim_probe_issue of include/rlsim_probe.h: the
// instruction rates the kernels' bounds rest on, measured on this device by
// kernels that do nothing else.  Each lane runs eight (MFMA: four)
// independent dependency chains of one instruction kind, so the time is set by
// issue throughput, not latency, once a SIMD holds enough waves.  Every chain
// ends in a value with a closed form, written out so that the work is kept and
// a test can check it.  Thread 0 of each workgroup can also record the shader
// clock cycles and real-time ticks its chains took, so that a rate can be put
// per clock: the shader clock of these parts follows their power draw, which
// depends on how many bits the data toggles, not only on the instructions.
// Part of the probe library's single translation unit (store_probe.hip).
#pragma once

#include "rlsim_probe.h"
#include "k_wide.hip.h"

namespace rlsim_dev {

enum : uint32_t {
    ISSUE_FMA = 0,         // v_fma_f32 x <- x * 1 + 1, the two 1s in two registers  (x0 + iters)
    ISSUE_SELECT_FMA = 1,  // t <- u ? b : -0; s <- fma(a, s, t)  (the per-lane padding update)
    ISSUE_EXP = 2,         // v_exp_f32 x <- 2^-x                  (converges to x = 2^-x)
    ISSUE_RCP = 3,         // v_rcp_f32 x <- 1 / x                 (x0 after an even count)
    ISSUE_MFMA = 4,        // v_mfma_f32_32x32x2_f32 C += A B, A = B = 1 (2 iters per element)
    ISSUE_MIXED = 5,       // even waves of a workgroup run ISSUE_MFMA, odd waves ISSUE_FMA
    ISSUE_MUL = 6,         // v_mul_f32 x <- x * 1                 (x0)
    ISSUE_FMA_SHARED = 7,  // ISSUE_FMA with both 1s read from one register
    ISSUE_REPLAY_TREE = 8, // the wide kernel's two-environment replay, 8 words each, per 32-step bit word
    ISSUE_REPLAY_FLAT = 9, // the same updates per step with no decisions (a fixed FMA / multiply pattern)
    ISSUE_KINDS = 10
};

__device__ __forceinline__ float issue_fma(uint32_t iters, uint32_t lane)
{
    float x[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = (float)(lane + (uint32_t)j);
    float one = 1.0f, one2 = 1.0f;
    asm volatile("" : "+v"(one), "+v"(one2));            // two registers holding 1
#pragma unroll 1
    for (uint32_t i = 0; i < iters; ++i) {
#pragma unroll
        for (int j = 0; j < 8; ++j) asm volatile("v_fma_f32 %0, %0, %1, %2" : "+v"(x[j]) : "v"(one), "v"(one2));
    }
    float sum = 0.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j) sum += x[j];
    return sum;
}

// The same chains with one register read twice: gfx950 issues this form at
// about half the rate of the one above.
__device__ __forceinline__ float issue_fma_shared(uint32_t iters, uint32_t lane)
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

// Bits of one 32-step word of the replay kinds: environment e's action word
// u[e] and done word d[e] from a hash of (k, e), about one done bit per 22
// steps per environment, like cart-pole episodes under random actions.
__device__ __forceinline__ uint32_t issue_hash(uint32_t x)
{
    x ^= x >> 16;
    x *= 0x7feb352du;
    x ^= x >> 15;
    x *= 0x846ca68bu;
    x ^= x >> 16;
    return x;
}

__device__ __forceinline__ void issue_replay_bits(uint32_t k, uint32_t (&u)[4], uint32_t (&d)[4])
{
    u[0] = issue_hash(4u * k);
    u[1] = issue_hash(4u * k + 1u);
    const uint32_t h = issue_hash(4u * k + 2u);
    d[0] = (1u << (h & 31u)) | ((h >> 5) % 3u == 0u ? 1u << ((h >> 8) & 31u) : 0u);
    d[1] = (1u << ((h >> 13) & 31u)) | ((h >> 18) % 3u == 0u ? 1u << ((h >> 21) & 31u) : 0u);
    u[2] = u[3] = d[2] = d[3] = 0u;
}

// The wide kernel's replay of two environments with 8 words per lane each
// (replay_multi<2, 8>: per step a two-level tree of scalar bit tests, then 16
// in-place updates), over `iters` bit words; a = b = 1, so each word ends as
// the number of action-1 steps since the environment's last done bit.
__device__ __forceinline__ float issue_replay_tree(uint32_t iters, uint32_t gwave)
{
    float s0[8], s1[8], s2[8], s3[8], a0[8], a1[8], b0[8], b1[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        s0[j] = s1[j] = s2[j] = s3[j] = 0.0f;
        a0[j] = a1[j] = b0[j] = b1[j] = 1.0f;
        asm volatile("" : "+v"(a0[j]), "+v"(a1[j]), "+v"(b0[j]), "+v"(b1[j]));   // each its own register
    }
#pragma unroll 1
    for (uint32_t w = 0; w < iters; ++w) {
        uint32_t u[4], d[4];
        issue_replay_bits(gwave * iters + w, u, d);
        replay_multi<2, 8>(s0, s1, s2, s3, a0, a1, a0, a1, b0, b1, b0, b1, u, d, 32u);
    }
    float sum = 0.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j) sum += s0[j] + s1[j];
    return sum;
}

// The same 16 updates per step with no decisions: 32 steps per word in a fixed
// pattern, each step one environment's 8 FMAs and the other's 8 multiplies
// (environment 0 takes the FMA at steps 0, 3, 4, 5 of every 8).  a = b = 1:
// both environments' words end at 16 iters.
#define ISSUE_FM RM_LEAF2(RM_R8, 1, 0)
#define ISSUE_MF RM_LEAF2(RM_R8, 0, 1)
#define ISSUE_FLAT8 ISSUE_FM ISSUE_MF ISSUE_MF ISSUE_FM ISSUE_FM ISSUE_FM ISSUE_MF ISSUE_MF
__device__ __forceinline__ float issue_replay_flat(uint32_t iters)
{
    float s0[8], s1[8], a0[8], a1[8], b0[8], b1[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        s0[j] = s1[j] = 0.0f;
        a0[j] = a1[j] = b0[j] = b1[j] = 1.0f;
        asm volatile("" : "+v"(a0[j]), "+v"(a1[j]), "+v"(b0[j]), "+v"(b1[j]));
    }
#pragma unroll 1
    for (uint32_t w = 0; w < iters; ++w) {
        uint32_t unused;
        asm volatile(ISSUE_FLAT8 ISSUE_FLAT8 ISSUE_FLAT8 ISSUE_FLAT8
                     : RM_R8(RM_OUT_S, 0) RM_R8(RM_OUT_S, 1)[unused] "=s"(unused)
                     : RM_R8(RM_IN_A, 0) RM_R8(RM_IN_A, 1) RM_R8(RM_IN_B, 0) RM_R8(RM_IN_B, 1)[w] "s"(w));
    }
    float sum = 0.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j) sum += s0[j] + s1[j];
    return sum;
}
#undef ISSUE_FLAT8
#undef ISSUE_MF
#undef ISSUE_FM

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
__global__ __launch_bounds__(256) void k_issue_probe(uint32_t iters, float* out, uint64_t* clocks)
{
    const uint32_t lane = threadIdx.x % 64u, wave = threadIdx.x / 64u;
    const uint64_t c0 = __builtin_amdgcn_s_memtime(), r0 = __builtin_amdgcn_s_memrealtime();
    float v;
    if (KIND == ISSUE_FMA) v = issue_fma(iters, lane);
    else if (KIND == ISSUE_FMA_SHARED) v = issue_fma_shared(iters, lane);
    else if (KIND == ISSUE_REPLAY_TREE) v = issue_replay_tree(iters, __builtin_amdgcn_readfirstlane(blockIdx.x * 4u + wave));
    else if (KIND == ISSUE_REPLAY_FLAT) v = issue_replay_flat(iters);
    else if (KIND == ISSUE_SELECT_FMA) v = issue_select_fma(iters, lane);
    else if (KIND == ISSUE_EXP) v = issue_exp(iters, lane);
    else if (KIND == ISSUE_RCP) v = issue_rcp(iters, lane);
    else if (KIND == ISSUE_MFMA) v = issue_mfma(iters, lane);
    else if (KIND == ISSUE_MUL) v = issue_mul(iters, lane);
    else v = ((blockIdx.x + wave) & 1u) ? issue_fma(16u * iters, lane) : issue_mfma(iters, lane);
    out[(size_t)blockIdx.x * 256u + threadIdx.x] = v;
    if (clocks && threadIdx.x == 0u) {
        const uint64_t c1 = __builtin_amdgcn_s_memtime(), r1 = __builtin_amdgcn_s_memrealtime();
        clocks[2u * blockIdx.x] = c1 - c0;
        clocks[2u * blockIdx.x + 1u] = r1 - r0;
    }
}

}  // namespace rlsim_dev

namespace rlsim_dev {
template <uint32_t KIND>
void launch_issue_probe(uint32_t blocks, uint32_t iters, float* out, uint64_t* clocks, hipStream_t s)
{
    hipLaunchKernelGGL(k_issue_probe<KIND>, dim3(blocks), dim3(256), 0, s, iters, out, clocks);
}
}  // namespace rlsim_dev

extern "C" int rlsim_probe_issue(uint32_t kind, uint32_t blocks, uint32_t iters, float* out, uint64_t* clocks,
                                 void* stream)
{
    using namespace rlsim_dev;
    if (kind >= ISSUE_KINDS || blocks == 0u || blocks > (1u << 20) || iters == 0u || iters > (1u << 22) ||
        (kind == ISSUE_MIXED && iters > (1u << 19)) ||
        ((kind == ISSUE_REPLAY_TREE || kind == ISSUE_REPLAY_FLAT) && iters > (1u << 16)) || !out ||
        (uintptr_t)out % 4u != 0u || (uintptr_t)clocks % 8u != 0u)
        return -1;
    hipStream_t s = (hipStream_t)stream;
    switch (kind) {
    case ISSUE_FMA: launch_issue_probe<ISSUE_FMA>(blocks, iters, out, clocks, s); break;
    case ISSUE_SELECT_FMA: launch_issue_probe<ISSUE_SELECT_FMA>(blocks, iters, out, clocks, s); break;
    case ISSUE_EXP: launch_issue_probe<ISSUE_EXP>(blocks, iters, out, clocks, s); break;
    case ISSUE_RCP: launch_issue_probe<ISSUE_RCP>(blocks, iters, out, clocks, s); break;
    case ISSUE_MFMA: launch_issue_probe<ISSUE_MFMA>(blocks, iters, out, clocks, s); break;
    case ISSUE_MIXED: launch_issue_probe<ISSUE_MIXED>(blocks, iters, out, clocks, s); break;
    case ISSUE_MUL: launch_issue_probe<ISSUE_MUL>(blocks, iters, out, clocks, s); break;
    case ISSUE_FMA_SHARED: launch_issue_probe<ISSUE_FMA_SHARED>(blocks, iters, out, clocks, s); break;
    case ISSUE_REPLAY_TREE: launch_issue_probe<ISSUE_REPLAY_TREE>(blocks, iters, out, clocks, s); break;
    default: launch_issue_probe<ISSUE_REPLAY_FLAT>(blocks, iters, out, clocks, s); break;
    }
    return hipGetLastError() == hipSuccess ? 0 : -3;
}

extern "C" int rlsim_probe_wall_clock_khz(uint32_t* khz)
{
    if (!khz) return -1;
    int dev = 0, rate = 0;
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&rate, hipDeviceAttributeWallClockRate, dev) != hipSuccess ||
        rate <= 0)
        return -3;
    *khz = (uint32_t)rate;
    return 0;
}
