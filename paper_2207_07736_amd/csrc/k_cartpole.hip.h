// k_cartpole.hip.h -- the fused K-step simulator kernel, one thread per
// environment, random actions, up to W padding words held in registers.
#pragma once

#include "device_common.hip.h"

namespace rlsim_dev {

constexpr int kBlock = 256;          // threads per workgroup = envs per stats block

struct StepArgs {
    DevParams p;
    uint32_t n;          // environments
    uint32_t D;          // padding words (<= W of the instantiation)
    uint32_t t0;         // global step of row 0
    uint32_t K;          // steps in this launch
    float* cart;         // [4][n]   x, x_dot, theta, theta_dot
    uint32_t* ep;        // [n]      steps taken in the current episode
    float* pad_s;        // [D][n]   padding words
    const float* pad_a;  // [D][n]
    const float* pad_b;  // [D][n]
    float* obs;          // [K][4][n]
    uint8_t* action;     // [K][n]
    float* reward;       // [K][n]
    uint8_t* done;       // [K][n]
    uint32_t* stats;     // [ceil(n/256)][4]
};

// Words of the action block that holds step t: the 32 action bits of steps
// t & ~31 .. (t & ~31) + 31, least significant first.
__device__ __forceinline__ uint32_t pick_word(const uint4& w, uint32_t q)
{
    return q == 0u ? w.x : q == 1u ? w.y : q == 2u ? w.z : w.w;
}

// Fused K-step loop.  The state of one environment lives in registers for all
// K steps; per step the only device-memory traffic is the trajectory row
// (22 bytes).  RNG words are drawn once per block of steps: one Philox call per
// 128 steps for the actions, one per 4 steps for the reset draw that an episode
// ending in that block would start from.
template <int W, bool REC, bool STATS>
__global__ __launch_bounds__(kBlock) void k_cartpole_fused(StepArgs a)
{
    const uint32_t env = blockIdx.x * kBlock + threadIdx.x;
    const bool live = env < a.n;
    const DevParams& p = a.p;
    uint32_t n_eps = 0u, n_len = 0u, n_term = 0u, n_trunc = 0u;

    if (live) {
        const uint32_t off = env * 4u;              // byte offset of a f32 column (n <= 2^30)
        const size_t plane = a.n;                   // entries per f32 plane
        float* const c0 = a.cart;
        float* const c1 = a.cart + plane;
        float* const c2 = a.cart + 2 * plane;
        float* const c3 = a.cart + 3 * plane;
        CartState s;
        s.x = *at(c0, off);
        s.xd = *at(c1, off);
        s.th = *at(c2, off);
        s.thd = *at(c3, off);
        uint32_t ep = a.ep[env];

        float ps[W > 0 ? W : 1], pa[W > 0 ? W : 1], pb[W > 0 ? W : 1];
#pragma unroll
        for (int j = 0; j < W; ++j) {
            const bool on = (uint32_t)j < a.D;
            const size_t q = (size_t)j * a.n + env;
            ps[j] = on ? a.pad_s[q] : 0.0f;
            pa[j] = on ? a.pad_a[q] : 0.0f;
            pb[j] = on ? a.pad_b[q] : 0.0f;
        }

        uint32_t t = a.t0;
        uint4 aw = philox(env, t >> 7, STREAM_ACTION, p.key0, p.key1);
        uint32_t abits = pick_word(aw, (t >> 5) & 3u) >> (t & 31u);
        uint4 rw = philox(env, (t + 1u) >> 2, STREAM_RESET, p.key0, p.key1);
        CartState rs = {uniform01_to(rw.x, p.reset_lo, p.reset_width), uniform01_to(rw.y, p.reset_lo, p.reset_width),
                        uniform01_to(rw.z, p.reset_lo, p.reset_width), uniform01_to(rw.w, p.reset_lo, p.reset_width)};

        float* obs = a.obs;
        uint8_t* act_row = a.action;
        float* rew_row = a.reward;
        uint8_t* done_row = a.done;

        for (uint32_t k = 0; k < a.K; ++k, ++t) {
            if (k != 0u) {
                if ((t & 127u) == 0u) aw = philox(env, t >> 7, STREAM_ACTION, p.key0, p.key1);
                if ((t & 31u) == 0u) abits = pick_word(aw, (t >> 5) & 3u);
                if (((t + 1u) & 3u) == 0u) {
                    rw = philox(env, (t + 1u) >> 2, STREAM_RESET, p.key0, p.key1);
                    rs.x = uniform01_to(rw.x, p.reset_lo, p.reset_width);
                    rs.xd = uniform01_to(rw.y, p.reset_lo, p.reset_width);
                    rs.th = uniform01_to(rw.z, p.reset_lo, p.reset_width);
                    rs.thd = uniform01_to(rw.w, p.reset_lo, p.reset_width);
                }
            }
            const uint32_t act = abits & 1u;
            abits >>= 1;

            const CartState nx = cartpole_step(p, s, act);
#pragma unroll
            for (int j = 0; j < W; ++j) ps[j] = __builtin_fmaf(pa[j], ps[j], act ? pb[j] : 0.0f);

            const uint32_t len = ep + 1u;
            const uint32_t term = crossed(p, nx);
            const uint32_t trunc = (uint32_t)((p.max_steps != 0u) & (len >= p.max_steps));
            const uint32_t d = term | (trunc << 1);

            if (REC) {
                *at(obs, off) = s.x;
                *at(obs + plane, off) = s.xd;
                *at(obs + 2 * plane, off) = s.th;
                *at(obs + 3 * plane, off) = s.thd;
                act_row[env] = (uint8_t)act;
                *at(rew_row, off) = 1.0f;
                done_row[env] = (uint8_t)d;
                obs += 4 * plane;
                act_row += a.n;
                rew_row += a.n;
                done_row += a.n;
            }

            const bool reset = d != 0u;
            s.x = reset ? rs.x : nx.x;
            s.xd = reset ? rs.xd : nx.xd;
            s.th = reset ? rs.th : nx.th;
            s.thd = reset ? rs.thd : nx.thd;
            ep = reset ? 0u : len;
#pragma unroll
            for (int j = 0; j < W; ++j) ps[j] = reset ? 0.0f : ps[j];
            if (STATS) {
                n_eps += reset ? 1u : 0u;
                n_len += reset ? len : 0u;
                n_term += term;
                n_trunc += trunc;
            }
        }

        *at(c0, off) = s.x;
        *at(c1, off) = s.xd;
        *at(c2, off) = s.th;
        *at(c3, off) = s.thd;
        a.ep[env] = ep;
#pragma unroll
        for (int j = 0; j < W; ++j)
            if ((uint32_t)j < a.D) a.pad_s[(size_t)j * a.n + env] = ps[j];
    }

    if (STATS) {
        __shared__ uint32_t part[kBlock / 64][4];
        const uint32_t v0 = wave_sum(n_eps), v1 = wave_sum(n_len), v2 = wave_sum(n_term), v3 = wave_sum(n_trunc);
        const uint32_t wave = threadIdx.x / 64u, lane = threadIdx.x % 64u;
        if (lane == 0u) {
            part[wave][0] = v0;
            part[wave][1] = v1;
            part[wave][2] = v2;
            part[wave][3] = v3;
        }
        __syncthreads();
        if (threadIdx.x < 4u) {
            uint32_t sum = 0u;
#pragma unroll
            for (int w = 0; w < kBlock / 64; ++w) sum += part[w][threadIdx.x];
            a.stats[(size_t)blockIdx.x * 4u + threadIdx.x] = sum;
        }
    }
}

// Initial state of every environment (episode beginning at step 0) and the
// padding parameters, for the register (structure-of-arrays) padding layout.
__global__ __launch_bounds__(kBlock) void k_reset_cart(DevParams p, uint32_t n, float* cart, uint32_t* ep)
{
    const uint32_t env = blockIdx.x * kBlock + threadIdx.x;
    if (env >= n) return;
    const uint4 w = philox(env, 0u, STREAM_RESET, p.key0, p.key1);
    const size_t plane = n;
    cart[env] = uniform01_to(w.x, p.reset_lo, p.reset_width);
    cart[plane + env] = uniform01_to(w.y, p.reset_lo, p.reset_width);
    cart[2 * plane + env] = uniform01_to(w.z, p.reset_lo, p.reset_width);
    cart[3 * plane + env] = uniform01_to(w.w, p.reset_lo, p.reset_width);
    ep[env] = 0u;
}

// Padding word j of env e lives at s[j * stride_j + e * stride_e]; one thread
// per (word, env) pair, grid-strided over all D * n pairs.
__global__ __launch_bounds__(kBlock) void k_reset_pad(DevParams p, uint32_t n, uint32_t D, size_t stride_j,
                                                      size_t stride_e, float a_lo, float a_width, float b_lo,
                                                      float b_width, float* s, float* pa, float* pb)
{
    const size_t total = (size_t)n * D;
    for (size_t i = (size_t)blockIdx.x * kBlock + threadIdx.x; i < total; i += (size_t)gridDim.x * kBlock) {
        // env-fastest enumeration keeps both layouts' writes mostly contiguous
        const uint32_t env = (uint32_t)(stride_e == 1 ? i % n : i / D);
        const uint32_t j = (uint32_t)(stride_e == 1 ? i / n : i % D);
        const uint4 w = philox(env, j, STREAM_PARAMS, p.key0, p.key1);
        const size_t q = (size_t)j * stride_j + (size_t)env * stride_e;
        pa[q] = uniform01_to(w.x, a_lo, a_width);
        pb[q] = uniform01_to(w.y, b_lo, b_width);
        s[q] = 0.0f;
    }
}

}  // namespace rlsim_dev
