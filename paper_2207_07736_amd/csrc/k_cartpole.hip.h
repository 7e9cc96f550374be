// k_cartpole.hip.h -- fused K-step simulator kernels with random actions.
//
//  k_cartpole_fused<W>: one thread per environment; the cart-pole state and up
//      to W padding words stay in registers for all K steps.
//  k_cartpole_split<W>: the same steps for up to W padding words with a
//      trajectory, with the stepping and the trajectory stores in separate
//      waves of a workgroup.
//  CartCore: the per-environment step loop every fused kernel shares (the
//      wide-padding kernel in k_wide.hip.h and the policy kernel included).
//  k_reset_cart, k_reset_pad: initial state and padding parameters.
#pragma once

#include "device_common.hip.h"

namespace rlsim_dev {

constexpr int kBlock = 256;          // threads per workgroup = envs per stats block

struct StepArgs {
    DevParams p;
    uint32_t n;          // environments
    uint32_t D;          // padding words
    uint32_t Dp;         // padded row length of the wide layout (multiple of 4)
    uint32_t t0;         // global step of row 0
    uint32_t K;          // steps in this launch
    float* cart;         // [4][n]   x, x_dot, theta, theta_dot
    uint32_t* ep;        // [n]      steps taken in the current episode
    float* pad_s;        // narrow: [D][n]; wide: [n][Dp]
    const float* pad_a;
    const float* pad_b;
    float* obs;          // [K][4][n]
    uint8_t* action;     // [K][n]
    float* reward;       // [K][n]
    uint8_t* done;       // [K][n]
    uint32_t* stats;     // [ceil(n/256)][4]
};

// The word of an action block that holds the 32 action bits of steps
// 32q .. 32q+31 (least significant bit first).
__device__ __forceinline__ uint32_t pick_word(const uint4& w, uint32_t q)
{
    return q == 0u ? w.x : q == 1u ? w.y : q == 2u ? w.z : w.w;
}

// Workgroups are dispatched to the 8 XCDs round-robin (hardware block b runs
// on XCD b mod 8).  This bijection hands XCD x the contiguous logical blocks
// [x per, (x+1) per), so each XCD's L2 and TLB see one contiguous slice of
// every trajectory row instead of a 1-in-8 comb across all of it.
__device__ __forceinline__ uint32_t xcd_block()
{
    const uint32_t nb = gridDim.x, b = blockIdx.x, per = nb / 8u;
    return b < per * 8u ? (b % 8u) * per + b / 8u : b;
}

// One environment's cart-pole state and RNG words, advanced step by step.
template <bool REC, bool STATS>
struct CartCore {
    const DevParams& p;
    uint32_t env;        // environment index within the handle
    uint32_t gid;        // global environment id: the RNG counters' first word
    CartState s;
    uint32_t ep;
    uint4 aw;            // action words of the current 128-step block
    uint32_t abits;      // remaining action bits of the current 32-step word
    CartState rs;        // reset draw for an episode beginning in the current 8-step block
    float* obs;          // trajectory row pointers (wave-uniform)
    uint8_t* act_row;
    float* rew_row;
    uint8_t* done_row;
    size_t plane;
    uint32_t ep_start = 0u;   // episode counter when the launch began
    uint32_t off4, off1a, off1d;   // per-lane byte offsets of this env in a row
    uint32_t n_eps = 0u, n_term = 0u, n_trunc = 0u;

    __device__ __forceinline__ CartCore(const DevParams& p_, uint32_t env_)
        : p(p_), env(env_), gid(env_ + p_.env0), off4(env_ * 4u), off1a(env_), off1d(env_) {}

    // Sum of the lengths of the episodes that ended in this launch: every step
    // adds one to the running episode, so the finished lengths plus the final
    // running length equal the starting length plus K (mod 2^32).
    __device__ __forceinline__ uint32_t finished_length_sum(uint32_t K) const { return ep_start + K - ep; }

    __device__ __forceinline__ void draw_reset(uint32_t block)
    {
        const uint4 w = philox(gid, block, STREAM_RESET, p.key0, p.key1);
        rs.x = uniform24_to(w.x, p.reset_lo, p.reset_width_u24);
        rs.xd = uniform24_to(w.y, p.reset_lo, p.reset_width_u24);
        rs.th = uniform24_to(w.z, p.reset_lo, p.reset_width_u24);
        rs.thd = uniform24_to(w.w, p.reset_lo, p.reset_width_u24);
    }

    // Called before the step at t when t is a multiple of 32.
    __device__ __forceinline__ void refresh_actions(uint32_t t)
    {
        if ((t & 127u) == 0u) aw = philox(gid, t >> 7, STREAM_ACTION, p.key0, p.key1);
        abits = pick_word(aw, (t >> 5) & 3u);
    }

    // Step t with the random action of the current action word.
    template <class Hook>
    __device__ __forceinline__ void step(Hook& hook)
    {
        const uint32_t act = abits & 1u;
        abits >>= 1;
        step_with(act, hook);
        if (REC) advance_rows();
    }

    __device__ __forceinline__ void advance_rows()
    {
        obs += 4 * plane;
        act_row += plane;
        rew_row += plane;
        done_row += plane;
    }

    // One step with the given action: record the row, Euler-step, terminate /
    // truncate, auto-reset.  hook.record(obs, act, done byte) sees the row this
    // step records and hook(act, reset) the action and whether the episode
    // ended.  The row pointers are left for the caller to advance.
    template <class Hook>
    __device__ __forceinline__ void step_with(uint32_t act, Hook& hook)
    {
        CartState nx = cartpole_step(p, s, act);
        // compute factor C > 1: the remaining Euler iterations of the step
        for (uint32_t c = 1; c < p.iters; ++c) nx = cartpole_step(p, nx, act);
        const uint32_t len = ep + 1u;
        const bool term = crossed(p, nx);
        const bool trunc = (p.max_steps != 0u) && (len >= p.max_steps);
        const uint32_t d = (trunc ? 2u : 0u) + (uint32_t)term;
        if (REC) {
            // the offsets are passed through an empty asm in place each step.
            // Byte planes first: about 1.5 % faster than obs first.  (Forcing
            // all seven stores back to back, the probe's fastest order, is
            // about 11 % slower here, with the step's arithmetic around them.)
            asm volatile("" : "+v"(off4), "+v"(off1a), "+v"(off1d));
            *at(act_row, off1a) = (uint8_t)act;
            *at(done_row, off1d) = (uint8_t)d;
            *at(obs, off4) = s.x;
            *at(obs + plane, off4) = s.xd;
            *at(obs + 2 * plane, off4) = s.th;
            *at(obs + 3 * plane, off4) = s.thd;
            *at(rew_row, off4) = 1.0f;
        }
        hook.record(s, act, d);
        const bool reset = term || trunc;
        s.x = reset ? rs.x : nx.x;
        s.xd = reset ? rs.xd : nx.xd;
        s.th = reset ? rs.th : nx.th;
        s.thd = reset ? rs.thd : nx.thd;
        ep = reset ? 0u : len;
        hook(act, reset);
        if (STATS) {
            n_eps += reset ? 1u : 0u;
            n_term += term ? 1u : 0u;
            n_trunc += trunc ? 1u : 0u;
        }
    }

    // Steps t0 .. t0+K-1.  The loop body covers the eight steps that share one
    // reset block ((t+1)/8 constant), so each reset draw is computed once, at a
    // fixed place, and the body has no data-dependent control flow.  A 32-step
    // action word can only begin at the second step of a body (t+1 = 0 mod 8).
    template <class Hook>
    __device__ __forceinline__ void run(uint32_t t0, uint32_t K, Hook& hook)
    {
        uint32_t t = t0, k = 0;
        aw = philox(gid, t >> 7, STREAM_ACTION, p.key0, p.key1);
        abits = pick_word(aw, (t >> 5) & 3u) >> (t & 31u);
        if (((t + 1u) & 7u) != 0u) {
            // up to seven steps before the first block boundary; none of them
            // but the first can start an action word (they are not multiples of 8)
            draw_reset((t + 1u) >> 3);
            while (k < K && ((t + 1u) & 7u) != 0u) {
                step(hook);
                ++t;
                ++k;
            }
        }
        // here t = 8m - 1: steps t .. t+7 draw resets from block m
        for (; K - k >= 8u; k += 8u, t += 8u) {
            draw_reset((t + 1u) >> 3);
            step(hook);
            if (((t + 1u) & 31u) == 0u) refresh_actions(t + 1u);
            // a rolled loop: row pointers advance by one scalar add per step
            // instead of eight precomputed per-step bases
#pragma unroll 1
            for (int i = 0; i < 7; ++i) step(hook);
        }
        if (k < K) {
            draw_reset((t + 1u) >> 3);
            step(hook);
            ++t;
            ++k;
            if (k < K && (t & 31u) == 0u) refresh_actions(t);
            for (; k < K; ++k) step(hook);
        }
    }

    __device__ __forceinline__ void set_rows(const StepArgs& a, uint32_t k0)
    {
        plane = a.n;
        obs = a.obs + (size_t)k0 * 4 * plane;
        act_row = a.action + (size_t)k0 * plane;
        rew_row = a.reward + (size_t)k0 * plane;
        done_row = a.done + (size_t)k0 * plane;
    }

    __device__ __forceinline__ void load(const StepArgs& a)
    {
        const size_t pl = a.n;
        s.x = a.cart[env];
        s.xd = a.cart[pl + env];
        s.th = a.cart[2 * pl + env];
        s.thd = a.cart[3 * pl + env];
        ep = a.ep[env];
        ep_start = ep;
    }

    __device__ __forceinline__ void store(const StepArgs& a)
    {
        const size_t pl = a.n;
        a.cart[env] = s.x;
        a.cart[pl + env] = s.xd;
        a.cart[2 * pl + env] = s.th;
        a.cart[3 * pl + env] = s.thd;
        a.ep[env] = ep;
    }
};

// Sums the four episode counters over a workgroup of kThreads threads and
// writes one row of the block statistics (all threads of the block must call
// this).
template <uint32_t kThreads = kBlock>
__device__ __forceinline__ void store_block_stats(uint32_t* stats, uint32_t blk, uint32_t c0, uint32_t c1, uint32_t c2,
                                                  uint32_t c3)
{
    __shared__ uint32_t part[kThreads / 64][4];
    const uint32_t v0 = wave_sum(c0), v1 = wave_sum(c1), v2 = wave_sum(c2), v3 = wave_sum(c3);
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
        for (int w = 0; w < (int)(kThreads / 64); ++w) sum += part[w][threadIdx.x];
        stats[(size_t)blk * 4u + threadIdx.x] = sum;
    }
}

// One padding word, s <- a s + b u rounded once: fma(a, s, b) when u = 1 and
// the product a s when u = 0.  fma(a, s, -0) equals the product bit for bit
// (x + -0 = x for every x, including both zeros), so a per-lane action costs
// one select and one FMA per word.
__device__ __forceinline__ float pad_update(float a, float s, float b, bool u)
{
    return __builtin_fmaf(a, s, u ? b : -0.0f);
}

struct NoPad {
    __device__ __forceinline__ void record(const CartState&, uint32_t, uint32_t) {}
    __device__ __forceinline__ void operator()(uint32_t, bool) {}
};

// Padding words held by one thread; zeroed when the episode ends.
template <int W>
struct RegisterPad {
    float s[W > 0 ? W : 1], a[W > 0 ? W : 1], b[W > 0 ? W : 1];
    __device__ __forceinline__ void record(const CartState&, uint32_t, uint32_t) {}
    __device__ __forceinline__ void operator()(uint32_t act, bool reset)
    {
#pragma unroll
        for (int j = 0; j < W; ++j) {
            const float v = pad_update(a[j], s[j], b[j], act != 0u);
            s[j] = reset ? 0.0f : v;
        }
    }
};

// Without padding words the kernel fits eight waves per SIMD (<= 64 VGPRs and
// <= 96 SGPRs); asking for it keeps the register allocator inside that budget.
template <int W, bool REC, bool STATS>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(W == 0 ? 8 : 1)))
void k_cartpole_fused(StepArgs a)
{
    const uint32_t blk = xcd_block();
    const uint32_t env = blk * kBlock + threadIdx.x;
    CartCore<REC, STATS> core(a.p, env);
    if (env < a.n) {
        core.load(a);
        if (REC) core.set_rows(a, 0);
        RegisterPad<W> pad;
#pragma unroll
        for (int j = 0; j < W; ++j) {
            const bool on = (uint32_t)j < a.D;
            const size_t q = (size_t)j * a.n + env;
            pad.s[j] = on ? a.pad_s[q] : 0.0f;
            pad.a[j] = on ? a.pad_a[q] : 0.0f;
            pad.b[j] = on ? a.pad_b[q] : 0.0f;
        }
        core.run(a.t0, a.K, pad);
        core.store(a);
#pragma unroll
        for (int j = 0; j < W; ++j)
            if ((uint32_t)j < a.D) a.pad_s[(size_t)j * a.n + env] = pad.s[j];
    }
    if (STATS) {
        const uint32_t len_sum = env < a.n ? core.finished_length_sum(a.K) : 0u;
        store_block_stats(a.stats, blk, core.n_eps, len_sum, core.n_term, core.n_trunc);
    }
}

// ---------------------------------------------------------------------------
// Warp-specialised stepping for up to W padding words with a trajectory.
// ---------------------------------------------------------------------------
// A workgroup of 512 threads covers 256 environments.  Its first four waves
// step them (one thread per environment, the CartCore loop with the state and
// up to W padding words in registers) and write each step's row into LDS
// instead of device memory; its last four waves copy the rows from LDS to the
// trajectory, each step's seven stores close together with none of the step's
// arithmetic between them.  The trajectory stores then run at 95-96 % of the
// rate of a store-only kernel, against 85 % when every wave interleaves them
// with the step's arithmetic.
//
// Rows are handed over in chunks of kHandSteps steps through two LDS buffers
// and one workgroup barrier per chunk: between barriers c and c+1 the stepping
// waves fill buffer (c+1) & 1 while the storing waves drain buffer c & 1, which
// the steppers filled before barrier c.  Both sides pass ceil(K / kHandSteps)
// barriers, then the one in the block statistics.  37 KB of LDS per workgroup
// leaves room for four workgroups (eight waves per SIMD) per CU.
constexpr uint32_t kHandSteps = 4;

// CartCore hook of the stepping waves: records each step's row in the current
// LDS buffer and passes a barrier after every kHandSteps steps.
struct RowHandOver {
    float (*obs)[kHandSteps][4][kBlock];     // [2 buffers][step][component][env]
    uint16_t (*act_done)[kHandSteps][kBlock];  // action | done byte << 8
    uint32_t col;                            // this thread's environment column
    uint32_t i = 0u, buf = 0u;               // step within the chunk, buffer
    __device__ __forceinline__ void record(const CartState& s, uint32_t act, uint32_t d)
    {
        obs[buf][i][0][col] = s.x;
        obs[buf][i][1][col] = s.xd;
        obs[buf][i][2][col] = s.th;
        obs[buf][i][3][col] = s.thd;
        act_done[buf][i][col] = (uint16_t)(act | (d << 8));
    }
    __device__ __forceinline__ void operator()(uint32_t, bool)
    {
        if (++i == kHandSteps) {
            i = 0u;
            buf ^= 1u;
            __syncthreads();
        }
    }
    // the barrier that hands over a last, partial chunk
    __device__ __forceinline__ void flush()
    {
        if (i != 0u) __syncthreads();
    }
};

// The storing waves' copy of one recorded step (row `row` of the call).
__device__ __forceinline__ void store_handed_row(const StepArgs& a, size_t row, uint32_t off4, uint32_t off1,
                                                 const float (*obs)[kBlock], const uint16_t* act_done, uint32_t col)
{
    const size_t plane = a.n;
    const float x = obs[0][col], xd = obs[1][col], th = obs[2][col], thd = obs[3][col];
    const uint32_t ad = act_done[col];
    float* o = a.obs + row * 4 * plane;
    *at(a.action + row * plane, off1) = (uint8_t)ad;
    *at(a.done + row * plane, off1) = (uint8_t)(ad >> 8);
    *at(o, off4) = x;
    *at(o + plane, off4) = xd;
    *at(o + 2 * plane, off4) = th;
    *at(o + 3 * plane, off4) = thd;
    *at(a.reward + row * plane, off4) = 1.0f;
}

// Both hooks of a stepping wave: the padding words' update and the hand-over.
template <int W>
struct PadHandOver {
    RegisterPad<W>& pad;
    RowHandOver& h;
    __device__ __forceinline__ void record(const CartState& s, uint32_t act, uint32_t d) { h.record(s, act, d); }
    __device__ __forceinline__ void operator()(uint32_t act, bool reset)
    {
        pad(act, reset);
        h(act, reset);
    }
};

template <int W, bool STATS>
__global__ __launch_bounds__(2 * kBlock) __attribute__((amdgpu_waves_per_eu(8)))
void k_cartpole_split(StepArgs a)
{
    __shared__ float lds_obs[2][kHandSteps][4][kBlock];
    __shared__ uint16_t lds_ad[2][kHandSteps][kBlock];
    const uint32_t blk = xcd_block();
    const uint32_t col = threadIdx.x % kBlock;
    const uint32_t env = blk * kBlock + col;
    const bool live = env < a.n;
    uint32_t c0 = 0u, c1 = 0u, c2 = 0u, c3 = 0u;
    if (threadIdx.x < kBlock) {
        // stepping waves; threads past n step a zero state so that every wave
        // passes the same barriers, and record nothing the storing side keeps
        CartCore<false, STATS> core(a.p, env);
        if (live) {
            core.load(a);
        } else {
            core.s = CartState{0.0f, 0.0f, 0.0f, 0.0f};
            core.ep = 0u;
        }
        RowHandOver h{lds_obs, lds_ad, col};
        RegisterPad<W> pad;
#pragma unroll
        for (int j = 0; j < W; ++j) {
            const bool on = live && (uint32_t)j < a.D;
            const size_t q = (size_t)j * a.n + env;
            pad.s[j] = on ? a.pad_s[q] : 0.0f;
            pad.a[j] = on ? a.pad_a[q] : 0.0f;
            pad.b[j] = on ? a.pad_b[q] : 0.0f;
        }
        PadHandOver<W> ph{pad, h};
        core.run(a.t0, a.K, ph);
        h.flush();
        if (live) {
#pragma unroll
            for (int j = 0; j < W; ++j)
                if ((uint32_t)j < a.D) a.pad_s[(size_t)j * a.n + env] = pad.s[j];
            core.store(a);
            c0 = core.n_eps;
            c1 = core.finished_length_sum(a.K);
            c2 = core.n_term;
            c3 = core.n_trunc;
        }
    } else {
        // storing waves: chunk c is complete after the c-th barrier
        const uint32_t off4 = env * 4u, off1 = env;
        const uint32_t n_chunks = a.K / kHandSteps + (a.K % kHandSteps != 0u ? 1u : 0u);
        for (uint32_t c = 0; c < n_chunks; ++c) {
            __syncthreads();
            const uint32_t b = c & 1u, k0 = c * kHandSteps, m = min(kHandSteps, a.K - k0);
            if (live && m == kHandSteps) {
#pragma unroll
                for (uint32_t i = 0; i < kHandSteps; ++i)
                    store_handed_row(a, (size_t)k0 + i, off4, off1, lds_obs[b][i], lds_ad[b][i], col);
            } else if (live) {
                for (uint32_t i = 0; i < m; ++i)
                    store_handed_row(a, (size_t)k0 + i, off4, off1, lds_obs[b][i], lds_ad[b][i], col);
            }
        }
    }
    if (STATS) store_block_stats<2 * kBlock>(a.stats, blk, c0, c1, c2, c3);
}

// ---------------------------------------------------------------------------
// Reset.
// ---------------------------------------------------------------------------
// Initial state of every environment (episode beginning at step 0).
__global__ __launch_bounds__(kBlock) void k_reset_cart(DevParams p, uint32_t n, float* cart, uint32_t* ep)
{
    const uint32_t env = blockIdx.x * kBlock + threadIdx.x;
    if (env >= n) return;
    const uint4 w = philox(env + p.env0, 0u, STREAM_RESET, p.key0, p.key1);
    const size_t plane = n;
    cart[env] = uniform01_to(w.x, p.reset_lo, p.reset_width);
    cart[plane + env] = uniform01_to(w.y, p.reset_lo, p.reset_width);
    cart[2 * plane + env] = uniform01_to(w.z, p.reset_lo, p.reset_width);
    cart[3 * plane + env] = uniform01_to(w.w, p.reset_lo, p.reset_width);
    ep[env] = 0u;
}

// Padding parameters and zero words: word j of env e lives at index
// j * stride_j + e * stride_e; one thread per (word, env) pair, grid-strided.
__global__ __launch_bounds__(kBlock) void k_reset_pad(DevParams p, uint32_t n, uint32_t D, size_t stride_j,
                                                      size_t stride_e, float a_lo, float a_width, float b_lo,
                                                      float b_width, float* s, float* pa, float* pb)
{
    const size_t total = (size_t)n * D;
    for (size_t i = (size_t)blockIdx.x * kBlock + threadIdx.x; i < total; i += (size_t)gridDim.x * kBlock) {
        // consecutive threads take consecutive addresses in either layout
        const uint32_t env = (uint32_t)(stride_e == 1 ? i % n : i / D);
        const uint32_t j = (uint32_t)(stride_e == 1 ? i / n : i % D);
        const uint4 w = philox(env + p.env0, j, STREAM_PARAMS, p.key0, p.key1);
        const size_t q = (size_t)j * stride_j + (size_t)env * stride_e;
        pa[q] = uniform01_to(w.x, a_lo, a_width);
        pb[q] = uniform01_to(w.y, b_lo, b_width);
        s[q] = 0.0f;
    }
}

}  // namespace rlsim_dev
