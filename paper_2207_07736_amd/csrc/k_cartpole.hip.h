// k_cartpole.hip.h -- fused K-step simulator kernels with random actions.
//
//  k_cartpole_fused<W>: one thread per environment; the cart-pole state and up
//      to W padding words stay in registers for all K steps.
//  k_cartpole_wide<G,W>: wide padding (the paper's state-size factor): phase 1
//      runs the cart-pole steps one thread per environment and leaves each
//      step's (action, done) bits in LDS; phase 2 gives every environment G
//      lanes holding W padding words each in registers and replays the steps
//      from those bits.  The padding words only feed on (action, done), so the
//      split is exact, and each word is still read and written once per launch.
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
    uint32_t env;
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
        : p(p_), env(env_), off4(env_ * 4u), off1a(env_), off1d(env_) {}

    // Sum of the lengths of the episodes that ended in this launch: every step
    // adds one to the running episode, so the finished lengths plus the final
    // running length equal the starting length plus K (mod 2^32).
    __device__ __forceinline__ uint32_t finished_length_sum(uint32_t K) const { return ep_start + K - ep; }

    __device__ __forceinline__ void draw_reset(uint32_t block)
    {
        const uint4 w = philox(env, block, STREAM_RESET, p.key0, p.key1);
        rs.x = uniform24_to(w.x, p.reset_lo, p.reset_width_u24);
        rs.xd = uniform24_to(w.y, p.reset_lo, p.reset_width_u24);
        rs.th = uniform24_to(w.z, p.reset_lo, p.reset_width_u24);
        rs.thd = uniform24_to(w.w, p.reset_lo, p.reset_width_u24);
    }

    // Called before the step at t when t is a multiple of 32.
    __device__ __forceinline__ void refresh_actions(uint32_t t)
    {
        if ((t & 127u) == 0u) aw = philox(env, t >> 7, STREAM_ACTION, p.key0, p.key1);
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
    // truncate, auto-reset.  hook(act, reset) sees the action and whether the
    // episode ended.  The row pointers are left for the caller to advance.
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
            // the offsets are passed through an empty asm in place each step
            asm volatile("" : "+v"(off4), "+v"(off1a), "+v"(off1d));
            *at(obs, off4) = s.x;
            *at(obs + plane, off4) = s.xd;
            *at(obs + 2 * plane, off4) = s.th;
            *at(obs + 3 * plane, off4) = s.thd;
            *at(act_row, off1a) = (uint8_t)act;
            *at(rew_row, off4) = 1.0f;
            *at(done_row, off1d) = (uint8_t)d;
        }
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
        aw = philox(env, t >> 7, STREAM_ACTION, p.key0, p.key1);
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

// Sums the four episode counters over the workgroup and writes one row of the
// block statistics (all threads of the block must call this).
__device__ __forceinline__ void store_block_stats(uint32_t* stats, uint32_t blk, uint32_t c0, uint32_t c1, uint32_t c2,
                                                  uint32_t c3)
{
    __shared__ uint32_t part[kBlock / 64][4];
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
        for (int w = 0; w < kBlock / 64; ++w) sum += part[w][threadIdx.x];
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
    __device__ __forceinline__ void operator()(uint32_t, bool) {}
};

// Padding words held by one thread; zeroed when the episode ends.
template <int W>
struct RegisterPad {
    float s[W > 0 ? W : 1], a[W > 0 ? W : 1], b[W > 0 ? W : 1];
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
// Wide padding.
// ---------------------------------------------------------------------------
constexpr uint32_t kChunk = 512;                 // steps per phase-1/phase-2 round
constexpr uint32_t kChunkWords = kChunk / 32u;   // 32-bit bit words per env per round

// Phase-1 hook: collects each step's action and done bits, 32 steps per word,
// into this thread's LDS columns.
struct BitRecorder {
    uint32_t* lds_u;     // [kChunkWords][kBlock]
    uint32_t* lds_d;
    uint32_t col;        // threadIdx.x
    uint32_t k = 0u;     // step index within the round
    uint32_t ub = 0u, db = 0u;
    __device__ __forceinline__ void operator()(uint32_t act, bool reset)
    {
        const uint32_t bit = k & 31u;
        ub |= act << bit;
        db |= (reset ? 1u : 0u) << bit;
        if (bit == 31u) {
            lds_u[(k >> 5) * kBlock + col] = ub;
            lds_d[(k >> 5) * kBlock + col] = db;
            ub = 0u;
            db = 0u;
        }
        ++k;
    }
    __device__ __forceinline__ void flush()
    {
        if ((k & 31u) != 0u) {
            lds_u[(k >> 5) * kBlock + col] = ub;
            lds_d[(k >> 5) * kBlock + col] = db;
        }
    }
};

// Wave-uniform replay of the padding recurrence (one environment per wave, so
// the action and done bits are scalars): for N words of this lane at offset O,
// run steps 0 .. m-1 of one 32-step bit word as a scalar loop around in-place
// VALU updates, i.e. one vector instruction per word per step.  Each step is
//   bit u set:   s <- fma(a, s, b)     (one rounding, v_fma_f32)
//   bit u clear: s <- a * s            (v_mul_f32)
//   bit d set:   s <- +0               (episode ended at this step)
// Written as one asm block because compiled if/else forms of it write the two
// paths to different registers and copy them back at the join, doubling the
// vector work.  Each update path carries its own copy of the loop tail, and
// the rare clearing sits out of line, so a step takes one taken branch after
// an FMA step and two after a multiply step.  The counter starts at 0 and the
// loop ends when it reaches m (1 <= m <= 32).
#define RL_REP4(X) X(0) X(1) X(2) X(3)
#define RL_REP8(X) RL_REP4(X) X(4) X(5) X(6) X(7)
#define RL_REP16(X) RL_REP8(X) X(8) X(9) X(10) X(11) X(12) X(13) X(14) X(15)
#define RL_REP32(X) \
    RL_REP16(X) X(16) X(17) X(18) X(19) X(20) X(21) X(22) X(23) X(24) X(25) X(26) X(27) X(28) X(29) X(30) X(31)
#define RL_FMA(i) "v_fma_f32 %[s" #i "], %[a" #i "], %[s" #i "], %[b" #i "]\n"
#define RL_MUL(i) "v_mul_f32 %[s" #i "], %[a" #i "], %[s" #i "]\n"
#define RL_ZERO(i) "v_mov_b32 %[s" #i "], 0\n"
#define RL_OUT_S(i) [s##i] "+v"(s[O + i]),
#define RL_IN_A(i) [a##i] "v"(pa[O + i]),
#define RL_IN_B(i) [b##i] "v"(pb[O + i]),
#define RL_TAIL                          \
    "s_bitcmp1_b32 %[db], %[c]\n"        \
    "s_cbranch_scc1 L_rl_zero%=\n"       \
    "s_add_u32 %[c], %[c], 1\n"          \
    "s_cmp_lt_u32 %[c], %[m]\n"          \
    "s_cbranch_scc1 L_rl_step%=\n"       \
    "s_branch L_rl_end%=\n"
#define RL_REPLAY_ASM(REP)                                                               \
    asm volatile("s_mov_b32 %[c], 0\n"                                                   \
                 "L_rl_step%=:\n"                                                        \
                 "s_bitcmp1_b32 %[ub], %[c]\n"                                           \
                 "s_cbranch_scc0 L_rl_mul%=\n" REP(RL_FMA) RL_TAIL                       \
                 "L_rl_mul%=:\n" REP(RL_MUL) RL_TAIL                                     \
                 "L_rl_zero%=:\n" REP(RL_ZERO)                                           \
                 "s_add_u32 %[c], %[c], 1\n"                                             \
                 "s_cmp_lt_u32 %[c], %[m]\n"                                             \
                 "s_cbranch_scc1 L_rl_step%=\n"                                          \
                 "L_rl_end%=:\n"                                                         \
                 : REP(RL_OUT_S)[c] "=&s"(cnt)                                           \
                 : REP(RL_IN_A) REP(RL_IN_B)[ub] "s"(ub), [db] "s"(db), [m] "s"(m)       \
                 : "scc")

template <int N, int O, int W>
__device__ __forceinline__ void replay_uniform_group(float (&s)[W], const float (&pa)[W], const float (&pb)[W],
                                                     uint32_t ub, uint32_t db, uint32_t m)
{
    static_assert(O + N <= W, "group outside the lane's words");
    uint32_t cnt;
    if constexpr (N == 32) RL_REPLAY_ASM(RL_REP32);
    else if constexpr (N == 16) RL_REPLAY_ASM(RL_REP16);
    else if constexpr (N == 8) RL_REPLAY_ASM(RL_REP8);
    else RL_REPLAY_ASM(RL_REP4);
}

// All W words of the lane, in groups of at most kReplayGroup.
constexpr int kReplayGroup = 32;
template <int W, int O = 0>
__device__ __forceinline__ void replay_uniform(float (&s)[W], const float (&pa)[W], const float (&pb)[W],
                                               uint32_t ub, uint32_t db, uint32_t m)
{
    if constexpr (O < W) {
        constexpr int R = W - O;
        constexpr int N = R >= kReplayGroup ? kReplayGroup : R >= 16 ? 16 : R >= 8 ? 8 : 4;
        replay_uniform_group<N, O, W>(s, pa, pb, ub, db, m);
        replay_uniform<W, O + N>(s, pa, pb, ub, db, m);
    }
}

// Phase 2: G lanes per environment, W consecutive words per lane (W a multiple
// of 4, loaded as float4).  Replays `steps` steps from the LDS bits for the
// 64 / G environments a wave covers at a time, for all of the wave's 64 envs.
template <int G, int W>
__device__ __forceinline__ void replay_padding(const StepArgs& a, const uint32_t* lds_u, const uint32_t* lds_d,
                                               uint32_t steps, uint32_t blk)
{
    static_assert(W % 4 == 0 && 64 % G == 0, "bad wide-padding shape");
    const uint32_t lane = threadIdx.x % 64u, wave = threadIdx.x / 64u;
    const uint32_t gi = lane / G, gl = lane % G;            // env slot in the wave, lane in its group
    const uint32_t chunk_words = (uint32_t)(G * W);
    const uint32_t n_chunks = (a.Dp + chunk_words - 1u) / chunk_words;
    // a pass covers 64 / G environments, so the wave's 64 take G passes
    for (uint32_t pass = 0; pass < (uint32_t)G; ++pass) {
        const uint32_t col = wave * 64u + pass * (64u / G) + gi;   // env column in the block
        const uint32_t env = blk * kBlock + col;
        const bool live = env < a.n;
        for (uint32_t c = 0; c < n_chunks; ++c) {
            // float4 q of this lane holds words base + q * 4G .. +3: the G lanes of
            // a group read and write 16 G contiguous bytes per instruction
            const uint32_t base = c * chunk_words + 4u * gl;
            float s[W], pa[W], pb[W];
            const size_t row = (size_t)env * a.Dp;
#pragma unroll
            for (int i = 0; i < W; i += 4) {
                const uint32_t j = base + (uint32_t)(i / 4) * (4u * G);
                const bool on = live && j < a.Dp;
                const float4 vs = on ? *reinterpret_cast<const float4*>(a.pad_s + row + j) : float4{0, 0, 0, 0};
                const float4 va = on ? *reinterpret_cast<const float4*>(a.pad_a + row + j) : float4{0, 0, 0, 0};
                const float4 vb = on ? *reinterpret_cast<const float4*>(a.pad_b + row + j) : float4{0, 0, 0, 0};
                s[i] = vs.x; s[i + 1] = vs.y; s[i + 2] = vs.z; s[i + 3] = vs.w;
                pa[i] = va.x; pa[i + 1] = va.y; pa[i + 2] = va.z; pa[i + 3] = va.w;
                pb[i] = vb.x; pb[i + 1] = vb.y; pb[i + 2] = vb.z; pb[i + 3] = vb.w;
            }
            for (uint32_t w32 = 0; w32 * 32u < steps; ++w32) {
                uint32_t ub = lds_u[w32 * kBlock + col];
                uint32_t db = lds_d[w32 * kBlock + col];
                const uint32_t m = min(32u, steps - w32 * 32u);
                if (G == 64) {
                    // one environment per wave: the bits are wave-uniform, so
                    // each step is a scalar branch and one FMA per word
                    replay_uniform<W>(s, pa, pb, __builtin_amdgcn_readfirstlane(ub), __builtin_amdgcn_readfirstlane(db),
                                      __builtin_amdgcn_readfirstlane(m));
                } else {
                    for (uint32_t i = 0; i < m; ++i) {
                        const bool u = (ub >> i) & 1u;
                        const bool d = (db >> i) & 1u;
#pragma unroll
                        for (int j = 0; j < W; ++j) s[j] = pad_update(pa[j], s[j], pb[j], u);
                        // episode ends are rare: clear words only in a wave that has one
                        if (__builtin_amdgcn_ballot_w64(d) != 0u) {
                            asm volatile("" ::: "memory");
#pragma unroll
                            for (int j = 0; j < W; ++j) s[j] = d ? 0.0f : s[j];
                        }
                    }
                }
            }
#pragma unroll
            for (int i = 0; i < W; i += 4) {
                const uint32_t j = base + (uint32_t)(i / 4) * (4u * G);
                if (live && j < a.Dp)
                    *reinterpret_cast<float4*>(a.pad_s + row + j) = float4{s[i], s[i + 1], s[i + 2], s[i + 3]};
            }
        }
    }
}

template <int G, int W, bool REC, bool STATS>
__global__ __launch_bounds__(kBlock) void k_cartpole_wide(StepArgs a)
{
    __shared__ uint32_t lds_u[kChunkWords * kBlock];
    __shared__ uint32_t lds_d[kChunkWords * kBlock];
    const uint32_t blk = xcd_block();
    const uint32_t env = blk * kBlock + threadIdx.x;
    const bool live = env < a.n;
    CartCore<REC, STATS> core(a.p, env);
    if (live) core.load(a);
    for (uint32_t k0 = 0; k0 < a.K; k0 += kChunk) {
        const uint32_t steps = min(kChunk, a.K - k0);
        BitRecorder rec{lds_u, lds_d, threadIdx.x};
        if (live) {
            if (REC) core.set_rows(a, k0);
            core.run(a.t0 + k0, steps, rec);
            rec.flush();
        }
        __syncthreads();
        replay_padding<G, W>(a, lds_u, lds_d, steps, blk);
        __syncthreads();
    }
    if (live) core.store(a);
    if (STATS) {
        const uint32_t len_sum = live ? core.finished_length_sum(a.K) : 0u;
        store_block_stats(a.stats, blk, core.n_eps, len_sum, core.n_term, core.n_trunc);
    }
}

// ---------------------------------------------------------------------------
// Reset.
// ---------------------------------------------------------------------------
// Initial state of every environment (episode beginning at step 0).
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
        const uint4 w = philox(env, j, STREAM_PARAMS, p.key0, p.key1);
        const size_t q = (size_t)j * stride_j + (size_t)env * stride_e;
        pa[q] = uniform01_to(w.x, a_lo, a_width);
        pb[q] = uniform01_to(w.y, b_lo, b_width);
        s[q] = 0.0f;
    }
}

}  // namespace rlsim_dev
