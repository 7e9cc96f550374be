// k_chain.hip.h -- the second simulator: a cart carrying a chain of N identical
// uniform rods (the heavier, multi-body kind of simulator the paper's Future
// Work points to), fused over K steps with random actions, one thread per
// environment and the whole state in registers.
//
// Generalised coordinates q = (x, phi_1 .. phi_N), phi_k the angle of link k
// from the upward vertical.  With mu_k = (N - k) m the mass beyond link k, L
// the link length, h_k = L (m/2 + mu_k), G_kk = L^2 (m/3 + mu_k) and
// G_jk = L h_k (j < k), Lagrange's equations are M(q) qdd = f(q, qd):
//   M_00 = mc + N m,  M_0k = h_k cos phi_k,  M_jk = G_jk cos(phi_j - phi_k),
//   f_0  = F + sum_k h_k sin(phi_k) phid_k^2,
//   f_j  = g h_j sin(phi_j) - sum_{k != j} G_jk sin(phi_j - phi_k) phid_k^2.
// Each step assembles M and f and solves them by Gaussian elimination without
// pivoting (M is positive definite) on the upper triangle, then takes an
// explicit-Euler step; the operation order is fixed (one IEEE rounding per
// operation, explicit FMAs) so that the results are reproducible bit for bit.
// The state words are (x, xd, phi_1, phid_1, ..., phi_N, phid_N).
#pragma once

#include "k_cartpole.hip.h"

namespace rlsim_dev {

constexpr int kMaxLinks = 4;

// Kernel-side constants of the chain, each one fp32 operation on the
// configured values (make_chain_params in rlsim.hip): the shared DevParams
// (step length, force, thresholds, reset box, RNG key) and the couplings.
struct ChainParams {
    DevParams p;
    float m00;                       // mc + N m
    float h[kMaxLinks + 1];          // [1..N] cart coupling h_k
    float gdiag[kMaxLinks + 1];      // G_kk
    float lh[kMaxLinks + 1];         // L h_k = G_jk for j < k
    float gh[kMaxLinks + 1];         // g h_k
};

struct ChainArgs {
    ChainParams c;
    uint32_t n;          // environments
    uint32_t t0;         // global step of row 0
    uint32_t K;          // steps in this launch
    float* state;        // [2N+2][n]
    uint32_t* ep;        // [n]
    float* obs;          // [K][2N+2][n]
    uint8_t* action;     // [K][n]
    float* reward;       // [K][n]
    uint8_t* done;       // [K][n]
    uint32_t* stats;     // [ceil(n/256)][4]
};

template <int N>
struct ChainState {
    float q[N + 1], qd[N + 1];       // q[0] = x, q[k] = phi_k
};

// Accelerations of the chain under the cart force F.
template <int N>
__device__ __forceinline__ void chain_accel(const ChainParams& c, const ChainState<N>& st, float force,
                                            float (&qdd)[N + 1])
{
    float s[N + 1], co[N + 1], w[N + 1];
#pragma unroll
    for (int j = 1; j <= N; ++j) {
        sincos_full(st.q[j], s[j], co[j]);
        w[j] = st.qd[j] * st.qd[j];
    }
    // mass matrix, upper triangle
    float A[N + 1][N + 1];
    A[0][0] = c.m00;
#pragma unroll
    for (int j = 1; j <= N; ++j) {
        A[0][j] = c.h[j] * co[j];
        A[j][j] = c.gdiag[j];
    }
#pragma unroll
    for (int j = 1; j <= N; ++j)
#pragma unroll
        for (int i = j + 1; i <= N; ++i) {
            const float cjk = __builtin_fmaf(co[j], co[i], s[j] * s[i]);      // cos(phi_j - phi_i)
            A[j][i] = c.lh[i] * cjk;
        }
    // forces: the cart's, then gravity and the links' velocity terms, pairs in
    // lexicographic order
    float f[N + 1];
    f[0] = force;
#pragma unroll
    for (int j = 1; j <= N; ++j) f[0] = __builtin_fmaf(c.h[j] * s[j], w[j], f[0]);
#pragma unroll
    for (int j = 1; j <= N; ++j) f[j] = c.gh[j] * s[j];
#pragma unroll
    for (int j = 1; j <= N; ++j)
#pragma unroll
        for (int i = j + 1; i <= N; ++i) {
            const float sjk = __builtin_fmaf(s[j], co[i], -(co[j] * s[i]));  // sin(phi_j - phi_i)
            const float P = c.lh[i] * sjk;
            f[j] = __builtin_fmaf(-P, w[i], f[j]);
            f[i] = __builtin_fmaf(P, w[j], f[i]);
        }
    // elimination on the upper triangle, then back substitution
    float inv[N + 1];
#pragma unroll
    for (int p = 0; p < N; ++p) {
        inv[p] = 1.0f / A[p][p];                                 // IEEE division
#pragma unroll
        for (int i = p + 1; i <= N; ++i) {
            const float l = A[p][i] * inv[p];
#pragma unroll
            for (int j = i; j <= N; ++j) A[i][j] = __builtin_fmaf(-l, A[p][j], A[i][j]);
            f[i] = __builtin_fmaf(-l, f[p], f[i]);
        }
    }
    inv[N] = 1.0f / A[N][N];
#pragma unroll
    for (int i = N; i >= 0; --i) {
        float acc = f[i];
#pragma unroll
        for (int j = i + 1; j <= N; ++j) acc = __builtin_fmaf(-A[i][j], qdd[j], acc);
        qdd[i] = acc * inv[i];
    }
}

// One explicit-Euler iteration; positions advance with the old velocities.
template <int N>
__device__ __forceinline__ ChainState<N> chain_euler(const ChainParams& c, const ChainState<N>& st, float force)
{
    float qdd[N + 1];
    chain_accel<N>(c, st, force, qdd);
    ChainState<N> o;
#pragma unroll
    for (int j = 0; j <= N; ++j) {
        o.q[j] = __builtin_fmaf(c.p.tau, st.qd[j], st.q[j]);
        o.qd[j] = __builtin_fmaf(c.p.tau, qdd[j], st.qd[j]);
    }
    return o;
}

// Strict thresholds on the cart position and every link angle (infinite when
// termination is disabled); NaN compares false.
template <int N>
__device__ __forceinline__ bool chain_crossed(const DevParams& p, const ChainState<N>& st)
{
    bool out = __builtin_fabsf(st.q[0]) > p.thr_x;
#pragma unroll
    for (int j = 1; j <= N; ++j) out = out || (__builtin_fabsf(st.q[j]) > p.thr_th);
    return out;
}

// The reset draw of an episode beginning in 8-step block `block`: state words
// 4j .. 4j+3 from Philox counter (env, block, RESET, j).
template <int N>
__device__ __forceinline__ void chain_reset_draw(const DevParams& p, uint32_t gid, uint32_t block, ChainState<N>& rs)
{
    constexpr int S = 2 * (N + 1);
    float v[((S + 3) / 4) * 4];
#pragma unroll
    for (int j = 0; 4 * j < S; ++j) {
        const uint4 w = philox(gid, block, STREAM_RESET, p.key0, p.key1, (uint32_t)j);
        v[4 * j] = uniform24_to(w.x, p.reset_lo, p.reset_width_u24);
        v[4 * j + 1] = uniform24_to(w.y, p.reset_lo, p.reset_width_u24);
        v[4 * j + 2] = uniform24_to(w.z, p.reset_lo, p.reset_width_u24);
        v[4 * j + 3] = uniform24_to(w.w, p.reset_lo, p.reset_width_u24);
    }
#pragma unroll
    for (int j = 0; j <= N; ++j) {
        rs.q[j] = v[2 * j];
        rs.qd[j] = v[2 * j + 1];
    }
}

// ChainCore hook that does nothing (the rows, if any, are stored by the core).
template <int N>
struct ChainNoHook {
    __device__ __forceinline__ void record(const ChainState<N>&, uint32_t, uint32_t) {}
    __device__ __forceinline__ void advance() {}
};

// One environment's chain state and RNG words, advanced step by step: the
// cart-pole's CartCore loop with the chain's state, step and reset draw.
template <int N, bool REC, bool STATS>
struct ChainCore {
    static constexpr int S = 2 * (N + 1);
    const ChainParams& c;
    uint32_t env, gid;
    ChainState<N> s, rs;
    uint32_t ep, ep_start = 0u;
    uint4 aw;
    uint32_t abits;
    float* obs;
    uint8_t* act_row;
    float* rew_row;
    uint8_t* done_row;
    size_t plane;
    uint32_t off4, off1;
    uint32_t n_eps = 0u, n_term = 0u, n_trunc = 0u;

    __device__ __forceinline__ ChainCore(const ChainParams& c_, uint32_t env_)
        : c(c_), env(env_), gid(env_ + c_.p.env0), off4(env_ * 4u), off1(env_) {}

    __device__ __forceinline__ uint32_t finished_length_sum(uint32_t K) const { return ep_start + K - ep; }

    __device__ __forceinline__ void refresh_actions(uint32_t t)
    {
        if ((t & 127u) == 0u) aw = philox(gid, t >> 7, STREAM_ACTION, c.p.key0, c.p.key1);
        abits = pick_word(aw, (t >> 5) & 3u);
    }

    // One step; hook.record(state, action, done byte) sees the row this step
    // records, and hook.advance() runs after the step is complete.
    template <class Hook>
    __device__ __forceinline__ void step(Hook& hook)
    {
        const uint32_t act = abits & 1u;
        abits >>= 1;
        const float force = act ? c.p.force_mag : -c.p.force_mag;
        ChainState<N> nx = chain_euler<N>(c, s, force);
        for (uint32_t it = 1; it < c.p.iters; ++it) nx = chain_euler<N>(c, nx, force);
        const uint32_t len = ep + 1u;
        const bool term = chain_crossed<N>(c.p, nx);
        const bool trunc = (c.p.max_steps != 0u) && (len >= c.p.max_steps);
        const uint32_t d = (trunc ? 2u : 0u) + (uint32_t)term;
        if (REC) {
            asm volatile("" : "+v"(off4), "+v"(off1));
            *at(act_row, off1) = (uint8_t)act;
            *at(done_row, off1) = (uint8_t)d;
#pragma unroll
            for (int j = 0; j <= N; ++j) {
                *at(obs + (2 * j) * plane, off4) = s.q[j];
                *at(obs + (2 * j + 1) * plane, off4) = s.qd[j];
            }
            *at(rew_row, off4) = 1.0f;
            obs += S * plane;
            act_row += plane;
            rew_row += plane;
            done_row += plane;
        }
        hook.record(s, act, d);
        const bool reset = term || trunc;
#pragma unroll
        for (int j = 0; j <= N; ++j) {
            s.q[j] = reset ? rs.q[j] : nx.q[j];
            s.qd[j] = reset ? rs.qd[j] : nx.qd[j];
        }
        ep = reset ? 0u : len;
        if (STATS) {
            n_eps += reset ? 1u : 0u;
            n_term += term ? 1u : 0u;
            n_trunc += trunc ? 1u : 0u;
        }
        hook.advance();
    }

    // Steps t0 .. t0+K-1 in bodies of the eight steps that share one reset
    // block, as CartCore::run.
    template <class Hook>
    __device__ __forceinline__ void run(uint32_t t0, uint32_t K, Hook& hook)
    {
        uint32_t t = t0, k = 0;
        aw = philox(gid, t >> 7, STREAM_ACTION, c.p.key0, c.p.key1);
        abits = pick_word(aw, (t >> 5) & 3u) >> (t & 31u);
        if (((t + 1u) & 7u) != 0u) {
            chain_reset_draw<N>(c.p, gid, (t + 1u) >> 3, rs);
            while (k < K && ((t + 1u) & 7u) != 0u) {
                step(hook);
                ++t;
                ++k;
            }
        }
        for (; K - k >= 8u; k += 8u, t += 8u) {
            chain_reset_draw<N>(c.p, gid, (t + 1u) >> 3, rs);
            step(hook);
            if (((t + 1u) & 31u) == 0u) refresh_actions(t + 1u);
#pragma unroll 1
            for (int i = 0; i < 7; ++i) step(hook);
        }
        if (k < K) {
            chain_reset_draw<N>(c.p, gid, (t + 1u) >> 3, rs);
            step(hook);
            ++t;
            ++k;
            if (k < K && (t & 31u) == 0u) refresh_actions(t);
            for (; k < K; ++k) step(hook);
        }
    }

    __device__ __forceinline__ void load(const ChainArgs& a)
    {
        const size_t pl = a.n;
#pragma unroll
        for (int j = 0; j <= N; ++j) {
            s.q[j] = a.state[(2 * j) * pl + env];
            s.qd[j] = a.state[(2 * j + 1) * pl + env];
        }
        ep = a.ep[env];
        ep_start = ep;
    }

    __device__ __forceinline__ void store(const ChainArgs& a)
    {
        const size_t pl = a.n;
#pragma unroll
        for (int j = 0; j <= N; ++j) {
            a.state[(2 * j) * pl + env] = s.q[j];
            a.state[(2 * j + 1) * pl + env] = s.qd[j];
        }
        a.ep[env] = ep;
    }
};

template <int N, bool REC, bool STATS>
__global__ __launch_bounds__(kBlock) void k_chain_fused(ChainArgs a)
{
    const uint32_t blk = xcd_block();
    const uint32_t env = blk * kBlock + threadIdx.x;
    ChainCore<N, REC, STATS> core(a.c, env);
    if (env < a.n) {
        core.load(a);
        if (REC) {
            core.plane = a.n;
            core.obs = a.obs;
            core.act_row = a.action;
            core.rew_row = a.reward;
            core.done_row = a.done;
        }
        ChainNoHook<N> none;
        core.run(a.t0, a.K, none);
        core.store(a);
    }
    if (STATS) {
        const uint32_t len_sum = env < a.n ? core.finished_length_sum(a.K) : 0u;
        store_block_stats(a.stats, blk, core.n_eps, len_sum, core.n_term, core.n_trunc);
    }
}

// k_chain_split<N>: the fused chain loop with a trajectory, warp-specialised as
// k_cartpole_split: in a 512-thread workgroup the first four waves step the
// block's 256 environments and write each step's row (2N + 2 obs words and
// action | done << 8) to LDS; the last four waves store the rows.  Rows are
// handed over in chunks of kChainHandSteps steps through two LDS buffers, one
// workgroup barrier per chunk: between barriers c and c+1 the stepping waves
// fill buffer (c+1) & 1 while the storing waves drain buffer c & 1.  Two-step
// chunks keep the LDS at 2 x 2 x (8 N + 10) x 256 B (N = 4: 42 KB).
constexpr uint32_t kChainHandSteps = 2;

template <int N>
struct ChainHandOver {
    static constexpr int S = 2 * (N + 1);
    float (*obs)[kChainHandSteps][S][kBlock];       // [2 buffers][step][word][env]
    uint16_t (*act_done)[kChainHandSteps][kBlock];  // action | done byte << 8
    uint32_t col;                                   // this thread's environment column
    uint32_t i = 0u, buf = 0u;                      // step within the chunk, buffer
    __device__ __forceinline__ void record(const ChainState<N>& st, uint32_t act, uint32_t d)
    {
#pragma unroll
        for (int j = 0; j <= N; ++j) {
            obs[buf][i][2 * j][col] = st.q[j];
            obs[buf][i][2 * j + 1][col] = st.qd[j];
        }
        act_done[buf][i][col] = (uint16_t)(act | (d << 8));
    }
    __device__ __forceinline__ void advance()
    {
        if (++i == kChainHandSteps) {
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

// The storing waves' copy of one recorded step (row `row` of the call):
// byte planes first, then the obs words and the reward.
template <int N>
__device__ __forceinline__ void store_chain_row(const ChainArgs& a, size_t row, uint32_t off4, uint32_t off1,
                                                const float (*obs)[kBlock], const uint16_t* act_done, uint32_t col)
{
    constexpr int S = 2 * (N + 1);
    const size_t plane = a.n;
    float v[S];
#pragma unroll
    for (int j = 0; j < S; ++j) v[j] = obs[j][col];
    const uint32_t ad = act_done[col];
    float* o = a.obs + row * S * plane;
    *at(a.action + row * plane, off1) = (uint8_t)ad;
    *at(a.done + row * plane, off1) = (uint8_t)(ad >> 8);
#pragma unroll
    for (int j = 0; j < S; ++j) *at(o + j * plane, off4) = v[j];
    *at(a.reward + row * plane, off4) = 1.0f;
}

template <int N, bool STATS>
__global__ __launch_bounds__(2 * kBlock) void k_chain_split(ChainArgs a)
{
    constexpr int S = 2 * (N + 1);
    __shared__ float lds_obs[2][kChainHandSteps][S][kBlock];
    __shared__ uint16_t lds_ad[2][kChainHandSteps][kBlock];
    const uint32_t blk = xcd_block();
    const uint32_t col = threadIdx.x % kBlock;
    const uint32_t env = blk * kBlock + col;
    const bool live = env < a.n;
    uint32_t c0 = 0u, c1 = 0u, c2 = 0u, c3 = 0u;
    if (threadIdx.x < kBlock) {
        // stepping waves; threads past n step the chain at rest so that every
        // wave passes the same barriers, and record nothing the storing side keeps
        ChainCore<N, false, STATS> core(a.c, env);
        if (live) {
            core.load(a);
        } else {
#pragma unroll
            for (int j = 0; j <= N; ++j) {
                core.s.q[j] = 0.0f;
                core.s.qd[j] = 0.0f;
            }
            core.ep = 0u;
        }
        ChainHandOver<N> h{lds_obs, lds_ad, col};
        core.run(a.t0, a.K, h);
        h.flush();
        if (live) {
            core.store(a);
            c0 = core.n_eps;
            c1 = core.finished_length_sum(a.K);
            c2 = core.n_term;
            c3 = core.n_trunc;
        }
    } else {
        // storing waves: chunk c is complete after the c-th barrier
        const uint32_t off4 = env * 4u, off1 = env;
        const uint32_t n_chunks = a.K / kChainHandSteps + (a.K % kChainHandSteps != 0u ? 1u : 0u);
        for (uint32_t c = 0; c < n_chunks; ++c) {
            __syncthreads();
            const uint32_t b = c & 1u, k0 = c * kChainHandSteps, m = min(kChainHandSteps, a.K - k0);
            if (live) {
                for (uint32_t i = 0; i < m; ++i)
                    store_chain_row<N>(a, (size_t)k0 + i, off4, off1, lds_obs[b][i], lds_ad[b][i], col);
            }
        }
    }
    if (STATS) store_block_stats<2 * kBlock>(a.stats, blk, c0, c1, c2, c3);
}

// Initial state of every environment (episode beginning at step 0).
template <int N>
__global__ __launch_bounds__(kBlock) void k_reset_chain(DevParams p, uint32_t n, float* state, uint32_t* ep)
{
    const uint32_t env = blockIdx.x * kBlock + threadIdx.x;
    if (env >= n) return;
    ChainState<N> rs;
    chain_reset_draw<N>(p, env + p.env0, 0u, rs);
    const size_t plane = n;
#pragma unroll
    for (int j = 0; j <= N; ++j) {
        state[(2 * j) * plane + env] = rs.q[j];
        state[(2 * j + 1) * plane + env] = rs.qd[j];
    }
    ep[env] = 0u;
}

}  // namespace rlsim_dev
