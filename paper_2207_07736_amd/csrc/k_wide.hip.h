// k_wide.hip.h -- cart-pole with a wide padding state (D > 16 words per
// environment, the state-size factor S of the paper's "Simulator Complexity"),
// too many to keep in one thread's registers.  Each 512-step round runs the
// cart-pole loop one thread per environment and records the action and done
// bits in LDS (phase 1), then replays the padding recurrence from those bits
// with the words spread over G lanes per environment (phase 2).  The padding
// words only feed on (action, done), so the split is exact, and each word is
// still read and written once per launch per round.
#pragma once

#include "k_cartpole.hip.h"

namespace rlsim_dev {

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
    __device__ __forceinline__ void record(const CartState&, uint32_t, uint32_t) {}
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
#define RL_REP64(X)                                                                                      \
    RL_REP32(X) X(32) X(33) X(34) X(35) X(36) X(37) X(38) X(39) X(40) X(41) X(42) X(43) X(44) X(45) X(46) \
        X(47) X(48) X(49) X(50) X(51) X(52) X(53) X(54) X(55) X(56) X(57) X(58) X(59) X(60) X(61) X(62) X(63)
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
    if constexpr (N == 64) RL_REPLAY_ASM(RL_REP64);
    else if constexpr (N == 32) RL_REPLAY_ASM(RL_REP32);
    else if constexpr (N == 16) RL_REPLAY_ASM(RL_REP16);
    else if constexpr (N == 8) RL_REPLAY_ASM(RL_REP8);
    else RL_REPLAY_ASM(RL_REP4);
}

// All W words of the lane, in groups of at most kReplayGroup.
constexpr int kReplayGroup = 64;
template <int W, int O = 0>
__device__ __forceinline__ void replay_uniform(float (&s)[W], const float (&pa)[W], const float (&pb)[W],
                                               uint32_t ub, uint32_t db, uint32_t m)
{
    if constexpr (O < W) {
        constexpr int R = W - O;
        constexpr int N = R >= kReplayGroup ? kReplayGroup : R >= 32 ? 32 : R >= 16 ? 16 : R >= 8 ? 8 : 4;
        replay_uniform_group<N, O, W>(s, pa, pb, ub, db, m);
        replay_uniform<W, O + N>(s, pa, pb, ub, db, m);
    }
}

// Phase 2: G lanes per environment, W words per lane (W a multiple of 4, held
// as W / 4 float4 runs interleaved across the group's lanes).  Replays `steps`
// steps from the LDS bits for the 64 / G environments a wave covers at a time,
// for all of the wave's 64 envs.
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
    // k0 advances by the round's own length, so it never passes K (a K within
    // one round of 2^32 cannot wrap it)
    for (uint32_t k0 = 0, steps = 0; k0 < a.K; k0 += steps) {
        steps = min(kChunk, a.K - k0);
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

}  // namespace rlsim_dev
