// k_wide.hip.h -- cart-pole with a wide padding state (D > 32 words per
// environment, the state-size factor S of the paper's "Simulator Complexity"),
// more than one thread's registers hold cheaply.  Each 512-step round of a block
// of 256 environments runs the cart-pole loop one thread per environment and
// records the action and done bits in LDS (phase 1); the padding recurrence is
// then replayed from those bits with each environment's words spread over the
// 64 lanes of a wave (phase 2), while the next round's phase 1 runs in other
// waves of the workgroup (k_cartpole_wide).  The padding words only feed on
// (action, done), so the split is exact, and each word is still read and
// written once per launch per round.
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
// Episode ends of one environment within one round of at most kChunk = 512
// steps, three 10-bit counts in one register: episodes ended (bits 0-9),
// terminated (10-19) and truncated (20-29).  The done byte d is term + 2 trunc.
template <bool STATS>
struct RoundCounts {
    uint32_t packed = 0u;
    __device__ __forceinline__ void add(uint32_t d)
    {
        if (STATS) packed += min(d, 1u) | ((d & 1u) << 10) | ((d & 2u) << 19);
    }
};
static_assert(kChunk < 1024u, "the per-round episode counts are 10-bit fields");

template <bool STATS>
struct BitRecorder {
    uint32_t* lds_u;     // [kChunkWords][kBlock]
    uint32_t* lds_d;
    uint32_t col;        // threadIdx.x
    uint32_t k = 0u;     // step index within the round
    uint32_t ub = 0u, db = 0u;
    RoundCounts<STATS> cnt{};
    __device__ __forceinline__ void record(const CartState&, uint32_t, uint32_t d) { cnt.add(d); }
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
// the action and done bits are scalars): for the 16 words of this lane,
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

// All 16 words of the lane in one asm block.
template <int W>
__device__ __forceinline__ void replay_uniform(float (&s)[W], const float (&pa)[W], const float (&pb)[W],
                                               uint32_t ub, uint32_t db, uint32_t m)
{
    static_assert(W == 16, "the one-environment replay holds 16 words per lane");
    constexpr int O = 0;
    uint32_t cnt;
    RL_REPLAY_ASM(RL_REP16);
}

// The same replay for E environments at once (E = 2 or 4): each lane holds W
// words of each of the E environments, and each step branches once on the E
// action bits together (a binary tree of scalar bit tests down to one of 2^E
// update paths, each E W in-place VALU updates), so the scalar work of a step
// covers E W words per lane instead of W.  The done bits of the E environments
// are tested together (their OR) and cleared out of line, each environment's
// words only when its own bit is set.
#define RM_FMA(e, i) "v_fma_f32 %[s" #e "_" #i "], %[a" #e "_" #i "], %[s" #e "_" #i "], %[b" #e "_" #i "]\n"
#define RM_MUL(e, i) "v_mul_f32 %[s" #e "_" #i "], %[a" #e "_" #i "], %[s" #e "_" #i "]\n"
#define RM_ZERO(e, i) "v_mov_b32 %[s" #e "_" #i "], 0\n"
#define RM_R4(X, e) X(e, 0) X(e, 1) X(e, 2) X(e, 3)
#define RM_R8(X, e) RM_R4(X, e) X(e, 4) X(e, 5) X(e, 6) X(e, 7)
#define RM_R16(X, e) RM_R8(X, e) X(e, 8) X(e, 9) X(e, 10) X(e, 11) X(e, 12) X(e, 13) X(e, 14) X(e, 15)
#define RM_ENV_1(R, e) R(RM_FMA, e)
#define RM_ENV_0(R, e) R(RM_MUL, e)
#define RM_CAT(a, b) a##b
// leaf of the tree: environment e's words take the FMA path when bit e of the
// leaf's code is set, the multiply path otherwise
#define RM_LEAF2(R, b0, b1) RM_CAT(RM_ENV_, b0)(R, 0) RM_CAT(RM_ENV_, b1)(R, 1)
#define RM_LEAF4(R, b0, b1, b2, b3) RM_LEAF2(R, b0, b1) RM_CAT(RM_ENV_, b2)(R, 2) RM_CAT(RM_ENV_, b3)(R, 3)
#define RM_TEST(u, lab) "s_bitcmp1_b32 %[" #u "], %[c]\n s_cbranch_scc1 " #lab "%=\n"
// every leaf but the last carries its own copy of the loop tail (done test,
// counter, loop branch), so a step takes one taken branch fewer than with a
// jump to a shared tail (262,144 envs x 500 steps: D = 256 1.73 against
// 1.84 ms, D = 512 2.43-2.47 against 2.46-2.56 ms)
#define RM_TO_TAIL                                                \
    "s_bitcmp1_b32 %[dor], %[c]\n s_cbranch_scc1 Lm_zero%=\n"     \
    "s_add_u32 %[c], %[c], 1\n s_cmp_lt_u32 %[c], %[m]\n"          \
    "s_cbranch_scc1 Lm_step%=\n s_branch Lm_end%=\n"
#define RM_CLEAR(R, e, d, next)                                  \
    "s_bitcmp1_b32 %[" #d "], %[c]\n s_cbranch_scc0 " #next "%=\n" R(RM_ZERO, e) #next "%=:\n"
#define RM_OUT_S(e, i) [s##e##_##i] "+v"(s##e[i]),
#define RM_IN_A(e, i) [a##e##_##i] "v"(a##e[i]),
#define RM_IN_B(e, i) [b##e##_##i] "v"(b##e[i]),
#define RM_TAIL                                                  \
    "Lm_tail%=:\n s_bitcmp1_b32 %[dor], %[c]\n s_cbranch_scc1 Lm_zero%=\n" \
    "Lm_next%=:\n s_add_u32 %[c], %[c], 1\n s_cmp_lt_u32 %[c], %[m]\n"   \
    "s_cbranch_scc1 Lm_step%=\n s_branch Lm_end%=\n"

#define RM_REPLAY2(R)                                                                                     \
    asm volatile("s_mov_b32 %[c], 0\n"                                                                    \
                 "Lm_step%=:\n" RM_TEST(u1, Lm_1x) RM_TEST(u0, Lm_01) RM_LEAF2(R, 0, 0) RM_TO_TAIL        \
                 "Lm_01%=:\n" RM_LEAF2(R, 1, 0) RM_TO_TAIL                                                 \
                 "Lm_1x%=:\n" RM_TEST(u0, Lm_11) RM_LEAF2(R, 0, 1) RM_TO_TAIL                              \
                 "Lm_11%=:\n" RM_LEAF2(R, 1, 1) RM_TAIL                                                    \
                 "Lm_zero%=:\n" RM_CLEAR(R, 0, d0, Lm_z0) RM_CLEAR(R, 1, d1, Lm_z1)                        \
                 "s_branch Lm_next%=\n"                                                                    \
                 "Lm_end%=:\n"                                                                             \
                 : R(RM_OUT_S, 0) R(RM_OUT_S, 1)[c] "=&s"(cnt)                                               \
                 : R(RM_IN_A, 0) R(RM_IN_A, 1) R(RM_IN_B, 0) R(RM_IN_B, 1)[u0] "s"(u[0]), [u1] "s"(u[1]),   \
                   [d0] "s"(d[0]), [d1] "s"(d[1]), [dor] "s"(dor), [m] "s"(m)                               \
                 : "scc")

#define RM_REPLAY4(R)                                                                                      \
    asm volatile("s_mov_b32 %[c], 0\n"                                                                     \
                 "Lm_step%=:\n" RM_TEST(u3, Lm_1xxx) RM_TEST(u2, Lm_01xx) RM_TEST(u1, Lm_001x)             \
                 RM_TEST(u0, Lm_0001) RM_LEAF4(R, 0, 0, 0, 0) RM_TO_TAIL                                     \
                 "Lm_0001%=:\n" RM_LEAF4(R, 1, 0, 0, 0) RM_TO_TAIL                                          \
                 "Lm_001x%=:\n" RM_TEST(u0, Lm_0011) RM_LEAF4(R, 0, 1, 0, 0) RM_TO_TAIL                     \
                 "Lm_0011%=:\n" RM_LEAF4(R, 1, 1, 0, 0) RM_TO_TAIL                                          \
                 "Lm_01xx%=:\n" RM_TEST(u1, Lm_011x) RM_TEST(u0, Lm_0101) RM_LEAF4(R, 0, 0, 1, 0) RM_TO_TAIL \
                 "Lm_0101%=:\n" RM_LEAF4(R, 1, 0, 1, 0) RM_TO_TAIL                                          \
                 "Lm_011x%=:\n" RM_TEST(u0, Lm_0111) RM_LEAF4(R, 0, 1, 1, 0) RM_TO_TAIL                     \
                 "Lm_0111%=:\n" RM_LEAF4(R, 1, 1, 1, 0) RM_TO_TAIL                                          \
                 "Lm_1xxx%=:\n" RM_TEST(u2, Lm_11xx) RM_TEST(u1, Lm_101x) RM_TEST(u0, Lm_1001)             \
                 RM_LEAF4(R, 0, 0, 0, 1) RM_TO_TAIL                                                          \
                 "Lm_1001%=:\n" RM_LEAF4(R, 1, 0, 0, 1) RM_TO_TAIL                                          \
                 "Lm_101x%=:\n" RM_TEST(u0, Lm_1011) RM_LEAF4(R, 0, 1, 0, 1) RM_TO_TAIL                     \
                 "Lm_1011%=:\n" RM_LEAF4(R, 1, 1, 0, 1) RM_TO_TAIL                                          \
                 "Lm_11xx%=:\n" RM_TEST(u1, Lm_111x) RM_TEST(u0, Lm_1101) RM_LEAF4(R, 0, 0, 1, 1) RM_TO_TAIL \
                 "Lm_1101%=:\n" RM_LEAF4(R, 1, 0, 1, 1) RM_TO_TAIL                                          \
                 "Lm_111x%=:\n" RM_TEST(u0, Lm_1111) RM_LEAF4(R, 0, 1, 1, 1) RM_TO_TAIL                     \
                 "Lm_1111%=:\n" RM_LEAF4(R, 1, 1, 1, 1) RM_TAIL                                             \
                 "Lm_zero%=:\n" RM_CLEAR(R, 0, d0, Lm_z0) RM_CLEAR(R, 1, d1, Lm_z1)                         \
                 RM_CLEAR(R, 2, d2, Lm_z2) RM_CLEAR(R, 3, d3, Lm_z3)                                         \
                 "s_branch Lm_next%=\n"                                                                     \
                 "Lm_end%=:\n"                                                                              \
                 : R(RM_OUT_S, 0) R(RM_OUT_S, 1) R(RM_OUT_S, 2) R(RM_OUT_S, 3)[c] "=&s"(cnt)                  \
                 : R(RM_IN_A, 0) R(RM_IN_A, 1) R(RM_IN_A, 2) R(RM_IN_A, 3) R(RM_IN_B, 0) R(RM_IN_B, 1)        \
                   R(RM_IN_B, 2) R(RM_IN_B, 3)[u0] "s"(u[0]), [u1] "s"(u[1]), [u2] "s"(u[2]), [u3] "s"(u[3]), \
                   [d0] "s"(d[0]), [d1] "s"(d[1]), [d2] "s"(d[2]), [d3] "s"(d[3]), [dor] "s"(dor), [m] "s"(m) \
                 : "scc")

// Steps 0 .. m-1 (1 <= m <= 32) of one 32-step bit word for E environments:
// u[e], d[e] their action and done bits (wave-uniform), s/a/b the lane's W
// words of each.
template <int E, int W>
__device__ __forceinline__ void replay_multi(float (&s0)[W], float (&s1)[W], float (&s2)[W], float (&s3)[W],
                                             const float (&a0)[W], const float (&a1)[W], const float (&a2)[W],
                                             const float (&a3)[W], const float (&b0)[W], const float (&b1)[W],
                                             const float (&b2)[W], const float (&b3)[W], const uint32_t (&u)[4],
                                             const uint32_t (&d)[4], uint32_t m)
{
    uint32_t cnt;
    const uint32_t dor = d[0] | d[1] | d[2] | d[3];
    if constexpr (E == 4 && W == 8) RM_REPLAY4(RM_R8);
    else if constexpr (E == 4 && W == 4) RM_REPLAY4(RM_R4);
    else if constexpr (E == 2 && W == 16) RM_REPLAY2(RM_R16);
    else if constexpr (E == 2 && W == 8) RM_REPLAY2(RM_R8);
    else if constexpr (E == 2 && W == 4) RM_REPLAY2(RM_R4);
    else static_assert(E == 0, "no replay for this (E, W)");
    (void)s2; (void)s3; (void)a2; (void)a3; (void)b2; (void)b3;
}

// A buffer resource over one environment's row of Dp padding words (none for
// an environment past n): loads outside it read 0 and stores outside it are
// dropped by the hardware's range check, so a wave-uniform resource and the
// lane's byte offset address every word, with no per-lane bounds test.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_rsrc(const float* row, uint32_t words)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(row), (short)0, (int)(words * 4u), 0x00020000);
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// E environments replayed together (columns col0 .. col0 + E - 1 of block
// blk): W words per lane per environment, loaded as float4 with the placement
// of replay_env.
template <int W, int E>
__device__ __forceinline__ void replay_group(const StepArgs& a, const uint32_t* lds_u, const uint32_t* lds_d,
                                             uint32_t steps, uint32_t blk, uint32_t col0)
{
    static_assert(W % 4 == 0 && (E == 2 || E == 4), "bad multi-environment replay shape");
    const uint32_t lane = threadIdx.x % 64u;
    const uint32_t chunk_words = 64u * W;
    const uint32_t n_chunks = (a.Dp + chunk_words - 1u) / chunk_words;
    uint32_t col[4], env[4];
    bool live[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        col[e] = col0 + (uint32_t)(e < E ? e : 0);
        env[e] = blk * kBlock + col[e];
        live[e] = e < E && env[e] < a.n;
    }
    // wave-uniform buffer resources over the E rows (scalar registers): each
    // load and store needs only the lane's byte offset in a VGPR
    __amdgpu_buffer_rsrc_t rs[4], ra[4], rb[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const size_t row = (size_t)env[e] * a.Dp;
        const uint32_t words = live[e] ? a.Dp : 0u;
        rs[e] = row_rsrc(a.pad_s + row, words);
        ra[e] = row_rsrc(a.pad_a + row, words);
        rb[e] = row_rsrc(a.pad_b + row, words);
    }
    for (uint32_t c = 0; c < n_chunks; ++c) {
        const uint32_t base = c * chunk_words + 4u * lane;
        float s[4][W], pa[4][W], pb[4][W];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
#pragma unroll
            for (int i = 0; i < W; i += 4) {
                const uint32_t jb = 4u * (base + (uint32_t)(i / 4) * 256u);
                u32x4 vs = {0u, 0u, 0u, 0u}, va = vs, vb = vs;
                if (e < E) {
                    vs = __builtin_amdgcn_raw_buffer_load_b128(rs[e], jb, 0, 0);
                    va = __builtin_amdgcn_raw_buffer_load_b128(ra[e], jb, 0, 0);
                    vb = __builtin_amdgcn_raw_buffer_load_b128(rb[e], jb, 0, 0);
                }
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    s[e][i + q] = __uint_as_float(vs[q]);
                    pa[e][i + q] = __uint_as_float(va[q]);
                    pb[e][i + q] = __uint_as_float(vb[q]);
                }
            }
        }
        for (uint32_t w32 = 0; w32 * 32u < steps; ++w32) {
            uint32_t ub[4], db[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                ub[e] = e < E ? __builtin_amdgcn_readfirstlane(lds_u[w32 * kBlock + col[e]]) : 0u;
                db[e] = e < E ? __builtin_amdgcn_readfirstlane(lds_d[w32 * kBlock + col[e]]) : 0u;
            }
            const uint32_t m = __builtin_amdgcn_readfirstlane(min(32u, steps - w32 * 32u));
            replay_multi<E, W>(s[0], s[1], s[2], s[3], pa[0], pa[1], pa[2], pa[3], pb[0], pb[1], pb[2], pb[3], ub,
                               db, m);
        }
#pragma unroll
        for (int e = 0; e < E; ++e) {
#pragma unroll
            for (int i = 0; i < W; i += 4) {
                const uint32_t jb = 4u * (base + (uint32_t)(i / 4) * 256u);
                const u32x4 v = {__float_as_uint(s[e][i]), __float_as_uint(s[e][i + 1]), __float_as_uint(s[e][i + 2]),
                                 __float_as_uint(s[e][i + 3])};
                __builtin_amdgcn_raw_buffer_store_b128(v, rs[e], jb, 0, 0);
            }
        }
    }
}

// Phase 2, one environment per wave at a time: the lane holds W words (W a
// multiple of 4, as W / 4 float4 runs: float4 q of lane l holds words
// 4 l + 256 q .. +3 of a 64 W-word chunk, so each float4 load and store of the
// wave covers 1 KB contiguously), and the bits are wave-uniform, so each step
// is a scalar branch and one FMA or multiply per word.  replay_env replays
// column col of block blk.
template <int W>
__device__ __forceinline__ void replay_env(const StepArgs& a, const uint32_t* lds_u, const uint32_t* lds_d,
                                           uint32_t steps, uint32_t blk, uint32_t col)
{
    static_assert(W % 4 == 0, "bad wide-padding shape");
    const uint32_t lane = threadIdx.x % 64u;
    const uint32_t chunk_words = 64u * W;
    const uint32_t n_chunks = (a.Dp + chunk_words - 1u) / chunk_words;
    const uint32_t env = blk * kBlock + col;
    const size_t row = (size_t)env * a.Dp;
    const uint32_t words = env < a.n ? a.Dp : 0u;
    const __amdgpu_buffer_rsrc_t rs = row_rsrc(a.pad_s + row, words), ra = row_rsrc(a.pad_a + row, words),
                                 rb = row_rsrc(a.pad_b + row, words);
    for (uint32_t c = 0; c < n_chunks; ++c) {
        const uint32_t base = c * chunk_words + 4u * lane;
        float s[W], pa[W], pb[W];
#pragma unroll
        for (int i = 0; i < W; i += 4) {
            const uint32_t jb = 4u * (base + (uint32_t)(i / 4) * 256u);
            const u32x4 vs = __builtin_amdgcn_raw_buffer_load_b128(rs, jb, 0, 0);
            const u32x4 va = __builtin_amdgcn_raw_buffer_load_b128(ra, jb, 0, 0);
            const u32x4 vb = __builtin_amdgcn_raw_buffer_load_b128(rb, jb, 0, 0);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                s[i + q] = __uint_as_float(vs[q]);
                pa[i + q] = __uint_as_float(va[q]);
                pb[i + q] = __uint_as_float(vb[q]);
            }
        }
        for (uint32_t w32 = 0; w32 * 32u < steps; ++w32) {
            const uint32_t ub = lds_u[w32 * kBlock + col];
            const uint32_t db = lds_d[w32 * kBlock + col];
            const uint32_t m = min(32u, steps - w32 * 32u);
            replay_uniform<W>(s, pa, pb, __builtin_amdgcn_readfirstlane(ub), __builtin_amdgcn_readfirstlane(db),
                              __builtin_amdgcn_readfirstlane(m));
        }
#pragma unroll
        for (int i = 0; i < W; i += 4) {
            const uint32_t jb = 4u * (base + (uint32_t)(i / 4) * 256u);
            const u32x4 v = {__float_as_uint(s[i]), __float_as_uint(s[i + 1]), __float_as_uint(s[i + 2]),
                             __float_as_uint(s[i + 3])};
            __builtin_amdgcn_raw_buffer_store_b128(v, rs, jb, 0, 0);
        }
    }
}

// ---------------------------------------------------------------------------
// One padding word per lane (at most 64 words), eight environments per step.
// ---------------------------------------------------------------------------
constexpr uint32_t kJtGroup = 8;                     // environments per replay group

// Phase-1 hook for the jump-table replay: each step's action and done bits of
// the wave's 64 environments (one ballot each), kept as one byte per group of
// eight consecutive environments -- bit e of byte g is environment 8 g + e of
// the wave -- in LDS rows [group][step].  Lane g of a wave writes its group's
// bytes; a group with a live environment has a live writer (environments past n
// are the wave's last lanes).
template <bool STATS>
struct ByteRecorder {
    uint8_t* lds_u;      // [kBlock / kJtGroup][kChunk]
    uint8_t* lds_d;
    uint32_t lane, wave;
    uint32_t k = 0u;     // step index within the round
    RoundCounts<STATS> cnt{};
    __device__ __forceinline__ void record(const CartState&, uint32_t, uint32_t d) { cnt.add(d); }
    __device__ __forceinline__ void operator()(uint32_t act, bool reset)
    {
        const uint64_t ub = __builtin_amdgcn_ballot_w64(act != 0u);
        const uint64_t db = __builtin_amdgcn_ballot_w64(reset);
        if (lane < 64u / kJtGroup) {
            const uint32_t row = (wave * (64u / kJtGroup) + lane) * kChunk + k;
            lds_u[row] = (uint8_t)(ub >> (kJtGroup * lane));
            lds_d[row] = (uint8_t)(db >> (kJtGroup * lane));
        }
        ++k;
    }
    __device__ __forceinline__ void flush() {}
};

// The replay of up to 32 steps of one group in one asm block.  Step c reads
// its action byte (byte c % 4 of u[c / 4]) and jumps with s_swappc_b64 to leaf
// number byte of a table of 256 leaves, each eight in-place updates -- the
// word of environment e takes v_fma_f32 (one rounding) when bit e is set and
// v_mul_f32 otherwise -- that returns with s_setpc_b64; every leaf is 68 bytes
// (eight 8-byte VOP3 instructions and the return), so leaf i starts at table +
// 68 i.  A nonzero done byte calls the clearing routine, which zeroes the words
// of the environments whose bit is set.  The 32 steps are unrolled; a second
// copy tests the step count m before each step, for a last, partial word.
// s36..s45 hold the table and routine addresses and the return addresses.
#define JT_M(e) "v_mul_f32_e64 %[s" #e "], %[a" #e "], %[s" #e "]\n"
#define JT_F(e) "v_fma_f32 %[s" #e "], %[a" #e "], %[s" #e "], %[b" #e "]\n"
#define JT_OP0(e) JT_M(e)
#define JT_OP1(e) JT_F(e)
#define JT_LEAF(b0, b1, b2, b3, b4, b5, b6, b7)                                                            \
    JT_OP##b0(0) JT_OP##b1(1) JT_OP##b2(2) JT_OP##b3(3) JT_OP##b4(4) JT_OP##b5(5) JT_OP##b6(6) JT_OP##b7(7) \
        "s_setpc_b64 s[44:45]\n"
#define JT_T0(b1, b2, b3, b4, b5, b6, b7) JT_LEAF(0, b1, b2, b3, b4, b5, b6, b7) JT_LEAF(1, b1, b2, b3, b4, b5, b6, b7)
#define JT_T1(b2, b3, b4, b5, b6, b7) JT_T0(0, b2, b3, b4, b5, b6, b7) JT_T0(1, b2, b3, b4, b5, b6, b7)
#define JT_T2(b3, b4, b5, b6, b7) JT_T1(0, b3, b4, b5, b6, b7) JT_T1(1, b3, b4, b5, b6, b7)
#define JT_T3(b4, b5, b6, b7) JT_T2(0, b4, b5, b6, b7) JT_T2(1, b4, b5, b6, b7)
#define JT_T4(b5, b6, b7) JT_T3(0, b5, b6, b7) JT_T3(1, b5, b6, b7)
#define JT_T5(b6, b7) JT_T4(0, b6, b7) JT_T4(1, b6, b7)
#define JT_T6(b7) JT_T5(0, b7) JT_T5(1, b7)
#define JT_TABLE JT_T6(0) JT_T6(1)
// one step: leaf call, then the done byte (SCC = byte != 0) and the call of
// the clearing routine through an out-of-line stub
#define JT_STEP(P, c, w, bc)                                     \
    "s_bfe_u32 s40, %[u" #w "], " #bc "\n"                      \
    "s_mul_i32 s40, s40, 68\n"                                   \
    "s_add_u32 s42, s36, s40\n"                                  \
    "s_addc_u32 s43, s37, 0\n"                                   \
    "s_swappc_b64 s[44:45], s[42:43]\n"                          \
    "s_bfe_u32 s41, %[d" #w "], " #bc "\n"                      \
    "s_cbranch_scc1 Lj" #P "c" #c "_%=\n"                        \
    "Lj" #P "r" #c "_%=:\n"
#define JT_PSTEP(c, w, bc) "s_cmp_le_u32 %[m], " #c "\n s_cbranch_scc1 Ljend%=\n" JT_STEP(p, c, w, bc)
#define JT_STUB(P, c) "Lj" #P "c" #c "_%=:\n s_swappc_b64 s[44:45], s[38:39]\n s_branch Lj" #P "r" #c "_%=\n"
#define JT_WORD(X, P, w, c0, c1, c2, c3) \
    X(P, c0, w, 0x80000) X(P, c1, w, 0x80008) X(P, c2, w, 0x80010) X(P, c3, w, 0x80018)
#define JT_FSTEP(P, c, w, bc) JT_STEP(P, c, w, bc)
#define JT_PSTEPX(P, c, w, bc) JT_PSTEP(c, w, bc)
#define JT_STEPS(X, P)                                                                                   \
    JT_WORD(X, P, 0, 0, 1, 2, 3) JT_WORD(X, P, 1, 4, 5, 6, 7) JT_WORD(X, P, 2, 8, 9, 10, 11)               \
        JT_WORD(X, P, 3, 12, 13, 14, 15) JT_WORD(X, P, 4, 16, 17, 18, 19) JT_WORD(X, P, 5, 20, 21, 22, 23) \
            JT_WORD(X, P, 6, 24, 25, 26, 27) JT_WORD(X, P, 7, 28, 29, 30, 31)
#define JT_STUBS(P)                                                                                       \
    JT_STUB(P, 0) JT_STUB(P, 1) JT_STUB(P, 2) JT_STUB(P, 3) JT_STUB(P, 4) JT_STUB(P, 5) JT_STUB(P, 6)      \
        JT_STUB(P, 7) JT_STUB(P, 8) JT_STUB(P, 9) JT_STUB(P, 10) JT_STUB(P, 11) JT_STUB(P, 12)             \
            JT_STUB(P, 13) JT_STUB(P, 14) JT_STUB(P, 15) JT_STUB(P, 16) JT_STUB(P, 17) JT_STUB(P, 18)      \
                JT_STUB(P, 19) JT_STUB(P, 20) JT_STUB(P, 21) JT_STUB(P, 22) JT_STUB(P, 23) JT_STUB(P, 24)  \
                    JT_STUB(P, 25) JT_STUB(P, 26) JT_STUB(P, 27) JT_STUB(P, 28) JT_STUB(P, 29)             \
                        JT_STUB(P, 30) JT_STUB(P, 31)
#define JT_CLR(e) "s_bitcmp1_b32 s41, " #e "\n s_cbranch_scc0 Ljz" #e "_%=\n v_mov_b32 %[s" #e "], 0\nLjz" #e "_%=:\n"
#define JT_INA(e) [a##e] "v"(pa[e]),
#define JT_INB(e) [b##e] "v"(pb[e]),
#define JT_INU(e) [u##e] "s"(u[e]),
#define JT_IND(e) [d##e] "s"(d[e]),
#define JT_R8(X) X(0) X(1) X(2) X(3) X(4) X(5) X(6) X(7)

__device__ __forceinline__ void replay_jt(float (&s)[8], const float (&pa)[8], const float (&pb)[8],
                                          const uint32_t (&u)[8], const uint32_t (&d)[8], uint32_t m)
{
    asm volatile("s_getpc_b64 s[36:37]\n"
                 "Ljbase0_%=:\n"
                 "s_add_u32 s36, s36, Ljtab%= - Ljbase0_%=\n"
                 "s_addc_u32 s37, s37, 0\n"
                 "s_getpc_b64 s[38:39]\n"
                 "Ljbase1_%=:\n"
                 "s_add_u32 s38, s38, Ljclr%= - Ljbase1_%=\n"
                 "s_addc_u32 s39, s39, 0\n"
                 "s_cmp_eq_u32 %[m], 32\n"
                 "s_cbranch_scc0 Ljpart%=\n"
                 JT_STEPS(JT_FSTEP, f)
                 "s_branch Ljend%=\n"
                 "Ljpart%=:\n"
                 JT_STEPS(JT_PSTEPX, p)
                 "s_branch Ljend%=\n"
                 JT_STUBS(f) JT_STUBS(p)
                 "Ljclr%=:\n" JT_R8(JT_CLR) "s_setpc_b64 s[44:45]\n"
                 "Ljtab%=:\n" JT_TABLE
                 "Ljend%=:\n"
                 : [s0] "+v"(s[0]), [s1] "+v"(s[1]), [s2] "+v"(s[2]), [s3] "+v"(s[3]), [s4] "+v"(s[4]),
                   [s5] "+v"(s[5]), [s6] "+v"(s[6]), [s7] "+v"(s[7])
                 : JT_R8(JT_INA) JT_R8(JT_INB) JT_R8(JT_INU) JT_R8(JT_IND)[m] "s"(m)
                 : "scc", "s36", "s37", "s38", "s39", "s40", "s41", "s42", "s43", "s44", "s45");
}

// Phase 2 of group g (columns 8 g .. 8 g + 7 of block blk): lane l holds word
// l of each of the eight environments.  Row addresses are recomputed at the
// store rather than held through the replay (fewer live registers).
__device__ __forceinline__ void replay_group_jt(const StepArgs& a, const uint8_t* lds_u, const uint8_t* lds_d,
                                                uint32_t steps, uint32_t blk, uint32_t g)
{
    const uint32_t lane = threadIdx.x % 64u;
    const uint32_t env0 = blk * kBlock + g * kJtGroup;
    const bool lane_on = lane < a.Dp;
    float s[8], pa[8], pb[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const bool on = lane_on && env0 + (uint32_t)e < a.n;
        const size_t row = (size_t)(env0 + (uint32_t)e) * a.Dp;
        s[e] = on ? a.pad_s[row + lane] : 0.0f;
        pa[e] = on ? a.pad_a[row + lane] : 0.0f;
        pb[e] = on ? a.pad_b[row + lane] : 0.0f;
    }
    for (uint32_t w32 = 0; w32 * 32u < steps; ++w32) {
        const uint32_t* pu = reinterpret_cast<const uint32_t*>(lds_u + g * kChunk + w32 * 32u);
        const uint32_t* pd = reinterpret_cast<const uint32_t*>(lds_d + g * kChunk + w32 * 32u);
        uint32_t u[8], d[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            u[q] = __builtin_amdgcn_readfirstlane(pu[q]);
            d[q] = __builtin_amdgcn_readfirstlane(pd[q]);
        }
        replay_jt(s, pa, pb, u, d, __builtin_amdgcn_readfirstlane(min(32u, steps - w32 * 32u)));
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const size_t row = (size_t)(env0 + (uint32_t)e) * a.Dp;
        if (lane_on && env0 + (uint32_t)e < a.n) a.pad_s[row + lane] = s[e];
    }
}

// k_cartpole_wide<W, E, NW>: the two phases, overlapped across the blocks of a
// persistent workgroup of NW waves (two workgroups per CU; workgroup g takes
// the 256-env blocks g, g + G, ... of a grid of G).  A work item is one 512-step
// round of one block, and the workgroup's items are its blocks round by round.
// In iteration j the first four waves run phase 1 of item j (the cart-pole loop
// with its trajectory stores, the action and done bits into LDS slot j & 1);
// the other waves replay item j - 1 from slot (j - 1) & 1, taking
// E-environment groups from an LDS counter; one workgroup barrier ends the
// iteration.  The stepping waves join the replay after the workgroup's last
// item: their cart-pole state and the replay's words then never share
// registers, which keeps the kernel within the 64 VGPRs of eight waves per SIMD.  Phase 1 of one block thus runs beside the replay
// of the one before it, and only the first item's phase 1 is exposed (262,144
// envs x 500 steps against the same phases run one after the other in 256-env
// workgroups: D = 512 2.11 against 2.45 ms, D = 2,048 6.33 against 8.59 ms).
// Block statistics go through LDS slot m & 1 of the workgroup's m-th block and
// are written out by wave 4 in the iteration after the block's last item.
// Two workgroups run per CU, eight waves per SIMD: the replay's scalar bit
// tests and branches, not its vector updates, set its pace, and more waves
// hide more of them (D = 64 0.88-0.93 against 0.99-1.05 ms with one workgroup,
// D = 512 2.00-2.04 against 2.17-2.29 ms).
template <int W, int E, int NW, bool REC, bool STATS>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(8)))
void k_cartpole_wide(StepArgs a)
{
    static_assert(NW >= 8 && NW <= 16, "the pipeline needs four stepping waves and at least four more");
    static_assert(W == 1 || W == 4 || W == 8 || W == 16, "shapes that fit 64 VGPRs");
    static_assert(W != 1 || E == (int)kJtGroup, "one word per lane takes the eight-environment jump table");
    __shared__ uint32_t lds_u[2][kChunkWords * kBlock];
    __shared__ uint32_t lds_d[2][kChunkWords * kBlock];
    __shared__ uint32_t next_group[2];
    __shared__ uint32_t blk_stats[2][4];
    const uint32_t G = gridDim.x, wg = blockIdx.x;
    const uint32_t n_blocks = (a.n + kBlock - 1u) / kBlock;
    const uint32_t my_blocks = wg < n_blocks ? (n_blocks - wg + G - 1u) / G : 0u;
    const uint32_t rounds = (a.K + kChunk - 1u) / kChunk;
    const uint32_t n_items = my_blocks * rounds;
    const uint32_t wave = threadIdx.x / 64u, lane = threadIdx.x % 64u;
    if (threadIdx.x < 8u) {
        blk_stats[threadIdx.x / 4u][threadIdx.x % 4u] = 0u;
        if (threadIdx.x < 2u) next_group[threadIdx.x] = 0u;
    }
    __syncthreads();

    // this wave's share of the replay of item i: groups of E columns taken
    // from the counter of slot i & 1 until none is left
    auto replay_item = [&](uint32_t i) {
        const uint32_t m = i / rounds, r = i % rounds;
        // wave-uniform by construction; readfirstlane keeps the compiler from
        // merging it with the same sum computed under the statistics' lane test,
        // which would make it, and every row address after it, per-lane
        const uint32_t blk = __builtin_amdgcn_readfirstlane(wg + m * G);
        const uint32_t k0 = r * kChunk, steps = min(kChunk, a.K - k0);
        const uint32_t cols = min((uint32_t)kBlock, a.n - blk * kBlock);
        const uint32_t n_groups = (cols + (uint32_t)E - 1u) / (uint32_t)E;
        const uint32_t sl = i & 1u;
        for (;;) {
            uint32_t g = 0u;
            if (lane == 0u) g = atomicAdd(&next_group[sl], 1u);
            g = __builtin_amdgcn_readfirstlane(g);
            if (g >= n_groups) break;
            if constexpr (W == 1)
                replay_group_jt(a, reinterpret_cast<const uint8_t*>(lds_u[sl]),
                                reinterpret_cast<const uint8_t*>(lds_d[sl]), steps, blk, g);
            else if constexpr (E > 1) replay_group<W, E>(a, lds_u[sl], lds_d[sl], steps, blk, g * (uint32_t)E);
            else replay_env<W>(a, lds_u[sl], lds_d[sl], steps, blk, g);
        }
    };

    if (wave < 4u) {
        // stepping waves: phase 1 of every item, in order, then their share of
        // the last item's replay
        const uint32_t col = threadIdx.x;
        uint32_t j = 0u;
        for (uint32_t m = 0; m < my_blocks; ++m) {
            const uint32_t blk = wg + m * G;
            const uint32_t env = blk * kBlock + col;
            const bool live = env < a.n;
            // the episode counts go through the recorder and LDS, not the core,
            // which keeps them out of the stepping loop's registers
            CartCore<REC, false> core(a.p, env);
            if (live) core.load(a);
            if (STATS) {
                // the block's finished episode lengths: the episode counters at the
                // start plus K per environment, minus the counters at the end
                const uint32_t e0 = wave_sum(live ? core.ep : 0u);
                const uint32_t nl = (uint32_t)__builtin_popcountll(__builtin_amdgcn_ballot_w64(live));
                if (lane == 0u) atomicAdd(&blk_stats[m & 1u][1], e0 + nl * a.K);
            }
            for (uint32_t r = 0; r < rounds; ++r, ++j) {
                const uint32_t k0 = r * kChunk, steps = min(kChunk, a.K - k0);
                // slot j & 1's counter was last used in iteration j - 1
                if (threadIdx.x == 0u) next_group[j & 1u] = 0u;
                uint32_t counts = 0u;
                if (live) {
                    if (REC) core.set_rows(a, k0);
                    if constexpr (W == 1) {
                        ByteRecorder<STATS> rec{reinterpret_cast<uint8_t*>(lds_u[j & 1u]),
                                                reinterpret_cast<uint8_t*>(lds_d[j & 1u]), lane, wave};
                        core.run(a.t0 + k0, steps, rec);
                        counts = rec.cnt.packed;
                    } else {
                        BitRecorder<STATS> rec{lds_u[j & 1u], lds_d[j & 1u], col};
                        core.run(a.t0 + k0, steps, rec);
                        rec.flush();
                        counts = rec.cnt.packed;
                    }
                }
                if (STATS) {
                    // a wave's sums of the 10-bit fields fit 16 bits (64 x 512)
                    const uint32_t lo = wave_sum((counts & 1023u) | (((counts >> 10) & 1023u) << 16));
                    const uint32_t hi = wave_sum(counts >> 20);
                    if (lane == 0u) {
                        atomicAdd(&blk_stats[m & 1u][0], lo & 0xFFFFu);
                        atomicAdd(&blk_stats[m & 1u][2], lo >> 16);
                        atomicAdd(&blk_stats[m & 1u][3], hi);
                    }
                }
                if (r + 1u == rounds) {
                    if (live) core.store(a);
                    if (STATS) {
                        const uint32_t e1 = wave_sum(live ? core.ep : 0u);
                        if (lane == 0u) atomicAdd(&blk_stats[m & 1u][1], 0u - e1);
                    }
                }
                __syncthreads();
            }
        }
        replay_item(n_items - 1u);
        __syncthreads();
    } else {
        for (uint32_t j = 0; j <= n_items; ++j) {
            // the statistics of a block whose last item was stepped in iteration j - 1
            if (STATS && j >= 1u && (j - 1u) % rounds == rounds - 1u && threadIdx.x < 4u * 64u + 4u &&
                threadIdx.x >= 4u * 64u) {
                const uint32_t m = (j - 1u) / rounds, q = threadIdx.x - 4u * 64u;
                a.stats[(size_t)(wg + m * G) * 4u + q] = blk_stats[m & 1u][q];
                blk_stats[m & 1u][q] = 0u;
            }
            if (j >= 1u) replay_item(j - 1u);
            __syncthreads();
        }
    }
}

}  // namespace rlsim_dev
