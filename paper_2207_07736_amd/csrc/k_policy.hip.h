// k_policy.hip.h -- the simulation/inference loop with an on-device MLP policy
// fused into the K-step kernel (the paper's Future Work: simulation/inference
// fusion).  Per step every environment evaluates
//     h1 = tanh(W1 obs + b1), h2 = tanh(W2 h1 + b2), logits = W3 h2 + b3,
//     p0 = softmax(logits)[0] = 1 / (1 + exp(l1 - l0)),
// samples action 0 when u < p0 (u from Philox stream POLICY), then takes the
// cart-pole step exactly as the random-action kernel does.  On request it also
// records what an actor-critic learner reads per step: log pi(a|obs) of the
// action taken and the value head v = Wv h2 + bv on the same trunk.
//
// Matrix layout.  A wave owns 64 environments (lane = environment for the
// cart-pole state) and runs the MLP as two 32-environment column tiles of the
// transposed product  Z^T = W * H^T  (weights = MFMA A operand, activations =
// B operand, environments = N).  With the 32x32 MFMA accumulator layout (lane l,
// register i holds row 8(i/4) + 4(l/32) + (i%4) of column l%32) each lane
// already holds the values the next layer's B operand needs from it, provided
// the next layer's K index runs over hidden units in that order; the weights are
// placed in that permuted order once per workgroup (in LDS, or in registers for
// the small tables), so activations never move between lanes.  The output layer puts logit rows at 0,1 (tile 0) and 4,5
// (tile 1) so that every lane finds its own environment's logits in its own
// registers 0 and 1, and the value row at 2 (tile 0) and 6 (tile 1), register 2.
#pragma once

#include "k_cartpole.hip.h"

namespace rlsim_dev {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

struct PolicyArgs {
    const void* w1;     // [64][4]  f32 or bf16 bits
    const float* b1;    // [64] or null
    const void* w2;     // [64][64]
    const float* b2;    // [64] or null
    const void* w3;     // [2][64]
    const float* b3;    // [2] or null
    const void* wv;     // [1][64] value head or null
    const float* bv;    // [1] or null
    float* p0;          // [K][n] or null
    float* logp;        // [K][n] or null
    float* value;       // [K][n] or null
};

// log pi(a) for two logits, from d = l1 - l0: with z = l_other - l_a,
// log pi(a) = -softplus(z) = -(max(z, 0) + log(1 + e^-|z|)).  e^-|z| is in
// (0, 1], so the log term is in [0, ln 2] and neither part can overflow.
__device__ __forceinline__ float log_pi(float d, uint32_t act)
{
    const float z = act ? -d : d;
    const float e = __builtin_amdgcn_exp2f(-__builtin_fabsf(z) * 1.44269504088896340736f);
    const float l1p = __builtin_amdgcn_logf(1.0f + e) * 0.69314718055994530942f;
    return -(__builtin_fmaxf(z, 0.0f) + l1p);
}

// Hidden unit held by accumulator register i of a lane in half h (0: lanes
// 0-31, 1: lanes 32-63) of row tile M.
__device__ __forceinline__ uint32_t acc_row(uint32_t M, uint32_t i, uint32_t h)
{
    return 32u * M + 8u * (i / 4u) + 4u * h + (i % 4u);
}

__device__ __forceinline__ float tanh_fast(float x)
{
    // tanh x = 1 - 2 / (1 + e^(2x)); e^(2x) = 2^(2 x log2 e) on the exp2 unit
    const float e = __builtin_amdgcn_exp2f(x * 2.88539008177792681472f);
    return __builtin_fmaf(-2.0f, __builtin_amdgcn_rcpf(1.0f + e), 1.0f);
}

// softmax over two logits, from d = l1 - l0: p0 = 1 / (1 + e^d)
__device__ __forceinline__ float policy_p0(float d)
{
    return __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(d * 1.44269504088896340736f));
}

__device__ __forceinline__ float weight_at(const void* w, bool bf16, uint32_t idx)
{
    if (bf16) {
        const uint16_t bits = reinterpret_cast<const uint16_t*>(w)[idx];
        return __uint_as_float((uint32_t)bits << 16);
    }
    return reinterpret_cast<const float*>(w)[idx];
}

__device__ __forceinline__ __bf16 to_bf16(float x) { return (__bf16)x; }

// Per-lane accumulator initialisation with the biases of row tile M.
__device__ __forceinline__ floatx16 bias_tile(const float* lds_b, uint32_t M, uint32_t h)
{
    floatx16 c;
#pragma unroll
    for (int i = 0; i < 16; ++i) c[i] = lds_b[acc_row(M, (uint32_t)i, h)];
    return c;
}

// ---------------------------------------------------------------------------
// bf16 MLP: all three layers on v_mfma_f32_32x32x16_bf16.
// ---------------------------------------------------------------------------
struct MlpBf16 {
    bf16x8 a1[2];        // layer 1, row tiles 0/1; K = obs in k 0-3 and 8-11
    float b3_0, b3_1, bv;

    // The lanes' operand vectors, staged once per workgroup in LDS as bfloat16
    // bits, [table][lane][8]: A1 [M 2][64] (obs weights in elements 0-3, zeros
    // in 4-7), A2 [Mo 2][s 4][64], A3 [s 4][64] (rows 0,1 / 4,5 the logits, 2 / 6
    // the value, per half).  The fill reads the weights in row-major order, so
    // global loads are coalesced, and scatters each to its permuted slot; each
    // lane then reads its 16-byte vectors: A1 once per launch into registers,
    // A2 and A3 at every step (1 % faster than holding those 48 VGPRs; the kernel
    // stays at two waves per SIMD either way).
    static constexpr uint32_t kA1 = 0, kA2 = 2 * 64, kA3 = kA2 + 8 * 64, kVecs = kA3 + 4 * 64;
    static constexpr int kLds = (int)kVecs * 4;   // floats: 16 B per vector

    // Layers 2 and 3 run over K steps s = 0..3 of 16 hidden units; element j of
    // step s, for a lane in half h, is hidden unit acc_row(s / 2, 8 (s % 2) + j, h),
    // the unit that lane holds in its previous layer's accumulator.  unit_slot
    // inverts that map: the (s, j, h) that reads hidden unit c.
    __device__ static void unit_slot(uint32_t c, uint32_t& s, uint32_t& j, uint32_t& h)
    {
        const uint32_t M = c / 32u, rem = c % 32u;
        const uint32_t i = 4u * (rem / 8u) + rem % 4u;
        h = (rem % 8u) / 4u;
        s = 2u * M + i / 8u;
        j = i % 8u;
    }

    __device__ static void fill_lds(const PolicyArgs& w, float* lds)
    {
        uint16_t* t = reinterpret_cast<uint16_t*>(lds);
        uint32_t* t32 = reinterpret_cast<uint32_t*>(lds);
        for (uint32_t q = threadIdx.x; q < kVecs * 4u; q += kBlock) t32[q] = 0u;
        __syncthreads();
        const uint16_t* w1 = reinterpret_cast<const uint16_t*>(w.w1);
        const uint16_t* w2 = reinterpret_cast<const uint16_t*>(w.w2);
        const uint16_t* w3 = reinterpret_cast<const uint16_t*>(w.w3);
        const uint16_t* wv = reinterpret_cast<const uint16_t*>(w.wv);
        for (uint32_t q = threadIdx.x; q < 64u * 4u; q += kBlock) {          // W1 [64][4]
            const uint32_t r = q / 4u, c = q % 4u, M = r / 32u, col = r % 32u;
            const uint16_t v = w1[q];
            t[((kA1 + M * 64u + col) * 8u) + c] = v;
            t[((kA1 + M * 64u + 32u + col) * 8u) + c] = v;
        }
        for (uint32_t q = threadIdx.x; q < 64u * 64u; q += kBlock) {         // W2 [64][64]
            const uint32_t r = q / 64u, Mo = r / 32u, col = r % 32u;
            uint32_t s, j, h;
            unit_slot(q % 64u, s, j, h);
            t[(kA2 + (Mo * 4u + s) * 64u + 32u * h + col) * 8u + j] = w2[q];
        }
        for (uint32_t q = threadIdx.x; q < 3u * 64u; q += kBlock) {          // W3 [2][64], Wv [64]
            const uint32_t o = q / 64u;
            if (o == 2u && wv == nullptr) continue;
            const uint16_t v = o < 2u ? w3[q] : wv[q % 64u];
            uint32_t s, j, h;
            unit_slot(q % 64u, s, j, h);
            t[(kA3 + s * 64u + 32u * h + o) * 8u + j] = v;
            t[(kA3 + s * 64u + 32u * h + 4u + o) * 8u + j] = v;
        }
    }

    __device__ void load(const PolicyArgs& w, uint32_t lane, const float* lds)
    {
        const bf16x8* T = reinterpret_cast<const bf16x8*>(lds);
#pragma unroll
        for (int M = 0; M < 2; ++M) a1[M] = T[kA1 + M * 64u + lane];
        b3_0 = w.b3 ? w.b3[0] : 0.0f;
        b3_1 = w.b3 ? w.b3[1] : 0.0f;
        bv = w.bv ? w.bv[0] : 0.0f;
    }

    // Logit difference d = l1 - l0 and value v of this lane's environment; obs
    // is this lane's pre-step state.  The value row rides in the output tile at
    // no extra cost, so VAL changes nothing here.
    template <bool VAL>
    __device__ void eval(const CartState& obs, const float* lds_b1, const float* lds_b2, const float* lds,
                         uint32_t lane, float& d, float& v) const
    {
        const bf16x8* ops = reinterpret_cast<const bf16x8*>(lds);
        const uint32_t h = lane / 32u;
        const bf16x8 zero8 = {};
        bf16x8 own = zero8;
        own[0] = to_bf16(obs.x);
        own[1] = to_bf16(obs.xd);
        own[2] = to_bf16(obs.th);
        own[3] = to_bf16(obs.thd);
        float l0 = 0.0f, l1 = 0.0f, lv = 0.0f;
#pragma unroll
        for (uint32_t T = 0; T < 2u; ++T) {
            // layer 1: tile T's environments live in half T
            const bf16x8 bin = (h == T) ? own : zero8;
            floatx16 c1[2];
#pragma unroll
            for (int M = 0; M < 2; ++M)
                c1[M] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[M], bin, bias_tile(lds_b1, M, h), 0, 0, 0);
            bf16x8 b1[4];
#pragma unroll
            for (int s = 0; s < 4; ++s)
#pragma unroll
                for (int j = 0; j < 8; ++j) b1[s][j] = to_bf16(tanh_fast(c1[s / 2][8 * (s % 2) + j]));
            // layer 2
            floatx16 c2[2];
#pragma unroll
            for (int Mo = 0; Mo < 2; ++Mo) {
                c2[Mo] = bias_tile(lds_b2, Mo, h);
#pragma unroll
                for (int s = 0; s < 4; ++s)
                    c2[Mo] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ops[kA2 + (Mo * 4u + s) * 64u + lane], b1[s],
                                                                     c2[Mo], 0, 0, 0);
            }
            bf16x8 b2[4];
#pragma unroll
            for (int s = 0; s < 4; ++s)
#pragma unroll
                for (int j = 0; j < 8; ++j) b2[s][j] = to_bf16(tanh_fast(c2[s / 2][8 * (s % 2) + j]));
            // layer 3: rows 0,1,2 (tile 0) / 4,5,6 (tile 1) are registers 0,1,2 of the owning half
            floatx16 c3 = {};
            c3[0] = b3_0;
            c3[1] = b3_1;
            c3[2] = bv;
#pragma unroll
            for (int s = 0; s < 4; ++s)
                c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ops[kA3 + s * 64u + lane], b2[s], c3, 0, 0, 0);
            if (h == T) {
                l0 = c3[0];
                l1 = c3[1];
                lv = c3[2];
            }
        }
        d = l1 - l0;
        v = lv;
    }
};

// ---------------------------------------------------------------------------
// fp32 MLP: layers 1 and 2 on v_mfma_f32_32x32x2_f32, layer 3 on the VALU.
// Both column tiles go through each layer together, so layer 2 runs as four
// independent accumulation chains that keep the matrix pipeline busy.
// ---------------------------------------------------------------------------
struct MlpF32 {
    float a1[2][2];      // layer 1 [row tile][K step]: W1[32 M + lane%32][2 s + lane/32]
    float b3_0, b3_1, bv;

    // LDS, filled once per workgroup:
    //  [0, 192): output-layer weights a lane of half h needs, [output][in tile][half][register]:
    //      W3[o][acc_row(Mi, i, h)] for the logits o = 0, 1 and Wv[acc_row(Mi, i, h)]
    //      (zero without a value head) as output 2;
    //  [192, 192 + 4096): layer-2 A operands, float4 (Mo, Mi, i/4, lane) holding
    //      W2[32 Mo + lane%32][acc_row(Mi, i, lane/32)] for i%4 = 0..3, so that a
    //      wave reads 1 KB of consecutive float4s per four matrix instructions
    //      (kept out of registers: 64 fewer VGPRs, one more wave per SIMD).
    static constexpr int kW3 = 3 * 2 * 2 * 16;
    static constexpr int kW2 = 2 * 2 * 16 * 64;
    static constexpr int kLds = kW3 + kW2;
    __device__ static void fill_lds(const PolicyArgs& w, float* lds)
    {
        for (uint32_t q = threadIdx.x; q < (uint32_t)kW3; q += kBlock) {
            const uint32_t o = q / 64u, Mi = (q / 32u) % 2u, h = (q / 16u) % 2u, i = q % 16u;
            lds[q] = o < 2u ? weight_at(w.w3, false, o * 64u + acc_row(Mi, i, h))
                            : (w.wv ? weight_at(w.wv, false, acc_row(Mi, i, h)) : 0.0f);
        }
        for (uint32_t q = threadIdx.x; q < (uint32_t)kW2; q += kBlock) {
            const uint32_t r = q % 4u, lane = (q / 4u) % 64u, i4 = (q / 256u) % 4u, Mi = (q / 1024u) % 2u,
                           Mo = q / 2048u;
            lds[kW3 + q] = weight_at(w.w2, false, (32u * Mo + lane % 32u) * 64u + acc_row(Mi, 4u * i4 + r, lane / 32u));
        }
    }

    __device__ void load(const PolicyArgs& w, uint32_t lane, const float*)
    {
        const uint32_t h = lane / 32u, col = lane % 32u;
#pragma unroll
        for (int M = 0; M < 2; ++M)
#pragma unroll
            for (int s = 0; s < 2; ++s) a1[M][s] = weight_at(w.w1, false, (32u * M + col) * 4u + 2u * s + h);
        b3_0 = w.b3 ? w.b3[0] : 0.0f;
        b3_1 = w.b3 ? w.b3[1] : 0.0f;
        bv = w.bv ? w.bv[0] : 0.0f;
    }

    // Logit difference d = l1 - l0 and (if VAL) value v of this lane's environment.
    template <bool VAL>
    __device__ void eval(const CartState& obs, const float* lds_b1, const float* lds_b2, const float* lds_w3,
                         uint32_t lane, float& d, float& v) const
    {
        const uint32_t h = lane / 32u;
        // layer 1, both tiles, two K steps of 2: K slot k of step s is obs component
        // 2 s + k of the tile's environment, supplied by the lanes of half k.  A lane
        // of half h holds its own environment (tile h); for the other tile it supplies
        // the environment of lane ^ 32, exchanged once per step.
        const float own0 = h ? obs.xd : obs.x, own1 = h ? obs.thd : obs.th;    // components h, 2 + h
        const float give0 = h ? obs.x : obs.xd, give1 = h ? obs.th : obs.thd;  // the partner's h
        const float other0 = __shfl_xor(give0, 32, 64), other1 = __shfl_xor(give1, 32, 64);
        floatx16 c1[2][2];
#pragma unroll
        for (uint32_t T = 0; T < 2u; ++T)
#pragma unroll
            for (int M = 0; M < 2; ++M) {
                c1[T][M] = bias_tile(lds_b1, M, h);
                c1[T][M] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1[M][0], h == T ? own0 : other0, c1[T][M], 0, 0, 0);
                c1[T][M] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1[M][1], h == T ? own1 : other1, c1[T][M], 0, 0, 0);
            }
#pragma unroll
        for (int T = 0; T < 2; ++T)
#pragma unroll
            for (int M = 0; M < 2; ++M)
#pragma unroll
                for (int i = 0; i < 16; ++i) c1[T][M][i] = tanh_fast(c1[T][M][i]);
        // layer 2: four independent chains [tile][out row tile]
        floatx16 c2[2][2];
#pragma unroll
        for (int T = 0; T < 2; ++T)
#pragma unroll
            for (int Mo = 0; Mo < 2; ++Mo) c2[T][Mo] = bias_tile(lds_b2, Mo, h);
        const float4* lds_a2 = reinterpret_cast<const float4*>(lds_w3 + kW3);
#pragma unroll
        for (int Mi = 0; Mi < 2; ++Mi)
#pragma unroll
            for (int i4 = 0; i4 < 4; ++i4) {
                float4 w4[2];
#pragma unroll
                for (int Mo = 0; Mo < 2; ++Mo) w4[Mo] = lds_a2[((Mo * 2 + Mi) * 4 + i4) * 64 + lane];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int i = 4 * i4 + r;
#pragma unroll
                    for (int T = 0; T < 2; ++T)
#pragma unroll
                        for (int Mo = 0; Mo < 2; ++Mo) {
                            const float a = r == 0 ? w4[Mo].x : r == 1 ? w4[Mo].y : r == 2 ? w4[Mo].z : w4[Mo].w;
                            c2[T][Mo] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, c1[T][Mi][i], c2[T][Mo], 0, 0, 0);
                        }
                }
            }
        // layer 3 on the VALU: this lane's half of the hidden units, for both tiles
        float part[2][3] = {{0.0f, 0.0f, 0.0f}, {0.0f, 0.0f, 0.0f}};   // [tile][logit 0, logit 1, value]
#pragma unroll
        for (int Mi = 0; Mi < 2; ++Mi)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const float w0 = lds_w3[(0 * 2 + Mi) * 32 + h * 16 + i];
                const float w1 = lds_w3[(1 * 2 + Mi) * 32 + h * 16 + i];
                const float wv = VAL ? lds_w3[(2 * 2 + Mi) * 32 + h * 16 + i] : 0.0f;
#pragma unroll
                for (int T = 0; T < 2; ++T) {
                    const float hv = tanh_fast(c2[T][Mi][i]);
                    part[T][0] = __builtin_fmaf(w0, hv, part[T][0]);
                    part[T][1] = __builtin_fmaf(w1, hv, part[T][1]);
                    if (VAL) part[T][2] = __builtin_fmaf(wv, hv, part[T][2]);
                }
            }
        // this lane's environment is column lane%32 of tile h; the other half of
        // its hidden units was summed by lane ^ 32 as that lane's "other tile"
        const float send0 = h ? part[0][0] : part[1][0];
        const float send1 = h ? part[0][1] : part[1][1];
        const float recv0 = __shfl_xor(send0, 32, 64);
        const float recv1 = __shfl_xor(send1, 32, 64);
        const float l0 = (h ? part[1][0] : part[0][0]) + recv0 + b3_0;
        const float l1 = (h ? part[1][1] : part[0][1]) + recv1 + b3_1;
        d = l1 - l0;
        v = 0.0f;
        if (VAL) {
            const float recv2 = __shfl_xor(h ? part[0][2] : part[1][2], 32, 64);
            v = (h ? part[1][2] : part[0][2]) + recv2 + bv;
        }
    }
};

// Fused policy + cart-pole kernel.  Every lane takes part in the MLP (the
// matrix instructions need the whole wave); lanes past n_envs carry a zero
// state and store nothing.  OUT: some of the per-step policy outputs (p0,
// log pi, value) are recorded; each row pointer may still be null.
template <class Mlp, bool REC, bool STATS, bool OUT>
__global__ __launch_bounds__(kBlock) void k_policy_fused(StepArgs a, PolicyArgs w)
{
    __shared__ float lds_b1[64];
    __shared__ float lds_b2[64];
    __shared__ __align__(16) float lds_w3[Mlp::kLds];
    if (threadIdx.x < 64u) {
        lds_b1[threadIdx.x] = w.b1 ? w.b1[threadIdx.x] : 0.0f;
        lds_b2[threadIdx.x] = w.b2 ? w.b2[threadIdx.x] : 0.0f;
    }
    Mlp::fill_lds(w, lds_w3);
    __syncthreads();

    const uint32_t blk = xcd_block();
    const uint32_t env = blk * kBlock + threadIdx.x;
    const uint32_t lane = threadIdx.x % 64u;
    const bool live = env < a.n;
    const DevParams& p = a.p;

    Mlp mlp;
    mlp.load(w, lane, lds_w3);

    CartCore<REC, STATS> core(p, env);
    if (live) {
        core.load(a);
    } else {
        core.s = CartState{0.0f, 0.0f, 0.0f, 0.0f};
        core.ep = 0u;
        core.ep_start = 0u;
    }
    if (REC) core.set_rows(a, 0);
    float* p0_row = w.p0;
    float* lp_row = w.logp;
    float* v_row = w.value;
    uint4 pw = make_uint4(0u, 0u, 0u, 0u);
    NoPad nopad;
    for (uint32_t k = 0; k < a.K; ++k) {
        const uint32_t t = a.t0 + k;
        if (k == 0u || ((t + 1u) & 7u) == 0u) core.draw_reset((t + 1u) >> 3);
        if (k == 0u || (t & 3u) == 0u) pw = philox(core.gid, t >> 2, STREAM_POLICY, p.key0, p.key1);
        const float u = u24(pick_word(pw, t & 3u));
        float d, v;
        mlp.template eval<OUT>(core.s, lds_b1, lds_b2, lds_w3, lane, d, v);
        const float p0 = policy_p0(d);
        const uint32_t act = (u < p0) ? 0u : 1u;
        if (live) {
            if (OUT) {
                if (p0_row) *at(p0_row, env * 4u) = p0;
                if (lp_row) *at(lp_row, env * 4u) = log_pi(d, act);
                if (v_row) *at(v_row, env * 4u) = v;
            }
            core.step_with(act, nopad);
        }
        // row pointers stay wave-uniform: advanced outside the lane branch
        if (OUT) {
            if (p0_row) p0_row += a.n;
            if (lp_row) lp_row += a.n;
            if (v_row) v_row += a.n;
        }
        if (REC) core.advance_rows();
    }
    if (live) core.store(a);
    if (STATS) {
        const uint32_t len_sum = live ? core.finished_length_sum(a.K) : 0u;
        store_block_stats(a.stats, blk, core.n_eps, len_sum, core.n_term, core.n_trunc);
    }
}

}  // namespace rlsim_dev
