/*
 * rlsim.h -- C ABI of the GPU-vectorised, kernel-fused cart-pole data collector.
 *
 * The operation is the data-collection loop of Gleeson et al., "Optimizing Data
 * Collection in Deep Reinforcement Learning" (2022): N simulator instances are
 * stepped together on the GPU (section "GPU Vectorization"), K consecutive
 * simulation steps run inside one kernel launch with the simulator state held
 * in registers (section "Simulator Kernel Fusion"), and each step feeds the
 * state to a policy whose action drives the next state and reward (Background,
 * "RL Training" and the data-collection figure).  The simulator is cart-pole
 * (Background, "Cartpole Simulator"), optionally widened by D extra state words
 * per environment (the state-size factor S of "Simulator Complexity"), or a
 * heavier multi-body simulator, a cart carrying a chain of N uniform rods (the
 * kind of simulator the paper's Future Work points to).
 *
 * Conventions for every call:
 *  - Returns RLSIM_OK (0) or a negative rlsim_status; rlsim_last_error() gives
 *    the message.  No exception crosses the ABI.
 *  - A handle is not thread-safe.  The library owns the simulator state (device
 *    memory it allocates in rlsim_create and frees in rlsim_destroy); the caller
 *    owns every buffer it passes in and the library never frees or keeps them.
 *  - Work is enqueued asynchronously on the handle's HIP stream (cfg.stream);
 *    only rlsim_get_state, rlsim_set_state and rlsim_destroy synchronise it.
 *    A kernel fault surfaces as RLSIM_EDEVICE at a later call.
 *  - "Device pointer" means memory the current HIP device can access (hipMalloc,
 *    torch tensors on that device).  Host pointers are plain process memory.
 */
#ifndef RLSIM_H
#define RLSIM_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    RLSIM_OK = 0,
    RLSIM_EINVAL = -1,       /* bad argument: sizes, NULLs, alignment, ranges */
    RLSIM_ENOMEM = -2,       /* device allocation failed */
    RLSIM_EDEVICE = -3,      /* a HIP runtime call failed (message has its text) */
    RLSIM_ESTATE = -4,       /* call not valid in the handle's state (step before reset) */
    RLSIM_EUNSUPPORTED = -5  /* valid request this build does not implement */
} rlsim_status;

enum { RLSIM_F32 = 0, RLSIM_BF16 = 1 };       /* rlsim_policy.dtype */
enum { RLSIM_F_NO_TERMINATION = 1u };         /* rlsim_cfg.flags: thresholds never fire */
enum { RLSIM_MODEL_CARTPOLE = 0u, RLSIM_MODEL_CHAIN = 1u };   /* rlsim_cfg.model */

typedef struct rlsim rlsim_t;                 /* opaque handle */

/* Simulator constants (fp32; the paper cites cart-pole but prints none) and the
 * stream the handle enqueues on.  rlsim_cfg_default fills the classic values:
 * g = 9.8, cart 1.0, pole 0.1, half length 0.5, force 10, tau 0.02, |x| limit
 * 2.4, |theta| limit = fp32(12 * 2 pi / 360), 500-step episodes, reset box
 * [-0.05, 0.05), padding a in [0.9, 0.99), b in [-1, 1), flags 0, compute
 * factor 1, env0 0, the cart-pole model, stream NULL.
 *
 * sin and cos of an angle are a degree-9/8 series on |angle| <= fp32(pi/4)
 * (every angle of a live cart-pole episode) and the same series after a
 * quadrant reduction beyond it, so every angle is valid (within 2.5e-7 of the
 * true sine and cosine).
 *
 * Reset draws are keyed by the 8-step block of the step an episode begins at
 * ((t+1) / 8 after an episode ends at step t; block 0 at rlsim_reset).  Two
 * episodes of one environment that begin in the same block therefore start
 * from the same state.  That needs an episode shorter than 8 steps: none is
 * with the default constants, but a time limit below 8 (or a much larger
 * force or step) makes it happen, as a defined part of the result.
 *
 * The chain model (model = RLSIM_MODEL_CHAIN, n_links = N in [1, 4]): a cart of
 * mass masscart carrying N identical uniform rods of mass masspole and length
 * 2 half_length, joined end to end; the state words are (x, x_dot, phi_1,
 * phi_1_dot, ..., phi_N, phi_N_dot), phi_k the angle of link k from the
 * upward vertical; termination is |x| > x_threshold or any
 * |phi_k| > theta_threshold_rad.  Every other constant means what it means for
 * the cart-pole. */
typedef struct {
    float gravity, masscart, masspole, half_length, force_mag, tau;
    float x_threshold, theta_threshold_rad;
    uint32_t max_episode_steps;            /* 0 = no time limit */
    float reset_low, reset_high;           /* initial-state box, each word */
    float pad_a_low, pad_a_high;           /* padding decay a_j */
    float pad_b_low, pad_b_high;           /* padding gain b_j */
    uint32_t flags;                        /* RLSIM_F_* */
    uint32_t compute_factor;               /* C >= 1: each step is C Euler iterations of
                                              length tau / C (the paper's compute factor,
                                              "Simulator Complexity"); default 1 */
    uint32_t env0;                         /* global id of environment 0: a handle holding
                                              global environments env0 .. env0 + n - 1 of
                                              a larger batch (one shard of the paper's N
                                              vectorised simulators, "GPU Vectorization")
                                              draws the same random numbers as those
                                              environments of a single handle; a multiple
                                              of 256; default 0 */
    uint32_t model;                        /* RLSIM_MODEL_CARTPOLE or RLSIM_MODEL_CHAIN */
    uint32_t n_links;                      /* chain model: links N in [1, 4]; else ignored */
    void* stream;                          /* hipStream_t; NULL = default stream */
} rlsim_cfg;

/* Fill *cfg with the defaults above.  NULL cfg: no effect. */
void rlsim_cfg_default(rlsim_cfg* cfg);

/* Create a simulator of n_envs environments on the current HIP device (the
 * paper's N simulator instances, "GPU Vectorization").  Cart-pole:
 * state_words = 4 + D fp32 words each, the 4 cart-pole words x, x_dot, theta,
 * theta_dot then D padding words, D being the state-size factor S of
 * "Simulator Complexity"; about (20 + 12 D) bytes per environment.  Chain
 * model: state_words = 2 n_links + 2 exactly.  Allocates the state on the
 * device.  cfg may be NULL (defaults).
 * Errors: EINVAL if out == NULL, n_envs == 0 or n_envs > 2^30, state_words < 4
 * or state_words > 2^24 + 4 (or != 2 n_links + 2 for the chain), a non-finite
 * or inconsistent constant (masses <= 0, half_length <= 0,
 * reset_low > reset_high, compute_factor == 0, env0 not a multiple of 256,
 * env0 + n_envs > 2^32, an unknown model, n_links outside [1, 4] for the
 * chain, ...); ENOMEM; EDEVICE.  On error *out is NULL. */
int rlsim_create(uint32_t n_envs, uint32_t state_words, const rlsim_cfg* cfg, rlsim_t** out);

/* Start every environment's first episode at global step t = 0 (Background,
 * "RL Training": the loop's initial simulator state).  The state is drawn from
 * Philox4x32-10 keyed by seed (stream RESET; counters use global environment
 * ids env0 + i), the episode counters are zeroed, the padding words set to +0
 * and their parameters a_j, b_j drawn (stream PARAMS).  Enqueues one kernel
 * per state array; does not synchronise.
 * Errors: EINVAL (h NULL), EDEVICE. */
int rlsim_reset(rlsim_t* h, uint64_t seed);

/* Caller-owned DEVICE buffers receiving rows 0..K-1 of one rlsim_step_fused
 * call; row k holds global step t + k.  Layout is structure-of-arrays so that
 * consecutive environments are consecutive addresses:
 *   obs        [K][S][n_envs] f32  state before the step; S = 4 (x, x_dot, th,
 *              th_dot) for the cart-pole, 2 n_links + 2 for the chain
 *   action     [K][n_envs]    u8   0 = push towards -x, 1 = towards +x
 *   reward     [K][n_envs]    f32  1.0 every step
 *   done       [K][n_envs]    u8   bit 0 terminated, bit 1 time limit reached
 *   block_stats[ceil(n_envs/256)][4] u32, optional, overwritten each call:
 *              per 256-environment block {episodes finished, sum of their
 *              lengths, terminated, truncated} over this call's K steps
 *   policy_p0  [K][n_envs]    f32  optional; policy runs only: the policy's
 *              probability of action 0 at each step
 *   logp       [K][n_envs]    f32  optional; policy runs only: log pi(a|obs) of
 *              the action taken, log softmax(logits)[a]
 *   value      [K][n_envs]    f32  optional; policy runs with a value head only:
 *              v(obs) = wv . h2 + bv
 * logp and value are what an actor-critic learner reads beside the trajectory
 * (the data-collection loop forms the learner's training data, Background,
 * "RL Training"); the caller's tensors are the learner's input as they stand.
 * obs, action, reward and done are all set or all NULL (no trajectory). */
typedef struct {
    float* obs;
    uint8_t* action;
    float* reward;
    uint8_t* done;
    uint32_t* block_stats;
    float* policy_p0;
    float* logp;
    float* value;
} rlsim_traj;

/* Caller-owned DEVICE weights of the MLP policy 4 -> 64 -> 64 -> 2 (tanh hidden
 * layers; the inference half of the simulation/inference loop, fused with the
 * simulator as the paper's Future Work proposes) and of an optional value head
 * 64 -> 1 on the second hidden layer h2.  Weights are row-major [out][in] in
 * dtype (RLSIM_F32: float, RLSIM_BF16: bfloat16 bits as uint16); biases are
 * always float and may be NULL (zero).  wv NULL = no value head. */
typedef struct {
    int dtype;
    const void* w1; const float* b1;    /* 64 x 4,  64 */
    const void* w2; const float* b2;    /* 64 x 64, 64 */
    const void* w3; const float* b3;    /* 2 x 64,  2  */
    const void* wv; const float* bv;    /* 1 x 64,  1  (value head, optional) */
} rlsim_policy;

/* Run global steps t .. t+K-1 of every environment in exactly one kernel launch
 * (the paper's fused simulation, "Simulator Kernel Fusion"), then t += K.  K = 1
 * is the unfused form: the state goes to and from device memory every step.
 * Each step: record obs; choose the action (random Philox bit, or sample the
 * policy: action 0 with probability p0 = softmax(logits)[0]); Euler-step the
 * simulator (the chain: assemble and solve its mass-matrix equations first);
 * update padding words s_j <- a_j s_j + b_j * action (one rounding);
 * terminated = a position or angle threshold crossed (strict), truncated
 * = episode length reached max_episode_steps; reward 1; after done at step
 * t+k the next episode starts from the reset draw of the 8-step block
 * (t+k+1) / 8 (see rlsim_cfg) with zero padding words.  block_stats row r
 * covers global environments env0 + 256 r .. env0 + 256 r + 255.
 * policy_or_null: NULL = random actions.  traj_or_null: NULL = record nothing.
 * Errors: EINVAL (h NULL, K == 0, t + K > 2^32 - 1, a mixed set of NULL
 * trajectory pointers, a float pointer not 4-byte aligned, policy_p0, logp or
 * value without a policy, value without wv, a policy with NULL w1/w2/w3 or
 * unknown dtype); ESTATE (before rlsim_reset); EUNSUPPORTED (a policy with
 * D > 0 or with the chain model); EDEVICE. */
int rlsim_step_fused(rlsim_t* h, uint32_t K, const rlsim_policy* policy_or_null,
                     const rlsim_traj* traj_or_null);

/* Copy the state to HOST memory and synchronise the stream.  host_state:
 * [state_words][n_envs] f32 (simulator words then padding words), host_ep:
 * [n_envs] u32 steps taken in the current episode, *t_out: next global step.
 * Any pointer may be NULL (skipped).  Errors: EINVAL, ESTATE, EDEVICE. */
int rlsim_get_state(rlsim_t* h, float* host_state, uint32_t* host_ep, uint64_t* t_out);

/* Overwrite the state from HOST memory (same layouts) and set the global step
 * to t (checkpoint resume; padding parameters stay those of the last reset).
 * NULL host_state / host_ep leave that part unchanged.  Synchronises.
 * Errors: EINVAL (t > 2^32 - 1), ESTATE (before reset), EDEVICE. */
int rlsim_set_state(rlsim_t* h, const float* host_state, const uint32_t* host_ep, uint64_t t);

/* Synchronise the stream and free the handle and its device memory.  NULL is
 * accepted (returns RLSIM_OK). */
int rlsim_destroy(rlsim_t* h);

/* Message of h's last failure ("" if none).  h == NULL: the calling thread's
 * last rlsim_create failure.  The string stays valid until the next call on h
 * (or the thread's next create). */
const char* rlsim_last_error(const rlsim_t* h);

#ifdef __cplusplus
}
#endif

#endif /* RLSIM_H */
