/*
 * rlsim_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * The plain, slow, single-threaded CPU definition of the data-collection step
 * of "Optimizing Data Collection in Deep Reinforcement Learning" (Gleeson et
 * al., 2022): N independent cart-pole simulators (Background, "Cartpole
 * Simulator") driven by a simulation/inference loop for K steps (Background,
 * "RL Training", and the data-collection figure).  The GPU library is checked
 * against this file; nothing in the product links, loads or runs it.  Only the
 * tests, the smoke check and the benchmark's CPU-baseline leg may use it.
 *
 * It shares no code, header or constant table with the HIP path.  Every
 * function below is written in the order of the definitions it follows, one
 * IEEE operation per line where rounding matters, so that a reader can check
 * it against the stated equations by eye.  Build: gcc -O2 -ffp-contract=off
 * (no fast-math, no FTZ): every fp32 product, sum and fmaf is rounded exactly
 * once, round-to-nearest-even.
 *
 * The paper gives no equations, constants, reward, reset rule or RNG; the
 * readings used here (cart + uniform rod, explicit Euler, Philox4x32-10 with a
 * block-grouped counter, strict thresholds, auto-reset) are the ones listed in
 * the design notes.  Parity of every function is pinned by the CPU tests
 * (known-answer Philox words, hand-derived rational cart-pole steps, a
 * 50-digit Euler-Lagrange solve, linearisation, conservation laws, closed
 * forms of the padding recurrence and of special MLP weights).
 *
 * Test helpers built on these definitions: orc_mlp_bounds (after the policy),
 * the interval enclosure of a device evaluation of the policy that serves as
 * its tolerance, and the teacher-forced row checkers.
 *
 * The second simulator, a cart carrying a chain of N uniform rods (the
 * heavier multi-body kind the paper's Future Work points to), closes the
 * file: its Lagrangian in mass-matrix form, solved by elimination every
 * step, with the same loop, RNG contract and checker.  Its pins: an
 * independent 50-digit assembly of the equations of motion from the links'
 * geometry, first-order energy and momentum drift, small-angle
 * linearisation, and the one-link case against the cart-pole.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel Random Numbers: As   */
/* Easy as 1, 2, 3", SC'11): ten rounds of a 4-word multiply/xor bijection    */
/* with a Weyl-sequence key schedule.                                        */
/* ------------------------------------------------------------------------ */
void orc_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4])
{
    uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
    uint32_t k0 = key_in[0], k1 = key_in[1];
    for (int round = 0; round < 10; ++round) {
        uint64_t p0 = (uint64_t)0xD2511F53u * (uint64_t)c0;
        uint64_t p1 = (uint64_t)0xCD9E8D57u * (uint64_t)c2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t n0 = hi1 ^ c1 ^ k0;
        uint32_t n1 = lo1;
        uint32_t n2 = hi0 ^ c3 ^ k1;
        uint32_t n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
        k0 += 0x9E3779B9u; /* the key bump after round 10 is never used */
        k1 += 0xBB67AE85u;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* Stream ids of the counter (third counter word). */
enum { ORC_STREAM_RESET = 0, ORC_STREAM_ACTION = 1, ORC_STREAM_PARAMS = 2, ORC_STREAM_POLICY = 3 };

static void orc_draw(uint64_t seed, uint32_t env, uint32_t block, uint32_t stream, uint32_t out[4])
{
    uint32_t ctr[4] = { env, block, stream, 0u };
    uint32_t key[2] = { (uint32_t)(seed & 0xFFFFFFFFu), (uint32_t)(seed >> 32) };
    orc_philox4x32_10(ctr, key, out);
}

/* Top 24 bits of a word as a float in [0, 1 - 2^-24]; exact. */
float orc_u24(uint32_t r)
{
    float m = (float)(r >> 8);
    return m * 0x1.0p-24f;
}

/* uniform on [lo, hi): lo + u24 * (hi - lo), the product-sum rounded once. */
float orc_uniform(uint32_t r, float lo, float hi)
{
    float width = hi - lo;
    return fmaf(orc_u24(r), width, lo);
}

/* ------------------------------------------------------------------------ */
/* Configuration (same meaning as the library's, declared independently).    */
/* ------------------------------------------------------------------------ */
typedef struct {
    float gravity, masscart, masspole, half_length, force_mag, tau;
    float x_threshold, theta_threshold_rad;
    uint32_t max_episode_steps;      /* 0 = no time limit */
    float reset_low, reset_high;
    float pad_a_low, pad_a_high, pad_b_low, pad_b_high;
    uint32_t no_termination;         /* nonzero: termination never fires */
    uint32_t compute_factor;         /* C >= 1 Euler sub-iterations of tau / C per step */
} orc_params;

/* ------------------------------------------------------------------------ */
/* sin and cos: a truncated Maclaurin series (degree 9 / 8, Horner form with  */
/* fmaf) on |theta| <= fp32(pi/4), the domain of every pre-step angle of a    */
/* live cart-pole episode.  Larger angles (a swinging chain link, a pole with */
/* termination disabled) are first reduced by quadrants: k = the integer      */
/* nearest theta * 2/pi (fp32 product, ties to even), r = theta - k pi/2 with */
/* pi/2 split into a high fp32 part (r1 = theta - k * hi is exact: both terms */
/* are multiples of 2^-24 and |r1| < 2) and a low part, then the quadrant     */
/* k mod 4 (formed exactly in fp32) picks and signs the series values:        */
/* sin(r + k pi/2) = sin r, cos r, -sin r, -cos r for k = 0, 1, 2, 3 mod 4.   */
/* A non-finite theta gives NaN.                                              */
/* ------------------------------------------------------------------------ */
float orc_sin_series(float th)
{
    const float s3 = (float)(-1.0 / 6.0);
    const float s5 = (float)(1.0 / 120.0);
    const float s7 = (float)(-1.0 / 5040.0);
    const float s9 = (float)(1.0 / 362880.0);
    float z = th * th;
    float q = fmaf(s9, z, s7);
    q = fmaf(q, z, s5);
    q = fmaf(q, z, s3);
    float th3 = th * z;
    return fmaf(th3, q, th);          /* th + th^3 (s3 + s5 z + s7 z^2 + s9 z^3) */
}

float orc_cos_series(float th)
{
    const float c2 = -0.5f;
    const float c4 = (float)(1.0 / 24.0);
    const float c6 = (float)(-1.0 / 720.0);
    const float c8 = (float)(1.0 / 40320.0);
    float z = th * th;
    float q = fmaf(c8, z, c6);
    q = fmaf(q, z, c4);
    q = fmaf(q, z, c2);
    return fmaf(z, q, 1.0f);          /* 1 + z (c2 + c4 z + c6 z^2 + c8 z^3) */
}

void orc_sincos(float th, float* s, float* c)
{
    const float quarter_pi = (float)(3.14159265358979323846 / 4.0);        /* 0x3F490FDB */
    const float two_over_pi = (float)(2.0 / 3.14159265358979323846);      /* 0x3F22F983 */
    const float half_pi_hi = (float)(3.14159265358979323846 / 2.0);       /* 0x3FC90FDB */
    const float half_pi_lo = -4.371138828673793e-08f;                     /* 0xB33BBD2E = fp32(pi/2 - hi) */
    if (fabsf(th) <= quarter_pi) {
        *s = orc_sin_series(th);
        *c = orc_cos_series(th);
        return;
    }
    float k = rintf(th * two_over_pi);
    float r = fmaf(-k, half_pi_hi, th);
    r = fmaf(-k, half_pi_lo, r);
    float quadrant = k - 4.0f * floorf(k * 0.25f);      /* k mod 4, exact; NaN for non-finite theta */
    float sr = orc_sin_series(r), cr = orc_cos_series(r);
    if (quadrant == 1.0f) {
        *s = cr;
        *c = -sr;
    } else if (quadrant == 2.0f) {
        *s = -sr;
        *c = -cr;
    } else if (quadrant == 3.0f) {
        *s = -cr;
        *c = sr;
    } else {
        *s = sr;
        *c = cr;
    }
}

float orc_sin(float th)
{
    float s, c;
    orc_sincos(th, &s, &c);
    return s;
}

float orc_cos(float th)
{
    float s, c;
    orc_sincos(th, &s, &c);
    return c;
}

/* ------------------------------------------------------------------------ */
/* One explicit-Euler step of the frictionless cart + uniform rod.           */
/*   Lagrangian L = 1/2 M xd^2 + m l xd thd cos th + 2/3 m l^2 thd^2         */
/*                  - m g l cos th      (M = cart + pole mass, l = half len) */
/*   => thacc = (g sin th - cos th * temp) / (l (4/3 - m cos^2 th / M)),     */
/*      temp  = (F + m l thd^2 sin th) / M,                                  */
/*      xacc  = temp - m l thacc cos th / M.                                 */
/* Positions advance with the old velocities.  a == 1 pushes towards +x.     */
/* ------------------------------------------------------------------------ */
void orc_cartpole_step(const orc_params* p, const float in[4], int action, float out[4])
{
    /* derived constants, one fp32 operation each */
    float total_mass = p->masscart + p->masspole;
    float pole_ml = p->masspole * p->half_length;
    float inv_total = 1.0f / total_mass;
    float m_over_M = p->masspole * inv_total;
    float ml_over_M = pole_ml * inv_total;
    float four_thirds = 4.0f / 3.0f;

    float x = in[0], xd = in[1], th = in[2], thd = in[3];
    float force = action ? p->force_mag : -p->force_mag;

    float sin_th, cos_th;
    orc_sincos(th, &sin_th, &cos_th);

    float thd2 = thd * thd;
    float ml_thd2 = pole_ml * thd2;
    float f_plus = fmaf(ml_thd2, sin_th, force);        /* F + m l thd^2 sin th */
    float temp = f_plus * inv_total;

    float g_sin = p->gravity * sin_th;
    float num = fmaf(-cos_th, temp, g_sin);             /* g sin th - cos th temp */
    float cos2 = cos_th * cos_th;
    float bracket = fmaf(-m_over_M, cos2, four_thirds); /* 4/3 - m cos^2 th / M */
    float den = p->half_length * bracket;
    float thacc = num / den;

    float k_th = ml_over_M * thacc;
    float xacc = fmaf(-k_th, cos_th, temp);             /* temp - m l thacc cos th / M */

    out[0] = fmaf(p->tau, xd, x);
    out[1] = fmaf(p->tau, xacc, xd);
    out[2] = fmaf(p->tau, thd, th);
    out[3] = fmaf(p->tau, thacc, thd);
}

/* One simulation step with the paper's compute factor C ("Simulator       */
/* Complexity"): C explicit-Euler iterations of length tau / C (one fp32    */
/* division), the action held for all of them.  C = 1 is the plain step.   */
void orc_env_step(const orc_params* p, const float in[4], int action, float out[4])
{
    uint32_t C = p->compute_factor;
    orc_params sub = *p;
    sub.tau = p->tau / (float)C;
    float cur[4] = { in[0], in[1], in[2], in[3] };
    for (uint32_t c = 0; c < C; ++c) {
        float nxt[4];
        orc_cartpole_step(&sub, cur, action, nxt);
        for (int q = 0; q < 4; ++q) cur[q] = nxt[q];
    }
    for (int q = 0; q < 4; ++q) out[q] = cur[q];
}

/* Strict threshold test on the post-step state; NaN compares false. */
int orc_terminated(const orc_params* p, const float s[4])
{
    if (p->no_termination) return 0;
    float x = s[0], th = s[2];
    return (x < -p->x_threshold) || (x > p->x_threshold) ||
           (th < -p->theta_threshold_rad) || (th > p->theta_threshold_rad);
}

/* Initial state of an episode that begins at global step t: stream RESET,  */
/* counter block t/8, words 0..3 -> x, xd, th, thd.  Episodes of one env    */
/* that begin in the same 8-step block would share a draw; with the default  */
/* constants every episode lasts at least 8 steps (shown for the whole reset */
/* box and every action sequence by interval arithmetic over the fp32 step,  */
/* tests/test_oracle_episode_bound.py), so none do.                          */
void orc_reset_draw(const orc_params* p, uint64_t seed, uint32_t env, uint32_t t, float out[4])
{
    uint32_t w[4];
    orc_draw(seed, env, t >> 3, ORC_STREAM_RESET, w);
    for (int c = 0; c < 4; ++c) out[c] = orc_uniform(w[c], p->reset_low, p->reset_high);
}

/* Random action at global step t: stream ACTION, counter block t/128,      */
/* bit (t mod 32) of word ((t/32) mod 4).                                    */
int orc_action_bit(uint64_t seed, uint32_t env, uint32_t t)
{
    uint32_t w[4];
    orc_draw(seed, env, t >> 7, ORC_STREAM_ACTION, w);
    return (int)((w[(t >> 5) & 3u] >> (t & 31u)) & 1u);
}

/* Uniform used to sample the policy's action at step t: stream POLICY,     */
/* counter block t/4, word (t mod 4).                                        */
float orc_policy_u(uint64_t seed, uint32_t env, uint32_t t)
{
    uint32_t w[4];
    orc_draw(seed, env, t >> 2, ORC_STREAM_POLICY, w);
    return orc_u24(w[t & 3u]);
}

/* Padding-word parameters: stream PARAMS, counter block j.                  */
void orc_pad_params(const orc_params* p, uint64_t seed, uint32_t env, uint32_t j, float* a, float* b)
{
    uint32_t w[4];
    orc_draw(seed, env, j, ORC_STREAM_PARAMS, w);
    *a = orc_uniform(w[0], p->pad_a_low, p->pad_a_high);
    *b = orc_uniform(w[1], p->pad_b_low, p->pad_b_high);
}

/* One padding word: s <- a s + b u with u the action (0 or 1), rounded once:
 * the fused a s + b when u = 1, the product a s when u = 0 (no b term). */
float orc_pad_update(float s, float a, float b, int u)
{
    if (u) return fmaf(a, s, b);
    return a * s;
}

/* ------------------------------------------------------------------------ */
/* MLP policy 4 -> 64 -> 64 -> 2, tanh hidden layers, weights row-major     */
/* [out][in], evaluated in double.  p0 = softmax(logits)[0].  An optional    */
/* value head 64 -> 1 reads the same second hidden layer (a shared trunk,    */
/* the usual actor-critic form of the learner the collected data feeds).     */
/* bf16 mode rounds the weights, the input and both hidden activations to    */
/* bfloat16 (round to nearest even) at the points where a bf16 kernel holds  */
/* them; biases and sums stay in double.  bf16 = 2 is bf16 mode over weight */
/* arrays that already hold bf16 values (rounding them again would change   */
/* nothing), so only the input and the activations are rounded.              */
/* ------------------------------------------------------------------------ */
typedef struct {
    int bf16;                                   /* 0 fp32, 1 bf16, 2 bf16 with rounded weights */
    const float *w1, *b1, *w2, *b2, *w3, *b3;   /* biases may be NULL (zero) */
    const float *wv, *bv;                       /* value head 1 x 64, 1; wv NULL = none */
} orc_policy;

/* Round a double to the nearest bfloat16 value (ties to even), returned as */
/* a double.  bfloat16 has an 8-bit significand and fp32's exponent range.  */
double orc_round_bf16(double v)
{
    if (v != v || v == 0.0 || isinf(v)) return v;
    int e;
    frexp(v, &e);                               /* |v| = f 2^e, f in [0.5, 1) */
    if (e < -125) e = -125;                     /* subnormal bf16 spacing      */
    double q = ldexp(1.0, e - 8);               /* spacing of 8-bit significand */
    double r = v / q;                           /* exact: power-of-two scale    */
    double fl = floor(r);
    double diff = r - fl;
    double k;
    if (diff > 0.5) k = fl + 1.0;
    else if (diff < 0.5) k = fl;
    else k = (fmod(fl, 2.0) == 0.0) ? fl : fl + 1.0;
    double out = k * q;
    if (fabs(out) > 3.3895313892515355e38) out = v > 0 ? INFINITY : -INFINITY;
    return out;
}

static double orc_w(const orc_policy* pol, const float* w, int idx)
{
    double v = (double)w[idx];
    return pol->bf16 == 1 ? orc_round_bf16(v) : v;
}

/* The trunk: h2 = tanh(W2 tanh(W1 obs + b1) + b2). */
static void orc_mlp_trunk(const orc_policy* pol, const float obs[4], double h2[64])
{
    double in[4], h1[64];
    for (int i = 0; i < 4; ++i) in[i] = pol->bf16 ? orc_round_bf16((double)obs[i]) : (double)obs[i];
    for (int o = 0; o < 64; ++o) {
        double acc = pol->b1 ? (double)pol->b1[o] : 0.0;
        for (int i = 0; i < 4; ++i) acc += orc_w(pol, pol->w1, o * 4 + i) * in[i];
        h1[o] = tanh(acc);
        if (pol->bf16) h1[o] = orc_round_bf16(h1[o]);
    }
    for (int o = 0; o < 64; ++o) {
        double acc = pol->b2 ? (double)pol->b2[o] : 0.0;
        for (int i = 0; i < 64; ++i) acc += orc_w(pol, pol->w2, o * 64 + i) * h1[i];
        h2[o] = tanh(acc);
        if (pol->bf16) h2[o] = orc_round_bf16(h2[o]);
    }
}

/* All policy outputs for one observation: the two logits W3 h2 + b3, p0, and  */
/* the value Wv h2 + bv (0 if the policy has no value head).                  */
void orc_mlp_eval(const orc_policy* pol, const float obs[4], double logit[2], double* p0, double* value)
{
    double h2[64];
    orc_mlp_trunk(pol, obs, h2);
    for (int o = 0; o < 2; ++o) {
        double acc = pol->b3 ? (double)pol->b3[o] : 0.0;
        for (int i = 0; i < 64; ++i) acc += orc_w(pol, pol->w3, o * 64 + i) * h2[i];
        logit[o] = acc;
    }
    /* softmax over two logits: p0 = e^l0 / (e^l0 + e^l1) = 1 / (1 + e^(l1 - l0)) */
    *p0 = 1.0 / (1.0 + exp(logit[1] - logit[0]));
    double v = 0.0;
    if (pol->wv) {
        v = pol->bv ? (double)pol->bv[0] : 0.0;
        for (int i = 0; i < 64; ++i) v += orc_w(pol, pol->wv, i) * h2[i];
    }
    *value = v;
}

double orc_mlp_p0(const orc_policy* pol, const float obs[4])
{
    double logit[2], p0, v;
    orc_mlp_eval(pol, obs, logit, &p0, &v);
    return p0;
}

/* log softmax(logits)[a] = l_a - log(e^l0 + e^l1), with the larger logit    */
/* taken out of the sum so that neither exponential overflows.               */
double orc_log_prob(const double logit[2], int a)
{
    double m = logit[0] > logit[1] ? logit[0] : logit[1];
    double lse = m + log(exp(logit[0] - m) + exp(logit[1] - m));
    return logit[a ? 1 : 0] - lse;
}

/* ------------------------------------------------------------------------ */
/* Tolerance of a device evaluation of the policy (a test helper): interval  */
/* enclosures of what any evaluation under the following error model may     */
/* return for one observation.                                               */
/*  - Each dot product bias + sum of n products is formed in fp32 with an    */
/*    error of at most err->acc * (n + 1) * (|bias| + sum |w x|), over the    */
/*    operands actually used (acc = 2^-23, twice fp32's unit roundoff per    */
/*    operation, covers any summation order and rounding direction; products */
/*    of bf16 values are exact in fp32, fp32 products round once).           */
/*  - tanh and p0 = 1 / (1 + e^d) are returned with an absolute error of at  */
/*    most err->tanh and err->p0, log pi with at most                         */
/*    err->logpi * (1 + |log pi|); d = l1 - l0 is one more fp32 rounding.     */
/*  - In bf16 mode inputs, weights and activations are rounded to bf16 at the */
/*    points the oracle rounds them.  Rounding is monotone, so rounding the   */
/*    ends of an interval encloses the rounding of every point inside it.    */
/* Intervals are carried as centre and radius through the dot products and   */
/* as end points through the monotone functions.  Out: lo/hi of p0, of        */
/* log pi(0), of log pi(1), and of the value head (0 without one).           */
/* ------------------------------------------------------------------------ */
typedef struct {
    double acc, tanh, p0, logpi;
} orc_errs;

typedef struct {
    double p0_lo, p0_hi, lp0_lo, lp0_hi, lp1_lo, lp1_hi, v_lo, v_hi;
} orc_bounds;

static double orc_dmax(double a, double b) { return a > b ? a : b; }

/* An activation interval from a pre-activation interval [z - r, z + r]. */
static void orc_act_interval(const orc_policy* pol, const orc_errs* e, double z, double r, double* lo, double* hi)
{
    double a = tanh(z - r) - e->tanh;
    double b = tanh(z + r) + e->tanh;
    if (pol->bf16) {
        a = orc_round_bf16(a);
        b = orc_round_bf16(b);
    }
    *lo = a;
    *hi = b;
}

/* -softplus(z), the log-probability of the action whose logit is z below the other's */
static double orc_neg_softplus(double z)
{
    return -(orc_dmax(z, 0.0) + log1p(exp(-fabs(z))));
}

void orc_mlp_bounds(const orc_policy* pol, const float obs[4], const orc_errs* e, orc_bounds* out)
{
    double x[4], lo1[64], hi1[64], lo2[64], hi2[64];
    for (int i = 0; i < 4; ++i) x[i] = pol->bf16 ? orc_round_bf16((double)obs[i]) : (double)obs[i];
    /* layer 1: exact inputs */
    for (int o = 0; o < 64; ++o) {
        double b = pol->b1 ? (double)pol->b1[o] : 0.0;
        double z = b, mag = fabs(b);
        for (int i = 0; i < 4; ++i) {
            double t = orc_w(pol, pol->w1, o * 4 + i) * x[i];
            z += t;
            mag += fabs(t);
        }
        orc_act_interval(pol, e, z, e->acc * 5.0 * mag, &lo1[o], &hi1[o]);
    }
    /* layer 2: interval inputs */
    for (int o = 0; o < 64; ++o) {
        double b = pol->b2 ? (double)pol->b2[o] : 0.0;
        double z = b, rad = 0.0, mag = fabs(b);
        for (int i = 0; i < 64; ++i) {
            double w = orc_w(pol, pol->w2, o * 64 + i);
            z += w * 0.5 * (lo1[i] + hi1[i]);
            rad += fabs(w) * 0.5 * (hi1[i] - lo1[i]);
            mag += fabs(w) * orc_dmax(fabs(lo1[i]), fabs(hi1[i]));
        }
        orc_act_interval(pol, e, z, rad + e->acc * 65.0 * mag, &lo2[o], &hi2[o]);
    }
    /* logits: d = l1 - l0 carried directly (l0 and l1 share h2) */
    double d = 0.0, rad_d = 0.0, mag0 = 0.0, mag1 = 0.0;
    {
        double b0 = pol->b3 ? (double)pol->b3[0] : 0.0, b1 = pol->b3 ? (double)pol->b3[1] : 0.0;
        d = b1 - b0;
        mag0 = fabs(b0);
        mag1 = fabs(b1);
        for (int i = 0; i < 64; ++i) {
            double w0 = orc_w(pol, pol->w3, i), w1 = orc_w(pol, pol->w3, 64 + i);
            double m = orc_dmax(fabs(lo2[i]), fabs(hi2[i]));
            d += (w1 - w0) * 0.5 * (lo2[i] + hi2[i]);
            rad_d += fabs(w1 - w0) * 0.5 * (hi2[i] - lo2[i]);
            mag0 += fabs(w0) * m;
            mag1 += fabs(w1) * m;
        }
        rad_d += e->acc * 65.0 * (mag0 + mag1);
        rad_d += 0.5 * e->acc * (fabs(d) + rad_d);      /* the subtraction l1 - l0 */
    }
    double dlo = d - rad_d, dhi = d + rad_d;
    out->p0_lo = 1.0 / (1.0 + exp(dhi)) - e->p0;         /* p0 decreases with d */
    out->p0_hi = 1.0 / (1.0 + exp(dlo)) + e->p0;
    /* log pi(0) = -softplus(d) decreases with d; log pi(1) = -softplus(-d) increases */
    double a0 = orc_neg_softplus(dhi), b0 = orc_neg_softplus(dlo);
    double a1 = orc_neg_softplus(-dlo), b1 = orc_neg_softplus(-dhi);
    out->lp0_lo = a0 - e->logpi * (1.0 + fabs(a0));
    out->lp0_hi = b0 + e->logpi * (1.0 + fabs(b0));
    out->lp1_lo = a1 - e->logpi * (1.0 + fabs(a1));
    out->lp1_hi = b1 + e->logpi * (1.0 + fabs(b1));
    if (pol->wv) {
        double bv = pol->bv ? (double)pol->bv[0] : 0.0;
        double v = bv, rad = 0.0, mag = fabs(bv);
        for (int i = 0; i < 64; ++i) {
            double w = orc_w(pol, pol->wv, i);
            v += w * 0.5 * (lo2[i] + hi2[i]);
            rad += fabs(w) * 0.5 * (hi2[i] - lo2[i]);
            mag += fabs(w) * orc_dmax(fabs(lo2[i]), fabs(hi2[i]));
        }
        rad += e->acc * 65.0 * mag;
        out->v_lo = v - rad;
        out->v_hi = v + rad;
    } else {
        out->v_lo = out->v_hi = 0.0;
    }
}

/* ------------------------------------------------------------------------ */
/* The vectorised simulator: a slice of n environments with global ids       */
/* env0 .. env0+n-1, each with 4 cart-pole words, D padding words, and an    */
/* episode step counter.  Host arrays, structure-of-arrays.                  */
/* ------------------------------------------------------------------------ */
typedef struct {
    uint32_t n, env0, D;
    orc_params p;
    uint64_t seed;
    uint32_t t;           /* global step of the next step */
    int has_reset;
    float* cart;          /* [4][n] */
    uint32_t* ep;         /* [n]    steps taken in the current episode */
    float* s;             /* [D][n] padding words */
    float* a;             /* [D][n] */
    float* b;             /* [D][n] */
} orc_sim;

void orc_destroy(orc_sim* sim)
{
    if (!sim) return;
    free(sim->cart); free(sim->ep); free(sim->s); free(sim->a); free(sim->b);
    free(sim);
}

orc_sim* orc_create(uint32_t n, uint32_t env0, uint32_t D, const orc_params* p)
{
    if (n == 0 || p->compute_factor == 0) return NULL;
    orc_sim* sim = (orc_sim*)calloc(1, sizeof(orc_sim));
    if (!sim) return NULL;
    sim->n = n; sim->env0 = env0; sim->D = D; sim->p = *p;
    sim->cart = (float*)calloc((size_t)4 * n, sizeof(float));
    sim->ep = (uint32_t*)calloc(n, sizeof(uint32_t));
    size_t nd = (size_t)D * n;
    sim->s = (float*)calloc(nd ? nd : 1, sizeof(float));
    sim->a = (float*)calloc(nd ? nd : 1, sizeof(float));
    sim->b = (float*)calloc(nd ? nd : 1, sizeof(float));
    if (!sim->cart || !sim->ep || !sim->s || !sim->a || !sim->b) { orc_destroy(sim); return NULL; }
    return sim;
}

/* Every environment starts an episode at global step 0. */
void orc_reset(orc_sim* sim, uint64_t seed)
{
    uint32_t n = sim->n;
    sim->seed = seed;
    sim->t = 0;
    sim->has_reset = 1;
    for (uint32_t i = 0; i < n; ++i) {
        uint32_t env = sim->env0 + i;
        float init[4];
        orc_reset_draw(&sim->p, seed, env, 0u, init);
        for (int c = 0; c < 4; ++c) sim->cart[(size_t)c * n + i] = init[c];
        sim->ep[i] = 0;
        for (uint32_t j = 0; j < sim->D; ++j) {
            float a, b;
            orc_pad_params(&sim->p, seed, env, j, &a, &b);
            sim->a[(size_t)j * n + i] = a;
            sim->b[(size_t)j * n + i] = b;
            sim->s[(size_t)j * n + i] = 0.0f;
        }
    }
}

/*
 * K steps of the data-collection loop for every environment of the slice.
 * Step t of one environment:
 *   obs   = the state before the step (recorded in the trajectory)
 *   a_t   = policy ? (u_t < p0(obs) ? 0 : 1) : random action bit
 *   next  = Euler step; padding words s <- a s + b a_t
 *   n     = ep + 1; terminated = threshold crossed by next;
 *   truncated = (max_episode_steps != 0 && n >= max_episode_steps)
 *   done  = terminated | truncated << 1;  reward = 1
 *   if done: the episode that begins at t+1 starts from the reset draw for
 *            t+1, ep = 0, padding words = +0;  else ep = n.
 * Outputs (each may be NULL), rows 0..K-1 of this call:
 *   obs [K][4][n] f32, act [K][n] u8, rew [K][n] f32, done [K][n] u8,
 *   p0, logp (log-probability of a_t), value [K][n] f64 (policy runs),
 *   stats [nblk][4] u32 over 256-env blocks of
 *   global env ids: {episodes finished, sum of their lengths, terminated,
 *   truncated}; nblk = (env0+n-1)/256 - env0/256 + 1.
 * Returns 0, or -1 before reset, -2 when t + K would pass 2^32 - 1.
 */
int orc_step(orc_sim* sim, uint32_t K, const orc_policy* pol,
             float* obs, uint8_t* act, float* rew, uint8_t* done, uint32_t* stats, double* p0_out,
             double* logp_out, double* value_out)
{
    if (!sim->has_reset) return -1;
    if ((uint64_t)sim->t + (uint64_t)K > 0xFFFFFFFFull) return -2;
    uint32_t n = sim->n;
    uint32_t blk0 = sim->env0 / 256u;
    if (stats) {
        uint32_t nblk = (sim->env0 + n - 1u) / 256u - blk0 + 1u;
        memset(stats, 0, (size_t)nblk * 4u * sizeof(uint32_t));
    }
    for (uint32_t k = 0; k < K; ++k) {
        uint32_t t = sim->t + k;
        for (uint32_t i = 0; i < n; ++i) {
            uint32_t env = sim->env0 + i;
            float cur[4], nxt[4];
            for (int c = 0; c < 4; ++c) cur[c] = sim->cart[(size_t)c * n + i];

            int a;
            if (pol) {
                double logit[2], p0, value;
                orc_mlp_eval(pol, cur, logit, &p0, &value);
                float u = orc_policy_u(sim->seed, env, t);
                a = ((double)u < p0) ? 0 : 1;
                if (p0_out) p0_out[(size_t)k * n + i] = p0;
                if (logp_out) logp_out[(size_t)k * n + i] = orc_log_prob(logit, a);
                if (value_out) value_out[(size_t)k * n + i] = value;
            } else {
                a = orc_action_bit(sim->seed, env, t);
            }

            orc_env_step(&sim->p, cur, a, nxt);
            for (uint32_t j = 0; j < sim->D; ++j) {
                size_t q = (size_t)j * n + i;
                sim->s[q] = orc_pad_update(sim->s[q], sim->a[q], sim->b[q], a);
            }

            uint32_t len = sim->ep[i] + 1u;
            int term = orc_terminated(&sim->p, nxt);
            int trunc = (sim->p.max_episode_steps != 0u) && (len >= sim->p.max_episode_steps);
            uint8_t d = (uint8_t)(term | (trunc << 1));

            if (obs) for (int c = 0; c < 4; ++c) obs[((size_t)k * 4 + c) * n + i] = cur[c];
            if (act) act[(size_t)k * n + i] = (uint8_t)a;
            if (rew) rew[(size_t)k * n + i] = 1.0f;
            if (done) done[(size_t)k * n + i] = d;

            if (d) {
                orc_reset_draw(&sim->p, sim->seed, env, t + 1u, nxt);
                sim->ep[i] = 0;
                for (uint32_t j = 0; j < sim->D; ++j) sim->s[(size_t)j * n + i] = 0.0f;
                if (stats) {
                    uint32_t* st = stats + (size_t)(env / 256u - blk0) * 4u;
                    st[0] += 1u;
                    st[1] += len;
                    st[2] += (uint32_t)term;
                    st[3] += (uint32_t)trunc;
                }
            } else {
                sim->ep[i] = len;
            }
            for (int c = 0; c < 4; ++c) sim->cart[(size_t)c * n + i] = nxt[c];
        }
    }
    sim->t += K;
    return 0;
}

/* State as [4 + D][n] words (cart-pole words, then padding), episode steps,
 * and the global step counter. */
void orc_get_state(const orc_sim* sim, float* state, uint32_t* ep, uint64_t* t)
{
    size_t n = sim->n;
    if (state) {
        memcpy(state, sim->cart, 4 * n * sizeof(float));
        if (sim->D) memcpy(state + 4 * n, sim->s, (size_t)sim->D * n * sizeof(float));
    }
    if (ep) memcpy(ep, sim->ep, n * sizeof(uint32_t));
    if (t) *t = sim->t;
}

/* Overwrite the state; the padding parameters stay those of the last reset. */
int orc_set_state(orc_sim* sim, const float* state, const uint32_t* ep, uint64_t t)
{
    if (!sim->has_reset) return -1;
    if (t > 0xFFFFFFFFull) return -2;
    size_t n = sim->n;
    if (state) {
        memcpy(sim->cart, state, 4 * n * sizeof(float));
        if (sim->D) memcpy(sim->s, state + 4 * n, (size_t)sim->D * n * sizeof(float));
    }
    if (ep) memcpy(sim->ep, ep, n * sizeof(uint32_t));
    sim->t = (uint32_t)t;
    return 0;
}

/* Padding parameters as [D][n] arrays (for tests of the recurrence). */
void orc_get_pad_params(const orc_sim* sim, float* a, float* b)
{
    size_t nd = (size_t)sim->D * sim->n;
    if (a && nd) memcpy(a, sim->a, nd * sizeof(float));
    if (b && nd) memcpy(b, sim->b, nd * sizeof(float));
}

/* ------------------------------------------------------------------------ */
/* Teacher-forced check of recorded random-action rows (a test helper: the    */
/* comparison rule that every recorded step follows from the one before it).  */
/* Rows k = 0..K-1 hold global steps t0 + k of environments env0 .. env0+n-1, */
/* laid out [K][4][n] (obs) and [K][n] (action, reward, done); ep0[i] is the   */
/* episode's step count at t0.  ep0 == NULL means every episode began at t0   */
/* (as after a reset), so row 0 must also be the reset draw for step t0.  For */
/* every env-step it recomputes, from the recorded obs and nothing else:      */
/*   the random action bit of (seed, env, t), reward 1,                       */
/*   next = the simulation step of (obs_t, action),                           */
/*   done = terminated(next) | truncated << 1 (episode length from ep0),      */
/*   obs_{t+1} (row k+1) = the reset draw for step t+1 if done, else next,    */
/* bit for bit.  final_state ([4][n]) and final_ep ([n]), each optional, are  */
/* the state and episode counters after the last row: they must equal the    */
/* last step's successor and episode length (mismatches count at row K-1).    */
/* Returns the number of mismatching env-steps and, if any, the row and env   */
/* index of the first in *bad_k, *bad_i.                                      */
/* ------------------------------------------------------------------------ */
uint64_t orc_check_rows(const orc_params* p, uint64_t seed, uint32_t env0, uint32_t n, uint32_t t0, uint32_t K,
                        const uint32_t* ep0, const float* obs, const uint8_t* act, const float* rew,
                        const uint8_t* done, const float* final_state, const uint32_t* final_ep,
                        uint32_t* bad_k, uint32_t* bad_i)
{
    uint64_t bad = 0;
    for (uint32_t i = 0; i < n; ++i) {
        uint32_t ep = ep0 ? ep0[i] : 0u;
        uint32_t env = env0 + i;
        for (uint32_t k = 0; k < K; ++k) {
            uint32_t t = t0 + k;
            float cur[4], nxt[4];
            for (int c = 0; c < 4; ++c) cur[c] = obs[((size_t)k * 4 + c) * n + i];
            int ok = 1;
            if (k == 0 && !ep0) {
                float start[4];
                orc_reset_draw(p, seed, env, t0, start);
                if (memcmp(start, cur, sizeof(start)) != 0) ok = 0;
            }
            int a = orc_action_bit(seed, env, t);
            orc_env_step(p, cur, a, nxt);
            uint32_t len = ep + 1u;
            int term = orc_terminated(p, nxt);
            int trunc = (p->max_episode_steps != 0u) && (len >= p->max_episode_steps);
            uint8_t d = (uint8_t)(term | (trunc << 1));
            if (act[(size_t)k * n + i] != (uint8_t)a || rew[(size_t)k * n + i] != 1.0f || done[(size_t)k * n + i] != d)
                ok = 0;
            if (d) {
                orc_reset_draw(p, seed, env, t + 1u, nxt);
                ep = 0u;
            } else {
                ep = len;
            }
            if (ok && k + 1 < K) {
                for (int c = 0; c < 4; ++c) {
                    float g = obs[((size_t)(k + 1) * 4 + c) * n + i];
                    if (memcmp(&g, &nxt[c], sizeof(float)) != 0) ok = 0;
                }
            }
            if (ok && k + 1 == K) {
                for (int c = 0; c < 4 && final_state; ++c) {
                    float g = final_state[(size_t)c * n + i];
                    if (memcmp(&g, &nxt[c], sizeof(float)) != 0) ok = 0;
                }
                if (final_ep && final_ep[i] != ep) ok = 0;
            }
            if (!ok) {
                if (bad == 0 && bad_k && bad_i) {
                    *bad_k = k;
                    *bad_i = i;
                }
                ++bad;
            }
        }
    }
    return bad;
}

/* ------------------------------------------------------------------------ */
/* Teacher-forced check of recorded policy rows (a test helper).  As          */
/* orc_check_rows, with the MLP policy choosing the action: for every         */
/* env-step, with u the POLICY-stream uniform of (seed, env, t) and p0g the   */
/* recorded probability of action 0:                                          */
/*   the recorded action is (u < p0g ? 0 : 1)               (exact);          */
/*   p0g, and log pi / value when given, lie in orc_mlp_bounds' enclosures    */
/*   for the recorded obs (the recorded action's log pi);                    */
/*   reward 1, the done byte, and the next row (reset draw after an episode   */
/*   end) follow from the simulation step of (obs, recorded action), bit for  */
/*   bit.                                                                    */
/* ep0 == NULL (episodes begin at t0) also checks row 0 against the reset    */
/* draw, and final_state / final_ep (optional) the state after the last row,  */
/* as orc_check_rows does.                                                    */
/* An action that differs from the oracle's own choice (u < p0) can only be   */
/* one whose u lies inside the p0 enclosure; these are counted in *exempt.    */
/* dp0_out ([K][n], may be NULL) receives |p0g - p0| of every env-step.        */
/* stats (may be NULL): [0] max |p0g - p0|, [1] max p0 enclosure width,        */
/* [2] sum of p0 enclosure widths.  Returns the number of failing env-steps;  */
/* *bad_k, *bad_i the first failure.                                          */
/* ------------------------------------------------------------------------ */
uint64_t orc_check_policy_rows(const orc_params* p, const orc_policy* pol, uint64_t seed, uint32_t env0, uint32_t n,
                               uint32_t t0, uint32_t K, const uint32_t* ep0, const float* obs, const uint8_t* act,
                               const float* rew, const uint8_t* done, const float* p0g, const float* logp,
                               const float* value, const orc_errs* errs, const float* final_state,
                               const uint32_t* final_ep, float* dp0_out, double stats[3], uint64_t* exempt,
                               uint32_t* bad_k, uint32_t* bad_i)
{
    uint64_t bad = 0, ex = 0;
    double worst = 0.0, wmax = 0.0, wsum = 0.0;
    /* a bf16 policy is evaluated over weight copies rounded once up front */
    float rw1[64 * 4], rw2[64 * 64], rw3[2 * 64], rwv[64];
    orc_policy rp = *pol;
    if (pol->bf16 == 1) {
        for (int j = 0; j < 64 * 4; ++j) rw1[j] = (float)orc_round_bf16((double)pol->w1[j]);
        for (int j = 0; j < 64 * 64; ++j) rw2[j] = (float)orc_round_bf16((double)pol->w2[j]);
        for (int j = 0; j < 2 * 64; ++j) rw3[j] = (float)orc_round_bf16((double)pol->w3[j]);
        for (int j = 0; j < 64 && pol->wv; ++j) rwv[j] = (float)orc_round_bf16((double)pol->wv[j]);
        rp.w1 = rw1;
        rp.w2 = rw2;
        rp.w3 = rw3;
        rp.wv = pol->wv ? rwv : NULL;
        rp.bf16 = 2;
    }
    for (uint32_t i = 0; i < n; ++i) {
        uint32_t ep = ep0 ? ep0[i] : 0u;
        uint32_t env = env0 + i;
        for (uint32_t k = 0; k < K; ++k) {
            uint32_t t = t0 + k;
            size_t q = (size_t)k * n + i;
            float cur[4], nxt[4];
            for (int c = 0; c < 4; ++c) cur[c] = obs[((size_t)k * 4 + c) * n + i];
            int a = act[q];
            float u = orc_policy_u(seed, env, t);
            double logit[2], p0, v;
            orc_bounds bd;
            orc_mlp_eval(&rp, cur, logit, &p0, &v);
            orc_mlp_bounds(&rp, cur, errs, &bd);
            double g = (double)p0g[q];
            if (fabs(g - p0) > worst) worst = fabs(g - p0);
            if (dp0_out) dp0_out[q] = (float)fabs(g - p0);
            if (bd.p0_hi - bd.p0_lo > wmax) wmax = bd.p0_hi - bd.p0_lo;
            wsum += bd.p0_hi - bd.p0_lo;
            int ok = (a == (u < p0g[q] ? 0 : 1)) && g >= bd.p0_lo && g <= bd.p0_hi;
            if (k == 0 && !ep0) {
                float start[4];
                orc_reset_draw(p, seed, env, t0, start);
                if (memcmp(start, cur, sizeof(start)) != 0) ok = 0;
            }
            if (a != (((double)u < p0) ? 0 : 1)) ++ex;
            if (logp) {
                double l = (double)logp[q];
                if (a ? (l < bd.lp1_lo || l > bd.lp1_hi) : (l < bd.lp0_lo || l > bd.lp0_hi)) ok = 0;
            }
            if (value && ((double)value[q] < bd.v_lo || (double)value[q] > bd.v_hi)) ok = 0;
            orc_env_step(p, cur, a, nxt);
            uint32_t len = ep + 1u;
            int term = orc_terminated(p, nxt);
            int trunc = (p->max_episode_steps != 0u) && (len >= p->max_episode_steps);
            uint8_t d = (uint8_t)(term | (trunc << 1));
            if (rew[q] != 1.0f || done[q] != d) ok = 0;
            if (d) {
                orc_reset_draw(p, seed, env, t + 1u, nxt);
                ep = 0u;
            } else {
                ep = len;
            }
            if (ok && k + 1 < K) {
                for (int c = 0; c < 4; ++c) {
                    float gnext = obs[((size_t)(k + 1) * 4 + c) * n + i];
                    if (memcmp(&gnext, &nxt[c], sizeof(float)) != 0) ok = 0;
                }
            }
            if (ok && k + 1 == K) {
                for (int c = 0; c < 4 && final_state; ++c) {
                    float gnext = final_state[(size_t)c * n + i];
                    if (memcmp(&gnext, &nxt[c], sizeof(float)) != 0) ok = 0;
                }
                if (final_ep && final_ep[i] != ep) ok = 0;
            }
            if (!ok) {
                if (bad == 0 && bad_k && bad_i) {
                    *bad_k = k;
                    *bad_i = i;
                }
                ++bad;
            }
        }
    }
    if (stats) {
        stats[0] = worst;
        stats[1] = wmax;
        stats[2] = wsum;
    }
    if (exempt) *exempt = ex;
    return bad;
}

/* ======================================================================== */
/* Second simulator: a cart carrying a chain of N identical uniform rods.    */
/* The paper's Future Work points to heavier, multi-body simulators (its      */
/* Related Work names rigid-body engines); it gives no model, so this one is  */
/* derived here from its Lagrangian.                                          */
/*                                                                            */
/* Cart of mass mc on a frictionless track; links k = 1..N, each a uniform    */
/* rod of mass m and length L = 2 l, joined end to end, link 1 hinged on the  */
/* cart.  Generalised coordinates q = (x, phi_1, ..., phi_N), phi_k the angle */
/* of link k from the upward vertical (a link leaning towards +x has          */
/* positive phi).  With mu_k = (N - k) m the mass beyond link k:              */
/*   h_k = L (m/2 + mu_k)      (cart coupling / first moment of link k)       */
/*   G_kk = L^2 (m/3 + mu_k),  G_jk = L h_k for j < k   (link coupling)       */
/* the kinetic energy is                                                      */
/*   T = 1/2 (mc + N m) xd^2 + sum_k h_k cos(phi_k) xd phid_k                 */
/*       + 1/2 sum_jk G_jk cos(phi_j - phi_k) phid_j phid_k                   */
/* and the potential V = g sum_k h_k cos(phi_k), so Lagrange's equations are  */
/* M(q) qdd = f(q, qd) with the symmetric mass matrix                         */
/*   M_00 = mc + N m,  M_0k = h_k cos(phi_k),  M_jk = G_jk cos(phi_j - phi_k) */
/* and the forces                                                             */
/*   f_0 = F + sum_k h_k sin(phi_k) phid_k^2                                  */
/*   f_j = g h_j sin(phi_j) - sum_{k != j} G_jk sin(phi_j - phi_k) phid_k^2.  */
/* N = 1 is the cart-pole above (h = m l, G = 4/3 m l^2).                     */
/*                                                                            */
/* The fp32 evaluation, in this order (the GPU kernel does the same):         */
/*  - constants from (mc, m, l, g), once, one operation each: L = 2 l,        */
/*    mu_k = (N - k) * m, h_k = L * (0.5 m + mu_k), G_kk = (L * L) *          */
/*    (m / 3 + mu_k), Lh_k = L * h_k, gh_k = g * h_k, M_00 = mc + N * m;      */
/*  - (s_k, c_k) = sincos(phi_k) (the full-range form above), w_k = phid_k^2; */
/*  - cos(phi_j - phi_k) = fma(c_j, c_k, s_j s_k) and                         */
/*    sin(phi_j - phi_k) = fma(s_j, c_k, -(c_j s_k)) for each pair j < k;     */
/*  - f_0 = F, then f_0 = fma(h_k s_k, w_k, f_0) for k = 1..N; f_j = gh_j s_j, */
/*    then for each pair j < k in lexicographic order, P = Lh_k sin(phi_j -   */
/*    phi_k): f_j = fma(-P, w_k, f_j), f_k = fma(P, w_j, f_k);                */
/*  - Gaussian elimination without pivoting (M is positive definite) on the  */
/*    upper triangle: for pivot p, inv_p = 1 / A_pp (IEEE division), for      */
/*    i > p: l = A_pi inv_p, A_ij = fma(-l, A_pj, A_ij) for j >= i,           */
/*    f_i = fma(-l, f_p, f_i); then back substitution                         */
/*    qdd_i = (f_i - sum_{j > i} A_ij qdd_j) inv_i, the sum as fmas from      */
/*    j = i + 1 upwards;                                                      */
/*  - explicit Euler: positions advance with the old velocities.             */
/* ======================================================================== */
#define ORC_CHAIN_MAX_LINKS 8

typedef struct {
    uint32_t N;
    float m00;                                    /* mc + N m */
    float h[ORC_CHAIN_MAX_LINKS + 1];             /* [1..N] */
    float g_diag[ORC_CHAIN_MAX_LINKS + 1];        /* G_kk */
    float lh[ORC_CHAIN_MAX_LINKS + 1];            /* L h_k = G_jk for j < k */
    float gh[ORC_CHAIN_MAX_LINKS + 1];            /* g h_k */
} orc_chain_consts;

int orc_chain_make_consts(const orc_params* p, uint32_t N, orc_chain_consts* k)
{
    if (N < 1 || N > ORC_CHAIN_MAX_LINKS) return -1;
    memset(k, 0, sizeof(*k));
    k->N = N;
    float m = p->masspole;
    float L = 2.0f * p->half_length;
    float LL = L * L;
    float half_m = 0.5f * m;
    float third_m = m / 3.0f;
    for (uint32_t j = 1; j <= N; ++j) {
        float mu = (float)(N - j) * m;
        float hm = half_m + mu;
        k->h[j] = L * hm;
        float gm = third_m + mu;
        k->g_diag[j] = LL * gm;
        k->lh[j] = L * k->h[j];
        k->gh[j] = p->gravity * k->h[j];
    }
    float nm = (float)N * m;
    k->m00 = p->masscart + nm;
    return 0;
}

/* Accelerations qdd = (xdd, phidd_1..N) of the state (x, xd, phi_1, phid_1, ...) */
/* under the cart force F. */
void orc_chain_accel(const orc_chain_consts* k, const float* st, float force, float* qdd)
{
    uint32_t N = k->N, S = N + 1;
    float s[ORC_CHAIN_MAX_LINKS + 1], c[ORC_CHAIN_MAX_LINKS + 1], w[ORC_CHAIN_MAX_LINKS + 1];
    float A[ORC_CHAIN_MAX_LINKS + 1][ORC_CHAIN_MAX_LINKS + 1], f[ORC_CHAIN_MAX_LINKS + 1];
    float inv[ORC_CHAIN_MAX_LINKS + 1];
    for (uint32_t j = 1; j <= N; ++j) {
        float phi = st[2 * j], phid = st[2 * j + 1];
        orc_sincos(phi, &s[j], &c[j]);
        w[j] = phid * phid;
    }
    /* mass matrix, upper triangle */
    A[0][0] = k->m00;
    for (uint32_t j = 1; j <= N; ++j) {
        A[0][j] = k->h[j] * c[j];
        A[j][j] = k->g_diag[j];
    }
    for (uint32_t j = 1; j <= N; ++j)
        for (uint32_t i = j + 1; i <= N; ++i) {
            float ss = s[j] * s[i];
            float cjk = fmaf(c[j], c[i], ss);             /* cos(phi_j - phi_i) */
            A[j][i] = k->lh[i] * cjk;
        }
    /* forces */
    f[0] = force;
    for (uint32_t j = 1; j <= N; ++j) {
        float hs = k->h[j] * s[j];
        f[0] = fmaf(hs, w[j], f[0]);                      /* + h_j sin(phi_j) phid_j^2 */
    }
    for (uint32_t j = 1; j <= N; ++j) f[j] = k->gh[j] * s[j];
    for (uint32_t j = 1; j <= N; ++j)
        for (uint32_t i = j + 1; i <= N; ++i) {
            float cs = c[j] * s[i];
            float sjk = fmaf(s[j], c[i], -cs);            /* sin(phi_j - phi_i) */
            float P = k->lh[i] * sjk;                     /* G_ji sin(phi_j - phi_i) */
            f[j] = fmaf(-P, w[i], f[j]);
            f[i] = fmaf(P, w[j], f[i]);                   /* sin(phi_i - phi_j) = -sjk */
        }
    /* elimination on the upper triangle */
    for (uint32_t p = 0; p + 1 < S; ++p) {
        inv[p] = 1.0f / A[p][p];
        for (uint32_t i = p + 1; i < S; ++i) {
            float l = A[p][i] * inv[p];
            for (uint32_t j = i; j < S; ++j) A[i][j] = fmaf(-l, A[p][j], A[i][j]);
            f[i] = fmaf(-l, f[p], f[i]);
        }
    }
    inv[S - 1] = 1.0f / A[S - 1][S - 1];
    /* back substitution */
    for (uint32_t ii = S; ii-- > 0;) {
        float acc = f[ii];
        for (uint32_t j = ii + 1; j < S; ++j) acc = fmaf(-A[ii][j], qdd[j], acc);
        qdd[ii] = acc * inv[ii];
    }
}

/* One explicit-Euler iteration of length tau; a == 1 pushes towards +x. */
void orc_chain_euler(const orc_chain_consts* k, float tau, float force_mag, const float* in, int action, float* out)
{
    uint32_t N = k->N;
    float qdd[ORC_CHAIN_MAX_LINKS + 1];
    float force = action ? force_mag : -force_mag;
    orc_chain_accel(k, in, force, qdd);
    for (uint32_t j = 0; j <= N; ++j) {
        out[2 * j] = fmaf(tau, in[2 * j + 1], in[2 * j]);
        out[2 * j + 1] = fmaf(tau, qdd[j], in[2 * j + 1]);
    }
}

/* One simulation step: compute_factor C iterations of tau / C, the action held. */
void orc_chain_env_step(const orc_params* p, const orc_chain_consts* k, const float* in, int action, float* out)
{
    uint32_t C = p->compute_factor, S = 2 * (k->N + 1);
    float sub_tau = p->tau / (float)C;
    float cur[2 * (ORC_CHAIN_MAX_LINKS + 1)];
    for (uint32_t q = 0; q < S; ++q) cur[q] = in[q];
    for (uint32_t c = 0; c < C; ++c) {
        float nxt[2 * (ORC_CHAIN_MAX_LINKS + 1)];
        orc_chain_euler(k, sub_tau, p->force_mag, cur, action, nxt);
        for (uint32_t q = 0; q < S; ++q) cur[q] = nxt[q];
    }
    for (uint32_t q = 0; q < S; ++q) out[q] = cur[q];
}

/* Strict thresholds on the cart position and on every link angle. */
int orc_chain_terminated(const orc_params* p, uint32_t N, const float* st)
{
    if (p->no_termination) return 0;
    float x = st[0];
    int out = (x < -p->x_threshold) || (x > p->x_threshold);
    for (uint32_t j = 1; j <= N; ++j) {
        float phi = st[2 * j];
        out |= (phi < -p->theta_threshold_rad) || (phi > p->theta_threshold_rad);
    }
    return out;
}

/* Initial state of an episode that begins at global step t: stream RESET,    */
/* counter (env, t / 8, RESET, j) for j = 0, 1, ... supplying the 2N + 2      */
/* state words four at a time in state order.  Episodes of one env that begin */
/* in the same 8-step block would share a draw; with the default constants    */
/* none lasts fewer than 8 steps.                                             */
#define ORC_CHAIN_RESET_SHIFT 3u
void orc_chain_reset_draw(const orc_params* p, uint32_t N, uint64_t seed, uint32_t env, uint32_t t, float* out)
{
    uint32_t S = 2 * (N + 1);
    uint32_t key[2] = { (uint32_t)(seed & 0xFFFFFFFFu), (uint32_t)(seed >> 32) };
    for (uint32_t j = 0; 4 * j < S; ++j) {
        uint32_t ctr[4] = { env, t >> ORC_CHAIN_RESET_SHIFT, ORC_STREAM_RESET, j };
        uint32_t w[4];
        orc_philox4x32_10(ctr, key, w);
        for (uint32_t q = 0; q < 4 && 4 * j + q < S; ++q) out[4 * j + q] = orc_uniform(w[q], p->reset_low, p->reset_high);
    }
}

/* The vectorised chain simulator: n environments with global ids env0 ..,    */
/* each 2N + 2 state words [S][n] and an episode step counter; random         */
/* actions, auto-reset, per-256-env block statistics as orc_step.            */
typedef struct {
    uint32_t n, env0, N;
    orc_params p;
    orc_chain_consts k;
    uint64_t seed;
    uint32_t t;
    int has_reset;
    float* st;            /* [2N+2][n] */
    uint32_t* ep;         /* [n] */
} orc_chain_sim;

void orc_chain_destroy(orc_chain_sim* sim)
{
    if (!sim) return;
    free(sim->st); free(sim->ep);
    free(sim);
}

orc_chain_sim* orc_chain_create(uint32_t n, uint32_t env0, uint32_t N, const orc_params* p)
{
    if (n == 0 || p->compute_factor == 0 || N < 1 || N > ORC_CHAIN_MAX_LINKS) return NULL;
    orc_chain_sim* sim = (orc_chain_sim*)calloc(1, sizeof(orc_chain_sim));
    if (!sim) return NULL;
    sim->n = n; sim->env0 = env0; sim->N = N; sim->p = *p;
    orc_chain_make_consts(p, N, &sim->k);
    sim->st = (float*)calloc((size_t)2 * (N + 1) * n, sizeof(float));
    sim->ep = (uint32_t*)calloc(n, sizeof(uint32_t));
    if (!sim->st || !sim->ep) { orc_chain_destroy(sim); return NULL; }
    return sim;
}

void orc_chain_reset(orc_chain_sim* sim, uint64_t seed)
{
    uint32_t n = sim->n, S = 2 * (sim->N + 1);
    sim->seed = seed;
    sim->t = 0;
    sim->has_reset = 1;
    for (uint32_t i = 0; i < n; ++i) {
        float init[2 * (ORC_CHAIN_MAX_LINKS + 1)];
        orc_chain_reset_draw(&sim->p, sim->N, seed, sim->env0 + i, 0u, init);
        for (uint32_t q = 0; q < S; ++q) sim->st[(size_t)q * n + i] = init[q];
        sim->ep[i] = 0;
    }
}

/* K steps of every environment; outputs as orc_step with obs [K][S][n]. */
int orc_chain_step(orc_chain_sim* sim, uint32_t K, float* obs, uint8_t* act, float* rew, uint8_t* done,
                   uint32_t* stats)
{
    if (!sim->has_reset) return -1;
    if ((uint64_t)sim->t + (uint64_t)K > 0xFFFFFFFFull) return -2;
    uint32_t n = sim->n, N = sim->N, S = 2 * (N + 1);
    uint32_t blk0 = sim->env0 / 256u;
    if (stats) {
        uint32_t nblk = (sim->env0 + n - 1u) / 256u - blk0 + 1u;
        memset(stats, 0, (size_t)nblk * 4u * sizeof(uint32_t));
    }
    for (uint32_t k = 0; k < K; ++k) {
        uint32_t t = sim->t + k;
        for (uint32_t i = 0; i < n; ++i) {
            uint32_t env = sim->env0 + i;
            float cur[2 * (ORC_CHAIN_MAX_LINKS + 1)], nxt[2 * (ORC_CHAIN_MAX_LINKS + 1)];
            for (uint32_t q = 0; q < S; ++q) cur[q] = sim->st[(size_t)q * n + i];
            int a = orc_action_bit(sim->seed, env, t);
            orc_chain_env_step(&sim->p, &sim->k, cur, a, nxt);
            uint32_t len = sim->ep[i] + 1u;
            int term = orc_chain_terminated(&sim->p, N, nxt);
            int trunc = (sim->p.max_episode_steps != 0u) && (len >= sim->p.max_episode_steps);
            uint8_t d = (uint8_t)(term | (trunc << 1));
            if (obs) for (uint32_t q = 0; q < S; ++q) obs[((size_t)k * S + q) * n + i] = cur[q];
            if (act) act[(size_t)k * n + i] = (uint8_t)a;
            if (rew) rew[(size_t)k * n + i] = 1.0f;
            if (done) done[(size_t)k * n + i] = d;
            if (d) {
                orc_chain_reset_draw(&sim->p, N, sim->seed, env, t + 1u, nxt);
                sim->ep[i] = 0;
                if (stats) {
                    uint32_t* sb = stats + (size_t)(env / 256u - blk0) * 4u;
                    sb[0] += 1u;
                    sb[1] += len;
                    sb[2] += (uint32_t)term;
                    sb[3] += (uint32_t)trunc;
                }
            } else {
                sim->ep[i] = len;
            }
            for (uint32_t q = 0; q < S; ++q) sim->st[(size_t)q * n + i] = nxt[q];
        }
    }
    sim->t += K;
    return 0;
}

void orc_chain_get_state(const orc_chain_sim* sim, float* st, uint32_t* ep, uint64_t* t)
{
    size_t n = sim->n, S = 2 * (sim->N + 1);
    if (st) memcpy(st, sim->st, S * n * sizeof(float));
    if (ep) memcpy(ep, sim->ep, n * sizeof(uint32_t));
    if (t) *t = sim->t;
}

int orc_chain_set_state(orc_chain_sim* sim, const float* st, const uint32_t* ep, uint64_t t)
{
    if (!sim->has_reset) return -1;
    if (t > 0xFFFFFFFFull) return -2;
    size_t n = sim->n, S = 2 * (sim->N + 1);
    if (st) memcpy(sim->st, st, S * n * sizeof(float));
    if (ep) memcpy(sim->ep, ep, n * sizeof(uint32_t));
    sim->t = (uint32_t)t;
    return 0;
}

/* Teacher-forced check of recorded chain rows ([K][S][n] obs, [K][n] action, */
/* reward, done), with the same rules, options and return values as          */
/* orc_check_rows.                                                            */
uint64_t orc_chain_check_rows(const orc_params* p, uint32_t N, uint64_t seed, uint32_t env0, uint32_t n, uint32_t t0,
                              uint32_t K, const uint32_t* ep0, const float* obs, const uint8_t* act, const float* rew,
                              const uint8_t* done, const float* final_state, const uint32_t* final_ep,
                              uint32_t* bad_k, uint32_t* bad_i)
{
    orc_chain_consts kc;
    if (orc_chain_make_consts(p, N, &kc) != 0) return (uint64_t)-1;
    uint32_t S = 2 * (N + 1);
    uint64_t bad = 0;
    for (uint32_t i = 0; i < n; ++i) {
        uint32_t ep = ep0 ? ep0[i] : 0u;
        uint32_t env = env0 + i;
        for (uint32_t k = 0; k < K; ++k) {
            uint32_t t = t0 + k;
            float cur[2 * (ORC_CHAIN_MAX_LINKS + 1)], nxt[2 * (ORC_CHAIN_MAX_LINKS + 1)];
            for (uint32_t q = 0; q < S; ++q) cur[q] = obs[((size_t)k * S + q) * n + i];
            int ok = 1;
            if (k == 0 && !ep0) {
                float start[2 * (ORC_CHAIN_MAX_LINKS + 1)];
                orc_chain_reset_draw(p, N, seed, env, t0, start);
                if (memcmp(start, cur, S * sizeof(float)) != 0) ok = 0;
            }
            int a = orc_action_bit(seed, env, t);
            orc_chain_env_step(p, &kc, cur, a, nxt);
            uint32_t len = ep + 1u;
            int term = orc_chain_terminated(p, N, nxt);
            int trunc = (p->max_episode_steps != 0u) && (len >= p->max_episode_steps);
            uint8_t d = (uint8_t)(term | (trunc << 1));
            if (act[(size_t)k * n + i] != (uint8_t)a || rew[(size_t)k * n + i] != 1.0f || done[(size_t)k * n + i] != d)
                ok = 0;
            if (d) {
                orc_chain_reset_draw(p, N, seed, env, t + 1u, nxt);
                ep = 0u;
            } else {
                ep = len;
            }
            if (ok && k + 1 < K) {
                for (uint32_t q = 0; q < S; ++q) {
                    float g = obs[((size_t)(k + 1) * S + q) * n + i];
                    if (memcmp(&g, &nxt[q], sizeof(float)) != 0) ok = 0;
                }
            }
            if (ok && k + 1 == K) {
                for (uint32_t q = 0; q < S && final_state; ++q) {
                    float g = final_state[(size_t)q * n + i];
                    if (memcmp(&g, &nxt[q], sizeof(float)) != 0) ok = 0;
                }
                if (final_ep && final_ep[i] != ep) ok = 0;
            }
            if (!ok) {
                if (bad == 0 && bad_k && bad_i) {
                    *bad_k = k;
                    *bad_i = i;
                }
                ++bad;
            }
        }
    }
    return bad;
}
