// rlsim.hip -- host runtime of the C ABI declared in include/rlsim.h:
// argument checks, device state ownership, kernel selection and launch.
#include "rlsim.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "k_chain.hip.h"
#include "k_policy.hip.h"
#include "k_wide.hip.h"

using namespace rlsim_dev;

struct rlsim {
    uint32_t n = 0;             // environments
    uint32_t D = 0;             // padding words per environment
    uint32_t model = RLSIM_MODEL_CARTPOLE;
    uint32_t links = 0;         // chain links N (chain model)
    uint32_t S = 4;             // simulator state words: 4, or 2N + 2 for the chain
    int device = 0;
    uint32_t cus = 1;           // compute units of the device (persistent-grid size)
    hipStream_t stream = nullptr;
    rlsim_cfg cfg{};
    DevParams dp{};
    ChainParams cp{};           // chain model: couplings (cp.p == dp)
    uint64_t t = 0;             // global step of the next step
    bool has_reset = false;
    float* cart = nullptr;      // [S][n]
    uint32_t* ep = nullptr;     // [n]
    bool wide = false;          // padding layout: false [D][n], true [n][Dp]
    uint32_t Dp = 0;            // wide row length (D rounded up to a multiple of 4)
    float* pad_s = nullptr;
    float* pad_a = nullptr;
    float* pad_b = nullptr;
    std::string err;
};

namespace {

thread_local std::string g_create_err;

int fail(rlsim* h, int code, const std::string& msg)
{
    if (h) h->err = msg;
    else g_create_err = msg;
    return code;
}

int hip_fail(rlsim* h, hipError_t e, const char* what)
{
    std::string m = std::string(what) + ": " + hipGetErrorString(e);
    return fail(h, RLSIM_EDEVICE, m);
}

// Makes the handle's device current for the scope, restoring the caller's.
struct DeviceGuard {
    int prev = -1;
    bool ok = true;
    explicit DeviceGuard(int dev)
    {
        if (hipGetDevice(&prev) != hipSuccess) { ok = false; return; }
        if (prev != dev && hipSetDevice(dev) != hipSuccess) ok = false;
    }
    ~DeviceGuard()
    {
        int cur = -1;
        if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
    }
};

bool finite(float v) { return std::isfinite(v); }

// Kernel constants, each one fp32 operation on the configured values.
DevParams make_dev_params(const rlsim_cfg& c, uint64_t seed)
{
    DevParams p{};
    volatile float total = c.masscart + c.masspole;    // volatile: one rounding per line
    volatile float pole_ml = c.masspole * c.half_length;
    volatile float inv_total = 1.0f / total;
    volatile float m_over_M = c.masspole * inv_total;
    volatile float ml_over_M = pole_ml * inv_total;
    volatile float width = c.reset_high - c.reset_low;
    volatile float tau_iter = c.tau / (float)c.compute_factor;
    p.gravity = c.gravity;
    p.force_mag = c.force_mag;
    p.tau = tau_iter;
    p.iters = c.compute_factor;
    p.half_length = c.half_length;
    p.pole_ml = pole_ml;
    p.inv_total = inv_total;
    p.m_over_M = m_over_M;
    p.ml_over_M = ml_over_M;
    const bool noterm = (c.flags & RLSIM_F_NO_TERMINATION) != 0u;
    p.thr_x = noterm ? INFINITY : c.x_threshold;
    p.thr_th = noterm ? INFINITY : c.theta_threshold_rad;
    p.max_steps = c.max_episode_steps;
    p.reset_lo = c.reset_low;
    p.reset_width = width;
    p.reset_width_u24 = std::ldexp((float)width, -24);   // exact: check_cfg bounds the width
    p.key0 = (uint32_t)(seed & 0xFFFFFFFFull);
    p.key1 = (uint32_t)(seed >> 32);
    p.env0 = c.env0;
    return p;
}

// The chain's couplings, each one fp32 operation on the configured values,
// in the order the kernel's definition fixes: L = 2 l, mu_k = (N - k) m,
// h_k = L (m/2 + mu_k), G_kk = (L L)(m/3 + mu_k), L h_k, g h_k, mc + N m.
ChainParams make_chain_params(const rlsim_cfg& c, uint32_t N, const DevParams& dp)
{
    ChainParams cp{};
    cp.p = dp;
    const float m = c.masspole;
    volatile float L = 2.0f * c.half_length;
    volatile float LL = L * L;
    volatile float half_m = 0.5f * m;
    volatile float third_m = m / 3.0f;
    for (uint32_t j = 1; j <= N; ++j) {
        volatile float mu = (float)(N - j) * m;
        volatile float hm = half_m + mu;
        volatile float h = L * hm;
        volatile float gm = third_m + mu;
        volatile float gd = LL * gm;
        volatile float lh = L * h;
        volatile float gh = c.gravity * h;
        cp.h[j] = h;
        cp.gdiag[j] = gd;
        cp.lh[j] = lh;
        cp.gh[j] = gh;
    }
    volatile float nm = (float)N * m;
    volatile float m00 = c.masscart + nm;
    cp.m00 = m00;
    return cp;
}

const char* check_cfg(const rlsim_cfg& c)
{
    const float vals[] = {c.gravity, c.masscart, c.masspole, c.half_length, c.force_mag, c.tau, c.x_threshold,
                          c.theta_threshold_rad, c.reset_low, c.reset_high, c.pad_a_low, c.pad_a_high,
                          c.pad_b_low, c.pad_b_high};
    for (float v : vals)
        if (!finite(v)) return "cfg: every constant must be finite";
    if (!(c.masscart > 0.0f) || !(c.masspole > 0.0f)) return "cfg: masses must be positive";
    if (!(c.half_length > 0.0f)) return "cfg: half_length must be positive";
    if (!(c.tau > 0.0f)) return "cfg: tau must be positive";
    if (c.reset_low > c.reset_high) return "cfg: reset_low > reset_high";
    {
        // the kernels scale the reset width by 2^-24, which must stay exact
        volatile float width = c.reset_high - c.reset_low;
        if (!std::isfinite((float)width)) return "cfg: reset range too wide";
        if (width != 0.0f && std::fabs((float)width) < 0x1.0p-100f) return "cfg: reset range narrower than 2^-100";
    }
    if (c.pad_a_low > c.pad_a_high || c.pad_b_low > c.pad_b_high) return "cfg: padding range low > high";
    if ((c.flags & ~(uint32_t)RLSIM_F_NO_TERMINATION) != 0u) return "cfg: unknown flag bits";
    if (c.compute_factor == 0u) return "cfg: compute_factor must be >= 1";
    if (c.env0 % 256u != 0u) return "cfg: env0 must be a multiple of 256";
    if (c.model != RLSIM_MODEL_CARTPOLE && c.model != RLSIM_MODEL_CHAIN) return "cfg: unknown model";
    if (c.model == RLSIM_MODEL_CHAIN && (c.n_links < 1u || c.n_links > (uint32_t)kMaxLinks))
        return "cfg: n_links must be in [1, 4] for the chain model";
    return nullptr;
}

void free_state(rlsim* h)
{
    if (h->cart) (void)hipFree(h->cart);
    if (h->ep) (void)hipFree(h->ep);
    if (h->pad_s) (void)hipFree(h->pad_s);
    if (h->pad_a) (void)hipFree(h->pad_a);
    if (h->pad_b) (void)hipFree(h->pad_b);
    h->cart = nullptr;
    h->ep = nullptr;
    h->pad_s = h->pad_a = h->pad_b = nullptr;
}

// Host-side layout conversion of the wide padding words, in 64 x 64 tiles:
// rows[env * Dp + j] <-> planes[j * n + env].
constexpr size_t kTile = 64;
void transpose_rows_to_planes(const float* rows, float* planes, size_t n, size_t D, size_t Dp)
{
    for (size_t e0 = 0; e0 < n; e0 += kTile)
        for (size_t j0 = 0; j0 < D; j0 += kTile)
            for (size_t j = j0; j < std::min(D, j0 + kTile); ++j)
                for (size_t e = e0; e < std::min(n, e0 + kTile); ++e) planes[j * n + e] = rows[e * Dp + j];
}
void transpose_planes_to_rows(const float* planes, float* rows, size_t n, size_t D, size_t Dp)
{
    for (size_t e0 = 0; e0 < n; e0 += kTile)
        for (size_t j0 = 0; j0 < D; j0 += kTile)
            for (size_t e = e0; e < std::min(n, e0 + kTile); ++e)
                for (size_t j = j0; j < std::min(D, j0 + kTile); ++j) rows[e * Dp + j] = planes[j * n + e];
}

bool aligned4(const void* ptr) { return ((uintptr_t)ptr & 3u) == 0u; }

unsigned grid_for(uint32_t n) { return (n + kBlock - 1u) / kBlock; }

// Largest padding count of the register-resident (one thread per env) kernel;
// above it the two-phase wide kernel holds the words.  (262,144 envs x 500
// steps: D = 32 0.82-0.87 ms in registers; the wide kernel's eight-environment
// jump table, one word per lane, costs the same at every D up to 64, 0.88-0.94 ms
// at D = 48 and 64, where the register form, every thread updating all 64 words,
// takes 1.07-1.13 ms.)
constexpr uint32_t kMaxRegisterWords = 32u;
// Fewest steps per call for which a trajectory-recording call runs the
// warp-specialised kernel: without padding words, and with 1-4 padding words.
// Below them the hand-over's pipeline fill and drain cost more than the faster
// stores save (4,194,304 envs, D = 0: 26.5 against 23.5 us per step at K = 8,
// 20.1 against 21.1 at K = 16; 262,144 envs, D = 4: 0.76 against 0.71 ms per
// 512 steps at K = 16, 0.60 against 0.62 at K = 100).
constexpr uint32_t kSplitMinSteps = 16u;
constexpr uint32_t kSplitPadMinSteps = 64u;
// Largest state: 2^24 padding words per environment (3 x 64 MiB of device
// memory per environment), which keeps the wide kernel's 32-bit word indices
// (row offsets, chunk counts) far from overflow.
constexpr uint32_t kMaxStateWords = (1u << 24) + 4u;

template <bool REC, bool STATS>
hipError_t launch_step(const StepArgs& a, bool wide, uint32_t cus, hipStream_t s)
{
    const dim3 grid(grid_for(a.n)), block(kBlock);
    if (!wide) {
        if (a.D == 0u && REC && a.K >= kSplitMinSteps)
            hipLaunchKernelGGL((k_cartpole_split<0, STATS>), grid, dim3(2 * kBlock), 0, s, a);
        else if (a.D <= 4u && REC && a.K >= kSplitPadMinSteps)
            hipLaunchKernelGGL((k_cartpole_split<4, STATS>), grid, dim3(2 * kBlock), 0, s, a);
        else if (a.D == 0u) hipLaunchKernelGGL((k_cartpole_fused<0, REC, STATS>), grid, block, 0, s, a);
        else if (a.D <= 4u) hipLaunchKernelGGL((k_cartpole_fused<4, REC, STATS>), grid, block, 0, s, a);
        else if (a.D <= 8u) hipLaunchKernelGGL((k_cartpole_fused<8, REC, STATS>), grid, block, 0, s, a);
        else if (a.D <= 16u) hipLaunchKernelGGL((k_cartpole_fused<16, REC, STATS>), grid, block, 0, s, a);
        else hipLaunchKernelGGL((k_cartpole_fused<32, REC, STATS>), grid, block, 0, s, a);
    } else {
        // one environment per wave in the replay (wave-uniform bits), W words
        // per lane; E environments replayed together where that pays
        // (262,144 envs x 500 steps, phases not overlapped: D = 256 1.84 / 1.98 /
        // 2.24 ms for E = 4 / 2 / 1, D = 512 3.10 / 2.55 / 2.81 ms).  Up to 64
        // words: one word per lane, eight environments per step through the
        // replay's jump table.  Above 512 words, 16 words per lane in chunks of
        // 1,024 (D = 2,048 / 4,096 / 5,000: 5.90-5.92 / 11.16-11.20 /
        // 13.84-13.85 ms against 6.01-6.10 / 11.61 / 16.4 ms with 32 words per
        // lane at four waves per SIMD, whose 2,048-word chunks waste more of the
        // last one, and 11.9-12.4 ms at D = 4,096 with 64 words at two waves).
        // Every shape fits the 64 VGPRs of eight waves per SIMD: two persistent
        // 16-wave workgroups per CU.
        const dim3 grid2(min(grid_for(a.n), 2u * cus)), block2(1024);
        if (a.D <= 64u) hipLaunchKernelGGL((k_cartpole_wide<1, 8, 16, REC, STATS>), grid2, block2, 0, s, a);
        else if (a.D <= 256u) hipLaunchKernelGGL((k_cartpole_wide<4, 4, 16, REC, STATS>), grid2, block2, 0, s, a);
        else if (a.D <= 512u) hipLaunchKernelGGL((k_cartpole_wide<8, 2, 16, REC, STATS>), grid2, block2, 0, s, a);
        else hipLaunchKernelGGL((k_cartpole_wide<16, 1, 16, REC, STATS>), grid2, block2, 0, s, a);
    }
    return hipGetLastError();
}

// Fewest steps per call for which a trajectory-recording chain call runs the
// warp-specialised chain kernel.
constexpr uint32_t kChainSplitMinSteps = 16u;

template <bool REC, bool STATS>
hipError_t launch_chain(const ChainArgs& a, uint32_t N, hipStream_t s)
{
    const dim3 grid(grid_for(a.n)), block(kBlock);
    if (REC && a.K >= kChainSplitMinSteps) {
        const dim3 wide_block(2 * kBlock);
        switch (N) {
        case 1: hipLaunchKernelGGL((k_chain_split<1, STATS>), grid, wide_block, 0, s, a); break;
        case 2: hipLaunchKernelGGL((k_chain_split<2, STATS>), grid, wide_block, 0, s, a); break;
        case 3: hipLaunchKernelGGL((k_chain_split<3, STATS>), grid, wide_block, 0, s, a); break;
        default: hipLaunchKernelGGL((k_chain_split<4, STATS>), grid, wide_block, 0, s, a); break;
        }
        return hipGetLastError();
    }
    switch (N) {
    case 1: hipLaunchKernelGGL((k_chain_fused<1, REC, STATS>), grid, block, 0, s, a); break;
    case 2: hipLaunchKernelGGL((k_chain_fused<2, REC, STATS>), grid, block, 0, s, a); break;
    case 3: hipLaunchKernelGGL((k_chain_fused<3, REC, STATS>), grid, block, 0, s, a); break;
    default: hipLaunchKernelGGL((k_chain_fused<4, REC, STATS>), grid, block, 0, s, a); break;
    }
    return hipGetLastError();
}

hipError_t launch_chain_reset(const DevParams& p, uint32_t N, uint32_t n, float* state, uint32_t* ep, hipStream_t s)
{
    const dim3 grid(grid_for(n)), block(kBlock);
    switch (N) {
    case 1: hipLaunchKernelGGL(k_reset_chain<1>, grid, block, 0, s, p, n, state, ep); break;
    case 2: hipLaunchKernelGGL(k_reset_chain<2>, grid, block, 0, s, p, n, state, ep); break;
    case 3: hipLaunchKernelGGL(k_reset_chain<3>, grid, block, 0, s, p, n, state, ep); break;
    default: hipLaunchKernelGGL(k_reset_chain<4>, grid, block, 0, s, p, n, state, ep); break;
    }
    return hipGetLastError();
}

template <class Mlp, bool REC, bool STATS>
hipError_t launch_policy(const StepArgs& a, const PolicyArgs& w, hipStream_t s)
{
    const dim3 grid(grid_for(a.n)), block(kBlock);
    if (w.p0 || w.logp || w.value) hipLaunchKernelGGL((k_policy_fused<Mlp, REC, STATS, true>), grid, block, 0, s, a, w);
    else hipLaunchKernelGGL((k_policy_fused<Mlp, REC, STATS, false>), grid, block, 0, s, a, w);
    return hipGetLastError();
}

template <class Mlp>
hipError_t launch_policy_any(const StepArgs& a, const PolicyArgs& w, bool rec, bool stats, hipStream_t s)
{
    if (rec && stats) return launch_policy<Mlp, true, true>(a, w, s);
    if (rec) return launch_policy<Mlp, true, false>(a, w, s);
    if (stats) return launch_policy<Mlp, false, true>(a, w, s);
    return launch_policy<Mlp, false, false>(a, w, s);
}

}  // namespace

extern "C" {

void rlsim_cfg_default(rlsim_cfg* c)
{
    if (!c) return;
    c->gravity = 9.8f;
    c->masscart = 1.0f;
    c->masspole = 0.1f;
    c->half_length = 0.5f;
    c->force_mag = 10.0f;
    c->tau = 0.02f;
    c->x_threshold = 2.4f;
    c->theta_threshold_rad = (float)(12.0 * 2.0 * 3.14159265358979323846 / 360.0);
    c->max_episode_steps = 500u;
    c->reset_low = -0.05f;
    c->reset_high = 0.05f;
    c->pad_a_low = 0.9f;
    c->pad_a_high = 0.99f;
    c->pad_b_low = -1.0f;
    c->pad_b_high = 1.0f;
    c->flags = 0u;
    c->compute_factor = 1u;
    c->env0 = 0u;
    c->model = RLSIM_MODEL_CARTPOLE;
    c->n_links = 0u;
    c->stream = nullptr;
}

int rlsim_create(uint32_t n_envs, uint32_t state_words, const rlsim_cfg* cfg, rlsim_t** out)
{
    if (!out) return fail(nullptr, RLSIM_EINVAL, "rlsim_create: out is NULL");
    *out = nullptr;
    if (n_envs == 0u || n_envs > (1u << 30)) return fail(nullptr, RLSIM_EINVAL, "rlsim_create: n_envs must be in [1, 2^30]");
    if (state_words < 4u || state_words > kMaxStateWords)
        return fail(nullptr, RLSIM_EINVAL, "rlsim_create: state_words must be in [4, 2^24 + 4]");
    rlsim_cfg c;
    if (cfg) c = *cfg;
    else rlsim_cfg_default(&c);
    if (const char* why = check_cfg(c)) return fail(nullptr, RLSIM_EINVAL, std::string("rlsim_create: ") + why);
    if ((uint64_t)c.env0 + n_envs > (1ull << 32))
        return fail(nullptr, RLSIM_EINVAL, "rlsim_create: env0 + n_envs must be <= 2^32 (global ids are 32-bit)");
    const bool chain = c.model == RLSIM_MODEL_CHAIN;
    const uint32_t S = chain ? 2u * (c.n_links + 1u) : 4u;
    if (chain && state_words != S)
        return fail(nullptr, RLSIM_EINVAL, "rlsim_create: the chain model takes state_words = 2 n_links + 2");
    const uint32_t D = state_words - S;

    rlsim* h = new (std::nothrow) rlsim();
    if (!h) return fail(nullptr, RLSIM_ENOMEM, "rlsim_create: host allocation failed");
    h->n = n_envs;
    h->D = D;
    h->model = c.model;
    h->links = chain ? c.n_links : 0u;
    h->S = S;
    h->wide = D > kMaxRegisterWords;
    h->Dp = h->wide ? (D + 3u) & ~3u : D;
    h->cfg = c;
    h->stream = (hipStream_t)c.stream;
    hipError_t e = hipGetDevice(&h->device);
    if (e != hipSuccess) {
        int rc = hip_fail(nullptr, e, "rlsim_create: hipGetDevice");
        delete h;
        return rc;
    }
    int cus = 0;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, h->device);
    if (e != hipSuccess) {
        int rc = hip_fail(nullptr, e, "rlsim_create: hipDeviceGetAttribute");
        delete h;
        return rc;
    }
    h->cus = cus > 0 ? (uint32_t)cus : 1u;
    const size_t n = n_envs;
    e = hipMalloc(&h->cart, (size_t)S * n * sizeof(float));
    if (e == hipSuccess) e = hipMalloc(&h->ep, n * sizeof(uint32_t));
    const size_t pad_bytes = (size_t)h->Dp * n * sizeof(float);
    if (e == hipSuccess && D) e = hipMalloc(&h->pad_s, pad_bytes);
    if (e == hipSuccess && D) e = hipMalloc(&h->pad_a, pad_bytes);
    if (e == hipSuccess && D) e = hipMalloc(&h->pad_b, pad_bytes);
    // the wide layout's row tails [D, Dp) stay zero for the handle's lifetime
    if (e == hipSuccess && h->wide) e = hipMemset(h->pad_s, 0, pad_bytes);
    if (e == hipSuccess && h->wide) e = hipMemset(h->pad_a, 0, pad_bytes);
    if (e == hipSuccess && h->wide) e = hipMemset(h->pad_b, 0, pad_bytes);
    if (e != hipSuccess) {
        int rc = (e == hipErrorOutOfMemory) ? fail(nullptr, RLSIM_ENOMEM, "rlsim_create: device allocation failed")
                                            : hip_fail(nullptr, e, "rlsim_create: hipMalloc");
        (void)hipGetLastError();
        free_state(h);
        delete h;
        return rc;
    }
    *out = h;
    return RLSIM_OK;
}

int rlsim_reset(rlsim_t* h, uint64_t seed)
{
    if (!h) return fail(nullptr, RLSIM_EINVAL, "rlsim_reset: handle is NULL");
    DeviceGuard g(h->device);
    if (!g.ok) return fail(h, RLSIM_EDEVICE, "rlsim_reset: cannot select the handle's device");
    h->dp = make_dev_params(h->cfg, seed);
    hipError_t e;
    if (h->model == RLSIM_MODEL_CHAIN) {
        h->cp = make_chain_params(h->cfg, h->links, h->dp);
        e = launch_chain_reset(h->dp, h->links, h->n, h->cart, h->ep, h->stream);
    } else {
        hipLaunchKernelGGL(k_reset_cart, dim3(grid_for(h->n)), dim3(kBlock), 0, h->stream, h->dp, h->n, h->cart,
                           h->ep);
        e = hipGetLastError();
    }
    if (e != hipSuccess) return hip_fail(h, e, "rlsim_reset: launch");
    if (h->D) {
        volatile float a_w = h->cfg.pad_a_high - h->cfg.pad_a_low;
        volatile float b_w = h->cfg.pad_b_high - h->cfg.pad_b_low;
        const size_t pairs = (size_t)h->n * h->D;
        const unsigned blocks = (unsigned)std::min<size_t>((pairs + kBlock - 1) / kBlock, 65536);
        const size_t stride_j = h->wide ? 1 : (size_t)h->n;
        const size_t stride_e = h->wide ? (size_t)h->Dp : 1;
        hipLaunchKernelGGL(k_reset_pad, dim3(blocks), dim3(kBlock), 0, h->stream, h->dp, h->n, h->D, stride_j,
                           stride_e, h->cfg.pad_a_low, (float)a_w, h->cfg.pad_b_low, (float)b_w, h->pad_s,
                           h->pad_a, h->pad_b);
        e = hipGetLastError();
        if (e != hipSuccess) return hip_fail(h, e, "rlsim_reset: launch");
    }
    h->t = 0;
    h->has_reset = true;
    h->err.clear();
    return RLSIM_OK;
}

int rlsim_step_fused(rlsim_t* h, uint32_t K, const rlsim_policy* policy, const rlsim_traj* traj)
{
    if (!h) return fail(nullptr, RLSIM_EINVAL, "rlsim_step_fused: handle is NULL");
    if (!h->has_reset) return fail(h, RLSIM_ESTATE, "rlsim_step_fused: called before rlsim_reset");
    if (K == 0u) return fail(h, RLSIM_EINVAL, "rlsim_step_fused: K must be >= 1");
    if (h->t + (uint64_t)K > 0xFFFFFFFFull) return fail(h, RLSIM_EINVAL, "rlsim_step_fused: global step would pass 2^32 - 1");
    rlsim_traj tr{};
    if (traj) tr = *traj;
    const int n_set = (tr.obs != nullptr) + (tr.action != nullptr) + (tr.reward != nullptr) + (tr.done != nullptr);
    if (n_set != 0 && n_set != 4)
        return fail(h, RLSIM_EINVAL, "rlsim_step_fused: obs, action, reward and done must be all set or all NULL");
    if (!aligned4(tr.obs) || !aligned4(tr.reward) || !aligned4(tr.block_stats) || !aligned4(tr.policy_p0) ||
        !aligned4(tr.logp) || !aligned4(tr.value))
        return fail(h, RLSIM_EINVAL, "rlsim_step_fused: f32/u32 pointers must be 4-byte aligned");
    if ((tr.policy_p0 || tr.logp || tr.value) && !policy)
        return fail(h, RLSIM_EINVAL, "rlsim_step_fused: policy_p0, logp and value need a policy");
    if (policy) {
        if (policy->dtype != RLSIM_F32 && policy->dtype != RLSIM_BF16)
            return fail(h, RLSIM_EINVAL, "rlsim_step_fused: unknown policy dtype");
        if (!policy->w1 || !policy->w2 || !policy->w3)
            return fail(h, RLSIM_EINVAL, "rlsim_step_fused: policy weights must not be NULL");
        if (tr.value && !policy->wv)
            return fail(h, RLSIM_EINVAL, "rlsim_step_fused: value output needs the value head wv");
        const size_t wal = policy->dtype == RLSIM_F32 ? 4 : 2;
        if (((uintptr_t)policy->w1 | (uintptr_t)policy->w2 | (uintptr_t)policy->w3 | (uintptr_t)policy->wv) % wal != 0 ||
            !aligned4(policy->b1) || !aligned4(policy->b2) || !aligned4(policy->b3) || !aligned4(policy->bv))
            return fail(h, RLSIM_EINVAL, "rlsim_step_fused: misaligned policy arrays");
        if (h->D != 0u)
            return fail(h, RLSIM_EUNSUPPORTED, "rlsim_step_fused: a policy with padding words is not supported");
        if (h->model != RLSIM_MODEL_CARTPOLE)
            return fail(h, RLSIM_EUNSUPPORTED, "rlsim_step_fused: the MLP policy reads the cart-pole's 4 state words");
    }

    DeviceGuard g(h->device);
    if (!g.ok) return fail(h, RLSIM_EDEVICE, "rlsim_step_fused: cannot select the handle's device");
    const bool rec = n_set == 4, stats = tr.block_stats != nullptr;
    hipError_t e;
    if (h->model == RLSIM_MODEL_CHAIN) {
        ChainArgs ca{};
        ca.c = h->cp;
        ca.n = h->n;
        ca.t0 = (uint32_t)h->t;
        ca.K = K;
        ca.state = h->cart;
        ca.ep = h->ep;
        ca.obs = tr.obs;
        ca.action = tr.action;
        ca.reward = tr.reward;
        ca.done = tr.done;
        ca.stats = tr.block_stats;
        if (rec && stats) e = launch_chain<true, true>(ca, h->links, h->stream);
        else if (rec) e = launch_chain<true, false>(ca, h->links, h->stream);
        else if (stats) e = launch_chain<false, true>(ca, h->links, h->stream);
        else e = launch_chain<false, false>(ca, h->links, h->stream);
        if (e != hipSuccess) return hip_fail(h, e, "rlsim_step_fused: launch");
        h->t += K;
        return RLSIM_OK;
    }
    StepArgs a{};
    a.p = h->dp;
    a.n = h->n;
    a.D = h->D;
    a.Dp = h->Dp;
    a.t0 = (uint32_t)h->t;
    a.K = K;
    a.cart = h->cart;
    a.ep = h->ep;
    a.pad_s = h->pad_s;
    a.pad_a = h->pad_a;
    a.pad_b = h->pad_b;
    a.obs = tr.obs;
    a.action = tr.action;
    a.reward = tr.reward;
    a.done = tr.done;
    a.stats = tr.block_stats;
    if (policy) {
        PolicyArgs w{policy->w1, policy->b1, policy->w2, policy->b2, policy->w3, policy->b3,
                     policy->wv, policy->bv, tr.policy_p0, tr.logp, tr.value};
        e = policy->dtype == RLSIM_BF16 ? launch_policy_any<MlpBf16>(a, w, rec, stats, h->stream)
                                        : launch_policy_any<MlpF32>(a, w, rec, stats, h->stream);
        if (e != hipSuccess) return hip_fail(h, e, "rlsim_step_fused: launch");
        h->t += K;
        return RLSIM_OK;
    }
    if (rec && stats) e = launch_step<true, true>(a, h->wide, h->cus, h->stream);
    else if (rec) e = launch_step<true, false>(a, h->wide, h->cus, h->stream);
    else if (stats) e = launch_step<false, true>(a, h->wide, h->cus, h->stream);
    else e = launch_step<false, false>(a, h->wide, h->cus, h->stream);
    if (e != hipSuccess) return hip_fail(h, e, "rlsim_step_fused: launch");
    h->t += K;
    return RLSIM_OK;
}

int rlsim_get_state(rlsim_t* h, float* host_state, uint32_t* host_ep, uint64_t* t_out)
{
    if (!h) return fail(nullptr, RLSIM_EINVAL, "rlsim_get_state: handle is NULL");
    if (!h->has_reset) return fail(h, RLSIM_ESTATE, "rlsim_get_state: called before rlsim_reset");
    DeviceGuard g(h->device);
    if (!g.ok) return fail(h, RLSIM_EDEVICE, "rlsim_get_state: cannot select the handle's device");
    const size_t n = h->n;
    std::vector<float> rows;     // wide layout staging, [n][Dp]
    hipError_t e = hipSuccess;
    if (host_state) {
        e = hipMemcpyAsync(host_state, h->cart, (size_t)h->S * n * sizeof(float), hipMemcpyDeviceToHost, h->stream);
        if (e == hipSuccess && h->D && !h->wide)
            e = hipMemcpyAsync(host_state + (size_t)h->S * n, h->pad_s, (size_t)h->D * n * sizeof(float), hipMemcpyDeviceToHost,
                               h->stream);
        if (e == hipSuccess && h->wide) {
            try {
                rows.resize((size_t)h->Dp * n);
            } catch (const std::bad_alloc&) {
                return fail(h, RLSIM_ENOMEM, "rlsim_get_state: host staging allocation failed");
            }
            e = hipMemcpyAsync(rows.data(), h->pad_s, rows.size() * sizeof(float), hipMemcpyDeviceToHost, h->stream);
        }
    }
    if (e == hipSuccess && host_ep) e = hipMemcpyAsync(host_ep, h->ep, n * sizeof(uint32_t), hipMemcpyDeviceToHost, h->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(h->stream);
    if (e != hipSuccess) return hip_fail(h, e, "rlsim_get_state");
    if (host_state && h->wide) transpose_rows_to_planes(rows.data(), host_state + (size_t)h->S * n, n, h->D, h->Dp);
    if (t_out) *t_out = h->t;
    return RLSIM_OK;
}

int rlsim_set_state(rlsim_t* h, const float* host_state, const uint32_t* host_ep, uint64_t t)
{
    if (!h) return fail(nullptr, RLSIM_EINVAL, "rlsim_set_state: handle is NULL");
    if (!h->has_reset) return fail(h, RLSIM_ESTATE, "rlsim_set_state: called before rlsim_reset");
    if (t > 0xFFFFFFFFull) return fail(h, RLSIM_EINVAL, "rlsim_set_state: t must be <= 2^32 - 1");
    DeviceGuard g(h->device);
    if (!g.ok) return fail(h, RLSIM_EDEVICE, "rlsim_set_state: cannot select the handle's device");
    const size_t n = h->n;
    std::vector<float> rows;
    if (host_state && h->wide) {
        try {
            rows.assign((size_t)h->Dp * n, 0.0f);
        } catch (const std::bad_alloc&) {
            return fail(h, RLSIM_ENOMEM, "rlsim_set_state: host staging allocation failed");
        }
        transpose_planes_to_rows(host_state + (size_t)h->S * n, rows.data(), n, h->D, h->Dp);
    }
    hipError_t e = hipSuccess;
    if (host_state) {
        e = hipMemcpyAsync(h->cart, host_state, (size_t)h->S * n * sizeof(float), hipMemcpyHostToDevice, h->stream);
        if (e == hipSuccess && h->D && !h->wide)
            e = hipMemcpyAsync(h->pad_s, host_state + (size_t)h->S * n, (size_t)h->D * n * sizeof(float), hipMemcpyHostToDevice,
                               h->stream);
        if (e == hipSuccess && h->wide)
            e = hipMemcpyAsync(h->pad_s, rows.data(), rows.size() * sizeof(float), hipMemcpyHostToDevice, h->stream);
    }
    if (e == hipSuccess && host_ep) e = hipMemcpyAsync(h->ep, host_ep, n * sizeof(uint32_t), hipMemcpyHostToDevice, h->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(h->stream);
    if (e != hipSuccess) return hip_fail(h, e, "rlsim_set_state");
    h->t = t;
    return RLSIM_OK;
}

int rlsim_destroy(rlsim_t* h)
{
    if (!h) return RLSIM_OK;
    int rc = RLSIM_OK;
    {
        DeviceGuard g(h->device);
        hipError_t e = hipStreamSynchronize(h->stream);
        if (e != hipSuccess) rc = RLSIM_EDEVICE;
        free_state(h);
    }
    delete h;
    return rc;
}

const char* rlsim_last_error(const rlsim_t* h)
{
    return h ? h->err.c_str() : g_create_err.c_str();
}

}  // extern "C"
