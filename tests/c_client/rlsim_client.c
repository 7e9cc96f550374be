/*
 * rlsim_client.c -- a plain C11 client of include/rlsim.h, with no Python and
 * no torch: device buffers come from the HIP runtime's C API.  Used by the GPU
 * tests to show that the C ABI stands on its own.
 *
 * usage: rlsim_client N K SEED OUT
 *   creates N cart-pole environments (no padding words), resets them with SEED,
 *   runs K fused steps in one rlsim_step_fused call with a trajectory, and writes
 *   to OUT, in this order: obs [K][4][N] f32, action [K][N] u8, reward [K][N] f32,
 *   done [K][N] u8, the final state [4][N] f32, the episode counters [N] u32 and
 *   the global step t (u64).  It also checks two argument errors (K = 0, and a
 *   step before reset on a second handle) for their status and message.
 * Exit status: 0 on success, 1 on a bad command line or a failed check, 2 on an
 * rlsim or HIP error (the message goes to stderr).
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "rlsim.h"

static int check(int rc, const rlsim_t* h, const char* what)
{
    if (rc != RLSIM_OK) {
        fprintf(stderr, "%s failed (%d): %s\n", what, rc, rlsim_last_error(h));
        return 0;
    }
    return 1;
}

static int hip_ok(hipError_t e, const char* what)
{
    if (e != hipSuccess) {
        fprintf(stderr, "%s: %s\n", what, hipGetErrorString(e));
        return 0;
    }
    return 1;
}

int main(int argc, char** argv)
{
    if (argc != 5) {
        fprintf(stderr, "usage: %s N K SEED OUT\n", argv[0]);
        return 1;
    }
    const uint32_t n = (uint32_t)strtoul(argv[1], NULL, 10);
    const uint32_t K = (uint32_t)strtoul(argv[2], NULL, 10);
    const uint64_t seed = strtoull(argv[3], NULL, 10);
    if (n == 0 || K == 0) return 1;

    rlsim_cfg cfg;
    rlsim_cfg_default(&cfg);
    rlsim_t* h = NULL;
    if (!check(rlsim_create(n, 4, &cfg, &h), NULL, "rlsim_create")) return 2;

    /* a step before any reset is a state error with a message */
    rlsim_t* fresh = NULL;
    if (!check(rlsim_create(n, 4, NULL, &fresh), NULL, "rlsim_create (second)")) return 2;
    if (rlsim_step_fused(fresh, 1, NULL, NULL) != RLSIM_ESTATE || rlsim_last_error(fresh)[0] == '\0') {
        fprintf(stderr, "step before reset was not reported as RLSIM_ESTATE\n");
        return 1;
    }
    if (!check(rlsim_destroy(fresh), NULL, "rlsim_destroy (second)")) return 2;

    if (!check(rlsim_reset(h, seed), h, "rlsim_reset")) return 2;
    if (rlsim_step_fused(h, 0, NULL, NULL) != RLSIM_EINVAL || rlsim_last_error(h)[0] == '\0') {
        fprintf(stderr, "K = 0 was not reported as RLSIM_EINVAL\n");
        return 1;
    }

    const size_t rows = (size_t)K * n;
    float *obs = NULL, *reward = NULL;
    uint8_t *action = NULL, *done = NULL;
    if (!hip_ok(hipMalloc((void**)&obs, rows * 4 * sizeof(float)), "hipMalloc obs") ||
        !hip_ok(hipMalloc((void**)&reward, rows * sizeof(float)), "hipMalloc reward") ||
        !hip_ok(hipMalloc((void**)&action, rows), "hipMalloc action") ||
        !hip_ok(hipMalloc((void**)&done, rows), "hipMalloc done"))
        return 2;
    rlsim_traj traj;
    memset(&traj, 0, sizeof traj);
    traj.obs = obs;
    traj.action = action;
    traj.reward = reward;
    traj.done = done;
    if (!check(rlsim_step_fused(h, K, NULL, &traj), h, "rlsim_step_fused")) return 2;

    float* h_obs = malloc(rows * 4 * sizeof(float));
    float* h_reward = malloc(rows * sizeof(float));
    uint8_t* h_action = malloc(rows);
    uint8_t* h_done = malloc(rows);
    float* h_state = malloc((size_t)4 * n * sizeof(float));
    uint32_t* h_ep = malloc((size_t)n * sizeof(uint32_t));
    if (!h_obs || !h_reward || !h_action || !h_done || !h_state || !h_ep) return 2;
    uint64_t t = 0;
    /* rlsim_get_state synchronises the handle's stream, so the trajectory is complete */
    if (!check(rlsim_get_state(h, h_state, h_ep, &t), h, "rlsim_get_state")) return 2;
    if (!hip_ok(hipMemcpy(h_obs, obs, rows * 4 * sizeof(float), hipMemcpyDeviceToHost), "copy obs") ||
        !hip_ok(hipMemcpy(h_reward, reward, rows * sizeof(float), hipMemcpyDeviceToHost), "copy reward") ||
        !hip_ok(hipMemcpy(h_action, action, rows, hipMemcpyDeviceToHost), "copy action") ||
        !hip_ok(hipMemcpy(h_done, done, rows, hipMemcpyDeviceToHost), "copy done"))
        return 2;

    FILE* f = fopen(argv[4], "wb");
    if (!f) return 2;
    int ok = fwrite(h_obs, sizeof(float), rows * 4, f) == rows * 4 && fwrite(h_action, 1, rows, f) == rows &&
             fwrite(h_reward, sizeof(float), rows, f) == rows && fwrite(h_done, 1, rows, f) == rows &&
             fwrite(h_state, sizeof(float), (size_t)4 * n, f) == (size_t)4 * n &&
             fwrite(h_ep, sizeof(uint32_t), n, f) == n && fwrite(&t, sizeof t, 1, f) == 1;
    ok = (fclose(f) == 0) && ok;

    (void)hipFree(obs);
    (void)hipFree(reward);
    (void)hipFree(action);
    (void)hipFree(done);
    free(h_obs);
    free(h_reward);
    free(h_action);
    free(h_done);
    free(h_state);
    free(h_ep);
    if (!check(rlsim_destroy(h), NULL, "rlsim_destroy")) return 2;
    return ok ? 0 : 2;
}
