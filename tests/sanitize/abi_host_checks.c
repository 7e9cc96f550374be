/*
 * abi_host_checks.c -- the C ABI's argument checks run in a process where the
 * library's host code is built with AddressSanitizer and
 * UndefinedBehaviorSanitizer (tests/test_abi_sanitized.py builds both).  Every
 * call here fails, or succeeds, before any device work: NULL handles and
 * outputs, out-of-range sizes, global env offsets and chain shapes, and seeded
 * draws of invalid configurations, each checked for its status and for a
 * non-empty message.  Exit status 0 when every expectation holds.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "rlsim.h"

static int failures = 0;

static void expect(int cond, const char* what)
{
    if (!cond) {
        fprintf(stderr, "FAILED: %s\n", what);
        ++failures;
    }
}

static void expect_create_einval(uint32_t n, uint32_t words, const rlsim_cfg* c, const char* what)
{
    rlsim_t* h = (rlsim_t*)0x1;
    int rc = rlsim_create(n, words, c, &h);
    expect(rc == RLSIM_EINVAL && h == NULL, what);
    const char* m = rlsim_last_error(NULL);
    expect(m != NULL && strlen(m) > 0, "create failure leaves a message");
}

/* splitmix64: a seeded stream for the invalid-configuration draws */
static uint64_t mix(uint64_t* s)
{
    uint64_t z = (*s += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

int main(void)
{
    rlsim_cfg c;
    rlsim_cfg_default(NULL);
    rlsim_cfg_default(&c);
    expect(c.max_episode_steps == 500u && c.compute_factor == 1u && c.env0 == 0u && c.model == RLSIM_MODEL_CARTPOLE,
           "defaults");

    /* NULL handles and outputs */
    expect(rlsim_destroy(NULL) == RLSIM_OK, "destroy(NULL)");
    expect(rlsim_reset(NULL, 1) == RLSIM_EINVAL, "reset(NULL)");
    expect(rlsim_step_fused(NULL, 1, NULL, NULL) == RLSIM_EINVAL, "step(NULL)");
    expect(rlsim_get_state(NULL, NULL, NULL, NULL) == RLSIM_EINVAL, "get_state(NULL)");
    expect(rlsim_set_state(NULL, NULL, NULL, 0) == RLSIM_EINVAL, "set_state(NULL)");
    expect(rlsim_create(16, 4, &c, NULL) == RLSIM_EINVAL, "create(out NULL)");
    expect(strlen(rlsim_last_error(NULL)) > 0, "message after create(out NULL)");

    /* sizes */
    expect_create_einval(0, 4, &c, "n = 0");
    expect_create_einval((1u << 30) + 1u, 4, &c, "n > 2^30");
    expect_create_einval(16, 3, &c, "state_words < 4");
    expect_create_einval(16, (1u << 24) + 5u, &c, "state_words > 2^24 + 4");
    expect_create_einval(16, 0xFFFFFFFFu, NULL, "state_words = 2^32 - 1, default cfg");

    /* global env offsets */
    rlsim_cfg e = c;
    e.env0 = 255u;
    expect_create_einval(16, 4, &e, "env0 not a multiple of 256");
    e.env0 = 0xFFFFFF00u;
    expect_create_einval(512, 4, &e, "env0 + n > 2^32");

    /* models and chain shapes */
    rlsim_cfg m = c;
    m.model = 7u;
    expect_create_einval(16, 4, &m, "unknown model");
    m.model = RLSIM_MODEL_CHAIN;
    m.n_links = 0u;
    expect_create_einval(16, 2, &m, "chain with 0 links");
    m.n_links = 5u;
    expect_create_einval(16, 12, &m, "chain with 5 links");
    m.n_links = 2u;
    expect_create_einval(16, 7, &m, "chain with padding words");

    /* seeded invalid configurations, one broken rule each */
    uint64_t st = 2024u;
    for (int i = 0; i < 500; ++i) {
        rlsim_cfg b = c;
        float* fields[] = {&b.gravity, &b.masscart, &b.masspole, &b.half_length, &b.force_mag, &b.tau,
                           &b.x_threshold, &b.theta_threshold_rad, &b.reset_low, &b.reset_high, &b.pad_a_low,
                           &b.pad_a_high, &b.pad_b_low, &b.pad_b_high};
        const uint64_t r = mix(&st);
        switch (r % 6u) {
        case 0: *fields[(r >> 8) % 14u] = ((r >> 16) & 1u) ? NAN : INFINITY; break;
        case 1: b.masscart = -(float)((r >> 8) % 100u) * 0.01f; break;
        case 2: b.reset_low = b.reset_high + 0.5f; break;
        case 3: b.flags = 2u + (uint32_t)(r >> 32) % 1000u; break;
        case 4: b.compute_factor = 0u; break;
        default: b.env0 = 1u + (uint32_t)(r >> 40) % 255u; break;
        }
        expect_create_einval(64, 4, &b, "seeded invalid cfg");
    }
    if (failures) {
        fprintf(stderr, "%d expectation(s) failed\n", failures);
        return 1;
    }
    printf("abi host checks: OK\n");
    return 0;
}
