/*
 * rlsim_probe.h -- C ABI of the measurement aids beside librlsim.so
 * (librlsim_probe.so): the store-only probe of the trajectory layout, a
 * read/write stream probe, and the error probe of the policy kernel's
 * elementwise functions.
 *
 * The fused simulator kernel's unavoidable work is writing the trajectory
 * (section "Simulator Kernel Fusion": fusion removes the state round trips,
 * not the trajectory the data-collection loop hands to the learner).  This
 * probe writes exactly the bytes, in exactly the layout and launch shape, of
 * K trajectory rows for n environments, with no simulation at all, so its
 * time is the ceiling the fused kernel's stores can reach on this device; the
 * fused kernel's time divided by the probe's is its distance from that ceiling.
 *
 * Conventions as in rlsim.h: 0 on success or a negative rlsim_status; work is
 * enqueued on `stream` (NULL = default stream) without synchronising; the
 * caller owns every buffer.
 */
#ifndef RLSIM_PROBE_H
#define RLSIM_PROBE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Write rows 0..K-1 of a trajectory for environments 0..n-1 into caller-owned
 * DEVICE buffers laid out as rlsim_traj (obs [K][4][n] f32, action [K][n] u8,
 * reward [K][n] f32, done [K][n] u8), one thread per environment, 256 per
 * workgroup, the same workgroup-to-environment mapping as the fused kernel.
 * Values (so that a test can check every byte):
 *   obs[k][c][e] = (e mod 65536) + k + c   (exact in fp32: K < 2^23)
 *   action[k][e] = (e + k) mod 2,  reward[k][e] = 1,  done[k][e] = (e xor k) mod 4
 * Errors: -1 (RLSIM_EINVAL) if n == 0, n > 2^30, K == 0 or K >= 2^23, a
 * pointer is NULL or a float pointer is not 4-byte aligned; -3
 * (RLSIM_EDEVICE) if the launch fails. */
int rlsim_probe_store(uint32_t n, uint32_t K, float* obs, uint8_t* action, float* reward, uint8_t* done,
                      void* stream);

/* Error of the MLP-policy kernel's elementwise functions, measured at every
 * fp32 value x whose bit pattern lies in [lo_bits, lo_bits + count) (NaN and
 * infinities skipped), against double-precision evaluations of what they
 * compute (the policy of rlsim.h: tanh hidden units, softmax over two logits,
 * log pi of the action taken):
 *   out_max[0] = max |tanh_kernel(x) - tanh(x)|
 *   out_max[1] = max |p0_kernel(x) - 1 / (1 + e^x)|          (x = l1 - l0)
 *   out_max[2] = max over a in {0, 1} of |log_pi_kernel(x, a) - r| / (1 + |r|),
 *                r = -softplus(a ? -x : x)
 * each as the bit pattern of a non-negative float rounded up, merged with
 * atomic max into the caller-owned DEVICE array out_max[3] (zero it first;
 * several calls over parts of a range merge).  The functions are those the
 * policy kernel itself calls, so the maxima over all 2^32 patterns bound the
 * kernel's elementwise error; the oracle's tolerance for the policy outputs is
 * built on them.
 * Errors: -1 if count == 0, lo_bits + count > 2^32, or out_max is NULL or not
 * 4-byte aligned; -3 if the launch fails. */
int rlsim_probe_policy_math(uint32_t lo_bits, uint64_t count, uint32_t* out_max, void* stream);

/* A plain stream with the traffic of one unfused step of the wide padding
 * state (section "Simulator Complexity": each word read and written once per
 * launch): for i < n4, s[i] <- fma(a[i], s[i], b[i]) on float4 units, each
 * component rounded once.  s, a and b are caller-owned DEVICE arrays of n4
 * float4 (16-byte aligned); 48 bytes are read and 16 written per float4.  Its
 * time is the ceiling that the K = 1 wide launches are compared with.
 * Errors: -1 if n4 == 0 or a pointer is NULL or not 16-byte aligned; -3 if the
 * launch fails. */
int rlsim_probe_stream(uint64_t n4, float* s, const float* a, const float* b, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* RLSIM_PROBE_H */
