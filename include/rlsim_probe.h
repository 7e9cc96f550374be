/*
 * rlsim_probe.h -- C ABI of the store-only probe of the trajectory layout
 * (librlsim_probe.so), a measurement aid beside librlsim.so.
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

#ifdef __cplusplus
}
#endif

#endif /* RLSIM_PROBE_H */
