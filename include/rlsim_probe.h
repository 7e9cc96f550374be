/*
 * rlsim_probe.h -- C ABI of the measurement aids beside librlsim.so
 * (librlsim_probe.so): the store-only probe of the trajectory layout, a
 * read/write stream probe, the error probe of the policy kernel's
 * elementwise functions, an instruction-rate probe and a fill probe of store
 * kernel shapes.
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

/* Instruction-rate probe: the throughputs that bound the kernels (section
 * "Simulator Complexity": the compute factor and state size make the step
 * compute-bound; "Future Work": simulation fused with MFMA inference).  One
 * launch of `blocks` workgroups of 256 threads (four waves; 256 blocks put
 * one wave on each SIMD of a 256-CU device, 256 w blocks w waves), each lane
 * running `iters` iterations of eight independent chains (MFMA: four) of one
 * instruction kind:
 *   kind 0  v_fma_f32 x <- x * 1 + 1, the two 1s in two registers,
 *           x0 = lane + j                                  -> x0 + iters
 *   kind 1  the per-lane padding update t <- u ? 1 : -0, s <- fma(1, s, t),
 *           u = (lane + i) odd, s0 = j                     -> s0 + #odd steps
 *   kind 2  v_exp_f32 x <- 2^-x                            -> the root of x = 2^-x
 *   kind 3  v_rcp_f32 x <- 1 / x, x0 = 2^j                 -> x0 (even iters)
 *   kind 4  v_mfma_f32_32x32x2_f32 C <- A B + C, A = B = 1 -> 2 iters per element
 *   kind 5  kind 4 with `iters` and kind 0 with 16 iters in alternate waves
 *           (workgroup b, wave w: MFMA when b + w is even), so that both
 *           share each SIMD
 *   kind 6  v_mul_f32 x <- x * 1, x0 = lane + j            -> x0
 *   kind 7  kind 0 with both 1s read from one register     -> x0 + iters
 *   kind 8  the wide kernel's padding replay of two environments, 8 words per
 *           lane each (per step a tree of scalar bit tests, then 16 in-place
 *           v_fma_f32 / v_mul_f32), over `iters` 32-step bit words; a = b = 1,
 *           so each word ends as the count of action-1 steps since its
 *           environment's last done bit.  The bits of word w of global wave g
 *           (g = 4 blockIdx + wave) come from hash(4k), hash(4k + 1) and
 *           hash(4k + 2), k = g iters + w (hash: x ^= x >> 16, x *= 0x7feb352d,
 *           x ^= x >> 15, x *= 0x846ca68b, x ^= x >> 16 on uint32): action words
 *           u0 = hash(4k), u1 = hash(4k + 1); with h = hash(4k + 2), done words
 *           d0 = 1 << (h & 31) | (((h >> 5) mod 3 == 0) << ((h >> 8) & 31)),
 *           d1 = 1 << ((h >> 13) & 31) | (((h >> 18) mod 3 == 0) << ((h >> 21) & 31))
 *   kind 9  the same 16 updates per step with no decisions: every 8 steps,
 *           environment 0 takes the FMA at steps 0, 3, 4, 5 and environment 1
 *           at the others                                  -> 16 iters per word
 * out (caller-owned DEVICE, blocks * 256 floats) receives per thread the sum
 * of its chains' final values (kinds 0-3, 6, 7: over j = 0..7; MFMA: elements
 * 0, 5, 10, 15 of the four accumulators, 8 iters; kinds 8, 9: over both
 * environments' 8 words).  clocks (caller-owned DEVICE, 2 blocks uint64, or
 * NULL) receives per workgroup the shader-clock cycles (s_memtime) and the
 * real-time ticks (s_memrealtime, at rlsim_probe_wall_clock_khz) that its
 * thread 0 took over its chains.  The caller times the launch.
 * Errors: -1 if kind > 9, blocks == 0 or > 2^20, iters == 0 or > 2^22 (kind
 * 5: > 2^19; kinds 8, 9: > 2^16), or out is NULL or not 4-byte aligned, or
 * clocks is not 8-byte aligned; -3 if the launch fails. */
int rlsim_probe_issue(uint32_t kind, uint32_t blocks, uint32_t iters, float* out, uint64_t* clocks, void* stream);

/* Frequency of the real-time counter that rlsim_probe_issue's clocks count in,
 * in kHz, for the current device, into *khz.  Errors: -1 if khz is NULL; -3 if
 * the device query fails. */
int rlsim_probe_wall_clock_khz(uint32_t* khz);

/* Store-rate probe of kernel shape (section "Simulator Kernel Fusion": what a
 * fused kernel's trajectory stores can reach depends on how they are issued):
 * a plain fill of n4 float4 at dst (caller-owned DEVICE, 16-byte aligned) by
 * workgroups of 256 threads, each thread storing per_thread float4 -- thread t
 * of workgroup b the indices b 256 per_thread + t + 256 j, j < per_thread --
 * so per_thread = 1 is one store per thread over a grid of many small
 * workgroups and large per_thread a long store loop per thread over a
 * workgroup-contiguous chunk (per_thread = 275 is the 1,126,400 bytes a
 * trajectory workgroup of 256 environments writes in 200 steps).
 * dst[i] = (v, v + 1, v + 2, v + 3) with v = i mod 2^20 (exact in fp32).
 * Errors: -1 if n4 == 0, per_thread == 0 or > 2^20, the grid would reach 2^31
 * workgroups, or dst is NULL or not 16-byte aligned; -3 if the launch fails. */
int rlsim_probe_fill(uint64_t n4, uint32_t per_thread, float* dst, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* RLSIM_PROBE_H */
