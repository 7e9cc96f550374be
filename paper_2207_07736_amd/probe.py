"""Thin ctypes binding of librlsim_probe.so (include/rlsim_probe.h): the
store-only probe of the trajectory layout, a read/write stream probe, the
error probe of the policy kernel's elementwise functions, the
instruction-rate probe and the fill probe of store kernel shapes, measurement
aids.  Argument
marshalling only; fails loudly if the library has not been built."""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
PROBE_LIB_PATH = os.path.join(_HERE, "librlsim_probe.so")
PROBE_EXPORTS = ("rlsim_probe_store", "rlsim_probe_policy_math", "rlsim_probe_stream", "rlsim_probe_issue",
                 "rlsim_probe_wall_clock_khz", "rlsim_probe_fill")
ISSUE_KINDS = ("fma", "select_fma", "exp", "rcp", "mfma", "mixed", "mul", "fma_shared", "replay_tree", "replay_flat")


def _load():
    if not os.path.exists(PROBE_LIB_PATH):
        raise ImportError(f"{PROBE_LIB_PATH} is missing: build it with paper_2207_07736_amd/build.py")
    L = ctypes.CDLL(PROBE_LIB_PATH)
    u32, vp = ctypes.c_uint32, ctypes.c_void_p
    L.rlsim_probe_store.argtypes = [u32, u32, vp, vp, vp, vp, vp]
    L.rlsim_probe_store.restype = ctypes.c_int
    L.rlsim_probe_policy_math.argtypes = [u32, ctypes.c_uint64, vp, vp]
    L.rlsim_probe_policy_math.restype = ctypes.c_int
    L.rlsim_probe_stream.argtypes = [ctypes.c_uint64, vp, vp, vp, vp]
    L.rlsim_probe_stream.restype = ctypes.c_int
    L.rlsim_probe_issue.argtypes = [u32, u32, u32, vp, vp, vp]
    L.rlsim_probe_issue.restype = ctypes.c_int
    L.rlsim_probe_wall_clock_khz.argtypes = [ctypes.POINTER(u32)]
    L.rlsim_probe_wall_clock_khz.restype = ctypes.c_int
    L.rlsim_probe_fill.argtypes = [ctypes.c_uint64, u32, vp, vp]
    L.rlsim_probe_fill.restype = ctypes.c_int
    return L


probe_lib = _load()


def _ptr(t):
    return None if t is None else t.data_ptr()


def probe_store(n: int, K: int, obs, action, reward, done, stream=None) -> None:
    """Write K trajectory rows for n envs (torch tensors laid out as rlsim_traj)
    with no simulation; raises ValueError on a rejected argument."""
    s = None if stream is None else (stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))
    rc = probe_lib.rlsim_probe_store(int(n), int(K), _ptr(obs), _ptr(action), _ptr(reward), _ptr(done), s)
    if rc != 0:
        raise ValueError(f"rlsim_probe_store rejected its arguments (status {rc})")


def probe_policy_math(lo_bits: int, count: int, out_max, stream=None) -> None:
    """Merge the policy functions' maximum errors over fp32 bit patterns
    [lo_bits, lo_bits + count) into out_max (a zeroed int32 device tensor of 3;
    read it with .view(torch.float32)); raises ValueError on a rejected argument."""
    s = None if stream is None else (stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))
    rc = probe_lib.rlsim_probe_policy_math(int(lo_bits), int(count), _ptr(out_max), s)
    if rc != 0:
        raise ValueError(f"rlsim_probe_policy_math rejected its arguments (status {rc})")


def probe_stream(s, a, b, stream=None) -> None:
    """s <- fma(a, s, b) elementwise over float32 device tensors of equal size
    (a multiple of 4, 16-byte aligned); raises ValueError on a rejected argument."""
    if not (s.numel() == a.numel() == b.numel()) or s.numel() % 4:
        raise ValueError("probe_stream needs three arrays of the same size, a multiple of 4")
    st = None if stream is None else (stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))
    rc = probe_lib.rlsim_probe_stream(s.numel() // 4, _ptr(s), _ptr(a), _ptr(b), st)
    if rc != 0:
        raise ValueError(f"rlsim_probe_stream rejected its arguments (status {rc})")


def probe_issue(kind: str, blocks: int, iters: int, out, stream=None, clocks=None) -> None:
    """Run the instruction-rate probe `kind` (one of ISSUE_KINDS) over `blocks`
    workgroups of 256 threads, `iters` iterations each, results into out (a
    float32 device tensor of blocks * 256) and, if given, each workgroup's
    shader cycles and real-time ticks into clocks (an int64 device tensor of
    blocks * 2); raises ValueError on a rejected argument."""
    if out.numel() < blocks * 256:
        raise ValueError("out must hold blocks * 256 floats")
    if clocks is not None and clocks.numel() < 2 * blocks:
        raise ValueError("clocks must hold 2 * blocks values")
    st = None if stream is None else (stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))
    rc = probe_lib.rlsim_probe_issue(ISSUE_KINDS.index(kind), int(blocks), int(iters), _ptr(out),
                                     None if clocks is None else _ptr(clocks), st)
    if rc != 0:
        raise ValueError(f"rlsim_probe_issue rejected its arguments (status {rc})")


def wall_clock_khz() -> int:
    """Frequency of the counter behind probe_issue's real-time ticks, in kHz."""
    khz = ctypes.c_uint32(0)
    rc = probe_lib.rlsim_probe_wall_clock_khz(ctypes.byref(khz))
    if rc != 0:
        raise RuntimeError(f"rlsim_probe_wall_clock_khz failed (status {rc})")
    return int(khz.value)


def probe_fill(dst, per_thread: int, stream=None) -> None:
    """Fill the float32 device tensor dst (a multiple of 4 elements, 16-byte
    aligned) with per_thread float4 stores per thread; raises ValueError on a
    rejected argument."""
    if dst.numel() % 4:
        raise ValueError("probe_fill needs a multiple of 4 floats")
    st = None if stream is None else (stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))
    rc = probe_lib.rlsim_probe_fill(dst.numel() // 4, int(per_thread), _ptr(dst), st)
    if rc != 0:
        raise ValueError(f"rlsim_probe_fill rejected its arguments (status {rc})")
