"""Thin Python binding of librlsim.so (include/rlsim.h): argument marshalling only.

Every step of the data-collection path runs in the library's HIP kernels; this
module converts Python values and torch tensors into the C structs and raises
``RlsimError`` on a negative status.  torch is used for device memory and the
current stream only.  There is no fallback: if the shared library is missing
the import fails.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "librlsim.so")

RLSIM_OK = 0
RLSIM_EINVAL = -1
RLSIM_ENOMEM = -2
RLSIM_EDEVICE = -3
RLSIM_ESTATE = -4
RLSIM_EUNSUPPORTED = -5
RLSIM_F32 = 0
RLSIM_BF16 = 1
RLSIM_F_NO_TERMINATION = 1

# every entry point include/rlsim.h declares
EXPORTS = ("rlsim_cfg_default", "rlsim_create", "rlsim_reset", "rlsim_step_fused", "rlsim_get_state",
           "rlsim_set_state", "rlsim_destroy", "rlsim_last_error")


class RlsimError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{msg} (status {code})")
        self.code = code


class rlsim_cfg(ctypes.Structure):
    _fields_ = [
        ("gravity", ctypes.c_float), ("masscart", ctypes.c_float), ("masspole", ctypes.c_float),
        ("half_length", ctypes.c_float), ("force_mag", ctypes.c_float), ("tau", ctypes.c_float),
        ("x_threshold", ctypes.c_float), ("theta_threshold_rad", ctypes.c_float),
        ("max_episode_steps", ctypes.c_uint32),
        ("reset_low", ctypes.c_float), ("reset_high", ctypes.c_float),
        ("pad_a_low", ctypes.c_float), ("pad_a_high", ctypes.c_float),
        ("pad_b_low", ctypes.c_float), ("pad_b_high", ctypes.c_float),
        ("flags", ctypes.c_uint32),
        ("compute_factor", ctypes.c_uint32),
        ("stream", ctypes.c_void_p),
    ]


class rlsim_traj(ctypes.Structure):
    _fields_ = [("obs", ctypes.c_void_p), ("action", ctypes.c_void_p), ("reward", ctypes.c_void_p),
                ("done", ctypes.c_void_p), ("block_stats", ctypes.c_void_p), ("policy_p0", ctypes.c_void_p),
                ("logp", ctypes.c_void_p), ("value", ctypes.c_void_p)]


class rlsim_policy(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int),
                ("w1", ctypes.c_void_p), ("b1", ctypes.c_void_p),
                ("w2", ctypes.c_void_p), ("b2", ctypes.c_void_p),
                ("w3", ctypes.c_void_p), ("b3", ctypes.c_void_p),
                ("wv", ctypes.c_void_p), ("bv", ctypes.c_void_p)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with paper_2207_07736_amd/build.py "
                          "(there is no CPU fallback)")
    L = ctypes.CDLL(LIB_PATH)
    vp, u32, u64 = ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint64
    L.rlsim_cfg_default.argtypes = [ctypes.POINTER(rlsim_cfg)]
    L.rlsim_cfg_default.restype = None
    L.rlsim_create.argtypes = [u32, u32, ctypes.POINTER(rlsim_cfg), ctypes.POINTER(vp)]
    L.rlsim_create.restype = ctypes.c_int
    L.rlsim_reset.argtypes = [vp, u64]
    L.rlsim_reset.restype = ctypes.c_int
    L.rlsim_step_fused.argtypes = [vp, u32, ctypes.POINTER(rlsim_policy), ctypes.POINTER(rlsim_traj)]
    L.rlsim_step_fused.restype = ctypes.c_int
    L.rlsim_get_state.argtypes = [vp, vp, vp, ctypes.POINTER(u64)]
    L.rlsim_get_state.restype = ctypes.c_int
    L.rlsim_set_state.argtypes = [vp, vp, vp, u64]
    L.rlsim_set_state.restype = ctypes.c_int
    L.rlsim_destroy.argtypes = [vp]
    L.rlsim_destroy.restype = ctypes.c_int
    L.rlsim_last_error.argtypes = [vp]
    L.rlsim_last_error.restype = ctypes.c_char_p
    return L


lib = _load()


def _check(rc: int, h) -> None:
    if rc != RLSIM_OK:
        msg = lib.rlsim_last_error(h)
        raise RlsimError(rc, msg.decode() if msg else "rlsim error")


def rlsim_last_error(h=None) -> str:
    m = lib.rlsim_last_error(h)
    return m.decode() if m else ""


def rlsim_cfg_default() -> rlsim_cfg:
    c = rlsim_cfg()
    lib.rlsim_cfg_default(ctypes.byref(c))
    return c


def make_cfg(values: dict | None = None, stream=None) -> rlsim_cfg:
    """rlsim_cfg from a dict of constants (the simulator's field names; the
    ``no_termination`` key maps to RLSIM_F_NO_TERMINATION) and a stream
    (torch.cuda.Stream, a raw hipStream_t int, or None for the default)."""
    c = rlsim_cfg_default()
    for k, v in (values or {}).items():
        if k == "no_termination":
            c.flags = (c.flags | RLSIM_F_NO_TERMINATION) if v else (c.flags & ~RLSIM_F_NO_TERMINATION)
        else:
            if not hasattr(c, k) or k in ("stream", "flags"):
                raise KeyError(k)
            setattr(c, k, v)
    if stream is not None:
        c.stream = stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
    return c


def rlsim_create(n_envs: int, state_words: int, cfg: rlsim_cfg | None = None) -> ctypes.c_void_p:
    h = ctypes.c_void_p()
    rc = lib.rlsim_create(int(n_envs), int(state_words), ctypes.byref(cfg) if cfg is not None else None,
                          ctypes.byref(h))
    _check(rc, None)
    return h


def rlsim_reset(h, seed: int) -> None:
    _check(lib.rlsim_reset(h, int(seed)), h)


def rlsim_step_fused(h, K: int, policy: rlsim_policy | None = None, traj: rlsim_traj | None = None) -> None:
    _check(lib.rlsim_step_fused(h, int(K), ctypes.byref(policy) if policy is not None else None,
                                ctypes.byref(traj) if traj is not None else None), h)


def rlsim_get_state(h, n_envs: int, state_words: int):
    """Returns (state [state_words][n_envs] f32, ep [n_envs] u32, t) as numpy arrays."""
    import numpy as np
    st = np.empty((state_words, n_envs), dtype=np.float32)
    ep = np.empty(n_envs, dtype=np.uint32)
    t = ctypes.c_uint64()
    _check(lib.rlsim_get_state(h, st.ctypes.data, ep.ctypes.data, ctypes.byref(t)), h)
    return st, ep, int(t.value)


def rlsim_set_state(h, state, ep, t: int) -> None:
    import numpy as np
    st = None if state is None else np.ascontiguousarray(state, dtype=np.float32)
    e = None if ep is None else np.ascontiguousarray(ep, dtype=np.uint32)
    _check(lib.rlsim_set_state(h, None if st is None else st.ctypes.data, None if e is None else e.ctypes.data,
                               int(t)), h)


def rlsim_destroy(h) -> None:
    if h:
        _check(lib.rlsim_destroy(h), None)


def _ptr(t):
    return None if t is None else t.data_ptr()


def traj_struct(obs=None, action=None, reward=None, done=None, block_stats=None, policy_p0=None,
                logp=None, value=None) -> rlsim_traj:
    """rlsim_traj from torch tensors (or None)."""
    return rlsim_traj(_ptr(obs), _ptr(action), _ptr(reward), _ptr(done), _ptr(block_stats), _ptr(policy_p0),
                      _ptr(logp), _ptr(value))


def policy_struct(dtype: int, w1, b1, w2, b2, w3, b3, wv=None, bv=None) -> rlsim_policy:
    """rlsim_policy from device tensors (weights fp32 or bf16, biases fp32 or
    None; wv/bv the optional value head)."""
    return rlsim_policy(int(dtype), _ptr(w1), _ptr(b1), _ptr(w2), _ptr(b2), _ptr(w3), _ptr(b3), _ptr(wv), _ptr(bv))


class Trajectory:
    """Device buffers of K trajectory rows for n environments (torch tensors).
    ``learner=True`` adds the per-step log pi(a|obs) and value planes."""

    def __init__(self, K: int, n: int, device="cuda", stats: bool = True, p0: bool = False, learner: bool = False):
        import torch
        self.K, self.n = K, n
        self.obs = torch.empty((K, 4, n), dtype=torch.float32, device=device)
        self.action = torch.empty((K, n), dtype=torch.uint8, device=device)
        self.reward = torch.empty((K, n), dtype=torch.float32, device=device)
        self.done = torch.empty((K, n), dtype=torch.uint8, device=device)
        self.block_stats = torch.empty(((n + 255) // 256, 4), dtype=torch.int32, device=device) if stats else None
        self.policy_p0 = torch.empty((K, n), dtype=torch.float32, device=device) if p0 else None
        self.logp = torch.empty((K, n), dtype=torch.float32, device=device) if learner else None
        self.value = torch.empty((K, n), dtype=torch.float32, device=device) if learner else None

    def rows(self, k0: int, k: int) -> rlsim_traj:
        """Struct addressing rows k0 .. k0+k-1 (for a call with K = k)."""
        if k0 < 0 or k0 + k > self.K:
            raise ValueError("row range outside the trajectory")
        part = lambda x: None if x is None else x[k0:k0 + k]  # noqa: E731
        return traj_struct(self.obs[k0:k0 + k], self.action[k0:k0 + k], self.reward[k0:k0 + k],
                           self.done[k0:k0 + k], self.block_stats, part(self.policy_p0), part(self.logp),
                           part(self.value))

    def learner_batch(self) -> dict:
        """The recorded rows as a learner reads them, as views of the buffers the
        kernel wrote (no copy): obs [K, n, 4], action, reward, done, and when
        recorded logp and value [K, n]."""
        out = dict(obs=self.obs.permute(0, 2, 1), action=self.action, reward=self.reward, done=self.done)
        if self.logp is not None:
            out["logp"], out["value"] = self.logp, self.value
        return out


class Simulator:
    """Owning wrapper of one rlsim handle (convenience for tests and the bench)."""

    def __init__(self, n_envs: int, D: int = 0, cfg_values: dict | None = None, stream=None):
        self.n, self.D = int(n_envs), int(D)
        self.cfg = make_cfg(cfg_values, stream)
        self.h = rlsim_create(self.n, 4 + self.D, self.cfg)

    def close(self):
        if self.h:
            h, self.h = self.h, None
            rlsim_destroy(h)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def reset(self, seed: int):
        rlsim_reset(self.h, seed)

    def step(self, K: int, traj: rlsim_traj | None = None, policy: rlsim_policy | None = None):
        rlsim_step_fused(self.h, K, policy, traj)

    def get_state(self):
        return rlsim_get_state(self.h, self.n, 4 + self.D)

    def set_state(self, state, ep, t):
        rlsim_set_state(self.h, state, ep, t)
