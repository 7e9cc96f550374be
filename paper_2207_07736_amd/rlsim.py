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
RLSIM_MODEL_CARTPOLE = 0
RLSIM_MODEL_CHAIN = 1

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
        ("env0", ctypes.c_uint32),
        ("model", ctypes.c_uint32),
        ("n_links", ctypes.c_uint32),
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


class TrajRows:
    """The rows one rlsim_step_fused call records, with the shape they were cut
    for: ``struct`` (the C struct), ``K`` steps (None for a statistics-only
    record, which suits any K), ``n`` environments and ``S`` state words.
    Simulator.step checks the shape against the call before anything is
    enqueued, so a mismatch raises instead of letting a kernel write past a
    buffer.  An output plane can be switched off by setting it to None."""

    _FIELDS = tuple(f for f, _ in rlsim_traj._fields_)

    def __init__(self, struct: rlsim_traj, K, n: int, S):
        object.__setattr__(self, "struct", struct)
        object.__setattr__(self, "K", K)
        object.__setattr__(self, "n", n)
        object.__setattr__(self, "S", S)

    def __getattr__(self, name):
        if name in TrajRows._FIELDS:
            return getattr(self.struct, name)
        raise AttributeError(name)

    def __setattr__(self, name, value):
        if name not in TrajRows._FIELDS:
            raise AttributeError(name)
        if value is not None:
            raise ValueError("a recorded plane can only be switched off (set to None)")
        setattr(self.struct, name, None)


def stats_only(block_stats, n: int) -> TrajRows:
    """A record of the per-256-env block statistics alone (no trajectory rows)
    for n environments; block_stats is a device tensor of at least
    ceil(n / 256) x 4 32-bit words."""
    need = 4 * ((n + 255) // 256)
    if block_stats.numel() * block_stats.element_size() < 4 * need or not block_stats.is_contiguous():
        raise ValueError(f"block_stats must hold {need} contiguous 32-bit words")
    return TrajRows(traj_struct(block_stats=block_stats), None, n, None)


class Trajectory:
    """Device buffers of K trajectory rows for n environments with S state words
    each (4 for the cart-pole, 2 N + 2 for an N-link chain), as torch tensors.
    ``learner=True`` adds the per-step log pi(a|obs) and value planes."""

    def __init__(self, K: int, n: int, device="cuda", stats: bool = True, p0: bool = False, learner: bool = False,
                 S: int = 4):
        import torch
        self.K, self.n, self.S = K, n, S
        self.obs = torch.empty((K, S, n), dtype=torch.float32, device=device)
        self.action = torch.empty((K, n), dtype=torch.uint8, device=device)
        self.reward = torch.empty((K, n), dtype=torch.float32, device=device)
        self.done = torch.empty((K, n), dtype=torch.uint8, device=device)
        self.block_stats = torch.empty(((n + 255) // 256, 4), dtype=torch.int32, device=device) if stats else None
        self.policy_p0 = torch.empty((K, n), dtype=torch.float32, device=device) if p0 else None
        self.logp = torch.empty((K, n), dtype=torch.float32, device=device) if learner else None
        self.value = torch.empty((K, n), dtype=torch.float32, device=device) if learner else None

    def rows(self, k0: int, k: int) -> TrajRows:
        """Rows k0 .. k0+k-1, for a call with K = k."""
        if k < 1 or k0 < 0 or k0 + k > self.K:
            raise ValueError("row range outside the trajectory")
        part = lambda x: None if x is None else x[k0:k0 + k]  # noqa: E731
        st = traj_struct(self.obs[k0:k0 + k], self.action[k0:k0 + k], self.reward[k0:k0 + k],
                         self.done[k0:k0 + k], self.block_stats, part(self.policy_p0), part(self.logp),
                         part(self.value))
        return TrajRows(st, k, self.n, self.S)

    def learner_batch(self) -> dict:
        """The recorded rows as a learner reads them, as views of the buffers the
        kernel wrote (no copy): obs [K, n, S], action, reward, done, and when
        recorded logp and value [K, n]."""
        out = dict(obs=self.obs.permute(0, 2, 1), action=self.action, reward=self.reward, done=self.done)
        if self.logp is not None:
            out["logp"], out["value"] = self.logp, self.value
        return out


class Simulator:
    """Owning wrapper of one rlsim handle (convenience for tests and the bench).
    ``links`` > 0 selects the chain model with that many links (no padding
    words); ``env0`` is the handle's first global environment id."""

    def __init__(self, n_envs: int, D: int = 0, cfg_values: dict | None = None, stream=None, links: int = 0,
                 env0: int = 0):
        self.n, self.D, self.links = int(n_envs), int(D), int(links)
        self.cfg = make_cfg(cfg_values, stream)
        self.cfg.env0 = int(env0)
        if self.links:
            self.cfg.model, self.cfg.n_links = RLSIM_MODEL_CHAIN, self.links
            self.S = 2 * (self.links + 1)
        else:
            self.S = 4
        self.h = rlsim_create(self.n, self.S + self.D, self.cfg)

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

    def step(self, K: int, traj: TrajRows | None = None, policy: rlsim_policy | None = None):
        """One rlsim_step_fused call of K steps recording into traj (rows cut
        for exactly this K and this simulator, or a statistics-only record)."""
        if traj is not None:
            if not isinstance(traj, TrajRows):
                raise TypeError("traj must come from Trajectory.rows() or stats_only()")
            if traj.n != self.n or (traj.K is not None and (traj.K != K or traj.S != self.S)):
                raise ValueError(f"rows cut for K={traj.K}, n={traj.n}, S={traj.S}; the call has K={K}, "
                                 f"n={self.n}, S={self.S}")
        rlsim_step_fused(self.h, K, policy, None if traj is None else traj.struct)

    def get_state(self):
        return rlsim_get_state(self.h, self.n, self.S + self.D)

    def set_state(self, state, ep, t):
        rlsim_set_state(self.h, state, ep, t)
