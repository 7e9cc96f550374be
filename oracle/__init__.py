"""CPU oracle of the data-collection step -- TEST INFRASTRUCTURE ONLY.

Plain, slow, single-threaded C (``rlsim_oracle.c``) behind a ctypes wrapper.
Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The GPU library never loads it, and it
shares no code with the GPU library: its configuration struct, constants and
RNG are declared here and in ``rlsim_oracle.c`` independently.

What it computes (one cart-pole environment per array column, Background,
"Cartpole Simulator"; the simulation/inference loop of Background, "RL
Training"; K steps per call as in "Simulator Kernel Fusion"):

* ``philox4x32_10`` -- the counter-based generator of Salmon et al. (SC'11).
* ``cartpole_step`` -- one explicit-Euler step of the frictionless cart and
  uniform rod, fp32, each operation rounded once; ``env_step`` -- a simulation
  step made of C such iterations of length tau / C (the compute factor).
* ``Sim`` -- N environments with auto-reset, the random-action or MLP-policy
  loop, padding words (the paper's state-size factor S, Simulator Complexity)
  and per-256-env block statistics.
* ``sincos`` -- the series sin/cos with a quadrant reduction for angles past
  pi/4 (a swinging link, a pole with termination disabled).
* ``chain_step`` / ``ChainSim`` -- the second, heavier simulator the paper's
  Future Work calls for: a cart carrying a chain of N uniform rods, its
  Lagrangian in mass-matrix form solved by elimination every step, with the
  same random-action loop, auto-reset and statistics.

Parity pins live in ``tests/test_oracle_*.py``.  Functions without an
independent pin: none.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "rlsim_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_CFLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared", "-Wall"]


def build() -> str:
    """Compile the oracle with gcc (no contraction, no fast-math)."""
    tmp = _LIB_PATH + ".tmp"
    subprocess.run(["gcc", *_CFLAGS, "-o", tmp, _SRC, "-lm"], check=True)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


class Params(ctypes.Structure):
    """Simulator configuration; field meaning as documented in rlsim_oracle.c."""

    _fields_ = [
        ("gravity", ctypes.c_float), ("masscart", ctypes.c_float), ("masspole", ctypes.c_float),
        ("half_length", ctypes.c_float), ("force_mag", ctypes.c_float), ("tau", ctypes.c_float),
        ("x_threshold", ctypes.c_float), ("theta_threshold_rad", ctypes.c_float),
        ("max_episode_steps", ctypes.c_uint32),
        ("reset_low", ctypes.c_float), ("reset_high", ctypes.c_float),
        ("pad_a_low", ctypes.c_float), ("pad_a_high", ctypes.c_float),
        ("pad_b_low", ctypes.c_float), ("pad_b_high", ctypes.c_float),
        ("no_termination", ctypes.c_uint32),
        ("compute_factor", ctypes.c_uint32),
    ]


class Errs(ctypes.Structure):
    """Error model of a device policy evaluation (orc_mlp_bounds): per-operation
    accumulation bound, and absolute errors of tanh, p0 and (relative to
    1 + |log pi|) log pi."""
    _fields_ = [("acc", ctypes.c_double), ("tanh", ctypes.c_double), ("p0", ctypes.c_double),
                ("logpi", ctypes.c_double)]


class Bounds(ctypes.Structure):
    _fields_ = [(name, ctypes.c_double) for name in ("p0_lo", "p0_hi", "lp0_lo", "lp0_hi", "lp1_lo", "lp1_hi",
                                                     "v_lo", "v_hi")]


class _Policy(ctypes.Structure):
    _fields_ = [("bf16", ctypes.c_int)] + [
        (name, ctypes.POINTER(ctypes.c_float)) for name in ("w1", "b1", "w2", "b2", "w3", "b3", "wv", "bv")
    ]


CHAIN_MAX_LINKS = 8


class ChainConsts(ctypes.Structure):
    """Derived constants of the chain simulator (orc_chain_make_consts)."""
    _fields_ = [("N", ctypes.c_uint32), ("m00", ctypes.c_float)] + [
        (name, ctypes.c_float * (CHAIN_MAX_LINKS + 1)) for name in ("h", "g_diag", "lh", "gh")]


_lib = None


def lib():
    """Load (building first if needed) the oracle shared library."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        build()
    L = ctypes.CDLL(_LIB_PATH)
    u32p = ctypes.POINTER(ctypes.c_uint32)
    f32p = ctypes.POINTER(ctypes.c_float)
    L.orc_philox4x32_10.argtypes = [u32p, u32p, u32p]
    L.orc_philox4x32_10.restype = None
    L.orc_u24.argtypes = [ctypes.c_uint32]
    L.orc_u24.restype = ctypes.c_float
    L.orc_uniform.argtypes = [ctypes.c_uint32, ctypes.c_float, ctypes.c_float]
    L.orc_uniform.restype = ctypes.c_float
    L.orc_sin.argtypes = [ctypes.c_float]
    L.orc_sin.restype = ctypes.c_float
    L.orc_cos.argtypes = [ctypes.c_float]
    L.orc_cos.restype = ctypes.c_float
    L.orc_sin_series.argtypes = [ctypes.c_float]
    L.orc_sin_series.restype = ctypes.c_float
    L.orc_cos_series.argtypes = [ctypes.c_float]
    L.orc_cos_series.restype = ctypes.c_float
    L.orc_sincos.argtypes = [ctypes.c_float, f32p, f32p]
    L.orc_sincos.restype = None
    L.orc_cartpole_step.argtypes = [ctypes.POINTER(Params), f32p, ctypes.c_int, f32p]
    L.orc_cartpole_step.restype = None
    L.orc_env_step.argtypes = [ctypes.POINTER(Params), f32p, ctypes.c_int, f32p]
    L.orc_env_step.restype = None
    L.orc_terminated.argtypes = [ctypes.POINTER(Params), f32p]
    L.orc_terminated.restype = ctypes.c_int
    L.orc_reset_draw.argtypes = [ctypes.POINTER(Params), ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint32, f32p]
    L.orc_reset_draw.restype = None
    L.orc_action_bit.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint32]
    L.orc_action_bit.restype = ctypes.c_int
    L.orc_policy_u.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint32]
    L.orc_policy_u.restype = ctypes.c_float
    L.orc_pad_params.argtypes = [ctypes.POINTER(Params), ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint32, f32p, f32p]
    L.orc_pad_params.restype = None
    L.orc_pad_update.argtypes = [ctypes.c_float, ctypes.c_float, ctypes.c_float, ctypes.c_int]
    L.orc_pad_update.restype = ctypes.c_float
    L.orc_round_bf16.argtypes = [ctypes.c_double]
    L.orc_round_bf16.restype = ctypes.c_double
    L.orc_mlp_p0.argtypes = [ctypes.POINTER(_Policy), f32p]
    L.orc_mlp_p0.restype = ctypes.c_double
    f64p = ctypes.POINTER(ctypes.c_double)
    L.orc_mlp_eval.argtypes = [ctypes.POINTER(_Policy), f32p, f64p, f64p, f64p]
    L.orc_mlp_eval.restype = None
    L.orc_log_prob.argtypes = [f64p, ctypes.c_int]
    L.orc_log_prob.restype = ctypes.c_double
    L.orc_create.argtypes = [ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint32, ctypes.POINTER(Params)]
    L.orc_create.restype = ctypes.c_void_p
    L.orc_destroy.argtypes = [ctypes.c_void_p]
    L.orc_destroy.restype = None
    L.orc_reset.argtypes = [ctypes.c_void_p, ctypes.c_uint64]
    L.orc_reset.restype = None
    L.orc_step.argtypes = [ctypes.c_void_p, ctypes.c_uint32, ctypes.POINTER(_Policy),
                           ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                           ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    L.orc_step.restype = ctypes.c_int
    L.orc_get_state.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.POINTER(ctypes.c_uint64)]
    L.orc_get_state.restype = None
    L.orc_set_state.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint64]
    L.orc_set_state.restype = ctypes.c_int
    L.orc_get_pad_params.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    L.orc_check_rows.argtypes = [ctypes.POINTER(Params), ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint32,
                                 ctypes.c_uint32, ctypes.c_uint32, ctypes.c_void_p, ctypes.c_void_p,
                                 ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                 ctypes.c_void_p, ctypes.POINTER(ctypes.c_uint32), ctypes.POINTER(ctypes.c_uint32)]
    L.orc_check_rows.restype = ctypes.c_uint64
    L.orc_mlp_bounds.argtypes = [ctypes.POINTER(_Policy), ctypes.POINTER(ctypes.c_float), ctypes.POINTER(Errs),
                                 ctypes.POINTER(Bounds)]
    L.orc_mlp_bounds.restype = None
    L.orc_check_policy_rows.argtypes = [ctypes.POINTER(Params), ctypes.POINTER(_Policy), ctypes.c_uint64,
                                        ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint32,
                                        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.POINTER(Errs), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.POINTER(ctypes.c_double),
                                        ctypes.POINTER(ctypes.c_uint64), ctypes.POINTER(ctypes.c_uint32),
                                        ctypes.POINTER(ctypes.c_uint32)]
    L.orc_check_policy_rows.restype = ctypes.c_uint64
    L.orc_get_pad_params.restype = None
    # the chain simulator
    L.orc_chain_make_consts.argtypes = [ctypes.POINTER(Params), ctypes.c_uint32, ctypes.POINTER(ChainConsts)]
    L.orc_chain_make_consts.restype = ctypes.c_int
    L.orc_chain_accel.argtypes = [ctypes.POINTER(ChainConsts), f32p, ctypes.c_float, f32p]
    L.orc_chain_accel.restype = None
    L.orc_chain_env_step.argtypes = [ctypes.POINTER(Params), ctypes.POINTER(ChainConsts), f32p, ctypes.c_int, f32p]
    L.orc_chain_env_step.restype = None
    L.orc_chain_terminated.argtypes = [ctypes.POINTER(Params), ctypes.c_uint32, f32p]
    L.orc_chain_terminated.restype = ctypes.c_int
    L.orc_chain_reset_draw.argtypes = [ctypes.POINTER(Params), ctypes.c_uint32, ctypes.c_uint64, ctypes.c_uint32,
                                       ctypes.c_uint32, f32p]
    L.orc_chain_reset_draw.restype = None
    L.orc_chain_create.argtypes = [ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint32, ctypes.POINTER(Params)]
    L.orc_chain_create.restype = ctypes.c_void_p
    L.orc_chain_destroy.argtypes = [ctypes.c_void_p]
    L.orc_chain_destroy.restype = None
    L.orc_chain_reset.argtypes = [ctypes.c_void_p, ctypes.c_uint64]
    L.orc_chain_reset.restype = None
    L.orc_chain_step.argtypes = [ctypes.c_void_p, ctypes.c_uint32] + [ctypes.c_void_p] * 5
    L.orc_chain_step.restype = ctypes.c_int
    L.orc_chain_get_state.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.POINTER(ctypes.c_uint64)]
    L.orc_chain_get_state.restype = None
    L.orc_chain_set_state.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint64]
    L.orc_chain_set_state.restype = ctypes.c_int
    L.orc_chain_check_rows.argtypes = [ctypes.POINTER(Params), ctypes.c_uint32, ctypes.c_uint64, ctypes.c_uint32,
                                       ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint32] + [ctypes.c_void_p] * 7 + [
                                       ctypes.POINTER(ctypes.c_uint32), ctypes.POINTER(ctypes.c_uint32)]
    L.orc_chain_check_rows.restype = ctypes.c_uint64
    _lib = L
    return L


def make_params(**overrides) -> Params:
    """Params from keyword values (every field must be given)."""
    p = Params()
    names = [f[0] for f in Params._fields_]
    missing = [n for n in names if n not in overrides]
    if missing:
        raise ValueError(f"missing oracle parameters: {missing}")
    for k, v in overrides.items():
        if k not in names:
            raise ValueError(f"unknown oracle parameter {k}")
        setattr(p, k, v)
    return p


def _u32(a):
    return np.ascontiguousarray(a, dtype=np.uint32)


def philox4x32_10(counter, key) -> np.ndarray:
    """Philox4x32-10 of one (counter[4], key[2]) pair -> 4 uint32 words."""
    c = _u32(counter)
    k = _u32(key)
    out = np.zeros(4, dtype=np.uint32)
    P = ctypes.POINTER(ctypes.c_uint32)
    lib().orc_philox4x32_10(c.ctypes.data_as(P), k.ctypes.data_as(P), out.ctypes.data_as(P))
    return out


def u24(r: int) -> float:
    return float(np.float32(lib().orc_u24(int(r))))


def uniform(r: int, lo: float, hi: float) -> np.float32:
    return np.float32(lib().orc_uniform(int(r), lo, hi))


def sin_poly(th: float) -> np.float32:
    return np.float32(lib().orc_sin(float(np.float32(th))))


def cos_poly(th: float) -> np.float32:
    return np.float32(lib().orc_cos(float(np.float32(th))))


def sin_series(th: float) -> np.float32:
    return np.float32(lib().orc_sin_series(float(np.float32(th))))


def cos_series(th: float) -> np.float32:
    return np.float32(lib().orc_cos_series(float(np.float32(th))))


def sincos(th: float):
    """(sin, cos) of an fp32 angle: the series on |th| <= fp32(pi/4), quadrant
    reduction outside it."""
    s, c = ctypes.c_float(), ctypes.c_float()
    lib().orc_sincos(float(np.float32(th)), ctypes.byref(s), ctypes.byref(c))
    return np.float32(s.value), np.float32(c.value)


def cartpole_step(params: Params, state, action: int) -> np.ndarray:
    """One Euler step from a 4-float state; returns the next 4 floats."""
    s = np.ascontiguousarray(state, dtype=np.float32)
    out = np.zeros(4, dtype=np.float32)
    P = ctypes.POINTER(ctypes.c_float)
    lib().orc_cartpole_step(ctypes.byref(params), s.ctypes.data_as(P), int(action), out.ctypes.data_as(P))
    return out


def env_step(params: Params, state, action: int) -> np.ndarray:
    """One simulation step: compute_factor Euler iterations of tau / C."""
    s = np.ascontiguousarray(state, dtype=np.float32)
    out = np.zeros(4, dtype=np.float32)
    P = ctypes.POINTER(ctypes.c_float)
    lib().orc_env_step(ctypes.byref(params), s.ctypes.data_as(P), int(action), out.ctypes.data_as(P))
    return out


def terminated(params: Params, state) -> bool:
    s = np.ascontiguousarray(state, dtype=np.float32)
    return bool(lib().orc_terminated(ctypes.byref(params), s.ctypes.data_as(ctypes.POINTER(ctypes.c_float))))


def reset_draw(params: Params, seed: int, env: int, t: int) -> np.ndarray:
    out = np.zeros(4, dtype=np.float32)
    lib().orc_reset_draw(ctypes.byref(params), seed, env, t, out.ctypes.data_as(ctypes.POINTER(ctypes.c_float)))
    return out


def action_bit(seed: int, env: int, t: int) -> int:
    return int(lib().orc_action_bit(seed, env, t))


def policy_u(seed: int, env: int, t: int) -> np.float32:
    return np.float32(lib().orc_policy_u(seed, env, t))


def pad_params(params: Params, seed: int, env: int, j: int):
    a = ctypes.c_float()
    b = ctypes.c_float()
    lib().orc_pad_params(ctypes.byref(params), seed, env, j, ctypes.byref(a), ctypes.byref(b))
    return np.float32(a.value), np.float32(b.value)


def pad_update(s: float, a: float, b: float, u: int) -> np.float32:
    return np.float32(lib().orc_pad_update(float(s), float(a), float(b), int(u)))


def round_bf16(v: float) -> float:
    return float(lib().orc_round_bf16(float(v)))


class Policy:
    """MLP weights (fp32 numpy, row-major [out][in]) for the oracle; wv (1 x 64)
    and bv (1,) are the optional value head."""

    def __init__(self, w1, b1, w2, b2, w3, b3, wv=None, bv=None, bf16: bool = False):
        self._arrs = [None if x is None else np.ascontiguousarray(x, dtype=np.float32)
                      for x in (w1, b1, w2, b2, w3, b3, wv, bv)]
        shapes = [(64, 4), (64,), (64, 64), (64,), (2, 64), (2,), (1, 64), (1,)]
        for a, shp in zip(self._arrs, shapes):
            if a is not None and a.shape != shp:
                raise ValueError(f"policy array shape {a.shape} != {shp}")
        for i in (0, 2, 4):
            if self._arrs[i] is None:
                raise ValueError("weights may not be None")
        self.has_value = self._arrs[6] is not None
        P = ctypes.POINTER(ctypes.c_float)
        self.struct = _Policy(int(bool(bf16)), *[
            ctypes.cast(None, P) if a is None else a.ctypes.data_as(P) for a in self._arrs])

    def p0(self, obs) -> float:
        o = np.ascontiguousarray(obs, dtype=np.float32)
        return float(lib().orc_mlp_p0(ctypes.byref(self.struct), o.ctypes.data_as(ctypes.POINTER(ctypes.c_float))))

    def eval(self, obs):
        """(logits [2] f64, p0, value) for one observation."""
        o = np.ascontiguousarray(obs, dtype=np.float32)
        logit = np.zeros(2, dtype=np.float64)
        p0 = ctypes.c_double()
        v = ctypes.c_double()
        lib().orc_mlp_eval(ctypes.byref(self.struct), o.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
                           logit.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), ctypes.byref(p0), ctypes.byref(v))
        return logit, float(p0.value), float(v.value)

    def log_prob(self, obs, action: int) -> float:
        logit, _, _ = self.eval(obs)
        return log_prob(logit, action)

    def bounds(self, obs, errs: "Errs") -> dict:
        """Enclosures (lo, hi) of p0, log pi(0), log pi(1) and the value that a
        device evaluation under the error model errs may return for obs."""
        o = np.ascontiguousarray(obs, dtype=np.float32)
        b = Bounds()
        lib().orc_mlp_bounds(ctypes.byref(self.struct), o.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
                             ctypes.byref(errs), ctypes.byref(b))
        return dict(p0=(b.p0_lo, b.p0_hi), logp0=(b.lp0_lo, b.lp0_hi), logp1=(b.lp1_lo, b.lp1_hi),
                    value=(b.v_lo, b.v_hi))


def log_prob(logit, action: int) -> float:
    """log softmax(logit)[action] for two logits."""
    lg = np.ascontiguousarray(logit, dtype=np.float64)
    return float(lib().orc_log_prob(lg.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), int(action)))


class Sim:
    """A slice of environments with global ids env0 .. env0+n-1."""

    def __init__(self, n_envs: int, D: int, params: Params, env0: int = 0):
        self.n, self.D, self.env0 = int(n_envs), int(D), int(env0)
        self.params = params
        self._h = lib().orc_create(self.n, self.env0, self.D, ctypes.byref(params))
        if not self._h:
            raise MemoryError("orc_create failed")

    def __del__(self):
        h = getattr(self, "_h", None)
        if h:
            lib().orc_destroy(h)
            self._h = None

    @property
    def n_blocks(self) -> int:
        return (self.env0 + self.n - 1) // 256 - self.env0 // 256 + 1

    def reset(self, seed: int) -> None:
        lib().orc_reset(self._h, int(seed))

    def step(self, K: int, policy: Policy | None = None, record: bool = True, stats: bool = True):
        """Run K steps; returns dict of trajectory arrays (or {} if not record)."""
        n = self.n
        out = {}
        ptr = lambda a: a.ctypes.data if a is not None else None  # noqa: E731
        if record:
            out["obs"] = np.empty((K, 4, n), dtype=np.float32)
            out["action"] = np.empty((K, n), dtype=np.uint8)
            out["reward"] = np.empty((K, n), dtype=np.float32)
            out["done"] = np.empty((K, n), dtype=np.uint8)
            if policy is not None:
                out["p0"] = np.empty((K, n), dtype=np.float64)
                out["logp"] = np.empty((K, n), dtype=np.float64)
                if policy.has_value:
                    out["value"] = np.empty((K, n), dtype=np.float64)
        if stats:
            out["stats"] = np.empty((self.n_blocks, 4), dtype=np.uint32)
        rc = lib().orc_step(self._h, int(K), ctypes.byref(policy.struct) if policy is not None else None,
                            ptr(out.get("obs")), ptr(out.get("action")), ptr(out.get("reward")),
                            ptr(out.get("done")), ptr(out.get("stats")), ptr(out.get("p0")),
                            ptr(out.get("logp")), ptr(out.get("value")))
        if rc != 0:
            raise RuntimeError(f"orc_step failed ({rc})")
        return out

    def get_state(self):
        st = np.empty((4 + self.D, self.n), dtype=np.float32)
        ep = np.empty(self.n, dtype=np.uint32)
        t = ctypes.c_uint64()
        lib().orc_get_state(self._h, st.ctypes.data, ep.ctypes.data, ctypes.byref(t))
        return st, ep, int(t.value)

    def set_state(self, state, ep, t: int) -> None:
        st = np.ascontiguousarray(state, dtype=np.float32)
        e = np.ascontiguousarray(ep, dtype=np.uint32)
        if st.shape != (4 + self.D, self.n) or e.shape != (self.n,):
            raise ValueError("state shape mismatch")
        rc = lib().orc_set_state(self._h, st.ctypes.data, e.ctypes.data, int(t))
        if rc != 0:
            raise RuntimeError(f"orc_set_state failed ({rc})")

    def pad_params(self):
        a = np.empty((self.D, self.n), dtype=np.float32)
        b = np.empty((self.D, self.n), dtype=np.float32)
        lib().orc_get_pad_params(self._h, a.ctypes.data, b.ctypes.data)
        return a, b


def check_rows(params: Params, seed: int, env0: int, t0: int, obs, action, reward, done, ep0=None,
               final_state=None, final_ep=None):
    """Teacher-forced check of recorded random-action rows ([K][4][n] obs,
    [K][n] action / reward / done for envs env0 ..).  ep0 None: every episode
    began at t0, so row 0 must be the reset draw for t0.  final_state ([4][n])
    and final_ep ([n]), optional, must be the state after the last row.
    Returns (number of mismatching env-steps, (k, i) of the first or None)."""
    obs = np.ascontiguousarray(obs, dtype=np.float32)
    action = np.ascontiguousarray(action, dtype=np.uint8)
    reward = np.ascontiguousarray(reward, dtype=np.float32)
    done = np.ascontiguousarray(done, dtype=np.uint8)
    K, four, n = obs.shape
    assert four == 4 and action.shape == reward.shape == done.shape == (K, n)
    c = lambda x, dt: None if x is None else np.ascontiguousarray(x, dtype=dt)  # noqa: E731
    e, fs, fe = c(ep0, np.uint32), c(final_state, np.float32), c(final_ep, np.uint32)
    assert fs is None or fs.shape == (4, n)
    assert fe is None or fe.shape == (n,)
    ptr = lambda x: None if x is None else x.ctypes.data  # noqa: E731
    bk, bi = ctypes.c_uint32(0), ctypes.c_uint32(0)
    bad = lib().orc_check_rows(ctypes.byref(params), int(seed), int(env0), int(n), int(t0), int(K),
                               ptr(e), obs.ctypes.data, action.ctypes.data, reward.ctypes.data, done.ctypes.data,
                               ptr(fs), ptr(fe), ctypes.byref(bk), ctypes.byref(bi))
    return int(bad), ((int(bk.value), int(bi.value)) if bad else None)


def check_policy_rows(params: Params, policy: "Policy", seed: int, env0: int, t0: int, obs, action, reward, done,
                      p0, errs: "Errs", logp=None, value=None, ep0=None, final_state=None, final_ep=None,
                      dp0_out=None):
    """Teacher-forced check of recorded policy rows against the enclosures of
    orc_mlp_bounds under errs.  Returns (failing env-steps, first failure (k, i)
    or None, stats) with stats = dict(worst: max |p0 - oracle p0|, max_width and
    mean_width of the p0 enclosures, exempt: actions that differ from the
    oracle's own choice, necessarily with u inside the enclosure).  ep0,
    final_state and final_ep as for check_rows; dp0_out, a float32 [K][n]
    array, receives |p0 - oracle p0| of every env-step."""
    c = lambda x, dt: None if x is None else np.ascontiguousarray(x, dtype=dt)  # noqa: E731
    obs, action, reward, done = c(obs, np.float32), c(action, np.uint8), c(reward, np.float32), c(done, np.uint8)
    p0, logp, value, ep0 = c(p0, np.float32), c(logp, np.float32), c(value, np.float32), c(ep0, np.uint32)
    fs, fe = c(final_state, np.float32), c(final_ep, np.uint32)
    K, four, n = obs.shape
    assert four == 4 and action.shape == reward.shape == done.shape == p0.shape == (K, n)
    if dp0_out is not None:
        assert dp0_out.dtype == np.float32 and dp0_out.shape == (K, n) and dp0_out.flags.c_contiguous
    ptr = lambda x: None if x is None else x.ctypes.data  # noqa: E731
    st = (ctypes.c_double * 3)()
    ex = ctypes.c_uint64(0)
    bk, bi = ctypes.c_uint32(0), ctypes.c_uint32(0)
    bad = lib().orc_check_policy_rows(ctypes.byref(params), ctypes.byref(policy.struct), int(seed), int(env0), int(n),
                                      int(t0), int(K), ptr(ep0), ptr(obs), ptr(action), ptr(reward), ptr(done),
                                      ptr(p0), ptr(logp), ptr(value), ctypes.byref(errs), ptr(fs), ptr(fe),
                                      ptr(dp0_out), st, ctypes.byref(ex),
                                      ctypes.byref(bk), ctypes.byref(bi))
    stats = dict(worst=st[0], max_width=st[1], mean_width=st[2] / max(1, K * n), exempt=int(ex.value))
    return int(bad), ((int(bk.value), int(bi.value)) if bad else None), stats


# ---------------------------------------------------------------------------
# The chain simulator: a cart carrying N identical uniform rods.
# ---------------------------------------------------------------------------
def chain_consts(params: Params, n_links: int) -> ChainConsts:
    k = ChainConsts()
    if lib().orc_chain_make_consts(ctypes.byref(params), int(n_links), ctypes.byref(k)) != 0:
        raise ValueError(f"n_links must be in [1, {CHAIN_MAX_LINKS}]")
    return k


def chain_accel(params: Params, n_links: int, state, force: float) -> np.ndarray:
    """Accelerations (xdd, phidd_1..N) of a chain state (x, xd, phi_1, phid_1, ...)."""
    k = chain_consts(params, n_links)
    s = np.ascontiguousarray(state, dtype=np.float32)
    assert s.shape == (2 * (n_links + 1),)
    out = np.zeros(n_links + 1, dtype=np.float32)
    P = ctypes.POINTER(ctypes.c_float)
    lib().orc_chain_accel(ctypes.byref(k), s.ctypes.data_as(P), float(force), out.ctypes.data_as(P))
    return out


def chain_step(params: Params, n_links: int, state, action: int) -> np.ndarray:
    """One simulation step of the chain (compute_factor Euler iterations)."""
    k = chain_consts(params, n_links)
    s = np.ascontiguousarray(state, dtype=np.float32)
    assert s.shape == (2 * (n_links + 1),)
    out = np.zeros_like(s)
    P = ctypes.POINTER(ctypes.c_float)
    lib().orc_chain_env_step(ctypes.byref(params), ctypes.byref(k), s.ctypes.data_as(P), int(action),
                             out.ctypes.data_as(P))
    return out


def chain_terminated(params: Params, n_links: int, state) -> bool:
    s = np.ascontiguousarray(state, dtype=np.float32)
    return bool(lib().orc_chain_terminated(ctypes.byref(params), int(n_links),
                                           s.ctypes.data_as(ctypes.POINTER(ctypes.c_float))))


def chain_reset_draw(params: Params, n_links: int, seed: int, env: int, t: int) -> np.ndarray:
    out = np.zeros(2 * (n_links + 1), dtype=np.float32)
    lib().orc_chain_reset_draw(ctypes.byref(params), int(n_links), int(seed), int(env), int(t),
                               out.ctypes.data_as(ctypes.POINTER(ctypes.c_float)))
    return out


class ChainSim:
    """A slice of chain environments with global ids env0 .. env0+n-1."""

    def __init__(self, n_envs: int, n_links: int, params: Params, env0: int = 0):
        self.n, self.N, self.env0 = int(n_envs), int(n_links), int(env0)
        self.S = 2 * (self.N + 1)
        self.params = params
        self._h = lib().orc_chain_create(self.n, self.env0, self.N, ctypes.byref(params))
        if not self._h:
            raise ValueError("orc_chain_create failed (bad n_links or compute_factor, or out of memory)")

    def __del__(self):
        h = getattr(self, "_h", None)
        if h:
            lib().orc_chain_destroy(h)
            self._h = None

    @property
    def n_blocks(self) -> int:
        return (self.env0 + self.n - 1) // 256 - self.env0 // 256 + 1

    def reset(self, seed: int) -> None:
        lib().orc_chain_reset(self._h, int(seed))

    def step(self, K: int, record: bool = True, stats: bool = True):
        n, S = self.n, self.S
        out = {}
        if record:
            out["obs"] = np.empty((K, S, n), dtype=np.float32)
            out["action"] = np.empty((K, n), dtype=np.uint8)
            out["reward"] = np.empty((K, n), dtype=np.float32)
            out["done"] = np.empty((K, n), dtype=np.uint8)
        if stats:
            out["stats"] = np.empty((self.n_blocks, 4), dtype=np.uint32)
        ptr = lambda key: out[key].ctypes.data if key in out else None  # noqa: E731
        rc = lib().orc_chain_step(self._h, int(K), ptr("obs"), ptr("action"), ptr("reward"), ptr("done"), ptr("stats"))
        if rc != 0:
            raise RuntimeError(f"orc_chain_step failed ({rc})")
        return out

    def get_state(self):
        st = np.empty((self.S, self.n), dtype=np.float32)
        ep = np.empty(self.n, dtype=np.uint32)
        t = ctypes.c_uint64()
        lib().orc_chain_get_state(self._h, st.ctypes.data, ep.ctypes.data, ctypes.byref(t))
        return st, ep, int(t.value)

    def set_state(self, state, ep, t: int) -> None:
        st = np.ascontiguousarray(state, dtype=np.float32)
        e = np.ascontiguousarray(ep, dtype=np.uint32)
        if st.shape != (self.S, self.n) or e.shape != (self.n,):
            raise ValueError("state shape mismatch")
        rc = lib().orc_chain_set_state(self._h, st.ctypes.data, e.ctypes.data, int(t))
        if rc != 0:
            raise RuntimeError(f"orc_chain_set_state failed ({rc})")


def chain_check_rows(params: Params, n_links: int, seed: int, env0: int, t0: int, obs, action, reward, done,
                     ep0=None, final_state=None, final_ep=None):
    """check_rows for the chain simulator ([K][2N+2][n] obs)."""
    c = lambda x, dt: None if x is None else np.ascontiguousarray(x, dtype=dt)  # noqa: E731
    obs, action, reward, done = c(obs, np.float32), c(action, np.uint8), c(reward, np.float32), c(done, np.uint8)
    e, fs, fe = c(ep0, np.uint32), c(final_state, np.float32), c(final_ep, np.uint32)
    K, S, n = obs.shape
    assert S == 2 * (n_links + 1) and action.shape == reward.shape == done.shape == (K, n)
    assert fs is None or fs.shape == (S, n)
    assert fe is None or fe.shape == (n,)
    ptr = lambda x: None if x is None else x.ctypes.data  # noqa: E731
    bk, bi = ctypes.c_uint32(0), ctypes.c_uint32(0)
    bad = lib().orc_chain_check_rows(ctypes.byref(params), int(n_links), int(seed), int(env0), int(n), int(t0), int(K),
                                     ptr(e), ptr(obs), ptr(action), ptr(reward), ptr(done), ptr(fs), ptr(fe),
                                     ctypes.byref(bk), ctypes.byref(bi))
    return int(bad), ((int(bk.value), int(bi.value)) if bad else None)
