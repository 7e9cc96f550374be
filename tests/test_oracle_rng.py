"""Pins of the oracle's random-number contract (CPU only).

* Philox4x32-10 against the published known-answer vectors and against
  rocRAND's independent implementation of the same bijection.
* The 24-bit uniform mapping: exact, inside [lo, hi].
* The stream contract: reset draws inside the initial-state box, fair action
  bits, and draws that depend only on (seed, env, step).
"""
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle
import workloads

HERE = os.path.dirname(os.path.abspath(__file__))


def _kat_rows():
    rows = []
    with open(os.path.join(HERE, "golden", "philox4x32_10_kat.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            v = [int(x, 16) for x in line.split()]
            rows.append((v[0:4], v[4:6], v[6:10]))
    return rows


def test_philox_known_answers():
    rows = _kat_rows()
    assert len(rows) == 3
    for ctr, key, want in rows:
        got = oracle.philox4x32_10(ctr, key)
        assert [int(x) for x in got] == want, (ctr, key)


def _build_rocrand_xcheck(tmp_path):
    hdr = "/opt/rocm/include/rocrand/rocrand_philox4x32_10.h"
    cxx = shutil.which("g++")
    if not (os.path.exists(hdr) and cxx):
        pytest.skip("rocRAND header or g++ not present: cross-check unavailable")
    exe = str(tmp_path / "philox_rocrand")
    subprocess.run([cxx, "-O1", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                    os.path.join(HERE, "xcheck", "philox_rocrand.cpp"), "-o", exe], check=True)
    return exe


def test_philox_matches_rocrand(tmp_path):
    exe = _build_rocrand_xcheck(tmp_path)
    rng = np.random.Generator(np.random.PCG64(1234))
    n = 20000
    pairs = rng.integers(0, 2**32, size=(n, 6), dtype=np.uint64).astype(np.uint32)
    # include the shapes the simulator uses: small env ids, block ids and stream ids
    pairs[: n // 2, 2] = rng.integers(0, 4, size=n // 2)
    pairs[: n // 2, 3] = 0
    res = subprocess.run([exe], input=pairs.tobytes(), capture_output=True, check=True)
    theirs = np.frombuffer(res.stdout, dtype=np.uint32).reshape(n, 4)
    for i in range(n):
        ours = oracle.philox4x32_10(pairs[i, :4], pairs[i, 4:])
        assert np.array_equal(ours, theirs[i]), i


def test_philox_bit_balance():
    # every output bit of consecutive counters is set about half the time
    words = np.array([oracle.philox4x32_10([i, 7, 1, 0], [3, 5]) for i in range(4096)], dtype=np.uint32)
    bits = ((words[:, :, None] >> np.arange(32, dtype=np.uint32)) & 1).reshape(-1, 32)
    freq = bits.mean(axis=0)
    # 16384 samples per bit: 5 sigma = 5 * 0.5 / sqrt(16384) = 0.0195
    assert np.all(np.abs(freq - 0.5) < 0.0195)


def test_u24_exact_and_in_range():
    for r in [0, 1, 255, 256, 0x12345678, 0xFFFFFF00, 0xFFFFFFFF]:
        want = (r >> 8) / 2.0**24          # exact in double, and representable in fp32
        assert oracle.u24(r) == want
    assert oracle.u24(0xFFFFFFFF) == 1.0 - 2.0**-24


def test_uniform_is_single_rounded_fma():
    # lo + u*(hi-lo) with one rounding: compare with exact rational arithmetic
    from fractions import Fraction
    lo, hi = np.float32(-0.05), np.float32(0.05)
    width = np.float32(hi - lo)
    rng = np.random.Generator(np.random.PCG64(7))
    for r in rng.integers(0, 2**32, size=2000, dtype=np.uint64):
        r = int(r)
        exact = Fraction(r >> 8, 2**24) * Fraction(float(width)) + Fraction(float(lo))
        got = oracle.uniform(r, float(lo), float(hi))
        # the correctly rounded fp32 of `exact` is the nearest float to it
        cand = np.float32(float(exact))
        err_got = abs(Fraction(float(got)) - exact)
        err_nb = min(abs(Fraction(float(np.nextafter(cand, np.float32(s)))) - exact) for s in (-1, 1))
        assert err_got <= abs(Fraction(float(cand)) - exact)
        assert err_got <= err_nb


def test_uniform_extremes_inside_box():
    p = workloads.CARTPOLE
    lo, hi = np.float32(p["reset_low"]), np.float32(p["reset_high"])
    assert oracle.uniform(0, float(lo), float(hi)) == lo
    top = oracle.uniform(0xFFFFFFFF, float(lo), float(hi))
    assert lo <= top <= hi
    a_lo, a_hi = np.float32(p["pad_a_low"]), np.float32(p["pad_a_high"])
    assert a_lo <= oracle.uniform(0xFFFFFFFF, float(a_lo), float(a_hi)) <= a_hi


def test_reset_draws_in_box_and_depend_on_block():
    P = oracle.make_params(**workloads.CARTPOLE)
    lo, hi = np.float32(-0.05), np.float32(0.05)
    seen = set()
    for seed in workloads.PARITY_SEEDS:
        for env in (0, 1, 255, 4194303):
            for t in range(0, 32):
                s = oracle.reset_draw(P, seed, env, t)
                assert np.all(s >= lo) and np.all(s <= hi)
                # the eight steps of a block share one draw (block-grouped counter)
                assert np.array_equal(s, oracle.reset_draw(P, seed, env, (t // 8) * 8))
                seen.add(s.tobytes())
    # distinct across blocks, envs and seeds: 3 seeds x 4 envs x 4 blocks
    assert len(seen) == 48


def test_high_seed_word_matters():
    # seeds that differ only above bit 32 give different streams
    a = [oracle.action_bit(7, 3, t) for t in range(256)]
    b = [oracle.action_bit(7 + (1 << 40), 3, t) for t in range(256)]
    assert a != b


def test_action_bits_fair_and_env_dependent():
    bits = np.array([[oracle.action_bit(0, env, t) for t in range(512)] for env in range(64)])
    m = bits.mean()
    # 32768 fair bits: 5 sigma = 0.0138
    assert abs(m - 0.5) < 0.0138
    assert not np.array_equal(bits[0], bits[1])
    # lag-1 correlation of the bit sequence is small
    x = bits.astype(np.float64) - 0.5
    corr = (x[:, 1:] * x[:, :-1]).mean() / 0.25
    assert abs(corr) < 0.03


def test_policy_uniform_range():
    us = np.array([oracle.policy_u(1, env, t) for env in range(16) for t in range(64)])
    assert us.min() >= 0.0 and us.max() < 1.0
    assert abs(us.mean() - 0.5) < 0.05


def test_action_block_carries_one_philox_output():
    """128 consecutive actions of a block are the 128 bits of one generator
    output (stream 1, counter block t/128), least significant bit first; the
    generator itself is pinned by the known-answer vectors above."""
    for seed, env, blk in ((0, 0, 0), (1, 77, 3), ((1 << 40) + 7, 4194303, 1)):
        bits = [oracle.action_bit(seed, env, blk * 128 + i) for i in range(128)]
        words = [sum(bits[32 * w + i] << i for i in range(32)) for w in range(4)]
        want = oracle.philox4x32_10([env, blk, 1, 0], [seed & 0xFFFFFFFF, seed >> 32])
        assert words == [int(x) for x in want]


def test_policy_uniform_is_word_of_block():
    for seed, env, t in ((0, 5, 0), (3, 9, 13), ((1 << 40) + 7, 1000, 255)):
        w = oracle.philox4x32_10([env, t // 4, 3, 0], [seed & 0xFFFFFFFF, seed >> 32])
        assert oracle.policy_u(seed, env, t) == (int(w[t % 4]) >> 8) / 2.0**24


def test_reset_and_param_draws_use_their_streams():
    P = oracle.make_params(**workloads.CARTPOLE)
    w = oracle.philox4x32_10([12, 2, 0, 0], [9, 0])
    want = [oracle.uniform(int(x), -0.05, 0.05) for x in w]
    assert list(oracle.reset_draw(P, 9, 12, 21)) == want
    w = oracle.philox4x32_10([12, 7, 2, 0], [9, 0])
    a, b = oracle.pad_params(P, 9, 12, 7)
    assert a == oracle.uniform(int(w[0]), 0.9, 0.99) and b == oracle.uniform(int(w[1]), -1.0, 1.0)


def test_padding_update_is_single_rounded_recurrence():
    """s <- a s + b u, one rounding: the fused a s + b for u = 1, the product a s
    for u = 0 (no b term, so the sign of a zero product is kept)."""
    from fractions import Fraction
    rng = np.random.Generator(np.random.PCG64(3))
    for _ in range(2000):
        s, a, b = (np.float32(v) for v in rng.standard_normal(3))
        for u in (0, 1):
            exact = Fraction(float(a)) * Fraction(float(s)) + (Fraction(float(b)) if u else 0)
            got = oracle.pad_update(s, a, b, u)
            cand = np.float32(float(exact))
            # nearest float: no neighbour of the result is closer to the exact value
            err = abs(Fraction(float(got)) - exact)
            for nb in (np.nextafter(got, np.float32(-np.inf)), np.nextafter(got, np.float32(np.inf))):
                assert err <= abs(Fraction(float(nb)) - exact)
            assert err <= abs(Fraction(float(cand)) - exact)
    assert np.signbit(oracle.pad_update(-0.0, 0.9, 0.5, 0))
    assert not np.signbit(oracle.pad_update(0.0, 0.9, -0.5, 0))
