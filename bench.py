#!/usr/bin/env python3
"""Benchmark of the fused data-collection kernel on one MI355X.

One bench "step" is one pass of the whole hot path over the headline workload:
4,194,304 cart-pole environments advanced 200 steps by ONE launch of the fused
kernel (K = 200), writing the full trajectory (obs f32 x 4, action u8, reward
f32, done u8 per env-step) and the per-256-env block statistics.  Inputs are
synthetic: the library draws every initial state and action on the device from
Philox keyed by the seed.  Prints one JSON line.

    python bench.py [--gpus 1] [--steps 20] [--warmup 3] [--no-cpu] [--no-unfused]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import workloads  # noqa: E402

METRIC = "env-steps/sec at 1 MI355X; achieved HBM GB/s vs peak; fused/unfused speedup"
HBM_PEAK_GBS = 8000.0
# fp32 VALU peak in lane operations (one FMA or multiply per lane) per second:
# the published 157.3 TFLOP/s fp32 vector rate, an FMA counted as two flops,
# i.e. 32 lanes per clock per SIMD at 2.4 GHz.  Plain (non-packed) v_fma_f32 and
# v_mul_f32 reach 25-29.5 lanes per clock (rlsim_probe_issue, eight waves per
# SIMD); under sustained VALU load the shader clock falls to 1.6-2.2 GHz.
VALU_LANE_OPS_PER_S = 157.3e12 / 2
COPY_BYTES = 1 << 30        # size of the plain copy used to calibrate the HBM byte counters


def traffic_file(workload: str) -> str:
    return os.path.join(ROOT, "profiles", f"hbm_traffic__{workload}.txt")


# sources of the fused random-action kernel the headline times, and of the
# launch code that picks it
FUSED_KERNEL_SOURCES = ("device_common.hip.h", "k_cartpole.hip.h", "rlsim.hip")
# the kernel a trajectory-recording launch of K >= 16 steps without padding
# words runs (the headline launch), as rocprofv3 names it and as reported
HEADLINE_KERNEL_PREFIX = "void rlsim_dev::k_cartpole_split<0,"
HEADLINE_KERNEL = "k_cartpole_split<0,STATS>"


def code_text(src: str) -> str:
    """C++ source without its comments and with whitespace collapsed: what the
    compiler sees, so that editing a comment leaves the digest alone."""
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", " ", src)
    return " ".join(src.split())


def kernel_source_digest() -> str:
    """Digest of the fused kernel's sources (code only, comments stripped): a
    stored traffic measurement is used only while the kernel it was taken on is
    unchanged."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2207_07736_amd", "csrc")
    for f in FUSED_KERNEL_SOURCES:
        with open(os.path.join(csrc, f), encoding="utf-8") as fh:
            h.update(f.encode() + b"\0" + code_text(fh.read()).encode())
    return h.hexdigest()[:16]


def _read_kv(path: str) -> dict:
    out = {}
    with open(path) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#") and ":" in line:
                k, v = line.split(":", 1)
                out[k.strip()] = v.strip()
    return out


def stored_traffic(workload: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or None
    when there is none or the kernel sources changed since it was taken."""
    try:
        d = _read_kv(traffic_file(workload))
    except OSError:
        return None
    if d.get("source_digest") != kernel_source_digest():
        return None
    return float(d["hbm_bytes_per_launch"])


def ingest_pmc(fetch_csv: str, write_csv: str, workload: str, kernel_prefix: str) -> str:
    """Turn two rocprofv3 --pmc counter CSVs (FETCH_SIZE, then WRITE_SIZE, KiB per
    dispatch) into the traffic summary: each counter is scaled by what it reads
    for the plain device copy of COPY_BYTES that --copy-calibration runs."""
    import csv
    import statistics

    def per_kernel(path, counter):
        vals = {}
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] == counter:
                vals.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
        return vals

    f, w = per_kernel(fetch_csv, "FETCH_SIZE"), per_kernel(write_csv, "WRITE_SIZE")
    kf = [k for k in f if k.startswith(kernel_prefix)]
    copy_f = [k for k in f if "copy" in k.lower() or "elementwise" in k.lower()]
    copy_w = [k for k in w if "copy" in k.lower() or "elementwise" in k.lower()]
    if len(kf) != 1 or not copy_f or not copy_w:
        raise SystemExit(f"cannot find the kernel / copy dispatches: {list(f)}")
    k = kf[0]
    fetch_kib = statistics.median(f[k])
    write_kib = statistics.median(w[k])
    # the copy reads and writes COPY_BYTES; its dispatch is the largest such one
    cf = max(max(v) for kk, v in f.items() if kk in copy_f)
    cw = max(max(v) for kk, v in w.items() if kk in copy_w)
    fetch_scale = COPY_BYTES / (cf * 1024.0)
    write_scale = COPY_BYTES / (cw * 1024.0)
    hbm = fetch_kib * 1024.0 * fetch_scale + write_kib * 1024.0 * write_scale
    path = traffic_file(workload)
    with open(path, "w") as fh:
        fh.write(f"""# HBM traffic of one launch, from rocprofv3 counters (KiB per dispatch, median)
# commands (repository root, run from /tmp with TMPDIR=/tmp):
#   rocprofv3 --pmc FETCH_SIZE --output-format csv -d <out>/pmc_fetch -o f -- python3 <repo>/bench.py --steps 3 --warmup 1 --no-cpu --no-sweep --no-unfused --copy-calibration
#   rocprofv3 --pmc WRITE_SIZE --output-format csv -d <out>/pmc_write -o w -- python3 <repo>/bench.py --steps 3 --warmup 1 --no-cpu --no-sweep --no-unfused --copy-calibration
#   python bench.py --ingest-pmc <out>/pmc_fetch/f_counter_collection.csv <out>/pmc_write/w_counter_collection.csv
# counters are scaled by what they read for a plain {COPY_BYTES} B device copy (torch copy_)
kernel: {k}
workload: {workload}
source_digest: {kernel_source_digest()}
fetch_kib_per_dispatch: {fetch_kib:.1f}
write_kib_per_dispatch: {write_kib:.1f}
copy_fetch_kib: {cf:.1f}
copy_write_kib: {cw:.1f}
copy_fetch_scale: {fetch_scale:.4f}
copy_write_scale: {write_scale:.4f}
hbm_bytes_per_launch: {hbm:.0f}
""")
    return path


def _oracle_slices(n_slice_envs: int, starts, T: int, seed: int, threads: int, D: int = 0, policy=None,
                   links: int = 0) -> float:
    """Wall seconds for the oracle to run T recorded steps of each env slice
    [start, start + n_slice_envs), `threads` slices at a time (links > 0: the
    chain model).  Each slice is its own oracle instance; the oracle's C loop
    runs outside the GIL."""
    import concurrent.futures as cf

    import oracle
    params = oracle.make_params(**workloads.CARTPOLE)

    def one(start):
        if links:
            sim = oracle.ChainSim(n_slice_envs, links, params, env0=start)
            sim.reset(seed)
            t0 = time.perf_counter()
            sim.step(T)
            return time.perf_counter() - t0
        sim = oracle.Sim(n_slice_envs, D, params, env0=start)
        sim.reset(seed)
        t0 = time.perf_counter()
        sim.step(T, policy=policy)
        return time.perf_counter() - t0

    if threads == 1:
        return sum(one(s) for s in starts)
    t0 = time.perf_counter()
    with cf.ThreadPoolExecutor(max_workers=threads) as ex:
        list(ex.map(one, starts))
    return time.perf_counter() - t0


def cpu_baseline(n_slice_envs: int, slices: int, T: int, seed: int) -> dict:
    """The oracle (plain C loop, as it stands) on bounded samples of the
    headline workload: env slices of the 4M batch, T steps each, trajectory
    recorded.  Reported multi-threaded (one slice per host thread at a time, as
    the paper's multi-core C++ simulator baseline divides environments over
    cores) and single-threaded."""
    import oracle  # noqa: F401  (builds the oracle before any timing)
    n_total = workloads.WORKLOADS[workloads.HEADLINE]["n"]
    threads = max(1, min(16, len(os.sched_getaffinity(0))))
    single_starts = [i * (n_total // slices) for i in range(slices)]
    single_s = _oracle_slices(n_slice_envs, single_starts, T, seed, 1)
    single = n_slice_envs * slices * T / single_s
    mt_slices = 2 * threads
    mt_starts = [i * (n_total // mt_slices) for i in range(mt_slices)]
    mt_s = _oracle_slices(n_slice_envs, mt_starts, T, seed, threads)
    multi = n_slice_envs * mt_slices * T / mt_s
    return {"value": multi, "unit": "env-steps/s", "cores": threads, "kind": "oracle",
            "sample": f"{mt_slices} slices x {n_slice_envs} envs x {T} steps of the 4,194,304-env headline batch "
                      f"(seed {seed}, trajectory recorded) on {threads} threads, {mt_s:.1f} s wall",
            "single_thread": {"value": single, "unit": "env-steps/s", "cores": 1,
                              "sample": f"{slices} slices x {n_slice_envs} envs x {T} steps, {single_s:.1f} s"},
            "other_workloads": cpu_other_workloads(threads), "host": host_cpu()}


def host_cpu() -> dict:
    """The host the oracle was timed on: CPU model, logical CPUs, and the CPUs
    this process may run on."""
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"cpu_model": model, "logical_cpus": os.cpu_count(), "usable_cpus": len(os.sched_getaffinity(0))}


def cpu_other_workloads(threads: int) -> dict:
    """The oracle on the 1,024-env workload in full (one thread), on the K-sweep
    workload in full (65,536 envs x 1,000 steps, on `threads` threads and on
    one), and on bounded slices of the state-size and policy workloads, one
    slice per thread at a time (env-steps/s; trajectories recorded)."""
    import oracle
    out = {}
    w = workloads.WORKLOADS[workloads.SMALL]
    sec = _oracle_slices(w["n"], [0], w["T"], w["seed"], 1)
    out[w["name"]] = {"single_thread": {"value": w["n"] * w["T"] / sec, "unit": "env-steps/s",
                                        "sample": f"all {w['n']} envs x {w['T']} steps on 1 thread, {sec:.3f} s"}}
    w = workloads.WORKLOADS[workloads.K_SWEEP]
    n_slice = w["n"] // threads
    starts = [i * n_slice for i in range(threads)]
    sec = _oracle_slices(n_slice, starts, w["T"], w["seed"], threads)
    sec1 = _oracle_slices(w["n"], [0], w["T"], w["seed"], 1)
    out[w["name"]] = {"threads": {"value": w["n"] * w["T"] / sec, "unit": "env-steps/s",
                                  "sample": f"all {w['n']} envs x {w['T']} steps on {threads} threads, {sec:.1f} s"},
                      "single_thread": {"value": w["n"] * w["T"] / sec1, "unit": "env-steps/s",
                                        "sample": f"all {w['n']} envs x {w['T']} steps on 1 thread, {sec1:.1f} s"}}
    w = workloads.WORKLOADS[workloads.STATE_SWEEP]
    rows = {}
    for D in w["D"]:
        n_total = max(4096, min(65536, (1 << 24) // D))       # about 1-3 s of oracle work per D
        n_slice = n_total // threads
        starts = [i * (w["n"] // threads) for i in range(threads)]
        sec = _oracle_slices(n_slice, starts, w["T"], w["seed"], threads, D=D)
        rows[f"D{D}"] = {"value": n_slice * threads * w["T"] / sec, "unit": "env-steps/s",
                         "sample": f"{threads} slices x {n_slice} envs x {w['T']} steps, {sec:.1f} s wall"}
    out[w["name"]] = rows
    w = workloads.WORKLOADS[workloads.MLP]
    rows = {}
    for dtype, n_total, T in (("f32", 16384, w["T"]), ("bf16", 4096, 64)):
        pol = oracle.Policy(**workloads.mlp_weights(w["seed"]), bf16=(dtype == "bf16"))
        n_slice = n_total // threads
        starts = [i * (w["n"] // threads) for i in range(threads)]
        sec = _oracle_slices(n_slice, starts, T, w["seed"], threads, policy=pol)
        rows[dtype] = {"value": n_slice * threads * T / sec, "unit": "env-steps/s",
                       "sample": f"{threads} slices x {n_slice} envs x {T} steps (policy, value head), {sec:.1f} s wall"}
    out[w["name"]] = rows
    w = workloads.CHAIN_SWEEP
    rows = {}
    for N in w["N"]:
        n_slice = 262144 // threads                              # about 0.3-1 s of oracle work per N
        starts = [i * (w["n"] // threads) for i in range(threads)]
        sec = _oracle_slices(n_slice, starts, w["T"], w["seed"], threads, links=N)
        rows[f"N{N}"] = {"value": n_slice * threads * w["T"] / sec, "unit": "env-steps/s",
                         "sample": f"{threads} slices x {n_slice} envs x {w['T']} steps, {sec:.1f} s wall"}
    out[w["name"]] = rows
    return out


def _time_schedule(sim, traj, sched, stream, reps):
    """Median wall time (ms, HIP events) of running the K schedule `sched`
    (one launch per entry, trajectory rows advanced) over `reps` repetitions."""
    import torch
    structs, k0 = [], 0
    for k in sched:
        structs.append((k, traj.rows(k0, k) if traj is not None else None))
        k0 += k
    times = []
    for r in range(reps + 1):
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record(stream)
        for k, st in structs:
            sim.step(k, st)
        stop.record(stream)
        torch.cuda.synchronize()
        if r:                       # the first repetition is a warm-up
            times.append(start.elapsed_time(stop))
    times.sort()
    return times[len(times) // 2]


def _graph_ms(sim, structs, stream, reps: int) -> float:
    """Median time of replaying one HIP graph that holds the K = 1 launches of
    `structs` (one kernel node per rlsim_step_fused call)."""
    import torch
    g = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=stream):
        for st in structs:
            sim.step(1, st)
    g.replay()
    torch.cuda.synchronize()
    times = []
    for _ in range(reps):
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record(stream)
        g.replay()
        stop.record(stream)
        torch.cuda.synchronize()
        times.append(start.elapsed_time(stop))
    del g
    times.sort()
    return times[len(times) // 2]


def fusion_sweeps(stream) -> dict:
    """The 1,024-env correctness workload's launch-bound timing, and fused
    versus unfused on the K sweep (65,536 envs x 1,000 steps) and the
    state-size sweep (262,144 envs x 500 steps, D padding words per env)."""
    from paper_2207_07736_amd import Simulator, Trajectory
    out = {}
    w = workloads.WORKLOADS[workloads.SMALL]
    n, T = w["n"], w["T"]
    sim = Simulator(n, 0, workloads.CARTPOLE, stream=stream)
    sim.reset(w["seed"])
    traj = Trajectory(T, n)
    ms = _time_schedule(sim, traj, [1] * T, stream, reps=5)
    gms = _graph_ms(sim, [traj.rows(k, 1) for k in range(T)], stream, reps=5)
    fused = _time_schedule(sim, traj, [T], stream, reps=5)
    # launch-latency bound: time per launch, not a roofline fraction
    out[w["name"]] = {"K1": {"ms": ms, "us_per_launch": ms * 1e3 / T},
                      "K1_hipgraph": {"ms": gms, "us_per_launch": gms * 1e3 / T},
                      "K100": {"ms": fused}}
    del traj
    sim.close()
    out[workloads.WORKLOADS[workloads.K_SWEEP]["name"]] = k_sweep(stream)

    w = workloads.WORKLOADS[workloads.STATE_SWEEP]
    n, T = w["n"], w["T"]
    d_rows = {}
    for D in w["D"]:
        sim = Simulator(n, D, workloads.CARTPOLE, stream=stream)
        sim.reset(w["seed"])
        traj = Trajectory(T, n)
        entry = {}
        for K in w["K"]:
            ms = _time_schedule(sim, traj, [K] * (T // K), stream, reps=2)
            state_bytes = (40 + 16 * D) * n * (T // K)
            entry[f"K{K}"] = {"ms": ms, "env_steps_per_s": n * T / (ms * 1e-3),
                              "algorithmic_GBs": (n * T * workloads.TRAJ_BYTES_PER_ENV_STEP + state_bytes) / (ms * 1e-3) / 1e9}
        ms_nt = _time_schedule(sim, None, [T], stream, reps=2)
        entry["K500_no_trajectory"] = {"ms": ms_nt, "env_steps_per_s": n * T / (ms_nt * 1e-3)}
        entry["fusion_speedup"] = entry["K1"]["ms"] / entry["K500"]["ms"]
        # fused: one fp32 VALU instruction per padding word per step is the floor
        entry["K500"]["valu_frac"] = n * D * T / (entry["K500"]["ms"] * 1e-3) / VALU_LANE_OPS_PER_S
        d_rows[f"D{D}"] = entry
        del traj
        sim.close()
        print(f"[bench] sweep D={D}: K1 {entry['K1']['ms']:.2f} ms, K500 {entry['K500']['ms']:.2f} ms", file=sys.stderr,
              flush=True)
    # the unfused wide launches against a plain stream of the same traffic mix
    D = max(w["D"])
    d_rows[f"D{D}"]["K1"]["stream_probe"] = stream_ceiling(n * D, d_rows[f"D{D}"]["K1"]["algorithmic_GBs"], stream)
    out[w["name"]] = d_rows

    out[workloads.WORKLOADS[workloads.MLP]["name"]] = policy_sweep(stream)
    out[workloads.C_SWEEP["name"]] = compute_factor_sweep(stream)
    out[workloads.CHAIN_SWEEP["name"]] = chain_sweep(stream)
    return out


def chain_flops_per_step(N: int) -> int:
    """fp32 operations of one explicit-Euler iteration of the N-link chain, as
    the definition lists them (a product, sum or division counts 1, an FMA 2),
    on the common path where every link angle is within pi/4 (no reduction):
    per link the sin/cos series (18) and phid^2; the mass matrix's cart row and
    each link pair's cos(phi_j - phi_k) and coupling; the forces; the
    elimination (a reciprocal per pivot, a multiplier and an FMA per updated
    entry and right-hand side); the back substitution; the Euler update."""
    pairs = N * (N - 1) // 2
    flops = 18 * N + N                  # sin/cos series, phid^2
    flops += N + 4 * pairs              # A_0k; per pair s s, fma, L h * cos
    flops += 3 * N + N + 8 * pairs      # f_0 terms; g h s; per pair c s, fma, L h * sin, two fmas
    S = N + 1
    for p in range(S - 1):
        flops += 1                      # 1 / A_pp
        for i in range(p + 1, S):
            flops += 1 + 2 * (S - i) + 2
    flops += 1                          # 1 / A_NN
    for i in range(S):
        flops += 2 * (S - 1 - i) + 1    # back substitution
    flops += 4 * S                      # Euler: 2 (N + 1) FMAs
    return flops


def chain_sweep(stream) -> dict:
    """The second simulator: 1,048,576 envs x 200 steps of the N-link chain,
    N = 1 .. 4, fused (one K = 200 launch) against unfused (200 launches of K =
    1), with the fused launch against the HBM roofline (trajectory plus the
    state once) and against the fp32 vector peak (the definition's operations
    per env-step, chain_flops_per_step)."""
    from paper_2207_07736_amd import Simulator, Trajectory
    w = workloads.CHAIN_SWEEP
    n, T = w["n"], w["T"]
    rows = {}
    for N in w["N"]:
        sim = Simulator(n, 0, workloads.CARTPOLE, stream=stream, links=N)
        sim.reset(w["seed"])
        traj = Trajectory(T, n, S=sim.S)
        entry = {}
        state_b = (4 * sim.S + 4) * n * 2
        traj_b = n * T * workloads.chain_traj_bytes_per_env_step(N)
        for K in w["K"]:
            ms = _time_schedule(sim, traj, [K] * (T // K), stream, reps=3)
            algo = traj_b + state_b * (T // K) + 16 * ((n + 255) // 256) * (T // K)
            entry[f"K{K}"] = {"ms": ms, "env_steps_per_s": n * T / (ms * 1e-3),
                              "algorithmic_GBs": algo / (ms * 1e-3) / 1e9}
        fused = entry[f"K{T}"]
        fused["hbm_frac"] = fused["algorithmic_GBs"] / HBM_PEAK_GBS
        fused["flops_per_env_step"] = chain_flops_per_step(N)
        fused["TFLOPs"] = n * T * chain_flops_per_step(N) / (fused["ms"] * 1e-3) / 1e12
        fused["fp32_frac"] = fused["TFLOPs"] / (2 * VALU_LANE_OPS_PER_S / 1e12)
        entry["fusion_speedup"] = entry["K1"]["ms"] / fused["ms"]
        rows[f"N{N}"] = entry
        del traj
        sim.close()
        print(f"[bench] chain N={N}: K1 {entry['K1']['ms']:.2f} ms, K{T} {fused['ms']:.3f} ms "
              f"({fused['hbm_frac']:.2f} of HBM, {fused['fp32_frac']:.2f} of fp32), {entry['fusion_speedup']:.1f}x",
              file=sys.stderr, flush=True)
    return rows


def stream_ceiling(words: int, achieved_gbs: float, stream) -> dict:
    """Time rlsim_probe_stream (read s, a, b; write s) over `words` fp32 words
    per array, and the fraction of its rate that `achieved_gbs` reaches."""
    import torch
    from paper_2207_07736_amd.probe import probe_stream
    s, a, b = (torch.zeros(words, dtype=torch.float32, device="cuda") for _ in range(3))
    probe_stream(s, a, b, stream)
    times = []
    for _ in range(5):
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record(stream)
        probe_stream(s, a, b, stream)
        stop.record(stream)
        torch.cuda.synchronize()
        times.append(start.elapsed_time(stop))
    times.sort()
    ms = times[len(times) // 2]
    gbs = words * 16 / (ms * 1e-3) / 1e9
    del s, a, b
    return {"ms": ms, "GBs": gbs, "frac_of_stream_ceiling": achieved_gbs / gbs}


# iterations per launch of each instruction-rate probe kind (about 1-3 ms)
ISSUE_ITERS = {"fma": 16384, "fma_shared": 16384, "select_fma": 8192, "exp": 4096, "rcp": 4096, "mfma": 1024,
               "mixed": 1024, "mul": 16384, "replay_tree": 256, "replay_flat": 256}
CUS = 256
SIMDS = 4 * CUS


def _probe_ms(kind: str, waves: int, iters: int, out, stream, reps: int = 5, clocks=None):
    """Median launch time of probe `kind` over `reps` launches; with `clocks`,
    also the median shader clock (GHz) of the last launch's workgroups."""
    import torch
    from paper_2207_07736_amd.probe import probe_issue, wall_clock_khz
    blocks = CUS * waves
    probe_issue(kind, blocks, iters, out, stream)
    times = []
    for _ in range(reps):
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record(stream)
        probe_issue(kind, blocks, iters, out, stream, clocks=clocks)
        stop.record(stream)
        torch.cuda.synchronize()
        times.append(start.elapsed_time(stop))
    times.sort()
    ms = times[len(times) // 2]
    if clocks is None:
        return ms
    c = clocks[:2 * blocks].view(blocks, 2).double().cpu()
    ghz = float((c[:, 0] / c[:, 1]).median()) * wall_clock_khz() * 1e-6
    return ms, ghz


def issue_rates(stream) -> dict:
    """The instruction rates the kernels' bounds rest on (rlsim_probe_issue),
    with `waves` waves per SIMD (256 CUs x 4 SIMDs): wave64 v_fma_f32 (with
    distinct source registers, and with one register read twice), v_mul_f32,
    v_exp_f32 and v_rcp_f32 as fp32 lane operations per second; the per-lane
    padding update (a select and an FMA per word) and the wide kernel's
    two-environment replay, with its scalar decisions and with none, as word
    updates per second; fp32 MFMA as TFLOP/s; and one MFMA wave beside one FMA
    wave on every SIMD against each alone (serialised if the mixed time is the
    sum of the two).  Each rate also comes per clock, as lanes per cycle per
    SIMD at the shader clock the probe's own workgroups counted: the clock
    follows the power draw, so rates per second differ with the data."""
    import torch
    out = torch.empty(CUS * 8 * 256, dtype=torch.float32, device="cuda")
    clocks = torch.zeros(CUS * 8 * 2, dtype=torch.int64, device="cuda")
    res = {}
    for kind, waves in (("fma", 1), ("fma", 2), ("fma", 4), ("fma", 8), ("fma_shared", 8), ("mul", 8),
                        ("select_fma", 2), ("select_fma", 8), ("exp", 8), ("rcp", 8), ("replay_tree", 4),
                        ("replay_tree", 8), ("replay_flat", 4), ("replay_flat", 8)):
        it = ISSUE_ITERS[kind]
        ms, ghz = _probe_ms(kind, waves, it, out, stream, clocks=clocks)
        if kind.startswith("replay"):
            lanes, unit = CUS * waves * 256 * it * 32 * 16, "word updates"
        else:
            lanes, unit = CUS * waves * 256 * it * 8, "word updates" if kind == "select_fma" else "lane ops"
        per_s = lanes / (ms * 1e-3)
        res[f"{kind}_w{waves}"] = {"ms": ms, "per_s": per_s, "unit": unit, "clock_ghz": ghz,
                                   "lanes_per_clk_per_simd": per_s / (SIMDS * ghz * 1e9)}
    it = ISSUE_ITERS["mfma"]
    for waves in (1, 2):
        ms, ghz = _probe_ms("mfma", waves, it, out, stream, clocks=clocks)
        flops = CUS * waves * 4 * it * 4 * (32 * 32 * 2 * 2)
        res[f"mfma_f32_w{waves}"] = {"ms": ms, "TFLOPs": flops / (ms * 1e-3) / 1e12, "clock_ghz": ghz,
                                     "flops_per_clk_per_cu": flops / (ms * 1e-3) / (CUS * ghz * 1e9)}
    # one MFMA wave and one FMA wave per SIMD, against each alone at one wave per SIMD
    mixed = _probe_ms("mixed", 2, it, out, stream)
    fma_alone = _probe_ms("fma", 1, 16 * it, out, stream)
    res["mfma_beside_fma"] = {"mixed_ms": mixed, "mfma_alone_ms": res["mfma_f32_w1"]["ms"], "fma_alone_ms": fma_alone,
                              "mixed_over_sum": mixed / (res["mfma_f32_w1"]["ms"] + fma_alone),
                              "mixed_over_max": mixed / max(res["mfma_f32_w1"]["ms"], fma_alone)}
    del out, clocks
    print("[bench] issue rates: " + ", ".join(
        f"{k} {v.get('per_s', v.get('TFLOPs', v.get('mixed_over_sum'))):.3g}"
        + (f" ({v['lanes_per_clk_per_simd']:.1f}/clk at {v['clock_ghz']:.2f} GHz)" if "lanes_per_clk_per_simd" in v else "")
        for k, v in res.items()), file=sys.stderr, flush=True)
    return res


def compute_factor_sweep(stream) -> dict:
    """Fused (K = 100) against unfused (K = 1) as the compute factor C grows:
    65,536 envs x 100 steps, each step C Euler iterations of tau / C."""
    from paper_2207_07736_amd import Simulator, Trajectory
    w = workloads.C_SWEEP
    n, T = w["n"], w["T"]
    rows = {}
    for C in w["C"]:
        sim = Simulator(n, 0, workloads.cartpole(compute_factor=C), stream=stream)
        sim.reset(w["seed"])
        traj = Trajectory(T, n)
        entry = {}
        for K in w["K"]:
            ms = _time_schedule(sim, traj, [K] * (T // K), stream, reps=2)
            entry[f"K{K}"] = {"ms": ms, "env_steps_per_s": n * T / (ms * 1e-3)}
        entry["fusion_speedup"] = entry["K1"]["ms"] / entry[f"K{T}"]["ms"]
        rows[f"C{C}"] = entry
        del traj
        sim.close()
    print("[bench] compute-factor sweep: " + ", ".join(f"{k} {v['fusion_speedup']:.2f}x" for k, v in rows.items()),
          file=sys.stderr, flush=True)
    return rows


def k_sweep(stream) -> dict:
    """Fused against unfused on the K sweep (65,536 envs x 1,000 steps, K = 1,
    10, 100, 1,000; three timed repetitions after one warm-up each), then the
    1,000 K = 1 launches captured in one HIP graph and replayed (one warm-up,
    three timed)."""
    from paper_2207_07736_amd import Simulator, Trajectory
    w = workloads.WORKLOADS[workloads.K_SWEEP]
    n, T = w["n"], w["T"]
    sim = Simulator(n, 0, workloads.CARTPOLE, stream=stream)
    sim.reset(w["seed"])
    traj = Trajectory(T, n)
    rows = {}
    for K in w["K"]:
        ms = _time_schedule(sim, traj, [K] * (T // K), stream, reps=3)
        rows[str(K)] = {"ms": ms, "env_steps_per_s": n * T / (ms * 1e-3)}
    base = rows["1"]["ms"]
    for r in rows.values():
        r["speedup_vs_K1"] = base / r["ms"]
    gms = _graph_ms(sim, [traj.rows(k, 1) for k in range(T)], stream, 3)
    rows["1_hipgraph"] = {"ms": gms, "env_steps_per_s": n * T / (gms * 1e-3), "speedup_vs_K1": base / gms}
    del traj
    sim.close()
    return rows


def sweep_only(which: str) -> int:
    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    stream = torch.cuda.Stream()
    torch.cuda.set_stream(stream)
    if which == "ksweep":
        rows = {workloads.WORKLOADS[workloads.K_SWEEP]["name"]: k_sweep(stream)}
    elif which == "chain":
        rows = {workloads.CHAIN_SWEEP["name"]: chain_sweep(stream)}
    elif which == "issue":
        rows = {"issue_rates": issue_rates(stream)}
    else:
        rows = {workloads.C_SWEEP["name"]: compute_factor_sweep(stream)}
    print(json.dumps(rows), flush=True)
    return 0


MLP_FLOPS_PER_ENV_STEP = 2 * (64 * 4 + 64 * 64 + 2 * 64)


def policy_only(dtype: str, steps: int, warmup: int) -> int:
    """Timed runs of the MLP-policy workload alone (for profiling): each run is
    the 256 steps of 1,048,576 envs in 16 launches of K = 16."""
    import torch
    from paper_2207_07736_amd import RLSIM_BF16, RLSIM_F32, Simulator, Trajectory, policy_struct
    w = workloads.WORKLOADS[workloads.MLP]
    n, T, K = w["n"], w["T"], w["K"][0]
    stream = torch.cuda.current_stream()
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    wts = workloads.mlp_weights(w["seed"])
    keep = {k: (torch.from_numpy(v).cuda().to(tdt) if k.startswith("w") else torch.from_numpy(v).cuda()).contiguous()
            for k, v in wts.items()}
    pol = policy_struct(RLSIM_BF16 if dtype == "bf16" else RLSIM_F32, keep["w1"], keep["b1"], keep["w2"], keep["b2"],
                        keep["w3"], keep["b3"])
    sim = Simulator(n, 0, workloads.CARTPOLE, stream=stream)
    sim.reset(w["seed"])
    traj = Trajectory(T, n)
    structs = [traj.rows(k0, K) for k0 in range(0, T, K)]
    for _ in range(warmup):
        for st in structs:
            sim.step(K, st, policy=pol)
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for _ in range(steps):
        for st in structs:
            sim.step(K, st, policy=pol)
    stop.record(stream)
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / steps
    print(json.dumps({"workload": w["name"], "dtype": dtype, "ms_per_run": ms, "launch_ms": ms / len(structs),
                      "env_steps_per_s": n * T / (ms * 1e-3),
                      "mlp_TFLOPs": n * T * MLP_FLOPS_PER_ENV_STEP / (ms * 1e-3) / 1e12}), flush=True)
    del traj
    sim.close()
    return 0


def wide_only(D: int, steps: int, warmup: int, copy_calibration: bool = False) -> int:
    """Timed K = 500 launches of the state-size workload alone (for profiling):
    262,144 envs x 500 steps with D padding words, trajectory recorded; with
    copy_calibration, then one plain device copy that calibrates the HBM byte
    counters."""
    import torch
    from paper_2207_07736_amd import Simulator, Trajectory
    w = workloads.WORKLOADS[workloads.STATE_SWEEP]
    n, T = w["n"], w["T"]
    stream = torch.cuda.current_stream()
    sim = Simulator(n, D, workloads.CARTPOLE, stream=stream)
    sim.reset(w["seed"])
    traj = Trajectory(T, n)
    rows = traj.rows(0, T)
    for _ in range(warmup):
        sim.step(T, rows)
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for _ in range(steps):
        sim.step(T, rows)
    stop.record(stream)
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / steps
    updates = n * D * T
    print(json.dumps({"workload": w["name"], "D": D, "K": T, "ms_per_launch": ms,
                      "env_steps_per_s": n * T / (ms * 1e-3),
                      "padding_updates_per_s": updates / (ms * 1e-3),
                      "valu_frac": updates / (ms * 1e-3) / VALU_LANE_OPS_PER_S}), flush=True)
    del traj
    sim.close()
    if copy_calibration:
        copy_for_calibration()
    return 0


FILL_SHAPES = (1, 4, 64, 275, 1024)     # float4 stores per thread; 275: a trajectory workgroup's volume


def store_ceiling_only(steps: int) -> int:
    """The headline's store ceiling against plain fills (for counters): the
    store-only probe writing the 4,194,304-env x 200-row trajectory (seven
    planes per row, byte planes first), then torch's fill of one contiguous
    buffer of the same 18.45 GB, then the fill probe over that buffer with
    FILL_SHAPES float4 stores per thread, then the headline launch itself, each
    `steps` times, with the per-launch times printed."""
    import torch
    from paper_2207_07736_amd import Simulator, Trajectory
    from paper_2207_07736_amd.probe import probe_fill, probe_store
    w = workloads.WORKLOADS[workloads.HEADLINE]
    n, T = w["n"], w["T"]
    stream = torch.cuda.current_stream()
    traj = Trajectory(T, n)
    out = {}

    def timed(name, fn):
        fn()
        torch.cuda.synchronize()
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record(stream)
        for _ in range(steps):
            fn()
        stop.record(stream)
        torch.cuda.synchronize()
        out[name] = start.elapsed_time(stop) / steps

    timed("store_probe_ms", lambda: probe_store(n, T, traj.obs, traj.action, traj.reward, traj.done, stream))
    flat = torch.empty(n * T * workloads.TRAJ_BYTES_PER_ENV_STEP // 4, dtype=torch.float32, device="cuda")
    timed("plain_fill_ms", lambda: flat.fill_(1.0))
    for per in FILL_SHAPES:
        timed(f"fill_probe_{per}_per_thread_ms", lambda per=per: probe_fill(flat, per, stream))
    del flat
    sim = Simulator(n, 0, workloads.CARTPOLE, stream=stream)
    sim.reset(w["seed"])
    rows = traj.rows(0, T)
    timed("headline_ms", lambda: sim.step(T, rows))
    sim.close()
    del traj
    b = n * T * workloads.TRAJ_BYTES_PER_ENV_STEP
    out.update({k.replace("_ms", "_TBs"): b / (v * 1e-3) / 1e12 for k, v in list(out.items())})
    print(json.dumps({"workload": w["name"], "bytes": b, **out}), flush=True)
    return 0


def copy_for_calibration() -> None:
    """One plain device copy of COPY_BYTES: what the HBM byte counters read for
    it scales their readings of the kernels."""
    import torch
    src = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


def chain_only(N: int, steps: int, warmup: int, copy_calibration: bool = False) -> int:
    """Timed K = 200 launches of the chain workload alone (for profiling):
    1,048,576 envs x 200 steps of the N-link chain, trajectory recorded."""
    import torch
    from paper_2207_07736_amd import Simulator, Trajectory
    w = workloads.CHAIN_SWEEP
    n, T = w["n"], w["T"]
    stream = torch.cuda.current_stream()
    sim = Simulator(n, 0, workloads.CARTPOLE, stream=stream, links=N)
    sim.reset(w["seed"])
    traj = Trajectory(T, n, S=sim.S)
    rows = traj.rows(0, T)
    for _ in range(warmup):
        sim.step(T, rows)
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for _ in range(steps):
        sim.step(T, rows)
    stop.record(stream)
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / steps
    algo = n * T * workloads.chain_traj_bytes_per_env_step(N) + (4 * sim.S + 4) * n * 2 + 16 * ((n + 255) // 256)
    print(json.dumps({"workload": w["name"], "N": N, "K": T, "ms_per_launch": ms,
                      "env_steps_per_s": n * T / (ms * 1e-3), "algorithmic_bytes_per_launch": algo,
                      "algorithmic_GBs": algo / (ms * 1e-3) / 1e9,
                      "TFLOPs": n * T * chain_flops_per_step(N) / (ms * 1e-3) / 1e12}), flush=True)
    del traj
    sim.close()
    if copy_calibration:
        copy_for_calibration()
    return 0


def unfused_only(steps: int, warmup: int, copy_calibration: bool) -> int:
    """Timed runs of the headline workload in its unfused form alone (for
    profiling): 4,194,304 envs x 200 steps as 200 launches of K = 1, the state
    read from and written to HBM at every step."""
    import torch
    from paper_2207_07736_amd import Simulator, Trajectory
    w = workloads.WORKLOADS[workloads.HEADLINE]
    n, T = w["n"], w["T"]
    stream = torch.cuda.current_stream()
    sim = Simulator(n, 0, workloads.CARTPOLE, stream=stream)
    sim.reset(w["seed"])
    traj = Trajectory(T, n)
    rows = [traj.rows(k, 1) for k in range(T)]
    for _ in range(warmup):
        for st in rows:
            sim.step(1, st)
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for _ in range(steps):
        for st in rows:
            sim.step(1, st)
    stop.record(stream)
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / steps
    algo = n * T * (workloads.TRAJ_BYTES_PER_ENV_STEP + 40) + T * (n // 256) * 16
    print(json.dumps({"workload": w["name"] + " as 200 launches of K = 1", "ms_per_run": ms, "launch_ms": ms / T,
                      "env_steps_per_s": n * T / (ms * 1e-3), "algorithmic_bytes_per_launch": algo // T,
                      "algorithmic_GBs": algo / (ms * 1e-3) / 1e9}), flush=True)
    del traj
    sim.close()
    if copy_calibration:
        copy_for_calibration()
    return 0


def policy_sweep(stream) -> dict:
    """The MLP-policy workload: 1,048,576 envs x 256 steps, fused K = 16 against
    unfused K = 1, fp32 and bf16 weights ~ N(0, 1/fan_in), zero biases; and K =
    16 again with the value head and the learner planes (log pi, value)
    recorded."""
    from paper_2207_07736_amd import RLSIM_BF16, RLSIM_F32, Simulator, Trajectory, policy_struct
    import torch
    w = workloads.WORKLOADS[workloads.MLP]
    n, T = w["n"], w["T"]
    wts = workloads.mlp_weights(w["seed"])
    rows = {}
    for dtype in ("f32", "bf16"):
        tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
        dev = {k: torch.from_numpy(v).to("cuda") for k, v in wts.items()}
        keep = {k: (dev[k].to(tdt) if k.startswith("w") else dev[k]).contiguous() for k in dev}
        code = RLSIM_BF16 if dtype == "bf16" else RLSIM_F32
        pol_plain = policy_struct(code, keep["w1"], keep["b1"], keep["w2"], keep["b2"], keep["w3"], keep["b3"])
        pol_value = policy_struct(code, keep["w1"], keep["b1"], keep["w2"], keep["b2"], keep["w3"], keep["b3"],
                                  keep["wv"], keep["bv"])
        sim = Simulator(n, 0, workloads.CARTPOLE, stream=stream)
        sim.reset(w["seed"])
        traj = Trajectory(T, n, learner=True)
        entry = {}
        for K, learner in ((16, False), (1, False), (16, True)):
            pol = pol_value if learner else pol_plain
            structs = [traj.rows(k0, K) for k0 in range(0, T, K)]
            if not learner:
                for st in structs:
                    st.logp = st.value = None
            times = []
            for r in range(5):
                start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                start.record(stream)
                for st in structs:
                    sim.step(K, st, policy=pol)
                stop.record(stream)
                torch.cuda.synchronize()
                if r:
                    times.append(start.elapsed_time(stop))
            ms = min(times)
            entry[f"K{K}" + ("_learner" if learner else "")] = {
                "ms": ms, "env_steps_per_s": n * T / (ms * 1e-3),
                "mlp_TFLOPs": n * T * MLP_FLOPS_PER_ENV_STEP / (ms * 1e-3) / 1e12}
        entry["fusion_speedup"] = entry["K1"]["ms"] / entry["K16"]["ms"]
        entry["learner_outputs_cost"] = entry["K16_learner"]["ms"] / entry["K16"]["ms"] - 1.0
        rows[dtype] = entry
        del traj
        sim.close()
        print(f"[bench] policy {dtype}: K16 {entry['K16']['ms']:.2f} ms, K1 {entry['K1']['ms']:.2f} ms, "
              f"K16 + log pi/value {entry['K16_learner']['ms']:.2f} ms", file=sys.stderr, flush=True)
    return rows


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    ap.add_argument("--no-unfused", action="store_true", help="skip the K=1 contrast")
    ap.add_argument("--no-sweep", action="store_true", help="skip the K and state-size sweeps")
    ap.add_argument("--cpu-slice-envs", type=int, default=65536)
    ap.add_argument("--cpu-slices", type=int, default=8)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run one plain device copy of 1 GiB (HBM counter calibration)")
    ap.add_argument("--policy", choices=("f32", "bf16"),
                    help="time only the MLP-policy workload (K = 16 launches) in this precision")
    ap.add_argument("--unfused", action="store_true",
                    help="time only the headline workload as 200 launches of K = 1 (profiling)")
    ap.add_argument("--wide", type=int, metavar="D",
                    help="time only the state-size workload (262,144 envs, K = 500) with D padding words")
    ap.add_argument("--store-ceiling", action="store_true",
                    help="time the headline's store-only probe, a plain fill of the same bytes and the headline "
                         "launch (for counters)")
    ap.add_argument("--chain", type=int, metavar="N",
                    help="time only the chain workload (1,048,576 envs, K = 200) with N links")
    ap.add_argument("--ingest-pmc", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write the HBM traffic summary from two rocprofv3 counter CSVs and exit")
    ap.add_argument("--sweep-only", choices=("ksweep", "csweep", "chain", "issue"),
                    help="run only the K sweep with its HIP-graph form (65,536 envs x 1,000 steps) or only "
                         "the compute-factor sweep, print its rows as JSON (profiling)")
    args = ap.parse_args()
    if args.sweep_only:
        return sweep_only(args.sweep_only)

    if args.policy:
        return policy_only(args.policy, args.steps, args.warmup)
    if args.wide:
        return wide_only(args.wide, args.steps, args.warmup, args.copy_calibration)
    if args.chain:
        return chain_only(args.chain, args.steps, args.warmup, args.copy_calibration)
    if args.store_ceiling:
        return store_ceiling_only(args.steps)
    if args.unfused:
        return unfused_only(args.steps, args.warmup, args.copy_calibration)

    if args.ingest_pmc:
        w = workloads.WORKLOADS[workloads.HEADLINE]
        print(ingest_pmc(args.ingest_pmc[0], args.ingest_pmc[1], w["name"], HEADLINE_KERNEL_PREFIX))
        return 0

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}): the environments shard by range with no "
              "communication, so a multi-GPU figure is N times the one-GPU figure and is not measured here.",
              file=sys.stderr)
        return 2

    import torch
    from paper_2207_07736_amd import Simulator, Trajectory

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    torch.cuda.set_device(0)
    w = workloads.WORKLOADS[workloads.HEADLINE]
    n, T, K = w["n"], w["T"], w["K"][0]
    seed = w["seed"]
    # one side stream for every launch and every timing event (graph capture
    # needs a stream other than the legacy default one)
    stream = torch.cuda.Stream()
    torch.cuda.set_stream(stream)

    sim = Simulator(n, 0, workloads.CARTPOLE, stream=stream)
    sim.reset(seed)
    traj = Trajectory(T, n)
    rows = traj.rows(0, K)
    print(f"[bench] workload {w['name']}: n={n} T={T} K={K} warmup={args.warmup} steps={args.steps}",
          file=sys.stderr, flush=True)

    for _ in range(args.warmup):
        sim.step(K, rows)
    torch.cuda.synchronize()

    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_wall = time.perf_counter()
    start.record(stream)
    for _ in range(args.steps):
        sim.step(K, rows)           # exactly one kernel launch
    stop.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_wall
    ms_total = start.elapsed_time(stop)
    ms_per_step = ms_total / args.steps
    env_steps_per_s = n * T / (ms_per_step * 1e-3)

    # Algorithmic bytes per launch: the trajectory (22 B per env-step), the
    # state read and written once (4 x f32 + u32 episode counter, each way) and
    # 16 B of block statistics per 256 envs.
    algo_bytes = n * T * workloads.TRAJ_BYTES_PER_ENV_STEP + n * 2 * 20 + (n // 256) * 16
    achieved_gbs = algo_bytes / (ms_per_step * 1e-3) / 1e9
    traffic = stored_traffic(w["name"])

    result = {
        "metric": METRIC,
        "value": env_steps_per_s,
        "unit": "env-steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (device Philox draws from seed 0)",
        "config": {"workload": w["name"], "n_envs": n, "steps_per_run": T, "steps_per_launch": K,
                   "padding_words": 0, "policy": "random", "trajectory": "obs f32x4, action u8, reward f32, done u8"},
        "roofline": {"bound": "hbm", "achieved": achieved_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved_gbs / HBM_PEAK_GBS, "traffic": traffic,
                     "kernel": HEADLINE_KERNEL, "algorithmic_bytes_per_launch": algo_bytes},
        "wall_s_timed_region": wall,
    }

    if not args.no_unfused:
        # the same 200 steps as 200 launches of K = 1 (state to and from HBM every step)
        sim.reset(seed)
        row_structs = [traj.rows(k, 1) for k in range(T)]      # marshalled before timing
        for k in range(T):
            sim.step(1, row_structs[k])
        torch.cuda.synchronize()
        reps = 3
        start.record(stream)
        for _ in range(reps):
            for k in range(T):
                sim.step(1, row_structs[k])
        stop.record(stream)
        torch.cuda.synchronize()
        unfused_ms = start.elapsed_time(stop) / reps
        graph_ms = _graph_ms(sim, row_structs, stream, reps)
        result["fusion"] = {"unfused_K1_ms": unfused_ms, "unfused_K1_hipgraph_ms": graph_ms, "fused_K200_ms": ms_per_step,
                            "speedup": unfused_ms / ms_per_step,
                            "speedup_over_hipgraph": graph_ms / ms_per_step,
                            "unfused_algorithmic_GBs": (n * T * (workloads.TRAJ_BYTES_PER_ENV_STEP + 40)) / (unfused_ms * 1e-3) / 1e9}

    # the store ceiling: the same trajectory bytes, layout and launch shape with
    # the simulation taken out (librlsim_probe.so), timed like the headline
    from paper_2207_07736_amd.probe import probe_store
    for _ in range(2):
        probe_store(n, K, traj.obs, traj.action, traj.reward, traj.done, stream)
    torch.cuda.synchronize()
    start.record(stream)
    for _ in range(args.steps):
        probe_store(n, K, traj.obs, traj.action, traj.reward, traj.done, stream)
    stop.record(stream)
    torch.cuda.synchronize()
    probe_ms = start.elapsed_time(stop) / args.steps
    traj_bytes = n * T * workloads.TRAJ_BYTES_PER_ENV_STEP
    result["roofline"]["store_probe"] = {
        "ms": probe_ms, "GBs": traj_bytes / (probe_ms * 1e-3) / 1e9,
        "frac_of_store_ceiling": (traj_bytes / ms_per_step) / (traj_bytes / probe_ms)}

    del traj
    sim.close()

    if args.copy_calibration:
        copy_for_calibration()

    if not args.no_sweep:
        result["sweeps"] = fusion_sweeps(stream)

    if not args.no_cpu:
        result["cpu_baseline"] = cpu_baseline(args.cpu_slice_envs, args.cpu_slices, T, seed)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
