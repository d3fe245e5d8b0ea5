"""Throughput of the MLIP energy/force/virial path on one MI355X.

A step is one velocity-Verlet NVE step of the whole path: half kick and drift,
a neighbour-list rebuild every 10 steps (or earlier when an atom has moved
more than skin/2), the fused energy/force/virial evaluation of every atom,
and the second half kick.  Inputs are resident in HBM before timing starts.

Default workload: 6-component equiatomic random FCC alloy, 128^3 cells =
8,388,608 atoms, a = 3.6 A, sigma = 0.1 A, cutoff 6.0 A, skin 0.5 A, k = 32,
l_max = 3, encoder 3 x 128, head 4 x 64, random N(0, 1/fan_in) weights with the
head's output layer scaled so forces are about 1 eV/A, as from a trained
potential near 300 K (the values change no work).

Prints one JSON line (rank 0, one GPU).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_TFLOPS = {64: 78.6, 32: 157.3}   # MI355X dense MFMA FP64 / FP32
PEAK_HBM_GBS = 8000.0
FUSED_SOURCE = os.path.join(ROOT, "paper_2608_16329_amd", "csrc", "fused.hip")


def traffic_summary_path(precision: int, fusion: str = "cached") -> str:
    tag = ("" if precision == 64 else "_f32") + ("" if fusion == "cached" else "_" + fusion)
    return os.path.join(ROOT, "profiles", f"k_fused{tag}_fcc-hea6-128_traffic.md")


def largest_system_run():
    """The largest system the committed capacity-sweep summary records as run
    on one GPU (atoms, bytes per atom), or None without that summary."""
    import re
    try:
        text = open(os.path.join(ROOT, "profiles", "capacity_sweep_bcc-hea6.md")).read()
    except OSError:
        return None
    m = re.search(r"Largest system run: ([\d,]+) atoms .*?, (\d+) bytes per atom", text)
    if not m:
        return None
    return {"atoms": int(m.group(1).replace(",", "")), "bytes_per_atom": int(m.group(2)),
            "source": "profiles/capacity_sweep_bcc-hea6.md (6-component BCC, totals only)"}


def fused_source_hash() -> str:
    import hashlib
    with open(FUSED_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def measured_traffic(workload: str, n_atoms: int, precision: int, fusion: str = "cached"):
    """HBM bytes per launch of the fused kernel from the committed rocprofv3
    FETCH_SIZE / WRITE_SIZE summary, scaled by the same counters on a plain
    copy of known size; None when the summary is for other kernel source,
    another workload, precision or fusion configuration."""
    try:
        with open(traffic_summary_path(precision, fusion)) as f:
            for line in f:
                if line.startswith("traffic_json:"):
                    t = json.loads(line.split(":", 1)[1])
                    if t["fused_source_sha256"] == fused_source_hash() and t["n_atoms"] == n_atoms \
                            and t["workload"] == workload and t.get("precision", 64) == precision \
                            and t.get("fusion", "cached") == fusion:
                        return t["traffic_bytes_per_launch"]
    except (OSError, KeyError, ValueError):
        pass
    return None


def flops_per_pair(hp) -> float:
    """Algorithmic FLOP per active pair: encoder forward and tangent
    (2 x 2 x MAC) plus the moment and the two W contractions (6 d k)."""
    W = hp.enc_width
    mac_enc = W + (hp.enc_hidden - 1) * W * W + W * hp.k
    if getattr(hp, "angular", 0) == 1:  # Cartesian monomials: (l+1)(l+2)/2 per order
        d = sum((l + 1) * (l + 2) // 2 for l in range(hp.lmax + 1))
    else:                               # irreducible harmonics: 2l+1 per order
        d = (hp.lmax + 1) ** 2
    return 4.0 * mac_enc + 6.0 * d * hp.k


def flops_per_atom(hp) -> float:
    """Algorithmic FLOP per atom for the energy head forward and backward."""
    R = hp.reg_width
    mac_head = (hp.lmax + 1) * hp.k * R + (hp.reg_hidden - 1) * R * R + R
    return 4.0 * mac_head


def summarize_traffic(fetch_dir: str, write_dir: str, bench_log: str, copy_bytes: int, command: str) -> None:
    """Write the traffic summary of the fused kernel from two rocprofv3 --pmc
    runs (FETCH_SIZE, then WRITE_SIZE, KiB per dispatch).  Each counter is
    scaled by what it reads for the calibration copy of copy_bytes bytes in
    the same run; the result is HBM-side (L2-to-fabric) bytes per launch."""
    import csv
    import glob

    def read(d, counter):
        path = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)[0]
        copy_vals, fused_vals = [], []
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            v = float(r["Counter_Value"])
            if "copyBuffer" in r["Kernel_Name"]:
                copy_vals.append(v)
            elif "k_fused" in r["Kernel_Name"]:
                fused_vals.append(v)
        return max(copy_vals), fused_vals

    fc, ff = read(fetch_dir, "FETCH_SIZE")
    wc, wf = read(write_dir, "WRITE_SIZE")
    f_scale = copy_bytes / (fc * 1024.0)
    w_scale = copy_bytes / (wc * 1024.0)
    fetch_b = float(np.mean(ff)) * 1024.0 * f_scale
    write_b = float(np.mean(wf)) * 1024.0 * w_scale
    b = None
    for line in open(bench_log):
        if line.startswith("{"):
            b = json.loads(line)
    precision = b["config"].get("precision", 64)
    fusion = b["config"].get("fusion", "cached")
    t = {"fused_source_sha256": fused_source_hash(), "workload": b["config"]["workload"],
         "n_atoms": b["config"]["n_atoms"], "precision": precision, "fusion": fusion,
         "fetch_kib_per_launch": float(np.mean(ff)),
         "write_kib_per_launch": float(np.mean(wf)), "copy_bytes": copy_bytes, "copy_fetch_kib": fc,
         "copy_write_kib": wc, "fetch_scale": f_scale, "write_scale": w_scale,
         "traffic_bytes_per_launch": fetch_b + write_b, "launches": len(ff)}
    with open(traffic_summary_path(precision, fusion), "w") as f:
        f.write(f"# HBM-side traffic of the fused energy/force/virial kernel (float{precision} network, "
                f"{fusion} configuration), 6-component FCC 128^3\n\n")
        f.write("Two rocprofv3 counter runs of the same command (one counter per run), from the repository\n"
                "root on the GPU host:\n\n")
        for ctr in ("FETCH_SIZE", "WRITE_SIZE"):
            f.write(f"    cd /tmp && export TMPDIR=/tmp && timeout -s KILL 240 rocprofv3 --pmc {ctr} --kernel-trace \\\n"
                    f"        -d <output-dir> -o run --output-format csv -- {command}\n\n")
        f.write(f"Calibration: the command first copies {copy_bytes} bytes device-to-device; that copy read "
                f"FETCH_SIZE = {fc:.0f} KiB and WRITE_SIZE = {wc:.0f} KiB, so fetch counts are scaled by "
                f"{f_scale:.3f} and write counts by {w_scale:.3f}.\n\n")
        f.write(f"Fused kernel, mean over {len(ff)} launches: FETCH_SIZE {np.mean(ff):.4g} KiB, WRITE_SIZE "
                f"{np.mean(wf):.4g} KiB; scaled traffic {fetch_b / 1e9:.1f} GB read + {write_b / 1e9:.1f} GB "
                f"written = {(fetch_b + write_b) / 1e9:.1f} GB per launch "
                f"({(fetch_b + write_b) / b['config']['n_atoms']:.0f} B per atom).\n\n")
        if fusion == "cached":
            ws = 2 * 2 * b["config"]["k"] * (precision // 8) * b["config"]["active_pairs_per_atom"]
            f.write(f"Most of it is the per-pair (m, dm) workspace that pass 1 writes and pass 2 reads back: 2k values "
                    f"per active pair each way, {ws:.0f} B per atom at {b['config']['active_pairs_per_atom']:.2f} active "
                    f"pairs per atom; the per-work-group workspace (about a megabyte per tile) does not stay in the 4 MB "
                    f"L2 of an XCD between the two passes. The rest "
                    f"({(fetch_b + write_b) / b['config']['n_atoms'] - ws:.0f} B per atom) is neighbour positions, "
                    f"neighbour-list entries, weights missing L2, and outputs. ")
        else:
            f.write("This configuration keeps no workspace: the traffic is neighbour positions, neighbour-list "
                    "entries, encoder weights missing L2, and the outputs. ")
        atomics = 3.0 * b["config"]["active_pairs_per_atom"] * b["config"]["n_atoms"]
        f.write(f"WRITE_SIZE counts each float64 atomic add of the force scatter (F_j -= f_ij, three per active "
                f"pair, {atomics:.3g} per launch) as a 32-byte write, {32 * atomics / 1e9:.1f} GB of the written "
                f"figure, although each carries 8 bytes. ")
        f.write("The counters see L2-to-fabric requests, which include Infinity Cache hits: no counter of this "
                "part separates Infinity Cache hits from HBM accesses.\n\n")
        f.write("traffic_json: " + json.dumps(t) + "\n")
    print(json.dumps(t))


def neighbour_build_record(events, first_ms: float, n_atoms: int, n_listed: int,
                           entry_bytes: int) -> dict:
    """Time and bandwidth of the neighbour-list build: HIP events around the
    rebuilds of the timed steps (the first build's wall time when none fell
    there).  Algorithmic bytes: positions and species read (28 B per atom),
    cell keys, permutation, sorted positions, row counts and int64 offsets
    written (44 B per atom), one entry (2 B coded, 4 B as an index) per listed
    pair written; candidate positions are re-read from cache and not counted."""
    ms = float(np.mean([a.elapsed_time(b) for a, b in events])) if events else first_ms
    nbytes = 72.0 * n_atoms + float(entry_bytes) * n_listed
    return {"ms": ms, "timed_rebuilds": len(events), "algorithmic_bytes": nbytes,
            "gbps": nbytes / (ms * 1e-3) / 1e9, "frac_of_hbm": nbytes / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS,
            "bound": "candidate scan (27 cells, about 500 distance tests per atom, twice)"}


def capacity_sweep(edges, steps: int, seed: int, bpa: float = 450.0, precision: int = 64) -> None:
    """6-component equiatomic random BCC alloy (a = 3.2 A, sigma = 0.1 A,
    cutoff 6 A) at growing supercell edges L; "max" picks the largest L the
    free device memory holds at the bytes per atom measured at the previous
    edge.  Energies and virials are reduced to totals only; the skin guard
    measures displacement against the library's build-time positions.  One
    JSON line per edge."""
    import torch
    import synth
    from paper_2608_16329_amd import Potential
    p = synth.PRESETS["bcc-hea6-sweep"]
    dev = torch.device("cuda:0")
    torch.cuda.init()
    for e in edges:
        torch.cuda.empty_cache()
        free0, total = torch.cuda.mem_get_info(dev)
        if e == "max":
            L = int(((0.93 * free0 / bpa) / 2.0) ** (1.0 / 3.0))
        else:
            L = int(e)
        N = 2 * L ** 3
        if N * bpa > 0.985 * free0:
            print(json.dumps({"sweep_edge": L, "n_atoms": N, "fits": False}), flush=True)
            continue
        hp = synth.HParams(n_species=p["C"], cutoff=p["cutoff"], skin=0.5, precision=precision)
        weights = synth.random_weights(hp, seed + 1, energy_scale=synth.PHYSICAL_ENERGY_SCALE)
        masses = np.array([synth.MASS[x] for x in p["masses"]])
        box = np.array([L * p["a"]] * 3)
        t0 = time.perf_counter()
        pos = torch.empty((N, 3), dtype=torch.float64, device=dev)
        vel = torch.empty((N, 3), dtype=torch.float64, device=dev)
        types = torch.empty(N, dtype=torch.int32, device=dev)
        F = torch.zeros((N, 3), dtype=torch.float64, device=dev)
        for first, cp, ct, cv in synth.lattice_stream("bcc", L, p["a"], p["C"], p["sigma"], masses, p["T"], seed):
            m = len(cp)
            if (first // m) % 8 == 0:
                log(f"[sweep] L={L}: generating, {first}/{N} sites")
            pos[first:first + m] = torch.from_numpy(cp).to(dev)
            vel[first:first + m] = torch.from_numpy(cv).to(dev)
            types[first:first + m] = torch.from_numpy(ct).to(dev)
        torch.cuda.synchronize()
        log(f"[sweep] L={L} N={N}: generated in {time.perf_counter() - t0:.1f}s")
        pot = Potential(hp, weights)
        pot.set_masses(masses)
        tb = time.perf_counter()
        pot.build_neighbors(pos, types, box)
        torch.cuda.synchronize()
        t_build = time.perf_counter() - tb
        pot.compute(pos, F)
        torch.cuda.synchronize()
        free1, _ = torch.cuda.mem_get_info(dev)
        used = free0 - free1
        bpa = used / N
        log(f"[sweep] L={L}: build {t_build:.2f}s, {bpa:.0f} B/atom")
        rebuilds = 0
        step = 0
        kern = []
        stream = torch.cuda.current_stream()

        def md_step(record):
            nonlocal step, rebuilds
            step += 1
            d2 = pot.md_first_half(pos, vel, F, 1.0, track=True)
            if step % 10 == 0 or d2 > 0.0625:
                pot.build_neighbors(pos, types, box)
                rebuilds += 1
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            pot.compute(pos, F)
            e1.record(stream)
            if record:
                kern.append((e0, e1))
            pot.md_second_half(vel, F, 1.0)

        if N < 200_000_000:   # at the largest sizes one step takes minutes: no warm-up step
            md_step(False)
            torch.cuda.synchronize()
            log(f"[sweep] L={L}: warm-up step done")
        rebuilds = 0
        t0 = time.perf_counter()
        for k in range(steps):
            md_step(True)
            torch.cuda.synchronize()
            log(f"[sweep] L={L}: step {k + 1}/{steps} {time.perf_counter() - t0:.1f}s")
        wall = time.perf_counter() - t0
        st = pot.stats()
        print(json.dumps({"sweep_edge": L, "n_atoms": N, "fits": True, "steps": steps, "precision": precision,
                          "atom_steps_per_s": N * steps / wall, "ms_per_step": wall / steps * 1e3,
                          "fused_kernel_ms": float(np.mean([a.elapsed_time(b) for a, b in kern])),
                          "hbm_bytes_per_atom": bpa, "library_bytes_per_atom": pot.memory_bytes() / N,
                          "device_total_bytes": total, "rebuilds_in_timed_steps": rebuilds,
                          "build_s": t_build, "listed_pairs_per_atom": st["n_listed_pairs"] / N,
                          "active_pairs_per_atom": st["n_active_pairs"] / N,
                          "list_entry_bytes": st["list_entry_bytes"],
                          "max_atoms_estimate": int(0.97 * total / bpa)}), flush=True)
        pot.close()
        del pos, vel, types, F


def recompute_record(pot, pos, F, E, V, stream, evals: int, flop: float, N: int, w, precision: int) -> dict:
    """The recompute configuration (one kernel, the encoder evaluated again in
    pass 2 instead of parked in a workspace: nothing but the outputs goes to
    HBM) at the final positions of the timed steps: HIP-event time of
    `evals` evaluations after one untimed, the same algorithmic FLOP."""
    import torch
    pot.set_fusion(1)
    lib_bytes = pot.memory_bytes()
    pot.compute(pos, F, E, V)
    ev = []
    for _ in range(evals):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        pot.compute(pos, F, E, V)
        e1.record(stream)
        ev.append((e0, e1))
    torch.cuda.synchronize()
    pot.set_fusion(0)
    ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))
    achieved = flop / (ms * 1e-3) / 1e12
    traffic = measured_traffic(w.description, N, precision, "recompute")
    log(f"[bench] recompute configuration: {ms:.1f} ms per evaluation")
    return {"fusion": "recompute", "evaluations": evals, "kernel_ms": ms, "atom_evals_per_s": N / (ms * 1e-3),
            "achieved": achieved, "peak": PEAK_TFLOPS[precision], "unit": "TFLOP/s",
            "frac": achieved / PEAK_TFLOPS[precision], "traffic": traffic,
            "traffic_gbps": traffic / (ms * 1e-3) / 1e9 if traffic else None,
            "library_bytes_per_atom": lib_bytes / N}


def log(msg: str) -> None:
    print(msg, file=sys.stderr, flush=True)


def _oracle_worker(args):
    import threadpoolctl
    with threadpoolctl.threadpool_limits(1):
        from oracle.model import Model, evaluate
        hp, weights, pos, types, box, off, idx, centres = args
        m = Model(hp, weights)
        t0 = time.perf_counter()
        evaluate(m, pos, types, box, off, idx, centres=centres)
        return time.perf_counter() - t0


def cpu_baseline(w, target_atoms: int) -> dict:
    """Oracle timed on this host's cores on a bounded sample of the workload:
    the centre atoms inside a cube of the supercell, with neighbours taken
    from the surrounding atoms (evaluation only, no neighbour search)."""
    import multiprocessing as mp
    from oracle.neighbors import cell_list_neighbors

    rl = w.hp.cutoff + w.hp.skin
    box = w.box
    d = w.pos - box / 2.0
    d -= box * np.round(d / box)
    rho = len(w.pos) / float(np.prod(box))
    half = 0.5 * (target_atoms / rho) ** (1.0 / 3.0)
    reach = half + rl + 0.5
    inner = np.all(np.abs(d) < half, axis=1)
    outer = np.all(np.abs(d) < reach, axis=1)
    loc = np.nonzero(outer)[0]
    # local, non-periodic frame: a box wide enough that no periodic image is in range
    lbox = np.full(3, 2.0 * reach + 2.0 * rl)
    lpos = d[loc] + reach + rl
    ltypes = w.types[loc]
    centres = np.nonzero(inner[loc])[0]
    t_nbr = time.perf_counter()
    off, idx = cell_list_neighbors(lpos, lbox, rl)
    t_nbr = time.perf_counter() - t_nbr
    host_cores = len(os.sched_getaffinity(0))
    # one GPU's share of a GPU host: at most 16 processes, whatever the host has
    cores = min(16, host_cores)
    chunks = np.array_split(centres, cores)
    jobs = [(w.hp, w.weights, lpos, ltypes, lbox, off, idx, c) for c in chunks if len(c)]
    ctx = mp.get_context("fork")
    t0 = time.perf_counter()
    with ctx.Pool(len(jobs)) as pool:
        pool.map(_oracle_worker, jobs)
    wall = time.perf_counter() - t0
    return {"value": len(centres) / (wall + t_nbr), "unit": "atom-steps/s", "cores": len(jobs), "kind": "oracle",
            "cpu_model": host_cpu_model(), "host_cores": host_cores,
            "cores_cap": "16 processes, one GPU's share of the GPU host's cores",
            "evaluation_only_value": len(centres) / wall,
            "sample": f"{len(centres)} centre atoms of the same workload (a cube at the box centre), "
                      f"one E+F+virial evaluation each, float64 NumPy, {len(jobs)} processes x 1 BLAS "
                      f"thread, {wall:.1f} s wall, plus the oracle's cell-list neighbour search of the "
                      f"{len(lpos)}-atom region around it in one process, {t_nbr:.1f} s"}


def host_cpu_model() -> str:
    """The host CPU's model name (first processor in /proc/cpuinfo)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="fcc-hea6-128")
    ap.add_argument("--cells", type=int, default=None, help="supercell edge override (cells)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--precision", type=int, choices=(64, 32), default=64,
                    help="network arithmetic: 64 (float64) or 32 (float32 network, float64 geometry and sums)")
    ap.add_argument("--fusion", choices=("cached", "recompute", "partial", "unfused"), default="cached",
                    help="fusion configuration: one kernel caching the encoder output (default), one kernel "
                         "recomputing it, three kernels with the descriptor in HBM, or ten kernels (one per "
                         "equation) with every intermediate in HBM")
    ap.add_argument("--scatter", choices=("atomic", "tile"), default="atomic",
                    help="F_j scatter of the cached kernel: one atomic per pair (default) or summed per distinct "
                         "neighbour of a tile in LDS first")
    ap.add_argument("--list", choices=("auto", "index"), default="auto",
                    help="neighbour-list entries: 2-byte codes where the cell buckets allow (default) or 4-byte "
                         "indices")
    ap.add_argument("--hp", default="",
                    help="comma-separated hyper-parameter overrides, e.g. k=64,lmax=2,enc_cond=1")
    ap.add_argument("--rebuild-every", type=int, default=10)
    ap.add_argument("--recompute-evals", type=int, default=3,
                    help="after the timed steps of the cached configuration, time this many evaluations of the "
                         "recompute configuration (0 disables)")
    ap.add_argument("--cpu-sample", type=int, default=100000, help="oracle sample size (atoms); 0 disables")
    ap.add_argument("--calibrate-copy-bytes", type=int, default=0,
                    help="first run one device-to-device copy of this many bytes (counter calibration)")
    ap.add_argument("--sweep", default=None,
                    help="capacity sweep over comma-separated BCC supercell edges (or 'max') and exit")
    ap.add_argument("--sweep-steps", type=int, default=20)
    ap.add_argument("--sweep-bpa", type=float, default=450.0,
                    help="device bytes per atom assumed before the first edge is measured")
    ap.add_argument("--summarize-traffic", nargs=3, metavar=("FETCH_DIR", "WRITE_DIR", "BENCH_LOG"),
                    help="write the traffic summary from two rocprofv3 --pmc runs and exit")
    args = ap.parse_args()
    if args.sweep:
        capacity_sweep(args.sweep.split(","), args.sweep_steps, args.seed, args.sweep_bpa, args.precision)
        return 0
    if args.summarize_traffic:
        summarize_traffic(*args.summarize_traffic, copy_bytes=args.calibrate_copy_bytes or 2147483648,
                          command="python3 <repo>/bench.py --steps 1 --warmup 0 --cpu-sample 0 --recompute-evals 0 "
                                  f"--calibrate-copy-bytes 2147483648 --precision {args.precision} "
                                  f"--fusion {args.fusion}")
        return 0

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(spatial decomposition across GPUs is not implemented)", file=sys.stderr)
        return 2

    import torch
    import synth
    from paper_2608_16329_amd import Potential

    t_gen = time.perf_counter()
    overrides = {"precision": args.precision}
    for item in filter(None, args.hp.split(",")):
        key, val = item.split("=")
        overrides[key.strip()] = int(val)
    w = synth.make_workload(args.workload, seed=args.seed, n=args.cells, hp_overrides=overrides,
                            energy_scale=synth.PHYSICAL_ENERGY_SCALE)
    N = len(w.pos)
    log(f"[bench] workload {w.description}: N={N} generated in {time.perf_counter() - t_gen:.1f}s")
    dev = torch.device("cuda:0")
    torch.cuda.init()
    if args.calibrate_copy_bytes > 0:
        src = torch.ones(args.calibrate_copy_bytes // 8, dtype=torch.float64, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        log(f"[bench] calibration copy of {args.calibrate_copy_bytes} bytes done")
    free0, total_mem = torch.cuda.mem_get_info(dev)
    pos = torch.from_numpy(w.pos).to(dev)
    vel = torch.from_numpy(w.vel).to(dev)
    types = torch.from_numpy(w.types).to(dev)
    F = torch.zeros((N, 3), dtype=torch.float64, device=dev)
    E = torch.zeros(N, dtype=torch.float64, device=dev)
    V = torch.zeros((N, 9), dtype=torch.float64, device=dev)
    ref = pos.clone()
    stream = torch.cuda.current_stream()
    pot = Potential(w.hp, w.weights, stream=stream)
    pot.set_fusion({"cached": 0, "recompute": 1, "partial": 2, "unfused": 3}[args.fusion])
    pot.set_scatter({"atomic": 0, "tile": 1}[args.scatter])
    pot.set_list_format({"auto": 0, "index": 1}[args.list])
    pot.set_masses(w.masses)
    t0 = time.perf_counter()
    pot.build_neighbors(pos, types, w.box)
    torch.cuda.synchronize()
    t_build = time.perf_counter() - t0
    pot.compute(pos, F, E, V)
    torch.cuda.synchronize()
    free1, _ = torch.cuda.mem_get_info(dev)
    st = pot.stats()
    log(f"[bench] build {t_build * 1e3:.1f} ms; stats {st}")

    dt = w.dt
    skin2 = (0.5 * w.hp.skin) ** 2
    step_no = 0
    rebuilds = 0
    compute_ms = []
    rebuild_ms = []

    def md_step(timed: bool):
        nonlocal step_no, rebuilds
        step_no += 1
        d2 = pot.md_first_half(pos, vel, F, dt, ref)
        if step_no % args.rebuild_every == 0 or d2 > skin2:
            b0 = torch.cuda.Event(enable_timing=True)
            b1 = torch.cuda.Event(enable_timing=True)
            b0.record(stream)
            pot.build_neighbors(pos, types, w.box)
            b1.record(stream)
            if timed:
                rebuild_ms.append((b0, b1))
            ref.copy_(pos)
            rebuilds += 1
        if timed:
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            pot.compute(pos, F, E, V)
            e1.record(stream)
            compute_ms.append((e0, e1))
        else:
            pot.compute(pos, F, E, V)
        pot.md_second_half(vel, F, dt)

    for _ in range(args.warmup):
        md_step(False)
    torch.cuda.synchronize()
    rebuilds = 0
    active_pairs = []
    t0 = time.perf_counter()
    for k in range(args.steps):
        md_step(True)
        torch.cuda.synchronize()
        active_pairs.append(pot.stats()["n_active_pairs"])
        log(f"[bench] step {k + 1}/{args.steps} done, {time.perf_counter() - t0:.2f}s")
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    kern = [a.elapsed_time(b) for a, b in compute_ms]
    ms_compute = float(np.mean(kern))
    ms_median = float(np.median(kern))
    flop = float(np.mean(active_pairs)) * flops_per_pair(w.hp) + N * flops_per_atom(w.hp)
    achieved = flop / (ms_compute * 1e-3) / 1e12
    value = N * args.steps / wall
    st = pot.stats()
    lib_bytes = pot.memory_bytes()
    caller_bytes = N * (24 + 24 + 4 + 24 + 8 + 72 + 24)  # pos, vel, types, F, E, virial, ref
    used = free0 - free1
    bpa = used / N

    traffic = (measured_traffic(w.description, N, args.precision, args.fusion)
               if args.scatter == "atomic" and args.list == "auto" else None)
    recompute = None
    if args.fusion == "cached" and args.recompute_evals > 0 and w.hp.k == 32 and w.hp.lmax <= 3 \
            and w.hp.angular == 0:
        recompute = recompute_record(pot, pos, F, E, V, stream, args.recompute_evals, flop, N, w, args.precision)
        if args.list != "auto":   # the committed traffic summary was taken with the default list entries
            recompute["traffic"] = recompute["traffic_gbps"] = None
    result = {
        "metric": "atom-steps/s (E+F+virial) at 1 GPU",
        "value": value,
        "unit": "atom-steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64" if args.precision == 64 else "f32",
        "data": "synthetic",
        "config": {"workload": w.description, "n_atoms": N, "n_species": w.hp.n_species, "k": w.hp.k,
                   "lmax": w.hp.lmax, "cutoff": w.hp.cutoff, "skin": w.hp.skin, "dt_fs": dt,
                   "rebuild_every": args.rebuild_every, "rebuilds_in_timed_steps": rebuilds,
                   "head_output_scale": synth.PHYSICAL_ENERGY_SCALE,
                   "active_pairs_per_atom": float(np.mean(active_pairs)) / N,
                   "listed_pairs_per_atom": st["n_listed_pairs"] / N, "tile_atoms": st["tile_atoms"],
                   "blocks": st["n_blocks"], "seed": args.seed, "precision": args.precision,
                   "enc_cond": w.hp.enc_cond, "reg_cond": w.hp.reg_cond, "enc_hidden": w.hp.enc_hidden,
                   "reg_hidden": w.hp.reg_hidden, "fusion": args.fusion, "scatter": args.scatter,
                   "list_entry_bytes": st["list_entry_bytes"]},
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": PEAK_TFLOPS[args.precision], "unit": "TFLOP/s",
                     "frac": achieved / PEAK_TFLOPS[args.precision],
                     "traffic": traffic,
                     "traffic_gbps": traffic / (ms_compute * 1e-3) / 1e9 if traffic else None,
                     "kernel": {"cached": "fused energy/force/virial (k_fused)",
                                "recompute": "fused energy/force/virial (k_fused)",
                                "partial": "encoding + regression + derivation kernels (k_fused modes 2-4)",
                                "unfused": "ten kernels, one per equation (setup, radial, angular, moment, "
                                           "descriptor, regression, adjoint, U, V, force)"}[args.fusion],
                     "kernel_ms": ms_compute,
                     "algorithmic_flop_per_launch": flop},
        "compute_only_atom_evals_per_s": N / (ms_median * 1e-3),
        "recompute": recompute,
        "hbm_bytes_per_atom": bpa,
        "library_bytes_per_atom": lib_bytes / N,
        "caller_bytes_per_atom": caller_bytes / N,
        "max_atoms_estimate": int(0.95 * total_mem / bpa),   # at this workload's bytes per atom
        "max_atoms_run": largest_system_run(),
        "build_ms": t_build * 1e3,
        "neighbour_build": neighbour_build_record(rebuild_ms, t_build * 1e3, N, st["n_listed_pairs"],
                                                  st["list_entry_bytes"]),
    }
    if args.cpu_sample > 0:
        log("[bench] timing the oracle on a bounded sample")
        result["cpu_baseline"] = cpu_baseline(w, args.cpu_sample)
    pot.close()
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
