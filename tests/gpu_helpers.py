"""Shared helpers of the GPU tests: run the HIP path through the C ABI and
the oracle on the same seeded inputs."""
import sys

import numpy as np

import synth


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def torch_mod():
    import torch
    return torch


def to_dev(a, dtype=None):
    torch = torch_mod()
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.to("cuda:0").contiguous()


def gpu_eval(hp, weights, pos, types, box, want_energy=True, want_virial=True):
    """Build neighbours and evaluate once on the GPU; returns host arrays."""
    torch = torch_mod()
    from paper_2608_16329_amd import Potential
    pot = Potential(hp, weights)
    p = to_dev(pos, torch.float64)
    t = to_dev(types.astype(np.int32))
    pot.build_neighbors(p, t, box)
    n = len(pos)
    F = torch.empty((n, 3), dtype=torch.float64, device="cuda:0")
    E = torch.empty(n, dtype=torch.float64, device="cuda:0") if want_energy else None
    V = torch.empty((n, 9), dtype=torch.float64, device="cuda:0") if want_virial else None
    tot = pot.compute(p, F, E, V, totals=True)
    torch.cuda.synchronize()
    out = {"F": F.cpu().numpy(), "totals": tot, "stats": pot.stats(), "pot": pot}
    if want_energy:
        out["E_i"] = E.cpu().numpy()
    if want_virial:
        out["virial"] = V.cpu().numpy()
    return out


def sorted_rows(off, idx):
    return [np.sort(idx[off[i]:off[i + 1]]) for i in range(len(off) - 1)]


def assert_same_neighbor_sets(off_a, idx_a, off_b, idx_b):
    ra, rb = sorted_rows(off_a, idx_a), sorted_rows(off_b, idx_b)
    assert len(ra) == len(rb)
    for i, (x, y) in enumerate(zip(ra, rb)):
        if not np.array_equal(x, y):
            raise AssertionError(f"row {i}: gpu-only {sorted(set(x) - set(y))}, oracle-only {sorted(set(y) - set(x))}")


def max_abs(a, b):
    return float(np.max(np.abs(np.asarray(a) - np.asarray(b)))) if np.size(a) else 0.0
