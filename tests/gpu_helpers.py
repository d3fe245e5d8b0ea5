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


def gpu_eval(hp, weights, pos, types, box, want_energy=True, want_virial=True, fusion=0):
    """Build neighbours and evaluate once on the GPU (in the given fusion
    configuration); returns host arrays."""
    torch = torch_mod()
    from paper_2608_16329_amd import Potential
    pot = Potential(hp, weights)
    if fusion:
        pot.set_fusion(fusion)
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


def local_cluster(pos, types, box, atom, radius):
    """Atoms within `radius` of `atom` (minimum image), re-centred in a box
    wide enough that no periodic image is in range.  Returns the local
    positions, species, box and the local index of `atom`."""
    d = pos - pos[atom]
    d -= box * np.round(d / box)
    sel = np.nonzero((d * d).sum(1) < radius * radius)[0]
    lbox = np.full(3, 4.0 * radius + 10.0)
    lpos = d[sel] + lbox / 2.0
    return lpos, types[sel], lbox, int(np.nonzero(sel == atom)[0][0]), sel


def oracle_sample(model, pos, types, box, atoms):
    """Oracle E_i, F_i and virial of selected atoms of a large periodic
    system, each from a local cluster holding every centre that contributes."""
    from oracle.model import forces_for
    from oracle.neighbors import neighbor_list
    rl = model.rc + model.skin
    assert np.min(box) > 2.0 * (2.0 * rl + 1.0), "box too small for a local cluster"
    E, F, V = [], [], []
    for a in atoms:
        lpos, ltypes, lbox, la, _ = local_cluster(pos, types, box, a, 2.0 * rl + 1.0)
        off, idx = neighbor_list(lpos, lbox, rl)
        r = forces_for(model, lpos, ltypes, lbox, [la], off, idx)
        E.append(r["E_i"][0])
        F.append(r["F"][0])
        V.append(r["virial"][0])
    return np.array(E), np.array(F), np.array(V)
