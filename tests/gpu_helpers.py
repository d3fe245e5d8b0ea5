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


# ---------------------------------------------------------------------------
# Oracle over many atoms: a cube (or the whole system) evaluated by worker
# processes over chunks of centre atoms, each with one BLAS thread.

def pool_size():
    """Worker processes for the oracle: the host cores this process may use,
    at most 16 (one GPU's share of a GPU host)."""
    import os
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


_SHARED = None   # (model, pos, types, box, offsets, idx), inherited by forked workers


def _centre_worker(centres):
    import threadpoolctl
    from oracle.model import evaluate
    with threadpoolctl.threadpool_limits(1):
        model, pos, types, box, off, idx = _SHARED
        r = evaluate(model, pos, types, box, off, idx, centres=centres, return_pairs=True)
        return centres, r["E_i"][centres], r["virial"][centres], r["pair_i"], r["pair_j"], r["pair_f"]


def oracle_centres(model, pos, types, box, off, idx, centres):
    """E_i and virial of the centres, and every force contribution their
    partial forces make (F [N][3]; exact for atoms all of whose listing
    centres are among `centres`)."""
    import multiprocessing as mp
    global _SHARED
    _SHARED = (model, pos, types, box, off, idx)
    nw = pool_size()
    chunks = [c for c in np.array_split(np.asarray(centres, dtype=np.int64), 4 * nw) if len(c)]
    try:
        with mp.get_context("fork").Pool(nw) as pool:
            parts = pool.map(_centre_worker, chunks)
    finally:
        _SHARED = None
    N = len(pos)
    E = np.full(N, np.nan)
    V = np.full((N, 9), np.nan)
    F = np.zeros((N, 3))
    for c, e, v, pi, pj, pf in parts:
        E[c] = e
        V[c] = v
        np.add.at(F, pi, pf)
        np.add.at(F, pj, -pf)
    return E, F, V


def oracle_full(model, pos, types, box):
    """Oracle E_i, F and virial of every atom of a periodic system, and its
    neighbour list (cell list, the same set as brute force)."""
    from oracle.neighbors import neighbor_list
    off, idx = neighbor_list(pos, box, model.rc + model.skin)
    E, F, V = oracle_centres(model, pos, types, box, off, idx, np.arange(len(pos)))
    return E, F, V, off, idx


def cube_members(pos, box, centre, half):
    """Indices of the atoms within the cube of half-edge `half` around
    `centre` (minimum image), and their displacement from it."""
    d = pos - np.asarray(centre, dtype=np.float64)
    d -= box * np.round(d / box)
    return np.nonzero(np.all(np.abs(d) < half, axis=1))[0]


def oracle_cube(model, pos, types, box, centre, half, index=None):
    """Oracle E_i, F_i and per-atom virial of every atom inside the cube of
    half-edge `half` around `centre` (minimum image) of a periodic system.

    pos/types may be any subset of the system that holds every atom within
    half + 2 (r_c + skin) + 1 of the centre (its global indices in `index`,
    default 0..len-1).  The subset is cut out around the centre into a
    non-periodic box wide enough that no image is within reach; the centres
    evaluated are the cube's atoms and their listed neighbours, so each
    cube atom's force is complete.  Returns (global indices, E, F, virial)."""
    from oracle.neighbors import cell_list_neighbors
    rl = model.rc + model.skin
    index = np.arange(len(pos)) if index is None else np.asarray(index)
    reach = half + 2.0 * rl + 1.0
    assert np.all(2.0 * reach < box), "cube too large for the box"
    d = pos - np.asarray(centre, dtype=np.float64)
    d -= box * np.round(d / box)
    sel = np.nonzero(np.all(np.abs(d) < reach, axis=1))[0]
    inner = np.all(np.abs(d[sel]) < half, axis=1)
    lbox = np.full(3, 2.0 * reach + 2.0 * rl + 2.0)
    lpos = d[sel] + lbox / 2.0
    ltypes = np.asarray(types)[sel]
    off, idx = cell_list_neighbors(lpos, lbox, rl)
    atoms = np.nonzero(inner)[0]
    nb = [idx[off[a]:off[a + 1]].astype(np.int64) for a in atoms]
    centres = np.unique(np.concatenate([atoms] + nb))
    E, F, V = oracle_centres(model, lpos, ltypes, lbox, off, idx, centres)
    return index[sel[atoms]], E[atoms], F[atoms], V[atoms]


def oracle_rows(pos, box, rl, rows_local):
    """Listed neighbours (exact definition on the caller's coordinates) of
    the given rows of a subset that holds every atom within rl + 1 of them;
    indices into the subset."""
    from oracle.neighbors import neighbors_of
    return neighbors_of(pos, box, rl, rows_local)


def compare_rows(got_rows, ref_rows, labels):
    """Neighbour rows as sets: identical, row by row."""
    for lab, g, r in zip(labels, got_rows, ref_rows):
        gs, rs = np.sort(np.asarray(g)), np.sort(np.asarray(r))
        if not np.array_equal(gs, rs):
            raise AssertionError(f"row of atom {lab}: gpu-only {sorted(set(gs.tolist()) - set(rs.tolist()))}, "
                                 f"oracle-only {sorted(set(rs.tolist()) - set(gs.tolist()))}")


def curved_head(hp, weights, pos, types, box):
    """Weights whose head operates in the curved region of its SiLUs: the
    first head layer A0 scaled by 1 / median |vec G| (the descriptor is
    unnormalised, so with N(0, 1/fan_in) weights most head pre-activations
    lie far out on the linear or zero branch).  Returns the new blob and, per
    head layer, the fraction of pre-activations with |z| < 4 (oracle values)."""
    from oracle.model import Model, evaluate, silu
    m = Model(hp, weights)
    r = evaluate(m, pos, types, box, return_descriptors=True)
    x = r["G"].reshape(len(r["G"]), -1)
    w2 = synth.scale_segments(hp, weights, ".A0", 1.0 / float(np.median(np.abs(x))))
    m2 = Model(hp, w2)
    rho = m2.head_index(np.asarray(types, dtype=np.int64))
    zs = [[] for _ in range(m2.nh_reg)]
    for t in np.unique(rho):
        h = m2.head[int(t)]
        z = x[rho == t] @ h["A0"].T + h["c0"]
        zs[0].append(z)
        y = silu(z)
        for li, (At, ct) in enumerate(h["hidden"]):
            z = y @ At.T + ct
            zs[li + 1].append(z)
            y = y + silu(z)
    return w2, [float(np.mean(np.abs(np.concatenate(z)) < 4.0)) for z in zs]
