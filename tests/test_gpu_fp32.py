"""GPU parity of the float32 network path (mlip_hparams.precision = 32)
against the float64 oracle on identical seeded inputs.

The bar is relative, in two parts, for each output array (E_i, F, per-atom
virial):
  * normwise: the largest absolute deviation from the oracle stays within
    1e-4 of the array's largest oracle magnitude;
  * per element: every entry whose oracle magnitude is at least a tenth of
    the array's largest deviates by at most 1e-4 of its own magnitude.
Smaller entries are sums whose terms cancel, and float32 rounding of those
terms is relative to the terms, not to the sum; their per-element figures
(floors 1e-2 and 1e-3 of the largest) are logged.  Neighbour sets do not
depend on the network precision and must be identical."""
import dataclasses

import numpy as np
import pytest

import synth
import oracle
from oracle.model import Model, evaluate
from oracle.neighbors import neighbor_list
from tests.gpu_helpers import (gpu_eval, assert_same_neighbor_sets, max_abs, log, oracle_sample, to_dev,
                               curved_head, oracle_cube)

pytestmark = pytest.mark.gpu

REL_TOL = 1e-4
ELEM_FLOOR = 0.1   # per-element check for entries at least this fraction of the array's largest


def rel_err(a, ref):
    scale = float(np.max(np.abs(ref)))
    return max_abs(a, ref) / scale if scale > 0 else max_abs(a, ref)


def elem_rel(a, ref, floor):
    """Largest per-element relative deviation over the entries whose oracle
    magnitude is at least `floor` times the array's largest."""
    a, ref = np.asarray(a).ravel(), np.asarray(ref).ravel()
    scale = float(np.max(np.abs(ref))) if ref.size else 0.0
    m = np.abs(ref) >= floor * scale
    if scale == 0.0 or not m.any():
        return 0.0
    return float(np.max(np.abs(a[m] - ref[m]) / np.abs(ref[m])))


def check_elementwise(label, pairs):
    """Log the per-element figures at three floors and assert the bar at
    ELEM_FLOOR."""
    parts = []
    for key, a, ref in pairs:
        parts.append(key + " " + " ".join(f"{f:g}:{elem_rel(a, ref, f):.1e}" for f in (0.1, 0.01, 0.001)))
    log(f"[fp32] {label}: per-element rel (floor:value) " + "; ".join(parts))
    for key, a, ref in pairs:
        e = elem_rel(a, ref, ELEM_FLOOR)
        assert e <= REL_TOL, (key, e)


def _hp32(hp):
    return dataclasses.replace(hp, precision=32)


def _compare(hp, weights, pos, types, box, label):
    hp = _hp32(hp)
    log(f"[fp32] {label}: N={len(pos)}")
    g = gpu_eval(hp, weights, pos, types, box)
    m = Model(hp, weights)
    off, idx = neighbor_list(pos, box, m.rc + m.skin)
    goff, gidx = g["pot"].neighbors()
    assert_same_neighbor_sets(goff, gidx, off, idx)
    ref = evaluate(m, pos, types, box, off, idx)
    eE, eF, eV = rel_err(g["E_i"], ref["E_i"]), rel_err(g["F"], ref["F"]), rel_err(g["virial"], ref["virial"])
    log(f"[fp32] {label}: rel dE={eE:.2e} dF={eF:.2e} dW={eV:.2e}")
    check_elementwise(label, [("E", g["E_i"], ref["E_i"]), ("F", g["F"], ref["F"]), ("W", g["virial"], ref["virial"])])
    assert eE <= REL_TOL, eE
    assert eF <= REL_TOL, eF
    assert eV <= REL_TOL, eV
    assert abs(g["totals"][0] - ref["E"]) <= REL_TOL * abs(ref["E"]) + REL_TOL * len(pos)
    st = g["stats"]
    assert st["n_active_pairs"] == len(oracle.neighbors.active_rows(pos, box, off, idx, m.rc)[0])
    g["pot"].close()
    return g, ref


VARIANTS = {
    "default": {},
    "lmax0": {"lmax": 0},
    "lmax2": {"lmax": 2},
    "enc_universal": {"enc_cond": 0},
    "head_universal": {"reg_cond": 0},
    "enc_hidden1": {"enc_hidden": 1},
    "deep": {"enc_hidden": 5, "reg_hidden": 6},
    "k16": {"k": 16},
    "k64": {"k": 64},
    "cartesian": {"angular": 1},
    "lmax4": {"lmax": 4},
    "lmax5": {"lmax": 5},
    "k16_lmax5": {"k": 16, "lmax": 5},
    "k64_lmax4": {"k": 64, "lmax": 4},
    "k64_lmax5": {"k": 64, "lmax": 5},
}


@pytest.mark.parametrize("name,n,over", [("fcc-binary-4", None, {}), ("fcc-hea6-128", 5, {}),
                                         ("fcc-binary-4", None, {"enc_hidden": 5, "reg_hidden": 6})])
def test_fp32_head_in_curved_region(name, n, over):
    """The head's first layer scaled so most head pre-activations lie where
    the SiLU curves (|z| < 4): the float32 sigmoid (hardware exp2 and
    reciprocal) and its backward factor away from the saturated branches."""
    w = synth.make_workload(name, seed=3, n=n, hp_overrides=over)
    wts, frac = curved_head(w.hp, w.weights, w.pos, w.types, w.box)
    log(f"[fp32] {name}/curved head {over}: fraction |z| < 4 per head layer {[round(f, 2) for f in frac]}")
    # most units curved: the first head layer, and the layers on average (deep
    # residual stacks drift outwards in their last layers)
    assert frac[0] > 0.5 and float(np.mean(frac)) > 0.5, frac
    _compare(w.hp, wts, w.pos, w.types, w.box, f"{name}/curved head {over}")


@pytest.mark.parametrize("variant", list(VARIANTS))
def test_fp32_binary_fcc_variants(variant):
    w = synth.make_workload("fcc-binary-4", seed=3, hp_overrides=VARIANTS[variant])
    _compare(w.hp, w.weights, w.pos, w.types, w.box, f"fcc-binary-4/{variant}")


@pytest.mark.parametrize("name,n", [("fcc-ternary-64", 4), ("fcc-hea6-128", 5), ("bcc-unary-32", 6)])
def test_fp32_preset_shapes(name, n):
    w = synth.make_workload(name, seed=5, n=n)
    _compare(w.hp, w.weights, w.pos, w.types, w.box, f"{name}/n={n}")


def test_fp32_ragged_and_sparse():
    rng = np.random.default_rng(21)
    w = synth.make_workload("fcc-hea6-128", seed=11, n=4)
    perm = rng.permutation(len(w.pos))
    pos = w.pos[perm] + w.box * rng.integers(-1, 2, (len(w.pos), 3))
    types = w.types[perm].copy()
    types[:29] = 2
    _compare(w.hp, w.weights, pos, types, w.box, "ragged")
    box = np.array([40.0, 41.0, 43.0])
    cl = synth.random_cluster(rng, 30, 3, 6.0, min_dist=2.0) + 20.0
    iso = np.array([[2.0, 2.0, 2.0], [35.0, 4.0, 30.0]])
    pos = np.concatenate([cl, iso])
    types = rng.integers(0, 3, len(pos)).astype(np.int32)
    hp = synth.HParams(n_species=3)
    g, _ = _compare(hp, synth.random_weights(hp, 8), pos, types, box, "sparse")


def test_fp32_agrees_with_fp64_path():
    """Both instantiations on the same input: the float32 path deviates from
    the float64 path by no more than from the oracle's bar."""
    w = synth.make_workload("fcc-hea6-128", seed=2, n=6)
    g64 = gpu_eval(w.hp, w.weights, w.pos, w.types, w.box)
    g32 = gpu_eval(_hp32(w.hp), w.weights, w.pos, w.types, w.box)
    for key in ("E_i", "F", "virial"):
        e = rel_err(g32[key], g64[key])
        log(f"[fp32] vs float64 path {key}: rel {e:.2e}")
        assert e <= REL_TOL
    g64["pot"].close()
    g32["pot"].close()


def test_fp32_full_size_sampled():
    """8,388,608-atom 6-component FCC in the launch configuration of the
    benchmark, float32 network: a corner cube of 2,456 lattice sites against
    the oracle."""
    import torch
    from paper_2608_16329_amd import Potential
    w = synth.make_workload("fcc-hea6-128", seed=0, hp_overrides={"precision": 32})
    N = len(w.pos)
    log(f"[fp32] full size N={N}")
    pot = Potential(w.hp, w.weights)
    p = to_dev(w.pos)
    t = to_dev(w.types)
    pot.build_neighbors(p, t, w.box)
    F = torch.empty((N, 3), dtype=torch.float64, device="cuda:0")
    E = torch.empty(N, dtype=torch.float64, device="cuda:0")
    V = torch.empty((N, 9), dtype=torch.float64, device="cuda:0")
    pot.compute(p, F, E, V)
    torch.cuda.synchronize()
    m = Model(w.hp, w.weights)
    log("[fp32] full size: oracle on a corner cube")
    atoms, Er, Fr, Vr = oracle_cube(m, w.pos, w.types, w.box, np.zeros(3), 15.5)
    assert len(atoms) >= 2000
    Eg, Fg, Vg = E.cpu().numpy()[atoms], F.cpu().numpy()[atoms], V.cpu().numpy()[atoms]
    eE, eF, eV = rel_err(Eg, Er), rel_err(Fg, Fr), rel_err(Vg, Vr)
    log(f"[fp32] full size, {len(atoms)} atoms: rel dE={eE:.2e} dF={eF:.2e} dW={eV:.2e}")
    check_elementwise("full size", [("E", Eg, Er), ("F", Fg, Fr), ("W", Vg, Vr)])
    assert eE <= REL_TOL and eF <= REL_TOL and eV <= REL_TOL
    pot.close()


def test_fp32_long_rows_small_tiles():
    """About 700 listed neighbours per atom: the float32 tiles shrink to what
    their entry capacity holds (weights scaled by 0.3 as in the float64 test)."""
    rng = np.random.default_rng(31)
    hp = synth.HParams(n_species=3, cutoff=12.0, skin=0.5)
    pos, box = synth.lattice("fcc", 7, 3.6)
    pos = pos + rng.normal(0.0, 0.1, pos.shape)
    types = rng.integers(0, 3, len(pos)).astype(np.int32)
    g, _ = _compare(hp, synth.random_weights(hp, 4, 0.3), pos, types, box, "long rows")
    st = g["stats"]
    assert st["max_row"] > 600 and 1 <= st["tile_atoms"] < 8 and st["tile_atoms"] * st["max_row"] <= 4096


def test_fp32_md_trajectory():
    """Ten velocity-Verlet steps with the float32 network; every step is fed
    to the oracle at the GPU's own positions."""
    import torch
    from paper_2608_16329_amd import Potential
    w = synth.make_workload("fcc-binary-4", seed=1, hp_overrides={"precision": 32})
    m = Model(w.hp, w.weights)
    pot = Potential(w.hp, w.weights)
    pot.set_masses(w.masses)
    pos, vel, types = to_dev(w.pos), to_dev(w.vel), to_dev(w.types)
    ref = pos.clone()
    F = torch.zeros((len(w.pos), 3), dtype=torch.float64, device="cuda:0")
    pot.build_neighbors(pos, types, w.box)
    pot.compute(pos, F)
    for step in range(1, 11):
        d2 = pot.md_first_half(pos, vel, F, 1.0, ref)
        if step % 10 == 0 or d2 > (0.5 * w.hp.skin) ** 2:
            pot.build_neighbors(pos, types, w.box)
            ref.copy_(pos)
        pot.compute(pos, F)
        pot.md_second_half(vel, F, 1.0)
        torch.cuda.synchronize()
        r = evaluate(m, pos.cpu().numpy(), w.types, w.box)
        e = rel_err(F.cpu().numpy(), r["F"])
        log(f"[fp32] md step {step}: rel dF={e:.2e}")
        assert e <= REL_TOL
        check_elementwise(f"md step {step}", [("F", F.cpu().numpy(), r["F"])])
    pot.close()
