"""GPU parity of the fusion configurations (Section 3.4, Table "Configurable
fusion"): the single kernel that recomputes the encoder in its second pass
(the paper's mega-fusion), the three-kernel split with G_i and dE/dG_i in
HBM (the paper's partial fusion) and the ten-kernel unfused pipeline with
every intermediate in HBM (the table's "before fusion" row), against the
oracle and against the default cached configuration."""
import dataclasses

import numpy as np
import pytest

import synth
from oracle.model import Model, evaluate
from oracle.neighbors import neighbor_list
from tests.gpu_helpers import gpu_eval, max_abs, log

pytestmark = pytest.mark.gpu

TOL64 = 1e-9
REL32 = 1e-4


def _eval(hp, w, fusion):
    return gpu_eval(hp, w.weights, w.pos, w.types, w.box, fusion=fusion)


def _rel(a, ref):
    return max_abs(a, ref) / max(float(np.max(np.abs(ref))), 1e-300)


@pytest.mark.parametrize("fusion", [1, 2, 3])
@pytest.mark.parametrize("precision", [64, 32])
@pytest.mark.parametrize("name,n,over", [("fcc-binary-4", None, {}), ("fcc-hea6-128", 5, {}),
                                         ("fcc-binary-4", None, {"lmax": 1, "enc_cond": 0, "reg_cond": 0}),
                                         ("bcc-unary-32", 6, {"enc_hidden": 2, "reg_hidden": 3})])
def test_fusion_configurations_match_oracle(fusion, precision, name, n, over):
    w = synth.make_workload(name, seed=13, n=n, hp_overrides=dict(over, precision=precision))
    label = f"{name}/{over}/fusion={fusion}/fp{precision}"
    log(f"[fusion] {label}: N={len(w.pos)}")
    g = _eval(w.hp, w, fusion)
    m = Model(w.hp, w.weights)
    off, idx = neighbor_list(w.pos, w.box, m.rc + m.skin)
    ref = evaluate(m, w.pos, w.types, w.box, off, idx)
    if precision == 64:
        eE, eF, eV = max_abs(g["E_i"], ref["E_i"]), max_abs(g["F"], ref["F"]), max_abs(g["virial"], ref["virial"])
        log(f"[fusion] {label}: max|dE|={eE:.2e} max|dF|={eF:.2e} max|dW|={eV:.2e}")
        assert max(eE, eF, eV) <= TOL64
        assert abs(g["totals"][0] - ref["E"]) <= TOL64 * len(w.pos)
        assert max_abs(g["totals"][1:], ref["W"]) <= TOL64 * len(w.pos)
    else:
        eE, eF, eV = _rel(g["E_i"], ref["E_i"]), _rel(g["F"], ref["F"]), _rel(g["virial"], ref["virial"])
        log(f"[fusion] {label}: rel dE={eE:.2e} dF={eF:.2e} dW={eV:.2e}")
        assert max(eE, eF, eV) <= REL32
    st = g["stats"]
    assert st["n_listed_pairs"] == len(idx)
    g["pot"].close()


def _unfused_bytes(n_atoms, n_listed, k, lmax, eb):
    """Intermediates of the unfused configuration: per listed entry the pair
    vector and distance (4 float64), g_rad and dg_rad/dr (2k), g_ang and its
    Jacobian (16 + 48), U and V rows (k + 16); per atom P and W (2 x 16k) and
    the descriptor buffer ((l_max + 1) k); each sub-buffer 256-byte aligned."""
    al = lambda b: (b + 255) // 256 * 256
    per_entry = [4 * 8, k * eb, k * eb, 16 * eb, 48 * eb, k * eb, 16 * eb]
    per_atom = [16 * k * eb, 16 * k * eb]
    return (sum(al(b * n_listed) for b in per_entry) + sum(al(b * n_atoms) for b in per_atom)
            + n_atoms * (lmax + 1) * k * eb)


def test_configurations_agree_and_hold_their_intermediates():
    """The four configurations on one input agree to rounding; the
    recompute one holds no workspace, the three-kernel one (l_max + 1) k
    values per atom more than the cached one, the unfused one every
    intermediate of Eqs. 1-10 and no workspace."""
    w = synth.make_workload("fcc-hea6-128", seed=3, n=6)
    out = {}
    for fusion in (0, 1, 2, 3):
        out[fusion] = _eval(w.hp, w, fusion)
    for fusion in (1, 2, 3):
        for key in ("E_i", "F", "virial"):
            d = max_abs(out[fusion][key], out[0][key])
            log(f"[fusion] {fusion} vs cached {key}: {d:.2e}")
            assert d <= TOL64
    st = out[0]["stats"]
    ws = out[0]["pot"].memory_bytes() - out[1]["pot"].memory_bytes()
    assert ws > 0 and ws % (8 * st["n_blocks"]) == 0     # one slot per work-group, held by cached only
    extra = out[2]["pot"].memory_bytes() - out[0]["pot"].memory_bytes()
    assert extra == len(w.pos) * (w.hp.lmax + 1) * w.hp.k * 8
    n_listed = out[3]["stats"]["n_listed_pairs"]
    extra = out[3]["pot"].memory_bytes() - out[1]["pot"].memory_bytes()
    assert extra == _unfused_bytes(len(w.pos), n_listed, w.hp.k, w.hp.lmax, 8)
    for g in out.values():
        g["pot"].close()


def test_unfused_md_steps_and_switching_back():
    """Ten velocity-Verlet steps in the unfused configuration track the cached
    configuration; switching a context back releases the intermediates."""
    import torch
    from paper_2608_16329_amd import Potential
    w = synth.make_workload("fcc-binary-4", seed=21)
    n = len(w.pos)
    runs = {}
    for fusion in (0, 3):
        pot = Potential(w.hp, w.weights)
        pot.set_fusion(fusion)
        pot.set_masses(w.masses)
        pos = torch.from_numpy(w.pos.copy()).to("cuda:0")
        vel = torch.from_numpy(w.vel.copy()).to("cuda:0")
        types = torch.from_numpy(w.types).to("cuda:0")
        F = torch.zeros((n, 3), dtype=torch.float64, device="cuda:0")
        pot.build_neighbors(pos, types, w.box)
        pot.compute(pos, F)
        for _ in range(10):
            pot.md_first_half(pos, vel, F, w.dt)
            pot.build_neighbors(pos, types, w.box)
            pot.compute(pos, F)
            pot.md_second_half(vel, F, w.dt)
        torch.cuda.synchronize()
        runs[fusion] = (pos.cpu().numpy(), F.cpu().numpy())
        if fusion == 3:
            held = pot.memory_bytes()
            pot.set_fusion(0)
            assert pot.memory_bytes() < held
        pot.close()
    dx = max_abs(runs[3][0], runs[0][0])
    dF = max_abs(runs[3][1], runs[0][1])
    log(f"[fusion] unfused vs cached after 10 steps: max|dx|={dx:.2e} max|dF|={dF:.2e}")
    assert dx <= 1e-10 and dF <= 1e-8


def test_fusion_argument_checks():
    from paper_2608_16329_amd import Potential, MlipError
    hp = synth.HParams(n_species=2)
    pot = Potential(hp, synth.random_weights(hp, 0))
    with pytest.raises(MlipError, match="ARG"):
        pot.set_fusion(7)
    pot.close()
    hp16 = dataclasses.replace(hp, k=16)
    pot = Potential(hp16, synth.random_weights(hp16, 0))
    for fusion in (1, 2, 3):
        with pytest.raises(MlipError, match="ARG"):
            pot.set_fusion(fusion)
    pot.set_fusion(0)
    pot.close()


@pytest.mark.parametrize("precision", [64, 32])
def test_configurations_agree_at_scale(precision):
    """At 16,000 atoms of the six-component BCC alloy (hundreds of tiles and
    work-groups, long unfused grids) every configuration matches the default
    cached one, which the other tests pin to the oracle, on all atoms."""
    w = synth.make_workload("bcc-hea6-sweep", seed=17, n=20, hp_overrides={"precision": precision})
    out = {f: _eval(w.hp, w, f) for f in (0, 1, 2, 3)}
    for f in (1, 2, 3):
        for key in ("E_i", "F", "virial"):
            if precision == 64:
                d = max_abs(out[f][key], out[0][key])
                log(f"[fusion] N={len(w.pos)} fp64 {f} vs cached {key}: {d:.2e}")
                assert d <= TOL64
            else:
                d = _rel(out[f][key], out[0][key])
                log(f"[fusion] N={len(w.pos)} fp32 {f} vs cached {key}: rel {d:.2e}")
                assert d <= REL32
        assert out[f]["stats"]["n_active_pairs"] == out[0]["stats"]["n_active_pairs"]
    for g in out.values():
        g["pot"].close()


def _eval_scatter(hp, weights, pos, types, box, scatter):
    import torch
    from paper_2608_16329_amd import Potential
    pot = Potential(hp, weights)
    pot.set_scatter(scatter)
    p = torch.from_numpy(np.ascontiguousarray(pos)).to("cuda:0")
    t = torch.from_numpy(np.ascontiguousarray(types, dtype=np.int32)).to("cuda:0")
    pot.build_neighbors(p, t, box)
    n = len(pos)
    F = torch.empty((n, 3), dtype=torch.float64, device="cuda:0")
    E = torch.empty(n, dtype=torch.float64, device="cuda:0")
    V = torch.empty((n, 9), dtype=torch.float64, device="cuda:0")
    tot = pot.compute(p, F, E, V, totals=True)
    torch.cuda.synchronize()
    out = {"F": F.cpu().numpy(), "E_i": E.cpu().numpy(), "virial": V.cpu().numpy(), "totals": tot,
           "stats": pot.stats()}
    pot.close()
    return out


@pytest.mark.parametrize("precision", [64, 32])
@pytest.mark.parametrize("name,n", [("fcc-binary-4", None), ("fcc-hea6-128", 5), ("bcc-hea6-sweep", 12)])
def test_tile_reduced_scatter_matches_oracle(precision, name, n):
    """The F_j scatter summed per distinct neighbour of a tile in LDS (one
    atomic per neighbour) against the oracle."""
    w = synth.make_workload(name, seed=19, n=n, hp_overrides={"precision": precision})
    label = f"{name}/tile scatter/fp{precision}"
    log(f"[scatter] {label}: N={len(w.pos)}")
    g = _eval_scatter(w.hp, w.weights, w.pos, w.types, w.box, 1)
    ref = evaluate(Model(w.hp, w.weights), w.pos, w.types, w.box)
    if precision == 64:
        e = [max_abs(g[k], ref[k]) for k in ("E_i", "F", "virial")]
        log(f"[scatter] {label}: max|dE|={e[0]:.2e} max|dF|={e[1]:.2e} max|dW|={e[2]:.2e}")
        assert max(e) <= TOL64
    else:
        e = [_rel(g[k], ref[k]) for k in ("E_i", "F", "virial")]
        log(f"[scatter] {label}: rel dE={e[0]:.2e} dF={e[1]:.2e} dW={e[2]:.2e}")
        assert max(e) <= REL32


def test_tile_reduced_scatter_long_rows():
    """A 12 A cutoff (about 700 neighbours, 2-atom tiles): the tile's table
    of 1024 slots runs nearly full, and contributions whose probes find no
    slot take the direct atomic."""
    rng = np.random.default_rng(31)
    hp = synth.HParams(n_species=3, cutoff=12.0, skin=0.5)
    pos, box = synth.lattice("fcc", 7, 3.6)
    pos = pos + rng.normal(0.0, 0.1, pos.shape)
    types = rng.integers(0, 3, len(pos)).astype(np.int32)
    wts = synth.random_weights(hp, 4, 0.3)
    g = _eval_scatter(hp, wts, pos, types, box, 1)
    ref = evaluate(Model(hp, wts), pos, types, box)
    e = [max_abs(g[k], ref[k]) for k in ("E_i", "F", "virial")]
    log(f"[scatter] long rows: tile {g['stats']['tile_atoms']}, max|dE|={e[0]:.2e} max|dF|={e[1]:.2e} "
        f"max|dW|={e[2]:.2e}")
    assert max(e) <= TOL64


def test_scatter_argument_checks():
    from paper_2608_16329_amd import Potential, MlipError
    hp = synth.HParams(n_species=2, k=16)
    pot = Potential(hp, synth.random_weights(hp, 0))
    with pytest.raises(MlipError, match="ARG"):
        pot.set_scatter(1)
    with pytest.raises(MlipError, match="ARG"):
        pot.set_scatter(5)
    pot.set_scatter(0)
    pot.close()
