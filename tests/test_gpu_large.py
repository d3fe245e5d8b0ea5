"""GPU parity at the full workload sizes, in the launch configuration the
benchmark times (same library calls, persistent grid over all CUs):
sampled atoms are checked against the oracle one by one (each from a local
cluster cut out of the periodic system), sampled neighbour rows against the
oracle's brute-force rows over all N atoms."""
import numpy as np
import pytest

import synth
from oracle.model import Model
from oracle.neighbors import neighbors_of
from tests.gpu_helpers import to_dev, oracle_sample, log, max_abs

pytestmark = pytest.mark.gpu

TOL = 1e-9


def _run(name, n_sample, seed=0):
    import torch
    from paper_2608_16329_amd import Potential
    log(f"[large] {name}: generating")
    w = synth.make_workload(name, seed=seed)
    N = len(w.pos)
    dev = torch.device("cuda:0")
    pot = Potential(w.hp, w.weights)
    pos = to_dev(w.pos)
    types = to_dev(w.types)
    F = torch.empty((N, 3), dtype=torch.float64, device=dev)
    E = torch.empty(N, dtype=torch.float64, device=dev)
    V = torch.empty((N, 9), dtype=torch.float64, device=dev)
    log(f"[large] {name}: N={N} build + compute")
    pot.build_neighbors(pos, types, w.box)
    tot = pot.compute(pos, F, E, V, totals=True)
    torch.cuda.synchronize()
    st = pot.stats()
    rng = np.random.default_rng(seed + 7)
    atoms = list(rng.choice(N, n_sample - 4, replace=False)) + [0, N - 1]
    for s in range(w.hp.n_species):       # one atom of each species, the rarest first
        idx = np.nonzero(w.types == s)[0]
        if len(idx):
            atoms.append(int(idx[len(idx) // 2]))
    atoms = sorted(set(int(a) for a in atoms))
    m = Model(w.hp, w.weights)
    log(f"[large] {name}: oracle on {len(atoms)} sampled atoms")
    oE, oF, oV = oracle_sample(m, w.pos, w.types, w.box, atoms)
    gE = E[atoms].cpu().numpy()
    gF = F[atoms].cpu().numpy()
    gV = V[atoms].cpu().numpy()
    eE, eF, eV = np.abs(gE - oE).max(), np.abs(gF - oF).max(), np.abs(gV - oV).max()
    log(f"[large] {name}: max|dE|={eE:.3e} max|dF|={eF:.3e} max|dW|={eV:.3e}")
    assert eE <= TOL and eF <= TOL and eV <= TOL
    # totals are the sums of the per-atom outputs
    Et = E.sum().item()
    assert abs(tot[0] - Et) <= 1e-9 * max(1.0, abs(Et)) * 10
    Wt = V.sum(0).cpu().numpy()
    assert np.abs(tot[1:] - Wt).max() <= 1e-9 * max(1.0, np.abs(Wt).max()) * 10
    # momentum: sum of forces vanishes up to rounding
    Fs = F.sum(0).cpu().numpy()
    assert np.abs(Fs).max() <= 1e-12 * N * F.abs().max().item()
    # neighbour rows of a few atoms, bit for bit
    log(f"[large] {name}: neighbour rows")
    goff, gidx = pot.neighbors()
    rl = w.hp.cutoff + w.hp.skin
    rows = atoms[:6]
    ref = neighbors_of(w.pos, w.box, rl, rows)
    for a, r in zip(rows, ref):
        assert np.array_equal(np.sort(gidx[goff[a]:goff[a + 1]]), r), a
    assert st["n_listed_pairs"] == goff[-1]
    pot.close()


def test_six_component_fcc_8m_sampled():
    _run("fcc-hea6-128", 14)


def test_ternary_fcc_1m_sampled():
    _run("fcc-ternary-64", 12)


def test_bcc_unary_nve_100_steps_sampled():
    """100 NVE steps of the 65,536-atom BCC metal on the GPU (rebuild every
    10 steps or on the skin guard); at steps 10, 50 and 100 the oracle is
    fed the GPU's own positions for sampled atoms."""
    import torch
    from paper_2608_16329_amd import Potential
    w = synth.make_workload("bcc-unary-32", seed=3)
    N = len(w.pos)
    m = Model(w.hp, w.weights)
    pot = Potential(w.hp, w.weights)
    pot.set_masses(w.masses)
    pos, vel, types = to_dev(w.pos), to_dev(w.vel), to_dev(w.types)
    ref = pos.clone()
    dev = torch.device("cuda:0")
    F = torch.zeros((N, 3), dtype=torch.float64, device=dev)
    E = torch.zeros(N, dtype=torch.float64, device=dev)
    V = torch.zeros((N, 9), dtype=torch.float64, device=dev)
    pot.build_neighbors(pos, types, w.box)
    pot.compute(pos, F, E, V)
    rng = np.random.default_rng(5)
    rebuilds = 0
    for step in range(1, 101):
        d2 = pot.md_first_half(pos, vel, F, 1.0, ref)
        if step % 10 == 0 or d2 > (0.5 * w.hp.skin) ** 2:
            pot.build_neighbors(pos, types, w.box)
            ref.copy_(pos)
            rebuilds += 1
        pot.compute(pos, F, E, V)
        pot.md_second_half(vel, F, 1.0)
        if step in (10, 50, 100):
            torch.cuda.synchronize()
            p = pos.cpu().numpy()
            atoms = sorted(int(a) for a in rng.choice(N, 6, replace=False))
            oE, oF, oV = oracle_sample(m, p, w.types, w.box, atoms)
            eE = np.abs(E[atoms].cpu().numpy() - oE).max()
            eF = np.abs(F[atoms].cpu().numpy() - oF).max()
            eV = np.abs(V[atoms].cpu().numpy() - oV).max()
            log(f"[md] step {step}: rebuilds {rebuilds} max|dE|={eE:.3e} max|dF|={eF:.3e} max|dW|={eV:.3e}")
            assert eE <= TOL and eF <= TOL and eV <= TOL
            goff, gidx = pot.neighbors()
            ref_rows = neighbors_of(p, w.box, w.hp.cutoff + w.hp.skin, atoms[:3])
            for a, r in zip(atoms[:3], ref_rows):
                assert np.array_equal(np.sort(gidx[goff[a]:goff[a + 1]]), r)
    pot.close()


def test_bcc_six_component_sweep_shape_sampled():
    """The capacity-sweep alloy (6-component BCC, a = 3.2 A) at L = 128
    (4,194,304 atoms) in the launch configuration of the sweep: sampled
    atoms against the oracle."""
    import torch
    from paper_2608_16329_amd import Potential
    w = synth.make_workload("bcc-hea6-sweep", seed=0, n=128)
    N = len(w.pos)
    log(f"[large] bcc sweep shape N={N}")
    pot = Potential(w.hp, w.weights)
    p = to_dev(w.pos)
    pot.build_neighbors(p, to_dev(w.types), w.box)
    F = torch.empty((N, 3), dtype=torch.float64, device="cuda:0")
    E = torch.empty(N, dtype=torch.float64, device="cuda:0")
    V = torch.empty((N, 9), dtype=torch.float64, device="cuda:0")
    pot.compute(p, F, E, V)
    torch.cuda.synchronize()
    atoms = np.random.default_rng(21).choice(N, 32, replace=False)
    Er, Fr, Vr = oracle_sample(Model(w.hp, w.weights), w.pos, w.types, w.box, atoms)
    eE = max_abs(E.cpu().numpy()[atoms], Er)
    eF = max_abs(F.cpu().numpy()[atoms], Fr)
    eV = max_abs(V.cpu().numpy()[atoms], Vr)
    log(f"[large] bcc sweep shape: max|dE|={eE:.2e} max|dF|={eF:.2e} max|dW|={eV:.2e}")
    assert max(eE, eF, eV) <= 1e-9
    pot.close()


def test_fusion_configurations_full_size():
    """On the 8.4M-atom six-component FCC workload the recompute and
    three-kernel configurations match the cached one (pinned to the oracle
    above) on every atom; the unfused one does not fit and reports OOM."""
    import torch
    from paper_2608_16329_amd import Potential, MlipError
    w = synth.make_workload("fcc-hea6-128", seed=0)
    N = len(w.pos)
    dev = torch.device("cuda:0")
    pot = Potential(w.hp, w.weights)
    pos = to_dev(w.pos)
    types = to_dev(w.types)
    pot.build_neighbors(pos, types, w.box)
    res = {}
    for fusion in (0, 1, 2):
        pot.set_fusion(fusion)
        F = torch.empty((N, 3), dtype=torch.float64, device=dev)
        E = torch.empty(N, dtype=torch.float64, device=dev)
        V = torch.empty((N, 9), dtype=torch.float64, device=dev)
        log(f"[large] fusion {fusion}: compute")
        pot.compute(pos, F, E, V)
        torch.cuda.synchronize()
        res[fusion] = (E, F, V)
    for fusion in (1, 2):
        d = [(res[fusion][k] - res[0][k]).abs().max().item() for k in range(3)]
        log(f"[large] fusion {fusion} vs cached on {N} atoms: max|dE|={d[0]:.2e} max|dF|={d[1]:.2e} max|dW|={d[2]:.2e}")
        assert max(d) <= TOL
    del res
    torch.cuda.empty_cache()
    pot.set_fusion(3)
    F = torch.empty((N, 3), dtype=torch.float64, device=dev)
    with pytest.raises(MlipError, match="OOM"):
        pot.compute(pos, F)
    pot.close()
