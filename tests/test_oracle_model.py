"""Pins for the oracle's energy/force/virial (Section 3.1, Eqs. 1-10) against
physics and mathematics that do not go through the oracle's own formulas:
finite differences, invariances, closed forms, and a separate PyTorch
autograd implementation that builds the descriptor from the Legendre
addition theorem instead of P_i (no Q_l, no monomials)."""
import math
import os

import numpy as np
import pytest

import synth
import oracle
from oracle.model import Model, evaluate, forces_for
from oracle.neighbors import neighbor_list

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _workload(seed=1, **hp):
    w = synth.make_workload("fcc-binary-4", seed=seed, hp_overrides=hp)
    return w, Model(w.hp, w.weights)


VARIANTS = {
    "default": {},
    "cartesian": {"angular": 1},
    "lmax0": {"lmax": 0},
    "lmax1": {"lmax": 1},
    "lmax2": {"lmax": 2},
    "enc_universal": {"enc_cond": 0},
    "enc_neighbour": {"enc_cond": 1},
    "head_universal": {"reg_cond": 0},
    "k16": {"k": 16},
    "k64_shallow": {"k": 64, "enc_hidden": 2, "reg_hidden": 2},
}


def test_architecture_parameter_counts():
    vals = {}
    with open(os.path.join(GOLD, "architecture.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                k, v = line.split()
                vals[k] = float(v)
    hp = synth.HParams(n_species=1)
    assert hp.k == vals["k"] and hp.lmax == vals["lmax"] and (hp.lmax + 1) ** 2 == vals["d"]
    assert hp.enc_width == vals["enc_width"] and hp.enc_hidden == vals["enc_hidden"]
    assert hp.reg_width == vals["reg_width"] and hp.reg_hidden == vals["reg_hidden"]
    assert hp.cutoff == vals["cutoff"]
    segs = synth.weight_segments(hp)
    enc = sum(n for name, n, _ in segs if name.startswith("enc0."))
    head = sum(n for name, n, _ in segs if name.startswith("head0."))
    assert enc == vals["enc_params_per_table"]
    assert head == vals["head_params_per_table"]
    m = Model(hp, synth.random_weights(hp, 0))
    assert m.d == 16
    with pytest.raises(ValueError):
        Model(hp, np.zeros(enc + head + 1))


@pytest.mark.parametrize("variant", list(VARIANTS))
def test_forces_match_central_differences(variant):
    w, m = _workload(seed=2, **VARIANTS[variant])
    off, idx = neighbor_list(w.pos, w.box, m.rc + m.skin)
    full = evaluate(m, w.pos, w.types, w.box, off, idx)
    rng = np.random.default_rng(0)
    atoms = rng.choice(len(w.pos), 3, replace=False)
    h = 1e-5
    for a in atoms:
        centres = np.unique(np.concatenate([[a], idx[off[a]:off[a + 1]]]))
        for ax in range(3):
            e = []
            for sgn in (1, -1):
                p = w.pos.copy()
                p[a, ax] += sgn * h
                e.append(evaluate(m, p, w.types, w.box, off, idx, centres=centres)["E"])
            fd = -(e[0] - e[1]) / (2 * h)
            F = full["F"][a, ax]
            assert abs(fd - F) <= 1e-6 * max(1.0, abs(F)), (variant, a, ax, fd, F)


def test_virial_matches_diagonal_strain_periodic():
    w, m = _workload(seed=3)
    off, idx = neighbor_list(w.pos, w.box, m.rc + m.skin)
    W = evaluate(m, w.pos, w.types, w.box, off, idx)["W"].reshape(3, 3)
    h = 1e-6
    for ax in range(3):
        e = []
        for sgn in (1, -1):
            s = np.ones(3)
            s[ax] += sgn * h
            e.append(evaluate(m, w.pos * s, w.types, w.box * s, off, idx)["E"])
        dE = (e[0] - e[1]) / (2 * h)
        assert abs(-dE - W[ax, ax]) <= 1e-6 * max(1.0, abs(W[ax, ax]))


def _cluster(seed, C=2, N=40, **hp):
    rng = np.random.default_rng(seed)
    pos = synth.random_cluster(rng, N, C, 7.0, min_dist=2.0) + 30.0
    types = rng.integers(0, C, N).astype(np.int32)
    box = np.array([60.0, 60.0, 60.0])
    hpo = synth.HParams(n_species=C, **hp)
    m = Model(hpo, synth.random_weights(hpo, seed + 1))
    return pos, types, box, m


def test_virial_matches_full_strain_cluster():
    """W[a][b] = -dE/d eps[b][a] for every component (isolated cluster)."""
    pos, types, box, m = _cluster(4)
    c = pos.mean(0)
    W = evaluate(m, pos, types, box)["W"].reshape(3, 3)
    h = 1e-6
    for a in range(3):
        for b in range(3):
            e = []
            for sgn in (1, -1):
                eps = np.zeros((3, 3))
                eps[b, a] = sgn * h
                p = c + (pos - c) @ (np.eye(3) + eps).T
                e.append(evaluate(m, p, types, box)["E"])
            dE = (e[0] - e[1]) / (2 * h)
            assert abs(-dE - W[a, b]) <= 1e-6 * max(1.0, abs(W[a, b])), (a, b)


def test_translation_invariance_and_zero_net_force():
    w, m = _workload(seed=5)
    r0 = evaluate(m, w.pos, w.types, w.box)
    r1 = evaluate(m, w.pos + np.array([3.3, -17.1, 40.2]), w.types, w.box)
    np.testing.assert_allclose(r1["E_i"], r0["E_i"], rtol=1e-12, atol=1e-9)
    np.testing.assert_allclose(r1["F"], r0["F"], atol=1e-9)
    scale = np.abs(r0["F"]).max()
    assert np.abs(r0["F"].sum(0)).max() < 1e-12 * scale * len(w.pos)


def test_rotation_equivariance_cluster():
    pos, types, box, m = _cluster(6)
    rng = np.random.default_rng(9)
    R, _ = np.linalg.qr(rng.normal(size=(3, 3)))
    if np.linalg.det(R) < 0:
        R[:, 0] *= -1
    c = pos.mean(0)
    r0 = evaluate(m, pos, types, box)
    r1 = evaluate(m, c + (pos - c) @ R.T, types, box)
    np.testing.assert_allclose(r1["E_i"], r0["E_i"], rtol=1e-11, atol=1e-9)
    np.testing.assert_allclose(r1["F"], r0["F"] @ R.T, atol=1e-9)
    w0 = r0["virial"].reshape(-1, 3, 3)
    w1 = r1["virial"].reshape(-1, 3, 3)
    np.testing.assert_allclose(w1, R @ w0 @ R.T, atol=1e-8)


def test_permutation_equivariance():
    w, m = _workload(seed=7)
    r0 = evaluate(m, w.pos, w.types, w.box)
    perm = np.random.default_rng(1).permutation(len(w.pos))
    r1 = evaluate(m, w.pos[perm], w.types[perm], w.box)
    np.testing.assert_allclose(r1["E_i"], r0["E_i"][perm], rtol=1e-12, atol=1e-9)
    np.testing.assert_allclose(r1["F"], r0["F"][perm], atol=1e-9)
    np.testing.assert_allclose(r1["virial"], r0["virial"][perm], atol=1e-8)


def test_per_atom_virial_is_symmetric():
    """Each E_i is rotation invariant in its own neighbourhood, so
    sum_j r_ij x f_ij = 0 and every centre-attributed w_i is symmetric."""
    w, m = _workload(seed=8)
    v = evaluate(m, w.pos, w.types, w.box)["virial"].reshape(-1, 3, 3)
    scale = np.abs(v).max()
    assert np.abs(v - v.transpose(0, 2, 1)).max() < 1e-12 * scale * 100


def test_dimer_closed_form():
    """Two atoms, no periodic images: G[0,c] = g_c, G[l,c] = g_c^2 K_l(1) with
    K_1(1) = 1, K_2(1) = 2/3, K_3(1) = 2/5; the force is along the bond and
    equals -dE/dr."""
    hp = synth.HParams(n_species=2)
    m = Model(hp, synth.random_weights(hp, 5))
    box = np.array([40.0, 40.0, 40.0])
    u = np.array([0.3, -0.5, 0.81])
    u /= np.linalg.norm(u)
    r = 3.1
    pos = np.array([[20.0, 20.0, 20.0], 20.0 + r * u])
    types = np.array([0, 1], dtype=np.int32)
    res = evaluate(m, pos, types, box, return_descriptors=True)
    g, _ = m.encoder(0 * 2 + 1, np.array([r]))
    G0 = res["G"][0]
    np.testing.assert_allclose(G0[0], g[0], rtol=1e-13)
    for l, K in ((1, 1.0), (2, 2 / 3), (3, 2 / 5)):
        np.testing.assert_allclose(G0[l], g[0] ** 2 * K, rtol=1e-12)
    F = res["F"]
    assert np.linalg.norm(np.cross(F[1], u)) < 1e-12 * max(1, np.linalg.norm(F[1]))
    h = 1e-6
    e = [evaluate(m, np.array([pos[0], pos[0] + (r + s * h) * u]), types, box)["E"] for s in (1, -1)]
    dEdr = (e[0] - e[1]) / (2 * h)
    np.testing.assert_allclose(F[1] @ u, -dEdr, rtol=1e-6, atol=1e-8)


def test_perfect_lattice_symmetry():
    """Unary perfect FCC: all E_i equal, F = 0, the l = 1..3 descriptor blocks
    vanish (the cubic point group has no invariant harmonics of degree 1-3),
    and the per-atom virial is isotropic."""
    pos, box = synth.lattice("fcc", 4, 3.6)
    types = np.zeros(len(pos), dtype=np.int32)
    hp = synth.HParams(n_species=1)
    m = Model(hp, synth.random_weights(hp, 11))
    res = evaluate(m, pos, types, box, return_descriptors=True)
    E = res["E_i"]
    assert np.ptp(E) < 1e-10 * max(1, abs(E).max())
    assert np.abs(res["F"]).max() < 1e-9
    G = res["G"]
    assert np.abs(G[:, 1:, :]).max() < 1e-10 * max(1.0, np.abs(G[:, 0, :]).max() ** 2)
    v = res["virial"].reshape(-1, 3, 3)
    for a in range(3):
        np.testing.assert_allclose(v[:, a, a], v[:, 0, 0], rtol=1e-10)
    off = v - np.eye(3) * v[:, :1, :1]
    assert np.abs(off).max() < 1e-9 * np.abs(v).max()


def test_lmax0_forces_are_radial():
    w, m = _workload(seed=12, lmax=0)
    res = evaluate(m, w.pos, w.types, w.box, return_pairs=True)
    off, idx = res["offsets"], res["idx"]
    from oracle.neighbors import wrap_positions, min_image
    wpos = wrap_positions(w.pos, w.box)
    rv = min_image(wpos[res["pair_j"]] - wpos[res["pair_i"]], w.box)
    cr = np.cross(rv, res["pair_f"])
    assert np.abs(cr).max() < 1e-11 * np.abs(res["pair_f"]).max() * 10


def test_species_relabelling():
    """Swapping species labels together with the weight tables leaves E_i."""
    w, m = _workload(seed=13)
    hp = w.hp
    segs = synth.weight_segments(hp)
    blob = {}
    p = 0
    for name, n, _ in segs:
        blob[name] = w.weights[p:p + n]
        p += n
    C = hp.n_species
    swap = [1, 0]
    out = []
    for name, n, _ in segs:
        tab, field = name.split(".")
        if tab.startswith("enc"):
            t = int(tab[3:])
            si, sj = divmod(t, C)
            src = f"enc{swap[si] * C + swap[sj]}.{field}"
        else:
            t = int(tab[4:])
            src = f"head{swap[t]}.{field}"
        out.append(blob[src])
    m2 = Model(hp, np.concatenate(out))
    types2 = np.array(swap)[w.types].astype(np.int32)
    r0 = evaluate(m, w.pos, w.types, w.box)
    r1 = evaluate(m2, w.pos, types2, w.box)
    np.testing.assert_allclose(r1["E_i"], r0["E_i"], rtol=1e-13, atol=1e-10)
    np.testing.assert_allclose(r1["F"], r0["F"], atol=1e-10)


def test_pair_conditioning_with_identical_tables_is_universal():
    w, m_univ = _workload(seed=14, enc_cond=0)
    hp_pair = synth.HParams(n_species=2, enc_cond=2)
    segs_u = synth.weight_segments(w.hp)
    n_enc = sum(n for name, n, _ in segs_u if name.startswith("enc0."))
    enc = w.weights[:n_enc]
    blob = np.concatenate([enc] * 4 + [w.weights[n_enc:]])
    m_pair = Model(hp_pair, blob)
    r0 = evaluate(m_univ, w.pos, w.types, w.box)
    r1 = evaluate(m_pair, w.pos, w.types, w.box)
    np.testing.assert_array_equal(r1["E_i"], r0["E_i"])
    np.testing.assert_array_equal(r1["F"], r0["F"])


def test_energy_continuous_at_cutoff():
    """A neighbour approaching r_c from inside contributes a vanishing amount
    (value and slope of the cosine cutoff both reach zero)."""
    hp = synth.HParams(n_species=1)
    m = Model(hp, synth.random_weights(hp, 15))
    box = np.array([40.0, 40.0, 40.0])
    types = np.zeros(2, dtype=np.int32)
    far = evaluate(m, np.array([[10.0, 10, 10], [30.0, 30, 30]]), types, box)["E"]
    es = []
    for dr in (1e-2, 1e-3, 1e-4):
        pos = np.array([[10.0, 10, 10], [10.0 + 6.0 - dr, 10, 10]])
        es.append(abs(evaluate(m, pos, types, box)["E"] - far))
    assert es[1] < es[0] * 0.02 and es[2] < es[1] * 0.02


# ---------------------------------------------------------------------------
# Independent formulation with PyTorch autograd (float64, CPU)
# ---------------------------------------------------------------------------
def _torch_pair_forces(hp, weights, pos, types, box):
    import torch
    torch.set_default_dtype(torch.float64)
    segs = synth.weight_segments(hp)
    blob, p = {}, 0
    for name, n, _ in segs:
        blob[name] = torch.tensor(weights[p:p + n])
        p += n
    C, k, Wd, R = hp.n_species, hp.k, hp.enc_width, hp.reg_width
    rl = hp.cutoff + hp.skin
    # pairs within the cutoff (plain O(N^2) min-image search)
    d = pos[None, :, :] - pos[:, None, :]
    d -= box * np.round(d / box)
    dist = np.linalg.norm(d, axis=2)
    np.fill_diagonal(dist, np.inf)
    I, J = np.nonzero(dist < hp.cutoff)
    rvec = torch.tensor(d[I, J], requires_grad=True)
    r = torch.sqrt((rvec * rvec).sum(1))
    u = rvec / r[:, None]
    silu = torch.nn.functional.silu
    g = torch.zeros(len(I), k)
    tau = {2: types[I] * C + types[J], 1: types[J], 0: np.zeros_like(I)}[hp.enc_cond]
    rows = []
    for t in np.unique(tau):
        sel = np.nonzero(tau == t)[0]
        x = r[sel][:, None]
        h = silu(x * blob[f"enc{t}.w0"] + blob[f"enc{t}.b0"])
        for hh in range(1, hp.enc_hidden):
            Wt = blob[f"enc{t}.W{hh}"].reshape(Wd, Wd)
            h = h + silu(h @ Wt.T + blob[f"enc{t}.b{hh}"])
        mm = h @ blob[f"enc{t}.Wout"].reshape(k, Wd).T + blob[f"enc{t}.bout"]
        fc = 0.5 * (1 + torch.cos(math.pi * x / hp.cutoff))
        rows.append((sel, fc * mm))
    g = torch.zeros(len(I), k)
    for sel, val in rows:
        g = g.index_put((torch.tensor(sel),), val)
    Es = []
    for i in range(len(pos)):
        sel = np.nonzero(I == i)[0]
        gi, ui = g[sel], u[sel]
        t = ui @ ui.T
        if hp.angular == 0:
            K = [torch.ones_like(t), t, t * t - 1.0 / 3.0, t * t * t - 0.6 * t]
        else:
            K = [t ** l for l in range(4)]
        G = [gi.sum(0)]
        for l in range(1, hp.lmax + 1):
            G.append(torch.einsum("jc,jk,kc->c", gi, K[l], gi))
        x = torch.cat(G)
        h = types[i] if hp.reg_cond == 1 else 0
        y = silu(blob[f"head{h}.A0"].reshape(R, -1) @ x + blob[f"head{h}.c0"])
        for hh in range(1, hp.reg_hidden):
            y = y + silu(blob[f"head{h}.A{hh}"].reshape(R, R) @ y + blob[f"head{h}.c{hh}"])
        Es.append(blob[f"head{h}.aout"] @ y + blob[f"head{h}.cout"][0])
    E = torch.stack(Es)
    E.sum().backward()
    return E.detach().numpy(), I, J, rvec.grad.numpy()


@pytest.mark.parametrize("variant", ["default", "cartesian", "lmax2", "enc_neighbour", "head_universal"])
def test_autograd_addition_theorem_formulation(variant):
    pos, types, box, _ = _cluster(20 + len(variant), N=24)
    hp = synth.HParams(n_species=2, **VARIANTS[variant])
    wts = synth.random_weights(hp, 99)
    m = Model(hp, wts)
    res = evaluate(m, pos, types, box, return_pairs=True)
    E, I, J, f = _torch_pair_forces(hp, wts, pos, types, box)
    np.testing.assert_allclose(res["E_i"], E, rtol=1e-11, atol=1e-9)
    ref = {(int(a), int(b)): v for a, b, v in zip(I, J, f)}
    assert len(ref) == len(res["pair_i"])
    for a, b, v in zip(res["pair_i"], res["pair_j"], res["pair_f"]):
        np.testing.assert_allclose(v, ref[(int(a), int(b))], rtol=1e-9, atol=1e-9)


def test_forces_for_subset_matches_full():
    w, m = _workload(seed=21)
    off, idx = neighbor_list(w.pos, w.box, m.rc + m.skin)
    full = evaluate(m, w.pos, w.types, w.box, off, idx)
    atoms = np.array([0, 17, 200, 255])
    sub = forces_for(m, w.pos, w.types, w.box, atoms, off, idx)
    np.testing.assert_allclose(sub["F"], full["F"][atoms], atol=1e-10)
    np.testing.assert_allclose(sub["E_i"], full["E_i"][atoms], rtol=1e-12)
    np.testing.assert_allclose(sub["virial"], full["virial"][atoms], rtol=1e-12, atol=1e-10)
