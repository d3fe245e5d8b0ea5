"""Pins for the oracle's velocity-Verlet driver and its active-pair filter,
against what mechanics and the neighbour definition fix independently of the
oracle's own formulas:

  * free flight: with no neighbours the force is zero, so positions follow
    x0 + n dt v exactly and the rebuild schedule is known in closed form;
  * energy conservation: the total energy K + E of an NVE run stays constant
    to O(dt^2) (velocity Verlet is second order), with the kinetic energy
    taken from CODATA constants rather than the driver's unit factor, so a
    wrong unit factor, mass lookup, kick weight or force sign breaks either
    the bound or the dt^2 convergence;
  * time reversibility: N steps, velocities negated, N steps return to the
    start (a stale force in the second half kick or unequal half kicks break
    it);
  * the active pairs r < r_c of a listed set: constructed pairs at exactly
    r_c and one ulp inside, across the periodic face (sign of r_ij = r_j -
    r_i), and SciPy's periodic k-d tree on random positions.
"""
import numpy as np
import pytest
from scipy.spatial import cKDTree

import synth
from oracle.md import velocity_verlet
from oracle.model import Model, evaluate
from oracle.neighbors import active_rows, brute_force_neighbors

# CODATA 2018: elementary charge (J per eV) and atomic mass constant (kg)
EV_J = 1.602176634e-19
AMU_KG = 1.66053906660e-27
# 1 amu A^2 / fs^2 in eV: kg m^2 / s^2 with A = 1e-10 m and fs = 1e-15 s
AMU_A2_FS2_EV = AMU_KG * 1e-20 / 1e-30 / EV_J


def _kinetic(vel, masses, types):
    m = np.asarray(masses)[np.asarray(types)]
    return 0.5 * AMU_A2_FS2_EV * float((m[:, None] * vel * vel).sum())


def _light_model(C, seed):
    # a small network keeps 100+ evaluations cheap; the driver does not
    # depend on the network's size
    hp = synth.HParams(n_species=C, k=16, lmax=2, enc_hidden=2, reg_hidden=2)
    return hp, Model(hp, synth.random_weights(hp, seed, energy_scale=0.05))


def _cluster(seed, n=28):
    rng = np.random.default_rng(seed)
    pos = synth.random_cluster(rng, n, 2, 5.5, min_dist=2.2) + 15.0
    types = rng.integers(0, 2, n).astype(np.int32)
    box = np.array([30.0, 30.0, 30.0])
    return rng, pos, types, box


def test_free_flight_closed_form_and_rebuild_schedule():
    hp, m = _light_model(2, 3)
    box = np.array([60.0, 60.0, 60.0])
    # eight atoms on a 20 A grid: no pair within r_c + skin, zero force
    g = np.array([[i, j, k] for i in range(2) for j in range(2) for k in range(2)], dtype=np.float64)
    pos0 = 10.0 + 20.0 * g
    types = np.array([0, 1] * 4, dtype=np.int32)
    rng = np.random.default_rng(0)
    vel0 = rng.uniform(-0.05, 0.05, (8, 3))
    vel0[5] = [0.09, 0.0, 0.0]        # the fastest atom: 0.09 A per step
    masses = np.array([10.0, 200.0])
    steps = 23
    seen = []
    pos, vel, res, rebuilds = velocity_verlet(m, pos0, vel0, types, masses, box, steps,
                                              callback=lambda s, p, v, r: seen.append((s, p.copy())))
    assert np.all(res["F"] == 0.0)
    np.testing.assert_array_equal(vel, vel0)
    for s, p in seen:
        np.testing.assert_allclose(p, pos0 + s * 1.0 * vel0, rtol=0, atol=1e-12)
    # rebuild at multiples of 10 and whenever the fastest atom has gone more
    # than skin/2 = 0.25 A since the last build: 0.27 A after 3 steps (a
    # threshold of 0.3 A would wait for the fourth)
    expect, last = [], 0
    for s in range(1, steps + 1):
        if s % 10 == 0 or (s - last) * 0.09 > 0.25:
            expect.append(s)
            last = s
    assert rebuilds == expect == [3, 6, 9, 10, 13, 16, 19, 20, 23]


def _energy_drift(m, pos0, vel0, types, masses, box, dt, t_total):
    steps = int(round(t_total / dt))
    H = []

    def cb(s, p, v, r):
        H.append(_kinetic(v, masses, types) + r["E"])

    r0 = evaluate(m, pos0, types, box)
    H0 = _kinetic(vel0, masses, types) + r0["E"]
    velocity_verlet(m, pos0, vel0, types, masses, box, steps, dt=dt, callback=cb)
    return np.abs(np.array(H) - H0).max(), H0


def test_energy_conservation_second_order():
    hp, m = _light_model(2, 5)
    rng, pos0, types, box = _cluster(11)
    masses = np.array([12.0, 190.0])   # strongly different masses expose a wrong lookup
    vel0 = synth.maxwell_boltzmann(rng, masses[types], 600.0)
    r0 = evaluate(m, pos0, types, box)
    fmax = np.abs(r0["F"]).max()
    assert fmax > 0.2, fmax       # forces large enough to matter
    d1, H0 = _energy_drift(m, pos0, vel0, types, masses, box, 1.0, 24.0)
    d2, _ = _energy_drift(m, pos0, vel0, types, masses, box, 0.5, 24.0)
    ke0 = _kinetic(vel0, masses, types)
    # the kinetic energy changes by a sizeable fraction over the run, while
    # the total stays constant to a small fraction of that
    assert d1 < 2e-3 * ke0, (d1, ke0)
    ratio = d1 / d2
    assert 3.0 < ratio < 5.5, ratio   # O(dt^2): halving dt divides the error by 4


def test_time_reversible():
    hp, m = _light_model(2, 7)
    rng, pos0, types, box = _cluster(13)
    masses = np.array([30.0, 90.0])
    vel0 = synth.maxwell_boltzmann(rng, masses[types], 800.0)
    p1, v1, _, _ = velocity_verlet(m, pos0, vel0, types, masses, box, 15)
    assert np.abs(p1 - pos0).max() > 0.1       # the atoms did move
    p2, v2, _, _ = velocity_verlet(m, p1, -v1, types, masses, box, 15)
    np.testing.assert_allclose(p2, pos0, rtol=0, atol=1e-10)
    np.testing.assert_allclose(-v2, vel0, rtol=0, atol=1e-11)


def test_active_rows_exact_boundaries_and_sign():
    box = np.array([20.0, 20.0, 20.0])
    rc = 6.0
    inside = np.nextafter(6.0, 0.0)
    pos = np.array([[1.0, 1.0, 1.0],
                    [7.0, 1.0, 1.0],               # dx = 6 exactly: r = r_c, not active
                    [1.0, 1.0 + inside, 1.0],      # one ulp inside r_c: active
                    [1.0, 1.0, 15.0],              # through the face: dz = -6, not active
                    [1.0, 17.0, 1.0],              # through the face: dy = -4, active
                    [3.0, 4.0, 1.0]])              # (2, 3, 0), active
    off, idx = brute_force_neighbors(pos, box, rc + 0.5)
    i, j, d = active_rows(pos, box, off, idx, rc)
    got = {(int(a), int(b)): tuple(v) for a, b, v in zip(i, j, d)}
    assert (0, 1) not in got and (1, 0) not in got
    assert (0, 3) not in got and (3, 0) not in got
    assert got[(0, 2)] == (0.0, inside, 0.0)
    assert got[(2, 0)] == (0.0, -inside, 0.0)
    assert got[(0, 4)] == (0.0, -4.0, 0.0)          # r_j - r_i with the minimum image
    assert got[(4, 0)] == (0.0, 4.0, 0.0)
    assert got[(0, 5)] == (2.0, 3.0, 0.0)
    # every listed pair is either active or has r >= r_c exactly
    listed = {(a, int(b)) for a in range(len(pos)) for b in idx[off[a]:off[a + 1]]}
    assert set(got) <= listed
    assert (0, 1) in listed and (0, 3) in listed


def test_active_rows_matches_periodic_kdtree():
    rng = np.random.default_rng(23)
    box = np.array([16.0, 18.0, 21.0])
    pos = rng.uniform(0.0, 1.0, (400, 3)) * box
    pos[:30] += box * rng.integers(-2, 3, (30, 3))     # outside [0, L)
    rc = 6.0
    off, idx = brute_force_neighbors(pos, box, rc + 0.5)
    i, j, d = active_rows(pos, box, off, idx, rc)
    tree = cKDTree(np.mod(pos, box), boxsize=box)
    ref = set()
    for a, b in tree.query_pairs(rc):
        ref.add((a, b))
        ref.add((b, a))
    assert set(zip(i.tolist(), j.tolist())) == ref
    # r_ij is r_j - r_i up to a lattice translation, and the shortest one
    raw = pos[j] - pos[i]
    shift = (raw - d) / box
    np.testing.assert_allclose(shift, np.round(shift), atol=1e-9)
    assert np.all(np.abs(d) <= box / 2)
    # and its length is the k-d tree's periodic distance
    dist = tree.sparse_distance_matrix(tree, rc, output_type="dict")
    np.testing.assert_allclose(np.linalg.norm(d, axis=1), [dist[(a, b)] for a, b in zip(i.tolist(), j.tolist())],
                               rtol=1e-12)
