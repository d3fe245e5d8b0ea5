"""Synthetic workload recipe: the head-output scale used by the MD workloads
multiplies energies, forces and virials exactly (the head's last layer is
linear, Eq. 6), leaves every other weight untouched, and brings forces on the
thermalised six-component alloy to the size of a trained potential's."""
import numpy as np

import synth
from oracle.model import Model, evaluate


def test_energy_scale_touches_only_the_head_output_layer():
    hp = synth.HParams(n_species=3)
    a = synth.random_weights(hp, 7)
    b = synth.random_weights(hp, 7, energy_scale=0.25)
    pos = 0
    for name, n, _ in synth.weight_segments(hp):
        sa, sb = a[pos:pos + n], b[pos:pos + n]
        if name.endswith(".aout") or name.endswith(".cout"):
            np.testing.assert_array_equal(sb, 0.25 * sa)
        else:
            np.testing.assert_array_equal(sb, sa)
        pos += n
    assert pos == len(a) == len(b)


def test_energy_scale_scales_energy_forces_and_virial():
    w1 = synth.make_workload("fcc-hea6-128", seed=4, n=4)
    ws = synth.make_workload("fcc-hea6-128", seed=4, n=4, energy_scale=synth.PHYSICAL_ENERGY_SCALE)
    np.testing.assert_array_equal(w1.pos, ws.pos)
    r1 = evaluate(Model(w1.hp, w1.weights), w1.pos, w1.types, w1.box)
    rs = evaluate(Model(ws.hp, ws.weights), ws.pos, ws.types, ws.box)
    s = synth.PHYSICAL_ENERGY_SCALE
    for key in ("E_i", "F", "virial"):
        np.testing.assert_allclose(rs[key], s * r1[key], rtol=1e-12, atol=1e-12 * np.abs(r1[key]).max())


def test_scaled_forces_have_physical_size():
    w = synth.make_workload("fcc-hea6-128", seed=0, n=4, energy_scale=synth.PHYSICAL_ENERGY_SCALE)
    r = evaluate(Model(w.hp, w.weights), w.pos, w.types, w.box)
    fn = np.linalg.norm(r["F"], axis=1)
    assert 0.2 < fn.mean() < 5.0, fn.mean()
    # a displacement bound over one list lifetime (10 steps of 1 fs) from the
    # largest acceleration and the fastest atom stays inside half the skin
    acc = fn / w.masses[w.types] * synth.FORCE_TO_ACC
    v = np.linalg.norm(w.vel, axis=1).max()
    assert v * 10 + 0.5 * acc.max() * 10 ** 2 < 0.5 * w.hp.skin
