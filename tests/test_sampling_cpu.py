"""The per-atom sampling used by the full-size GPU parity tests (a local
cluster cut out of the periodic system around each sampled atom) reproduces
the oracle's full periodic evaluation."""
import numpy as np

import synth
from oracle.model import Model, evaluate
from tests.gpu_helpers import oracle_sample


def test_local_cluster_sampling_matches_full_evaluation():
    w = synth.make_workload("bcc-hea6-sweep", seed=3, n=10)   # 2,000 atoms, 32 A box
    m = Model(w.hp, w.weights)
    full = evaluate(m, w.pos, w.types, w.box)
    atoms = [0, 100, 777, 1999]
    E, F, V = oracle_sample(m, w.pos, w.types, w.box, atoms)
    np.testing.assert_allclose(E, full["E_i"][atoms], rtol=1e-13, atol=1e-10)
    np.testing.assert_allclose(F, full["F"][atoms], atol=1e-10)
    np.testing.assert_allclose(V, full["virial"][atoms], atol=1e-10)


def test_cube_cutout_matches_periodic_evaluation():
    """The cube cut-out used at full size (a corner cube, so it straddles
    every periodic face) gives the oracle's periodic E_i, F_i and virial."""
    from oracle.model import forces_for
    from oracle.neighbors import neighbor_list
    from tests.gpu_helpers import oracle_cube
    w = synth.make_workload("bcc-hea6-sweep", seed=4, n=14)    # 5,488 atoms, 44.8 A box
    m = Model(w.hp, w.weights)
    atoms, E, F, V = oracle_cube(m, w.pos, w.types, w.box, np.zeros(3), 5.0)
    assert len(atoms) > 40
    pick = np.arange(0, len(atoms), max(1, len(atoms) // 6))
    off, idx = neighbor_list(w.pos, w.box, m.rc + m.skin)
    ref = forces_for(m, w.pos, w.types, w.box, atoms[pick], off, idx)
    np.testing.assert_allclose(E[pick], ref["E_i"], rtol=1e-13, atol=1e-10)
    np.testing.assert_allclose(F[pick], ref["F"], atol=1e-10)
    np.testing.assert_allclose(V[pick], ref["virial"], atol=1e-10)
