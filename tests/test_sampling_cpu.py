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
