"""mlip_compute_noalloc, the entry point that allocates nothing (a fixed
per-device scratch holds the fused kernel's workspace, totals and counter),
against mlip_compute on the same context: two calls in a row, the second on
a smaller system, in both single-kernel configurations and both precisions;
the configurations it does not run and a workspace beyond the scratch are
rejected with MLIP_E_ARG."""
import numpy as np
import pytest

import synth
from tests.gpu_helpers import to_dev, log, max_abs

pytestmark = pytest.mark.gpu


def _outputs(n, fill):
    import torch
    dev = torch.device("cuda:0")
    return (torch.full((n, 3), fill, dtype=torch.float64, device=dev),
            torch.full((n,), fill, dtype=torch.float64, device=dev),
            torch.full((n, 9), fill, dtype=torch.float64, device=dev))


def _bar(precision, ref):
    # the bar of the parity tests: 1e-9 absolute in float64, 1e-4 of the
    # array's largest magnitude in float32
    return 1e-9 if precision == 64 else 1e-4 * max(1.0, float(np.abs(ref).max()))


@pytest.mark.parametrize("precision", [64, 32])
@pytest.mark.parametrize("fusion", [0, 1])
def test_noalloc_matches_compute_twice_second_smaller(precision, fusion):
    import torch
    from paper_2608_16329_amd import Potential
    big = synth.make_workload("fcc-hea6-128", seed=31, n=8, hp_overrides={"precision": precision})   # 2,048 atoms
    small = synth.make_workload("fcc-hea6-128", seed=32, n=5, hp_overrides={"precision": precision})  # 500 atoms
    pot = Potential(big.hp, big.weights)
    pot.set_fusion(fusion)
    for call, w in enumerate((big, small)):
        n = len(w.pos)
        pos, types = to_dev(w.pos), to_dev(w.types)
        pot.build_neighbors(pos, types, w.box)
        F0, E0, V0 = _outputs(n, 0.0)
        t0 = pot.compute(pos, F0, E0, V0, totals=True)
        act0 = pot.stats()["n_active_pairs"]
        F1, E1, V1 = _outputs(n, float("nan"))    # every entry must be written
        t1 = pot.compute_noalloc(pos, F1, E1, V1, totals=True)
        torch.cuda.synchronize()
        act1 = pot.stats()["n_active_pairs"]
        res = [(a.cpu().numpy(), b.cpu().numpy()) for a, b in ((E0, E1), (F0, F1), (V0, V1))]
        errs = [max_abs(a, b) for a, b in res]
        log(f"[noalloc] precision {precision} fusion {fusion} call {call + 1}: N={n} max|dE|={errs[0]:.2e} "
            f"max|dF|={errs[1]:.2e} max|dW|={errs[2]:.2e}")
        for (a, b), e in zip(res, errs):
            assert np.all(np.isfinite(b))
            assert e <= _bar(precision, a), e
        assert max_abs(t0, t1) <= 1e-9 * n * max(1.0, float(np.abs(t0).max()))
        assert act0 == act1 > 0
    pot.close()


def test_noalloc_rejects_what_it_cannot_run():
    """The three-kernel configuration (per-atom intermediates) and a
    workspace larger than the scratch: MLIP_E_ARG with the reason; the same
    context still evaluates through mlip_compute."""
    import torch
    from paper_2608_16329_amd import Potential, MlipError
    w = synth.make_workload("fcc-binary-4", seed=5)
    pot = Potential(w.hp, w.weights)
    pos, types = to_dev(w.pos), to_dev(w.types)
    pot.build_neighbors(pos, types, w.box)
    F, E, V = _outputs(len(w.pos), 0.0)
    pot.set_fusion(2)
    with pytest.raises(MlipError, match="ARG.*single-kernel"):
        pot.compute_noalloc(pos, F, E, V)
    pot.close()
    # 16 species, k = 64, cutoff 6.5: 8-atom tiles of about 110 neighbours
    # in up to 16 species buckets need about 1.2 MB of workspace per
    # work-group, beyond 256 MiB over 256 work-groups
    rng = np.random.default_rng(7)
    hp = synth.HParams(n_species=16, k=64, cutoff=6.5)
    p, box = synth.lattice("fcc", 8, 3.6)
    p = p + rng.normal(0.0, 0.05, p.shape)
    t = rng.integers(0, 16, len(p)).astype(np.int32)
    pot = Potential(hp, synth.random_weights(hp, 3))
    pos = to_dev(p)
    pot.build_neighbors(pos, to_dev(t), box)
    st = pot.stats()
    log(f"[noalloc] 16 species k=64: {st['n_blocks']} work-groups, tile {st['tile_atoms']}, max row {st['max_row']}")
    F, E, V = _outputs(len(p), 0.0)
    with pytest.raises(MlipError, match="ARG.*workspace needs"):
        pot.compute_noalloc(pos, F, E, V)
    pot.compute(pos, F, E, V)
    torch.cuda.synchronize()
    assert np.all(np.isfinite(F.cpu().numpy())) and float(F.abs().max()) > 0.0
    pot.close()
