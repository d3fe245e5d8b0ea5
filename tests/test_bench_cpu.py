"""Accounting in bench.py: the algorithmic FLOP counts behind the roofline
fraction against the closed forms of the architecture (encoder 1 -> 128,
two 128 -> 128 layers, 128 -> k, forward and tangent; head (l_max+1)k -> 64,
three 64 -> 64 layers, 64 -> 1, forward and backward; Eqs. 2-10), and the
neighbour-build record's byte count."""
import bench
import synth


def test_flops_per_pair_and_atom_closed_forms():
    hp = synth.HParams()
    # per pair: 2 FLOP per MAC x (forward + tangent) x (128 + 2 * 128^2 + 128 k), plus
    # the moment and the two W contractions, 2 FLOP x d k each
    assert bench.flops_per_pair(hp) == 151_040
    assert bench.flops_per_atom(hp) == 4 * (4 * 32 * 64 + 3 * 64 * 64 + 64) == 82_176
    for k, want in ((16, 141_312), (64, 170_496)):
        hp.k = k
        assert bench.flops_per_pair(hp) == want
    hp = synth.HParams(angular=1)   # Cartesian basis to l = 3: 1 + 3 + 6 + 10 = 20 rows
    assert bench.flops_per_pair(hp) == 4 * (128 + 2 * 128 * 128 + 128 * 32) + 6 * 20 * 32
    hp = synth.HParams(lmax=5)      # irreducible to l = 5: 36 rows; head input 6 k
    assert bench.flops_per_pair(hp) == 4 * (128 + 2 * 128 * 128 + 128 * 32) + 6 * 36 * 32
    assert bench.flops_per_atom(hp) == 4 * (6 * 32 * 64 + 3 * 64 * 64 + 64)


def test_neighbour_build_record_without_timed_rebuilds():
    r = bench.neighbour_build_record([], 40.0, 1000, 90_000, 4)
    assert r["ms"] == 40.0 and r["timed_rebuilds"] == 0
    assert r["algorithmic_bytes"] == 72 * 1000 + 4 * 90_000
    assert bench.neighbour_build_record([], 40.0, 1000, 90_000, 2)["algorithmic_bytes"] == 72 * 1000 + 2 * 90_000
    assert abs(r["gbps"] - r["algorithmic_bytes"] / 0.040 / 1e9) < 1e-12
    assert abs(r["frac_of_hbm"] - r["gbps"] / bench.PEAK_HBM_GBS) < 1e-15


def test_more_than_one_gpu_is_refused_with_a_message():
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and not r.stdout.strip()


def test_largest_system_run_is_read_from_the_sweep_summary():
    r = bench.largest_system_run()
    assert r is not None and r["atoms"] > 10 ** 9 and 100 < r["bytes_per_atom"] < 1000
