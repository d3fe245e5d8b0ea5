"""Seeded synthetic inputs for the MLIP energy/force/virial path.

This module is the only code shared by the CPU oracle side (tests, the
oracle's CPU baseline) and the HIP side (tests, bench, smoke).  It draws
random numbers and lays them out; it holds none of the method's arithmetic
(no descriptor, network, force or neighbour computation).

Workloads follow the shapes of the paper's bulk-material evaluation
(Section 4.1: unary, ternary and six-component alloys, cutoff 6 A,
k = 32, l_max = 3, encoder 3 x 128, head 4 x 64): cubic FCC/BCC supercells
with Gaussian displacements, species drawn per site, random-init weights
N(0, 1/fan_in).  The paper's trained models and DFT datasets are not used;
these seeded inputs stand in for them.

Weight-blob layout (flat float64, row-major, matrices stored [out][in]):

  encoder tables, index tau = s_i*C + s_j (pair conditioning),
  s_j (neighbour conditioning) or 0 (universal), each:
      w0[W], b0[W],
      then for t = 1 .. enc_hidden-1:  W_t[W][W], b_t[W],
      W_out[k][W], b_out[k]
  head tables, index rho = s_i (species conditioning) or 0, each:
      A0[R][(l_max+1)*k], c0[R],
      then for t = 1 .. reg_hidden-1:  A_t[R][R], c_t[R],
      a_out[R], c_out[1]

with W = enc_width and R = reg_width.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Tuple

import numpy as np

# Public standard atomic weights (amu) used as synthetic species masses.
MASS = {
    "Cu": 63.546, "Ni": 58.693, "Mo": 95.95, "Al": 26.982, "Mg": 24.305,
    "Ta": 180.948, "Nb": 92.906, "W": 183.84, "V": 50.942, "Sn": 118.71,
}

# Boltzmann constant in eV/K (metal units).
KB_EV = 8.617333262e-5
# (eV/A) / amu -> A/fs^2
FORCE_TO_ACC = 9.648533212e-3


@dataclasses.dataclass
class HParams:
    """Hyper-parameters of the model (Section 3, Section 4.1 architecture)."""

    n_species: int = 1
    cutoff: float = 6.0
    skin: float = 0.5
    k: int = 32
    lmax: int = 3
    angular: int = 0      # 0 irreducible harmonic basis, 1 Cartesian monomials
    enc_cond: int = 2     # 2 (s_i, s_j) pairs, 1 s_j, 0 universal
    reg_cond: int = 1     # 1 s_i, 0 universal
    enc_width: int = 128
    enc_hidden: int = 3
    reg_width: int = 64
    reg_hidden: int = 4
    precision: int = 64

    def n_enc_tables(self) -> int:
        C = self.n_species
        return {2: C * C, 1: C, 0: 1}[self.enc_cond]

    def n_head_tables(self) -> int:
        return self.n_species if self.reg_cond == 1 else 1

    def head_in(self) -> int:
        return (self.lmax + 1) * self.k


def weight_segments(hp: HParams) -> List[Tuple[str, int, int]]:
    """(name, count, fan_in) for every segment of the weight blob, in order."""
    W, R, k = hp.enc_width, hp.reg_width, hp.k
    segs: List[Tuple[str, int, int]] = []
    for t in range(hp.n_enc_tables()):
        segs += [(f"enc{t}.w0", W, 1), (f"enc{t}.b0", W, 1)]
        for h in range(1, hp.enc_hidden):
            segs += [(f"enc{t}.W{h}", W * W, W), (f"enc{t}.b{h}", W, W)]
        segs += [(f"enc{t}.Wout", k * W, W), (f"enc{t}.bout", k, W)]
    for t in range(hp.n_head_tables()):
        segs += [(f"head{t}.A0", R * hp.head_in(), hp.head_in()), (f"head{t}.c0", R, hp.head_in())]
        for h in range(1, hp.reg_hidden):
            segs += [(f"head{t}.A{h}", R * R, R), (f"head{t}.c{h}", R, R)]
        segs += [(f"head{t}.aout", R, R), (f"head{t}.cout", 1, R)]
    return segs


def weight_count(hp: HParams) -> int:
    return sum(n for _, n, _ in weight_segments(hp))


# Factor on the energy head's output layer for workloads that run MD.  With
# every layer drawn N(0, 1/fan_in) the descriptor is unnormalised and a
# thermalised alloy sees forces of about 100 eV/A, which carry atoms past half
# the neighbour-list skin within a few 1 fs steps and melt the lattice.  Scaled
# by this factor the mean force is about 1 eV/A, the size a trained potential
# gives near 300 K, so the list lasts its 10 steps as in production runs.  The
# values change no work: every pair and atom is evaluated the same way.
PHYSICAL_ENERGY_SCALE = 0.01


def random_weights(hp: HParams, seed: int, scale: float = 1.0, energy_scale: float = 1.0) -> np.ndarray:
    """Weights and biases drawn N(0, scale^2/fan_in), segment by segment; the
    head's output layer (weights and bias) is then multiplied by energy_scale,
    which scales energies, forces and virials by the same factor."""
    rng = np.random.default_rng(seed)
    segs = weight_segments(hp)
    parts = [rng.normal(0.0, scale / math.sqrt(fan), n) for _, n, fan in segs]
    if energy_scale != 1.0:
        for i, (name, _, _) in enumerate(segs):
            if name.endswith(".aout") or name.endswith(".cout"):
                parts[i] = parts[i] * energy_scale
    return np.concatenate(parts).astype(np.float64)


def scale_segments(hp: HParams, weights: np.ndarray, suffix: str, factor: float) -> np.ndarray:
    """Copy of a weight blob with every segment whose name ends in `suffix`
    (for example ".A0", the head's first layer in each head table)
    multiplied by `factor`."""
    out = np.array(weights, dtype=np.float64, copy=True)
    pos = 0
    for name, n, _ in weight_segments(hp):
        if name.endswith(suffix):
            out[pos:pos + n] *= factor
        pos += n
    assert pos == len(out)
    return out


def lattice(kind: str, n: int, a: float) -> Tuple[np.ndarray, np.ndarray]:
    """Cubic n x n x n supercell of an FCC or BCC lattice, sites ordered
    (ix, iy, iz, basis).  Returns positions [N][3] and the box edges."""
    if kind == "fcc":
        basis = np.array([[0, 0, 0], [0, .5, .5], [.5, 0, .5], [.5, .5, 0]])
    elif kind == "bcc":
        basis = np.array([[0, 0, 0], [.5, .5, .5]])
    else:
        raise ValueError(kind)
    g = np.arange(n, dtype=np.float64)
    ix, iy, iz = np.meshgrid(g, g, g, indexing="ij")
    cells = np.stack([ix.ravel(), iy.ravel(), iz.ravel()], axis=1)
    pos = (cells[:, None, :] + basis[None, :, :]).reshape(-1, 3) * a
    box = np.array([n * a] * 3, dtype=np.float64)
    return pos.astype(np.float64), box


def species_exact(rng: np.random.Generator, N: int, fractions) -> np.ndarray:
    counts = [int(round(f * N)) for f in fractions]
    counts[0] += N - sum(counts)
    t = np.concatenate([np.full(c, s, dtype=np.int32) for s, c in enumerate(counts)])
    rng.shuffle(t)
    return t


def species_iid(rng: np.random.Generator, N: int, C: int) -> np.ndarray:
    return rng.integers(0, C, N).astype(np.int32)


def maxwell_boltzmann(rng: np.random.Generator, masses: np.ndarray, T: float) -> np.ndarray:
    """Velocities (A/fs) at temperature T with zero total momentum, rescaled
    so the kinetic temperature over 3N-3 degrees of freedom is exactly T."""
    N = masses.shape[0]
    v = rng.normal(size=(N, 3)) * np.sqrt(KB_EV * T * FORCE_TO_ACC / masses)[:, None]
    p = (masses[:, None] * v).sum(0)
    v -= p / masses.sum()
    ke = 0.5 * (masses[:, None] * v * v).sum() / FORCE_TO_ACC
    dof = max(3 * N - 3, 1)
    if ke > 0:
        v *= math.sqrt(0.5 * dof * KB_EV * T / ke)
    return v


@dataclasses.dataclass
class Workload:
    name: str
    pos: np.ndarray          # [N][3] float64, A
    types: np.ndarray        # [N] int32
    box: np.ndarray          # [3] float64, A
    vel: np.ndarray          # [N][3] float64, A/fs
    masses: np.ndarray       # [C] float64, amu
    hp: HParams
    weights: np.ndarray      # flat float64 blob
    steps: int
    rebuild_every: int
    dt: float
    seed: int
    description: str


# Named workloads: shapes of the paper's bulk systems (binary FCC, unary
# BCC metal, dilute ternary FCC, six-component random FCC, BCC capacity sweep).
PRESETS: Dict[str, dict] = {
    "fcc-binary-4": dict(kind="fcc", n=4, a=3.6, C=2, frac=(0.5, 0.5), sigma=0.05, cutoff=6.0,
                         T=300.0, steps=10, masses=("Cu", "Ni"),
                         desc="binary FCC 4^3 (256 atoms), a=3.6, 50/50, sigma=0.05, rc=6.0"),
    "bcc-unary-32": dict(kind="bcc", n=32, a=3.2, C=1, frac=(1.0,), sigma=0.08, cutoff=6.0,
                         T=300.0, steps=100, masses=("Mo",),
                         desc="unary BCC 32^3 (65,536 atoms), a=3.2, sigma=0.08, rc=6.0"),
    "fcc-ternary-64": dict(kind="fcc", n=64, a=4.05, C=3, frac=(0.90, 0.05, 0.05), sigma=0.1,
                           cutoff=6.5, T=600.0, steps=100, masses=("Al", "Cu", "Mg"),
                           desc="dilute ternary FCC 64^3 (1,048,576 atoms), a=4.05, 0.90/0.05/0.05, "
                                "sigma=0.1, rc=6.5"),
    "fcc-hea6-128": dict(kind="fcc", n=128, a=3.6, C=6, frac=None, sigma=0.1, cutoff=6.0,
                         T=300.0, steps=50, masses=("Ta", "Nb", "W", "Mo", "V", "Al"),
                         desc="6-component equiatomic random FCC 128^3 (8,388,608 atoms), a=3.6, "
                              "sigma=0.1, rc=6.0"),
    "bcc-hea6-sweep": dict(kind="bcc", n=128, a=3.2, C=6, frac=None, sigma=0.1, cutoff=6.0,
                           T=300.0, steps=20, masses=("Ta", "Nb", "W", "Mo", "V", "Al"),
                           desc="6-component equiatomic random BCC L^3 capacity sweep, a=3.2, "
                                "sigma=0.1, rc=6.0"),
}


def make_workload(name: str, seed: int = 0, n: Optional[int] = None, skin: float = 0.5,
                  hp_overrides: Optional[dict] = None, weight_scale: float = 1.0,
                  energy_scale: float = 1.0) -> Workload:
    """Build a named workload.  `n` overrides the supercell edge (in cells)."""
    p = PRESETS[name]
    rng = np.random.default_rng(seed)
    ncell = p["n"] if n is None else n
    pos, box = lattice(p["kind"], ncell, p["a"])
    N = pos.shape[0]
    C = p["C"]
    if p["frac"] is not None:
        types = species_exact(rng, N, p["frac"])
    else:
        types = species_iid(rng, N, C)
    pos = pos + rng.normal(0.0, p["sigma"], (N, 3))
    masses = np.array([MASS[e] for e in p["masses"]], dtype=np.float64)
    vel = maxwell_boltzmann(rng, masses[types], p["T"])
    hp = HParams(n_species=C, cutoff=p["cutoff"], skin=skin)
    for key, val in (hp_overrides or {}).items():
        setattr(hp, key, val)
    weights = random_weights(hp, seed + 1, weight_scale, energy_scale)
    return Workload(name=name, pos=pos, types=types, box=box, vel=vel, masses=masses, hp=hp,
                    weights=weights, steps=p["steps"], rebuild_every=10, dt=1.0, seed=seed,
                    description=p["desc"] if n is None else f"{p['desc']} (edge {ncell})")


def random_cluster(rng: np.random.Generator, N: int, C: int, radius: float,
                   min_dist: float = 1.8) -> np.ndarray:
    """Non-periodic cluster: N points in a ball, rejection-sampled so no two
    are closer than min_dist.  Returns positions [N][3]."""
    pts: List[np.ndarray] = []
    while len(pts) < N:
        p = rng.uniform(-radius, radius, 3)
        if np.linalg.norm(p) > radius:
            continue
        if all(np.linalg.norm(p - q) >= min_dist for q in pts):
            pts.append(p)
    return np.array(pts, dtype=np.float64)


def lattice_stream(kind: str, n: int, a: float, C: int, sigma: float, masses, T: float, seed: int,
                   planes: int = 16):
    """Large cubic supercells generated a few ix-planes at a time (same site
    order as `lattice`): yields (first_site, positions, species, velocities)
    chunks so that no host array of the full system is needed.  Species are
    i.i.d. uniform over C; velocities are Maxwell-Boltzmann at T per site
    (no total-momentum removal or exact rescaling at this size)."""
    if kind == "fcc":
        basis = np.array([[0, 0, 0], [0, .5, .5], [.5, 0, .5], [.5, .5, 0]])
    elif kind == "bcc":
        basis = np.array([[0, 0, 0], [.5, .5, .5]])
    else:
        raise ValueError(kind)
    rng = np.random.default_rng(seed)
    masses = np.asarray(masses, dtype=np.float64)
    g = np.arange(n, dtype=np.float64)
    iy, iz = np.meshgrid(g, g, indexing="ij")
    plane = np.stack([iy.ravel(), iz.ravel()], axis=1)
    first = 0
    for x0 in range(0, n, planes):
        xs = np.arange(x0, min(n, x0 + planes), dtype=np.float64)
        cells = np.concatenate([np.column_stack([np.full(len(plane), x), plane]) for x in xs])
        pos = ((cells[:, None, :] + basis[None, :, :]).reshape(-1, 3) * a)
        m = len(pos)
        types = rng.integers(0, C, m).astype(np.int32)
        pos += rng.normal(0.0, sigma, (m, 3))
        vel = rng.normal(size=(m, 3)) * np.sqrt(KB_EV * T * FORCE_TO_ACC / masses[types])[:, None]
        yield first, pos, types, vel
        first += m
