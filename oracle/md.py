"""Velocity-Verlet NVE driver around the oracle (the paper runs its MLIP
inside LAMMPS molecular dynamics with a 1 fs step, Section 4.1).

Metal units: A, fs, amu, eV.  Acceleration = F/m * 9.648533212e-3 A/fs^2 per
(eV/A)/amu.  Schedule per step s = 1..steps: half kick, drift, rebuild the
neighbour list when s is a multiple of `rebuild_every` or when some atom has
moved more than skin/2 since the last build, evaluate forces, half kick.
This is a driver for trajectory comparisons, not part of the method.
"""
from __future__ import annotations

import numpy as np

from .model import evaluate
from .neighbors import neighbor_list

ACC_PER_FORCE_MASS = 9.648533212e-3


def velocity_verlet(model, pos, vel, types, masses, box, steps, dt=1.0, rebuild_every=10,
                    callback=None):
    pos = np.array(pos, dtype=np.float64)
    vel = np.array(vel, dtype=np.float64)
    inv_m = ACC_PER_FORCE_MASS / np.asarray(masses, dtype=np.float64)[np.asarray(types)]
    rl = model.rc + model.skin
    offsets, idx = neighbor_list(pos, box, rl)
    ref = pos.copy()
    res = evaluate(model, pos, types, box, offsets, idx)
    rebuilds = []
    for s in range(1, steps + 1):
        vel += 0.5 * dt * res["F"] * inv_m[:, None]
        pos += dt * vel
        disp2 = ((pos - ref) ** 2).sum(1).max()
        if s % rebuild_every == 0 or disp2 > (0.5 * model.skin) ** 2:
            offsets, idx = neighbor_list(pos, box, rl)
            ref = pos.copy()
            rebuilds.append(s)
        res = evaluate(model, pos, types, box, offsets, idx)
        vel += 0.5 * dt * res["F"] * inv_m[:, None]
        if callback is not None:
            callback(s, pos, vel, res)
    return pos, vel, res, rebuilds
