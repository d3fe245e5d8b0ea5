"""Neighbour sets N(i) for the oracle (Section 3.1: the neighbours of atom i
are the atoms within the cutoff; Section 4.1: lists are built by binning
with a Verlet skin).

Definition used here (periodic orthorhombic box, minimum image):

  * each coordinate is wrapped into [0, L):  w = fmod(x, L); if w < 0 then
    w = w + L; if w >= L then w = w - L  (fmod is exact in IEEE arithmetic);
  * for atoms i, j: dx = w_j - w_i; if dx > L/2 then dx = dx - L, else if
    dx < -L/2 then dx = dx + L  (per component);
  * d2 = (dx*dx + dy*dy) + dz*dz, evaluated in that order without fused
    multiply-add;
  * j is a listed neighbour of i iff j != i and d2 < rl*rl, rl = cutoff+skin.

Every operation is a correctly rounded IEEE double operation, so the set is
exactly reproducible by any implementation that performs the same steps.
Rows are returned sorted by neighbour index (the list is a set; order is not
part of the definition).  The minimum image is only unique when
rl <= min(L)/2, which is required.
"""
from __future__ import annotations

from typing import Iterable, Tuple

import numpy as np


def wrap_positions(pos: np.ndarray, box: np.ndarray) -> np.ndarray:
    box = np.asarray(box, dtype=np.float64)
    w = np.fmod(np.asarray(pos, dtype=np.float64), box)
    w = np.where(w < 0.0, w + box, w)
    w = np.where(w >= box, w - box, w)
    return w


def min_image(d: np.ndarray, box: np.ndarray) -> np.ndarray:
    box = np.asarray(box, dtype=np.float64)
    half = 0.5 * box
    return np.where(d > half, d - box, np.where(d < -half, d + box, d))


def _sq_dist(d: np.ndarray) -> np.ndarray:
    # (dx*dx + dy*dy) + dz*dz, elementwise, no contraction in NumPy
    return (d[..., 0] * d[..., 0] + d[..., 1] * d[..., 1]) + d[..., 2] * d[..., 2]


def _check_box(box: np.ndarray, rl: float) -> None:
    if not rl <= 0.5 * float(np.min(box)):
        raise ValueError(f"list radius {rl} exceeds half the smallest box edge {np.min(box)}")


def _to_csr(rows) -> Tuple[np.ndarray, np.ndarray]:
    counts = np.array([len(r) for r in rows], dtype=np.int64)
    offsets = np.zeros(len(rows) + 1, dtype=np.int64)
    np.cumsum(counts, out=offsets[1:])
    idx = np.concatenate(rows).astype(np.int32) if rows else np.zeros(0, np.int32)
    return offsets, idx


def neighbors_of(pos: np.ndarray, box: np.ndarray, rl: float, rows: Iterable[int]):
    """Brute-force neighbour rows for selected atoms only (O(N) each)."""
    box = np.asarray(box, dtype=np.float64)
    _check_box(box, rl)
    w = wrap_positions(pos, box)
    rl2 = rl * rl
    out = []
    for i in rows:
        d = min_image(w - w[i], box)
        m = _sq_dist(d) < rl2
        m[i] = False
        out.append(np.nonzero(m)[0].astype(np.int32))
    return out


def brute_force_neighbors(pos: np.ndarray, box: np.ndarray, rl: float) -> Tuple[np.ndarray, np.ndarray]:
    """O(N^2) neighbour list; CSR (offsets int64 [N+1], idx int32)."""
    return _to_csr(neighbors_of(pos, box, rl, range(len(pos))))


def cell_list_neighbors(pos: np.ndarray, box: np.ndarray, rl: float) -> Tuple[np.ndarray, np.ndarray]:
    """Same set as brute_force_neighbors, found through a cell list.

    Cells have edge L/nc >= rl, so every pair within rl lies in the same or
    an adjacent cell (periodically); adjacent cell indices are deduplicated
    when nc < 3.  The distance test is the same exact test as above."""
    box = np.asarray(box, dtype=np.float64)
    _check_box(box, rl)
    w = wrap_positions(pos, box)
    N = len(w)
    nc = np.maximum(1, np.floor(box / (rl * (1.0 + 1e-9))).astype(np.int64))
    cidx = np.minimum((w / (box / nc)).astype(np.int64), nc - 1)
    flat = (cidx[:, 2] * nc[1] + cidx[:, 1]) * nc[0] + cidx[:, 0]
    order = np.argsort(flat, kind="stable")
    ncell = int(nc.prod())
    start = np.searchsorted(flat[order], np.arange(ncell + 1))
    rl2 = rl * rl
    rows = [None] * N

    def adj(c, n):
        return sorted({(c + o) % n for o in (-1, 0, 1)})

    for cz in range(nc[2]):
        for cy in range(nc[1]):
            for cx in range(nc[0]):
                c = (cz * nc[1] + cy) * nc[0] + cx
                mine = order[start[c]:start[c + 1]]
                if len(mine) == 0:
                    continue
                cand = []
                for zz in adj(cz, nc[2]):
                    for yy in adj(cy, nc[1]):
                        for xx in adj(cx, nc[0]):
                            cc = (zz * nc[1] + yy) * nc[0] + xx
                            cand.append(order[start[cc]:start[cc + 1]])
                cand = np.concatenate(cand)
                d = min_image(w[cand][None, :, :] - w[mine][:, None, :], box)
                m = _sq_dist(d) < rl2
                m &= cand[None, :] != mine[:, None]
                for r, i in enumerate(mine):
                    rows[i] = np.sort(cand[m[r]]).astype(np.int32)
    return _to_csr(rows)


def neighbor_list(pos: np.ndarray, box: np.ndarray, rl: float) -> Tuple[np.ndarray, np.ndarray]:
    """Brute force for small systems, cell list otherwise (same set)."""
    if len(pos) <= 5000:
        return brute_force_neighbors(pos, box, rl)
    return cell_list_neighbors(pos, box, rl)


def active_rows(pos: np.ndarray, box: np.ndarray, offsets: np.ndarray, idx: np.ndarray, rc: float):
    """Listed pairs (i, j) with distance below the cutoff, and their r_ij
    vectors (Eq. 1: r_ij = r_j - r_i, minimum image)."""
    box = np.asarray(box, dtype=np.float64)
    N = len(offsets) - 1
    i = np.repeat(np.arange(N, dtype=np.int64), np.diff(offsets))
    j = idx.astype(np.int64)
    w = wrap_positions(pos, box)
    d = min_image(w[j] - w[i], box)
    keep = _sq_dist(d) < rc * rc
    return i[keep], j[keep], d[keep]


def list_radius(cutoff: float, skin: float) -> float:
    return cutoff + skin


__all__ = ["wrap_positions", "min_image", "neighbors_of", "brute_force_neighbors",
           "cell_list_neighbors", "neighbor_list", "active_rows", "list_radius"]
