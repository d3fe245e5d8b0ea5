"""Angular feature vectors (Section 3.3).

The order-l block of the canonical (reducible) angular feature holds every
Cartesian monomial u_x^a u_y^b u_z^c of the unit direction u with
a + b + c = l (Eq. for the reducible dimension: sum of C(l+2, 2)).  Monomials
are ordered lexicographically with x first, e.g. l = 2: x^2, xy, xz, y^2,
yz, z^2, as listed in the paper.

The irreducible harmonic projection (Section 3.3, "Irreducible Harmonic
Projection") left-multiplies the order-l block by Q_l with (2l+1) rows,
fixed by two constraints: L_l Q_l^T = 0, where L_l is the Laplacian acting on
coefficient vectors of degree-l homogeneous polynomials, and
Q_l D_l^{-1} Q_l^T = I, where D_l = diag(l! / (a! b! c!)).

Readings of the paper taken here:
  * the paper also writes Q_l Q_l^T = I; the two-constraint definition with
    D_l^{-1} is the one used (the other is inconsistent with it for l >= 2);
  * D_l is square of size C(l+2, 2) (the printed size l x l is a typo);
  * Q_l is unique up to a (2l+1) x (2l+1) orthogonal factor; the descriptor
    uses only squared norms for l >= 1, so it does not depend on that factor.
    For l = 0 the single row is fixed to +1 (the descriptor's l = 0 block is
    linear, so its sign matters);
  * the metric C_l of Eq. 5 is the identity for the irreducible basis and
    D_l (the Cartesian multiplicities) for the canonical basis.

Construction: a basis of ker(L_l) from the SVD of L_l, then symmetric
(Loewdin) orthonormalisation in the D_l^{-1} inner product.
"""
from __future__ import annotations

import math
from functools import lru_cache
from typing import List, Tuple

import numpy as np


def monomial_exponents(l: int) -> List[Tuple[int, int, int]]:
    out = []
    for a in range(l, -1, -1):
        for b in range(l - a, -1, -1):
            out.append((a, b, l - a - b))
    return out


def multinomial_diag(l: int) -> np.ndarray:
    return np.array([math.factorial(l) / (math.factorial(a) * math.factorial(b) * math.factorial(c))
                     for a, b, c in monomial_exponents(l)], dtype=np.float64)


def laplacian_matrix(l: int) -> np.ndarray:
    """L_l: coefficients of a degree-l polynomial -> coefficients of its
    Laplacian (degree l-2).  Shape [C(l,2)][C(l+2,2)]."""
    cols = monomial_exponents(l)
    if l < 2:
        return np.zeros((0, len(cols)))
    rows = {e: r for r, e in enumerate(monomial_exponents(l - 2))}
    L = np.zeros((len(rows), len(cols)))
    for c, (a, b, cc) in enumerate(cols):
        if a >= 2:
            L[rows[(a - 2, b, cc)], c] += a * (a - 1)
        if b >= 2:
            L[rows[(a, b - 2, cc)], c] += b * (b - 1)
        if cc >= 2:
            L[rows[(a, b, cc - 2)], c] += cc * (cc - 1)
    return L


@lru_cache(maxsize=None)
def harmonic_projection(l: int) -> np.ndarray:
    """Q_l, shape [2l+1][C(l+2,2)], satisfying L_l Q_l^T = 0 and
    Q_l D_l^{-1} Q_l^T = I."""
    n = (l + 1) * (l + 2) // 2
    if l == 0:
        return np.ones((1, 1))
    L = laplacian_matrix(l)
    if L.shape[0] == 0:
        basis = np.eye(n)
    else:
        _, s, vt = np.linalg.svd(L)
        rank = int(np.sum(s > 1e-10 * s.max()))
        basis = vt[rank:]                                  # rows span ker(L)
    dinv = np.diag(1.0 / multinomial_diag(l))
    gram = basis @ dinv @ basis.T
    ev, U = np.linalg.eigh(gram)
    q = (U @ np.diag(ev ** -0.5) @ U.T) @ basis
    q.setflags(write=False)
    return q


def angular_basis(lmax: int, kind: int):
    """Per-order blocks (projection P_l mapping monomials to features, metric
    C_l).  kind 0 = irreducible (P_l = Q_l, C_l = I), kind 1 = Cartesian
    (P_l = I, C_l = D_l)."""
    blocks = []
    for l in range(lmax + 1):
        n = (l + 1) * (l + 2) // 2
        if kind == 0:
            proj = harmonic_projection(l)
            metric = np.eye(2 * l + 1)
        elif kind == 1:
            proj = np.eye(n)
            metric = np.diag(multinomial_diag(l))
        else:
            raise ValueError(kind)
        blocks.append((proj, metric))
    return blocks


def angular_dim(lmax: int, kind: int) -> int:
    return sum(b[0].shape[0] for b in angular_basis(lmax, kind))


def _monomials(u: np.ndarray, l: int):
    """Values [n][C(l+2,2)] and gradients [n][C(l+2,2)][3] w.r.t. u."""
    ex = monomial_exponents(l)
    n = u.shape[0]
    val = np.empty((n, len(ex)))
    grad = np.zeros((n, len(ex), 3))
    for c, e in enumerate(ex):
        val[:, c] = u[:, 0] ** e[0] * u[:, 1] ** e[1] * u[:, 2] ** e[2]
        for ax in range(3):
            if e[ax] == 0:
                continue
            e2 = list(e)
            e2[ax] -= 1
            grad[:, c, ax] = e[ax] * u[:, 0] ** e2[0] * u[:, 1] ** e2[1] * u[:, 2] ** e2[2]
    return val, grad


def angular_features(u: np.ndarray, lmax: int, kind: int = 0):
    """g^angular (Eq. 3) at unit vectors u [n][3]: values [n][d] and the
    gradient with respect to u, [n][d][3] (u treated as a free vector)."""
    vals, grads = [], []
    for l, (proj, _) in enumerate(angular_basis(lmax, kind)):
        m, dm = _monomials(u, l)
        vals.append(m @ proj.T)
        grads.append(np.einsum("pq,nqa->npa", proj, dm))
    return np.concatenate(vals, axis=1), np.concatenate(grads, axis=1)


def block_slices(lmax: int, kind: int):
    """Row ranges of each order-l block inside the d-dimensional feature."""
    out, s = [], 0
    for proj, metric in angular_basis(lmax, kind):
        out.append((slice(s, s + proj.shape[0]), metric))
        s += proj.shape[0]
    return out
