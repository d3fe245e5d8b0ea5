"""Pins for the oracle's angular basis (Section 3.3) against values the
paper prints and against mathematics independent of the oracle's own
construction (Legendre polynomials, numerical Laplacians, sphere quadrature)."""
import math
import os

import numpy as np
import pytest
from scipy.special import eval_legendre

from oracle import angular

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _rows(name):
    out = []
    with open(os.path.join(GOLD, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                out.append([float(x) for x in line.split()])
    return out


def test_dimension_table_matches_paper():
    for lmax, orig, red in _rows("angular_dims.txt"):
        lmax = int(lmax)
        assert angular.angular_dim(lmax, 1) == int(orig)
        assert angular.angular_dim(lmax, 0) == int(red)
        # Eq. for the reducible dimension and (lmax+1)^2 for the reduced one
        assert int(orig) == (lmax + 1) * (lmax + 2) * (lmax + 3) // 6
        assert int(red) == (lmax + 1) ** 2


def test_monomial_order_matches_paper():
    rows = _rows("monomial_order.txt")
    got = [(l, e) for l in range(3) for e in angular.monomial_exponents(l)]
    assert len(got) == len(rows)
    for (l, e), r in zip(got, rows):
        assert l == int(r[0]) and e == tuple(int(x) for x in r[1:])


@pytest.mark.parametrize("l", range(6))
def test_projection_constraints(l):
    q = angular.harmonic_projection(l)
    D = angular.multinomial_diag(l)
    assert q.shape == (2 * l + 1, (l + 1) * (l + 2) // 2)
    np.testing.assert_allclose(q @ np.diag(1 / D) @ q.T, np.eye(2 * l + 1), atol=1e-12)
    L = angular.laplacian_matrix(l)
    if L.size:
        np.testing.assert_allclose(L @ q.T, 0.0, atol=1e-12)
    assert np.linalg.matrix_rank(q) == 2 * l + 1
    if l == 0:
        assert q[0, 0] == 1.0


def test_multinomial_diag_values():
    # l!/(a!b!c!) for the l = 2 order x^2, xy, xz, y^2, yz, z^2
    np.testing.assert_array_equal(angular.multinomial_diag(2), [1, 2, 2, 1, 2, 1])
    # sum of multinomial coefficients of degree l in 3 variables is 3^l
    for l in range(6):
        assert angular.multinomial_diag(l).sum() == 3 ** l


@pytest.mark.parametrize("l", range(6))
def test_rows_are_harmonic_by_finite_differences(l):
    """Each row of Q_l, read as a polynomial in R^3, has zero Laplacian
    (checked with a numerical 7-point Laplacian, independent of L_l)."""
    q = angular.harmonic_projection(l)
    ex = angular.monomial_exponents(l)
    rng = np.random.default_rng(l)
    x = rng.normal(size=(20, 3))

    def poly(p):
        return sum(q[:, c] * (p[0] ** e[0] * p[1] ** e[1] * p[2] ** e[2]) for c, e in enumerate(ex))

    h = 1e-3
    for p in x:
        lap = -6 * poly(p)
        for ax in range(3):
            dp = np.zeros(3)
            dp[ax] = h
            lap = lap + poly(p + dp) + poly(p - dp)
        lap = lap / h ** 2
        assert np.max(np.abs(lap)) < 1e-4 * max(1.0, np.max(np.abs(poly(p))))


@pytest.mark.parametrize("l", range(6))
def test_addition_theorem_closed_form(l):
    """With Q D^-1 Q^T = I:  m(a)^T Q^T Q m(b) = l!/(2l-1)!! P_l(a.b),
    the Legendre polynomial from scipy (independent of the oracle)."""
    rng = np.random.default_rng(100 + l)
    a = rng.normal(size=(50, 3))
    b = rng.normal(size=(50, 3))
    a /= np.linalg.norm(a, axis=1, keepdims=True)
    b /= np.linalg.norm(b, axis=1, keepdims=True)
    fa, _ = angular.angular_features(a, l, 0)
    fb, _ = angular.angular_features(b, l, 0)
    sl = slice(l * l, (l + 1) ** 2)
    lhs = (fa[:, sl] * fb[:, sl]).sum(1)
    dfact = math.prod(range(2 * l - 1, 0, -2)) if l > 0 else 1
    rhs = math.factorial(l) / dfact * eval_legendre(l, (a * b).sum(1))
    np.testing.assert_allclose(lhs, rhs, atol=1e-13)


def test_sphere_orthogonality_by_quadrature():
    """Features of different orders and different rows are orthogonal on the
    sphere, and rows of one order have equal norms (Gauss-Legendre x uniform
    phi quadrature, exact for these polynomial degrees)."""
    lmax = 5
    xg, wg = np.polynomial.legendre.leggauss(12)
    phi = np.arange(24) * (2 * np.pi / 24)
    ct, ph = np.meshgrid(xg, phi, indexing="ij")
    wt = np.repeat(wg, len(phi)) * (2 * np.pi / len(phi))
    st = np.sqrt(1 - ct ** 2)
    u = np.stack([(st * np.cos(ph)).ravel(), (st * np.sin(ph)).ravel(), ct.ravel()], 1)
    f, _ = angular.angular_features(u, lmax, 0)
    gram = (f * wt[:, None]).T @ f
    for l in range(lmax + 1):
        sl = slice(l * l, (l + 1) ** 2)
        blk = gram[sl, sl]
        np.testing.assert_allclose(blk, blk[0, 0] * np.eye(2 * l + 1), atol=1e-12)
    off = gram - np.diag(np.diag(gram))
    np.testing.assert_allclose(off, 0.0, atol=1e-12)


def test_cartesian_vs_irreducible_identities():
    """G_cart[l] = sum_jj' g g' t^l (multinomial theorem with C_l = D_l) and
    G_irr = G_cart minus lower orders via the Legendre expansion:
    G_irr[1] = G_cart[1], G_irr[2] = G_cart[2] - G0^2/3,
    G_irr[3] = G_cart[3] - 3/5 G_cart[1]."""
    rng = np.random.default_rng(7)
    n = 9
    u = rng.normal(size=(n, 3))
    u /= np.linalg.norm(u, axis=1, keepdims=True)
    g = rng.normal(size=n)
    G = {}
    for kind in (0, 1):
        f, _ = angular.angular_features(u, 3, kind)
        P = f.T @ g
        out = [P[0]]
        for l, (sl, metric) in enumerate(angular.block_slices(3, kind)):
            if l:
                out.append(P[sl] @ metric @ P[sl])
        G[kind] = np.array(out)
    t = u @ u.T
    gg = np.outer(g, g)
    for l in (1, 2, 3):
        np.testing.assert_allclose(G[1][l], (gg * t ** l).sum(), rtol=1e-12)
    np.testing.assert_allclose(G[0][1], G[1][1], rtol=1e-12)
    np.testing.assert_allclose(G[0][2], G[1][2] - G[0][0] ** 2 / 3, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(G[0][3], G[1][3] - 0.6 * G[1][1], rtol=1e-11, atol=1e-12)


@pytest.mark.parametrize("kind", [0, 1])
def test_feature_gradient_by_finite_differences(kind):
    rng = np.random.default_rng(3)
    u = rng.normal(size=(10, 3))
    f, df = angular.angular_features(u, 3, kind)
    h = 1e-6
    for ax in range(3):
        du = np.zeros(3)
        du[ax] = h
        fp, _ = angular.angular_features(u + du, 3, kind)
        fm, _ = angular.angular_features(u - du, 3, kind)
        np.testing.assert_allclose((fp - fm) / (2 * h), df[:, :, ax], atol=1e-7)
