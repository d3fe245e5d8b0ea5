"""The MLIP's energy, forces and virial, written out plainly (Section 3.1).

Pipeline (Eqs. 1-10 of Section 3.1, architecture of Section 4.1):

  Eq. 1   r_ij = r_j - r_i (minimum image), r_ij = |r_ij|, u = r_ij / r_ij
  Eq. 2   g_rad_ij = E(r_ij; chi_E), a residual SiLU network per encoder
          table, times a smooth cutoff
  Eq. 3   g_ang_ij = Omega(u) (angular.py)
  Eq. 4   P_i = G_ang_i^T G_rad_i = sum_j g_ang_ij (x) g_rad_ij   [d x k]
  Eq. 5   G_i[0, c] = P_i[0, c];  G_i[l, c] = p_l^T C_l p_l  (l >= 1)
  Eq. 6   E_i = R(G_i; chi_R), a residual SiLU network per head table
  Eq. 7   W_i = dE_i / dP_i
  Eq. 8   U_i = G_ang_i W_i          (row j: u_ij = W_i^T g_ang_ij)
  Eq. 9   V_i = G_rad_i W_i^T        (row j: v_ij = W_i g_rad_ij)
  Eq. 10  f_ij = dE_i/dr_ij = J_rad_ij^T u_ij + J_ang_ij^T v_ij
  forces  the scatter-sum of partial forces: F_i += f_ij, F_j -= f_ij
          (F = -grad E with E = sum_i E_i and r_ij = r_j - r_i)

Readings of points the paper leaves open (each is stated where it is used):
  * network form: encoder h1 = silu(w0 r + b0), then (enc_hidden - 1)
    residual layers h <- h + silu(W h + b), then a linear output layer; the
    head likewise with reg_hidden hidden layers of width reg_width and a
    linear scalar output.  The SiLU activation and the residual connections
    apply to both networks (Section 4.1, architecture);
  * encoder input is the raw distance in Angstrom; no descriptor
    normalisation; no per-species reference energy beyond the output bias;
  * the radial feature is multiplied by the cosine cutoff
    fc(r) = (1 + cos(pi r / rc)) / 2 for r < rc (0 beyond), so energies and
    forces are continuous at rc;
  * encoder tables: one per ordered species pair (s_i, s_j), per neighbour
    species, or one universal table; head tables: one per centre species or
    one universal table (Section 3.2, "Differentiating Atom Species");
  * head input is vec(G_i) in l-major order, index l*k + c;
  * virial: per-atom, centre-attributed, w_i = - sum_j r_ij (x) f_ij
    (w[a][b] = - sum_j r_ij[a] f_ij[b]); the total W = sum_i w_i equals
    - dE/d(strain)^T.  The paper does not define a virial.
"""
from __future__ import annotations

import math
from typing import Dict, Optional, Sequence

import numpy as np

from .angular import angular_features, block_slices
from .neighbors import neighbor_list, wrap_positions, min_image


def sigmoid(z):
    return 1.0 / (1.0 + np.exp(-z))


def silu(z):
    return z * sigmoid(z)


def dsilu(z):
    s = sigmoid(z)
    return s * (1.0 + z * (1.0 - s))


def cutoff_function(r, rc):
    """fc(r) = (1 + cos(pi r/rc))/2 and its derivative, zero for r >= rc."""
    inside = r < rc
    fc = np.where(inside, 0.5 * (1.0 + np.cos(math.pi * r / rc)), 0.0)
    dfc = np.where(inside, -0.5 * math.pi / rc * np.sin(math.pi * r / rc), 0.0)
    return fc, dfc


def _hp(hp, name):
    return hp[name] if isinstance(hp, dict) else getattr(hp, name)


class Model:
    """Weights of one model, unpacked from the flat float64 blob.

    Blob order: encoder tables then head tables.  Encoder table:
    w0[W], b0[W], (W_t[W][W], b_t[W]) for t = 1..enc_hidden-1, W_out[k][W],
    b_out[k].  Head table: A0[R][(lmax+1)k], c0[R], (A_t[R][R], c_t[R]) for
    t = 1..reg_hidden-1, a_out[R], c_out.  Matrices are [out][in]."""

    def __init__(self, hp, weights: np.ndarray):
        g = lambda n: _hp(hp, n)
        self.C = int(g("n_species"))
        self.rc = float(g("cutoff"))
        self.skin = float(g("skin"))
        self.k = int(g("k"))
        self.lmax = int(g("lmax"))
        self.kind = int(g("angular"))
        self.enc_cond = int(g("enc_cond"))
        self.reg_cond = int(g("reg_cond"))
        self.W = int(g("enc_width"))
        self.nh_enc = int(g("enc_hidden"))
        self.R = int(g("reg_width"))
        self.nh_reg = int(g("reg_hidden"))
        self.blocks = block_slices(self.lmax, self.kind)
        self.d = self.blocks[-1][0].stop
        w = np.asarray(weights, dtype=np.float64)
        pos = 0

        def take(n, shape):
            nonlocal pos
            out = w[pos:pos + n].reshape(shape)
            pos += n
            return out

        n_enc = {2: self.C * self.C, 1: self.C, 0: 1}[self.enc_cond]
        n_head = self.C if self.reg_cond == 1 else 1
        W, R, k = self.W, self.R, self.k
        self.enc = []
        for _ in range(n_enc):
            t = {"w0": take(W, (W,)), "b0": take(W, (W,)), "hidden": []}
            for _h in range(1, self.nh_enc):
                t["hidden"].append((take(W * W, (W, W)), take(W, (W,))))
            t["Wout"] = take(k * W, (k, W))
            t["bout"] = take(k, (k,))
            self.enc.append(t)
        nin = (self.lmax + 1) * k
        self.head = []
        for _ in range(n_head):
            t = {"A0": take(R * nin, (R, nin)), "c0": take(R, (R,)), "hidden": []}
            for _h in range(1, self.nh_reg):
                t["hidden"].append((take(R * R, (R, R)), take(R, (R,))))
            t["aout"] = take(R, (R,))
            t["cout"] = float(take(1, (1,))[0])
            self.head.append(t)
        if pos != w.size:
            raise ValueError(f"weight blob has {w.size} values, model needs {pos}")

    # -- species conditioning (Section 3.2) ---------------------------------
    def enc_index(self, si, sj):
        if self.enc_cond == 2:
            return si * self.C + sj
        if self.enc_cond == 1:
            return sj
        return np.zeros_like(sj)

    def head_index(self, si):
        return si if self.reg_cond == 1 else np.zeros_like(si)

    # -- Eq. 2: radial encoder and its derivative in r ----------------------
    def encoder(self, tau: int, r: np.ndarray):
        """g_rad(r) [n][k] and d g_rad / dr [n][k] for encoder table tau."""
        t = self.enc[tau]
        z = r[:, None] * t["w0"][None, :] + t["b0"][None, :]
        h = silu(z)
        dh = dsilu(z) * t["w0"][None, :]
        for Wt, bt in t["hidden"]:
            z = h @ Wt.T + bt
            dz = dh @ Wt.T
            h = h + silu(z)
            dh = dh + dsilu(z) * dz
        m = h @ t["Wout"].T + t["bout"]
        dm = dh @ t["Wout"].T
        fc, dfc = cutoff_function(r, self.rc)
        g = fc[:, None] * m
        dg = dfc[:, None] * m + fc[:, None] * dm
        return g, dg

    # -- Eq. 6 and its gradient ---------------------------------------------
    def regression(self, rho: int, x: np.ndarray):
        """E [n] and dE/dx [n][(lmax+1)k] for head table rho."""
        t = self.head[rho]
        zeta0 = x @ t["A0"].T + t["c0"]
        y = silu(zeta0)
        zetas = []
        for At, ct in t["hidden"]:
            zt = y @ At.T + ct
            zetas.append(zt)
            y = y + silu(zt)
        E = y @ t["aout"] + t["cout"]
        delta = np.broadcast_to(t["aout"], y.shape).copy()
        for (At, _), zt in zip(reversed(t["hidden"]), reversed(zetas)):
            delta = delta + (dsilu(zt) * delta) @ At
        dEdx = (dsilu(zeta0) * delta) @ t["A0"]
        return E, dEdx

    # -- Eq. 5 ----------------------------------------------------------------
    def descriptor(self, P: np.ndarray) -> np.ndarray:
        """G [n][lmax+1][k] from P [n][d][k]."""
        n = P.shape[0]
        G = np.empty((n, self.lmax + 1, self.k))
        for l, (sl, metric) in enumerate(self.blocks):
            p = P[:, sl, :]
            if l == 0:
                G[:, 0, :] = p[:, 0, :]
            else:
                G[:, l, :] = np.einsum("nmc,mq,nqc->nc", p, metric, p)
        return G

    # -- Eq. 7 ----------------------------------------------------------------
    def moment_adjoint(self, P: np.ndarray, dEdG: np.ndarray) -> np.ndarray:
        """W = dE/dP [n][d][k] given dE/dG [n][lmax+1][k]."""
        Wm = np.empty_like(P)
        for l, (sl, metric) in enumerate(self.blocks):
            if l == 0:
                Wm[:, sl, :] = dEdG[:, 0, None, :]
            else:
                Wm[:, sl, :] = 2.0 * np.einsum("mq,nqc->nmc", metric, P[:, sl, :]) * dEdG[:, l, None, :]
        return Wm


def evaluate(model: Model, pos: np.ndarray, types: np.ndarray, box: np.ndarray,
             offsets: Optional[np.ndarray] = None, idx: Optional[np.ndarray] = None,
             centres: Optional[Sequence[int]] = None, batch: int = 512,
             return_pairs: bool = False, return_descriptors: bool = False) -> Dict[str, np.ndarray]:
    """Evaluate E_i, forces and per-atom virial.

    offsets/idx: listed neighbours (CSR, rows in atom order); built with
    r_list = cutoff + skin when omitted.  Only pairs with |r_ij| < cutoff
    take part (beyond it the cutoff function is zero).

    centres: evaluate only these centre atoms.  E_i and the virial are then
    valid for the centres; forces are partial sums of their partial forces
    (use `forces_for` for exact forces of chosen atoms).

    Returns dict with E_i [N] (NaN for atoms not evaluated), F [N][3],
    virial [N][9] (row-major 3x3, NaN rows for atoms not evaluated), E, W [9],
    and optionally pair_i, pair_j, pair_f and P, G per centre."""
    pos = np.asarray(pos, dtype=np.float64)
    types = np.asarray(types)
    box = np.asarray(box, dtype=np.float64)
    N = len(pos)
    if offsets is None:
        offsets, idx = neighbor_list(pos, box, model.rc + model.skin)
    centres = np.arange(N) if centres is None else np.asarray(centres, dtype=np.int64)
    w = wrap_positions(pos, box)
    E_i = np.full(N, np.nan)
    F = np.zeros((N, 3))
    vir = np.full((N, 9), np.nan)
    pi_l, pj_l, pf_l, P_l, G_l = [], [], [], [], []
    rc2 = model.rc * model.rc
    for b0 in range(0, len(centres), batch):
        cb = centres[b0:b0 + batch]
        counts = offsets[cb + 1] - offsets[cb]
        ci_local = np.repeat(np.arange(len(cb)), counts)
        j = np.concatenate([idx[offsets[c]:offsets[c + 1]] for c in cb]).astype(np.int64) \
            if len(cb) else np.zeros(0, np.int64)
        i = cb[ci_local]
        # Eq. 1
        rvec = min_image(w[j] - w[i], box)
        d2 = (rvec[:, 0] * rvec[:, 0] + rvec[:, 1] * rvec[:, 1]) + rvec[:, 2] * rvec[:, 2]
        keep = d2 < rc2
        ci_local, i, j, rvec = ci_local[keep], i[keep], j[keep], rvec[keep]
        r = np.sqrt((rvec * rvec).sum(1))
        u = rvec / r[:, None]
        # Eq. 2 (grouped by encoder table)
        tau = model.enc_index(types[i].astype(np.int64), types[j].astype(np.int64))
        g = np.zeros((len(r), model.k))
        dg = np.zeros((len(r), model.k))
        for t in np.unique(tau):
            sel = tau == t
            g[sel], dg[sel] = model.encoder(int(t), r[sel])
        # Eq. 3
        a, da = angular_features(u, model.lmax, model.kind)
        # Eq. 4
        P = np.zeros((len(cb), model.d, model.k))
        np.add.at(P, ci_local, a[:, :, None] * g[:, None, :])
        # Eq. 5
        G = model.descriptor(P)
        x = G.reshape(len(cb), -1)
        # Eq. 6
        rho = model.head_index(types[cb].astype(np.int64))
        E = np.zeros(len(cb))
        dEdx = np.zeros_like(x)
        for t in np.unique(rho):
            sel = rho == t
            E[sel], dEdx[sel] = model.regression(int(t), x[sel])
        # Eq. 7
        Wm = model.moment_adjoint(P, dEdx.reshape(G.shape))
        # Eqs. 8-9, row by row of U_i and V_i
        Wp = Wm[ci_local]
        U = np.einsum("pd,pdk->pk", a, Wp)
        V = np.einsum("pdk,pk->pd", Wp, g)
        # Eq. 10 with explicit Jacobians w.r.t. r_ij
        J_rad = dg[:, :, None] * u[:, None, :]
        proj = (np.eye(3)[None] - u[:, :, None] * u[:, None, :]) / r[:, None, None]
        J_ang = np.einsum("pdb,pba->pda", da, proj)
        f = np.einsum("pk,pka->pa", U, J_rad) + np.einsum("pd,pda->pa", V, J_ang)
        # scatter-sum and per-atom virial
        np.add.at(F, i, f)
        np.add.at(F, j, -f)
        wv = np.zeros((len(cb), 3, 3))
        np.add.at(wv, ci_local, -rvec[:, :, None] * f[:, None, :])
        E_i[cb] = E
        vir[cb] = wv.reshape(len(cb), 9)
        if return_pairs:
            pi_l.append(i), pj_l.append(j), pf_l.append(f)
        if return_descriptors:
            P_l.append(P), G_l.append(G)
    out = {"E_i": E_i, "F": F, "virial": vir,
           "E": float(np.nansum(E_i[centres])), "W": np.nansum(vir[centres], axis=0),
           "offsets": offsets, "idx": idx}
    if return_pairs:
        out["pair_i"] = np.concatenate(pi_l) if pi_l else np.zeros(0, np.int64)
        out["pair_j"] = np.concatenate(pj_l) if pj_l else np.zeros(0, np.int64)
        out["pair_f"] = np.concatenate(pf_l) if pf_l else np.zeros((0, 3))
    if return_descriptors:
        out["P"] = np.concatenate(P_l) if P_l else np.zeros((0, model.d, model.k))
        out["G"] = np.concatenate(G_l) if G_l else np.zeros((0, model.lmax + 1, model.k))
    return out


def forces_for(model: Model, pos, types, box, atoms: Sequence[int], offsets, idx) -> Dict[str, np.ndarray]:
    """Exact E_i, F_i and virial for selected atoms only.

    F_a needs f_aj (centre a) and f_ia for every centre i that lists a;
    with a full list those centres are exactly the listed neighbours of a.
    So the centres evaluated are atoms plus their listed neighbours."""
    atoms = np.asarray(atoms, dtype=np.int64)
    nb = [idx[offsets[a]:offsets[a + 1]] for a in atoms]
    centres = np.unique(np.concatenate([atoms] + [n.astype(np.int64) for n in nb]))
    res = evaluate(model, pos, types, box, offsets, idx, centres=centres, return_pairs=True)
    slot = np.full(len(pos), -1, dtype=np.int64)
    slot[atoms] = np.arange(len(atoms))
    F = np.zeros((len(atoms), 3))
    si = slot[res["pair_i"]]
    sj = slot[res["pair_j"]]
    np.add.at(F, si[si >= 0], res["pair_f"][si >= 0])
    np.add.at(F, sj[sj >= 0], -res["pair_f"][sj >= 0])
    return {"E_i": res["E_i"][atoms], "F": F, "virial": res["virial"][atoms]}
