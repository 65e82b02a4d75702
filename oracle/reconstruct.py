"""Online Error-Accumulation-Minimization reconstruction (M) -- TEST
INFRASTRUCTURE ONLY.

Plain fp64 numpy evaluation of Sec. 4 of arXiv 2501.19090 and of Part 1 of
Algorithm "MPIFA" (appendix "Experiment Details"), in the paper's order, for
row-major calibration batches (samples are rows here, columns in the paper):

  S  = sum_i x_u^i x_u^i^T                   (eq. lsq_online: X X^T, online)
  T  = sum_i y_t^i x_u^i^T,  y_t^i = lam W x_o^i + (1 - lam) W x_u^i
                                               (eq. mix_original_output)
  U_r   = T V (V^T S V)^-1                    (eq. lsq_online with Y_t)
  V_r^T = (U_r^T U_r)^-1 U_r^T (T + a W) (S + a I)^-1      (eq. lsq_v_reg)

V is n x r in the paper; these functions take and return V^T (r x n), the
layout the low-rank layer uses.  Library primitives (matmul, solve, lstsq)
are the steps; nothing is blocked or reordered.  Only tests/ may import this.
"""
from __future__ import annotations

import numpy as np


class OnlineAccumulator:
    """The two running sums of Algorithm "MPIFA", Part 1, steps 3 and 4."""

    def __init__(self, W, lam: float):
        self.W = np.asarray(W, np.float64)
        self.lam = float(lam)
        n = self.W.shape[1]
        self.S = np.zeros((n, n))
        self.T = np.zeros((self.W.shape[0], n))

    def add(self, Xo, Xu):
        """One batch of dense-flow inputs Xo and low-rank-flow inputs Xu (rows)."""
        Xo = np.asarray(Xo, np.float64)
        Xu = np.asarray(Xu, np.float64)
        for xo, xu in zip(Xo, Xu):  # sample by sample, as the sums are written
            self.S += np.outer(xu, xu)
            yt = self.lam * (self.W @ xo) + (1.0 - self.lam) * (self.W @ xu)
            self.T += np.outer(yt, xu)


def reconstruct(S, T, W, Vt, alpha: float):
    """Steps 5 and 6 (with the regularised V update): returns (U_r, V_r^T)."""
    S = np.asarray(S, np.float64)
    T = np.asarray(T, np.float64)
    W = np.asarray(W, np.float64)
    V = np.asarray(Vt, np.float64).T  # n x r, the paper's V
    U_r = np.linalg.solve((V.T @ S @ V).T, (T @ V).T).T
    G = U_r.T @ U_r
    H = U_r.T @ (T + alpha * W)
    Vt_r = np.linalg.solve(S + alpha * np.eye(S.shape[0]), np.linalg.solve(G, H).T).T
    return U_r, Vt_r


def full_batch(Xo, Xu, W, Vt, lam: float, alpha: float):
    """The same two minimisations solved from the whole calibration set at
    once by least squares (eq. lsq and eq. lsq_v_reg as stacked systems),
    without normal equations: an independent route to (U_r, V_r^T)."""
    Xo = np.asarray(Xo, np.float64).T  # n x b, the paper's layout
    Xu = np.asarray(Xu, np.float64).T
    W = np.asarray(W, np.float64)
    Yt = lam * (W @ Xo) + (1.0 - lam) * (W @ Xu)
    D = np.asarray(Vt, np.float64) @ Xu  # V^T X, r x b
    U_r = np.linalg.lstsq(D.T, Yt.T, rcond=None)[0].T  # min || Y_t - U D ||
    # min ||Y_t - U V^T X||^2 + a ||W - U V^T||^2 = || [Y_t, sqrt(a) W] - U V^T [X, sqrt(a) I] ||^2
    n = Xu.shape[0]
    Xs = np.concatenate([Xu, np.sqrt(alpha) * np.eye(n)], axis=1)
    Ys = np.concatenate([Yt, np.sqrt(alpha) * W], axis=1)
    Z = np.linalg.lstsq(U_r, Ys, rcond=None)[0]          # U^+ [Y_t, sqrt(a) W]
    Vt_r = np.linalg.lstsq(Xs.T, Z.T, rcond=None)[0].T   # (...) [X, sqrt(a) I]^+
    return U_r, Vt_r
