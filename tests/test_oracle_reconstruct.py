"""Pins for the reconstruction oracle (oracle/reconstruct.py), CPU only.

The online normal equations (Sec. 4, Algorithm "MPIFA" Part 1) are checked
against the same minimisations solved from the whole calibration set by
least squares (no normal equations), against exact recovery of a rank-r W,
and against batch-split invariance; planted mistakes must fail the pins.
"""
import numpy as np
import pytest

from oracle import reconstruct as rec


def _data(n=24, m=30, r=6, b=300, seed=0, same_flow=False):
    rng = np.random.default_rng(seed)
    W = rng.standard_normal((m, n)) / np.sqrt(n)
    Vt = rng.standard_normal((r, n)) / np.sqrt(n)
    Xu = rng.standard_normal((b, n))
    Xo = Xu.copy() if same_flow else Xu + 0.1 * rng.standard_normal((b, n))
    return W, Vt, Xo, Xu


def _online(W, Xo, Xu, lam, batches=3):
    acc = rec.OnlineAccumulator(W, lam)
    for xo, xu in zip(np.array_split(Xo, batches), np.array_split(Xu, batches)):
        acc.add(xo, xu)
    return acc


def _rel(a, b):
    return np.linalg.norm(a - b) / np.linalg.norm(b)


@pytest.mark.parametrize("lam,alpha", [(0.25, 1e-3), (1.0, 1e-3), (0.0, 0.1), (0.5, 0.0)])
def test_online_equals_full_batch_least_squares(lam, alpha):
    W, Vt, Xo, Xu = _data()
    acc = _online(W, Xo, Xu, lam)
    U_r, Vt_r = rec.reconstruct(acc.S, acc.T, W, Vt, alpha)
    U_f, Vt_f = rec.full_batch(Xo, Xu, W, Vt, lam, alpha)
    assert _rel(U_r, U_f) <= 1e-9
    assert _rel(Vt_r, Vt_f) <= 1e-9


def test_rank_r_weight_is_recovered_exactly():
    """W = U0 V0^T of rank r and one data flow (X_o = X_u): the objective can
    reach zero, so U_r V_r^T = W for a generic starting V."""
    rng = np.random.default_rng(3)
    n, m, r = 20, 26, 5
    W = rng.standard_normal((m, r)) @ rng.standard_normal((r, n))
    _, Vt, Xo, Xu = _data(n, m, r, 200, seed=4, same_flow=True)
    acc = _online(W, Xo, Xu, 0.25)
    U_r, Vt_r = rec.reconstruct(acc.S, acc.T, W, Vt, 1e-3)
    assert _rel(U_r @ Vt_r, W) <= 1e-9


def test_accumulators_are_batch_split_invariant_and_equal_gram():
    W, Vt, Xo, Xu = _data(seed=5)
    a = _online(W, Xo, Xu, 0.25, batches=1)
    b = _online(W, Xo, Xu, 0.25, batches=7)
    assert _rel(a.S, b.S) <= 1e-13 and _rel(a.T, b.T) <= 1e-13
    assert _rel(a.S, Xu.T @ Xu) <= 1e-13
    assert _rel(a.T, W @ (0.25 * Xo + 0.75 * Xu).T @ Xu) <= 1e-13


def test_planted_mistakes_are_caught():
    W, Vt, Xo, Xu = _data(seed=6)
    lam, alpha = 0.25, 1e-3
    U_f, Vt_f = rec.full_batch(Xo, Xu, W, Vt, lam, alpha)
    acc = _online(W, Xo, Xu, lam)
    S, T = acc.S, acc.T
    V = Vt.T
    wrong = {
        "mix ratio swapped": _online(W, Xo, Xu, 1 - lam),
    }
    U_w, _ = rec.reconstruct(wrong["mix ratio swapped"].S, wrong["mix ratio swapped"].T, W, Vt, alpha)
    assert _rel(U_w, U_f) > 1e-4
    # regularisation added to the wrong factor
    U_r = np.linalg.solve((V.T @ S @ V).T, (T @ V).T).T
    bad = np.linalg.solve(S, np.linalg.solve(U_r.T @ U_r + alpha * np.eye(U_r.shape[1]),
                                             U_r.T @ (T + alpha * W)).T).T
    assert _rel(bad, Vt_f) > 1e-6
    # the Gram factor (V^T S V)^-1 dropped from the U update
    assert _rel(T @ V, U_f) > 1e-4
    # the dense-flow inputs used as the regressor instead of the low-rank ones
    acc_o = rec.OnlineAccumulator(W, lam)
    acc_o.add(Xu, Xo)
    U_x, _ = rec.reconstruct(acc_o.S, acc_o.T, W, Vt, alpha)
    assert _rel(U_x, U_f) > 1e-4
