"""fp64 reference of the owner's SOAP update (test infrastructure only; see package docstring).

Paper passage followed: Section 5.7 ("Generality beyond Muon"): the owner, holding each 2D matrix
whole, runs a single-device matrix optimizer on it unchanged; besides Shampoo the paper runs SOAP,
which it describes as Adam run in the eigenbasis of Shampoo's preconditioner statistics. The paper
does not restate SOAP, so the published algorithm is followed: Vyas, Morwani, Zhao, Shapira,
Brandfonbrener, Janson and Kakade, "SOAP: Improving and Stabilizing Shampoo using Adam" (2024), the
matrix case, whose eigenbasis is refreshed by one step of power iteration followed by a QR
decomposition. Per step, with the bases Q_L (m x m) and Q_R (n x n) of the previous refresh:

    G' = Q_L^T G Q_R                        gradient in the eigenbasis
    M  <- beta1 M + (1 - beta1) G           first moment, kept in the original coordinates
    M' = Q_L^T M Q_R
    V  <- beta2 V + (1 - beta2) G' * G'     second moment, kept in the eigenbasis coordinates
    N' = Adam direction from M', V          (bias-corrected, below)
    N  = Q_L N' Q_R^T                       back to the original coordinates
    p  <- p (1 - lr wd) - lr N
    L  <- beta_s L + w_s G G^T,  R <- beta_s R + w_s G^T G          (Shampoo statistics)
    refresh: Q_L <- orthonormal factor of QR(L Q_L), Q_R <- of QR(R Q_R)

Readings (the paper fixes none of them):
* bias correction as PyTorch AdamW: N' = (M'/(1 - beta1^t)) / (sqrt(V)/sqrt(1 - beta2^t) + eps), so
  that with Q_L = Q_R = I one SOAP step is exactly one AdamW step.
* decoupled weight decay on the old parameter (as AdamW and the Muon/Shampoo steps here).
* the statistics are updated as Shampoo's (beta_s L + w_s G G^T and beta_s R + w_s G^T G, as in
  ``shampoo.update_statistics``; the published SOAP uses the EMA w_s = 1 - beta_s) and start at zero; the bases start at the
  identity, so the first steps are AdamW and the first refresh begins the power iteration (the
  published code starts from a full eigendecomposition instead; ``refresh_iters`` > 1 repeats the
  power step + QR, i.e. runs orthogonal iteration towards the eigenvectors).
* V is left unchanged when the basis is refreshed, as in the published algorithm.
* the QR factor is the Householder one with LAPACK's sign convention (LAPACK's geqrf/orgqr through
  scipy.linalg.qr). Column signs of a basis do not change N (each column enters N twice).
* one-sided preconditioning, as the published optimizer's maximum preconditioned dimension: a side
  longer than ``max_precond_dim`` keeps the identity basis and no statistic (its Q and statistic
  are returned as None), so on that side G', M' and N are untransformed; with both sides beyond
  it the step is AdamW.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Tuple

import numpy as np
import scipy.linalg

from .muon import _f64


@dataclasses.dataclass
class SoapHParams:
    lr: float = 3e-3
    weight_decay: float = 0.0
    beta1: float = 0.95
    beta2: float = 0.95
    eps: float = 1e-8
    shampoo_beta: float = 0.95
    shampoo_weight: float = 0.05
    refresh: bool = False
    refresh_iters: int = 1
    max_precond_dim: int = 4096


def orthonormal_factor(A: np.ndarray) -> np.ndarray:
    """Q of the Householder QR decomposition A = Q R (square A; LAPACK's geqrf/orgqr with their sign
    convention, as numpy.linalg.qr, through scipy.linalg.qr)."""
    Q, _ = scipy.linalg.qr(np.asarray(A, dtype=np.float64), mode="economic", check_finite=False)
    return Q


def refresh_basis(S: np.ndarray, Q: np.ndarray, iters: int = 1) -> np.ndarray:
    """`iters` steps of power iteration with QR on the statistic S, from the basis Q."""
    S = np.asarray(S, dtype=np.float64)
    Q = np.asarray(Q, dtype=np.float64)
    for _ in range(int(iters)):
        Q = orthonormal_factor(S @ Q)
    return Q


def adam_direction(Mp: np.ndarray, V: np.ndarray, beta1: float, beta2: float, eps: float,
                   step: int) -> np.ndarray:
    """Bias-corrected Adam direction (M/(1 - beta1^t)) / (sqrt(V)/sqrt(1 - beta2^t) + eps)."""
    if step < 1:
        raise ValueError("step is counted from 1")
    bc1 = 1.0 - beta1 ** step
    bc2 = 1.0 - beta2 ** step
    return (Mp / bc1) / (np.sqrt(V) / math.sqrt(bc2) + eps)


def soap_step(param: np.ndarray, grad: np.ndarray, exp_avg: np.ndarray, exp_avg_sq: np.ndarray,
              L, R, QL, QR, step: int, hp: SoapHParams):
    """One owner-local SOAP step on one whole m x n matrix at step number ``step`` (t >= 1).
    Returns (param', M', V', L', R', Q_L', Q_R', N) in float64. A side longer than
    hp.max_precond_dim is not preconditioned: its basis is the identity, its statistic is not kept,
    and its L (or R) and Q_L (or Q_R) come back as None (the inputs are ignored)."""
    G = _f64(grad)
    m, n = G.shape
    left, right = m <= hp.max_precond_dim, n <= hp.max_precond_dim
    QLm = np.asarray(QL, dtype=np.float64) if left else None
    QRm = np.asarray(QR, dtype=np.float64) if right else None

    def to_basis(X):      # Q_L^T X Q_R, a side without a basis being the identity
        X = QLm.T @ X if left else X
        return X @ QRm if right else X

    def from_basis(X):    # Q_L X Q_R^T
        X = QLm @ X if left else X
        return X @ QRm.T if right else X

    Gp = to_basis(G)
    M = hp.beta1 * _f64(exp_avg) + (1.0 - hp.beta1) * G
    Mp = to_basis(M)
    V = hp.beta2 * _f64(exp_avg_sq) + (1.0 - hp.beta2) * Gp * Gp
    Np = adam_direction(Mp, V, hp.beta1, hp.beta2, hp.eps, step)
    N = from_basis(Np)
    p_new = _f64(param) * (1.0 - hp.lr * hp.weight_decay) - hp.lr * N
    L2 = hp.shampoo_beta * np.asarray(L, dtype=np.float64) + hp.shampoo_weight * (G @ G.T) if left else None
    R2 = hp.shampoo_beta * np.asarray(R, dtype=np.float64) + hp.shampoo_weight * (G.T @ G) if right else None
    QLo, QRo = QLm, QRm
    if hp.refresh:
        if left:
            QLo = refresh_basis(L2, QLm, hp.refresh_iters)
        if right:
            QRo = refresh_basis(R2, QRm, hp.refresh_iters)
    return p_new, M, V, L2, R2, QLo, QRo, N
