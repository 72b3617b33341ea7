"""fp64 reference of the owner's Shampoo update (test infrastructure only; see package docstring).

Paper passage followed: Section 5.7 ("Generality beyond Muon"): because the owner holds each 2D matrix
whole, a single-device matrix optimizer runs on it unchanged; the paper swaps Muon for Shampoo with
full left and right preconditioners and the inverse fourth root, in float32. The paper does not
restate Shampoo, so the published definition is used: Gupta, Koren and Singer, "Shampoo:
Preconditioned Stochastic Tensor Optimization" (ICML 2018), the matrix case:

    L <- L + G G^T          (m x m)
    R <- R + G^T G          (n x n)
    W <- W - lr * L^{-1/4} G R^{-1/4}

Readings (the paper fixes none of them):
* statistics decay: L <- beta L + weight G G^T (and R alike); beta = weight = 1 is the published
  accumulation, beta = 1 - weight an exponential moving average. The statistics start at zero.
* regularisation: the root is taken of S + rho I with rho = eps + eps_rel * ||S||_F (an absolute
  ridge, as the published eps I, plus one relative to the statistic's Frobenius norm, which keeps
  float32 root iterations well conditioned whatever the gradient scale).
* refresh: the preconditioners P_L, P_R are recomputed from the updated statistics when refresh is
  set, else the stored ones are used (the published method recomputes every step; practical
  implementations every few steps).
* decoupled weight decay as for Muon: p' = p (1 - lr wd) - lr U, both terms on the old parameter.
* no momentum and no grafting (the paper names neither for Shampoo).

The inverse root here is the plain definition through a symmetric eigendecomposition.
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Tuple

import numpy as np

from .muon import _f64


def ridge(S: np.ndarray, eps: float, eps_rel: float) -> float:
    """rho = eps + eps_rel * ||S||_F."""
    return float(eps) + float(eps_rel) * float(np.linalg.norm(np.asarray(S, dtype=np.float64)))


def inverse_root(S: np.ndarray, p: int, eps: float = 0.0, eps_rel: float = 0.0) -> np.ndarray:
    """(S + rho I)^{-1/p} for symmetric positive semidefinite S, through S = V diag(w) V^T."""
    S = np.asarray(S, dtype=np.float64)
    d = S.shape[0]
    Sr = 0.5 * (S + S.T) + ridge(S, eps, eps_rel) * np.eye(d)
    w, V = np.linalg.eigh(Sr)
    if w.size and w.min() <= 0.0:
        raise ValueError("S + rho I is not positive definite")
    return (V * w ** (-1.0 / p)) @ V.T


def update_statistics(L: np.ndarray, R: np.ndarray, grad: np.ndarray, beta: float,
                      weight: float) -> Tuple[np.ndarray, np.ndarray]:
    """L' = beta L + weight G G^T, R' = beta R + weight G^T G."""
    G = _f64(grad)
    return (beta * np.asarray(L, dtype=np.float64) + weight * (G @ G.T),
            beta * np.asarray(R, dtype=np.float64) + weight * (G.T @ G))


@dataclasses.dataclass
class ShampooHParams:
    lr: float = 1e-3
    weight_decay: float = 0.0
    beta: float = 1.0
    weight: float = 1.0
    eps: float = 0.0
    eps_rel: float = 1e-6
    refresh: bool = True
    root: int = 4


def shampoo_step(param: np.ndarray, grad: np.ndarray, L: np.ndarray, R: np.ndarray,
                 PL: Optional[np.ndarray], PR: Optional[np.ndarray], hp: ShampooHParams):
    """One owner-local Shampoo step on one whole m x n matrix.
    Returns (param', L', R', P_L, P_R, U) with U = P_L G P_R."""
    G = _f64(grad)
    L2, R2 = update_statistics(L, R, G, hp.beta, hp.weight)
    if hp.refresh:
        PL = inverse_root(L2, hp.root, hp.eps, hp.eps_rel)
        PR = inverse_root(R2, hp.root, hp.eps, hp.eps_rel)
    else:
        PL = np.asarray(PL, dtype=np.float64)
        PR = np.asarray(PR, dtype=np.float64)
    U = PL @ G @ PR
    p_new = _f64(param) * (1.0 - hp.lr * hp.weight_decay) - hp.lr * U
    return p_new, L2, R2, PL, PR, U
