"""fp64 reference of the owner's Muon update (test infrastructure only; see package docstring).

Paper passages followed:
* Section 3 ("Approach: Owner-Shaped ZeRO-3"): the owner runs NS on the complete reduced gradient of
  each matrix it owns and updates its parameter and Muon state locally.
* Section 2 ("Motivation"): NS iterations are made of whole-matrix products X X^T.
* Section 5.1 ("Setup", Optimizers/timing): Muon is torch.optim.Muon; the run uses lr, weight decay,
  momentum, the number of NS steps and the ``match_rms_adamw`` learning-rate adjustment as
  arguments. Those are arguments here too.

The quintic iteration is X <- a X + (b A + c A^2) X with A = X X^T, applied to the short side
(the matrix is transposed when it has more rows than columns) after Frobenius normalisation with a
clamped norm. The momentum buffer is an exponential moving average of the gradient with a Nesterov
look-ahead. Everything is float64.

Per-step coefficient schedules (one (a_k, b_k, c_k) per NS step) generalise the fixed triple; the
paper does not use them (it runs one fixed triple), and with a constant schedule the iteration is
exactly the paper's.
"""
from __future__ import annotations

import math
from typing import Tuple

import numpy as np


def bf16_widen(bits: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) -> float64, exactly (a bf16 is the top half of an fp32)."""
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def _f64(x: np.ndarray) -> np.ndarray:
    x = np.asarray(x)
    if x.dtype == np.uint16:
        return bf16_widen(x)
    return x.astype(np.float64)


def momentum_update(grad: np.ndarray, buf: np.ndarray, beta: float,
                    nesterov: bool = True) -> Tuple[np.ndarray, np.ndarray]:
    """Muon momentum (Section 5.1: torch.optim.Muon's buffer; Section 3: "Muon state").

    The buffer is an exponential moving average: buf' = buf + (1 - beta) (g - buf).
    With Nesterov the NS input is the look-ahead u = g + beta (buf' - g); without it u = buf'.
    Returns (buf', u).
    """
    g = _f64(grad)
    b = _f64(buf)
    b_new = b + (1.0 - beta) * (g - b)
    if nesterov:
        u = g + beta * (b_new - g)
    else:
        u = b_new.copy()
    return b_new, u


def reduce_gradients(parts, scale: float = 1.0) -> np.ndarray:
    """Owner-side gradient reduction (Section 4.2, owner-segment collectives): every rank of the
    shard span contributes its full-gradient buffer for the matrix and the owner keeps the
    reduced result. Reading: the reduction is the sum of the W contributions times ``scale``
    (1 / W for the data-parallel mean), formed here exactly in float64."""
    parts = [_f64(p) for p in parts]
    if not parts:
        raise ValueError("at least one gradient part")
    total = np.zeros_like(parts[0])
    for p in parts:
        if p.shape != total.shape:
            raise ValueError("gradient parts must share one shape")
        total = total + p
    return total * float(scale)


def frobenius_normalize(x: np.ndarray, eps: float) -> np.ndarray:
    """X0 = X / max(||X||_F, eps): bounds the spectral norm by 1 before NS (clamped-norm reading)."""
    x = _f64(x)
    nrm = math.sqrt(float(np.sum(x * x)))
    return x / max(nrm, eps)


def ns_quintic_step(x: np.ndarray, a: float, b: float, c: float) -> np.ndarray:
    """One quintic NS step on a short-side-first matrix X (r x s, r <= s).

    A = X X^T (Section 2's whole-matrix product), B = b A + c A A, X' = a X + B X.
    """
    A = x @ x.T
    B = b * A + c * (A @ A)
    return a * x + B @ x


def step_coefficients(a: float, b: float, c: float, steps: int, schedule=None):
    """The (a_k, b_k, c_k) of each of the ``steps`` NS steps: the fixed triple, or ``schedule``."""
    if schedule is None:
        return [(a, b, c)] * steps
    sched = [tuple(float(v) for v in t) for t in schedule]
    if len(sched) != steps or any(len(t) != 3 for t in sched):
        raise ValueError("schedule needs one (a, b, c) triple per NS step")
    return sched


def newton_schulz(u: np.ndarray, a: float, b: float, c: float, steps: int,
                  eps: float = 1e-7, schedule=None) -> np.ndarray:
    """NS orthogonalisation of the whole matrix u (m x n), returned in u's orientation.

    Transpose when m > n (work on the short side), normalise by the clamped Frobenius norm, take
    ``steps`` quintic steps (step k with schedule[k] if a schedule is given), transpose back.
    """
    x = _f64(u)
    if x.ndim != 2:
        raise ValueError("NS needs a 2D matrix")
    if not 0 <= steps < 100:
        raise ValueError("steps must be in [0, 100)")
    tall = x.shape[0] > x.shape[1]
    if tall:
        x = x.T
    coeffs = step_coefficients(a, b, c, steps, schedule)
    x = frobenius_normalize(x, eps)
    for ak, bk, ck in coeffs:
        x = ns_quintic_step(x, ak, bk, ck)
    return np.ascontiguousarray(x.T if tall else x)


def lr_factor(m: int, n: int, mode: str) -> float:
    """Shape adjustment of the learning rate (Section 5.1 names ``match_rms_adamw``).

    * "original":        sqrt(max(1, rows / cols))   (torch.optim.Muon's default)
    * "match_rms_adamw": 0.2 * sqrt(max(rows, cols))
    * "none":            1
    rows, cols are the parameter's stored shape.
    """
    if mode == "original":
        return math.sqrt(max(1.0, m / n))
    if mode == "match_rms_adamw":
        return 0.2 * math.sqrt(max(m, n))
    if mode == "none":
        return 1.0
    raise ValueError(f"unknown lr adjustment {mode!r}")


def apply_update(param: np.ndarray, update: np.ndarray, lr: float, weight_decay: float,
                 factor: float) -> np.ndarray:
    """Decoupled weight decay then the scaled step: p' = p (1 - lr wd) - lr f O.

    The decay uses the unadjusted lr; both terms act on the old parameter.
    """
    p = _f64(param)
    return p * (1.0 - lr * weight_decay) - (lr * factor) * update


def muon_step(param: np.ndarray, grad: np.ndarray, buf: np.ndarray, *, lr: float,
              weight_decay: float, momentum: float, nesterov: bool, a: float, b: float, c: float,
              ns_steps: int, eps: float = 1e-7, lr_adjust: str = "original", ns_schedule=None
              ) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """One owner-local Muon step on one whole matrix (Section 3). Returns (param', buf', O)."""
    m, n = np.asarray(grad).shape
    buf_new, u = momentum_update(grad, buf, momentum, nesterov)
    O = newton_schulz(u, a, b, c, ns_steps, eps, ns_schedule)
    p_new = apply_update(param, O, lr, weight_decay, lr_factor(m, n, lr_adjust))
    return p_new, buf_new, O
