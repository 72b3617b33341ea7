"""fp64 reference of the tail owner's AdamW update (test infrastructure only).

Section 3 and Section 4.4 of the paper route a block's non-matrix tensors (its "tail") to AdamW on
the tail owner; Section 5.1 fixes PyTorch AdamW with betas (0.9, 0.999), eps 1e-8 and lr / weight
decay 1e-3 / 1e-2. AdamW (Loshchilov & Hutter) is bias-corrected Adam with decoupled weight decay.
"""
from __future__ import annotations

import math
from typing import Tuple

import numpy as np

from .muon import _f64


def adamw_step(param: np.ndarray, grad: np.ndarray, exp_avg: np.ndarray, exp_avg_sq: np.ndarray,
               *, lr: float, beta1: float, beta2: float, eps: float, weight_decay: float,
               step: int) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """One AdamW step at step number ``step`` (t >= 1, counted after increment).

    p <- p (1 - lr wd)
    m <- beta1 m + (1 - beta1) g
    v <- beta2 v + (1 - beta2) g^2
    p <- p - lr / (1 - beta1^t) * m / (sqrt(v) / sqrt(1 - beta2^t) + eps)
    Returns (p, m, v) in float64.
    """
    if step < 1:
        raise ValueError("step is counted from 1")
    p = _f64(param) * (1.0 - lr * weight_decay)
    g = _f64(grad)
    m = beta1 * _f64(exp_avg) + (1.0 - beta1) * g
    v = beta2 * _f64(exp_avg_sq) + (1.0 - beta2) * g * g
    bc1 = 1.0 - beta1 ** step
    bc2 = 1.0 - beta2 ** step
    denom = np.sqrt(v) / math.sqrt(bc2) + eps
    p = p - (lr / bc1) * (m / denom)
    return p, m, v
