"""Shared test helpers: host<->device marshalling of the synthetic inputs and error measures."""
import numpy as np

import synth


def to_dev(arr: np.ndarray, dtype: str, device="cuda"):
    import torch
    if dtype == synth.BF16:
        return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).to(device)


def from_dev(t) -> np.ndarray:
    """Device tensor -> float64 numpy (bf16 widened exactly)."""
    import torch
    if t.dtype == torch.bfloat16:
        bits = t.view(torch.int16).cpu().numpy().view(np.uint16)
        return synth.bf16_bits_to_f32(bits).astype(np.float64)
    return t.float().cpu().numpy().astype(np.float64)


def rel_fro(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / den) if den > 0 else float(np.linalg.norm(a - b))


def tile_rel_errors(a, b, tile: int = 256) -> np.ndarray:
    """Relative Frobenius error of a against b on every tile x tile block (edge blocks partial):
    a defect confined to one block of the output shows here even where the whole-matrix error,
    which averages it over all blocks, stays small."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    m, n = b.shape
    tm, tn = -(-m // tile), -(-n // tile)
    d2 = np.zeros((tm * tile, tn * tile))
    b2 = np.zeros((tm * tile, tn * tile))
    d2[:m, :n] = (a - b) ** 2
    b2[:m, :n] = b ** 2
    num = d2.reshape(tm, tile, tn, tile).sum(axis=(1, 3))
    den = b2.reshape(tm, tile, tn, tile).sum(axis=(1, 3))
    return np.sqrt(num / np.where(den > 0, den, 1.0))


def bf16_half_ulp(x: np.ndarray) -> np.ndarray:
    """Half a bf16 ulp at |x| (8 significant bits); tiny values use the subnormal spacing."""
    ax = np.maximum(np.abs(np.asarray(x, dtype=np.float64)), 2.0 ** -126)
    return 0.5 * 2.0 ** (np.floor(np.log2(ax)) - 7)


def check_bf16_param(p_gpu, p_or, lr_f_update_norm: float, tol: float) -> float:
    """Rounding-aware parameter check: the fp64 parameter rounded to bf16 can be off by half an
    ulp per element; on top of that the update may differ by `tol` relative. Returns the ratio of
    the error to the allowed bound (must be <= 1)."""
    err = np.linalg.norm(p_gpu - p_or)
    bound = tol * lr_f_update_norm + np.linalg.norm(bf16_half_ulp(p_or)) * (1 + 2.0 ** -6)
    return float(err / bound)
