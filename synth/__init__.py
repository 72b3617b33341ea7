"""Seeded synthetic owner shares for the owner-local Muon/AdamW step.

This module is shared by the tests, the benchmark and the CPU oracle's callers. It only draws
random numbers and packs them into storage formats; it holds none of the optimizer's arithmetic.

Every tensor is drawn from its own counter-free numpy stream (PCG64 seeded through a
``SeedSequence`` tree), so any single entry can be regenerated on its own and large shares can be
drawn in parallel without changing a single bit:

    root = SeedSequence([workload seed])
    root.spawn(1 + n_muon + n_adamw)
      child 0            -> (unused; the uneven plan draws its shapes from default_rng(4))
      child 1 + i        -> Muon entry i:   spawn(3) = (param, grad, momentum)
      child 1 + n_muon+j -> AdamW entry j:  spawn(2) = (param, grad)
    each tensor stream spawns one grand-child per 2**24-element chunk, in order.

bf16 tensors are returned as their uint16 bit patterns (round-to-nearest-even from the float32
draw); fp32 tensors as float32 arrays. The shapes follow the workloads of the paper's evaluation
(Section 5.1): GPT-2-small-like and Llama-like decoder layers whose 2D weights are owned whole by
one rank, with non-matrix tensors (norm weights, and an embedding in the uneven stress plan) on
AdamW.
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor
from typing import List, Optional, Tuple

import numpy as np

F32 = "f32"
BF16 = "bf16"
_CHUNK = 1 << 24

# Default Newton-Schulz coefficients of the quintic iteration used by Muon.
NS_COEFFS = (3.4445, -4.7750, 2.0315)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest-even) and return the uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bfloat16 bit patterns to float32 (exact)."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclasses.dataclass
class Dist:
    """Normal(mean, std^2), or a constant when std == 0."""
    std: float
    mean: float = 0.0


@dataclasses.dataclass
class MuonSpec:
    m: int
    n: int
    name: str = ""
    param_dtype: str = BF16
    grad_dtype: str = BF16
    param: Dist = dataclasses.field(default_factory=lambda: Dist(0.02))
    grad: Dist = dataclasses.field(default_factory=lambda: Dist(1e-3))
    momentum: Dist = dataclasses.field(default_factory=lambda: Dist(1e-3))


@dataclasses.dataclass
class AdamWSpec:
    numel: int
    name: str = ""
    param_dtype: str = BF16
    grad_dtype: str = BF16
    param: Dist = dataclasses.field(default_factory=lambda: Dist(0.02, 1.0))
    grad: Dist = dataclasses.field(default_factory=lambda: Dist(0.02))


@dataclasses.dataclass
class MuonHParams:
    lr: float = 0.02
    weight_decay: float = 0.01
    momentum: float = 0.95
    nesterov: bool = True
    a: float = NS_COEFFS[0]
    b: float = NS_COEFFS[1]
    c: float = NS_COEFFS[2]
    ns_steps: int = 5
    eps: float = 1e-7
    lr_adjust: str = "original"    # "none" | "original" | "match_rms_adamw"
    ns_dtype: str = BF16
    ns_schedule: tuple = None      # None, or one (a, b, c) triple per NS step


@dataclasses.dataclass
class AdamWHParams:
    lr: float = 1e-3
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    weight_decay: float = 0.01
    step: int = 1


@dataclasses.dataclass
class Workload:
    name: str
    seed: int
    muon: List[MuonSpec]
    adamw: List[AdamWSpec]
    hp: MuonHParams
    adamw_hp: AdamWHParams
    description: str = ""

    def ns_flops_nominal(self) -> float:
        """Nominal NS flops K * sum(4 r^2 s + 2 r^3), r = short side, s = long side."""
        tot = 0.0
        for e in self.muon:
            r, s = min(e.m, e.n), max(e.m, e.n)
            tot += 4.0 * r * r * s + 2.0 * r ** 3
        return tot * self.hp.ns_steps

    def muon_elements(self) -> int:
        return sum(e.m * e.n for e in self.muon)

    def adamw_elements(self) -> int:
        return sum(e.numel for e in self.adamw)


# ----------------------------------------------------------------------------------------------
# The five owner shares.
# ----------------------------------------------------------------------------------------------

def _uneven_shapes(rng: np.random.Generator, count: int = 64) -> List[Tuple[int, int]]:
    """Shapes m, n in {512, ..., 8192} (multiples of 128), aspect ratio at most 4:1."""
    out = []
    while len(out) < count:
        k = rng.integers(0, 61, size=2)
        m, n = 512 + 128 * int(k[0]), 512 + 128 * int(k[1])
        if max(m, n) <= 4 * min(m, n):
            out.append((m, n))
    return out


def workload(index: int) -> Workload:
    """The numbered owner share (1..5). Seed = index."""
    if index == 1:
        return Workload(
            name="single_fp32_256x512", seed=1,
            muon=[MuonSpec(256, 512, "w", F32, F32, Dist(0.02), Dist(1.0), Dist(0.0))],
            adamw=[],
            hp=MuonHParams(lr=0.02, weight_decay=0.0, ns_dtype=F32),
            adamw_hp=AdamWHParams(),
            description="one fp32 256x512 matrix, zero momentum, fp32 Newton-Schulz")
    if index == 2:
        d, f = 768, 3072
        mu = []
        for layer in range(2):
            for nm in ("q", "k", "v", "o"):
                mu.append(MuonSpec(d, d, f"l{layer}.{nm}", grad=Dist(0.02)))
            mu.append(MuonSpec(f, d, f"l{layer}.fc", grad=Dist(0.02)))
            mu.append(MuonSpec(d, f, f"l{layer}.proj", grad=Dist(0.02)))
        ad = [AdamWSpec(d, f"ln{i}") for i in range(4)]
        return Workload(
            name="gpt2_small_share_2x768", seed=2, muon=mu, adamw=ad,
            hp=MuonHParams(lr=0.02, weight_decay=0.01), adamw_hp=AdamWHParams(weight_decay=0.01),
            description="2 GPT-2-small layers (d=768, ffn=3072): 12 matrices + 4 LayerNorm vectors")
    if index == 3:
        mu = []
        for layer in range(4):
            mu += [MuonSpec(4096, 4096, f"l{layer}.wq"), MuonSpec(1024, 4096, f"l{layer}.wk"),
                   MuonSpec(1024, 4096, f"l{layer}.wv"), MuonSpec(4096, 4096, f"l{layer}.wo"),
                   MuonSpec(14336, 4096, f"l{layer}.gate"), MuonSpec(14336, 4096, f"l{layer}.up"),
                   MuonSpec(4096, 14336, f"l{layer}.down")]
        ad = [AdamWSpec(4096, f"rms{i}", grad=Dist(1e-3)) for i in range(8)]
        return Workload(
            name="llama3_8b_share_4of32_layers", seed=3, muon=mu, adamw=ad,
            hp=MuonHParams(lr=0.02, weight_decay=0.01), adamw_hp=AdamWHParams(weight_decay=0.01),
            description="4 of 32 Llama-3-8B layers: 28 matrices + 8 RMSNorm vectors of 4096")
    if index == 4:
        # shapes first, from the plain seeded generator: 25 tall, 38 wide, 1 square, 1485.4 M elements
        shapes = _uneven_shapes(np.random.default_rng(4))
        mu = [MuonSpec(m, n, f"u{i}") for i, (m, n) in enumerate(shapes)]
        ad = [AdamWSpec(128256 * 4096, "embed", param=Dist(0.02), grad=Dist(1e-3))]
        ad += [AdamWSpec(4096, f"norm{i}", grad=Dist(1e-3)) for i in range(32)]
        return Workload(
            name="uneven_64_plus_embedding", seed=4, muon=mu, adamw=ad,
            hp=MuonHParams(lr=0.02, weight_decay=0.01), adamw_hp=AdamWHParams(weight_decay=0.01),
            description="64 seed-drawn shapes (512..8192, multiples of 128, aspect <= 4) + "
                        "AdamW on a 128256x4096 embedding and 32 vectors of 4096")
    if index == 5:
        mu = [MuonSpec(8192, 8192, "wq"), MuonSpec(1024, 8192, "wk"), MuonSpec(1024, 8192, "wv"),
              MuonSpec(8192, 8192, "wo"), MuonSpec(28672, 8192, "gate"), MuonSpec(28672, 8192, "up"),
              MuonSpec(8192, 28672, "down"), MuonSpec(28672, 8192, "gate_b"),
              MuonSpec(8192, 28672, "down_b")]
        return Workload(
            name="llama3_70b_heavy_share_9", seed=5, muon=mu, adamw=[],
            hp=MuonHParams(lr=0.02, weight_decay=0.1), adamw_hp=AdamWHParams(weight_decay=0.1),
            description="heavy 1/64 share of Llama-3-70B: one layer's 7 matrices + one extra "
                        "gate and down (9 matrices)")
    raise ValueError(f"no workload {index}")


# ----------------------------------------------------------------------------------------------
# Drawing values.
# ----------------------------------------------------------------------------------------------

def _tensor_seeds(wl: Workload) -> List[np.random.SeedSequence]:
    root = np.random.SeedSequence([wl.seed])
    return root.spawn(1 + len(wl.muon) + len(wl.adamw))


def _draw(seed: np.random.SeedSequence, numel: int, dist: Dist, dtype: str,
          pool: Optional[ThreadPoolExecutor] = None) -> np.ndarray:
    nchunk = max(1, -(-numel // _CHUNK))
    seeds = seed.spawn(nchunk)
    out = np.empty(numel, dtype=np.float32)

    def fill(i):
        lo, hi = i * _CHUNK, min(numel, (i + 1) * _CHUNK)
        if dist.std == 0.0:
            out[lo:hi] = dist.mean
            return
        rng = np.random.Generator(np.random.PCG64(seeds[i]))
        v = rng.standard_normal(hi - lo, dtype=np.float32)
        if dist.std != 1.0:
            v *= np.float32(dist.std)
        if dist.mean != 0.0:
            v += np.float32(dist.mean)
        out[lo:hi] = v

    if pool is not None and nchunk > 1:
        list(pool.map(fill, range(nchunk)))
    else:
        for i in range(nchunk):
            fill(i)
    if dtype == BF16:
        return f32_to_bf16_bits(out)
    return out


@dataclasses.dataclass
class MuonTensors:
    param: np.ndarray      # (m, n) uint16 bf16 bits or float32
    grad: np.ndarray
    momentum: np.ndarray   # (m, n) float32


@dataclasses.dataclass
class AdamWTensors:
    param: np.ndarray
    grad: np.ndarray
    exp_avg: np.ndarray
    exp_avg_sq: np.ndarray


def muon_entry(wl: Workload, i: int, pool: Optional[ThreadPoolExecutor] = None) -> MuonTensors:
    e = wl.muon[i]
    s_param, s_grad, s_mom = _tensor_seeds(wl)[1 + i].spawn(3)
    numel = e.m * e.n
    p = _draw(s_param, numel, e.param, e.param_dtype, pool).reshape(e.m, e.n)
    g = _draw(s_grad, numel, e.grad, e.grad_dtype, pool).reshape(e.m, e.n)
    mo = _draw(s_mom, numel, e.momentum, F32, pool).reshape(e.m, e.n)
    return MuonTensors(p, g, mo)


def adamw_entry(wl: Workload, j: int, pool: Optional[ThreadPoolExecutor] = None) -> AdamWTensors:
    e = wl.adamw[j]
    s_param, s_grad = _tensor_seeds(wl)[1 + len(wl.muon) + j].spawn(2)
    p = _draw(s_param, e.numel, e.param, e.param_dtype, pool)
    g = _draw(s_grad, e.numel, e.grad, e.grad_dtype, pool)
    z = np.zeros(e.numel, dtype=np.float32)
    return AdamWTensors(p, g, z, z.copy())


def thread_pool(max_workers: Optional[int] = None) -> ThreadPoolExecutor:
    n = max_workers or min(16, os.cpu_count() or 1)
    return ThreadPoolExecutor(n)


def random_muon_tensors(rng: np.random.Generator, m: int, n: int, param_dtype: str = BF16,
                        grad_dtype: str = BF16, g_std: float = 1e-3, m_std: float = 1e-3,
                        p_std: float = 0.02) -> MuonTensors:
    """Small ad-hoc tensors for tests (param, grad, momentum in that draw order)."""
    def cast(x, dt):
        return f32_to_bf16_bits(x) if dt == BF16 else x.astype(np.float32)
    p = cast(rng.standard_normal((m, n), dtype=np.float32) * np.float32(p_std), param_dtype)
    g = cast(rng.standard_normal((m, n), dtype=np.float32) * np.float32(g_std), grad_dtype)
    mo = (rng.standard_normal((m, n), dtype=np.float32) * np.float32(m_std)).astype(np.float32)
    return MuonTensors(p, g, mo)


# ----------------------------------------------------------------------------------------------
# Parameter lists for owner planning: (block, numel, is_matrix) per parameter, plus names and
# 2D shapes. Only shapes; no planning arithmetic.
# ----------------------------------------------------------------------------------------------

@dataclasses.dataclass
class PlanParam:
    block: int
    numel: int
    is_matrix: bool
    name: str
    shape: Tuple[int, ...]

    def tuple(self) -> Tuple[int, int, bool]:
        return (self.block, self.numel, self.is_matrix)


def decoder_plan_params(layers: int, hidden: int = 4096, intermediate: int = 16384,
                        kv_hidden: Optional[int] = None, vocab: int = 0,
                        norm: str = "rms") -> List[PlanParam]:
    """A decoder-only transformer wrapped one block per layer (Section 5.1 shapes: hidden 4096,
    intermediate 16384, 32 heads for the latency sweeps; hidden 768, intermediate 3072, vocab 50257
    for the convergence model). Per layer: q, o (hidden x hidden), k, v (kv_hidden x hidden),
    gate, up (intermediate x hidden), down (hidden x intermediate) as 2D matrices, and the two norm
    weights (plus biases for norm="layer") as non-2D tensors. vocab > 0 adds an embedding block
    before the layers and a final block with the final norm and an untied LM head, both 2D."""
    kv = hidden if kv_hidden is None else kv_hidden
    out: List[PlanParam] = []
    blk = 0

    def vec(b, name):
        out.append(PlanParam(b, hidden, False, name, (hidden,)))
        if norm == "layer":
            out.append(PlanParam(b, hidden, False, name + ".bias", (hidden,)))

    if vocab > 0:
        out.append(PlanParam(blk, vocab * hidden, True, "embed", (vocab, hidden)))
        blk += 1
    for layer in range(layers):
        vec(blk, f"l{layer}.attn_norm")
        for nm, shp in (("q", (hidden, hidden)), ("k", (kv, hidden)), ("v", (kv, hidden)),
                        ("o", (hidden, hidden))):
            out.append(PlanParam(blk, shp[0] * shp[1], True, f"l{layer}.{nm}", shp))
        vec(blk, f"l{layer}.ffn_norm")
        for nm, shp in (("gate", (intermediate, hidden)), ("up", (intermediate, hidden)),
                        ("down", (hidden, intermediate))):
            out.append(PlanParam(blk, shp[0] * shp[1], True, f"l{layer}.{nm}", shp))
        blk += 1
    if vocab > 0:
        vec(blk, "final_norm")
        out.append(PlanParam(blk, vocab * hidden, True, "lm_head", (vocab, hidden)))
    return out


def random_plan_params(rng: np.random.Generator, blocks: int, max_matrices: int = 6,
                       max_tail: int = 3, max_numel: int = 4096,
                       tie_prob: float = 0.5) -> List[Tuple[int, int, bool]]:
    """Random planner instances: `blocks` blocks (indices shuffled into the parameter order, some
    left empty), each with 0..max_matrices matrices and 0..max_tail non-2D tensors. With
    probability tie_prob the sizes come from a small set so that equal-size roles are common."""
    sizes = rng.integers(0, max_numel + 1, size=4)
    params = []
    order = rng.permutation(blocks)
    for b in order:
        b = int(b)
        if rng.random() < 0.1:
            continue
        items = [True] * int(rng.integers(0, max_matrices + 1)) + [False] * int(rng.integers(0, max_tail + 1))
        rng.shuffle(items)
        for is_m in items:
            if rng.random() < tie_prob:
                numel = int(sizes[int(rng.integers(0, 4))])
            else:
                numel = int(rng.integers(0, max_numel + 1))
            params.append((b, numel, bool(is_m)))
    return params
