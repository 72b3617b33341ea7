"""torch.optim front ends of the owner-local step.

`OwnerMuon`, `OwnerShampoo` and `OwnerSOAP` take the parameters a rank owns (whole tensors, as owner
placement gives them). Each step makes one grouped library call per parameter group for the 2D
matrices (Muon, Shampoo or SOAP) and one for the remaining tensors (AdamW), on torch's current
stream. Optimizer state (fp32 momentum, Shampoo statistics and preconditioners, SOAP moments and
bases, AdamW moments) lives in
`self.state` like torch's own optimizers, so `state_dict()` / `load_state_dict()` work unchanged.
These classes only marshal arguments: every arithmetic step runs in libmfsdp.so, and there is no
CPU path (CUDA tensors are required).
"""
from __future__ import annotations

from typing import Dict, List, Tuple

import torch

from . import native

_MUON_DEFAULTS = dict(lr=1e-3, weight_decay=0.1, momentum=0.95, nesterov=True,
                      ns_coefficients=(3.4445, -4.7750, 2.0315), ns_steps=5, eps=1e-7,
                      lr_adjust="original", ns_dtype="bf16", adamw_lr=1e-3, adamw_betas=(0.9, 0.999),
                      adamw_eps=1e-8, adamw_weight_decay=0.01)
_SHAMPOO_DEFAULTS = dict(lr=1e-3, weight_decay=0.0, beta=1.0, weight=1.0, eps=1e-12, eps_rel=1e-6,
                         root_iters=20, precondition_frequency=1, adamw_lr=1e-3,
                         adamw_betas=(0.9, 0.999), adamw_eps=1e-8, adamw_weight_decay=0.01)

_SOAP_DEFAULTS = dict(lr=3e-3, weight_decay=0.01, beta1=0.95, beta2=0.95, eps=1e-8, shampoo_beta=0.95,
                      precondition_frequency=10, refresh_iters=1, max_precond_dim=4096, adamw_lr=1e-3,
                      adamw_betas=(0.9, 0.999), adamw_eps=1e-8, adamw_weight_decay=0.01)


def _check_tensor(p: torch.Tensor, what: str) -> None:
    if not p.is_cuda:
        raise ValueError(f"{what}: the owner step runs on the GPU only; got a {p.device} tensor")
    if p.dtype not in (torch.float32, torch.bfloat16):
        raise TypeError(f"{what}: dtype must be float32 or bfloat16, got {p.dtype}")
    if p.layout != torch.strided:
        raise ValueError(f"{what}: must be a dense (strided) tensor, got {p.layout}")
    if not p.is_contiguous():
        raise ValueError(f"{what}: must be contiguous")


class _OwnerOptimizer(torch.optim.Optimizer):
    """Shared parts: grouping into matrices and tails, AdamW on the tails, workspace caching."""

    def __init__(self, params, defaults):
        super().__init__(params, defaults)
        self._ws: Dict[Tuple[int, str], Tuple[tuple, torch.Tensor]] = {}

    def _split(self, group) -> Tuple[List[torch.Tensor], List[torch.Tensor]]:
        """The group's parameters with a gradient, 2D matrices and the rest; empty tensors have
        nothing to update and are left out. Every tensor must be a dense CUDA tensor on one device."""
        mats, tails = [], []
        device = None
        for p in group["params"]:
            if p.grad is None or p.numel() == 0:
                continue
            _check_tensor(p, "parameter")
            _check_tensor(p.grad, "gradient")
            if p.grad.device != p.device or p.grad.shape != p.shape:
                raise ValueError("gradient: must have the parameter's shape and device")
            if device is None:
                device = p.device
            elif p.device != device:
                raise ValueError(f"parameters of one group must be on one GPU; got {device} and {p.device}")
            (mats if p.dim() == 2 else tails).append(p)
        return mats, tails

    @torch.no_grad()
    def step(self, closure=None):
        loss = None
        if closure is not None:
            with torch.enable_grad():
                loss = closure()
        for gi, group in enumerate(self.param_groups):
            mats, tails = self._split(group)
            if not mats and not tails:
                continue
            # the library launches on the current device's stream: make it the parameters' device
            with torch.cuda.device((mats or tails)[0].device):
                self._step_group(gi, group, mats, tails)
        return loss

    def _step_group(self, gi: int, group: dict, mats: List[torch.Tensor], tails: List[torch.Tensor]) -> None:
        raise NotImplementedError

    def load_state_dict(self, state_dict) -> None:
        """As torch.optim.Optimizer.load_state_dict, except that the state tensors keep float32:
        the library's momentum, moments, statistics and preconditioners are fp32 whatever the
        parameter dtype (the base class would cast them to the parameter dtype)."""
        saved_state = state_dict["state"]
        saved_groups = state_dict["param_groups"]
        super().load_state_dict(state_dict)
        for sg, g in zip(saved_groups, self.param_groups):
            for sid, p in zip(sg["params"], g["params"]):
                for k, v in saved_state.get(sid, {}).items():
                    if isinstance(v, torch.Tensor) and v.is_floating_point():
                        self.state[p][k] = v.detach().to(device=p.device, dtype=torch.float32).clone()

    def _workspace(self, gi: int, kind: str, key: tuple, size_fn, device) -> torch.Tensor:
        cached = self._ws.get((gi, kind))
        if cached is not None and cached[0] == key:
            return cached[1]
        ws = torch.empty(max(int(size_fn()), 256), dtype=torch.uint8, device=device)
        self._ws[(gi, kind)] = (key, ws)
        return ws

    def _adamw(self, group, tails: List[torch.Tensor]) -> None:
        # the library takes one step count per call: tensors are grouped by their own count
        by_step: Dict[int, list] = {}
        for p in tails:
            st = self.state[p]
            if "exp_avg" not in st:
                st["exp_avg"] = torch.zeros_like(p, dtype=torch.float32)
                st["exp_avg_sq"] = torch.zeros_like(p, dtype=torch.float32)
                st["step"] = 0
            st["step"] += 1
            by_step.setdefault(st["step"], []).append(
                native.adamw_entry_t(p, p.grad, st["exp_avg"], st["exp_avg_sq"]))
        b1, b2 = group["adamw_betas"]
        for step, ents in by_step.items():
            native.adamw_step_t(ents, lr=group["adamw_lr"], beta1=b1, beta2=b2, eps=group["adamw_eps"],
                                weight_decay=group["adamw_weight_decay"], step=step)


class OwnerMuon(_OwnerOptimizer):
    """Muon on the owned 2D matrices (momentum with Nesterov, Frobenius normalisation, quintic
    Newton-Schulz, shape-scaled lr, decoupled weight decay) and AdamW on the other tensors.

    Hyperparameters: lr, weight_decay, momentum, nesterov, ns_coefficients (a, b, c) or
    ns_schedule (one triple per NS step), ns_steps, eps, lr_adjust ("original", "match_rms_adamw",
    "none"), ns_dtype ("bf16" MFMA or "f32"); adamw_lr, adamw_betas, adamw_eps, adamw_weight_decay.
    """

    def __init__(self, params, **kw):
        d = dict(_MUON_DEFAULTS, ns_schedule=None)
        unknown = set(kw) - set(d)
        if unknown:
            raise TypeError(f"unknown hyperparameters: {sorted(unknown)}")
        d.update(kw)
        super().__init__(params, d)

    def _step_group(self, gi: int, group: dict, mats: List[torch.Tensor], tails: List[torch.Tensor]) -> None:
        if mats:
            ents = []
            for p in mats:
                st = self.state[p]
                if "momentum_buffer" not in st:
                    st["momentum_buffer"] = torch.zeros_like(p, dtype=torch.float32)
                ents.append(native.muon_entry_t(p, p.grad, st["momentum_buffer"]))
            a, b, c = group["ns_coefficients"]
            hp = native.muon_hparams(lr=group["lr"], weight_decay=group["weight_decay"],
                                     momentum=group["momentum"], nesterov=group["nesterov"], a=a, b=b,
                                     c=c, ns_steps=group["ns_steps"], eps=group["eps"],
                                     lr_adjust=group["lr_adjust"], ns_dtype=group["ns_dtype"],
                                     ns_schedule=group["ns_schedule"])
            key = (tuple((tuple(p.shape), p.dtype, p.grad.dtype) for p in mats), group["ns_steps"],
                   group["ns_dtype"])
            ws = self._workspace(gi, "muon", key, lambda: native.mfsdp_muon_workspace_size(ents, hp),
                                 mats[0].device)
            native.muon_step_t(ents, hp, ws)
        if tails:
            self._adamw(group, tails)


class OwnerShampoo(_OwnerOptimizer):
    """Shampoo on the owned 2D matrices (statistics L, R, inverse fourth-root preconditioners
    recomputed every `precondition_frequency` steps, decoupled weight decay) and AdamW on the other
    tensors. fp32 math on the GPU.

    Hyperparameters: lr, weight_decay, beta and weight (S <- beta S + weight G G^T), eps and
    eps_rel (ridge eps + eps_rel ||S||_F), root_iters, precondition_frequency; adamw_lr,
    adamw_betas, adamw_eps, adamw_weight_decay.
    """

    def __init__(self, params, **kw):
        d = dict(_SHAMPOO_DEFAULTS)
        unknown = set(kw) - set(d)
        if unknown:
            raise TypeError(f"unknown hyperparameters: {sorted(unknown)}")
        d.update(kw)
        if int(d["precondition_frequency"]) < 1:
            raise ValueError("precondition_frequency must be >= 1")
        super().__init__(params, d)

    def _step_group(self, gi: int, group: dict, mats: List[torch.Tensor], tails: List[torch.Tensor]) -> None:
        # one call per refresh decision: matrices whose preconditioners are due, and the rest
        due: Dict[bool, list] = {True: [], False: []}
        for p in mats:
            st = self.state[p]
            if "L" not in st:
                m, n = p.shape
                for name, d in (("L", m), ("R", n), ("PL", m), ("PR", n)):
                    st[name] = torch.zeros((d, d), dtype=torch.float32, device=p.device)
                st["step"] = 0
            refresh = st["step"] % int(group["precondition_frequency"]) == 0
            st["step"] += 1
            due[refresh].append(p)
        for refresh, ps in due.items():
            if not ps:
                continue
            ents = [native.shampoo_entry_t(p, p.grad, self.state[p]["L"], self.state[p]["R"],
                                           self.state[p]["PL"], self.state[p]["PR"]) for p in ps]
            hp = native.shampoo_hparams(lr=group["lr"], weight_decay=group["weight_decay"],
                                        beta=group["beta"], weight=group["weight"], eps=group["eps"],
                                        eps_rel=group["eps_rel"], refresh=refresh,
                                        root_iters=group["root_iters"])
            key = (tuple((tuple(p.shape), p.dtype, p.grad.dtype) for p in ps), refresh,
                   group["root_iters"])
            ws = self._workspace(gi, "shampoo" + ("+" if refresh else "-"), key,
                                 lambda: native.mfsdp_shampoo_workspace_size(ents, hp), ps[0].device)
            native.shampoo_step_t(ents, hp, ws)
        if tails:
            self._adamw(group, tails)


class OwnerSOAP(_OwnerOptimizer):
    """SOAP on the owned 2D matrices (Adam in the eigenbasis of the Shampoo statistics; the bases
    start at the identity and are refreshed by a power step + QR after the first step and then
    every `precondition_frequency` steps) and AdamW on the other tensors. fp32 math on the GPU. A
    matrix side longer than `max_precond_dim` (at most 4096) has no basis and no statistic (the
    identity on that side); sides up to 65536.

    Hyperparameters: lr, weight_decay, beta1, beta2, eps (Adam in the eigenbasis), shampoo_beta
    (statistics S <- shampoo_beta S + (1 - shampoo_beta) G G^T), precondition_frequency,
    refresh_iters, max_precond_dim; adamw_lr, adamw_betas, adamw_eps, adamw_weight_decay.
    """

    def __init__(self, params, **kw):
        d = dict(_SOAP_DEFAULTS)
        unknown = set(kw) - set(d)
        if unknown:
            raise TypeError(f"unknown hyperparameters: {sorted(unknown)}")
        d.update(kw)
        if int(d["precondition_frequency"]) < 1:
            raise ValueError("precondition_frequency must be >= 1")
        if not 1 <= int(d["max_precond_dim"]) <= 4096:
            raise ValueError("max_precond_dim must be in [1, 4096]")
        super().__init__(params, d)

    def _step_group(self, gi: int, group: dict, mats: List[torch.Tensor], tails: List[torch.Tensor]) -> None:
        # the library takes one step count and one refresh decision per call
        calls: Dict[Tuple[int, bool], list] = {}
        maxd = int(group["max_precond_dim"])
        for p in mats:
            if max(p.shape) > native.SOAP_MAX_SIDE:
                raise ValueError(f"SOAP supports matrix sides up to {native.SOAP_MAX_SIDE}, got {tuple(p.shape)}")
            st = self.state[p]
            if "exp_avg" not in st:
                m, n = p.shape
                st["exp_avg"] = torch.zeros((m, n), dtype=torch.float32, device=p.device)
                st["exp_avg_sq"] = torch.zeros((m, n), dtype=torch.float32, device=p.device)
                # a side beyond max_precond_dim keeps no statistic and no basis
                if m <= maxd:
                    st["L"] = torch.zeros((m, m), dtype=torch.float32, device=p.device)
                    st["QL"] = torch.eye(m, dtype=torch.float32, device=p.device)
                if n <= maxd:
                    st["R"] = torch.zeros((n, n), dtype=torch.float32, device=p.device)
                    st["QR"] = torch.eye(n, dtype=torch.float32, device=p.device)
                st["step"] = 0
            st["step"] += 1
            t = st["step"]
            refresh = t == 1 or t % int(group["precondition_frequency"]) == 0
            calls.setdefault((t, refresh), []).append(p)
        for (t, refresh), ps in calls.items():
            ents = [native.soap_entry_t(p, p.grad, self.state[p]["exp_avg"], self.state[p]["exp_avg_sq"],
                                        self.state[p].get("L"), self.state[p].get("R"), self.state[p].get("QL"),
                                        self.state[p].get("QR")) for p in ps]
            beta_s = float(group["shampoo_beta"])
            hp = native.soap_hparams(lr=group["lr"], weight_decay=group["weight_decay"], beta1=group["beta1"],
                                     beta2=group["beta2"], eps=group["eps"], shampoo_beta=beta_s,
                                     shampoo_weight=1.0 - beta_s, step=t, refresh=refresh,
                                     refresh_iters=group["refresh_iters"], max_precond_dim=maxd)
            key = (tuple((tuple(p.shape), p.dtype, p.grad.dtype) for p in ps), refresh, group["refresh_iters"],
                   maxd)
            ws = self._workspace(gi, "soap" + ("+" if refresh else "-"), key,
                                 lambda: native.mfsdp_soap_workspace_size(ents, hp), ps[0].device)
            native.soap_step_t(ents, hp, ws)
        if tails:
            self._adamw(group, tails)
