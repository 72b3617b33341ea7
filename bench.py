#!/usr/bin/env python3
"""Owner-local Muon step on one MI355X: latency, NS TFLOP/s and roofline fractions.

One "step" is the whole owner update for one synthetic owner share: mfsdp_muon_step over every
owned matrix (momentum + Nesterov, Frobenius normalisation, K quintic Newton-Schulz steps on bf16
MFMA, shape-scaled lr with decoupled weight decay) followed by mfsdp_adamw_step over the tail
tensors. Inputs are resident in HBM before the timed region starts.

Default workload: 4 of 32 Llama-3-8B layers (28 matrices: Wq, Wo 4096x4096; Wk, Wv 1024x4096;
gate, up 14336x4096; down 4096x14336 per layer) plus 8 RMSNorm vectors of 4096 on AdamW.

Prints ONE JSON line. `value` is nominal NS TFLOP/s over the whole step (NS flops / step time);
`roofline` describes the NS GEMM kernel; `cpu_baseline` is the fp64 oracle timed on a bounded
sample of the same share on the host cores. `planner` reports the owner planner (Algorithm 1) on the
paper's decoder sweep (planner time, rank-load imbalance, gamma_B per policy); with --plan-span W it
also runs every rank's planned share on the GPU and reports the step-time imbalance over ranks.
`shampoo` times the Shampoo owner step (fp32 accuracy; products on the bf16 MFMA with split
operands, rates given against the fp32 MFMA peak and the split-product ceiling) on the GPT-2-small share, with and without
preconditioner refresh; `soap` times the SOAP owner step (Adam in the eigenbasis of the Shampoo
statistics) on the same share, with and without the basis refresh (power step + Householder QR), and
`soap_llama_layer` on one Llama-3-8B layer's seven matrices (sides up to 4096 preconditioned: the
14336-long FFN sides keep the identity basis).
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6   # dense bf16 MFMA: 256 CU x 2.4 GHz x 4096 flop/clk/CU
PEAK_HBM_GBS = 8000.0       # HBM3E
PEAK_F32_TFLOPS = 157.3     # dense fp32 MFMA (the fp32 NS path runs v_mfma_f32_32x32x2f32)
METRIC = "owner Muon-step latency (ms) and NS TFLOP/s (% MFMA bf16 peak) at 1 MI355X"
GEMM_KERNEL = "gemm_bf16_kernel"
GEMM_SOURCE = os.path.join(ROOT, "paper_2607_05895_amd", "csrc", "kernels_gemm.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gemm_bf16_traffic_llama3_8b_share.json")


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


class HipEvents:
    """hipEvent_t helpers from the HIP runtime torch already loaded (same runtime instance)."""

    def __init__(self):
        self.hip = ctypes.CDLL("libamdhip64.so.7")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self) -> int:
        ev = ctypes.c_void_p()
        rc = self.hip.hipEventCreate(ctypes.byref(ev))
        if rc != 0:
            raise RuntimeError(f"hipEventCreate failed: {rc}")
        return ev.value

    def record(self, ev: int, stream: int) -> None:
        rc = self.hip.hipEventRecord(ev, stream)
        if rc != 0:
            raise RuntimeError(f"hipEventRecord failed: {rc}")

    def elapsed_ms(self, a: int, b: int) -> float:
        out = ctypes.c_float()
        rc = self.hip.hipEventElapsedTime(ctypes.byref(out), a, b)
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed: {rc}")
        return float(out.value)


def _to_dev(arr, dtype, torch, dev):
    import numpy as np
    import synth
    if dtype == synth.BF16:
        return torch.from_numpy(arr.view(np.int16)).view(torch.bfloat16).to(dev)
    return torch.from_numpy(arr).to(dev)


def device_info(torch) -> dict:
    """The device the numbers come from: name, architecture and CU count from the runtime, and the
    shader clock level the driver marks as current right after the timed region (read from the
    device's sysfs `pp_dpm_sclk`, no child process; null where the file is not readable). Under a long
    MFMA load the clock settles below its maximum."""
    pr = torch.cuda.get_device_properties(0)
    info = {"name": pr.name, "arch": getattr(pr, "gcnArchName", None), "compute_units": pr.multi_processor_count,
            "sclk_after_timing": None}
    try:
        path = (f"/sys/bus/pci/devices/{pr.pci_domain_id:04x}:{pr.pci_bus_id:02x}:"
                f"{pr.pci_device_id:02x}.0/pp_dpm_sclk")
        with open(path) as f:
            for line in f:
                if line.rstrip().endswith("*"):
                    info["sclk_after_timing"] = line.rstrip().rstrip("*").strip()
                    break
    except (OSError, AttributeError, TypeError, ValueError):
        pass
    return info


def cpu_baseline(wl, sample_idx, pool) -> dict:
    """Time the fp64 oracle on a bounded sample of the share (host cores)."""
    import numpy as np
    import oracle
    import synth
    try:
        import threadpoolctl
        threads = max([i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = os.cpu_count() or 1
    hp = wl.hp
    flops = 0.0
    elapsed = 0.0
    for i in sample_idx:
        t = synth.muon_entry(wl, i, pool)
        e = wl.muon[i]
        r, s = min(e.m, e.n), max(e.m, e.n)
        flops += hp.ns_steps * (4.0 * r * r * s + 2.0 * r ** 3)
        t0 = time.perf_counter()
        oracle.muon_step(t.param, t.grad, t.momentum, lr=hp.lr, weight_decay=hp.weight_decay,
                         momentum=hp.momentum, nesterov=hp.nesterov, a=hp.a, b=hp.b, c=hp.c,
                         ns_steps=hp.ns_steps, eps=hp.eps, lr_adjust=hp.lr_adjust)
        elapsed += time.perf_counter() - t0
    names = [wl.muon[i].name + f" {wl.muon[i].m}x{wl.muon[i].n}" for i in sample_idx]
    return {"value": flops / elapsed / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": f"full fp64 oracle Muon step of {len(sample_idx)} of the share's "
                      f"{len(wl.muon)} matrices ({', '.join(names)}): {elapsed:.1f} s for "
                      f"{flops:.3e} nominal NS flop; estimated whole-share step "
                      f"{elapsed * wl.ns_flops_nominal() / flops:.0f} s"}


def _oracle_threads() -> int:
    try:
        import threadpoolctl
        return max([i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        return os.cpu_count() or 1


def cpu_baseline_matrix_opt(which: str, refresh: bool) -> dict:
    """The fp64 oracle's Shampoo or SOAP step with refresh on the GPT-2-small share, timed on one
    matrix of each distinct shape and extrapolated to the share by the shape counts (host cores)."""
    import numpy as np
    import oracle
    import synth
    shapes = [(e.m, e.n) for e in synth.workload(2).muon]
    counts = {}
    for sh in shapes:
        counts[sh] = counts.get(sh, 0) + 1
    rng = np.random.default_rng(11)
    total, sample = 0.0, 0.0
    for (m, n), c in counts.items():
        g = rng.standard_normal((m, n)) * 0.02
        p = rng.standard_normal((m, n)) * 0.02
        t0 = time.perf_counter()
        if which == "shampoo":
            oracle.shampoo.shampoo_step(p, g, np.zeros((m, m)), np.zeros((n, n)), None, None,
                                        oracle.shampoo.ShampooHParams(lr=1e-3, weight_decay=0.01, beta=0.95,
                                                                      weight=0.05, eps=1e-12, eps_rel=1e-6,
                                                                      refresh=refresh))
        else:
            oracle.soap.soap_step(p, g, np.zeros((m, n)), np.zeros((m, n)), np.zeros((m, m)), np.zeros((n, n)),
                                  np.eye(m), np.eye(n), 1, oracle.soap.SoapHParams(lr=3e-3, weight_decay=0.01,
                                                                                  refresh=refresh))
        dt = time.perf_counter() - t0
        sample += dt
        total += c * dt
    return {"ms_per_step": round(total * 1e3, 1), "cores": _oracle_threads(), "kind": "oracle",
            "sample": f"fp64 oracle {which} step with refresh on one matrix of each shape "
                      f"({', '.join(f'{m}x{n}' for (m, n) in counts)}): {sample:.1f} s, extrapolated to "
                      f"the share's {len(shapes)} matrices by shape counts"}


def traffic_record(workload_name: str):
    """HBM traffic of the NS GEMM kernel per launch from the committed rocprofv3 FETCH_SIZE /
    WRITE_SIZE runs (scaled by the plain-copy calibration), if they were taken on the current
    kernel source and on this workload; else None."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    try:
        rec = json.load(open(TRAFFIC_FILE))
        sha = hashlib.sha256(open(GEMM_SOURCE, "rb").read()).hexdigest()
        if rec.get("kernel_source_sha256") != sha or rec.get("workload") != workload_name:
            return None
        return rec
    except Exception:
        return None


def time_reduction(args, native, wl, keep, ents, h, ws, stream, hev, plain_step_ms, plain_prep_ms, es_g):
    """Time mfsdp_muon_step_reduce with W gradient parts per matrix (parts derived on the device
    from each matrix's gradient: the values do not change the cost). The reduction runs inside the
    momentum pass, so its time is the step time minus the plain step's, plus the plain pass."""
    import torch
    import synth
    W = args.grad_parts
    parts = []
    for (p, g, mo) in keep[:len(ents)]:
        parts.append([(g.float() * (1.0 + 0.01 * w)).to(g.dtype) for w in range(W)])
    torch.cuda.synchronize()

    def rstep():
        native.muon_step_reduce_t(ents, parts, 1.0 / W, h, ws)
    for _ in range(args.warmup):
        rstep()
    torch.cuda.synchronize()
    e0, e1 = hev.create(), hev.create()
    hev.record(e0, stream)
    for _ in range(args.steps):
        rstep()
    hev.record(e1, stream)
    torch.cuda.synchronize()
    step_ms = hev.elapsed_ms(e0, e1) / args.steps
    prep_ms = plain_prep_ms + (step_ms - plain_step_ms)
    elts = wl.muon_elements()
    es_ns = 2 if wl.hp.ns_dtype == synth.BF16 else 4
    nbytes = elts * (W * es_g + 8 + 2 * es_ns)      # W parts, momentum in/out, u and u^T
    log(f"reduction W={W}: step {step_ms:.3f} ms, fused momentum+reduction pass ~{prep_ms:.3f} ms "
        f"({nbytes / (prep_ms * 1e-3) / 1e9:.0f} GB/s)")
    return {"grad_parts": W, "ms_per_step": round(step_ms, 4), "reduce_prep_ms": round(prep_ms, 4),
            "reduce_prep_bytes": nbytes,
            "reduce_prep_GBps": round(nbytes / (prep_ms * 1e-3) / 1e9, 1),
            "reduce_prep_frac_hbm": round(nbytes / (prep_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
            "note": "pass time = reduce-step time - plain-step time + plain momentum-pass time"}


# the paper's weak-scaling sweep: decoder layers (hidden 4096, intermediate 16384) per shard span
PLAN_SWEEP = {8: 16, 16: 32, 32: 64, 64: 128}


def _plan_share(params, owner, rank):
    mats = sorted((p.shape for p, o in zip(params, owner) if o == rank and p.is_matrix), reverse=True)
    tails = sorted((p.numel for p, o in zip(params, owner) if o == rank and not p.is_matrix), reverse=True)
    return tuple(mats), tuple(tails)


def _time_share(native, torch, dev, hev, stream, share, hp, ah, steps, warmup, gen):
    """ms per owner step (Muon over the matrices + AdamW over the tail tensors) of one rank's share;
    seeded device-drawn values (the step time does not depend on them)."""
    mats, tails = share
    keep, ents, aents = [], [], []
    for (m, n) in mats:
        p = (torch.randn(m, n, device=dev, generator=gen) * 0.02).to(torch.bfloat16)
        g = (torch.randn(m, n, device=dev, generator=gen) * 1e-3).to(torch.bfloat16)
        mo = torch.randn(m, n, device=dev, generator=gen) * 1e-3
        keep.append((p, g, mo))
        ents.append(native.muon_entry_t(p, g, mo))
    for numel in tails:
        t = (torch.ones(numel, device=dev, dtype=torch.bfloat16),
             (torch.randn(numel, device=dev, generator=gen) * 1e-3).to(torch.bfloat16),
             torch.zeros(numel, device=dev), torch.zeros(numel, device=dev))
        keep.append(t)
        aents.append(native.adamw_entry_t(*t))
    ws = native.muon_workspace_t(ents, hp, device=dev) if ents else None
    a, b = hev.create(), hev.create()

    def step():
        if ents:
            native.mfsdp_muon_step(ents, hp, ws.data_ptr(), ws.numel(), stream)
        if aents:
            native.mfsdp_adamw_step(aents, ah.lr, ah.beta1, ah.beta2, ah.eps, ah.weight_decay, ah.step, stream)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    hev.record(a, stream)
    for _ in range(steps):
        step()
    hev.record(b, stream)
    torch.cuda.synchronize()
    ms = hev.elapsed_ms(a, b) / steps
    del keep, ws
    return ms


def planner_report(native, spans, gpu_span, ctx=None) -> dict:
    """Owner planning (Algorithm 1) on the paper's sweep: planner time, rank-load (resident
    parameter) imbalance max/avg and gamma_B per policy; for gpu_span, every rank's share under
    RoleGreedy and ScopeGreedy (CostAware returns one of the two) run on the GPU, and the
    optimizer-step imbalance max/avg over ranks."""
    import synth
    names = {0: "role_greedy", 1: "scope_greedy", 2: "cost_aware"}
    out = {"model": "decoder, hidden 4096, intermediate 16384, 32 heads (q, k, v, o, gate, up, "
                    "down per layer; 2 RMSNorm vectors per layer as the block tail)",
           "spans": {}}
    for span in spans:
        layers = PLAN_SWEEP[span]
        params = synth.decoder_plan_params(layers)
        tuples = [p.tuple() for p in params]
        rec = {"layers": layers, "parameters": len(params), "numel": sum(p.numel for p in params)}
        owners = {}
        for pol in (0, 1, 2):
            reps, best = 5, float("inf")
            for _ in range(reps):
                t0 = time.perf_counter()
                owner, loads, gam, used = native.mfsdp_plan_owners(tuples, span, pol, 0.0)
                best = min(best, time.perf_counter() - t0)
            avg = sum(loads) / span
            rec[names[pol]] = {"plan_ms": round(best * 1e3, 3),
                               "load_max_over_avg": round(max(loads) / avg, 4),
                               "gamma_max": round(max(gam), 4),
                               "gamma_mean": round(sum(gam) / len(gam), 4),
                               "policy_used": names[used]}
            owners[pol] = owner
        if span == gpu_span and ctx is not None:
            torch, dev, hev, stream, hp, ah, steps, warmup = ctx
            gen = torch.Generator(device=dev)
            gen.manual_seed(span)
            cache = {}
            for pol in (0, 1):
                shares = [_plan_share(params, owners[pol], r) for r in range(span)]
                for r, sh in enumerate(shares):
                    if sh not in cache:
                        log(f"planner: span {span}, {names[pol]}: timing rank {r}'s share ({len(sh[0])} "
                            f"matrices, {len(sh[1])} tail tensors)")
                        cache[sh] = _time_share(native, torch, dev, hev, stream, sh, hp, ah, steps, warmup, gen)
                ms = [cache[sh] for sh in shares]
                heavy = max(range(span), key=lambda r: ms[r])
                rec[names[pol]]["gpu_owner_step"] = {
                    "distinct_shares": len(set(shares)),
                    "ms_max": round(max(ms), 4), "ms_mean": round(sum(ms) / span, 4), "ms_min": round(min(ms), 4),
                    "step_max_over_avg": round(max(ms) / (sum(ms) / span), 4),
                    "heaviest_rank": heavy,
                    "heaviest_share_matrices": [list(x) for x in shares[heavy][0]],
                    "heaviest_share_tail_tensors": len(shares[heavy][1])}
        out["spans"][str(span)] = rec
    return out


PEAK_F32_MFMA_TFLOPS = 157.3  # dense fp32 MFMA
# Shampoo / SOAP products run on the bf16 MFMA with each fp32 operand split into three bf16 parts
# (six bf16 products per fp32 product): their ceiling in fp32 flop is the bf16 peak / 6
PEAK_SPLIT_TFLOPS = PEAK_BF16_TFLOPS / 6.0


def shampoo_nominal_flop(shapes, iters: int, refresh: bool) -> float:
    """Nominal flop of one Shampoo step: statistics G G^T and G^T G, P_L G and (P_L G) P_R, and on
    refresh 4 iters - 3 products of d x d per side (the last iteration forms X only)."""
    tot = 0.0
    for m, n in shapes:
        tot += 2.0 * m * m * n + 2.0 * m * n * n          # statistics
        tot += 2.0 * m * m * n + 2.0 * m * n * n          # U = P_L G P_R
        if refresh:
            tot += (4 * iters - 3) * 2.0 * (m ** 3 + n ** 3)
    return tot


def _dist_draw(torch, shape, dist, dtype, dev, gen):
    """Seeded device draw of N(dist.mean, dist.std^2) (a constant when std == 0)."""
    x = torch.randn(*shape, device=dev, generator=gen) * dist.std + dist.mean
    return x.to(dtype)


def share_record(native, torch, dev, hev, stream, index, steps, warmup) -> dict:
    """One owner share (synth.workload(index)) timed like the headline share: values drawn on the
    device from a seeded generator with the share's distributions (the cost does not depend on them),
    warmup + `steps` whole owner steps (Muon over every matrix, then AdamW over the tail tensors),
    phase events from mfsdp_muon_step_timed. The share's largest AdamW tensor (the uneven plan's
    128256 x 4096 embedding) is also timed on its own."""
    import synth
    wl = synth.workload(index)
    hp = wl.hp
    gen = torch.Generator(device=dev)
    gen.manual_seed(1000 + index)
    tdt = {synth.BF16: torch.bfloat16, synth.F32: torch.float32}
    keep, ents, aents = [], [], []
    for e in wl.muon:
        p = _dist_draw(torch, (e.m, e.n), e.param, tdt[e.param_dtype], dev, gen)
        g = _dist_draw(torch, (e.m, e.n), e.grad, tdt[e.grad_dtype], dev, gen)
        mo = _dist_draw(torch, (e.m, e.n), e.momentum, torch.float32, dev, gen)
        keep.append((p, g, mo))
        ents.append(native.muon_entry_t(p, g, mo))
    for e in wl.adamw:
        t = (_dist_draw(torch, (e.numel,), e.param, tdt[e.param_dtype], dev, gen),
             _dist_draw(torch, (e.numel,), e.grad, tdt[e.grad_dtype], dev, gen),
             torch.zeros(e.numel, device=dev), torch.zeros(e.numel, device=dev))
        keep.append(t)
        aents.append(native.adamw_entry_t(*t))
    h = native.muon_hparams(lr=hp.lr, weight_decay=hp.weight_decay, momentum=hp.momentum,
                            nesterov=hp.nesterov, a=hp.a, b=hp.b, c=hp.c, ns_steps=hp.ns_steps,
                            eps=hp.eps, lr_adjust=hp.lr_adjust, ns_dtype=hp.ns_dtype)
    ws = native.muon_workspace_t(ents, h, device=dev)
    ah = wl.adamw_hp
    ev = [[hev.create() for _ in range(4)] for _ in range(steps)]
    e0, e1 = hev.create(), hev.create()

    def step(events=None):
        native.mfsdp_muon_step_timed(ents, h, ws.data_ptr(), ws.numel(), stream, events or [None] * 4)
        if aents:
            native.mfsdp_adamw_step(aents, ah.lr, ah.beta1, ah.beta2, ah.eps, ah.weight_decay, ah.step, stream)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    hev.record(e0, stream)
    for k in range(steps):
        step(ev[k])
    hev.record(e1, stream)
    torch.cuda.synchronize()
    ms = hev.elapsed_ms(e0, e1) / steps
    prep_ms = sum(hev.elapsed_ms(x[0], x[1]) for x in ev) / steps
    ns_ms = sum(hev.elapsed_ms(x[1], x[2]) for x in ev) / steps
    bf16_ns = hp.ns_dtype == synth.BF16
    peak = PEAK_BF16_TFLOPS if bf16_ns else PEAK_F32_TFLOPS
    flops = wl.ns_flops_nominal()
    es = {synth.BF16: 2, synth.F32: 4}
    prep_bytes = sum(e.m * e.n * (es[e.grad_dtype] + 8 + 2 * es[hp.ns_dtype]) for e in wl.muon)
    rec = {"workload": wl.name, "description": wl.description, "muon_matrices": len(wl.muon),
           "muon_elements": wl.muon_elements(), "adamw_elements": wl.adamw_elements(),
           "ns_dtype": "bf16" if bf16_ns else "f32", "steps": steps, "warmup": warmup,
           "ms_per_step": round(ms, 4), "ns_ms": round(ns_ms, 4), "prep_norm_ms": round(prep_ms, 4),
           "nominal_ns_flop_per_step": flops,
           "ns_tflops": round(flops / (ns_ms * 1e-3) / 1e12, 2),
           "ns_frac_peak": round(flops / (ns_ms * 1e-3) / 1e12 / peak, 4), "peak_tflops": peak,
           "prep_GBps": round(prep_bytes / (prep_ms * 1e-3) / 1e9, 1),
           "prep_frac_hbm": round(prep_bytes / (prep_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
           "data": "seeded device draws with the share's distributions"}
    log(f"share {wl.name}: {ms:.3f} ms per step, NS {ns_ms:.3f} ms ({rec['ns_tflops']} TFLOP/s, "
        f"{rec['ns_frac_peak']:.3f} of peak), prep {rec['prep_GBps']} GB/s")
    del ws
    big = max(range(len(wl.adamw)), key=lambda j: wl.adamw[j].numel, default=None)
    if big is not None and wl.adamw[big].numel >= (1 << 24):
        e = wl.adamw[big]
        one = [aents[big]]
        for _ in range(warmup):
            native.mfsdp_adamw_step(one, ah.lr, ah.beta1, ah.beta2, ah.eps, ah.weight_decay, ah.step, stream)
        torch.cuda.synchronize()
        hev.record(e0, stream)
        for _ in range(steps):
            native.mfsdp_adamw_step(one, ah.lr, ah.beta1, ah.beta2, ah.eps, ah.weight_decay, ah.step, stream)
        hev.record(e1, stream)
        torch.cuda.synchronize()
        ams = hev.elapsed_ms(e0, e1) / steps
        nb = e.numel * (2 * es[e.param_dtype] + es[e.grad_dtype] + 16)
        rec["adamw_largest"] = {"tensor": e.name, "numel": e.numel, "bytes": nb, "ms": round(ams, 4),
                                "GBps": round(nb / (ams * 1e-3) / 1e9, 1),
                                "frac_hbm": round(nb / (ams * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}
        log(f"AdamW on {e.name} ({e.numel / 1e6:.1f} M elements): {ams:.3f} ms, "
            f"{rec['adamw_largest']['GBps']} GB/s")
    del keep, ents, aents
    torch.cuda.empty_cache()
    return rec


def time_shampoo(native, torch, dev, hev, stream, steps, warmup, iters=20) -> dict:
    """The Shampoo owner step (Section 5.7) on the GPT-2-small share's 12 matrices, fp32 accuracy."""
    import synth
    wl = synth.workload(2)
    shapes = [(e.m, e.n) for e in wl.muon]
    gen = torch.Generator(device=dev)
    gen.manual_seed(2)
    keep, ents = [], []
    for m, n in shapes:
        t = ((torch.randn(m, n, device=dev, generator=gen) * 0.02).to(torch.bfloat16),
             (torch.randn(m, n, device=dev, generator=gen) * 0.02).to(torch.bfloat16),
             torch.zeros(m, m, device=dev), torch.zeros(n, n, device=dev),
             torch.zeros(m, m, device=dev), torch.zeros(n, n, device=dev))
        keep.append(t)
        ents.append(native.shampoo_entry_t(*t))
    out = {"workload": wl.name + " (12 matrices: 8 x 768x768, 2 x 3072x768, 2 x 768x3072)",
           "root_iters": iters, "ridge": "1e-12 + 1e-6 ||S||_F", "dtype": "f32"}
    for refresh in (True, False):
        hp = native.shampoo_hparams(lr=1e-3, weight_decay=0.01, beta=0.95, weight=0.05, eps=1e-12,
                                    eps_rel=1e-6, refresh=refresh, root_iters=iters)
        ws = native.shampoo_workspace_t(ents, hp, device=dev)
        for _ in range(warmup):
            native.shampoo_step_t(ents, hp, ws)
        torch.cuda.synchronize()
        a, b = hev.create(), hev.create()
        hev.record(a, stream)
        for _ in range(steps):
            native.shampoo_step_t(ents, hp, ws)
        hev.record(b, stream)
        torch.cuda.synchronize()
        ms = hev.elapsed_ms(a, b) / steps
        fl = shampoo_nominal_flop(shapes, iters, refresh)
        key = "refresh" if refresh else "stale_preconditioners"
        out[key] = {"ms_per_step": round(ms, 4), "nominal_flop_per_step": fl,
                    "nominal_tflops": round(fl / (ms * 1e-3) / 1e12, 2),
                    "x_fp32_mfma_peak": round(fl / (ms * 1e-3) / 1e12 / PEAK_F32_MFMA_TFLOPS, 4),
                    "frac_split_bf16_peak": round(fl / (ms * 1e-3) / 1e12 / PEAK_SPLIT_TFLOPS, 4),
                    "workspace_gib": round(ws.numel() / 2 ** 30, 3)}
        log(f"shampoo ({key}): {ms:.3f} ms per step, {fl / (ms * 1e-3) / 1e12:.1f} nominal TFLOP/s")
        del ws
    return out


def soap_nominal_flop(shapes, refresh_iters: int, refresh: bool, max_precond_dim: int = 4096) -> float:
    """Nominal flop of one SOAP step: per side with a basis (length <= max_precond_dim), on the left
    Q_L^T [G | M] (4 m^2 n), Q_L N' (2 m^2 n) and the statistic G G^T (2 m^2 n), on the right [G' | M']
    Q_R (4 m n^2), (Q_L N') Q_R^T (2 m n^2) and G^T G (2 m n^2); per refresh iteration and side the
    power step S Q (2 d^3) and a Householder QR with the explicit Q (LAPACK's count, 4/3 d^3 for the
    factorization and 4/3 d^3 for forming Q)."""
    tot = 0.0
    for m, n in shapes:
        for d, other in ((m, n), (n, m)):
            if d <= max_precond_dim:
                tot += 8.0 * d * d * other
                if refresh:
                    tot += refresh_iters * (2.0 + 8.0 / 3.0) * d ** 3
    return tot


def time_soap(native, torch, dev, hev, stream, steps, warmup, shapes=None, label=None,
              max_precond_dim=4096, tag="soap") -> dict:
    """The SOAP owner step (Section 5.7), fp32 math, bases starting at the identity and statistics at
    zero (the cost does not depend on the values): by default on the GPT-2-small share's 12
    matrices; sides longer than max_precond_dim keep the identity basis."""
    import synth
    if shapes is None:
        wl = synth.workload(2)
        shapes = [(e.m, e.n) for e in wl.muon]
        label = wl.name + " (12 matrices: 8 x 768x768, 2 x 3072x768, 2 x 768x3072)"
    gen = torch.Generator(device=dev)
    gen.manual_seed(3)
    keep, ents = [], []
    for m, n in shapes:
        t = ((torch.randn(m, n, device=dev, generator=gen) * 0.02).to(torch.bfloat16),
             (torch.randn(m, n, device=dev, generator=gen) * 0.02).to(torch.bfloat16),
             torch.zeros(m, n, device=dev), torch.zeros(m, n, device=dev),
             torch.zeros(m, m, device=dev) if m <= max_precond_dim else None,
             torch.zeros(n, n, device=dev) if n <= max_precond_dim else None,
             torch.eye(m, device=dev) if m <= max_precond_dim else None,
             torch.eye(n, device=dev) if n <= max_precond_dim else None)
        keep.append(t)
        ents.append(native.soap_entry_t(*t))
    out = {"workload": label, "dtype": "f32", "betas": [0.95, 0.95], "shampoo_beta": 0.95,
           "max_precond_dim": max_precond_dim}
    step_no = 1
    for refresh in (True, False):
        hp = native.soap_hparams(lr=3e-3, weight_decay=0.01, refresh=refresh, refresh_iters=1,
                                 max_precond_dim=max_precond_dim)
        ws = native.soap_workspace_t(ents, hp, device=dev)

        def one():
            nonlocal step_no
            hp.step = step_no
            native.soap_step_t(ents, hp, ws)
            step_no += 1
        for _ in range(warmup):
            one()
        torch.cuda.synchronize()
        a, b = hev.create(), hev.create()
        hev.record(a, stream)
        for _ in range(steps):
            one()
        hev.record(b, stream)
        torch.cuda.synchronize()
        ms = hev.elapsed_ms(a, b) / steps
        fl = soap_nominal_flop(shapes, 1, refresh, max_precond_dim)
        key = "refresh" if refresh else "no_refresh"
        out[key] = {"ms_per_step": round(ms, 4), "nominal_flop_per_step": fl,
                    "nominal_tflops": round(fl / (ms * 1e-3) / 1e12, 2),
                    "x_fp32_mfma_peak": round(fl / (ms * 1e-3) / 1e12 / PEAK_F32_MFMA_TFLOPS, 4),
                    "frac_split_bf16_peak": round(fl / (ms * 1e-3) / 1e12 / PEAK_SPLIT_TFLOPS, 4),
                    "workspace_gib": round(ws.numel() / 2 ** 30, 3)}
        log(f"{tag} ({key}): {ms:.3f} ms per step, {fl / (ms * 1e-3) / 1e12:.1f} nominal TFLOP/s")
        del ws
    del keep, ents
    torch.cuda.empty_cache()
    return out


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", type=int, default=3, help="owner share 1..5 (default 3: Llama-3-8B)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--grad-parts", type=int, default=0,
                    help="also time the owner-side gradient reduction fused with the step: each "
                         "matrix's gradient arrives as this many full-size parts (shard span W)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="before timing, run one plain 1 GiB -> 1 GiB elementwise copy kernel (the "
                         "reference dispatch for scaling HBM counters)")
    ap.add_argument("--plan-span", type=int, default=0, choices=[0] + sorted(PLAN_SWEEP),
                    help="also run every rank's owner share of the planned decoder sweep model at this "
                         "shard span on the GPU and report the step-time imbalance over ranks")
    ap.add_argument("--no-shampoo", action="store_true",
                    help="skip timing the Shampoo owner step on the GPT-2-small share")
    ap.add_argument("--shampoo", action="store_true", help=argparse.SUPPRESS)  # (the default)
    ap.add_argument("--no-soap", action="store_true", help="skip the SOAP owner-step timing")
    ap.add_argument("--no-other-shares", action="store_true",
                    help="skip timing the other owner shares (1, 2, 4, 5 besides the default 3)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on exactly one GPU: the owner-local Muon "
                                   "step has no cross-GPU work; run with --gpus 1"}), flush=True)
        return 2
    if int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print(json.dumps({"error": "launched with WORLD_SIZE > 1; this benchmark is single-GPU"}))
        return 2

    import numpy as np
    import torch

    import synth
    from paper_2607_05895_amd import native

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    wl = synth.workload(args.workload)
    hp = wl.hp
    pool = synth.thread_pool()
    log(f"workload {wl.name}: {len(wl.muon)} matrices, {wl.muon_elements() / 1e6:.1f} M Muon "
        f"elements, {wl.adamw_elements() / 1e6:.2f} M AdamW elements; generating inputs")
    t0 = time.time()
    keep, ents = [], []
    for i, e in enumerate(wl.muon):
        t = synth.muon_entry(wl, i, pool)
        p = _to_dev(t.param, e.param_dtype, torch, dev)
        g = _to_dev(t.grad, e.grad_dtype, torch, dev)
        mo = _to_dev(t.momentum, synth.F32, torch, dev)
        keep.append((p, g, mo))
        ents.append(native.muon_entry_t(p, g, mo))
    aents = []
    for j, e in enumerate(wl.adamw):
        t = synth.adamw_entry(wl, j, pool)
        tens = (_to_dev(t.param, e.param_dtype, torch, dev), _to_dev(t.grad, e.grad_dtype, torch, dev),
                _to_dev(t.exp_avg, synth.F32, torch, dev), _to_dev(t.exp_avg_sq, synth.F32, torch, dev))
        keep.append(tens)
        aents.append(native.adamw_entry_t(*tens))
    h = native.muon_hparams(lr=hp.lr, weight_decay=hp.weight_decay, momentum=hp.momentum,
                            nesterov=hp.nesterov, a=hp.a, b=hp.b, c=hp.c, ns_steps=hp.ns_steps,
                            eps=hp.eps, lr_adjust=hp.lr_adjust, ns_dtype=hp.ns_dtype)
    ws = native.muon_workspace_t(ents, h, device=dev)
    torch.cuda.synchronize()
    log(f"inputs resident ({time.time() - t0:.1f} s); workspace {ws.numel() / 2**30:.2f} GiB")

    if args.copy_calibration:
        x = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        y = torch.empty_like(x)
        torch.mul(x, 2.0, out=y)
        torch.cuda.synchronize()
        log("copy calibration: one elementwise kernel reading 1 GiB and writing 1 GiB")
        del x, y

    ah = wl.adamw_hp
    stream = torch.cuda.current_stream().cuda_stream
    hev = HipEvents()
    n_ev = args.steps
    ev = [[hev.create() for _ in range(6)] for _ in range(n_ev)]
    ev_start, ev_stop = hev.create(), hev.create()

    def step(events=None, aev=None):
        native.mfsdp_muon_step_timed(ents, h, ws.data_ptr(), ws.numel(), stream,
                                     events if events else [None] * 4)
        if aents:
            if aev:
                hev.record(aev[0], stream)
            native.mfsdp_adamw_step(aents, ah.lr, ah.beta1, ah.beta2, ah.eps, ah.weight_decay,
                                    ah.step, stream)
            if aev:
                hev.record(aev[1], stream)

    for w in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"warmup done ({args.warmup} steps); timing {args.steps} steps")
    hev.record(ev_start, stream)
    for k in range(args.steps):
        step(ev[k][:4], ev[k][4:6])
    hev.record(ev_stop, stream)
    torch.cuda.synchronize()
    total_ms = hev.elapsed_ms(ev_start, ev_stop)
    ms_per_step = total_ms / args.steps
    # per-step times: from one step's first event to the next step's (the last one to the stop)
    step_ms = sorted(hev.elapsed_ms(ev[k][0], ev[k + 1][0] if k + 1 < n_ev else ev_stop)
                     for k in range(n_ev))
    prep_ms = sum(hev.elapsed_ms(e[0], e[1]) for e in ev) / n_ev
    ns_ms = sum(hev.elapsed_ms(e[1], e[2]) for e in ev) / n_ev
    apply_ms = sum(hev.elapsed_ms(e[2], e[3]) for e in ev) / n_ev
    adamw_ms = (sum(hev.elapsed_ms(e[4], e[5]) for e in ev) / n_ev) if aents else 0.0
    log(f"step {ms_per_step:.3f} ms: prep+norm {prep_ms:.3f}, NS {ns_ms:.3f}, apply {apply_ms:.3f}, "
        f"AdamW {adamw_ms:.3f}")
    if hp.ns_dtype == synth.BF16 and hp.ns_steps >= 1:
        apply_ms = 0.0  # the events around the (absent) apply pass bracket no kernel

    flops = wl.ns_flops_nominal()
    bf16_ns = hp.ns_dtype == synth.BF16
    peak = PEAK_BF16_TFLOPS if bf16_ns else PEAK_F32_TFLOPS
    launches = 3 * hp.ns_steps
    ns_tflops = flops / (ns_ms * 1e-3) / 1e12 if ns_ms > 0 else 0.0
    value = flops / (ms_per_step * 1e-3) / 1e12
    elts = wl.muon_elements()
    es_g = 2 if all(e.grad_dtype == synth.BF16 for e in wl.muon) else 4
    es_p = 2 if all(e.param_dtype == synth.BF16 for e in wl.muon) else 4
    es_ns = 2 if hp.ns_dtype == synth.BF16 else 4
    prep_bytes = elts * (es_g + 4 + 4 + 2 * es_ns)       # g, m in/out, u and u^T
    # on the bf16 path the parameter update runs in the last NS update's epilogue (no apply pass)
    apply_fused = hp.ns_dtype == synth.BF16 and hp.ns_steps >= 1
    apply_bytes = 0 if apply_fused else elts * (es_ns + 2 * es_p)   # O, p in/out
    alg_bytes = elts * (es_g + 8 + 2 * es_p)              # g, m in/out, p in/out
    adamw_bytes = sum(e.numel * ({"bf16": 2, "f32": 4}[e.param_dtype] * 2 +
                                 {"bf16": 2, "f32": 4}[e.grad_dtype] + 16) for e in wl.adamw)
    trec = traffic_record(wl.name)
    traffic = trec["bytes_per_launch"] if trec else None
    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if hp.ns_dtype == synth.BF16 else "f32",
        "data": "synthetic (seeded Gaussian gradients/params/momentum of the share's shapes)",
        "config": {"workload": wl.name, "description": wl.description,
                   "muon_matrices": len(wl.muon), "muon_elements": elts,
                   "adamw_tensors": len(wl.adamw), "adamw_elements": wl.adamw_elements(),
                   "ns_steps": hp.ns_steps, "ns_coefficients": [hp.a, hp.b, hp.c],
                   "momentum": hp.momentum, "nesterov": hp.nesterov, "lr": hp.lr,
                   "weight_decay": hp.weight_decay, "lr_adjust": hp.lr_adjust,
                   "nominal_ns_flop_per_step": flops},
        "roofline": {
            "kernel": GEMM_KERNEL if bf16_ns else "gemm_f32_kernel",
            "bound": "mfma",
            "achieved": round(ns_tflops, 2),
            "peak": peak,
            "unit": "TFLOP/s",
            "frac": round(ns_tflops / peak, 4),
            "traffic": traffic,
            "traffic_unit": "bytes per launch (HBM, calibrated rocprofv3 FETCH_SIZE + WRITE_SIZE)",
            "algorithmic_bytes_per_launch": trec["algorithmic_bytes_per_launch"] if trec else None,
            "launches_per_step": launches,
            "avg_launch_ms": round(ns_ms / launches, 4) if launches else 0.0,
            "nominal_flop_per_launch": flops / launches if launches else 0.0,
        },
        "step_ms_stats": {"median": round(step_ms[len(step_ms) // 2], 4), "min": round(step_ms[0], 4),
                          "max": round(step_ms[-1], 4)},
        "device": device_info(torch),
        # (nominal NS flop / MFMA peak + algorithmic elementwise bytes / HBM peak) / step time
        "step_roofline_frac": round((flops / (peak * 1e12) + (alg_bytes + adamw_bytes) / (PEAK_HBM_GBS * 1e9))
                                    / (ms_per_step * 1e-3), 4),
        "phases_ms": {"prep_norm": round(prep_ms, 4), "ns": round(ns_ms, 4),
                      "apply": round(apply_ms, 4), "adamw": round(adamw_ms, 4)},
        "elementwise": {
            "prep_GBps": round(prep_bytes / (prep_ms * 1e-3) / 1e9, 1) if prep_ms else None,
            "apply_fused_into_ns": apply_fused,
            "apply_GBps": (round(apply_bytes / (apply_ms * 1e-3) / 1e9, 1)
                           if apply_ms and not apply_fused else None),
            "muon_elementwise_frac_hbm": (round((prep_bytes + apply_bytes) / ((prep_ms + apply_ms) * 1e-3) / 1e9
                                                / PEAK_HBM_GBS, 4) if (prep_ms + apply_ms) else None),
            "muon_algorithmic_bytes": alg_bytes,
            "adamw_GBps": round(adamw_bytes / (adamw_ms * 1e-3) / 1e9, 1) if adamw_ms else None,
        },
    }
    if args.grad_parts > 0:
        out["grad_reduction"] = time_reduction(args, native, wl, keep, ents, h, ws, stream, hev,
                                               ms_per_step, prep_ms, es_g)
    log("owner planner on the decoder sweep" + (f" (GPU shares at span {args.plan_span})"
                                                  if args.plan_span else ""))
    pctx = (torch, dev, hev, stream, h, ah, 5, 2) if args.plan_span else None
    out["planner"] = planner_report(native, sorted(PLAN_SWEEP), args.plan_span, pctx)
    if not args.no_other_shares:
        # the other owner shares, each timed on its own (the headline stays the share above)
        others = [i for i in (1, 2, 3, 4, 5) if i != args.workload]
        del ws
        torch.cuda.empty_cache()
        out["other_shares"] = {}
        for i in others:
            log(f"timing owner share {i}")
            out["other_shares"][synth.workload(i).name] = share_record(
                native, torch, dev, hev, stream, i, max(5, args.steps // 4), 2)
    if not args.no_shampoo:
        # nominal_flop counts every product of all root iterations in full; iterations skipped
        # after convergence and the upper-tile-only symmetric products execute less
        out["shampoo"] = time_shampoo(native, torch, dev, hev, stream, max(3, args.steps // 4), 1)
    if not args.no_soap:
        out["soap"] = time_soap(native, torch, dev, hev, stream, max(3, args.steps // 4), 1)
        # one Llama-3-8B layer: q, k, v, o, gate, up, down
        layer = [(4096, 4096), (1024, 4096), (1024, 4096), (4096, 4096), (14336, 4096), (14336, 4096),
                 (4096, 14336)]
        out["soap_llama_layer"] = time_soap(
            native, torch, dev, hev, stream, 3, 1, layer,
            "llama3_8b_layer (q, k, v, o 4096x4096 / 1024x4096, gate, up 14336x4096, down 4096x14336)",
            tag="soap_llama_layer")
    if not args.no_cpu_baseline:
        # about 10-30 s of fp64 work on the host: one matrix of each Llama-3-8B shape
        sample = {3: [0, 1, 4, 6], 2: list(range(12)), 1: [0], 4: [0, 1], 5: [1]}.get(args.workload, [0])
        log("timing the fp64 oracle on a bounded sample (cpu_baseline)")
        out["cpu_baseline"] = cpu_baseline(wl, sample, pool)
        for key in ("shampoo", "soap"):
            if key in out:
                log(f"timing the fp64 {key} oracle on one matrix of each shape")
                out[key]["cpu_baseline"] = cpu_baseline_matrix_opt(key, True)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
