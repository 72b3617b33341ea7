"""ctypes binding of libmfsdp.so (the C ABI in include/mfsdp.h).

Argument marshalling only: every step of the owner update runs in the library's HIP kernels.
The functions keep the C names; the ``*_t`` helpers accept torch tensors and pass their device
pointers and the current HIP stream. Loading fails loudly if the library has not been built.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence, Tuple

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libmfsdp.so")

F32, BF16 = 0, 1
LR_NONE, LR_ORIGINAL, LR_MATCH_RMS_ADAMW = 0, 1, 2
OK, E_INVALID, E_WORKSPACE, E_HIP = 0, -1, -2, -3
_NS_DT = {"bf16": BF16, "f32": F32}
_LR_MODES = {"none": LR_NONE, "original": LR_ORIGINAL, "match_rms_adamw": LR_MATCH_RMS_ADAMW}
EXPORTS = ("mfsdp_muon_workspace_size", "mfsdp_muon_step", "mfsdp_muon_step_timed", "mfsdp_ns_workspace_size",
           "mfsdp_newton_schulz", "mfsdp_newton_schulz_schedule", "mfsdp_adamw_step", "mfsdp_last_error",
           "mfsdp_status_string", "mfsdp_abi_version", "mfsdp_muon_step_reduce", "mfsdp_plan_owners",
           "mfsdp_shampoo_workspace_size", "mfsdp_shampoo_step", "mfsdp_inverse_root_workspace_size",
           "mfsdp_inverse_root", "mfsdp_soap_workspace_size", "mfsdp_soap_step",
           "mfsdp_orthonormal_factor_workspace_size", "mfsdp_orthonormal_factor", "mfsdp_build_id",
           "mfsdp_muon_step_noalloc", "mfsdp_plan_layouts")
NOALLOC_SCRATCH_BYTES = 64 << 20
MAX_GRAD_PARTS = 64
ABI_VERSION = 6
SOAP_MAX_DIM = 4096     # longest side with a basis (max_precond_dim at most this)
SOAP_MAX_SIDE = 65536   # longest side of a SOAP matrix


class MuonEntry(ctypes.Structure):
    _fields_ = [("param", ctypes.c_void_p), ("grad", ctypes.c_void_p),
                ("momentum", ctypes.c_void_p), ("m", ctypes.c_int64), ("n", ctypes.c_int64),
                ("param_dtype", ctypes.c_int32), ("grad_dtype", ctypes.c_int32),
                ("update_out", ctypes.c_void_p)]


class MuonHParams(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_double), ("weight_decay", ctypes.c_double),
                ("momentum", ctypes.c_double), ("nesterov", ctypes.c_int32),
                ("a", ctypes.c_double), ("b", ctypes.c_double), ("c", ctypes.c_double),
                ("ns_steps", ctypes.c_int32), ("eps", ctypes.c_double),
                ("lr_adjust", ctypes.c_int32), ("ns_dtype", ctypes.c_int32),
                ("ns_schedule", ctypes.POINTER(ctypes.c_double))]


class AdamWEntry(ctypes.Structure):
    _fields_ = [("param", ctypes.c_void_p), ("grad", ctypes.c_void_p),
                ("exp_avg", ctypes.c_void_p), ("exp_avg_sq", ctypes.c_void_p),
                ("numel", ctypes.c_int64), ("param_dtype", ctypes.c_int32),
                ("grad_dtype", ctypes.c_int32)]


class ShampooEntry(ctypes.Structure):
    _fields_ = [("param", ctypes.c_void_p), ("grad", ctypes.c_void_p), ("L", ctypes.c_void_p),
                ("R", ctypes.c_void_p), ("PL", ctypes.c_void_p), ("PR", ctypes.c_void_p),
                ("m", ctypes.c_int64), ("n", ctypes.c_int64), ("param_dtype", ctypes.c_int32),
                ("grad_dtype", ctypes.c_int32), ("update_out", ctypes.c_void_p)]


class ShampooHParams(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_double), ("weight_decay", ctypes.c_double), ("beta", ctypes.c_double),
                ("weight", ctypes.c_double), ("eps", ctypes.c_double), ("eps_rel", ctypes.c_double),
                ("refresh", ctypes.c_int32), ("root_iters", ctypes.c_int32)]


class SoapEntry(ctypes.Structure):
    _fields_ = [("param", ctypes.c_void_p), ("grad", ctypes.c_void_p), ("exp_avg", ctypes.c_void_p),
                ("exp_avg_sq", ctypes.c_void_p), ("L", ctypes.c_void_p), ("R", ctypes.c_void_p),
                ("QL", ctypes.c_void_p), ("QR", ctypes.c_void_p), ("m", ctypes.c_int64), ("n", ctypes.c_int64),
                ("param_dtype", ctypes.c_int32), ("grad_dtype", ctypes.c_int32), ("update_out", ctypes.c_void_p)]


class SoapHParams(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_double), ("weight_decay", ctypes.c_double), ("beta1", ctypes.c_double),
                ("beta2", ctypes.c_double), ("eps", ctypes.c_double), ("shampoo_beta", ctypes.c_double),
                ("shampoo_weight", ctypes.c_double), ("step", ctypes.c_int32), ("refresh", ctypes.c_int32),
                ("refresh_iters", ctypes.c_int32), ("max_precond_dim", ctypes.c_int32)]


class PlanParam(ctypes.Structure):
    _fields_ = [("block", ctypes.c_int32), ("is_matrix", ctypes.c_int32), ("numel", ctypes.c_int64)]


PLAN_ROLE_GREEDY, PLAN_SCOPE_GREEDY, PLAN_COST_AWARE = 0, 1, 2


class MfsdpError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{msg} (status {status})")
        self.status = status


_lib = None


def lib() -> ctypes.CDLL:
    """Load libmfsdp.so once. Raises if it is missing, or if it was built from other sources than the
    ones in the tree (its embedded build identifier differs): there is no fallback path."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2607_05895_amd.build_lib`")
        # torch (the memory/stream plumbing) must be loaded first so the library binds to the same
        # HIP runtime instance (its libamdhip64 carries the soname the library links against)
        try:
            import torch  # noqa: F401
        except ImportError:
            pass
        L = ctypes.CDLL(LIB_PATH)
        vp, i64, i32, f64, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_double, ctypes.c_size_t
        L.mfsdp_muon_workspace_size.argtypes = [ctypes.POINTER(MuonEntry), i64, ctypes.POINTER(MuonHParams)]
        L.mfsdp_muon_workspace_size.restype = sz
        L.mfsdp_muon_step.argtypes = [ctypes.POINTER(MuonEntry), i64, ctypes.POINTER(MuonHParams), vp, sz, vp]
        L.mfsdp_muon_step.restype = ctypes.c_int
        L.mfsdp_muon_step_timed.argtypes = [ctypes.POINTER(MuonEntry), i64, ctypes.POINTER(MuonHParams),
                                            vp, sz, vp, ctypes.POINTER(ctypes.c_void_p)]
        L.mfsdp_muon_step_timed.restype = ctypes.c_int
        L.mfsdp_muon_step_noalloc.argtypes = [ctypes.POINTER(MuonEntry), i64, ctypes.POINTER(MuonHParams), vp]
        L.mfsdp_muon_step_noalloc.restype = ctypes.c_int
        L.mfsdp_muon_step_reduce.argtypes = [ctypes.POINTER(MuonEntry), i64, ctypes.POINTER(ctypes.c_void_p),
                                             i32, f64, ctypes.POINTER(ctypes.c_void_p),
                                             ctypes.POINTER(MuonHParams), vp, sz, vp]
        L.mfsdp_muon_step_reduce.restype = ctypes.c_int
        L.mfsdp_ns_workspace_size.argtypes = [i64, i64, i32]
        L.mfsdp_ns_workspace_size.restype = sz
        L.mfsdp_newton_schulz.argtypes = [vp, i32, vp, i32, i64, i64, f64, f64, f64, i32, f64, i32, vp, sz, vp]
        L.mfsdp_newton_schulz_schedule.restype = ctypes.c_int
        L.mfsdp_newton_schulz_schedule.argtypes = [vp, i32, vp, i32, i64, i64, ctypes.POINTER(f64), i32, f64,
                                                   i32, vp, sz, vp]
        L.mfsdp_newton_schulz.restype = ctypes.c_int
        L.mfsdp_adamw_step.argtypes = [ctypes.POINTER(AdamWEntry), i64, f64, f64, f64, f64, f64, i64, vp]
        L.mfsdp_adamw_step.restype = ctypes.c_int
        L.mfsdp_last_error.argtypes = []
        L.mfsdp_last_error.restype = ctypes.c_char_p
        L.mfsdp_status_string.argtypes = [ctypes.c_int]
        L.mfsdp_status_string.restype = ctypes.c_char_p
        L.mfsdp_abi_version.argtypes = []
        L.mfsdp_abi_version.restype = ctypes.c_int
        L.mfsdp_plan_owners.argtypes = [ctypes.POINTER(PlanParam), i64, i32, i32, f64, ctypes.POINTER(i32),
                                        ctypes.POINTER(i64), ctypes.POINTER(f64), ctypes.POINTER(i32)]
        L.mfsdp_plan_owners.restype = ctypes.c_int
        L.mfsdp_plan_layouts.argtypes = [ctypes.POINTER(PlanParam), i64, i32, ctypes.POINTER(i32),
                                         ctypes.POINTER(i64), ctypes.POINTER(i64), ctypes.POINTER(i64)]
        L.mfsdp_plan_layouts.restype = ctypes.c_int
        L.mfsdp_shampoo_workspace_size.argtypes = [ctypes.POINTER(ShampooEntry), i64, ctypes.POINTER(ShampooHParams)]
        L.mfsdp_shampoo_workspace_size.restype = sz
        L.mfsdp_shampoo_step.argtypes = [ctypes.POINTER(ShampooEntry), i64, ctypes.POINTER(ShampooHParams), vp,
                                         sz, vp]
        L.mfsdp_shampoo_step.restype = ctypes.c_int
        L.mfsdp_inverse_root_workspace_size.argtypes = [i64, i32, i32]
        L.mfsdp_inverse_root_workspace_size.restype = sz
        L.mfsdp_inverse_root.argtypes = [vp, vp, i64, i32, f64, f64, i32, vp, sz, vp]
        L.mfsdp_inverse_root.restype = ctypes.c_int
        L.mfsdp_soap_workspace_size.argtypes = [ctypes.POINTER(SoapEntry), i64, ctypes.POINTER(SoapHParams)]
        L.mfsdp_soap_workspace_size.restype = sz
        L.mfsdp_soap_step.argtypes = [ctypes.POINTER(SoapEntry), i64, ctypes.POINTER(SoapHParams), vp, sz, vp]
        L.mfsdp_soap_step.restype = ctypes.c_int
        L.mfsdp_orthonormal_factor_workspace_size.argtypes = [i64]
        L.mfsdp_orthonormal_factor_workspace_size.restype = sz
        L.mfsdp_orthonormal_factor.argtypes = [vp, vp, i64, vp, sz, vp]
        L.mfsdp_orthonormal_factor.restype = ctypes.c_int
        L.mfsdp_build_id.argtypes = []
        L.mfsdp_build_id.restype = ctypes.c_char_p
        from . import build_lib
        built, tree = L.mfsdp_build_id().decode(), build_lib.source_id()
        if built != tree:
            raise ImportError(f"{LIB_PATH} was built from other sources (build id {built}, sources {tree}); "
                              "rebuild it with `python -m paper_2607_05895_amd.build_lib`")
        _lib = L
    return _lib


def _check(status: int) -> None:
    if status != OK:
        raise MfsdpError(status, lib().mfsdp_last_error().decode())


def _entries(arr, cls):
    arr = list(arr)
    return (cls * max(1, len(arr)))(*arr), len(arr)


# ------------------------------------------------------------------- C names, raw arguments

def mfsdp_abi_version() -> int:
    return lib().mfsdp_abi_version()


def mfsdp_build_id() -> str:
    return lib().mfsdp_build_id().decode()


def mfsdp_last_error() -> str:
    return lib().mfsdp_last_error().decode()


def mfsdp_status_string(status: int) -> str:
    return lib().mfsdp_status_string(status).decode()


def mfsdp_plan_owners(params, world: int, policy: int, gamma_cap: float = 0.0):
    """params: (block, numel, is_matrix) per parameter. Returns (owner list, rank loads, per-block
    gamma_B list indexed by block, policy used). Host only: no GPU is touched."""
    params = list(params)
    arr = (PlanParam * max(1, len(params)))(*[PlanParam(int(b), int(bool(mx)), int(n)) for b, n, mx in params])
    nblocks = 1 + max((int(b) for b, _, _ in params), default=-1)
    owner = (ctypes.c_int32 * max(1, len(params)))()
    loads = (ctypes.c_int64 * max(1, world))()
    gam = (ctypes.c_double * max(1, nblocks))()
    used = ctypes.c_int32(-1)
    _check(lib().mfsdp_plan_owners(arr, len(params), world, policy, gamma_cap, owner, loads, gam,
                                   ctypes.byref(used)))
    return list(owner[:len(params)]), list(loads[:world]), list(gam[:nblocks]), used.value


def mfsdp_plan_layouts(params, world: int, owner):
    """params: (block, numel, is_matrix) per parameter; owner: one rank per parameter. Returns
    (global offsets, local offsets, per-block lists of the ranks' local buffer lengths). Host only."""
    params = list(params)
    n = len(params)
    arr = (PlanParam * max(1, n))(*[PlanParam(int(b), int(bool(mx)), int(k)) for b, k, mx in params])
    own = (ctypes.c_int32 * max(1, n))(*[int(o) for o in owner])
    nblocks = 1 + max((int(b) for b, _, _ in params), default=-1)
    g = (ctypes.c_int64 * max(1, n))()
    loc = (ctypes.c_int64 * max(1, n))()
    lens = (ctypes.c_int64 * max(1, nblocks * world))()
    _check(lib().mfsdp_plan_layouts(arr, n, world, own, g, loc, lens))
    return list(g[:n]), list(loc[:n]), [list(lens[b * world:(b + 1) * world]) for b in range(nblocks)]


def mfsdp_shampoo_workspace_size(entries: Sequence[ShampooEntry], hp: ShampooHParams) -> int:
    arr, n = _entries(entries, ShampooEntry)
    return lib().mfsdp_shampoo_workspace_size(arr, n, ctypes.byref(hp))


def mfsdp_shampoo_step(entries: Sequence[ShampooEntry], hp: ShampooHParams, workspace: int,
                       workspace_bytes: int, stream: int) -> None:
    arr, n = _entries(entries, ShampooEntry)
    _check(lib().mfsdp_shampoo_step(arr, n, ctypes.byref(hp), workspace, workspace_bytes, stream))


def mfsdp_soap_workspace_size(entries: Sequence[SoapEntry], hp: SoapHParams) -> int:
    arr, n = _entries(entries, SoapEntry)
    return lib().mfsdp_soap_workspace_size(arr, n, ctypes.byref(hp))


def mfsdp_soap_step(entries: Sequence[SoapEntry], hp: SoapHParams, workspace: int, workspace_bytes: int,
                    stream: int = 0) -> None:
    arr, n = _entries(entries, SoapEntry)
    _check(lib().mfsdp_soap_step(arr, n, ctypes.byref(hp), workspace, workspace_bytes, stream))


def mfsdp_orthonormal_factor_workspace_size(d: int) -> int:
    return lib().mfsdp_orthonormal_factor_workspace_size(d)


def mfsdp_orthonormal_factor(a: int, q: int, d: int, workspace: int, workspace_bytes: int,
                             stream: int = 0) -> None:
    _check(lib().mfsdp_orthonormal_factor(a, q, d, workspace, workspace_bytes, stream))


def mfsdp_inverse_root_workspace_size(d: int, p: int, iters: int) -> int:
    return lib().mfsdp_inverse_root_workspace_size(d, p, iters)


def mfsdp_inverse_root(a: int, out: int, d: int, p: int, eps: float, eps_rel: float, iters: int,
                       workspace: int, workspace_bytes: int, stream: int) -> None:
    _check(lib().mfsdp_inverse_root(a, out, d, p, eps, eps_rel, iters, workspace, workspace_bytes, stream))


def mfsdp_muon_workspace_size(entries: Sequence[MuonEntry], hp: MuonHParams) -> int:
    arr, n = _entries(entries, MuonEntry)
    size = lib().mfsdp_muon_workspace_size(arr, n, ctypes.byref(hp))
    if size == 0 and n > 0:
        raise MfsdpError(E_INVALID, mfsdp_last_error())
    return size


def mfsdp_muon_step(entries: Sequence[MuonEntry], hp: MuonHParams, workspace: int,
                    workspace_bytes: int, stream: int = 0) -> None:
    arr, n = _entries(entries, MuonEntry)
    _check(lib().mfsdp_muon_step(arr, n, ctypes.byref(hp), workspace, workspace_bytes, stream))


def mfsdp_muon_step_noalloc(entries: Sequence[MuonEntry], hp: MuonHParams, stream: int = 0) -> None:
    arr, n = _entries(entries, MuonEntry)
    _check(lib().mfsdp_muon_step_noalloc(arr, n, ctypes.byref(hp), stream))


def mfsdp_muon_step_timed(entries: Sequence[MuonEntry], hp: MuonHParams, workspace: int,
                          workspace_bytes: int, stream: int, events: Sequence[int]) -> None:
    arr, n = _entries(entries, MuonEntry)
    ev = (ctypes.c_void_p * 4)(*list(events))
    _check(lib().mfsdp_muon_step_timed(arr, n, ctypes.byref(hp), workspace, workspace_bytes,
                                       stream, ev))


def mfsdp_muon_step_reduce(entries: Sequence[MuonEntry], grad_parts: Sequence[Sequence[int]],
                           grad_scale: float, reduced_out: Optional[Sequence[Optional[int]]],
                           hp: MuonHParams, workspace: int, workspace_bytes: int, stream: int = 0) -> None:
    """grad_parts[i]: the nparts device pointers of entry i (same count for every entry)."""
    arr, n = _entries(entries, MuonEntry)
    nparts = len(grad_parts[0]) if grad_parts else 0
    flat = [p for parts in grad_parts for p in parts]
    pa = (ctypes.c_void_p * max(1, len(flat)))(*flat)
    ro = (ctypes.c_void_p * max(1, n))(*list(reduced_out)) if reduced_out is not None else None
    _check(lib().mfsdp_muon_step_reduce(arr, n, pa, nparts, grad_scale, ro, ctypes.byref(hp),
                                        workspace, workspace_bytes, stream))


def mfsdp_ns_workspace_size(m: int, n: int, ns_dtype: int) -> int:
    size = lib().mfsdp_ns_workspace_size(m, n, ns_dtype)
    if size == 0:
        raise MfsdpError(E_INVALID, mfsdp_last_error())
    return size


def mfsdp_newton_schulz(x: int, x_dtype: int, out: int, out_dtype: int, m: int, n: int, a: float,
                        b: float, c: float, steps: int, eps: float, ns_dtype: int, workspace: int,
                        workspace_bytes: int, stream: int = 0) -> None:
    _check(lib().mfsdp_newton_schulz(x, x_dtype, out, out_dtype, m, n, a, b, c, steps, eps,
                                     ns_dtype, workspace, workspace_bytes, stream))


def _coeff_array(triples):
    flat = [float(v) for t in triples for v in t]
    return (ctypes.c_double * max(len(flat), 1))(*flat)


def mfsdp_newton_schulz_schedule(x: int, x_dtype: int, out: int, out_dtype: int, m: int, n: int,
                                 schedule, eps: float, ns_dtype: int, workspace: int,
                                 workspace_bytes: int, stream: int = 0) -> None:
    """schedule: a sequence of (a_k, b_k, c_k), one per NS step."""
    arr = _coeff_array(schedule)
    _check(lib().mfsdp_newton_schulz_schedule(x, x_dtype, out, out_dtype, m, n, arr, len(schedule),
                                              eps, ns_dtype, workspace, workspace_bytes, stream))


def mfsdp_adamw_step(entries: Sequence[AdamWEntry], lr: float, beta1: float, beta2: float,
                     eps: float, weight_decay: float, step: int, stream: int = 0) -> None:
    arr, n = _entries(entries, AdamWEntry)
    _check(lib().mfsdp_adamw_step(arr, n, lr, beta1, beta2, eps, weight_decay, step, stream))


# ------------------------------------------------------------------- torch tensor helpers

def _dt(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _stream() -> int:
    import torch
    return torch.cuda.current_stream().cuda_stream


_FLOAT = ("bfloat16", "float32")


def _ptr(t, what: str, shape=None, dtypes=_FLOAT) -> int:
    """Data pointer of a tensor handed to the library, after checking what the C ABI cannot: that it
    is a dense, contiguous tensor on the current GPU (the calls run on that GPU's current stream)
    with the shape and dtype the call reads and writes. The library trusts pointers and sizes, so a
    tensor that is smaller than the call assumes would be written past its end."""
    import torch
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{what}: expected a torch.Tensor, got {type(t).__name__}")
    if not t.is_cuda or t.layout != torch.strided:
        raise ValueError(f"{what}: must be a dense CUDA tensor, got {t.layout} on {t.device}")
    if t.device.index != torch.cuda.current_device():
        raise ValueError(f"{what}: is on {t.device} but the current device is cuda:{torch.cuda.current_device()}")
    if not t.is_contiguous():
        raise ValueError(f"{what}: must be contiguous")
    if str(t.dtype).replace("torch.", "") not in dtypes:
        raise TypeError(f"{what}: dtype must be one of {dtypes}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{what}: shape {tuple(t.shape)} where {tuple(shape)} is required")
    return t.data_ptr()


def _ws(workspace) -> Tuple[int, int]:
    return _ptr(workspace, "workspace", dtypes=("uint8",)), workspace.numel()


def muon_hparams(lr=0.02, weight_decay=0.0, momentum=0.95, nesterov=True, a=3.4445, b=-4.7750,
                 c=2.0315, ns_steps=5, eps=1e-7, lr_adjust="original", ns_dtype="bf16",
                 ns_schedule=None) -> MuonHParams:
    """ns_schedule: None, or one (a_k, b_k, c_k) per NS step (the array is kept on the struct)."""
    hp = MuonHParams(lr, weight_decay, momentum, int(bool(nesterov)), a, b, c, ns_steps, eps,
                     _LR_MODES[lr_adjust] if isinstance(lr_adjust, str) else int(lr_adjust),
                     _NS_DT[ns_dtype] if isinstance(ns_dtype, str) else int(ns_dtype), None)
    if ns_schedule is not None:
        hp._schedule = _coeff_array(ns_schedule)  # keeps the memory alive as long as hp
        hp.ns_schedule = hp._schedule
    return hp


def muon_entry_t(param, grad, momentum, update_out=None) -> MuonEntry:
    if param.dim() != 2:
        raise ValueError(f"param: a Muon entry is a 2D matrix, got shape {tuple(param.shape)}")
    m, n = param.shape
    return MuonEntry(_ptr(param, "param"), _ptr(grad, "grad", (m, n)),
                     _ptr(momentum, "momentum", (m, n), ("float32",)), m, n, _dt(param), _dt(grad),
                     _ptr(update_out, "update_out", (m, n), ("float32",)) if update_out is not None else None)


def muon_workspace_t(entries: Sequence[MuonEntry], hp: MuonHParams, device="cuda"):
    import torch
    size = mfsdp_muon_workspace_size(entries, hp)
    return torch.empty(max(size, 256), dtype=torch.uint8, device=device)


def muon_step_t(entries: Sequence[MuonEntry], hp: MuonHParams, workspace) -> None:
    mfsdp_muon_step(entries, hp, *_ws(workspace), _stream())


def muon_step_noalloc_t(entries: Sequence[MuonEntry], hp: MuonHParams) -> None:
    """The allocation-free step on the current device's torch stream (no workspace tensor)."""
    mfsdp_muon_step_noalloc(entries, hp, _stream())


def muon_step_reduce_t(entries: Sequence[MuonEntry], parts, grad_scale: float, hp: MuonHParams,
                       workspace, reduced_out=None) -> None:
    """parts[i]: list of gradient-part tensors of entry i; reduced_out: None or a list of tensors
    (or None) receiving the reduced gradients."""
    if len(parts) != len(entries) or (reduced_out is not None and len(reduced_out) != len(entries)):
        raise ValueError("parts (and reduced_out) need one item per entry")
    dts = {BF16: ("bfloat16",), F32: ("float32",)}
    ptrs = [[_ptr(t, f"parts[{i}]", (e.m, e.n), dts.get(e.grad_dtype, ())) for t in ps]
            for i, (e, ps) in enumerate(zip(entries, parts))]
    outs = ([_ptr(t, f"reduced_out[{i}]", (e.m, e.n), dts.get(e.grad_dtype, ())) if t is not None else None
             for i, (e, t) in enumerate(zip(entries, reduced_out))] if reduced_out is not None else None)
    mfsdp_muon_step_reduce(entries, ptrs, grad_scale, outs, hp, *_ws(workspace), _stream())


def newton_schulz_t(x, out, a=3.4445, b=-4.7750, c=2.0315, steps=5, eps=1e-7, ns_dtype="bf16",
                    workspace=None) -> None:
    import torch
    m, n = x.shape
    nsd = BF16 if ns_dtype in ("bf16", BF16) else F32
    if workspace is None:
        workspace = torch.empty(mfsdp_ns_workspace_size(m, n, nsd), dtype=torch.uint8, device=x.device)
    mfsdp_newton_schulz(_ptr(x, "x"), _dt(x), _ptr(out, "out", (m, n)), _dt(out), m, n, a, b, c, steps, eps,
                        nsd, *_ws(workspace), _stream())


def newton_schulz_schedule_t(x, out, schedule, eps=1e-7, ns_dtype="bf16", workspace=None) -> None:
    import torch
    m, n = x.shape
    nsd = BF16 if ns_dtype in ("bf16", BF16) else F32
    if workspace is None:
        workspace = torch.empty(mfsdp_ns_workspace_size(m, n, nsd), dtype=torch.uint8, device=x.device)
    mfsdp_newton_schulz_schedule(_ptr(x, "x"), _dt(x), _ptr(out, "out", (m, n)), _dt(out), m, n, schedule,
                                 eps, nsd, *_ws(workspace), _stream())


def adamw_entry_t(param, grad, exp_avg, exp_avg_sq) -> AdamWEntry:
    sh = tuple(param.shape)
    return AdamWEntry(_ptr(param, "param"), _ptr(grad, "grad", sh),
                      _ptr(exp_avg, "exp_avg", sh, ("float32",)), _ptr(exp_avg_sq, "exp_avg_sq", sh, ("float32",)),
                      param.numel(), _dt(param), _dt(grad))


def adamw_step_t(entries: Sequence[AdamWEntry], lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8,
                 weight_decay=1e-2, step=1) -> None:
    mfsdp_adamw_step(entries, lr, beta1, beta2, eps, weight_decay, step, _stream())


def shampoo_hparams(lr=1e-3, weight_decay=0.0, beta=1.0, weight=1.0, eps=1e-12, eps_rel=1e-6,
                    refresh=True, root_iters=20) -> ShampooHParams:
    return ShampooHParams(lr, weight_decay, beta, weight, eps, eps_rel, int(bool(refresh)), root_iters)


def shampoo_entry_t(param, grad, L, R, PL, PR, update_out=None) -> ShampooEntry:
    if param.dim() != 2:
        raise ValueError(f"param: a Shampoo entry is a 2D matrix, got shape {tuple(param.shape)}")
    m, n = param.shape
    f = ("float32",)
    return ShampooEntry(_ptr(param, "param"), _ptr(grad, "grad", (m, n)), _ptr(L, "L", (m, m), f),
                        _ptr(R, "R", (n, n), f), _ptr(PL, "PL", (m, m), f), _ptr(PR, "PR", (n, n), f),
                        m, n, _dt(param), _dt(grad),
                        _ptr(update_out, "update_out", (m, n), f) if update_out is not None else None)


def shampoo_workspace_t(entries: Sequence[ShampooEntry], hp: ShampooHParams, device="cuda"):
    import torch
    size = mfsdp_shampoo_workspace_size(entries, hp)
    return torch.empty(max(size, 256), dtype=torch.uint8, device=device)


def shampoo_step_t(entries: Sequence[ShampooEntry], hp: ShampooHParams, workspace) -> None:
    mfsdp_shampoo_step(entries, hp, *_ws(workspace), _stream())


def inverse_root_t(a, out, p=4, eps=1e-12, eps_rel=1e-6, iters=20, workspace=None) -> None:
    import torch
    d = a.shape[0]
    if workspace is None:
        workspace = torch.empty(mfsdp_inverse_root_workspace_size(d, p, iters), dtype=torch.uint8,
                                device=a.device)
    f = ("float32",)
    mfsdp_inverse_root(_ptr(a, "a", (d, d), f), _ptr(out, "out", (d, d), f), d, p, eps, eps_rel, iters,
                       *_ws(workspace), _stream())


def soap_hparams(lr=3e-3, weight_decay=0.0, beta1=0.95, beta2=0.95, eps=1e-8, shampoo_beta=0.95,
                 shampoo_weight=0.05, step=1, refresh=False, refresh_iters=1, max_precond_dim=0) -> SoapHParams:
    """max_precond_dim: sides longer than it have no basis (0: 4096)."""
    return SoapHParams(lr, weight_decay, beta1, beta2, eps, shampoo_beta, shampoo_weight, int(step),
                       int(bool(refresh)), int(refresh_iters), int(max_precond_dim))


def soap_entry_t(param, grad, exp_avg, exp_avg_sq, L, R, QL, QR, update_out=None) -> SoapEntry:
    """L and QL (or R and QR) may be None for a side longer than the call's max_precond_dim."""
    if param.dim() != 2:
        raise ValueError(f"param: a SOAP entry is a 2D matrix, got shape {tuple(param.shape)}")
    m, n = param.shape
    f = ("float32",)
    opt = lambda t, what, shape: _ptr(t, what, shape, f) if t is not None else None  # noqa: E731
    return SoapEntry(_ptr(param, "param"), _ptr(grad, "grad", (m, n)), _ptr(exp_avg, "exp_avg", (m, n), f),
                     _ptr(exp_avg_sq, "exp_avg_sq", (m, n), f), opt(L, "L", (m, m)), opt(R, "R", (n, n)),
                     opt(QL, "QL", (m, m)), opt(QR, "QR", (n, n)), m, n, _dt(param), _dt(grad),
                     _ptr(update_out, "update_out", (m, n), f) if update_out is not None else None)


def soap_workspace_t(entries: Sequence[SoapEntry], hp: SoapHParams, device="cuda"):
    import torch
    size = mfsdp_soap_workspace_size(entries, hp)
    return torch.empty(max(size, 256), dtype=torch.uint8, device=device)


def soap_step_t(entries: Sequence[SoapEntry], hp: SoapHParams, workspace) -> None:
    mfsdp_soap_step(entries, hp, *_ws(workspace), _stream())


def orthonormal_factor_t(a, q, workspace=None) -> None:
    import torch
    d = a.shape[0]
    if workspace is None:
        workspace = torch.empty(max(mfsdp_orthonormal_factor_workspace_size(d), 256), dtype=torch.uint8,
                                device=a.device)
    f = ("float32",)
    mfsdp_orthonormal_factor(_ptr(a, "a", (d, d), f), _ptr(q, "q", (d, d), f), d, *_ws(workspace), _stream())
