"""mfsdp_muon_step_timed (the owner step with caller events at its phase boundaries, which the
benchmark's phase times come from) gives bitwise the results of mfsdp_muon_step, with the four events
and with events = NULL, and records its events in order."""
import ctypes
import sys

import numpy as np
import pytest

import synth
from tests.helpers import to_dev

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


class _Events:
    """hipEvent_t handles from the HIP runtime torch loaded."""

    def __init__(self):
        self.hip = ctypes.CDLL("libamdhip64.so.7")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self):
        ev = ctypes.c_void_p()
        assert self.hip.hipEventCreate(ctypes.byref(ev)) == 0
        return ev.value

    def elapsed(self, a, b):
        out = ctypes.c_float()
        assert self.hip.hipEventElapsedTime(ctypes.byref(out), a, b) == 0
        return out.value

    def destroy(self, ev):
        self.hip.hipEventDestroy(ev)


def _share(rng, shapes):
    host = [synth.random_muon_tensors(rng, m, n, synth.BF16, synth.BF16) for (m, n) in shapes]

    def device():
        import torch
        out = []
        for t, (m, n) in zip(host, shapes):
            out.append((to_dev(t.param, synth.BF16), to_dev(t.grad, synth.BF16), to_dev(t.momentum, synth.F32),
                        torch.empty((m, n), dtype=torch.float32, device="cuda")))
        return out
    return device


@pytest.mark.parametrize("ns_dtype", ["bf16", "f32"])
def test_timed_step_is_the_plain_step(ns_dtype):
    import torch
    from paper_2607_05895_amd import native
    _say(f"timed step {ns_dtype}")
    rng = np.random.default_rng(31)
    make = _share(rng, [(256, 512), (512, 256), (300, 300), (1, 50)])
    hp = native.muon_hparams(lr=0.02, weight_decay=0.01, ns_dtype=ns_dtype)
    runs = []
    ev = _Events()
    events = [ev.create() for _ in range(4)]
    stream = torch.cuda.current_stream().cuda_stream
    for mode in ("plain", "timed", "timed_null"):
        ts = make()
        ents = [native.muon_entry_t(p, g, m, u) for (p, g, m, u) in ts]
        ws = native.muon_workspace_t(ents, hp)
        if mode == "plain":
            native.muon_step_t(ents, hp, ws)
        elif mode == "timed":
            native.mfsdp_muon_step_timed(ents, hp, ws.data_ptr(), ws.numel(), stream, events)
        else:
            native.mfsdp_muon_step_timed(ents, hp, ws.data_ptr(), ws.numel(), stream, [None] * 4)
        torch.cuda.synchronize()
        runs.append(ts)
        if mode == "timed":
            e = [ev.elapsed(events[0], events[k]) for k in range(1, 4)]
            assert 0.0 <= e[0] <= e[1] <= e[2], e
    for ev_ in events:
        ev.destroy(ev_)
    for other in runs[1:]:
        for a, b in zip(runs[0], other):
            for x, y in zip(a, b):
                xv = x.view(torch.int16) if x.dtype == torch.bfloat16 else x
                yv = y.view(torch.int16) if y.dtype == torch.bfloat16 else y
                assert torch.equal(xv, yv)
