"""moe_layer_forward_traced on the GPU: the traced layer's output equals the untraced one bit for
bit whether every step boundary, only some (NULL entries are not recorded) or none is asked for;
recorded intervals are ordered and add up to the whole step; with T == 0 every asked-for event is
still recorded."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2607_18631_amd import moe
from paper_2607_18631_amd import workloads as wl

pytestmark = pytest.mark.gpu

NSTEP = len(moe.MOE_STEP_NAMES)


class _Events:
    """hipEvent_t handles through the HIP runtime's C API."""

    def __init__(self):
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.made = []

    def create(self):
        h = ctypes.c_void_p()
        assert self.hip.hipEventCreate(ctypes.byref(h)) == 0
        self.made.append(h)
        return h

    def ms(self, a, b):
        v = ctypes.c_float()
        assert self.hip.hipEventElapsedTime(ctypes.byref(v), a, b) == 0
        return v.value

    def close(self):
        for h in self.made:
            self.hip.hipEventDestroy(h)


@pytest.fixture
def events():
    ev = _Events()
    yield ev
    ev.close()


def _layer():
    sh = wl.MoEShape(T=700, d=256, E=32, top_k=4, F=128, E_local=8, e_begin=8, F_shared=128,
                     gate=wl.GATE_SIGMOID, n_group=4, topk_group=2, routed_scale=2.5)
    return moe.DeviceLayer(wl.custom_inputs(sh, seed=5), device="cuda:0")


def test_traced_output_matches_untraced(events):
    layer = _layer()
    layer.forward()
    torch.cuda.synchronize()
    ref = moe.bf16_bits(layer.out)

    full = (ctypes.c_void_p * (NSTEP + 1))(*[events.create() for _ in range(NSTEP + 1)])
    layer.out.zero_()
    layer.forward_traced(full)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(moe.bf16_bits(layer.out), ref)
    steps = [events.ms(full[j], full[j + 1]) for j in range(NSTEP)]
    total = events.ms(full[0], full[NSTEP])
    assert all(s >= 0 for s in steps) and total > 0
    assert abs(sum(steps) - total) <= 1e-3 * max(1.0, total) + 1e-3, (steps, total)

    up = moe.MOE_STEP_NAMES.index("ffn_up")
    sparse = (ctypes.c_void_p * (NSTEP + 1))()
    for j in (0, up, up + 1, NSTEP):
        sparse[j] = events.create()
    layer.out.zero_()
    layer.forward_traced(sparse)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(moe.bf16_bits(layer.out), ref)
    t_all = events.ms(sparse[0], sparse[NSTEP])
    t_up = events.ms(sparse[up], sparse[up + 1])
    assert 0 < t_up <= t_all
    assert events.ms(sparse[0], sparse[up]) >= 0 and events.ms(sparse[up + 1], sparse[NSTEP]) >= 0


def test_traced_empty_batch_records_events(events):
    layer = _layer()
    sh0 = layer.shape.replace(T=0)
    ev = (ctypes.c_void_p * (NSTEP + 1))()
    ev[0], ev[NSTEP] = events.create(), events.create()
    moe.moe_layer_forward_traced(sh0, None, None, None, None, None, None, None, None, None, ev)
    torch.cuda.synchronize()
    assert events.ms(ev[0], ev[NSTEP]) >= 0
