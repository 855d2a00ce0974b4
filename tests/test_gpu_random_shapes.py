"""Seeded sweep of random layer shapes on the GPU against the fp64 oracle, forward and backward.

Each case draws (from a fixed seed, so the set is the same on every run) the token count, hidden
size, expert count, top-k, gating mode (softmax with or without a Zipf router bias, sigmoid with
or without a group limit, renormalised or not, scaled or not), the rank's expert slice, the expert
and shared-expert widths, the row layout (offsets or masked-decode capacity with drops) and the
kernel structure (gather / combine folded or not).  Checked per case: the routing protocol
(R1-R3), counts / offsets / permutation bit-exact against the oracle's of the GPU's decision, the
layer output within rel. Frobenius 5e-3, and -- where the backward applies (combine not folded,
E % 8 == 0) -- every gradient within 5e-3 of the oracle's layer backward.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import moe_backward as obwd
from paper_2607_18631_amd import moe
from paper_2607_18631_amd import workloads as wl

from parity_util import REL_TOL, check_routing, dev_bits, oracle_routing_with_gpu_ties, rel_fro, run_route

pytestmark = pytest.mark.gpu

N_CASES = 24
GRADS = ("dx", "dw_router", "dw13", "dw2", "dws13", "dws2")


def _draw(i):
    rng = np.random.default_rng(90210 + i)
    E = int(rng.choice([8, 16, 24, 32, 40, 64, 96, 128]))
    top_k = int(rng.integers(1, min(8, E) + 1))
    gate = int(rng.integers(0, 2))
    n_group, topk_group = 1, 1
    if gate == wl.GATE_SIGMOID and rng.random() < 0.5:
        divs = [g for g in range(2, 9) if E % g == 0 and E // g >= 2]
        n_group = int(rng.choice(divs))
        gsz = E // n_group
        lo = max(1, -(-top_k // gsz))
        topk_group = int(rng.integers(lo, n_group + 1))
    E_local = int(rng.integers(1, E + 1))
    e_begin = int(rng.integers(0, E - E_local + 1))
    d = 8 * int(rng.integers(8, 129))
    F = 8 * int(rng.integers(2, 97))
    F_shared = int(rng.choice([0, F, 8 * int(rng.integers(2, 65))]))
    T = int(rng.integers(1, 701))
    C = int(rng.integers(1, T + 1)) if rng.random() < 0.3 else 0
    fusion = int(rng.choice(list(wl.FUSION_VARIANTS.values()) + [0]))
    sh = wl.MoEShape(T=T, d=d, E=E, top_k=top_k, F=F, E_local=E_local, e_begin=e_begin, F_shared=F_shared,
                     gate=gate, n_group=n_group, topk_group=topk_group, renormalize=int(rng.integers(0, 2)),
                     routed_scale=float(rng.choice([1.0, 2.5])), expert_capacity=C, fusion=fusion)
    zipf = 1.2 if gate == wl.GATE_SOFTMAX and rng.random() < 0.4 else 0.0
    router_std = float(rng.choice([d ** -0.5, 2 * d ** -0.5]))
    return sh, router_std, zipf


@pytest.mark.parametrize("i", range(N_CASES))
def test_random_shape_forward_backward(i):
    sh, router_std, zipf = _draw(i)
    print(f"[random] case {i}: {sh} router_std={router_std:.3g} zipf={zipf}", flush=True)
    inputs = wl.custom_inputs(sh, seed=500 + i, router_std=router_std, zipf_s=zipf)
    layer = moe.DeviceLayer(inputs)
    out = layer.forward()
    torch.cuda.synchronize()
    g_idx, g_w, g_keys = run_route(layer)
    o_idx, o_w, keys64, near = check_routing(inputs, g_idx, g_w, g_keys)
    T, k, cap, C = sh.T, sh.top_k, sh.capacity, sh.expert_capacity
    reg = lambda r, dt, shp: layer.region(r, dt, shp).cpu().numpy()
    np.testing.assert_array_equal(reg(moe.MOE_REGION_TOPK_IDX, torch.int32, (T, k)), g_idx)
    counts, offsets = oracle.counts_offsets(g_idx, sh.e_begin, sh.E_local, C)
    row_token, slot_row = oracle.permutation(g_idx, sh.e_begin, sh.E_local, C)
    np.testing.assert_array_equal(reg(moe.MOE_REGION_COUNTS, torch.int32, (sh.E_local,)), counts)
    np.testing.assert_array_equal(reg(moe.MOE_REGION_OFFSETS, torch.int32, (sh.E_local + 1,)), offsets)
    np.testing.assert_array_equal(reg(moe.MOE_REGION_SLOT_ROW, torch.int32, (T, k)), slot_row)
    g_rt = reg(moe.MOE_REGION_ROW_TOKEN, torch.int32, (cap,))
    if C > 0:                                   # rows past an expert's valid prefix are not written
        live = row_token >= 0
        np.testing.assert_array_equal(g_rt[live], row_token[live])
    else:                                       # rows past offsets[E_local] are not written
        np.testing.assert_array_equal(g_rt[:row_token.size], row_token)
    idx, w = oracle_routing_with_gpu_ties(o_idx, o_w, keys64, g_idx, near, sh)
    ref = oracle.layer_forward(inputs, routing=(idx, w))
    err = rel_fro(oracle.bf16_to_f64(dev_bits(out)), ref["out"])
    print(f"[random] case {i}: forward rel_fro={err:.2e} near_ties={len(near)}", flush=True)
    assert err <= REL_TOL, err

    if (sh.fusion & wl.FUSE_COMBINE) or sh.E % 8:
        return
    dout = wl.f32_to_bf16_bits(np.random.default_rng(700 + i).standard_normal((T, sh.d)).astype(np.float32))
    grads = layer.backward(moe.to_device_bf16(dout))
    torch.cuda.synchronize()
    rb = obwd.layer_backward(inputs, oracle.bf16_to_f64(dout), routing=(idx, w))
    errs = {}
    for key in GRADS:
        if rb[key] is None:
            assert grads[key] is None, key
            continue
        errs[key] = rel_fro(oracle.bf16_to_f64(dev_bits(grads[key])), rb[key])
    print(f"[random] case {i}: backward " + ", ".join(f"{a}={b:.2e}" for a, b in errs.items()), flush=True)
    for key, v in errs.items():
        assert v <= REL_TOL, (key, v)
