"""Pins of the fp64 expert-MLP backward oracle (CPU): central finite differences of the
scalar <dY, Y>, torch.autograd in float64 (an independent differentiation of the same
forward), the closed form of silu' and the grouped segment bookkeeping."""
import numpy as np
import pytest
import torch

import oracle
from oracle import moe_backward as bwd
from paper_2607_18631_amd import workloads as wl


def _expert(rng, m, d, F, scale=0.5):
    x = rng.standard_normal((m, d))
    w13 = rng.standard_normal((2 * F, d)) * scale
    w2 = rng.standard_normal((d, F)) * scale
    dy = rng.standard_normal((m, d))
    return x, w13, w2, dy


def test_silu_grad_closed_forms():
    assert bwd.silu_grad(np.array(0.0)) == 0.5                  # s(0) = 1/2, h = 0
    # large |h|: silu'(h) -> 1 for h -> +inf, -> 0 for h -> -inf
    assert abs(bwd.silu_grad(np.array(40.0)) - 1.0) < 1e-12
    assert abs(bwd.silu_grad(np.array(-40.0))) < 1e-12
    # against a central difference of silu itself
    h = np.linspace(-6, 6, 25)
    silu = lambda v: v / (1 + np.exp(-v))
    eps = 1e-6
    np.testing.assert_allclose(bwd.silu_grad(h), (silu(h + eps) - silu(h - eps)) / (2 * eps), rtol=0, atol=1e-8)


def test_backward_matches_finite_differences():
    """Every entry of dX, dW13, dW2 against a central difference of L = <dY, Y>."""
    rng = np.random.default_rng(0)
    x, w13, w2, dy = _expert(rng, 3, 4, 2)
    loss = lambda x_, w13_, w2_: float(np.sum(dy * oracle.swiglu_ffn(x_, w13_, w2_)))
    gx, g13, g2 = bwd.swiglu_ffn_backward(x, w13, w2, dy)
    eps = 1e-6
    for arr, grad, which in ((x, gx, 0), (w13, g13, 1), (w2, g2, 2)):
        num = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            args_p = [x.copy(), w13.copy(), w2.copy()]
            args_m = [x.copy(), w13.copy(), w2.copy()]
            args_p[which][idx] += eps
            args_m[which][idx] -= eps
            num[idx] = (loss(*args_p) - loss(*args_m)) / (2 * eps)
        np.testing.assert_allclose(grad, num, rtol=1e-6, atol=1e-7, err_msg=f"operand {which}")


def test_backward_matches_torch_autograd():
    rng = np.random.default_rng(1)
    x, w13, w2, dy = _expert(rng, 7, 12, 5)
    tx = torch.tensor(x, dtype=torch.float64, requires_grad=True)
    t13 = torch.tensor(w13, dtype=torch.float64, requires_grad=True)
    t2 = torch.tensor(w2, dtype=torch.float64, requires_grad=True)
    F = 5
    y = (torch.nn.functional.silu(tx @ t13[:F].T) * (tx @ t13[F:].T)) @ t2.T
    y.backward(torch.tensor(dy, dtype=torch.float64))
    gx, g13, g2 = bwd.swiglu_ffn_backward(x, w13, w2, dy)
    np.testing.assert_allclose(gx, tx.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(g13, t13.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(g2, t2.grad.numpy(), rtol=1e-12, atol=1e-12)


def test_swapped_gate_and_up_halves_are_caught():
    """The gate (W1) and up (W3) halves play different roles: swapping them changes dX."""
    rng = np.random.default_rng(2)
    x, w13, w2, dy = _expert(rng, 4, 6, 3)
    gx, _, _ = bwd.swiglu_ffn_backward(x, w13, w2, dy)
    swapped = np.concatenate([w13[3:], w13[:3]])
    gx2, _, _ = bwd.swiglu_ffn_backward(x, swapped, w2, dy)
    assert np.abs(gx - gx2).max() > 1e-3


@pytest.mark.parametrize("capacity", [0, 3])
def test_grouped_backward_segments(capacity):
    """Per-expert segments: an empty expert gets zero weight gradients, rows outside every
    segment get zero dX, and each segment equals the single-expert backward."""
    rng = np.random.default_rng(3)
    E, d, F = 4, 8, 4
    w13 = wl.f32_to_bf16_bits((rng.standard_normal((E, 2 * F, d)) * 0.4).astype(np.float32))
    w2 = wl.f32_to_bf16_bits((rng.standard_normal((E, d, F)) * 0.4).astype(np.float32))
    if capacity:
        counts = np.array([2, 0, 5, 1])                     # expert 2 keeps 3 of its 5
        offsets = counts
        cap = E * capacity
        segs = [(0, 2), (3, 3), (6, 9), (9, 10)]
    else:
        offsets = np.array([0, 2, 2, 7, 8])
        cap = 9
        segs = [(0, 2), (2, 2), (2, 7), (7, 8)]
    assert bwd.expert_segments(offsets, E, capacity) == segs
    x = rng.standard_normal((cap, d))
    dy = rng.standard_normal((cap, d))
    dx, dw13, dw2 = bwd.grouped_ffn_backward(x, offsets, w13, w2, dy, E, capacity)
    covered = np.zeros(cap, bool)
    for e, (a, b) in enumerate(segs):
        covered[a:b] = True
        if a == b:
            assert not dw13[e].any() and not dw2[e].any()
            continue
        gx, g13, g2 = bwd.swiglu_ffn_backward(x[a:b], oracle.bf16_to_f64(w13[e]), oracle.bf16_to_f64(w2[e]), dy[a:b])
        np.testing.assert_array_equal(dx[a:b], gx)
        np.testing.assert_array_equal(dw13[e], g13)
        np.testing.assert_array_equal(dw2[e], g2)
    assert not dx[~covered].any()


# ---------------------------------------------------------------------------------------
# the whole layer: an independent float64 torch implementation of the forward, differentiated
# by torch.autograd with the oracle's expert choice held fixed
# ---------------------------------------------------------------------------------------
def _torch_layer_grads(inputs, dout):
    sh = inputs["shape"]
    t = lambda a: torch.tensor(oracle.bf16_to_f64(a), dtype=torch.float64, requires_grad=True)
    x, wr, w13, w2 = t(inputs["x"]), t(inputs["w_router"]), t(inputs["w13"]), t(inputs["w2"])
    ws13 = t(inputs["ws13"]) if sh.F_shared else None
    ws2 = t(inputs["ws2"]) if sh.F_shared else None
    res = oracle.layer_forward(inputs)                        # expert choice (held fixed)
    idx = torch.tensor(res["topk_idx"].astype(np.int64))
    logits = x @ wr.T
    if sh.gate == wl.GATE_SOFTMAX:
        keys = logits + (torch.tensor(inputs["bias"], dtype=torch.float64) if inputs.get("bias") is not None else 0)
        sel = keys.gather(1, idx)
        if sh.renormalize:
            gates = torch.softmax(sel, dim=1)
        else:
            gates = torch.softmax(keys, dim=1).gather(1, idx)
    else:
        keys = torch.sigmoid(logits)
        sel = keys.gather(1, idx)
        gates = sel / sel.sum(dim=1, keepdim=True) if sh.renormalize else sel
    gates = gates * sh.routed_scale
    keep = torch.tensor(oracle.keep_mask(res["topk_idx"], sh.e_begin, sh.E_local, sh.expert_capacity))
    F = sh.F
    out = torch.zeros_like(x)
    for tok in range(sh.T):
        for j in range(sh.top_k):
            e = int(idx[tok, j]) - sh.e_begin
            if not keep[tok, j]:
                continue
            h = w13[e, :F] @ x[tok]
            u = w13[e, F:] @ x[tok]
            out[tok] = out[tok] + gates[tok, j] * (w2[e] @ (torch.nn.functional.silu(h) * u))
    if sh.F_shared:
        Fs = sh.F_shared
        out = out + (torch.nn.functional.silu(x @ ws13[:Fs].T) * (x @ ws13[Fs:].T)) @ ws2.T
    out.backward(torch.tensor(dout, dtype=torch.float64))
    g = {"dx": x.grad, "dw_router": wr.grad, "dw13": w13.grad, "dw2": w2.grad}
    if sh.F_shared:
        g["dws13"], g["dws2"] = ws13.grad, ws2.grad
    return {k: v.numpy() for k, v in g.items()}


LAYER_CASES = {
    "softmax_bias_renorm": (wl.MoEShape(T=9, d=12, E=6, top_k=2, F=5, E_local=6), 1.0),
    "softmax_full_scaled": (wl.MoEShape(T=8, d=10, E=5, top_k=3, F=4, E_local=5, renormalize=0, routed_scale=1.5),
                            0.0),
    "sigmoid_groups_shared_slice": (wl.MoEShape(T=10, d=16, E=8, top_k=3, F=6, E_local=4, e_begin=2, F_shared=4,
                                                gate=wl.GATE_SIGMOID, n_group=4, topk_group=2, routed_scale=2.5), 0.0),
    "sigmoid_raw": (wl.MoEShape(T=7, d=8, E=6, top_k=2, F=4, E_local=6, gate=wl.GATE_SIGMOID, renormalize=0), 0.0),
    "masked_capacity_drops": (wl.MoEShape(T=12, d=8, E=4, top_k=2, F=4, E_local=4, expert_capacity=3), 0.0),
}


@pytest.mark.parametrize("name", list(LAYER_CASES))
def test_layer_backward_matches_torch_autograd(name):
    sh, zipf = LAYER_CASES[name]
    inputs = wl.custom_inputs(sh, seed=31, router_std=1.0, zipf_s=zipf)
    if name == "softmax_bias_renorm":
        inputs["bias"] = np.linspace(-0.5, 0.7, sh.E).astype(np.float32)
    dout = np.random.default_rng(5).standard_normal((sh.T, sh.d))
    got = bwd.layer_backward(inputs, dout)
    ref = _torch_layer_grads(inputs, dout)
    for key, val in ref.items():
        np.testing.assert_allclose(got[key], val, rtol=1e-10, atol=1e-11, err_msg=key)


def test_layer_backward_finite_differences():
    """dx and dW_router against central differences of <dout, out> (the expert choice is
    checked to be unchanged by every perturbation)."""
    sh = wl.MoEShape(T=4, d=6, E=4, top_k=2, F=3, E_local=4, F_shared=2, gate=wl.GATE_SIGMOID)
    inputs = wl.custom_inputs(sh, seed=7, router_std=1.0)
    dout = np.random.default_rng(8).standard_normal((sh.T, sh.d))
    got = bwd.layer_backward(inputs, dout)
    base_idx = oracle.layer_forward(inputs)["topk_idx"]
    xd = oracle.bf16_to_f64(inputs["x"])
    wr = oracle.bf16_to_f64(inputs["w_router"])

    def loss(xv, wrv):
        idx, w, _ = oracle.route(xv, wrv, sh)
        assert (idx == base_idx).all()
        out = oracle.expert_outputs_for_tokens(xv, idx, w, sh, inputs["w13"], inputs["w2"], inputs["ws13"],
                                               inputs["ws2"])
        return float((dout * out).sum())

    eps = 1e-6
    for name, arr, grad in (("dx", xd, got["dx"]), ("dw_router", wr, got["dw_router"])):
        num = np.zeros_like(arr)
        for ix in np.ndindex(arr.shape):
            a, b = arr.copy(), arr.copy()
            a[ix] += eps
            b[ix] -= eps
            num[ix] = (loss(a, wr) - loss(b, wr)) / (2 * eps) if name == "dx" else \
                (loss(xd, a) - loss(xd, b)) / (2 * eps)
        np.testing.assert_allclose(grad, num, rtol=1e-6, atol=1e-7, err_msg=name)
