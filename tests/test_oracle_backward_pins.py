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
