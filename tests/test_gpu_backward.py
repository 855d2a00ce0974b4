"""GPU parity of the expert-MLP backward (moe_grouped_ffn_backward, through the C ABI)
against the fp64 oracle: dX per expert segment, dW13 and dW2 per expert, rel. Frobenius
<= 5e-3 (bf16 operands and results, fp32 accumulation, dA / [dH dU] / activation rounded to
bf16 once each).  Experts without rows must get exactly zero weight gradients, and rows
outside every segment of dX must stay untouched.

Cases: ragged segment lengths around the 32/64/128/256-row tile edges with K tails in every
GEMM (d = 264, F = 136), decode-sized segments (the small-tile path), the masked-decode
layout with dropped slots, the DeepSeek-V3 expert shape (d = 7168, F = 2048) on four
experts, and a call with no tokens.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import moe_backward as obwd
from paper_2607_18631_amd import moe
from paper_2607_18631_amd import workloads as wl

from parity_util import REL_TOL, dev_bits, rel_fro

pytestmark = pytest.mark.gpu

S = wl.MoEShape


def _bits(rng, shape, std):
    return wl.f32_to_bf16_bits((rng.standard_normal(shape) * std).astype(np.float32))


def _run(sh, counts_or_offsets, seed):
    """Random x_perm / dy_perm / weights for the segments, the GPU backward, and the oracle."""
    rng = np.random.default_rng(seed)
    E, d, F, cap = sh.E_local, sh.d, sh.F, sh.capacity
    x = _bits(rng, (cap, d), 1.0)
    dy = _bits(rng, (cap, d), 1.0)
    w13 = _bits(rng, (E, 2 * F, d), d ** -0.5)
    w2 = _bits(rng, (E, d, F), F ** -0.5)
    dev = "cuda"
    offs = torch.from_numpy(np.asarray(counts_or_offsets, np.int32)).to(dev)
    dx = torch.full((cap, d), float("nan"), dtype=torch.bfloat16, device=dev)
    dw13 = torch.full((E, 2 * F, d), float("nan"), dtype=torch.bfloat16, device=dev)
    dw2 = torch.full((E, d, F), float("nan"), dtype=torch.bfloat16, device=dev)
    print(f"[backward] {sh} segments {list(counts_or_offsets)[:12]}...", flush=True)
    moe.moe_grouped_ffn_backward(sh, moe.to_device_bf16(x), offs, moe.to_device_bf16(w13), moe.to_device_bf16(w2),
                                 moe.to_device_bf16(dy), dx, dw13, dw2,
                                 moe.alloc_workspace(sh, moe.MOE_WS_FFN_BWD))
    torch.cuda.synchronize()
    return x, dy, w13, w2, dev_bits(dx), dev_bits(dw13), dev_bits(dw2)


def _check(sh, segs_arg, x, dy, w13, w2, g_dx, g_dw13, g_dw2, experts=None):
    E, C = sh.E_local, sh.expert_capacity
    segs = obwd.expert_segments(segs_arg, E, C)
    xd, dyd = oracle.bf16_to_f64(x), oracle.bf16_to_f64(dy)
    covered = np.zeros(sh.capacity, bool)
    worst = 0.0
    for e, (a, b) in enumerate(segs):
        covered[a:b] = True
        if experts is not None and e not in experts:
            continue
        if b <= a:
            assert not g_dw13[e].any() and not g_dw2[e].any(), f"expert {e} has no rows but nonzero dW"
            continue
        rdx, r13, r2 = obwd.swiglu_ffn_backward(xd[a:b], oracle.bf16_to_f64(w13[e]), oracle.bf16_to_f64(w2[e]),
                                                dyd[a:b])
        errs = (rel_fro(oracle.bf16_to_f64(g_dx[a:b]), rdx), rel_fro(oracle.bf16_to_f64(g_dw13[e]), r13),
                rel_fro(oracle.bf16_to_f64(g_dw2[e]), r2))
        worst = max(worst, *errs)
        assert max(errs) <= REL_TOL, (e, b - a, errs)
    # rows outside every segment were not written (still NaN)
    outside = oracle.bf16_to_f64(g_dx[~covered])
    assert np.isnan(outside).all(), "dX written outside the expert segments"
    print(f"[backward] worst rel_fro {worst:.3e}", flush=True)


def test_backward_ragged_segments_and_k_tails():
    lengths = [1, 0, 31, 32, 33, 63, 64, 65, 96, 127, 128, 129, 160, 191, 255, 256, 273, 612]
    E = len(lengths)
    offs = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    sh = S(T=int(offs[-1]) + 5, d=264, E=E, top_k=1, F=136, E_local=E)      # cap = T: 5 spare rows
    out = _run(sh, offs, 1)
    _check(sh, offs, *out)


def test_backward_decode_sized_segments():
    lengths = [3, 0, 1, 7, 2, 9, 0, 5, 4, 6, 1, 8, 2, 0, 3, 1]
    E = len(lengths)
    offs = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    sh = S(T=int(offs[-1]), d=512, E=E, top_k=1, F=256, E_local=E)
    out = _run(sh, offs, 2)
    _check(sh, offs, *out)


def test_backward_masked_layout():
    C = 20
    counts = np.array([25, 0, 20, 3, 19, 40, 1, 8], np.int32)                # experts 0 and 5 drop rows
    E = counts.size
    sh = S(T=64, d=256, E=E, top_k=4, F=128, E_local=E, expert_capacity=C)
    out = _run(sh, counts, 3)
    _check(sh, counts, *out)


def test_backward_dsv3_expert_shape():
    lengths = [250, 0, 263, 300]
    E = len(lengths)
    offs = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    sh = S(T=int(offs[-1]), d=7168, E=E, top_k=1, F=2048, E_local=E)
    out = _run(sh, offs, 4)
    _check(sh, offs, *out)


def test_backward_no_tokens_zero_weight_gradients():
    E, d, F = 3, 64, 32
    sh = S(T=0, d=d, E=E, top_k=1, F=F, E_local=E)
    dev = "cuda"
    offs = torch.zeros(E + 1, dtype=torch.int32, device=dev)
    w = torch.zeros(8, dtype=torch.bfloat16, device=dev)
    dw13 = torch.full((E, 2 * F, d), float("nan"), dtype=torch.bfloat16, device=dev)
    dw2 = torch.full((E, d, F), float("nan"), dtype=torch.bfloat16, device=dev)
    moe.moe_grouped_ffn_backward(sh, None, offs, w, w, None, None, dw13, dw2, None)
    torch.cuda.synchronize()
    assert (dw13.float() == 0).all() and (dw2.float() == 0).all()
