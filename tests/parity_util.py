"""Helpers of the GPU parity tests: run the C ABI on device tensors and compare with the
fp64 oracle under the routing protocol

  R1  decision exactness: the oracle's decision replayed on the GPU's own float32 keys
      (group sums as float32 additions) equals the GPU's topk_idx bit for bit, and the
      oracle's counts / offsets / permutation of the GPU's topk_idx equal the GPU's;
  R2  end to end: the GPU's topk_idx equals the fp64 decision except at rounding
      near-ties (every swapped pair's fp64 keys within 16x the token's key error);
  R3  gates: |w_gpu - w_fp64| <= 1e-5 * max(1, routed_scale) on matched tokens.

Outputs: relative Frobenius error <= 5e-3 against the oracle (bf16 storage, fp32
accumulation), on every row at small sizes and on sampled rows at full sizes.
"""
import numpy as np
import torch

import oracle
from paper_2607_18631_amd import moe

REL_TOL = 5e-3


def rel_fro(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.linalg.norm(ref)
    return np.linalg.norm(got - ref) / (den if den > 0 else 1.0)


def dev_bits(t):
    return moe.bf16_bits(t)


def run_route(layer: "moe.DeviceLayer"):
    sh = layer.shape
    dev = layer.device
    idx = torch.empty((sh.T, sh.top_k), dtype=torch.int32, device=dev)
    w = torch.empty((sh.T, sh.top_k), dtype=torch.float32, device=dev)
    keys = torch.empty((sh.T, sh.E), dtype=torch.float32, device=dev)
    ws = moe.alloc_workspace(sh, moe.MOE_WS_ROUTE, dev)
    moe.moe_route(sh, layer.x, layer.w_router, layer.bias, idx, w, keys, ws)
    torch.cuda.synchronize()
    return idx.cpu().numpy(), w.cpu().numpy(), keys.cpu().numpy()


def check_routing(inputs, g_idx, g_w, g_keys, xd=None):
    """R1/R2/R3.  Returns (oracle idx, oracle w, oracle keys64, near-tie token list)."""
    sh = inputs["shape"]
    if xd is None:
        xd = oracle.bf16_to_f64(inputs["x"])
    L = oracle.router_logits(xd, oracle.bf16_to_f64(inputs["w_router"]))
    keys64 = oracle.gating_keys(L, sh.gate, inputs.get("bias"))
    # R1: replay on the GPU's float32 keys
    r1 = oracle.decide_topk(g_keys.astype(np.float32), sh.top_k, sh.n_group, sh.topk_group)
    np.testing.assert_array_equal(g_idx, r1, err_msg="R1: GPU decision differs from its own keys' decision")
    # the GPU keys are the fp64 keys up to float32 rounding of the logits
    kerr = np.abs(g_keys.astype(np.float64) - keys64)
    assert kerr.max() < 1e-3 * max(1.0, np.abs(keys64).max()), kerr.max()
    # R2
    o_idx = oracle.decide_topk(keys64, sh.top_k, sh.n_group, sh.topk_group)
    bad = np.nonzero((o_idx != g_idx).any(axis=1))[0]
    near = []
    for t in bad:
        delta = 16.0 * kerr[t].max() + 1e-12
        ka = keys64[t, g_idx[t]]
        kb = keys64[t, o_idx[t]]
        assert np.all(np.abs(np.sort(ka) - np.sort(kb)) <= 2 * delta), \
            f"token {t}: GPU {g_idx[t]} vs oracle {o_idx[t]} is not a rounding near-tie"
        near.append(int(t))
    # R3 on matched tokens
    o_w = oracle.gate_weights(keys64, o_idx, sh.gate, sh.renormalize, sh.routed_scale)
    ok = np.ones(sh.T, bool)
    ok[near] = False
    np.testing.assert_allclose(g_w[ok], o_w[ok], rtol=0, atol=1e-5 * max(1.0, sh.routed_scale))
    return o_idx, o_w, keys64, near


def oracle_routing_with_gpu_ties(o_idx, o_w, keys64, g_idx, near, sh):
    """Oracle routing, except near-tie tokens take the GPU's (equally valid) choice."""
    idx = o_idx.copy()
    w = o_w.copy()
    if near:
        idx[near] = g_idx[near]
        w[near] = oracle.gate_weights(keys64[near], g_idx[near], sh.gate, sh.renormalize, sh.routed_scale)
    return idx, w
