"""Helpers of the GPU parity tests: run the C ABI on device tensors and compare with the
fp64 oracle under the routing protocol

  R1  decision exactness: the oracle's decision replayed on the GPU's own float32 keys
      (group sums as float32 additions) equals the GPU's topk_idx bit for bit, and the
      oracle's counts / offsets / permutation of the GPU's topk_idx equal the GPU's;
  R2  end to end: the GPU's topk_idx equals the fp64 decision except at rounding
      near-ties.  A near-tie is explained when every decision that differs sits on an
      fp64 margin of at most NEAR_TIE_FACTOR x the token's largest key error: a differing
      choice of groups by the fp64 group scores of the swapped groups, a differing slot by
      the fp64 keys of the two experts that trade places (a swap needs a margin of at most
      twice the key error, a group swap at most four times);
  R3  gates: |w_gpu - w_fp64| <= 1e-5 * max(1, routed_scale) on matched tokens.

Outputs: relative Frobenius error <= 5e-3 against the oracle (bf16 storage, fp32
accumulation) over the whole [T, d] output and over the live rows of every expert.
"""
import numpy as np
import torch

import oracle
from paper_2607_18631_amd import moe

REL_TOL = 5e-3
NEAR_TIE_FACTOR = 8.0


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


def _kept_groups(keys, n_group, topk_group):
    """Groups kept per token (sorted ids) by the oracle's group rule in the keys' own dtype."""
    gs = oracle.group_scores(keys, n_group)
    order = np.lexsort((np.broadcast_to(np.arange(n_group), gs.shape), -gs), axis=1)
    return np.sort(order[:, :topk_group], axis=1)


def explain_near_tie(t, sh, keys64, g_keys, g_idx, o_idx, kerr_t):
    """Assert that token t's differing decision is a rounding near-tie (see R2)."""
    delta = NEAR_TIE_FACTOR * kerr_t + 1e-12
    if sh.n_group > 1:
        k64 = keys64[t:t + 1]
        g_grp = _kept_groups(g_keys[t:t + 1].astype(np.float32), sh.n_group, sh.topk_group)[0]
        o_grp = _kept_groups(k64, sh.n_group, sh.topk_group)[0]
        if not np.array_equal(g_grp, o_grp):
            gs = oracle.group_scores(k64, sh.n_group)[0]
            a = np.sort(gs[np.setdiff1d(g_grp, o_grp)])
            b = np.sort(gs[np.setdiff1d(o_grp, g_grp)])
            assert np.all(np.abs(a - b) <= delta), \
                f"token {t}: groups {g_grp} vs oracle {o_grp}, fp64 scores {a} vs {b} beyond {delta:.3e}"
            return "group"
    diff = np.nonzero(g_idx[t] != o_idx[t])[0]
    ka = keys64[t, g_idx[t, diff]]
    kb = keys64[t, o_idx[t, diff]]
    assert np.all(np.abs(ka - kb) <= delta), \
        f"token {t}: GPU {g_idx[t]} vs oracle {o_idx[t]} is not a rounding near-tie ({ka} vs {kb}, {delta:.3e})"
    return "expert"


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
        explain_near_tie(int(t), sh, keys64, g_keys, g_idx, o_idx, float(kerr[t].max()))
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


def expert_segments(sh, counts, offsets):
    """(expert, first row, live rows) of every local expert with rows: the monotone offsets, or
    the valid prefix of each equal-stride segment in the masked-decode layout."""
    C = sh.expert_capacity
    segs = []
    for e in range(sh.E_local):
        if C > 0:
            a, n = e * C, min(int(counts[e]), C)
        else:
            a, n = int(offsets[e]), int(offsets[e + 1] - offsets[e])
        if n > 0:
            segs.append((e, a, n))
    return segs


def live_y_rows(layer, segs):
    """float64 values of the live rows of the layer's y_perm region only (rows outside every
    segment are never written and are not decoded)."""
    sh = layer.shape
    y = layer.region(moe.MOE_REGION_Y_PERM, torch.bfloat16, (sh.capacity, sh.d))
    return {e: oracle.bf16_to_f64(dev_bits(y[a:a + n])) for e, a, n in segs}


def check_expert_rows(inputs, xd, segs, rows_by_expert, row_token):
    """Every live expert row against the oracle's SwiGLU MLP of its token, expert by expert.
    Returns (worst per-expert rel_fro, rel_fro over all live rows)."""
    worst, num, den = 0.0, 0.0, 0.0
    for e, a, n in segs:
        ref = oracle.swiglu_ffn(xd[row_token[a:a + n]], oracle.bf16_to_f64(inputs["w13"][e]),
                                oracle.bf16_to_f64(inputs["w2"][e]))
        got = rows_by_expert[e]
        err = rel_fro(got, ref)
        assert err <= REL_TOL, f"expert {e} ({n} rows): rel_fro {err:.3e}"
        worst = max(worst, err)
        num += float(np.sum((got - ref) ** 2))
        den += float(np.sum(ref ** 2))
    return worst, (num ** 0.5) / (den ** 0.5 if den > 0 else 1.0)
