"""GPU parity of the layer's four kernel structures (the paper's fuse_gather x fuse_combine
matrix): unfused, gather folded into the up-projection, combine folded into the
down-projection (float32 atomics), both.

Gather folding changes no arithmetic: those variants are bit-identical to the default.  The
folded combine adds unrounded expert rows in no fixed order, so it is checked against the
oracle to the output tolerance, with routing and permutation still bit-exact.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_18631_amd import moe
from paper_2607_18631_amd import workloads as wl

from parity_util import (REL_TOL, check_routing, dev_bits, oracle_routing_with_gpu_ties, rel_fro,
                         run_route)

pytestmark = pytest.mark.gpu

S = wl.MoEShape
CASES = {
    # shared expert narrower than the routed ones: its own launches
    "group_limited_slice": S(T=300, d=520, E=64, top_k=8, F=1000, E_local=8, e_begin=8, F_shared=264,
                             gate=wl.GATE_SIGMOID, n_group=8, topk_group=4, routed_scale=2.5),
    # shared expert as wide as the routed ones: inside the routed launches
    "decode_merged_shared": S(T=5, d=1024, E=96, top_k=8, F=256, E_local=12, F_shared=256, gate=wl.GATE_SIGMOID),
    "ragged_T257": S(T=257, d=264, E=16, top_k=2, F=136, E_local=16),
    "masked_drops": S(T=64, d=512, E=32, top_k=4, F=256, E_local=16, expert_capacity=6, F_shared=256),
}


def _layer_out(inputs, fusion):
    sh = inputs["shape"].replace(fusion=fusion)
    layer = moe.DeviceLayer(dict(inputs, shape=sh))
    out = dev_bits(layer.forward())
    torch.cuda.synchronize()
    return layer, out


def _oracle_out(inputs, layer, toks=None):
    sh = inputs["shape"]
    g_idx, g_w, g_keys = run_route(layer)
    xd = oracle.bf16_to_f64(inputs["x"])
    o_idx, o_w, keys64, near = check_routing(inputs, g_idx, g_w, g_keys, xd)
    idx, w = oracle_routing_with_gpu_ties(o_idx, o_w, keys64, g_idx, near, sh)
    keep = oracle.keep_mask(idx, sh.e_begin, sh.E_local, sh.expert_capacity) if sh.expert_capacity else None
    if toks is None:
        toks = np.arange(sh.T)
    return oracle.expert_outputs_for_tokens(xd[toks], idx[toks], w[toks], sh, inputs["w13"], inputs["w2"],
                                            inputs.get("ws13"), inputs.get("ws2"),
                                            None if keep is None else keep[toks]), g_idx


@pytest.mark.parametrize("name", list(CASES))
def test_fusion_matrix_small(name):
    sh = CASES[name]
    inputs = wl.custom_inputs(sh, seed=23, zipf_s=1.1 if sh.expert_capacity else 0.0)
    print(f"[fusion] {name}: {sh}", flush=True)
    _, base = _layer_out(inputs, 0)
    for v in ("unfused", "gather"):
        _, out = _layer_out(inputs, wl.FUSION_VARIANTS[v])
        np.testing.assert_array_equal(out, base, err_msg=f"{v} differs from the default structure")
    for v in ("combine", "both"):
        layer, out = _layer_out(inputs, wl.FUSION_VARIANTS[v])
        ref, g_idx = _oracle_out(inputs, layer)
        # routing and permutation are the default's, bit for bit
        C = sh.expert_capacity
        row_token, slot_row = oracle.permutation(g_idx, sh.e_begin, sh.E_local, C)
        np.testing.assert_array_equal(layer.region(moe.MOE_REGION_SLOT_ROW, torch.int32, (sh.T, sh.top_k))
                                      .cpu().numpy(), slot_row)
        err = rel_fro(oracle.bf16_to_f64(out), ref)
        diff = rel_fro(oracle.bf16_to_f64(out), oracle.bf16_to_f64(base))
        print(f"[fusion] {name} {v}: rel_fro vs oracle {err:.3e}, vs default structure {diff:.3e}", flush=True)
        assert err <= REL_TOL


@pytest.mark.parametrize("name", ["dsv3", "mixtral", "k2decode"])
def test_fused_combine_full_workload(name):
    """Both folds at the full workload sizes (the benchmark's fusion-matrix configuration):
    every output token against the oracle."""
    print(f"[fusion] full workload {name}: generating inputs", flush=True)
    inputs = wl.make_inputs(name)
    sh = inputs["shape"]
    layer, out = _layer_out(inputs, wl.FUSION_VARIANTS["both"])
    ref, _ = _oracle_out(inputs, layer)
    got = oracle.bf16_to_f64(out)
    err = rel_fro(got, ref)
    blk = max(rel_fro(got[i:i + 128], ref[i:i + 128]) for i in range(0, sh.T, 128))
    print(f"[fusion] {name} both: rel_fro={err:.3e} over all {sh.T} tokens (worst 128-token block {blk:.3e})",
          flush=True)
    assert err <= REL_TOL and blk <= 2 * REL_TOL
    # the folded combine is the unfolded one up to summation order and one bf16 rounding
    _, base = _layer_out(inputs, 0)
    assert rel_fro(got, oracle.bf16_to_f64(base)) <= REL_TOL
