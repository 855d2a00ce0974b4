"""GPU parity of the masked-decode layout (equal-stride expert segments of capacity C, the
slots ranked past C dropped) against the fp64 oracle, plus HIP-graph replay of the layer.

Cases: drops in most experts, C = 1, a single token, a ragged token count, a rank slice in
the middle of a group-limited sigmoid router with a shared expert, and C at least every
expert's count (no drop: output bit-identical to the offsets layout).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_18631_amd import moe
from paper_2607_18631_amd import workloads as wl

import parity_util
from parity_util import (REL_TOL, check_routing, dev_bits, oracle_routing_with_gpu_ties, rel_fro,
                         run_route)

pytestmark = pytest.mark.gpu

S = wl.MoEShape
MASKED = {
    # mean rows per expert 8 > C = 6, skewed: the popular experts drop slots
    "drops_skewed": (S(T=64, d=512, E=32, top_k=4, F=256, E_local=16, expert_capacity=6), 2 * 512 ** -0.5, 1.1),
    "capacity_one": (S(T=40, d=256, E=16, top_k=4, F=128, E_local=16, expert_capacity=1), None, 0.0),
    "single_token": (S(T=1, d=1024, E=64, top_k=6, F=512, E_local=64, expert_capacity=2), None, 0.0),
    "ragged_T257": (S(T=257, d=264, E=16, top_k=2, F=136, E_local=16, expert_capacity=24), None, 0.8),
    "sigmoid_slice_shared": (S(T=100, d=1024, E=64, top_k=6, F=512, E_local=16, e_begin=16, F_shared=512,
                               gate=wl.GATE_SIGMOID, n_group=8, topk_group=4, routed_scale=2.5,
                               expert_capacity=8), None, 0.0),
}


def _inputs(name):
    sh, rstd, zipf = MASKED[name]
    return wl.custom_inputs(sh, seed=17, router_std=rstd, zipf_s=zipf)


def _regions(layer):
    sh = layer.shape
    T, k, cap = sh.T, sh.top_k, sh.capacity
    g = lambda r, dt, shp: layer.region(r, dt, shp).cpu().numpy()
    return {
        "topk_idx": g(moe.MOE_REGION_TOPK_IDX, torch.int32, (T, k)),
        "counts": g(moe.MOE_REGION_COUNTS, torch.int32, (sh.E_local,)),
        "offsets": g(moe.MOE_REGION_OFFSETS, torch.int32, (sh.E_local + 1,)),
        "row_token": g(moe.MOE_REGION_ROW_TOKEN, torch.int32, (cap,)),
        "slot_row": g(moe.MOE_REGION_SLOT_ROW, torch.int32, (T, k)),
    }


def _check_masked_permutation(sh, reg, g_idx):
    """Counts (before the drop), offsets e * C, slot rows (-1 for dropped slots) and the tokens
    of the kept rows, bit-exact against the oracle on the GPU's own routing."""
    C = sh.expert_capacity
    counts, offsets = oracle.counts_offsets(g_idx, sh.e_begin, sh.E_local, C)
    row_token, slot_row = oracle.permutation(g_idx, sh.e_begin, sh.E_local, C)
    np.testing.assert_array_equal(reg["counts"], counts)
    np.testing.assert_array_equal(reg["offsets"], offsets)
    np.testing.assert_array_equal(reg["slot_row"], slot_row)
    kept = row_token >= 0
    np.testing.assert_array_equal(reg["row_token"][kept], row_token[kept])
    return counts, row_token


@pytest.mark.parametrize("name", list(MASKED))
def test_masked_layer_parity(name):
    inputs = _inputs(name)
    sh = inputs["shape"]
    C = sh.expert_capacity
    print(f"[masked] {name}: {sh}", flush=True)
    layer = moe.DeviceLayer(inputs)
    out = layer.forward()
    torch.cuda.synchronize()
    g_idx, g_w, g_keys = run_route(layer)
    o_idx, o_w, keys64, near = check_routing(inputs, g_idx, g_w, g_keys)
    reg = _regions(layer)
    np.testing.assert_array_equal(reg["topk_idx"], g_idx)
    counts, row_token = _check_masked_permutation(sh, reg, g_idx)
    dropped = int(np.maximum(counts - C, 0).sum())
    # per-expert rows of the valid prefix of each segment (only those rows are decoded: the rest
    # of a segment is never written)
    xd = oracle.bf16_to_f64(inputs["x"])
    segs = parity_util.expert_segments(sh, counts, reg["offsets"])
    parity_util.check_expert_rows(inputs, xd, segs, parity_util.live_y_rows(layer, segs), row_token)
    # layer output: the kept slots of the whole batch's routing
    idx, w = oracle_routing_with_gpu_ties(o_idx, o_w, keys64, g_idx, near, sh)
    keep = oracle.keep_mask(idx, sh.e_begin, sh.E_local, C)
    ref = oracle.expert_outputs_for_tokens(xd, idx, w, sh, inputs["w13"], inputs["w2"], inputs.get("ws13"),
                                           inputs.get("ws2"), keep)
    err = rel_fro(oracle.bf16_to_f64(dev_bits(out)), ref)
    print(f"[masked] {name}: rel_fro={err:.3e} dropped={dropped} near_ties={len(near)}", flush=True)
    assert err <= REL_TOL


@pytest.mark.parametrize("name", ["drops_skewed", "sigmoid_slice_shared"])
def test_masked_components_compose_to_layer(name):
    """moe_permute -> moe_grouped_ffn (counts as the segment lengths) -> moe_combine in the
    masked layout == the layer, bit for bit."""
    inputs = _inputs(name)
    sh = inputs["shape"]
    layer = moe.DeviceLayer(inputs)
    ref = layer.forward().clone()
    dev = "cuda"
    T, k, cap = sh.T, sh.top_k, sh.capacity
    idx = torch.empty((T, k), dtype=torch.int32, device=dev)
    w = torch.empty((T, k), dtype=torch.float32, device=dev)
    moe.moe_route(sh, layer.x, layer.w_router, layer.bias, idx, w, None, moe.alloc_workspace(sh, moe.MOE_WS_ROUTE))
    counts = torch.empty(sh.E_local, dtype=torch.int32, device=dev)
    offsets = torch.empty(sh.E_local + 1, dtype=torch.int32, device=dev)
    row_token = torch.empty(cap, dtype=torch.int32, device=dev)
    slot_row = torch.empty((T, k), dtype=torch.int32, device=dev)
    x_perm = torch.empty((cap, sh.d), dtype=torch.bfloat16, device=dev)
    moe.moe_permute(sh, idx, layer.x, counts, offsets, row_token, slot_row, x_perm,
                    moe.alloc_workspace(sh, moe.MOE_WS_PERMUTE))
    torch.cuda.synchronize()
    # the kept rows of x_perm are bit-exact copies of their tokens
    g_idx = idx.cpu().numpy()
    o_row_token, _ = oracle.permutation(g_idx, sh.e_begin, sh.E_local, sh.expert_capacity)
    kept = np.nonzero(o_row_token >= 0)[0]
    np.testing.assert_array_equal(dev_bits(x_perm)[kept], inputs["x"][o_row_token[kept]])
    y_perm = torch.empty((cap, sh.d), dtype=torch.bfloat16, device=dev)
    moe.moe_grouped_ffn(sh, x_perm, counts, layer.w13, layer.w2, y_perm, moe.alloc_workspace(sh, moe.MOE_WS_FFN))
    shared_y = None
    if sh.F_shared:
        ssh = sh.replace(E=1, top_k=1, e_begin=0, E_local=1, F=sh.F_shared, F_shared=0, n_group=1, topk_group=1,
                         expert_capacity=0)
        soff = torch.tensor([0, T], dtype=torch.int32, device=dev)
        shared_y = torch.empty((T, sh.d), dtype=torch.bfloat16, device=dev)
        moe.moe_grouped_ffn(ssh, layer.x, soff, layer.ws13, layer.ws2, shared_y,
                            moe.alloc_workspace(ssh, moe.MOE_WS_FFN))
    out = torch.empty((T, sh.d), dtype=torch.bfloat16, device=dev)
    moe.moe_combine(sh, y_perm, slot_row, w, shared_y, out)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(dev_bits(out), dev_bits(ref))


def test_masked_without_drops_equals_offsets_layout():
    """C at least every expert's count (and at least T * top_k / E, so both layouts pick the
    same GEMM tiles): every slot is kept and the output is bit-identical to the offsets layout."""
    sh0 = S(T=300, d=520, E=64, top_k=8, F=1000, E_local=8, e_begin=8, F_shared=264, gate=wl.GATE_SIGMOID,
            n_group=8, topk_group=4, routed_scale=2.5)
    inputs = wl.custom_inputs(sh0, seed=11)
    base = moe.DeviceLayer(inputs)
    a = dev_bits(base.forward())
    counts = base.region(moe.MOE_REGION_COUNTS, torch.int32, (sh0.E_local,)).cpu().numpy()
    C = int(max(counts.max(), sh0.T * sh0.top_k // sh0.E + 1))
    masked = moe.DeviceLayer(dict(inputs, shape=sh0.replace(expert_capacity=C)))
    b = dev_bits(masked.forward())
    torch.cuda.synchronize()
    np.testing.assert_array_equal(b, a)


@pytest.mark.parametrize("capacity", [0, 6])
def test_layer_graph_replay(capacity):
    """The layer captured in a HIP graph (torch.cuda.graph on the library's stream argument):
    three replays on new token rows, with eager layer calls and synchronizations between them,
    each bit-identical to the eager layer on the same rows."""
    sh = S(T=64, d=512, E=32, top_k=4, F=256, E_local=8, F_shared=256, expert_capacity=capacity)
    inputs = wl.custom_inputs(sh, seed=3, router_std=2 * 512 ** -0.5, zipf_s=1.1)
    graphed = moe.DeviceLayer(inputs)
    eager = moe.DeviceLayer(inputs)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        graphed.forward()                                         # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        graphed.forward()
    rng = np.random.default_rng(99)
    for rep in range(3):
        x = wl.f32_to_bf16_bits(rng.standard_normal((sh.T, sh.d)).astype(np.float32))
        xt = moe.to_device_bf16(x)
        graphed.x.copy_(xt)
        g.replay()
        torch.cuda.synchronize()
        got = dev_bits(graphed.out)
        eager.x.copy_(xt)
        want = dev_bits(eager.forward())
        torch.cuda.synchronize()
        print(f"[graph] capacity={capacity} replay {rep}: checked", flush=True)
        np.testing.assert_array_equal(got, want)
