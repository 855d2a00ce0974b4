"""GPU parity of the layer backward (moe_layer_backward, through the C ABI) against the fp64
oracle (``oracle.moe_backward.layer_backward``): dx, dw_router, the routed experts' dw13 / dw2
and the shared expert's dws13 / dws2, each within rel. Frobenius 5e-3 (bf16 storage, fp32
accumulation; rounded to bf16 once each on the way: the expert rows' output gradients,
dlogits, and the expert-MLP backward's dA, [dH dU] and recomputed activation).

The routing is the forward's; where the GPU took a rounding near-tie the other way, the
oracle uses the GPU's (equally valid) choice for that token (the routing protocol of the
forward tests).  Cases: every gating mode (softmax renormalised, softmax over all experts
with a scale, softmax with a Zipf router bias, sigmoid renormalised with a group limit and a
scale, raw sigmoid), a rank slice with slots routed elsewhere, a shared expert of another
width (own launches) and of the routed width, the masked-decode layout with dropped slots, a
shape whose routed products take 320-row tiles, the forward with and without the gather folded (bit-identical gradients), run-to-run
determinism, no tokens, and the full DeepSeek-V3-shaped workload.
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

S = wl.MoEShape
CASES = {
    "tiny": (wl.WORKLOADS["tiny"].shape, 0.02, 0.0),
    "group_limited_slice_shared": (S(T=300, d=520, E=64, top_k=8, F=1000, E_local=8, e_begin=8, F_shared=264,
                                     gate=wl.GATE_SIGMOID, n_group=8, topk_group=4, routed_scale=2.5), None, 0.0),
    "skewed_bias": (S(T=700, d=256, E=32, top_k=8, F=96, E_local=32), 2 * 256 ** -0.5, 1.2),
    "softmax_all_experts_scaled": (S(T=200, d=128, E=16, top_k=4, F=64, E_local=16, renormalize=0,
                                     routed_scale=1.5), None, 0.0),
    "sigmoid_raw_slice_end": (S(T=150, d=64, E=40, top_k=5, F=40, E_local=8, e_begin=32, gate=wl.GATE_SIGMOID,
                                renormalize=0), None, 0.0),
    "merged_shared_decode": (S(T=5, d=1024, E=96, top_k=8, F=256, E_local=12, F_shared=256,
                               gate=wl.GATE_SIGMOID), None, 0.0),
    "masked_drops": (S(T=120, d=192, E=16, top_k=4, F=64, E_local=16, expert_capacity=12, F_shared=64), None, 0.0),
    # 256 rows per expert on average over 32 experts, d and 2F multiples of 64: the routed dX runs
    # on the 320-row tile without K-tail code, the recomputed up-projection on 320-row tiles
    "tile320_rows": (S(T=1024, d=2048, E=32, top_k=8, F=1024, E_local=32), None, 0.0),
    # the logit partials of a K split with uneven chunks (16 chunks of 7 slices of 64, the last 5,
    # its last slice 24 wide) summed again for the gate gradients; router dW over token chunks
    "router_ksplit_ragged": (S(T=4096, d=7000, E=128, top_k=8, F=64, E_local=8, e_begin=40), None, 0.0),
}
GRADS = ("dx", "dw_router", "dw13", "dw2", "dws13", "dws2")


def _dout(sh, seed):
    rng = np.random.default_rng(seed)
    return wl.f32_to_bf16_bits(rng.standard_normal((sh.T, sh.d)).astype(np.float32))


def _gpu_backward(inputs, dout_bits):
    layer = moe.DeviceLayer(inputs)
    layer.forward()
    g = layer.backward(moe.to_device_bf16(dout_bits))
    torch.cuda.synchronize()
    return layer, {k: (dev_bits(v) if v is not None else None) for k, v in g.items()}


def _oracle(inputs, layer, dout_bits):
    g_idx, g_w, g_keys = run_route(layer)
    o_idx, o_w, keys64, near = check_routing(inputs, g_idx, g_w, g_keys)
    idx, w = oracle_routing_with_gpu_ties(o_idx, o_w, keys64, g_idx, near, inputs["shape"])
    return obwd.layer_backward(inputs, oracle.bf16_to_f64(dout_bits), routing=(idx, w)), near


def _compare(name, got, ref):
    errs = {}
    for k in GRADS:
        if ref[k] is None:
            assert got[k] is None, k
            continue
        errs[k] = rel_fro(oracle.bf16_to_f64(got[k]), ref[k])
    print(f"[layer backward] {name}: " + ", ".join(f"{k}={v:.2e}" for k, v in errs.items()), flush=True)
    for k, v in errs.items():
        assert v <= REL_TOL, (name, k, v)
    return errs


@pytest.mark.parametrize("name", list(CASES))
def test_layer_backward_small(name):
    sh, rstd, zipf = CASES[name]
    print(f"[layer backward] case {name}: {sh}", flush=True)
    inputs = wl.custom_inputs(sh, seed=21, router_std=rstd, zipf_s=zipf)
    dout = _dout(sh, 5)
    layer, got = _gpu_backward(inputs, dout)
    ref, near = _oracle(inputs, layer, dout)
    _compare(name, got, ref)
    # experts without rows get exactly zero weight gradients
    counts = layer.region(moe.MOE_REGION_COUNTS, torch.int32, (sh.E_local,)).cpu().numpy()
    for e in np.nonzero(counts == 0)[0]:
        assert not got["dw13"][e].any() and not got["dw2"][e].any(), e


def test_layer_backward_gather_structures_and_determinism():
    """The forward with the gather folded (rows read through row_token, x_perm never written)
    and unfolded leaves the same state for the backward: gradients bit-identical; two
    backward calls give bit-identical results."""
    sh, rstd, zipf = CASES["group_limited_slice_shared"]
    inputs = wl.custom_inputs(sh, seed=22, router_std=rstd, zipf_s=zipf)
    dout = _dout(sh, 6)
    outs = []
    for fusion in (wl.FUSION_VARIANTS["gather"], wl.FUSION_VARIANTS["unfused"]):
        print(f"[layer backward] fusion {fusion:#x}", flush=True)
        layer = moe.DeviceLayer(dict(inputs, shape=sh.replace(fusion=fusion)))
        layer.forward()
        d = moe.to_device_bf16(dout)
        a = {k: dev_bits(v) for k, v in layer.backward(d).items() if v is not None}
        b = {k: dev_bits(v) for k, v in layer.backward(d).items() if v is not None}
        torch.cuda.synchronize()
        for k in a:
            assert np.array_equal(a[k], b[k]), f"backward not deterministic: {k}"
        outs.append(a)
    for k in outs[0]:
        assert np.array_equal(outs[0][k], outs[1][k]), f"gather structures differ: {k}"


def test_layer_backward_no_tokens_zero_weight_gradients():
    sh = S(T=0, d=64, E=8, top_k=2, F=32, E_local=8, F_shared=16)
    dev = "cuda"
    bf = torch.bfloat16
    g = {"dw_router": (sh.E, sh.d), "dw13": (sh.E_local, 2 * sh.F, sh.d), "dw2": (sh.E_local, sh.d, sh.F),
         "dws13": (2 * sh.F_shared, sh.d), "dws2": (sh.d, sh.F_shared)}
    t = {k: torch.full(v, float("nan"), dtype=bf, device=dev) for k, v in g.items()}
    moe.moe_layer_backward(sh, None, None, None, None, None, None, None, None, None, None, t["dw_router"],
                           t["dw13"], t["dw2"], t["dws13"], t["dws2"], None)
    torch.cuda.synchronize()
    for k, v in t.items():
        assert (v.float() == 0).all(), k


@pytest.mark.parametrize("name", ["dsv3"])
def test_layer_backward_full_workload(name):
    """The DeepSeek-V3-shaped rank share at full size (the configuration the benchmark times),
    every gradient against the fp64 oracle over the whole batch (the oracle takes ~40-70 s of
    host time here; the decode-sized, skewed and every-gating-mode cases run at small sizes
    above)."""
    print(f"[layer backward] full workload {name}: generating inputs", flush=True)
    inputs = wl.make_inputs(name)
    sh = inputs["shape"]
    dout = _dout(sh, 7)
    layer, got = _gpu_backward(inputs, dout)
    print(f"[layer backward] {name}: GPU backward ran, oracle on {sh.T} tokens", flush=True)
    ref, near = _oracle(inputs, layer, dout)
    _compare(name, got, ref)


@pytest.mark.parametrize("capacity", [0, 6])
def test_forward_backward_graph_replay(capacity):
    """Forward and backward captured together in one HIP graph (the library issues no memset,
    allocation or host synchronisation): three replays on new token rows and output gradients,
    with eager calls and synchronisations between them, every gradient of every replay
    bit-identical to the eager forward + backward on the same inputs."""
    sh = S(T=64, d=512, E=32, top_k=4, F=256, E_local=8, F_shared=256, expert_capacity=capacity)
    inputs = wl.custom_inputs(sh, seed=4, router_std=2 * 512 ** -0.5, zipf_s=1.1)
    graphed = moe.DeviceLayer(inputs)
    eager = moe.DeviceLayer(inputs)
    dout = moe.to_device_bf16(_dout(sh, 1))
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        graphed.forward()                                         # warm-up (allocates the workspaces)
        graphed.backward(dout)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        graphed.forward()
        grads = graphed.backward(dout)
    rng = np.random.default_rng(98)
    for rep in range(3):
        xt = moe.to_device_bf16(wl.f32_to_bf16_bits(rng.standard_normal((sh.T, sh.d)).astype(np.float32)))
        dt = moe.to_device_bf16(wl.f32_to_bf16_bits(rng.standard_normal((sh.T, sh.d)).astype(np.float32)))
        graphed.x.copy_(xt)
        dout.copy_(dt)
        g.replay()
        torch.cuda.synchronize()
        got = {k: dev_bits(v) for k, v in grads.items() if v is not None}
        eager.x.copy_(xt)
        eager.forward()
        want = {k: dev_bits(v) for k, v in eager.backward(dt).items() if v is not None}
        torch.cuda.synchronize()
        print(f"[graph] capacity={capacity} replay {rep}: checked", flush=True)
        for k in want:
            np.testing.assert_array_equal(got[k], want[k], err_msg=k)
