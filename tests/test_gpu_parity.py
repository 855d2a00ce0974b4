"""GPU parity of the HIP path (through the C ABI) against the fp64 oracle.

Small cases compare every output and every intermediate; the five full-size workloads
run moe_layer_forward in the launch configuration the benchmark times and compare
routing, counts, offsets and the permutation on all tokens, every live expert row and
the whole layer output.  Edge cases: ragged and single-token batches, non-tile-multiple d and F,
zero-token experts, one hot expert, a rank slice in the middle of the experts, E = 1024
with top-16, E = 1 with top-1 (a dense SwiGLU MLP), T = 0.
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
SMALL = {
    "tiny": (wl.WORKLOADS["tiny"].shape, 0.02, 0.0),
    "tiny_T257": (wl.WORKLOADS["tiny"].shape.replace(T=257), 0.02, 0.0),
    "tiny_T1": (wl.WORKLOADS["tiny"].shape.replace(T=1), 0.02, 0.0),
    "group_limited_slice": (S(T=300, d=520, E=64, top_k=8, F=1000, E_local=8, e_begin=8, F_shared=264,
                              gate=wl.GATE_SIGMOID, n_group=8, topk_group=4, routed_scale=2.5), None, 0.0),
    "skewed_small": (S(T=1000, d=256, E=32, top_k=8, F=96, E_local=32), 2 * 256 ** -0.5, 1.2),
    "decode_small": (S(T=5, d=1024, E=96, top_k=8, F=256, E_local=12, F_shared=256, gate=wl.GATE_SIGMOID),
                     None, 0.0),
    "dense_identity": (S(T=130, d=136, E=1, top_k=1, F=72, E_local=1), None, 0.0),
    "softmax_no_renorm": (S(T=200, d=128, E=16, top_k=4, F=64, E_local=16, renormalize=0, routed_scale=1.5),
                          None, 0.0),
    "sigmoid_slice_end": (S(T=150, d=64, E=40, top_k=5, F=40, E_local=7, e_begin=33, gate=wl.GATE_SIGMOID,
                            renormalize=0), None, 0.0),
    "max_experts_top16": (S(T=70, d=64, E=1024, top_k=16, F=16, E_local=1024), None, 0.0),
    # 256 rows per expert on average over 32 experts with K tails in both projections (d, F not
    # multiples of 64): enough tiles that both projections take 320-row tiles, with tail slices
    "tile320_ktail": (S(T=1024, d=2000, E=32, top_k=8, F=1000, E_local=32), None, 0.0),
    # router logits on 256 x 256 tiles with a K split whose chunks are uneven: 110 slices of 64
    # (the last 24 wide) in 16 chunks of 7, the last chunk 5 slices
    "router_ksplit_ragged": (S(T=4096, d=7000, E=128, top_k=8, F=64, E_local=8, e_begin=40), None, 0.0),
    # permutation count tables too wide for the placement kernel to scan itself (10 super-chunks of
    # 512 tokens x 1024 experts; 79 super-chunks x 16 experts): the separate scan launch
    "wide_count_table": (S(T=5000, d=64, E=1024, top_k=16, F=16, E_local=1024), None, 0.0),
    "many_super_chunks": (S(T=40000, d=64, E=16, top_k=2, F=16, E_local=16), None, 0.0),
    # the kernel-crossover shape at expert multiplicities 4 and 32
    "crossover_me4": (wl.crossover(4).shape, None, 0.0),
    "crossover_me32": (wl.crossover(32).shape, None, 0.0),
}


def _inputs(name):
    sh, rstd, zipf = SMALL[name]
    return wl.custom_inputs(sh, seed=11, router_std=rstd, zipf_s=zipf)


def _intermediates(layer):
    sh = layer.shape
    T, k, cap = sh.T, sh.top_k, sh.capacity
    g = lambda r, dt, shp: layer.region(r, dt, shp).cpu().numpy()
    return {
        "topk_idx": g(moe.MOE_REGION_TOPK_IDX, torch.int32, (T, k)),
        "topk_w": g(moe.MOE_REGION_TOPK_W, torch.float32, (T, k)),
        "counts": g(moe.MOE_REGION_COUNTS, torch.int32, (sh.E_local,)),
        "offsets": g(moe.MOE_REGION_OFFSETS, torch.int32, (sh.E_local + 1,)),
        "row_token": g(moe.MOE_REGION_ROW_TOKEN, torch.int32, (cap,)),
        "slot_row": g(moe.MOE_REGION_SLOT_ROW, torch.int32, (T, k)),
    }


def _check_standalone_permute(layer, inputs, inter, n):
    """moe_permute on the layer's routing: same indices as the layer, x_perm rows bit-exact copies
    (the layer itself reads the token rows through row_token and writes no x_perm)."""
    sh = layer.shape
    dev = "cuda"
    T, k, cap = sh.T, sh.top_k, sh.capacity
    idx = layer.region(moe.MOE_REGION_TOPK_IDX, torch.int32, (T, k))
    counts = torch.empty(sh.E_local, dtype=torch.int32, device=dev)
    offsets = torch.empty(sh.E_local + 1, dtype=torch.int32, device=dev)
    row_token = torch.empty(cap, dtype=torch.int32, device=dev)
    slot_row = torch.empty((T, k), dtype=torch.int32, device=dev)
    x_perm = torch.empty((cap, sh.d), dtype=torch.bfloat16, device=dev)
    moe.moe_permute(sh, idx, layer.x, counts, offsets, row_token, slot_row, x_perm,
                    moe.alloc_workspace(sh, moe.MOE_WS_PERMUTE))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(offsets.cpu().numpy(), inter["offsets"])
    np.testing.assert_array_equal(row_token.cpu().numpy()[:n], inter["row_token"][:n])
    np.testing.assert_array_equal(slot_row.cpu().numpy(), inter["slot_row"])
    np.testing.assert_array_equal(dev_bits(x_perm[:n]), inputs["x"][inter["row_token"][:n]])


def _check_permutation(sh, inter, g_idx):
    counts, offsets = oracle.counts_offsets(g_idx, sh.e_begin, sh.E_local)
    row_token, slot_row = oracle.permutation(g_idx, sh.e_begin, sh.E_local)
    np.testing.assert_array_equal(inter["topk_idx"], g_idx)
    np.testing.assert_array_equal(inter["counts"], counts)
    np.testing.assert_array_equal(inter["offsets"], offsets)
    n = int(offsets[-1])
    np.testing.assert_array_equal(inter["row_token"][:n], row_token)
    np.testing.assert_array_equal(inter["slot_row"], slot_row)
    return n


@pytest.mark.parametrize("name", list(SMALL))
def test_small_layer_parity(name):
    inputs = _inputs(name)
    sh = inputs["shape"]
    print(f"[parity] small case {name}: {sh}", flush=True)
    layer = moe.DeviceLayer(inputs)
    out = layer.forward()
    torch.cuda.synchronize()
    g_idx, g_w, g_keys = run_route(layer)
    o_idx, o_w, keys64, near = check_routing(inputs, g_idx, g_w, g_keys)
    inter = _intermediates(layer)
    np.testing.assert_array_equal(inter["topk_w"], g_w)
    n = _check_permutation(sh, inter, g_idx)
    # the standalone permutation: same indices, x_perm rows bit-exact copies
    _check_standalone_permute(layer, inputs, inter, n)
    # per-expert MLP rows (the live rows only: rows past offsets[E_local] are never written)
    xd = oracle.bf16_to_f64(inputs["x"])
    segs = parity_util.expert_segments(sh, inter["counts"], inter["offsets"])
    parity_util.check_expert_rows(inputs, xd, segs, parity_util.live_y_rows(layer, segs), inter["row_token"])
    # layer output
    idx, w = oracle_routing_with_gpu_ties(o_idx, o_w, keys64, g_idx, near, sh)
    ref = oracle.expert_outputs_for_tokens(xd, idx, w, sh, inputs["w13"], inputs["w2"], inputs.get("ws13"),
                                           inputs.get("ws2"))
    got = oracle.bf16_to_f64(dev_bits(out))
    err = rel_fro(got, ref)
    print(f"[parity] {name}: rel_fro={err:.3e} near_ties={len(near)} local_rows={n}", flush=True)
    assert err <= REL_TOL


@pytest.mark.parametrize("name", ["tiny_T257", "group_limited_slice", "decode_small"])
def test_components_compose_to_layer(name):
    """route -> permute -> grouped_ffn (+ shared as one group over x) -> combine == layer, bit for bit."""
    inputs = _inputs(name)
    sh = inputs["shape"]
    layer = moe.DeviceLayer(inputs)
    ref = layer.forward().clone()
    dev = "cuda"
    T, k, cap = sh.T, sh.top_k, sh.capacity
    idx = torch.empty((T, k), dtype=torch.int32, device=dev)
    w = torch.empty((T, k), dtype=torch.float32, device=dev)
    moe.moe_route(sh, layer.x, layer.w_router, layer.bias, idx, w, None,
                  moe.alloc_workspace(sh, moe.MOE_WS_ROUTE))
    counts = torch.empty(sh.E_local, dtype=torch.int32, device=dev)
    offsets = torch.empty(sh.E_local + 1, dtype=torch.int32, device=dev)
    row_token = torch.empty(cap, dtype=torch.int32, device=dev)
    slot_row = torch.empty((T, k), dtype=torch.int32, device=dev)
    x_perm = torch.empty((cap, sh.d), dtype=torch.bfloat16, device=dev)
    moe.moe_permute(sh, idx, layer.x, counts, offsets, row_token, slot_row, x_perm,
                    moe.alloc_workspace(sh, moe.MOE_WS_PERMUTE))
    y_perm = torch.empty((cap, sh.d), dtype=torch.bfloat16, device=dev)
    moe.moe_grouped_ffn(sh, x_perm, offsets, layer.w13, layer.w2, y_perm, moe.alloc_workspace(sh, moe.MOE_WS_FFN))
    shared_y = None
    if sh.F_shared:
        ssh = sh.replace(E=1, top_k=1, e_begin=0, E_local=1, F=sh.F_shared, F_shared=0, n_group=1, topk_group=1)
        soff = torch.tensor([0, T], dtype=torch.int32, device=dev)
        shared_y = torch.empty((T, sh.d), dtype=torch.bfloat16, device=dev)
        moe.moe_grouped_ffn(ssh, layer.x, soff, layer.ws13, layer.ws2, shared_y,
                            moe.alloc_workspace(ssh, moe.MOE_WS_FFN))
    out = torch.empty((T, sh.d), dtype=torch.bfloat16, device=dev)
    moe.moe_combine(sh, y_perm, slot_row, w, shared_y, out)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(dev_bits(out), dev_bits(ref))


def test_metamorphic_determinism_scaling_and_token_order():
    inputs = _inputs("group_limited_slice")
    sh = inputs["shape"]
    layer = moe.DeviceLayer(inputs)
    a = dev_bits(layer.forward().clone())
    b = dev_bits(layer.forward().clone())
    np.testing.assert_array_equal(a, b)                           # run to run
    # doubling W2 and the shared W2 doubles every output exactly
    layer.w2.mul_(2)
    layer.ws2.mul_(2)
    c = oracle.bf16_to_f64(dev_bits(layer.forward().clone()))
    np.testing.assert_array_equal(c, 2 * oracle.bf16_to_f64(a))
    # permuting tokens permutes output rows bit for bit
    perm = np.random.default_rng(0).permutation(sh.T)
    inp2 = dict(inputs, x=inputs["x"][perm])
    layer2 = moe.DeviceLayer(inp2)
    d = dev_bits(layer2.forward())
    torch.cuda.synchronize()
    np.testing.assert_array_equal(d, a[perm])


def test_expert_relabel_invariance():
    inputs = _inputs("skewed_small")
    sh = inputs["shape"]
    a = dev_bits(moe.DeviceLayer(inputs).forward())
    pi = np.random.default_rng(1).permutation(sh.E)                # new id of old expert e is pi[e]
    inv = np.argsort(pi)
    inp2 = dict(inputs, w_router=inputs["w_router"][inv], bias=inputs["bias"][inv], w13=inputs["w13"][inv],
                w2=inputs["w2"][inv])
    b = dev_bits(moe.DeviceLayer(inp2).forward())
    torch.cuda.synchronize()
    np.testing.assert_array_equal(a, b)


def test_single_hot_expert():
    sh = S(T=700, d=192, E=8, top_k=2, F=128, E_local=8)
    inputs = wl.custom_inputs(sh, seed=5)
    bias = np.zeros(8, np.float32)
    bias[3] = 40.0                                                 # every token picks expert 3 first
    inputs["bias"] = bias
    layer = moe.DeviceLayer(inputs)
    out = layer.forward()
    torch.cuda.synchronize()
    inter = _intermediates(layer)
    assert inter["counts"][3] == sh.T and (inter["topk_idx"][:, 0] == 3).all()
    g_idx, g_w, g_keys = run_route(layer)
    o_idx, o_w, keys64, near = check_routing(inputs, g_idx, g_w, g_keys)
    _check_permutation(sh, inter, g_idx)
    idx, w = oracle_routing_with_gpu_ties(o_idx, o_w, keys64, g_idx, near, sh)
    ref = oracle.expert_outputs_for_tokens(oracle.bf16_to_f64(inputs["x"]), idx, w, sh, inputs["w13"],
                                           inputs["w2"])
    assert rel_fro(oracle.bf16_to_f64(dev_bits(out)), ref) <= REL_TOL


def test_zero_tokens_noop_on_device():
    sh = wl.WORKLOADS["tiny"].shape.replace(T=0)
    moe.moe_layer_forward(sh, None, None, None, None, None, None, None, None, None)


# ---------------------------------------------------------------------------------------
# full-size workloads, launch configuration of the benchmark
# ---------------------------------------------------------------------------------------
def full_layer_check(inputs, layer, out, label):
    """Routing (R1-R3) and the permutation on every token, every live y_perm row expert by
    expert, and the whole [T, d] output against the oracle.  Returns the printed summary."""
    sh = inputs["shape"]
    g_idx, g_w, g_keys = run_route(layer)
    xd = oracle.bf16_to_f64(inputs["x"])
    o_idx, o_w, keys64, near = check_routing(inputs, g_idx, g_w, g_keys, xd)
    inter = _intermediates(layer)
    np.testing.assert_array_equal(inter["topk_w"], g_w)
    C = sh.expert_capacity
    if C > 0:
        counts, offsets = oracle.counts_offsets(g_idx, sh.e_begin, sh.E_local, C)
        row_token, slot_row = oracle.permutation(g_idx, sh.e_begin, sh.E_local, C)
        np.testing.assert_array_equal(inter["topk_idx"], g_idx)
        np.testing.assert_array_equal(inter["counts"], counts)
        np.testing.assert_array_equal(inter["offsets"], offsets)
        np.testing.assert_array_equal(inter["slot_row"], slot_row)
        kept = row_token >= 0
        np.testing.assert_array_equal(inter["row_token"][kept], row_token[kept])
        n = int(kept.sum())
    else:
        n = _check_permutation(sh, inter, g_idx)
        _check_standalone_permute(layer, inputs, inter, n)
    segs = parity_util.expert_segments(sh, inter["counts"], inter["offsets"])
    rows = parity_util.live_y_rows(layer, segs)
    worst_e, err_rows = parity_util.check_expert_rows(inputs, xd, segs, rows, inter["row_token"])
    idx, w = oracle_routing_with_gpu_ties(o_idx, o_w, keys64, g_idx, near, sh)
    keep = oracle.keep_mask(idx, sh.e_begin, sh.E_local, C) if C > 0 else None
    ref = oracle.expert_outputs_for_tokens(xd, idx, w, sh, inputs["w13"], inputs["w2"], inputs.get("ws13"),
                                           inputs.get("ws2"), keep)
    got = oracle.bf16_to_f64(dev_bits(out))
    err = rel_fro(got, ref)
    # the worst 128-row block of tokens, so that one wrong tile is not diluted by the others
    blk = max(rel_fro(got[i:i + 128], ref[i:i + 128]) for i in range(0, sh.T, 128))
    cnt = inter["counts"]
    msg = (f"[parity] {label}: rel_fro={err:.3e} over all {sh.T} tokens (worst 128-token block {blk:.3e}), "
           f"y_perm rel_fro={err_rows:.3e} over {n} live rows (worst expert {worst_e:.3e}), "
           f"near_ties={len(near)}, counts min/median/max={cnt.min()}/{int(np.median(cnt))}/{cnt.max()}")
    print(msg, flush=True)
    assert err <= REL_TOL and blk <= 2 * REL_TOL
    return err


@pytest.mark.parametrize("name", list(wl.WORKLOADS))
def test_full_workload_parity(name):
    print(f"[parity] full workload {name}: generating inputs", flush=True)
    inputs = wl.make_inputs(name)
    layer = moe.DeviceLayer(inputs)
    out = layer.forward()
    torch.cuda.synchronize()
    print(f"[parity] {name}: layer ran, checking every token and every live row", flush=True)
    full_layer_check(inputs, layer, out, name)


@pytest.mark.parametrize("name,e_begin", [("dsv3", 224), ("k2decode", 336)])
def test_full_workload_last_rank(name, e_begin):
    """The full-size workload on the last expert-parallel rank's slice (DeepSeek-V3: experts
    224-255, the last routing group; Kimi-K2 decode: experts 336-383): every token and every live
    row against the oracle."""
    print(f"[parity] full workload {name}, experts from {e_begin}: generating inputs", flush=True)
    base = wl.make_inputs(name)
    inputs = dict(base, shape=base["shape"].replace(e_begin=e_begin))
    layer = moe.DeviceLayer(inputs)
    out = layer.forward()
    torch.cuda.synchronize()
    full_layer_check(inputs, layer, out, f"{name} e_begin={e_begin}")


@pytest.mark.parametrize("capacity", [2, 8, 64])
def test_k2decode_masked_layout_full(capacity):
    """The masked-decode layout at the Kimi-K2 decode shape (T = 64, 48 of 384 experts local,
    shared expert): C = 2 drops the slots ranked past 2 in the busier experts, C = 8 and C = T keep
    every slot of this batch."""
    print(f"[parity] k2decode masked C={capacity}: generating inputs", flush=True)
    base = wl.make_inputs("k2decode")
    inputs = dict(base, shape=base["shape"].replace(expert_capacity=capacity))
    layer = moe.DeviceLayer(inputs)
    out = layer.forward()
    torch.cuda.synchronize()
    full_layer_check(inputs, layer, out, f"k2decode masked C={capacity}")


@pytest.mark.parametrize("capacity", [240, 320])
def test_dsv3_masked_layout_full(capacity):
    """The masked-decode layout at the DeepSeek-V3 size (32 local experts with 230-293 slots each):
    C = 240 drops the slots ranked past 240 in most experts, C = 320 keeps every slot (its segments
    fill the 320-row tiles the launch uses)."""
    print(f"[parity] dsv3 masked C={capacity}: generating inputs", flush=True)
    base = wl.make_inputs("dsv3")
    inputs = dict(base, shape=base["shape"].replace(expert_capacity=capacity))
    layer = moe.DeviceLayer(inputs)
    out = layer.forward()
    torch.cuda.synchronize()
    full_layer_check(inputs, layer, out, f"dsv3 masked C={capacity}")


def test_grouped_ffn_ragged_tail_blocks():
    """moe_grouped_ffn on hand-picked segment lengths: the last m-tile of a segment holds every
    count of live 32-row blocks (1 .. 8, block edges +-1), plus empty segments, multi-tile
    segments and K tails in both GEMMs (d = 264, F = 136); each segment against the oracle."""
    lengths = [1, 0, 31, 32, 33, 63, 64, 65, 96, 127, 128, 129, 160, 191, 224, 255, 256, 0, 273, 612]
    E = len(lengths)
    T = int(sum(lengths))
    sh = S(T=T, d=264, E=E, top_k=1, F=136, E_local=E)
    rng = np.random.default_rng(2024)
    x = wl.f32_to_bf16_bits(rng.standard_normal((T, sh.d)).astype(np.float32))
    w13 = wl.f32_to_bf16_bits((rng.standard_normal((E, 2 * sh.F, sh.d)) * sh.d ** -0.5).astype(np.float32))
    w2 = wl.f32_to_bf16_bits((rng.standard_normal((E, sh.d, sh.F)) * sh.F ** -0.5).astype(np.float32))
    offs = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    dev = "cuda"
    y = torch.full((sh.capacity, sh.d), float("nan"), dtype=torch.bfloat16, device=dev)
    moe.moe_grouped_ffn(sh, moe.to_device_bf16(x), torch.from_numpy(offs).to(dev), moe.to_device_bf16(w13),
                        moe.to_device_bf16(w2), y, moe.alloc_workspace(sh, moe.MOE_WS_FFN))
    torch.cuda.synchronize()
    got = y.float().cpu().numpy()
    assert np.isfinite(got[:T]).all()
    xd = oracle.bf16_to_f64(x)
    for e in range(E):
        a, b = offs[e], offs[e + 1]
        if a == b:
            continue
        ref = oracle.swiglu_ffn(xd[a:b], oracle.bf16_to_f64(w13[e]), oracle.bf16_to_f64(w2[e]))
        err = rel_fro(got[a:b], ref)
        assert err <= REL_TOL, (e, lengths[e], err)


def test_grouped_ffn_more_rounds_than_the_tile_list():
    """moe_grouped_ffn with 1024 groups of 60..140 rows and d = 2048: the down-projection launch
    has more than 64 rounds of tiles per workgroup even at two workgroups per CU, so the tiles past
    a workgroup's 64-entry LDS tile list are decoded on the fly.  The first groups, a spread of
    middle ones and all of the last ones (whose tiles come last) against the oracle.  Inputs from
    torch's seeded GPU generator (0.6 G values); the checked groups are copied back for the oracle."""
    E, d, F = 1024, 2048, 64
    rng = np.random.default_rng(77)
    lengths = rng.integers(60, 141, size=E)
    T = int(lengths.sum())
    sh = S(T=T, d=d, E=E, top_k=1, F=F, E_local=E)
    # at most two workgroups per CU on 256 CUs, 64-row tiles, 128-wide output tiles
    tiles_down = int(sum((l + 63) // 64 for l in lengths)) * (d // 128)
    assert tiles_down > 64 * 512, tiles_down
    dev = "cuda"
    g = torch.Generator(device=dev).manual_seed(77)
    x = torch.randn(T, d, device=dev, generator=g).bfloat16()
    w13 = (torch.randn(E, 2 * F, d, device=dev, generator=g) * d ** -0.5).bfloat16()
    w2 = (torch.randn(E, d, F, device=dev, generator=g) * F ** -0.5).bfloat16()
    offs = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    y = torch.full((sh.capacity, d), float("nan"), dtype=torch.bfloat16, device=dev)
    moe.moe_grouped_ffn(sh, x, torch.from_numpy(offs).to(dev), w13, w2, y, moe.alloc_workspace(sh, moe.MOE_WS_FFN))
    torch.cuda.synchronize()
    assert bool(torch.isfinite(y[:T].float()).all())
    check = list(range(4)) + list(range(100, E - 64, 97)) + list(range(E - 64, E))
    worst = 0.0
    for e in check:
        a, b = int(offs[e]), int(offs[e + 1])
        ref = oracle.swiglu_ffn(oracle.bf16_to_f64(dev_bits(x[a:b])), oracle.bf16_to_f64(dev_bits(w13[e])),
                                oracle.bf16_to_f64(dev_bits(w2[e])))
        err = rel_fro(oracle.bf16_to_f64(dev_bits(y[a:b])), ref)
        worst = max(worst, err)
        assert err <= REL_TOL, (e, b - a, err)
    print(f"[parity] grouped_ffn {E} groups, {tiles_down} down-projection tiles: worst rel_fro {worst:.3e} "
          f"over {len(check)} groups", flush=True)


def test_library_loaded_before_torch():
    """The binding loaded before anything imported torch (a fresh process) still runs the layer:
    the library must bind to the HIP runtime torch uses, not to a second copy of it."""
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    code = ("import sys; sys.path.insert(0, %r)\n"
            "from paper_2607_18631_amd import moe\n"
            "moe.lib()\n"
            "import torch\n"
            "from paper_2607_18631_amd import workloads as wl\n"
            "layer = moe.DeviceLayer(wl.make_inputs('tiny'))\n"
            "out = layer.forward()\n"
            "torch.cuda.synchronize()\n"
            "assert bool(torch.isfinite(out.float()).all())\n"
            "print('ok')\n") % root
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), r.stdout[-2000:] + r.stderr[-2000:]
