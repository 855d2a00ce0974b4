"""moe_permute_noalloc (scratch in the library's fixed device array, no workspace argument)
against moe_permute (caller workspace), through the C ABI: two calls in a row on the same
GPU, the second on a smaller batch, every output bit for bit (counts, offsets, the live
rows of row_token, slot_row and the live rows of x_perm), in both row layouts."""
import numpy as np
import pytest
import torch

from paper_2607_18631_amd import moe
from paper_2607_18631_amd import workloads as wl

pytestmark = pytest.mark.gpu

S = wl.MoEShape


def _route(sh, seed):
    inputs = wl.custom_inputs(sh, seed=seed, router_std=2 * sh.d ** -0.5, zipf_s=1.1)
    dev = "cuda"
    x = moe.to_device_bf16(inputs["x"], dev)
    wr = moe.to_device_bf16(inputs["w_router"], dev)
    bias = torch.from_numpy(inputs["bias"]).to(dev)
    idx = torch.empty((sh.T, sh.top_k), dtype=torch.int32, device=dev)
    w = torch.empty((sh.T, sh.top_k), dtype=torch.float32, device=dev)
    moe.moe_route(sh, x, wr, bias, idx, w, None, moe.alloc_workspace(sh, moe.MOE_WS_ROUTE))
    return x, idx


def _outputs(sh, dev="cuda"):
    cap = sh.capacity
    return {"counts": torch.full((sh.E_local,), -7, dtype=torch.int32, device=dev),
            "offsets": torch.full((sh.E_local + 1,), -7, dtype=torch.int32, device=dev),
            "row_token": torch.full((cap,), -7, dtype=torch.int32, device=dev),
            "slot_row": torch.full((sh.T, sh.top_k), -7, dtype=torch.int32, device=dev),
            "x_perm": torch.zeros((cap, sh.d), dtype=torch.bfloat16, device=dev)}


def _live(sh, o):
    counts = o["counts"].cpu().numpy()
    offsets = o["offsets"].cpu().numpy()
    slot_row = o["slot_row"].cpu().numpy()
    rows = np.unique(slot_row[slot_row >= 0])
    return {"counts": counts, "offsets": offsets, "slot_row": slot_row,
            "row_token": o["row_token"].cpu().numpy()[rows], "x_perm": moe.bf16_bits(o["x_perm"])[rows]}


@pytest.mark.parametrize("capacity", [0, 5])
def test_permute_noalloc_matches_workspace_call(capacity):
    big = S(T=3000, d=264, E=64, top_k=6, F=64, E_local=48, e_begin=8, expert_capacity=capacity)
    small = S(T=130, d=264, E=64, top_k=6, F=64, E_local=40, e_begin=16, expert_capacity=capacity)
    for i, sh in enumerate((big, small)):
        print(f"[noalloc] call {i}: {sh}", flush=True)
        x, idx = _route(sh, seed=31 + i)
        ref = _outputs(sh)
        moe.moe_permute(sh, idx, x, ref["counts"], ref["offsets"], ref["row_token"], ref["slot_row"],
                        ref["x_perm"], moe.alloc_workspace(sh, moe.MOE_WS_PERMUTE))
        got = _outputs(sh)
        moe.moe_permute_noalloc(sh, idx, x, got["counts"], got["offsets"], got["row_token"], got["slot_row"],
                                got["x_perm"])
        torch.cuda.synchronize()
        a, b = _live(sh, ref), _live(sh, got)
        assert a["slot_row"].max() >= 0
        for k in a:
            np.testing.assert_array_equal(b[k], a[k], err_msg=f"call {i}: {k}")
        print(f"[noalloc] call {i}: {int((a['slot_row'] >= 0).sum())} rows bit-identical", flush=True)
