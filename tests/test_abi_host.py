"""C-ABI checks that need no GPU: the library loads, exports every declared symbol, sizes
workspaces, and rejects invalid calls on the host with the right status and a verbatim
reason -- before any HIP call.  (No valid compute call is made here: pointers passed are
never dereferenced because every call below fails validation first.)"""
import ctypes
import os
import re

import pytest

from paper_2607_18631_amd import moe
from paper_2607_18631_amd import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "moe.h")

FAKE = ctypes.c_void_p(0x100000)        # aligned, never dereferenced (validation fails first)
MISALIGNED = ctypes.c_void_p(0x100002)


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(moe_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    L = moe.lib()
    names = _declared()
    assert set(names) == set(moe.EXPORTS), names
    for n in names:
        assert hasattr(L, n), n
    assert L.moe_abi_version() == 5


def test_status_strings():
    L = moe.lib()
    for s in range(5):
        assert L.moe_status_string(s).decode().startswith(
            ["MOE_OK", "MOE_ERR_INVALID_ARG", "MOE_ERR_UNSUPPORTED", "MOE_ERR_WORKSPACE", "MOE_ERR_HIP"][s])


def test_explicit_gather_fold_beyond_offset_range_is_rejected():
    sh = BASE.replace(T=2 ** 22, d=1024, fusion=wl.FUSION_VARIANTS["gather"])
    st, msg = _layer_call(sh)
    assert st == moe.MOE_ERR_UNSUPPORTED and "MOE_FUSE_GATHER" in msg, (st, msg)
    # the default structure copies the rows instead (passes validation up to the workspace)
    st, msg = _layer_call(sh.replace(fusion=0))
    assert st == moe.MOE_ERR_WORKSPACE, (st, msg)


def test_fused_combine_workspace():
    """The folded combine adds a float32 [T, d] accumulator and a gate per row."""
    base = moe.workspace_size(BASE, moe.MOE_WS_LAYER)
    fused = moe.workspace_size(BASE.replace(fusion=wl.FUSION_VARIANTS["both"]), moe.MOE_WS_LAYER)
    assert fused >= base + BASE.T * BASE.d * 4 + BASE.capacity * 4
    assert moe.workspace_size(BASE.replace(fusion=wl.FUSION_VARIANTS["gather"]), moe.MOE_WS_LAYER) == base


def test_masked_layout_workspace():
    """The masked-decode layout sizes the permuted buffers by E_local * C rows."""
    C = 5
    sh = BASE.replace(expert_capacity=C)
    cap = sh.E_local * C
    assert sh.capacity == cap
    off = [moe.workspace_offset(sh, r) for r in range(9)]
    assert off[moe.MOE_REGION_X_PERM] - off[moe.MOE_REGION_ROW_TOKEN] >= cap * 4
    assert off[moe.MOE_REGION_Y_PERM] - off[moe.MOE_REGION_X_PERM] >= cap * sh.d * 2
    assert moe.workspace_size(sh, moe.MOE_WS_FFN) >= cap * sh.F * 2


@pytest.mark.parametrize("name", list(wl.WORKLOADS))
def test_workspace_sizes(name):
    sh = wl.WORKLOADS[name].shape
    for kind in range(6):
        n = moe.workspace_size(sh, kind)
        assert n > 0 and n % 256 == 0
    layer = moe.workspace_size(sh, moe.MOE_WS_LAYER)
    cap, d = sh.capacity, sh.d
    assert layer >= 2 * cap * d * 2 + cap * sh.F * 2          # x_perm, y_perm, activation
    offs = [moe.workspace_offset(sh, r) for r in range(9)]
    sizes = [sh.T * sh.top_k * 4, sh.T * sh.top_k * 4, sh.E_local * 4, (sh.E_local + 1) * 4, cap * 4,
             sh.T * sh.top_k * 4, cap * d * 2, cap * d * 2, sh.T * d * 2 if sh.F_shared else 0]
    for i in range(8):
        assert offs[i] % 256 == 0 and offs[i] + sizes[i] <= offs[i + 1]
    assert offs[8] + sizes[8] <= layer


def _status(fn, *args):
    st = fn(*args)
    return st, moe.last_error()


def _layer_call(sh, x=FAKE, wr=FAKE, bias=None, w13=FAKE, w2=FAKE, ws13=None, ws2=None, out=FAKE, ws=FAKE,
                ws_bytes=0):
    return _status(moe.lib().moe_layer_forward, ctypes.byref(moe.shape_c(sh)) if sh is not None else None,
                   x, wr, bias, w13, w2, ws13, ws2, out, ws, ws_bytes, None)


BASE = wl.MoEShape(T=64, d=64, E=8, top_k=2, F=64, E_local=8)


@pytest.mark.parametrize("sh,status,needle", [
    (BASE.replace(d=60), moe.MOE_ERR_UNSUPPORTED, "d (60) % 8 != 0"),
    (BASE.replace(F=12), moe.MOE_ERR_UNSUPPORTED, "F (12) % 8 != 0"),
    (BASE.replace(F_shared=-8), moe.MOE_ERR_INVALID_ARG, "F_shared (-8) < 0"),
    (BASE.replace(E=2000), moe.MOE_ERR_UNSUPPORTED, "E (2000) outside [1, 1024]"),
    (BASE.replace(top_k=9), moe.MOE_ERR_UNSUPPORTED, "top_k (9)"),
    (BASE.replace(E=64, top_k=17), moe.MOE_ERR_UNSUPPORTED, "top_k (17)"),
    (BASE.replace(e_begin=4, E_local=5), moe.MOE_ERR_INVALID_ARG, "local slice"),
    (BASE.replace(E_local=0), moe.MOE_ERR_INVALID_ARG, "local slice"),
    (BASE.replace(n_group=3), moe.MOE_ERR_INVALID_ARG, "E (8) % n_group (3) != 0"),
    (BASE.replace(n_group=8, topk_group=4), moe.MOE_ERR_INVALID_ARG, "group size"),
    (BASE.replace(n_group=4, topk_group=5), moe.MOE_ERR_INVALID_ARG, "topk_group (5)"),
    (BASE.replace(E=16, top_k=6, n_group=4, topk_group=1), moe.MOE_ERR_INVALID_ARG, "< top_k (6)"),
    (BASE.replace(gate=7), moe.MOE_ERR_UNSUPPORTED, "gate (7)"),
    (BASE.replace(renormalize=2), moe.MOE_ERR_INVALID_ARG, "renormalize (2)"),
    (BASE.replace(routed_scale=float("nan")), moe.MOE_ERR_INVALID_ARG, "routed_scale"),
    (BASE.replace(T=-1), moe.MOE_ERR_INVALID_ARG, "T (-1) < 0"),
    (BASE.replace(T=2 ** 30, top_k=2), moe.MOE_ERR_UNSUPPORTED, "T * top_k"),
    (BASE.replace(expert_capacity=-1), moe.MOE_ERR_INVALID_ARG, "expert_capacity (-1) < 0"),
    (BASE.replace(expert_capacity=2 ** 28), moe.MOE_ERR_UNSUPPORTED, "E_local * expert_capacity"),
    (BASE.replace(fusion=wl.FUSE_COMBINE), moe.MOE_ERR_INVALID_ARG, "fusion (0x2)"),
    (BASE.replace(fusion=wl.FUSION_SET | 0x4), moe.MOE_ERR_INVALID_ARG, "fusion (0x14)"),
])
def test_shape_validation(sh, status, needle):
    st, msg = _layer_call(sh)
    assert st == status and needle in msg, (st, msg)
    assert moe.lib().moe_workspace_size(ctypes.byref(moe.shape_c(sh)), moe.MOE_WS_LAYER) == 0


def test_null_shape():
    st, msg = _layer_call(None)
    assert st == moe.MOE_ERR_INVALID_ARG and "shape is NULL" in msg


def test_pointer_and_workspace_validation():
    need = moe.workspace_size(BASE, moe.MOE_WS_LAYER)
    st, msg = _layer_call(BASE, x=None)
    assert st == moe.MOE_ERR_INVALID_ARG and "x is NULL" in msg
    st, msg = _layer_call(BASE, w13=MISALIGNED)
    assert st == moe.MOE_ERR_INVALID_ARG and "w13" in msg and "16-byte aligned" in msg
    st, msg = _layer_call(BASE, out=None)
    assert st == moe.MOE_ERR_INVALID_ARG and "out is NULL" in msg
    st, msg = _layer_call(BASE, ws=None, ws_bytes=need)
    assert st == moe.MOE_ERR_WORKSPACE and "workspace is NULL" in msg
    st, msg = _layer_call(BASE, ws_bytes=need - 1)
    assert st == moe.MOE_ERR_WORKSPACE and f"required ({need})" in msg
    sh = BASE.replace(F_shared=64)
    st, msg = _layer_call(sh, ws_bytes=10 ** 12)
    assert st == moe.MOE_ERR_INVALID_ARG and "ws13 is NULL" in msg
    sig = BASE.replace(gate=wl.GATE_SIGMOID)
    st, msg = _layer_call(sig, bias=FAKE)
    assert st == moe.MOE_ERR_UNSUPPORTED and "bias" in msg


def test_component_validation():
    L = moe.lib()
    sp = ctypes.byref(moe.shape_c(BASE))
    assert L.moe_route(sp, FAKE, FAKE, None, None, FAKE, None, FAKE, 1 << 40, None) == moe.MOE_ERR_INVALID_ARG
    assert "topk_idx is NULL" in moe.last_error()
    assert L.moe_route(sp, FAKE, FAKE, None, FAKE, FAKE, None, FAKE, 16, None) == moe.MOE_ERR_WORKSPACE
    assert L.moe_permute(sp, FAKE, FAKE, FAKE, FAKE, FAKE, MISALIGNED, FAKE, FAKE, 1 << 40,
                         None) == moe.MOE_ERR_INVALID_ARG
    assert "slot_row" in moe.last_error()
    assert L.moe_grouped_ffn(sp, FAKE, None, FAKE, FAKE, FAKE, FAKE, 1 << 40, None) == moe.MOE_ERR_INVALID_ARG
    assert "offsets is NULL" in moe.last_error()
    assert L.moe_combine(sp, FAKE, FAKE, FAKE, MISALIGNED, FAKE, None) == moe.MOE_ERR_INVALID_ARG
    assert "shared_y" in moe.last_error()


def test_zero_tokens_is_a_noop():
    # T = 0 returns before any pointer is looked at or any HIP call is made
    sh = BASE.replace(T=0)
    st, msg = _layer_call(sh, x=None, wr=None, w13=None, w2=None, out=None, ws=None)
    assert st == moe.MOE_OK and msg == ""


def _bwd_call(sh, dout=FAKE, fwd_ws=FAKE, fwd_bytes=1 << 44, dx=FAKE, dwr=FAKE, dw13=FAKE, dw2=FAKE, dws13=None,
              dws2=None, ws=FAKE, ws_bytes=1 << 44, bias=None):
    return _status(moe.lib().moe_layer_backward, ctypes.byref(moe.shape_c(sh)), FAKE, FAKE, bias, FAKE, FAKE,
                   FAKE if sh.F_shared else None, FAKE if sh.F_shared else None, dout, fwd_ws, fwd_bytes, dx, dwr,
                   dw13, dw2, dws13, dws2, ws, ws_bytes, None)


def test_layer_backward_workspace():
    """Gradient rows of the experts (cap x d, twice), the router and shared rows (T x d),
    dlogits (T x E bf16), gate gradients and the expert-MLP backward's intermediates."""
    for name in wl.WORKLOADS:
        sh = wl.WORKLOADS[name].shape
        need = moe.workspace_size(sh, moe.MOE_WS_LAYER_BWD)
        cap, T, d = sh.capacity, sh.T, sh.d
        low = 2 * cap * d * 2 + T * d * 2 * (2 if sh.F_shared else 1) + T * sh.E * 2 + T * sh.top_k * 4
        low += max(4 * cap * sh.F * 2, 4 * T * sh.F_shared * 2)
        assert need % 256 == 0 and need >= low, (name, need, low)


@pytest.mark.parametrize("kw,status,needle", [
    (dict(fusion=wl.FUSION_VARIANTS["both"]), moe.MOE_ERR_UNSUPPORTED, "MOE_FUSE_COMBINE"),
    (dict(E=12, E_local=12), moe.MOE_ERR_UNSUPPORTED, "E (12) % 8 != 0"),
    (dict(F=12), moe.MOE_ERR_UNSUPPORTED, "F (12) % 8 != 0"),
])
def test_layer_backward_shape_validation(kw, status, needle):
    st, msg = _bwd_call(BASE.replace(**kw))
    assert st == status and needle in msg, (st, msg)


def test_layer_backward_pointer_and_workspace_validation():
    st, msg = _bwd_call(BASE, dout=None)
    assert st == moe.MOE_ERR_INVALID_ARG and "dout is NULL" in msg
    st, msg = _bwd_call(BASE, dwr=MISALIGNED)
    assert st == moe.MOE_ERR_INVALID_ARG and "dw_router" in msg
    st, msg = _bwd_call(BASE.replace(F_shared=64))
    assert st == moe.MOE_ERR_INVALID_ARG and "dws13 is NULL" in msg
    need_f = moe.workspace_size(BASE, moe.MOE_WS_LAYER)
    st, msg = _bwd_call(BASE, fwd_bytes=need_f - 1)
    assert st == moe.MOE_ERR_WORKSPACE and f"required ({need_f})" in msg
    need_b = moe.workspace_size(BASE, moe.MOE_WS_LAYER_BWD)
    st, msg = _bwd_call(BASE, ws_bytes=need_b - 1)
    assert st == moe.MOE_ERR_WORKSPACE and f"required ({need_b})" in msg
    st, msg = _bwd_call(BASE.replace(gate=wl.GATE_SIGMOID), bias=FAKE)
    assert st == moe.MOE_ERR_UNSUPPORTED and "bias" in msg


def test_permute_noalloc_validation():
    """The allocation-free permutation validates on the host like moe_permute, and rejects a
    request whose scratch would not fit its fixed 1 MiB device array (no HIP call is made)."""
    L = moe.lib()
    sp = ctypes.byref(moe.shape_c(BASE))
    assert L.moe_permute_noalloc(sp, FAKE, FAKE, FAKE, FAKE, FAKE, MISALIGNED, FAKE, None) == moe.MOE_ERR_INVALID_ARG
    assert "slot_row" in moe.last_error()
    assert L.moe_permute_noalloc(sp, None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None) == moe.MOE_ERR_INVALID_ARG
    assert "topk_idx is NULL" in moe.last_error()
    # per 64-token chunk and local expert a lane mask and a base (12 bytes): T = 2^16 tokens over
    # 128 local experts needs 1.5 MiB
    big = BASE.replace(T=2 ** 16, E=128, E_local=128, top_k=8)
    assert moe.workspace_size(big, moe.MOE_WS_PERMUTE) > 1 << 20
    assert L.moe_permute_noalloc(ctypes.byref(moe.shape_c(big)), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                                 None) == moe.MOE_ERR_UNSUPPORTED
    assert "scratch" in moe.last_error() and "1048576" in moe.last_error()
    # the largest DeepSeek-V3 and skewed batches fit
    for name in ("dsv3", "skewed", "mixtral", "k2decode"):
        assert moe.workspace_size(wl.WORKLOADS[name].shape, moe.MOE_WS_PERMUTE) <= 1 << 20
    # T = 0 is a no-op before any pointer is looked at
    z = ctypes.byref(moe.shape_c(BASE.replace(T=0)))
    assert L.moe_permute_noalloc(z, None, None, None, None, None, None, None, None) == moe.MOE_OK


def test_missing_library_fails_loudly():
    """With the HIP library absent the binding raises: there is no other path to fall back to.
    Run in a fresh process so this process's loaded library is untouched."""
    import subprocess
    import sys
    code = ("from paper_2607_18631_amd import moe\n"
            "moe.LIB_PATH = '/nonexistent/libmoe_mi355x.so'\n"
            "try:\n"
            "    moe.lib()\n"
            "except RuntimeError as e:\n"
            "    print('raised:', e)\n"
            "    raise SystemExit(0)\n"
            "raise SystemExit(3)\n")
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, (r.returncode, r.stdout, r.stderr)
    assert "is missing" in r.stdout
