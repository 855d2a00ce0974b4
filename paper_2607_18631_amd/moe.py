"""Thin ctypes binding of libmoe_mi355x.so (include/moe.h), same names as the C ABI.

Argument marshalling only: every step of the layer runs in the library's HIP kernels.
Tensors are torch device tensors (torch provides device memory and streams); each call
passes their data pointers and the current torch stream.  If the library is not built,
``lib()`` raises -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from .workloads import MoEShape

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmoe_mi355x.so")

MOE_OK, MOE_ERR_INVALID_ARG, MOE_ERR_UNSUPPORTED, MOE_ERR_WORKSPACE, MOE_ERR_HIP = range(5)
MOE_WS_ROUTE, MOE_WS_PERMUTE, MOE_WS_FFN, MOE_WS_LAYER, MOE_WS_FFN_BWD, MOE_WS_LAYER_BWD = range(6)
MOE_FUSION_SET, MOE_FUSE_GATHER, MOE_FUSE_COMBINE = 0x10, 0x1, 0x2
(MOE_REGION_TOPK_IDX, MOE_REGION_TOPK_W, MOE_REGION_COUNTS, MOE_REGION_OFFSETS, MOE_REGION_ROW_TOKEN,
 MOE_REGION_SLOT_ROW, MOE_REGION_X_PERM, MOE_REGION_Y_PERM, MOE_REGION_SHARED_Y) = range(9)

EXPORTS = ["moe_abi_version", "moe_status_string", "moe_last_error", "moe_workspace_size",
           "moe_workspace_offset", "moe_route", "moe_permute", "moe_grouped_ffn", "moe_combine",
           "moe_layer_forward", "moe_layer_forward_traced", "moe_grouped_ffn_backward", "moe_layer_backward",
           "moe_permute_noalloc"]
MOE_STEP_NAMES = ["router_gemm", "gate", "histogram", "permute", "ffn_up", "ffn_down", "shared_up",
                  "shared_down", "combine"]


class MoEShapeC(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int64), ("d", ctypes.c_int32), ("E", ctypes.c_int32),
                ("top_k", ctypes.c_int32), ("e_begin", ctypes.c_int32), ("E_local", ctypes.c_int32),
                ("F", ctypes.c_int32), ("F_shared", ctypes.c_int32), ("gate", ctypes.c_int32),
                ("n_group", ctypes.c_int32), ("topk_group", ctypes.c_int32),
                ("renormalize", ctypes.c_int32), ("routed_scale", ctypes.c_float),
                ("expert_capacity", ctypes.c_int32), ("fusion", ctypes.c_int32)]


class MoEError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"status {status}: {message}")
        self.status = status


_lib = None
_vp = ctypes.c_void_p


def lib():
    """Load the built library (once).  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it first (python -m paper_2607_18631_amd.build)")
        # torch ships its own HIP runtime under the same soname (libamdhip64.so.7) as the system
        # one the library is linked against.  Loading torch first makes the library bind to that
        # runtime; loaded the other way round, the process holds two runtimes and the library's
        # kernels are not found for torch's device memory ("invalid device function").
        import torch  # noqa: F401
        L = ctypes.CDLL(LIB_PATH)
        sp = ctypes.POINTER(MoEShapeC)
        L.moe_abi_version.restype = ctypes.c_int
        L.moe_status_string.restype = ctypes.c_char_p
        L.moe_status_string.argtypes = [ctypes.c_int]
        L.moe_last_error.restype = ctypes.c_char_p
        L.moe_workspace_size.restype = ctypes.c_size_t
        L.moe_workspace_size.argtypes = [sp, ctypes.c_int]
        L.moe_workspace_offset.restype = ctypes.c_size_t
        L.moe_workspace_offset.argtypes = [sp, ctypes.c_int]
        L.moe_route.argtypes = [sp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp]
        L.moe_permute.argtypes = [sp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp]
        L.moe_grouped_ffn.argtypes = [sp, _vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp]
        L.moe_permute_noalloc.argtypes = [sp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp]
        L.moe_combine.argtypes = [sp, _vp, _vp, _vp, _vp, _vp, _vp]
        L.moe_grouped_ffn_backward.argtypes = [sp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_size_t,
                                               _vp]
        L.moe_layer_backward.argtypes = [sp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_size_t,
                                         _vp, _vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp]
        L.moe_layer_forward.argtypes = [sp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp]
        L.moe_layer_forward_traced.argtypes = [sp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_size_t,
                                               ctypes.POINTER(_vp), _vp]
        for f in ("moe_route", "moe_permute", "moe_grouped_ffn", "moe_combine", "moe_layer_forward",
                  "moe_layer_forward_traced", "moe_grouped_ffn_backward", "moe_layer_backward"):
            getattr(L, f).restype = ctypes.c_int
        _lib = L
    return _lib


def shape_c(sh: MoEShape) -> MoEShapeC:
    return MoEShapeC(sh.T, sh.d, sh.E, sh.top_k, sh.e_begin, sh.E_local, sh.F, sh.F_shared, sh.gate,
                     sh.n_group, sh.topk_group, sh.renormalize, sh.routed_scale, sh.expert_capacity,
                     sh.fusion)


def last_error() -> str:
    return lib().moe_last_error().decode()


def _check(status: int):
    if status != MOE_OK:
        raise MoEError(status, last_error())


def _p(t):
    """Data pointer of a tensor (or None)."""
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is not None:
        return ctypes.c_void_p(stream)
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def workspace_size(sh: MoEShape, kind: int) -> int:
    n = lib().moe_workspace_size(ctypes.byref(shape_c(sh)), kind)
    if n == 0:
        raise MoEError(MOE_ERR_INVALID_ARG, last_error())
    return n


def workspace_offset(sh: MoEShape, region: int) -> int:
    n = lib().moe_workspace_offset(ctypes.byref(shape_c(sh)), region)
    if n == ctypes.c_size_t(-1).value:
        raise MoEError(MOE_ERR_INVALID_ARG, last_error())
    return n


def alloc_workspace(sh: MoEShape, kind: int, device="cuda"):
    import torch
    return torch.empty(workspace_size(sh, kind), dtype=torch.uint8, device=device)


def moe_route(sh, x, w_router, bias, topk_idx, topk_w, keys_out=None, ws=None, stream=None):
    _check(lib().moe_route(ctypes.byref(shape_c(sh)), _p(x), _p(w_router), _p(bias), _p(topk_idx), _p(topk_w),
                           _p(keys_out), _p(ws), 0 if ws is None else ws.numel(), _stream(stream)))


def moe_permute(sh, topk_idx, x, counts, offsets, row_token, slot_row, x_perm, ws=None, stream=None):
    _check(lib().moe_permute(ctypes.byref(shape_c(sh)), _p(topk_idx), _p(x), _p(counts), _p(offsets),
                             _p(row_token), _p(slot_row), _p(x_perm), _p(ws), 0 if ws is None else ws.numel(),
                             _stream(stream)))


def moe_permute_noalloc(sh, topk_idx, x, counts, offsets, row_token, slot_row, x_perm, stream=None):
    _check(lib().moe_permute_noalloc(ctypes.byref(shape_c(sh)), _p(topk_idx), _p(x), _p(counts), _p(offsets),
                                     _p(row_token), _p(slot_row), _p(x_perm), _stream(stream)))


def moe_grouped_ffn(sh, x_perm, offsets, w13, w2, y_perm, ws=None, stream=None):
    _check(lib().moe_grouped_ffn(ctypes.byref(shape_c(sh)), _p(x_perm), _p(offsets), _p(w13), _p(w2), _p(y_perm),
                                 _p(ws), 0 if ws is None else ws.numel(), _stream(stream)))


def moe_grouped_ffn_backward(sh, x_perm, offsets, w13, w2, dy_perm, dx_perm, dw13, dw2, ws=None, stream=None):
    _check(lib().moe_grouped_ffn_backward(ctypes.byref(shape_c(sh)), _p(x_perm), _p(offsets), _p(w13), _p(w2),
                                          _p(dy_perm), _p(dx_perm), _p(dw13), _p(dw2), _p(ws),
                                          0 if ws is None else ws.numel(), _stream(stream)))


def moe_layer_backward(sh, x, w_router, bias, w13, w2, ws13, ws2, dout, fwd_ws, dx, dw_router, dw13, dw2, dws13,
                       dws2, ws, stream=None):
    _check(lib().moe_layer_backward(ctypes.byref(shape_c(sh)), _p(x), _p(w_router), _p(bias), _p(w13), _p(w2),
                                    _p(ws13), _p(ws2), _p(dout), _p(fwd_ws), 0 if fwd_ws is None else fwd_ws.numel(),
                                    _p(dx), _p(dw_router), _p(dw13), _p(dw2), _p(dws13), _p(dws2), _p(ws),
                                    0 if ws is None else ws.numel(), _stream(stream)))


def moe_combine(sh, y_perm, slot_row, topk_w, shared_y, out, stream=None):
    _check(lib().moe_combine(ctypes.byref(shape_c(sh)), _p(y_perm), _p(slot_row), _p(topk_w), _p(shared_y),
                             _p(out), _stream(stream)))


def moe_layer_forward(sh, x, w_router, bias, w13, w2, ws13, ws2, out, ws, stream=None):
    _check(lib().moe_layer_forward(ctypes.byref(shape_c(sh)), _p(x), _p(w_router), _p(bias), _p(w13), _p(w2),
                                   _p(ws13), _p(ws2), _p(out), _p(ws), 0 if ws is None else ws.numel(),
                                   _stream(stream)))


def moe_layer_forward_traced(sh, x, w_router, bias, w13, w2, ws13, ws2, out, ws, events, stream=None):
    """``events``: ctypes array of len(MOE_STEP_NAMES) + 1 hipEvent_t handles (or None); a NULL
    entry is not recorded."""
    _check(lib().moe_layer_forward_traced(ctypes.byref(shape_c(sh)), _p(x), _p(w_router), _p(bias), _p(w13),
                                          _p(w2), _p(ws13), _p(ws2), _p(out), _p(ws),
                                          0 if ws is None else ws.numel(), events, _stream(stream)))


# ---------------------------------------------------------------------------------------
# device placement helpers (torch is plumbing: memory and streams)
# ---------------------------------------------------------------------------------------
def to_device_bf16(bits: np.ndarray, device="cuda"):
    """uint16 bf16 bit patterns -> torch.bfloat16 device tensor (bit-exact)."""
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(device).view(torch.bfloat16)


def bf16_bits(t) -> np.ndarray:
    """torch.bfloat16 tensor -> uint16 bit patterns on the host."""
    import torch
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


class DeviceLayer:
    """Inputs of one workload resident on the GPU, with a layer workspace.

    ``forward()`` runs ``moe_layer_forward``; ``region(...)`` views the intermediates
    it left in the workspace (routing, permutation, permuted rows).
    """

    def __init__(self, inputs: dict, device="cuda"):
        import torch
        self.shape = sh = inputs["shape"]
        self.device = device
        self.x = to_device_bf16(inputs["x"], device)
        self.w_router = to_device_bf16(inputs["w_router"], device)
        self.bias = None if inputs.get("bias") is None else torch.from_numpy(inputs["bias"]).to(device)
        self.w13 = to_device_bf16(inputs["w13"], device)
        self.w2 = to_device_bf16(inputs["w2"], device)
        self.ws13 = to_device_bf16(inputs["ws13"], device) if sh.F_shared > 0 else None
        self.ws2 = to_device_bf16(inputs["ws2"], device) if sh.F_shared > 0 else None
        self.out = torch.empty((sh.T, sh.d), dtype=torch.bfloat16, device=device)
        self.ws = alloc_workspace(sh, MOE_WS_LAYER, device)

    def forward(self, stream=None):
        moe_layer_forward(self.shape, self.x, self.w_router, self.bias, self.w13, self.w2, self.ws13, self.ws2,
                          self.out, self.ws, stream)
        return self.out

    def forward_traced(self, events, stream=None):
        moe_layer_forward_traced(self.shape, self.x, self.w_router, self.bias, self.w13, self.w2, self.ws13,
                                 self.ws2, self.out, self.ws, events, stream)
        return self.out

    def backward(self, dout, stream=None):
        """``moe_layer_backward`` for output gradient ``dout`` of the last ``forward()``; returns
        the gradients as a dict of device tensors (dx, dw_router, dw13, dw2, dws13, dws2)."""
        import torch
        sh = self.shape
        dev = self.device
        bf = torch.bfloat16
        g = {"dx": torch.empty((sh.T, sh.d), dtype=bf, device=dev),
             "dw_router": torch.empty((sh.E, sh.d), dtype=bf, device=dev),
             "dw13": torch.empty((sh.E_local, 2 * sh.F, sh.d), dtype=bf, device=dev),
             "dw2": torch.empty((sh.E_local, sh.d, sh.F), dtype=bf, device=dev),
             "dws13": torch.empty((2 * sh.F_shared, sh.d), dtype=bf, device=dev) if sh.F_shared > 0 else None,
             "dws2": torch.empty((sh.d, sh.F_shared), dtype=bf, device=dev) if sh.F_shared > 0 else None}
        if getattr(self, "ws_bwd", None) is None:
            self.ws_bwd = alloc_workspace(sh, MOE_WS_LAYER_BWD, dev)
        moe_layer_backward(sh, self.x, self.w_router, self.bias, self.w13, self.w2, self.ws13, self.ws2, dout,
                           self.ws, g["dx"], g["dw_router"], g["dw13"], g["dw2"], g["dws13"], g["dws2"],
                           self.ws_bwd, stream)
        return g

    def region(self, region: int, dtype, shape):
        import torch
        off = workspace_offset(self.shape, region)
        nbytes = int(np.prod(shape)) * torch.empty((), dtype=dtype).element_size()
        return self.ws[off:off + nbytes].view(dtype).view(*shape)
