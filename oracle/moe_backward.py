"""fp64 CPU oracle of the expert-MLP backward -- TEST INFRASTRUCTURE ONLY.

Only the test suite may import this module; the product path never calls it, and it
shares no code with the HIP kernels.

The paper's training leg (Section 4, engine registration) wraps the generated expert
kernels in an autograd function: the forward composes the expert MLP's two GEMMs, the
backward composes the dual GEMMs in transposed layout for the activation gradients and
per-expert products for the weight gradients.  For one expert with rows X [m, d],
w13 = [W1; W3] ([2F, d]), W2 [d, F] and the gradient dY [m, d] of its output

    H = X W1^T,  U = X W3^T,  A = silu(H) * U,  Y = A W2^T          (the forward)

the chain rule gives, with s = 1 / (1 + exp(-H)), silu(H) = H s and
silu'(H) = s (1 + H (1 - s)):

    dA   = dY W2                         [m, F]
    dW2  = dY^T A                        [d, F]
    dH   = dA * U * silu'(H)             [m, F]
    dU   = dA * silu(H)                  [m, F]
    dX   = dH W1 + dU W3 = [dH dU] w13   [m, d]
    dW13 = [dH dU]^T X                   [2F, d]

Each expert's rows are a segment of the expert-ordered row buffer: [offs[e], offs[e+1])
(monotone offsets) or [e C, e C + min(count_e, C)) (masked-decode layout).  An expert with
no rows has zero weight gradients.  Everything is float64.
"""
from __future__ import annotations

import numpy as np

from .moe_oracle import GATE_SOFTMAX, bf16_to_f64


def silu_grad(h: np.ndarray) -> np.ndarray:
    """d/dh of h / (1 + exp(-h))."""
    s = 1.0 / (1.0 + np.exp(-h))
    return s * (1.0 + h * (1.0 - s))


def swiglu_ffn_backward(xr, w13, w2, dy):
    """Gradients (dX, dW13, dW2) of one expert's SwiGLU MLP for output gradient dy."""
    xr = np.asarray(xr, np.float64)
    w13 = np.asarray(w13, np.float64)
    w2 = np.asarray(w2, np.float64)
    dy = np.asarray(dy, np.float64)
    F = w13.shape[0] // 2
    h = xr @ w13[:F].T
    u = xr @ w13[F:].T
    s = 1.0 / (1.0 + np.exp(-h))
    a = h * s * u
    da = dy @ w2
    dw2 = dy.T @ a
    dh = da * u * silu_grad(h)
    du = da * h * s
    dhu = np.concatenate([dh, du], axis=1)
    dx = dhu @ w13
    dw13 = dhu.T @ xr
    return dx, dw13, dw2


def expert_segments(offsets, E_local: int, expert_capacity: int = 0):
    """(start, stop) row range of every local expert: monotone offsets, or, in the
    masked-decode layout, offsets holds the per-expert counts and expert e owns
    [e C, e C + min(count_e, C))."""
    offsets = np.asarray(offsets, np.int64)
    if expert_capacity > 0:
        C = expert_capacity
        return [(e * C, e * C + int(min(max(offsets[e], 0), C))) for e in range(E_local)]
    return [(int(offsets[e]), int(offsets[e + 1])) for e in range(E_local)]


def grouped_ffn_backward(x_rows, offsets, w13_bits, w2_bits, dy_rows, E_local: int, expert_capacity: int = 0):
    """Per-expert backward over the expert-ordered rows.

    x_rows, dy_rows: float64 [cap, d]; w13_bits [E_local, 2F, d], w2_bits [E_local, d, F]
    (bf16 bit patterns).  Returns dX rows [cap, d] (rows outside every segment are 0),
    dW13 [E_local, 2F, d] and dW2 [E_local, d, F].
    """
    x_rows = np.asarray(x_rows, np.float64)
    dy_rows = np.asarray(dy_rows, np.float64)
    E2F, d = w13_bits.shape[1], w13_bits.shape[2]
    F = E2F // 2
    dx = np.zeros_like(x_rows)
    dw13 = np.zeros((E_local, 2 * F, d))
    dw2 = np.zeros((E_local, d, F))
    for e, (a, b) in enumerate(expert_segments(offsets, E_local, expert_capacity)):
        if b <= a:
            continue
        gx, g13, g2 = swiglu_ffn_backward(x_rows[a:b], bf16_to_f64(w13_bits[e]), bf16_to_f64(w2_bits[e]),
                                          dy_rows[a:b])
        dx[a:b] = gx
        dw13[e] = g13
        dw2[e] = g2
    return dx, dw13, dw2


# ----------------------------------------------------------------------------------------
# the whole layer (one rank's share): combine, expert MLPs, shared expert, gates, router
# ----------------------------------------------------------------------------------------
def gate_weights_backward(keys, topk_idx, dgate, gate: int, renormalize: int = 1, routed_scale: float = 1.0):
    """d loss / d key for every expert, given d loss / d gate of every chosen slot.

    The choice of experts is piecewise constant in the keys, so it carries no gradient; the
    gates are differentiated as the functions of the keys the forward evaluates (see
    ``gate_weights``): with s = routed_scale,
      softmax, renormalised:   w_j = s p_j,  p = softmax over the chosen keys
                               dkey_i = s p_i (dw_i - sum_j p_j dw_j)      (chosen i; 0 else)
      softmax, full:           w_j = s P_j,  P = softmax over all keys
                               dkey_i = s P_i ([i chosen] dw_i - sum_j P_j dw_j)
      sigmoid key, renorm.:    w_j = s k_j / S,  S = sum of the chosen keys
                               dkey_i = (s / S) (dw_i - sum_j (k_j / S) dw_j)  (chosen i)
      sigmoid key, raw:        w_j = s k_j,  dkey_i = s dw_i                  (chosen i)
    """
    keys = np.asarray(keys, np.float64)
    dgate = np.asarray(dgate, np.float64)
    T, E = keys.shape
    idx = np.asarray(topk_idx, np.int64)
    s = float(routed_scale)
    rows = np.arange(T)[:, None]
    dkey = np.zeros((T, E))
    sel = np.take_along_axis(keys, idx, axis=1)
    if gate == GATE_SOFTMAX:
        if renormalize:
            p = np.exp(sel - sel.max(axis=1, keepdims=True))
            p /= p.sum(axis=1, keepdims=True)
            inner = (p * dgate).sum(axis=1, keepdims=True)
            np.add.at(dkey, (rows, idx), s * p * (dgate - inner))
        else:
            P = np.exp(keys - keys.max(axis=1, keepdims=True))
            P /= P.sum(axis=1, keepdims=True)
            psel = np.take_along_axis(P, idx, axis=1)
            inner = (psel * dgate).sum(axis=1, keepdims=True)
            dkey = -s * P * inner
            np.add.at(dkey, (rows, idx), s * psel * dgate)
    else:                                                     # sigmoid scores as keys
        if renormalize:
            S = sel.sum(axis=1, keepdims=True)
            inner = ((sel / S) * dgate).sum(axis=1, keepdims=True)
            np.add.at(dkey, (rows, idx), (s / S) * (dgate - inner))
        else:
            np.add.at(dkey, (rows, idx), s * dgate)
    return dkey


def logits_backward(dkey, keys, gate: int):
    """d loss / d logit: the softmax key is the (biased) logit itself; the sigmoid key is
    sigma(L), whose derivative is k (1 - k)."""
    dkey = np.asarray(dkey, np.float64)
    if gate == GATE_SOFTMAX:
        return dkey
    k = np.asarray(keys, np.float64)
    return dkey * k * (1.0 - k)


def layer_backward(inputs: dict, dout, routing=None):
    """Gradients of the layer forward (``moe_oracle.layer_forward``) for output gradient dout.

    The routing decision is the forward's (``routing`` = (topk_idx, topk_w) overrides it,
    as for the forward).  Slots routed to other ranks or dropped by the capacity contribute
    nothing on this rank: their gate gradient is 0.  Returns dx [T, d], dw_router [E, d],
    dw13 / dw2 of the local experts, dws13 / dws2 of the shared expert (or None), the gate
    gradient dgate [T, k] and dlogits [T, E].
    """
    from . import moe_oracle as mo
    sh = inputs["shape"]
    xd = mo.bf16_to_f64(inputs["x"])
    wr = mo.bf16_to_f64(inputs["w_router"])
    dout = np.asarray(dout, np.float64)
    idx, w, keys = mo.route(xd, wr, sh, inputs.get("bias"))
    if routing is not None:
        idx, w = routing
    C = getattr(sh, "expert_capacity", 0)
    keep = mo.keep_mask(idx, sh.e_begin, sh.E_local, C)
    le = np.where(keep, mo.local_expert(idx, sh.e_begin, sh.E_local), -1)
    T, k = idx.shape
    F, d = sh.F, sh.d
    dx = np.zeros((T, d))
    dgate = np.zeros((T, k))
    dw13 = np.zeros((sh.E_local, 2 * F, d))
    dw2 = np.zeros((sh.E_local, d, F))
    for e in np.unique(le[le >= 0]):
        tok, slot = np.nonzero(le == e)
        w13e, w2e = mo.bf16_to_f64(inputs["w13"][e]), mo.bf16_to_f64(inputs["w2"][e])
        y = mo.swiglu_ffn(xd[tok], w13e, w2e)
        dgate[tok, slot] = (dout[tok] * y).sum(axis=1)
        gx, dw13[e], dw2[e] = swiglu_ffn_backward(xd[tok], w13e, w2e, w[tok, slot][:, None] * dout[tok])
        np.add.at(dx, tok, gx)
    dws13 = dws2 = None
    if sh.F_shared > 0:
        gx, dws13, dws2 = swiglu_ffn_backward(xd, mo.bf16_to_f64(inputs["ws13"]), mo.bf16_to_f64(inputs["ws2"]),
                                              dout)
        dx += gx
    dkey = gate_weights_backward(keys, idx, dgate, sh.gate, sh.renormalize, sh.routed_scale)
    dlogits = logits_backward(dkey, keys, sh.gate)
    dx += dlogits @ wr
    return {"dx": dx, "dw_router": dlogits.T @ xd, "dw13": dw13, "dw2": dw2, "dws13": dws13, "dws2": dws2,
            "dgate": dgate, "dlogits": dlogits}
