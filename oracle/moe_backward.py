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

from .moe_oracle import bf16_to_f64


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
