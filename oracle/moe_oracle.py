"""fp64 CPU oracle of the MoE-layer forward -- TEST INFRASTRUCTURE ONLY.

Only the test suite, the package smoke check and the benchmark's CPU-baseline leg
may import this module.  The product path never calls it, and it shares no code
with the HIP kernels (it reads the same seeded bf16 bit patterns, nothing else).

What it computes (one MoE layer on one expert-parallel rank):

  1. router logits        L[t, e] = sum_i x[t, i] * Wr[e, i]
  2. gating keys          softmax mode: key = L + bias (bias inside the softmax);
                          sigmoid mode: key = s = 1 / (1 + exp(-L))
  3. group limit          (n_group > 1) experts split into n_group contiguous groups;
                          group score = sum of the two largest keys in the group;
                          the topk_group best groups stay eligible
  4. top-k                the top_k largest eligible keys, slot order = key
                          descending, ties to the lower expert (group) index
  5. gates                softmax: exp(key_j - m) / sum over chosen (renormalised)
                          or over all experts (not renormalised);
                          sigmoid: s_j / sum over chosen (renormalised) or s_j,
                          times routed_scale
  6. local slice          experts [e_begin, e_begin + E_local); other slots dropped
  7. counts / offsets     per-local-expert histogram and its exclusive scan, the
                          monotone [E_local + 1] row-offset array of the paper's
                          kernel-generation section (expert e owns rows
                          [offs[e], offs[e + 1]))
  8. permutation          rows grouped by expert, ascending token inside an expert;
                          masked-decode layout (expert_capacity C > 0, the equal-stride
                          capacity segments of the kernel-generation section): expert e
                          owns rows [e C, e C + min(count_e, C)); a slot whose rank
                          inside its expert (ascending token) is >= C is dropped
  9. expert FFN (SwiGLU)  y = W2_e (silu(W1_e x) * (W3_e x)); the forward composes
                          the two GEMMs of the expert MLP (Section 4, kernel
                          generation / engine registration)
 10. shared expert        the same SwiGLU on every token, weight 1
 11. combine              out[t] = sum_j w[t, j] * y[t, j] + y_shared[t]

The paper states the layer only in prose (Section 2 background: tokens routed to a
small subset of experts; Section 3.1 IR: permute folded into the grouped-GEMM
prologue, weighted combine folded into the epilogue; Section 4 kernel generation:
the [E+1] offsets).  The gating formulas (2-5), the SwiGLU form (9) and the
shared-expert rule (10) are the layer definitions the workloads are stated with;
every reading taken where the paper is silent is listed in the design notes.

Everything is float64 unless a function says otherwise.  ``decide_topk`` can also
run in float32 so that a decision taken by the GPU on its own float32 keys can be
replayed exactly (group sums as single IEEE float32 additions).
"""
from __future__ import annotations

import numpy as np

GATE_SOFTMAX = 0
GATE_SIGMOID = 1


# ----------------------------------------------------------------------------------------
# bf16 decoding
# ----------------------------------------------------------------------------------------
def bf16_to_f64(bits) -> np.ndarray:
    """Exact value of bf16 bit patterns: a bf16 is the upper half of an IEEE binary32."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


# ----------------------------------------------------------------------------------------
# routing
# ----------------------------------------------------------------------------------------
def router_logits(x: np.ndarray, w_router: np.ndarray) -> np.ndarray:
    """L[t, e] = sum_i x[t, i] * Wr[e, i]   (x: [T, d], Wr: [E, d])."""
    return np.asarray(x, np.float64) @ np.asarray(w_router, np.float64).T


def gating_keys(logits: np.ndarray, gate: int, bias=None) -> np.ndarray:
    """The per-expert key the selection is taken on.

    softmax: the biased logit (softmax is monotone, so the largest probabilities are
    the largest keys); sigmoid: the sigmoid score itself (group scores add scores).
    """
    L = np.asarray(logits, np.float64)
    if gate == GATE_SOFTMAX:
        return L if bias is None else L + np.asarray(bias, np.float64)[None, :]
    if gate == GATE_SIGMOID:
        if bias is not None:
            raise ValueError("sigmoid gating takes no router bias")
        return 1.0 / (1.0 + np.exp(-L))
    raise ValueError(f"unknown gate {gate}")


def _order_desc(vals: np.ndarray, eligible: np.ndarray) -> np.ndarray:
    """Indices of each row ordered: eligible first, then key descending, then index ascending."""
    T, n = vals.shape
    idx = np.broadcast_to(np.arange(n), (T, n))
    # np.lexsort sorts by the last key first
    return np.lexsort((idx, -vals, ~eligible), axis=1)


def group_scores(keys: np.ndarray, n_group: int) -> np.ndarray:
    """Score of each contiguous expert group: the sum of its two largest keys.

    The addition is done in the keys' own dtype (float64 for the oracle's keys,
    float32 when replaying the GPU's keys), as one IEEE addition.
    """
    T, E = keys.shape
    g = keys.reshape(T, n_group, E // n_group)
    srt = np.sort(g, axis=2)
    return srt[:, :, -1] + srt[:, :, -2]


def decide_topk(keys: np.ndarray, top_k: int, n_group: int = 1, topk_group: int = 1) -> np.ndarray:
    """Chosen experts per token, in slot order (key descending, ties to lower index).

    With n_group > 1 only experts of the topk_group best groups are eligible
    (group ties go to the lower group index).
    """
    keys = np.asarray(keys)
    T, E = keys.shape
    eligible = np.ones((T, E), bool)
    if n_group > 1:
        gs = group_scores(keys, n_group)
        gorder = _order_desc(gs, np.ones_like(gs, bool))
        keep = np.zeros((T, n_group), bool)
        np.put_along_axis(keep, gorder[:, :topk_group], True, axis=1)
        eligible = np.repeat(keep, E // n_group, axis=1)
    order = _order_desc(keys, eligible)
    return order[:, :top_k].astype(np.int32)


def gate_weights(keys: np.ndarray, topk_idx: np.ndarray, gate: int, renormalize: int = 1,
                 routed_scale: float = 1.0) -> np.ndarray:
    """Gate of each chosen slot (float64)."""
    keys = np.asarray(keys, np.float64)
    sel = np.take_along_axis(keys, topk_idx.astype(np.int64), axis=1)
    if gate == GATE_SOFTMAX:
        m = keys.max(axis=1, keepdims=True)
        num = np.exp(sel - m)
        den = num.sum(axis=1, keepdims=True) if renormalize else np.exp(keys - m).sum(axis=1, keepdims=True)
        w = num / den
    else:
        w = sel / sel.sum(axis=1, keepdims=True) if renormalize else sel
    return w * float(routed_scale)


def route(x, w_router, shape, bias=None):
    """Oracle routing of a whole batch: (topk_idx [T,k] int32, topk_w [T,k] f64, keys [T,E] f64)."""
    L = router_logits(x, w_router)
    keys = gating_keys(L, shape.gate, bias)
    idx = decide_topk(keys, shape.top_k, shape.n_group, shape.topk_group)
    w = gate_weights(keys, idx, shape.gate, shape.renormalize, shape.routed_scale)
    return idx, w, keys


# ----------------------------------------------------------------------------------------
# histogram, scan, permutation
# ----------------------------------------------------------------------------------------
def local_expert(topk_idx: np.ndarray, e_begin: int, E_local: int) -> np.ndarray:
    """Local expert id of every slot, or -1 for a slot routed to another rank."""
    le = np.asarray(topk_idx, np.int64) - e_begin
    return np.where((le >= 0) & (le < E_local), le, -1)


def counts_offsets(topk_idx: np.ndarray, e_begin: int, E_local: int, expert_capacity: int = 0):
    """counts[e] = local slots routed to local expert e (before any capacity drop);
    offsets = [0, cumsum(counts)], or the equal-stride segment starts e * C (e = 0 .. E_local)
    in the masked-decode layout."""
    le = local_expert(topk_idx, e_begin, E_local)
    counts = np.bincount(le[le >= 0], minlength=E_local).astype(np.int32)
    if expert_capacity > 0:
        offsets = (np.arange(E_local + 1) * expert_capacity).astype(np.int32)
    else:
        offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    return counts, offsets


def expert_rank(topk_idx: np.ndarray, e_begin: int, E_local: int) -> np.ndarray:
    """Rank of every local slot among the slots of its expert in ascending token order
    (the token-major slot list; two slots of one token never share an expert), -1 elsewhere."""
    T, k = topk_idx.shape
    le = local_expert(topk_idx, e_begin, E_local).reshape(-1)
    slots = np.nonzero(le >= 0)[0]
    order = slots[np.argsort(le[slots], kind="stable")]              # stable: token order kept
    counts = np.bincount(le[slots], minlength=E_local)
    first = np.concatenate([[0], np.cumsum(counts)])[:-1]
    rank = np.full(T * k, -1, np.int64)
    rank[order] = np.arange(order.size) - first[le[order]]
    return rank.reshape(T, k)


def keep_mask(topk_idx: np.ndarray, e_begin: int, E_local: int, expert_capacity: int = 0) -> np.ndarray:
    """Slots that reach this rank's experts: local, and (masked-decode layout) ranked below the
    expert capacity inside their expert."""
    rank = expert_rank(topk_idx, e_begin, E_local)
    keep = rank >= 0
    if expert_capacity > 0:
        keep &= rank < expert_capacity
    return keep


def permutation(topk_idx: np.ndarray, e_begin: int, E_local: int, expert_capacity: int = 0):
    """Expert-contiguous row order: row_token[r] = token of row r; slot_row[t, j] = row or -1.

    Rows of one expert are in ascending token order (a stable counting sort of the
    token-major slot list).  Masked-decode layout (expert_capacity C > 0): row_token has
    E_local * C entries (-1 for rows past an expert's valid prefix); slot (t, j) of local
    expert e with rank r < C sits in row e * C + r, a slot with r >= C is dropped (-1).
    """
    T, k = topk_idx.shape
    le = local_expert(topk_idx, e_begin, E_local)
    rank = expert_rank(topk_idx, e_begin, E_local)
    if expert_capacity > 0:
        keep = (rank >= 0) & (rank < expert_capacity)
        slot_row = np.where(keep, le * expert_capacity + rank, -1).astype(np.int32)
        row_token = np.full(E_local * expert_capacity, -1, np.int32)
        tt, jj = np.nonzero(keep)
        row_token[slot_row[tt, jj]] = tt
        return row_token, slot_row
    counts = np.bincount(le[le >= 0], minlength=E_local)
    first = np.concatenate([[0], np.cumsum(counts)])
    slot_row = np.where(rank >= 0, first[np.maximum(le, 0)] + rank, -1).astype(np.int32)
    row_token = np.zeros(int(counts.sum()), np.int32)
    tt, jj = np.nonzero(rank >= 0)
    row_token[slot_row[tt, jj]] = tt
    return row_token, slot_row


# ----------------------------------------------------------------------------------------
# expert FFN and combine
# ----------------------------------------------------------------------------------------
def swiglu_ffn(xr: np.ndarray, w13: np.ndarray, w2: np.ndarray) -> np.ndarray:
    """SwiGLU expert MLP on rows xr [m, d]: W2 (silu(W1 x) * (W3 x)).

    w13 is [2F, d] with rows [0, F) = W1 (gate) and rows [F, 2F) = W3 (up);
    w2 is [d, F]; silu(h) = h / (1 + exp(-h)).
    """
    xr = np.asarray(xr, np.float64)
    w13 = np.asarray(w13, np.float64)
    F = w13.shape[0] // 2
    h = xr @ w13[:F].T
    u = xr @ w13[F:].T
    a = h / (1.0 + np.exp(-h)) * u
    return a @ np.asarray(w2, np.float64).T


def combine(y_rows: np.ndarray, slot_row: np.ndarray, topk_w: np.ndarray, shared=None) -> np.ndarray:
    """out[t] = sum over local slots j of w[t, j] * y_rows[slot_row[t, j]]  (+ shared[t])."""
    T, k = slot_row.shape
    out = np.zeros((T, y_rows.shape[1]), np.float64)
    for j in range(k):
        r = slot_row[:, j]
        m = r >= 0
        out[m] += np.asarray(topk_w, np.float64)[m, j:j + 1] * y_rows[r[m]]
    if shared is not None:
        out += shared
    return out


def expert_outputs_for_tokens(xd: np.ndarray, topk_idx: np.ndarray, topk_w: np.ndarray, shape,
                              w13_bits, w2_bits, ws13_bits=None, ws2_bits=None, keep=None) -> np.ndarray:
    """Layer output rows for a set of tokens, straight from the definition.

    xd: [n, d] float64 token rows; topk_idx / topk_w: their routing.  Each local
    expert's weights are decoded once and applied to the tokens that chose it.
    keep: optional [n, k] mask of the slots that reach the experts (the masked-decode
    layout drops slots past an expert's capacity; the mask comes from the whole batch).
    """
    n = xd.shape[0]
    out = np.zeros((n, shape.d), np.float64)
    le = local_expert(topk_idx, shape.e_begin, shape.E_local)
    if keep is not None:
        le = np.where(keep, le, -1)
    for e in np.unique(le[le >= 0]):
        rows, slots = np.nonzero(le == e)
        y = swiglu_ffn(xd[rows], bf16_to_f64(w13_bits[e]), bf16_to_f64(w2_bits[e]))
        for i in range(rows.size):   # slot order per token is irrelevant in exact arithmetic
            out[rows[i]] += topk_w[rows[i], slots[i]] * y[i]
    if shape.F_shared > 0 and ws13_bits is not None:
        out += swiglu_ffn(xd, bf16_to_f64(ws13_bits), bf16_to_f64(ws2_bits))
    return out


def layer_forward(inputs: dict, routing=None):
    """Whole-layer oracle on a workload dict from the input generator.

    ``routing`` may supply (topk_idx, topk_w) to take instead of the oracle's own
    decision (used only for tokens whose choice is a rounding near-tie).
    Returns a dict with the routing, the permutation and ``out`` [T, d] float64.
    """
    sh = inputs["shape"]
    xd = bf16_to_f64(inputs["x"])
    idx, w, keys = route(xd, bf16_to_f64(inputs["w_router"]), sh, inputs.get("bias"))
    if routing is not None:
        idx, w = routing
    C = getattr(sh, "expert_capacity", 0)
    counts, offsets = counts_offsets(idx, sh.e_begin, sh.E_local, C)
    row_token, slot_row = permutation(idx, sh.e_begin, sh.E_local, C)
    keep = keep_mask(idx, sh.e_begin, sh.E_local, C) if C > 0 else None
    out = expert_outputs_for_tokens(xd, idx, w, sh, inputs["w13"], inputs["w2"],
                                    inputs.get("ws13"), inputs.get("ws2"), keep)
    return {"topk_idx": idx, "topk_w": w, "keys": keys, "counts": counts, "offsets": offsets,
            "row_token": row_token, "slot_row": slot_row, "out": out}
