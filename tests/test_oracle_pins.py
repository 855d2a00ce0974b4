"""Pins of the fp64 oracle against facts fixed outside it (CPU only).

Each test checks the oracle against something it does not compute itself: hand-
worked closed forms, brute force over all candidate subsets, an independent
library's bf16 conversion, per-element ``math.fsum`` loops, and identities of the
layer (one expert with top-1 is a dense SwiGLU MLP; the shared expert adds).  The
cases are chosen so that a dropped term, a wrong sign, a swapped W1/W3, a
transposed operand or a wrong tie rule fails at least one of them.
"""
import itertools
import json
import math
import os
from collections import Counter

import numpy as np
import pytest
import torch

import oracle
from paper_2607_18631_amd import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ----------------------------------------------------------------------------------------
# bf16 decoding and the input generator's rounding
# ----------------------------------------------------------------------------------------
def test_bf16_decode_known_patterns():
    bits = np.array([0x3F80, 0xC000, 0x4049, 0x0001, 0x7F7F, 0x8000, 0x7F80], np.uint16)
    v = oracle.bf16_to_f64(bits)
    assert v[0] == 1.0 and v[1] == -2.0 and v[2] == 3.140625
    assert v[3] == 2.0 ** -133
    assert v[4] == (2.0 - 2.0 ** -7) * 2.0 ** 127
    assert v[5] == 0.0 and math.copysign(1.0, v[5]) == -1.0
    assert v[6] == math.inf


def test_bf16_decode_matches_torch():
    rng = np.random.default_rng(1)
    bits = rng.integers(0, 1 << 16, size=20000, dtype=np.uint32).astype(np.uint16)
    bits = bits[((bits >> 7) & 0xFF) != 0xFF]          # drop inf/NaN exponents
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(oracle.bf16_to_f64(bits), ref)


def test_rne_encoder_matches_torch():
    rng = np.random.default_rng(2)
    a = (rng.standard_normal(50000) * 10.0 ** rng.integers(-6, 6, 50000)).astype(np.float32)
    # exact halfway cases: 1 + 2^-8 -> 1 (even), 1 + 3*2^-8 -> 1 + 2^-6 (even)
    a = np.concatenate([a, np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8)], np.float32)])
    ref = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = wl.f32_to_bf16_bits(a)
    np.testing.assert_array_equal(got, ref)
    assert oracle.bf16_to_f64(got[-3:]).tolist() == [1.0, 1.0 + 2 ** -6, -1.0]


# ----------------------------------------------------------------------------------------
# router logits
# ----------------------------------------------------------------------------------------
def test_router_logits_hand():
    x = np.array([[1.0, 2.0, 3.0], [0.0, -1.0, 0.5]])
    wr = np.array([[1.0, 0, 0], [0, 1.0, 0], [1.0, 1.0, 1.0], [0, 0, -1.0]])
    np.testing.assert_array_equal(oracle.router_logits(x, wr),
                                  [[1.0, 2.0, 6.0, -3.0], [0.0, -1.0, -0.5, -0.5]])


def test_router_logits_fsum_loops():
    rng = np.random.default_rng(3)
    x, wr = rng.standard_normal((5, 7)), rng.standard_normal((3, 7))
    ref = [[math.fsum(x[t, i] * wr[e, i] for i in range(7)) for e in range(3)] for t in range(5)]
    np.testing.assert_allclose(oracle.router_logits(x, wr), ref, rtol=0, atol=1e-13)


# ----------------------------------------------------------------------------------------
# top-k and group limit
# ----------------------------------------------------------------------------------------
def _brute_topk(keys, k, eligible=None):
    E = len(keys)
    cand = range(E) if eligible is None else [e for e in range(E) if eligible[e]]
    best = max(itertools.combinations(cand, k), key=lambda s: math.fsum(keys[e] for e in s))
    return sorted(best, key=lambda e: -keys[e])


def test_topk_bruteforce():
    rng = np.random.default_rng(4)
    for E, k in [(8, 2), (8, 3), (10, 4), (6, 6), (5, 1)]:
        keys = rng.standard_normal((20, E))
        got = oracle.decide_topk(keys, k)
        for t in range(20):
            assert got[t].tolist() == _brute_topk(keys[t], k)


def test_topk_ties_rank_formula():
    rng = np.random.default_rng(5)
    keys = rng.integers(0, 4, size=(50, 9)).astype(np.float64)   # many exact ties
    k = 4
    got = oracle.decide_topk(keys, k)
    for t in range(50):
        kk = keys[t]
        rank = [sum(1 for j in range(9) if kk[j] > kk[e] or (kk[j] == kk[e] and j < e)) for e in range(9)]
        expect = sorted([e for e in range(9) if rank[e] < k], key=lambda e: rank[e])
        assert got[t].tolist() == expect


def _brute_group_topk(keys, k, n_group, topk_group):
    E = len(keys)
    gsz = E // n_group
    gscore = [max(keys[a] + keys[b] for a in range(g * gsz, (g + 1) * gsz)
                  for b in range(g * gsz, (g + 1) * gsz) if a != b) for g in range(n_group)]
    best = max(itertools.combinations(range(n_group), topk_group),
               key=lambda s: math.fsum(gscore[g] for g in s))
    eligible = [(e // gsz) in best for e in range(E)]
    return _brute_topk(keys, k, eligible)


def test_group_limited_bruteforce():
    rng = np.random.default_rng(6)
    for E, n_group, topk_group, k in [(16, 4, 2, 3), (16, 8, 4, 4), (12, 3, 1, 2), (24, 4, 3, 8)]:
        keys = 1.0 / (1.0 + np.exp(-rng.standard_normal((15, E))))
        got = oracle.decide_topk(keys, k, n_group, topk_group)
        for t in range(15):
            assert got[t].tolist() == _brute_group_topk(keys[t], k, n_group, topk_group)


def test_group_limited_hand():
    # group 0 holds the single largest key (0.95) but group 1 has the larger top-2 sum
    # (0.9 + 0.8 = 1.7 > 0.95 + 0.1 = 1.05): with one group kept, expert 0 is excluded.
    keys = np.array([[0.95, 0.10, 0.05, 0.02, 0.9, 0.8, 0.3, 0.2]])
    assert oracle.decide_topk(keys, 2, n_group=2, topk_group=1).tolist() == [[4, 5]]
    assert oracle.decide_topk(keys, 2).tolist() == [[0, 4]]
    np.testing.assert_allclose(oracle.group_scores(keys, 2), [[1.05, 1.7]])


def test_group_sum_precision_replay():
    # Two groups whose top-2 sums differ in float64 but tie once added in float32:
    # the float32 replay must take the tie rule (lower group), float64 the larger sum.
    # float32 sums are multiples of 2^-25 near 0.75; 0.75 + 2^-25 is a tie that rounds to even (0.75)
    a, b = np.float32(0.5), np.float32(0.25)
    c, d = np.float32(0.5), np.float32(0.25 + 2.0 ** -25)
    keys32 = np.array([[a, b, 0.0, 0.0, c, d, 0.0, 0.0]], np.float32)
    s64 = oracle.group_scores(keys32.astype(np.float64), 2)
    s32 = oracle.group_scores(keys32, 2)
    assert s32.dtype == np.float32
    assert s64[0, 0] < s64[0, 1] and s32[0, 0] == s32[0, 1]
    assert oracle.decide_topk(keys32, 1, 2, 1).tolist() == [[0]]
    assert oracle.decide_topk(keys32.astype(np.float64), 1, 2, 1).tolist() == [[4]]


# ----------------------------------------------------------------------------------------
# gates
# ----------------------------------------------------------------------------------------
def test_softmax_gates_hand():
    L = np.array([[0.0, math.log(3.0), -5.0]])
    idx = oracle.decide_topk(oracle.gating_keys(L, oracle.GATE_SOFTMAX), 2)
    assert idx.tolist() == [[1, 0]]
    w = oracle.gate_weights(L, idx, oracle.GATE_SOFTMAX, renormalize=1)
    np.testing.assert_allclose(w, [[0.75, 0.25]], rtol=1e-15)
    # not renormalised: full-softmax probabilities
    z = 1.0 + 3.0 + math.exp(-5.0)
    w = oracle.gate_weights(L, idx, oracle.GATE_SOFTMAX, renormalize=0)
    np.testing.assert_allclose(w, [[3.0 / z, 1.0 / z]], rtol=1e-15)


def test_softmax_gates_equal_renormalised_full_softmax():
    rng = np.random.default_rng(7)
    L = rng.standard_normal((30, 16)) * 3
    bias = rng.standard_normal(16)
    keys = oracle.gating_keys(L, oracle.GATE_SOFTMAX, bias)
    idx = oracle.decide_topk(keys, 4)
    w = oracle.gate_weights(keys, idx, oracle.GATE_SOFTMAX, 1)
    for t in range(30):
        p = [math.exp(L[t, e] + bias[e]) for e in range(16)]
        p = [v / math.fsum(p) for v in p]
        sel = [p[e] for e in idx[t]]
        np.testing.assert_allclose(w[t], [v / math.fsum(sel) for v in sel], rtol=1e-13)
        assert abs(w[t].sum() - 1.0) < 1e-14
        # the bias changes the selection: chosen = largest L + bias
        assert set(idx[t]) == set(np.argsort(-(L[t] + bias))[:4])


def test_sigmoid_gates_hand():
    L = np.array([[0.0, math.log(3.0), -2.0]])
    s = oracle.gating_keys(L, oracle.GATE_SIGMOID)
    np.testing.assert_allclose(s[0, :2], [0.5, 0.75], rtol=1e-15)
    idx = oracle.decide_topk(s, 2)
    assert idx.tolist() == [[1, 0]]
    w = oracle.gate_weights(s, idx, oracle.GATE_SIGMOID, renormalize=1, routed_scale=2.5)
    np.testing.assert_allclose(w, [[1.5, 1.0]], rtol=1e-15)
    w = oracle.gate_weights(s, idx, oracle.GATE_SIGMOID, renormalize=0, routed_scale=2.0)
    np.testing.assert_allclose(w, [[1.5, 1.0]], rtol=1e-15)


def test_sigmoid_rejects_bias():
    with pytest.raises(ValueError):
        oracle.gating_keys(np.zeros((1, 4)), oracle.GATE_SIGMOID, np.zeros(4))


# ----------------------------------------------------------------------------------------
# histogram, scan, permutation
# ----------------------------------------------------------------------------------------
def _brute_perm(idx, e_begin, E_local):
    T, k = idx.shape
    pairs = sorted((int(idx[t, j]) - e_begin, t, j) for t in range(T) for j in range(k)
                   if 0 <= idx[t, j] - e_begin < E_local)
    cnt = Counter(p[0] for p in pairs)
    counts = [cnt.get(e, 0) for e in range(E_local)]
    offsets = [0]
    for c in counts:
        offsets.append(offsets[-1] + c)
    row_token = [p[1] for p in pairs]
    slot_row = [[-1] * k for _ in range(T)]
    for r, (_, t, j) in enumerate(pairs):
        slot_row[t][j] = r
    return counts, offsets, row_token, slot_row


@pytest.mark.parametrize("E,k,e_begin,E_local,T", [(8, 2, 0, 8, 40), (16, 4, 4, 5, 33), (32, 8, 0, 32, 17),
                                                   (12, 3, 11, 1, 25), (8, 1, 0, 8, 1)])
def test_counts_offsets_permutation_bruteforce(E, k, e_begin, E_local, T):
    rng = np.random.default_rng(E * 100 + k)
    idx = np.array([rng.permutation(E)[:k] for _ in range(T)], np.int32)
    counts, offsets = oracle.counts_offsets(idx, e_begin, E_local)
    row_token, slot_row = oracle.permutation(idx, e_begin, E_local)
    bc, bo, brt, bsr = _brute_perm(idx, e_begin, E_local)
    assert counts.tolist() == bc and offsets.tolist() == bo
    assert row_token.tolist() == brt and slot_row.tolist() == bsr
    # round trip: every local slot appears exactly once and points back to its token
    rows = slot_row[slot_row >= 0]
    assert sorted(rows.tolist()) == list(range(offsets[-1]))
    for t in range(T):
        for j in range(k):
            if slot_row[t, j] >= 0:
                r = slot_row[t, j]
                assert row_token[r] == t and offsets[idx[t, j] - e_begin] <= r < offsets[idx[t, j] - e_begin + 1]


def _brute_capacity_perm(idx, e_begin, E_local, C):
    """The masked-decode drop rule by a sequential walk: tokens in order, slots in order, each
    local expert keeps its first C slots in rows e*C, e*C+1, ...; the rest are dropped."""
    T, k = idx.shape
    taken = [0] * E_local
    slot_row = [[-1] * k for _ in range(T)]
    row_token = [-1] * (E_local * C)
    for t in range(T):
        for j in range(k):
            e = int(idx[t, j]) - e_begin
            if 0 <= e < E_local:
                if taken[e] < C:
                    slot_row[t][j] = e * C + taken[e]
                    row_token[e * C + taken[e]] = t
                taken[e] += 1
    return taken, row_token, slot_row


def test_capacity_layout_hand():
    """Experts 0..2 local, capacity 2: expert 0 keeps tokens 0, 1 and drops 2, 3; expert 1 keeps
    tokens 0, 2 and drops 3; expert 2 keeps token 1."""
    idx = np.array([[0, 1], [0, 2], [1, 0], [0, 1]], np.int32)
    counts, offsets = oracle.counts_offsets(idx, 0, 3, 2)
    row_token, slot_row = oracle.permutation(idx, 0, 3, 2)
    assert counts.tolist() == [4, 3, 1] and offsets.tolist() == [0, 2, 4, 6]
    assert slot_row.tolist() == [[0, 2], [1, 4], [3, -1], [-1, -1]]
    assert row_token.tolist() == [0, 1, 0, 2, 1, -1]
    assert oracle.keep_mask(idx, 0, 3, 2).tolist() == [[True, True], [True, True], [True, False], [False, False]]


@pytest.mark.parametrize("E,k,e_begin,E_local,T,C", [(8, 2, 0, 8, 40, 1), (8, 2, 0, 8, 40, 6), (16, 4, 4, 5, 33, 3),
                                                     (32, 8, 0, 32, 17, 2), (12, 3, 11, 1, 25, 4),
                                                     (8, 3, 2, 4, 29, 100)])
def test_capacity_layout_bruteforce(E, k, e_begin, E_local, T, C):
    rng = np.random.default_rng(E * 1000 + k * 10 + C)
    idx = np.array([rng.permutation(E)[:k] for _ in range(T)], np.int32)
    counts, offsets = oracle.counts_offsets(idx, e_begin, E_local, C)
    row_token, slot_row = oracle.permutation(idx, e_begin, E_local, C)
    taken, brt, bsr = _brute_capacity_perm(idx, e_begin, E_local, C)
    assert counts.tolist() == taken
    assert offsets.tolist() == [e * C for e in range(E_local + 1)]
    assert row_token.tolist() == brt and slot_row.tolist() == bsr
    assert (oracle.keep_mask(idx, e_begin, E_local, C) == (slot_row >= 0)).all()


def test_capacity_layout_without_drops_matches_offsets_layout():
    """With C >= every expert count nothing is dropped: ranks and layer output are those of the
    monotone-offsets layout, rows moved to e*C + rank."""
    sh = wl.MoEShape(T=30, d=16, E=8, top_k=2, F=8, E_local=4, e_begin=2, F_shared=8)
    inp = wl.custom_inputs(sh, seed=6)
    plain = oracle.layer_forward(inp)
    C = int(plain["counts"].max())
    capped = oracle.layer_forward(dict(inp, shape=sh.replace(expert_capacity=C)))
    np.testing.assert_array_equal(capped["out"], plain["out"])
    le = oracle.local_expert(plain["topk_idx"], sh.e_begin, sh.E_local)
    rank = plain["slot_row"] - np.where(le >= 0, plain["offsets"][np.maximum(le, 0)], 0)
    np.testing.assert_array_equal(capped["slot_row"], np.where(le >= 0, le * C + rank, -1))


def test_capacity_layer_output_by_loops():
    """Layer with drops (capacity 1) against per-token loops: a dropped slot contributes nothing."""
    sh = wl.MoEShape(T=10, d=8, E=4, top_k=2, F=6, E_local=4, expert_capacity=1)
    inp = wl.custom_inputs(sh, seed=8)
    res = oracle.layer_forward(inp)
    xd = oracle.bf16_to_f64(inp["x"])
    taken = [0] * 4
    for t in range(10):
        out = np.zeros(8)
        for j in range(2):
            e = int(res["topk_idx"][t, j])
            if taken[e] < 1:
                out += res["topk_w"][t, j] * _dense_swiglu_loops(
                    xd[t:t + 1], oracle.bf16_to_f64(inp["w13"][e]), oracle.bf16_to_f64(inp["w2"][e]))[0]
            taken[e] += 1
        np.testing.assert_allclose(res["out"][t], out, rtol=1e-11, atol=1e-12)
    assert sum(taken) == 20 and (res["slot_row"] >= 0).sum() == 4


# ----------------------------------------------------------------------------------------
# SwiGLU expert MLP, combine and the layer
# ----------------------------------------------------------------------------------------
def _silu(h):
    return h / (1.0 + math.exp(-h))


def test_swiglu_hand():
    # d=2, F=2; distinct W1 / W3 so a swap changes the answer; W2 non-symmetric
    x = np.array([[1.0, 3.0]])
    w13 = np.array([[1.0, 0.0], [0.0, -1.0],      # W1 (gate) rows
                    [0.0, 2.0], [1.0, 1.0]])      # W3 (up) rows
    w2 = np.array([[1.0, 0.5], [-1.0, 0.0]])      # [d, F]
    h = [1.0, -3.0]
    u = [6.0, 4.0]
    a = [_silu(h[0]) * u[0], _silu(h[1]) * u[1]]
    expect = [a[0] + 0.5 * a[1], -a[0]]
    np.testing.assert_allclose(oracle.swiglu_ffn(x, w13, w2), [expect], rtol=1e-15)


def test_swiglu_fsum_loops():
    rng = np.random.default_rng(8)
    m, d, F = 3, 6, 5
    x, w13, w2 = rng.standard_normal((m, d)), rng.standard_normal((2 * F, d)), rng.standard_normal((d, F))
    ref = np.zeros((m, d))
    for r in range(m):
        a = [_silu(math.fsum(w13[f, i] * x[r, i] for i in range(d))) *
             math.fsum(w13[F + f, i] * x[r, i] for i in range(d)) for f in range(F)]
        for o in range(d):
            ref[r, o] = math.fsum(w2[o, f] * a[f] for f in range(F))
    np.testing.assert_allclose(oracle.swiglu_ffn(x, w13, w2), ref, rtol=1e-12, atol=1e-13)


def test_combine_hand():
    y = np.array([[1.0, 2.0], [10.0, 20.0], [100.0, 200.0]])
    slot_row = np.array([[1, -1, 0], [-1, 2, -1]])
    w = np.array([[0.5, 9.0, 0.25], [7.0, 2.0, 5.0]])
    shared = np.array([[1.0, 1.0], [0.0, -1.0]])
    out = oracle.combine(y, slot_row, w, shared)
    np.testing.assert_array_equal(out, [[0.5 * 10 + 0.25 * 1 + 1, 0.5 * 20 + 0.25 * 2 + 1],
                                        [2.0 * 100, 2.0 * 200 - 1]])


def _dense_swiglu_loops(xd, w13, w2):
    F = w13.shape[0] // 2
    out = np.zeros((xd.shape[0], w2.shape[0]))
    for t in range(xd.shape[0]):
        a = [_silu(math.fsum(w13[f] * xd[t])) * math.fsum(w13[F + f] * xd[t]) for f in range(F)]
        out[t] = [math.fsum(w2[o, f] * a[f] for f in range(F)) for o in range(w2.shape[0])]
    return out


@pytest.mark.parametrize("gate", [oracle.GATE_SOFTMAX, oracle.GATE_SIGMOID])
def test_layer_one_expert_top1_is_dense_swiglu(gate):
    sh = wl.MoEShape(T=9, d=16, E=1, top_k=1, F=12, E_local=1, gate=gate)
    inp = wl.custom_inputs(sh, seed=3)
    res = oracle.layer_forward(inp)
    assert res["topk_idx"].tolist() == [[0]] * 9
    np.testing.assert_allclose(res["topk_w"], 1.0, rtol=0, atol=1e-15)
    ref = _dense_swiglu_loops(oracle.bf16_to_f64(inp["x"]), oracle.bf16_to_f64(inp["w13"][0]),
                              oracle.bf16_to_f64(inp["w2"][0]))
    np.testing.assert_allclose(res["out"], ref, rtol=1e-12, atol=1e-12)


def test_layer_shared_expert_adds_and_offrank_tokens_get_only_shared():
    sh = wl.MoEShape(T=40, d=16, E=8, top_k=2, F=8, E_local=2, e_begin=3, F_shared=8,
                     gate=oracle.GATE_SIGMOID, renormalize=1, routed_scale=2.5)
    inp = wl.custom_inputs(sh, seed=4)
    res = oracle.layer_forward(inp)
    xd = oracle.bf16_to_f64(inp["x"])
    ys = _dense_swiglu_loops(xd, oracle.bf16_to_f64(inp["ws13"]), oracle.bf16_to_f64(inp["ws2"]))
    no_shared = dict(inp, ws13=None, ws2=None, shape=sh.replace(F_shared=0))
    routed = oracle.layer_forward(no_shared)["out"]
    np.testing.assert_allclose(res["out"], routed + ys, rtol=1e-12, atol=1e-12)
    local = (res["slot_row"] >= 0).any(axis=1)
    assert (~local).any() and local.any()
    np.testing.assert_array_equal(routed[~local], 0.0)
    np.testing.assert_allclose(res["topk_w"].sum(axis=1), 2.5, rtol=1e-14)


def test_layer_routed_output_by_loops():
    """Whole layer on a small softmax case against per-token loops of the definition."""
    sh = wl.MoEShape(T=12, d=8, E=4, top_k=2, F=6, E_local=4)
    inp = wl.custom_inputs(sh, seed=5, zipf_s=1.2)
    res = oracle.layer_forward(inp)
    xd = oracle.bf16_to_f64(inp["x"])
    wr = oracle.bf16_to_f64(inp["w_router"])
    for t in range(12):
        key = [math.fsum(xd[t] * wr[e]) + float(inp["bias"][e]) for e in range(4)]
        chosen = sorted(range(4), key=lambda e: (-key[e], e))[:2]
        z = math.fsum(math.exp(key[e]) for e in chosen)
        out = np.zeros(8)
        for e in chosen:
            out += math.exp(key[e]) / z * _dense_swiglu_loops(
                xd[t:t + 1], oracle.bf16_to_f64(inp["w13"][e]), oracle.bf16_to_f64(inp["w2"][e]))[0]
        assert res["topk_idx"][t].tolist() == chosen
        np.testing.assert_allclose(res["out"][t], out, rtol=1e-11, atol=1e-12)


def test_hand_layer_golden():
    """A hand-worked two-token layer (tests/golden/hand_layer.json), closed forms only."""
    with open(os.path.join(GOLDEN, "hand_layer.json")) as f:
        g = json.load(f)
    sh = wl.MoEShape(**g["shape"])
    f32 = lambda a: wl.f32_to_bf16_bits(np.array(a, np.float32))   # values are exact in bf16
    inp = {"shape": sh, "x": f32(g["x"]), "w_router": f32(g["w_router"]), "bias": None,
           "w13": f32(g["w13"]), "w2": f32(g["w2"]), "ws13": None, "ws2": None}
    res = oracle.layer_forward(inp)
    env = {"exp": math.exp, "log": math.log}
    assert res["topk_idx"].tolist() == g["expect_topk_idx"]
    np.testing.assert_allclose(res["topk_w"], [[eval(s, env) for s in r] for r in g["expect_topk_w"]],
                               rtol=1e-14)
    np.testing.assert_allclose(res["out"], [[eval(s, env) for s in r] for r in g["expect_out"]],
                               rtol=1e-14, atol=1e-15)
    assert res["offsets"].tolist() == g["expect_offsets"]
    assert res["row_token"].tolist() == g["expect_row_token"]


# ----------------------------------------------------------------------------------------
# workload readings
# ----------------------------------------------------------------------------------------
def test_skewed_workload_load_ratio_in_band():
    """Zipf(1.2) router bias gives hot experts 10-50x the tokens of the median expert."""
    inp = wl.make_inputs("skewed", with_experts=False)
    sh = inp["shape"]
    idx, w, _ = oracle.route(oracle.bf16_to_f64(inp["x"]), oracle.bf16_to_f64(inp["w_router"]), sh,
                             inp["bias"])
    counts, _ = oracle.counts_offsets(idx, 0, sh.E_local)
    ratio = counts.max() / np.median(counts)
    assert 10 <= ratio <= 50, ratio
    np.testing.assert_allclose(w.sum(axis=1), 1.0, rtol=1e-13)


def test_dsv3_local_slice_is_group0():
    sh = wl.WORKLOADS["dsv3"].shape
    assert sh.E // sh.n_group == sh.E_local and sh.e_begin == 0
    assert sh.topk_group * (sh.E // sh.n_group) >= sh.top_k
