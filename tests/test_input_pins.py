"""The input recipe is pinned: the SHA-256 of each workload's seeded input bytes (token rows,
router weight and bias, the first and last local expert's weights, the shared expert's
weights) equals the digest recorded in tests/golden/input_sha256.json.  A change of the
random generator, of a stream's seed layout, of a standard deviation or of the bf16 rounding
changes these bytes.  Also checks that the batch generator and the per-expert generator the
digests are taken from produce the same bytes."""
import json
import os
import sys

import numpy as np
import pytest

from paper_2607_18631_amd import workloads as wl

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "golden"))
import make_input_sha256  # noqa: E402

with open(os.path.join(HERE, "golden", "input_sha256.json")) as f:
    PINS = json.load(f)


@pytest.mark.parametrize("name", list(wl.WORKLOADS))
def test_input_bytes_pinned(name):
    assert make_input_sha256.digests(name) == PINS[name]


def test_batch_generator_matches_per_expert_generator():
    inp = wl.make_inputs("tiny")
    for le in range(inp["shape"].E_local):
        w13, w2 = wl.expert_tensors("tiny", le)
        np.testing.assert_array_equal(inp["w13"][le], w13)
        np.testing.assert_array_equal(inp["w2"][le], w2)
    sh = wl.MoEShape(T=16, d=64, E=8, top_k=2, F=32, E_local=3, e_begin=4, F_shared=16)
    inp = wl.custom_inputs(sh, seed=7)
    w = wl.Workload("custom", sh, router_std=sh.d ** -0.5, seed=7)
    ws13, ws2 = wl.shared_tensors(w)
    np.testing.assert_array_equal(inp["ws13"], ws13)
    np.testing.assert_array_equal(inp["ws2"], ws2)
    np.testing.assert_array_equal(inp["w13"][2], wl.expert_tensors(w, 2)[0])
