"""Write input_sha256.json: the SHA-256 of the seeded input bytes of each workload.

The digests pin the input recipe (numpy PCG64 streams per tensor and expert, the scaling by
the standard deviation, the round-to-nearest-even bf16 encoding): a change in any of them
changes every workload, and the CPU test that recomputes these digests fails.  Hashed per
workload: the token rows, the router weight, the router bias (if any), the first and the last
local expert's W13 and W2, and the shared expert's weights (if any).  Only the input
generator is called here (no kernel and no oracle arithmetic).

    python tests/golden/make_input_sha256.py
"""
import hashlib
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_2607_18631_amd import workloads as wl  # noqa: E402


def digests(name):
    w = wl.WORKLOADS[name]
    sh = w.shape
    inp = wl.make_inputs(name, with_experts=False)
    h = lambda a: hashlib.sha256(a.tobytes()).hexdigest()
    out = {"x": h(inp["x"]), "w_router": h(inp["w_router"])}
    if inp["bias"] is not None:
        out["bias"] = h(inp["bias"])
    for le in sorted({0, sh.E_local - 1}):
        w13, w2 = wl.expert_tensors(name, le)
        out[f"w13[{le}]"] = h(w13)
        out[f"w2[{le}]"] = h(w2)
    ws13, ws2 = wl.shared_tensors(name)
    if ws13 is not None:
        out["ws13"] = h(ws13)
        out["ws2"] = h(ws2)
    return out


def main():
    res = {name: digests(name) for name in wl.WORKLOADS}
    with open(os.path.join(HERE, "input_sha256.json"), "w") as f:
        json.dump(res, f, indent=1, sort_keys=True)
        f.write("\n")


if __name__ == "__main__":
    main()
