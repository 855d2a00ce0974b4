"""Benchmark of the MoE-layer forward on one MI355X.

    python bench.py [--gpus 1] [--steps 30] [--warmup 40] [--workload dsv3] [--no-cpu-baseline]

One step = one moe_layer_forward (router logits, gating/top-k, histogram + scan,
permutation, grouped SwiGLU expert MLP, shared expert, combine) over one batch of
seeded synthetic input already resident in HBM.  Prints ONE JSON line.

Default workload: the DeepSeek-V3-shaped rank share (T=8192, d=7168, 256 routed experts,
top-8 sigmoid gating with 8 groups / top-4 groups, 32 local experts of width 2048 plus
one shared expert of width 2048), the configuration the grouped-GEMM and HBM targets
are quoted on.

Timing follows the paper's kernel protocol on the timed steps: every step records HIP events
between its launches (moe_layer_forward_traced, on the library's stream), and each figure is the
median over 3 rounds of the per-round medians; the synchronised wall clock of the same steps is
reported beside it.  The dominant kernel's roofline figure comes from those events; the CPU
baseline times the fp64 oracle on a bounded sample of the same batch on the host cores.  The
standalone permutation and combine are timed back to back, on the same buffers (warm: inputs
partly in the 256 MB MALL) and rotating through buffer sets larger than the MALL (hbm).
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


class HipEvents:
    """hipEvent_t handles through the HIP runtime's C API (timing events)."""

    def __init__(self):
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.hip.hipEventSynchronize.argtypes = [ctypes.c_void_p]

    def create(self, n):
        arr = (ctypes.c_void_p * n)()
        for i in range(n):
            h = ctypes.c_void_p()
            if self.hip.hipEventCreate(ctypes.byref(h)) != 0:
                raise RuntimeError("hipEventCreate failed")
            arr[i] = h
        return arr

    def elapsed_ms(self, a, b):
        ms = ctypes.c_float()
        if self.hip.hipEventElapsedTime(ctypes.byref(ms), a, b) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def destroy(self, arr):
        for h in arr:
            self.hip.hipEventDestroy(h)


def gating_desc(sh):
    g = "softmax" if sh.gate == 0 else "sigmoid"
    if sh.n_group > 1:
        g += f", {sh.n_group} groups / top-{sh.topk_group}"
    g += ", renormalised" if sh.renormalize else ""
    if sh.routed_scale != 1.0:
        g += f" x{sh.routed_scale:g}"
    return g


TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "gemm_swiglu_dsv3_traffic.md")
GEMM_SOURCE = os.path.join(ROOT, "paper_2607_18631_amd", "csrc", "gemm.hip")


def measured_traffic(workload):
    """HBM bytes per launch of the SwiGLU GEMM from the committed rocprofv3 FETCH_SIZE / WRITE_SIZE
    summary, or None when the kernel source changed since the counters were taken (or another
    workload is benchmarked)."""
    import hashlib
    if workload != "dsv3" or not os.path.exists(TRAFFIC_SUMMARY):
        return None
    fields = {}
    with open(TRAFFIC_SUMMARY) as f:
        for line in f:
            line = line.strip().strip("`")
            if ":" in line and line.startswith(("traffic_bytes_per_launch", "kernel_source_sha256")):
                k, v = line.split(":", 1)
                fields[k.strip()] = v.strip()
    with open(GEMM_SOURCE, "rb") as f:
        sha = hashlib.sha256(f.read()).hexdigest()
    if fields.get("kernel_source_sha256") != sha or "traffic_bytes_per_launch" not in fields:
        return None
    return float(fields["traffic_bytes_per_launch"])


WARM_S = 0.1   # least busy time before any timed call: an idle part takes ~50 ms of load to reach its clock


def warm_up(fn, calls):
    """Batches of `calls` calls of `fn`, each batch synchronised, until at least WARM_S of wall time
    has passed since the first call (at least one batch)."""
    import torch
    t0 = time.perf_counter()
    while True:
        for _ in range(max(1, calls)):
            fn()
        torch.cuda.synchronize()
        if time.perf_counter() - t0 >= WARM_S:
            return


def timed_median(fn, reps, rounds=3, warmup=10):
    """Median over `rounds` of the median per-call time (ms) of `reps` calls, each call between
    two events on the current stream, after `warmup` calls (more if they take under WARM_S)."""
    import numpy as np
    import torch
    warm_up(fn, warmup)
    meds = []
    for _ in range(rounds):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
        ev[0].record()
        for i in range(reps):
            fn()
            ev[i + 1].record()
        torch.cuda.synchronize()
        meds.append(float(np.median([ev[i].elapsed_time(ev[i + 1]) for i in range(reps)])))
    return float(np.median(meds))


SCRUB_BYTES = 512 << 20          # read between calls for cold-cache figures (> the 256 MB MALL)
ROTATE_BYTES = 768 << 20         # buffer sets rotated through for the HBM (cold) streaming figures


class ReadProbe:
    """libmoe_probe.so: a read-only stream kernel (the read ceiling, and the cache scrub of the
    cold figures: reading leaves clean lines, so the next kernel pays no write-back)."""

    def __init__(self):
        import torch
        from paper_2607_18631_amd import build as _b
        self.lib = ctypes.CDLL(_b.PROBE_LIB)
        self.lib.probe_read_stream.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p]
        self.lib.probe_read_sink_words.restype = ctypes.c_int64
        self.sink = torch.empty(int(self.lib.probe_read_sink_words()), dtype=torch.int32, device="cuda:0")
        self.lib.probe_mfma_loop.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
        self.lib.probe_mfma_blocks.restype = ctypes.c_int64
        self.lib.probe_mfma_flops.argtypes = [ctypes.c_int]
        self.lib.probe_mfma_flops.restype = ctypes.c_double
        self.mfma_sink = None
        self.lib.probe_lds_read.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        self.lib.probe_lds_blocks.restype = ctypes.c_int64
        self.lib.probe_lds_bytes.argtypes = [ctypes.c_int]
        self.lib.probe_lds_bytes.restype = ctypes.c_double
        self.lds_sink = self.lds_cycles = None

    def read(self, buf):
        import torch
        st = torch.cuda.current_stream().cuda_stream
        rc = self.lib.probe_read_stream(buf.data_ptr(), buf.numel() * buf.element_size(), self.sink.data_ptr(), st)
        if rc != 0:
            raise RuntimeError(f"probe_read_stream failed ({rc})")

    def mfma(self, iters):
        """One launch of the MFMA loop probe; returns its flops."""
        import torch
        if self.mfma_sink is None:
            self.mfma_sink = torch.empty(int(self.lib.probe_mfma_blocks()) * 256, dtype=torch.float32,
                                         device="cuda:0")
        rc = self.lib.probe_mfma_loop(iters, self.mfma_sink.data_ptr(), torch.cuda.current_stream().cuda_stream)
        if rc != 0:
            raise RuntimeError(f"probe_mfma_loop failed ({rc})")
        return self.lib.probe_mfma_flops(iters)

    def lds(self, iters):
        """One launch of the LDS read probe (two workgroups of 4 waves per CU); returns its bytes."""
        import torch
        if self.lds_sink is None:
            nb = int(self.lib.probe_lds_blocks())
            self.lds_sink = torch.empty(nb * 256, dtype=torch.int32, device="cuda:0")
            self.lds_cycles = torch.empty(2 * nb, dtype=torch.int64, device="cuda:0")
        rc = self.lib.probe_lds_read(iters, self.lds_sink.data_ptr(), self.lds_cycles.data_ptr(),
                                     torch.cuda.current_stream().cuda_stream)
        if rc != 0:
            raise RuntimeError(f"probe_lds_read failed ({rc})")
        return self.lib.probe_lds_bytes(iters)

    def lds_clock_ghz(self):
        """Shader clock (GHz) during the last probe_lds_read call: each workgroup's s_memtime cycles
        over its 100 MHz s_memrealtime ticks (median)."""
        import numpy as np
        import torch
        torch.cuda.synchronize()
        c = self.lds_cycles.cpu().numpy().reshape(-1, 2).astype(np.float64)
        return float(np.median(c[:, 0] / c[:, 1])) * 0.1


def back_to_back_ms(fn, calls, rounds=3, warmup=3):
    """Median over `rounds` of the mean per-call time (ms) of `calls` calls issued back to back
    between two events (no event between calls), after `warmup` calls (more if they take under
    WARM_S)."""
    import numpy as np
    import torch
    warm_up(fn, warmup)
    res = []
    for _ in range(rounds):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(calls):
            fn()
        e1.record()
        torch.cuda.synchronize()
        res.append(e0.elapsed_time(e1) / calls)
    return float(np.median(res))


def cold_ms(fn, scrub, reps):
    """Median time (ms) of one call of `fn` right after `scrub()` has streamed a buffer larger than
    the MALL through the caches, so the call's inputs come from HBM; each call between two events."""
    import numpy as np
    import torch
    fn()
    torch.cuda.synchronize()
    ts = []
    for _ in range(reps):
        scrub()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        fn()
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    return float(np.median(ts))


def crossover_run():
    """The paper's RQ4 kernel-crossover workload: per-token latency over the global token count
    me * E / top_k, for the grouped expert MLP alone (exactly me rows per local expert, the
    figure's single-card expert compute) and for the whole layer on that many tokens.  Protocol:
    warmup 10 calls and >= 0.1 s, 200 calls per round for me < 16 else 50, median of 3 round medians."""
    import numpy as np
    import torch

    from paper_2607_18631_amd import moe
    from paper_2607_18631_amd import workloads as wl
    rows = []
    for me in wl.CROSSOVER_ME:
        w = wl.crossover(me)
        inputs = wl.make_inputs(w)
        sh = inputs["shape"]
        layer = moe.DeviceLayer(inputs, device="cuda:0")
        reps = 200 if me < 16 else 50
        n = me * sh.E_local
        offsets = torch.arange(0, n + 1, me, dtype=torch.int32, device="cuda:0")
        x_perm = layer.x[:n].contiguous()                  # n = T / 4 distinct token rows
        ffn_sh = sh.replace(T=n, top_k=1)              # capacity n rows
        y = torch.empty((n, sh.d), dtype=torch.bfloat16, device="cuda:0")
        ws = moe.alloc_workspace(ffn_sh, moe.MOE_WS_FFN, "cuda:0")
        t_ffn = timed_median(lambda: moe.moe_grouped_ffn(ffn_sh, x_perm, offsets, layer.w13, layer.w2, y, ws), reps)
        t_layer = timed_median(layer.forward, reps)
        tokens = me * sh.E // sh.top_k
        rows.append({"me": me, "global_tokens": tokens, "expert_mlp_us": t_ffn * 1e3,
                     "expert_mlp_us_per_token": t_ffn * 1e3 / tokens,
                     "expert_mlp_tflops": 6.0 * sh.d * sh.F * n / (t_ffn * 1e-3) / 1e12,
                     "layer_us": t_layer * 1e3, "layer_us_per_token": t_layer * 1e3 / tokens})
        log(f"me={me}: expert MLP {t_ffn * 1e3:.1f} us ({rows[-1]['expert_mlp_us_per_token']:.4f} us/token), "
            f"layer {t_layer * 1e3:.1f} us")
        del layer, x_perm, y, ws
        torch.cuda.empty_cache()
    return rows


def masked_decode_run(workload, capacity):
    """One decode step in the offsets layout and in the masked-decode layout (equal segments of
    `capacity` rows per local expert; capacity T keeps every slot), each called eagerly and
    replayed from a HIP graph captured once.  Per-call times follow the paper's protocol (warmup
    10, 200 calls per round under 100 us else 50, median of 3 round medians); the HBM figure
    counts the weights of the experts that received rows, the shared-expert and router weights,
    token rows in and out and the routing arrays."""
    import numpy as np
    import torch

    from paper_2607_18631_amd import moe
    from paper_2607_18631_amd import workloads as wl
    base = wl.make_inputs(workload)
    sh0 = base["shape"]
    C = capacity if capacity > 0 else sh0.T
    rows, outs, dropped = [], {}, 0
    for name, sh in (("offsets", sh0), ("masked", sh0.replace(expert_capacity=C))):
        layer = moe.DeviceLayer(dict(base, shape=sh), device="cuda:0")
        layer.forward()
        torch.cuda.synchronize()
        t_eager = timed_median(layer.forward, 50)
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            layer.forward()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            layer.forward()
        t_graph = timed_median(g.replay, 50)
        g.replay()
        torch.cuda.synchronize()
        outs[name] = moe.bf16_bits(layer.out)
        counts = layer.region(moe.MOE_REGION_COUNTS, torch.int32, (sh.E_local,)).cpu().numpy()
        d, F, Fs, T, k = sh.d, sh.F, sh.F_shared, sh.T, sh.top_k
        active = int((counts > 0).sum())
        layer_bytes = (active * 3 * d * F * 2 + 3 * d * Fs * 2 + sh.E * d * 2 + 2 * T * d * 2 + T * k * 8)
        kept = int(np.minimum(counts, C).sum()) if sh.expert_capacity > 0 else int(counts.sum())
        dropped = max(dropped, int(counts.sum()) - kept)
        rows.append({"layout": name, "expert_capacity": sh.expert_capacity, "buffer_rows": sh.capacity,
                     "local_rows": kept, "active_local_experts": active,
                     "eager_us": t_eager * 1e3, "graph_us": t_graph * 1e3,
                     "graph_tokens_per_s": T / (t_graph * 1e-3),
                     "graph_hbm_gbs": layer_bytes / (t_graph * 1e-3) / 1e9,
                     "eager_hbm_gbs": layer_bytes / (t_eager * 1e-3) / 1e9})
        log(f"{name}: eager {t_eager * 1e3:.1f} us, graph replay {t_graph * 1e3:.1f} us, "
            f"{rows[-1]['graph_hbm_gbs']:.0f} GB/s")
        del g, layer
        torch.cuda.empty_cache()
    # with no slot dropped both layouts compute the same rows with the same tiles
    same = bool(np.array_equal(outs["offsets"], outs["masked"])) if dropped == 0 else None
    return sh0, C, rows, same


def fusion_matrix_run(workload, steps):
    """The layer in the paper's four kernel structures (fuse_gather x fuse_combine): per-call
    time (warmup 10 calls and >= 0.1 s, median of 3 round medians of `steps` calls) and the
    per-step split of one traced pass per call, averaged."""
    import numpy as np
    import torch

    from paper_2607_18631_amd import moe
    from paper_2607_18631_amd import workloads as wl
    base = wl.make_inputs(workload)
    sh0 = base["shape"]
    ev = HipEvents()
    nstep = len(moe.MOE_STEP_NAMES)
    rows = []
    for name, fusion in wl.FUSION_VARIANTS.items():
        sh = sh0.replace(fusion=fusion)
        layer = moe.DeviceLayer(dict(base, shape=sh), device="cuda:0")
        t = timed_median(layer.forward, steps)
        events = [ev.create(nstep + 1) for _ in range(steps)]
        for i in range(steps):
            layer.forward_traced(events[i])
        torch.cuda.synchronize()
        split = np.array([[ev.elapsed_ms(e[j], e[j + 1]) for j in range(nstep)] for e in events]).mean(axis=0)
        for e in events:
            ev.destroy(e)
        rows.append({"variant": name, "fusion": fusion, "layer_us": t * 1e3, "tokens_per_s": sh.T / (t * 1e-3),
                     "step_us": {n: round(float(split[i]) * 1e3, 2) for i, n in enumerate(moe.MOE_STEP_NAMES)}})
        log(f"{name}: {t * 1e3:.1f} us per layer")
        del layer
        torch.cuda.empty_cache()
    return sh0, rows


def backward_run(workload, steps):
    """The expert-MLP backward (moe_grouped_ffn_backward) on the expert-ordered rows of one
    routed batch of the workload (its forward run unfused, so x_perm is materialised), next to
    the forward expert MLP (moe_grouped_ffn) on the same rows.  Per-call times: warmup 10 calls
    and >= 0.1 s, median of 3 round medians of `steps` calls."""
    import numpy as np
    import torch

    from paper_2607_18631_amd import moe
    from paper_2607_18631_amd import workloads as wl
    inputs = wl.make_inputs(workload)
    sh = inputs["shape"].replace(fusion=wl.FUSION_VARIANTS["unfused"])
    layer = moe.DeviceLayer(dict(inputs, shape=sh), device="cuda:0")
    layer.forward()
    torch.cuda.synchronize()
    cap, d, F, E = sh.capacity, sh.d, sh.F, sh.E_local
    x_perm = layer.region(moe.MOE_REGION_X_PERM, torch.bfloat16, (cap, d))
    offsets = layer.region(moe.MOE_REGION_OFFSETS, torch.int32, (E + 1,))
    n_loc = int(offsets[-1].item())
    g = torch.Generator(device="cuda:0").manual_seed(5)
    dy = torch.randn((cap, d), generator=g, device="cuda:0").to(torch.bfloat16)
    dx = torch.empty((cap, d), dtype=torch.bfloat16, device="cuda:0")
    dw13 = torch.empty((E, 2 * F, d), dtype=torch.bfloat16, device="cuda:0")
    dw2 = torch.empty((E, d, F), dtype=torch.bfloat16, device="cuda:0")
    ws = moe.alloc_workspace(sh, moe.MOE_WS_FFN_BWD, "cuda:0")
    y = torch.empty((cap, d), dtype=torch.bfloat16, device="cuda:0")
    ws_f = moe.alloc_workspace(sh, moe.MOE_WS_FFN, "cuda:0")
    t_bwd = timed_median(lambda: moe.moe_grouped_ffn_backward(sh, x_perm, offsets, layer.w13, layer.w2, dy, dx,
                                                              dw13, dw2, ws), steps)
    t_fwd = timed_median(lambda: moe.moe_grouped_ffn(sh, x_perm, offsets, layer.w13, layer.w2, y, ws_f), steps)
    assert bool(torch.isfinite(dw13.float()).all()) and bool(torch.isfinite(dx[:n_loc].float()).all())
    unit = d * F * n_loc
    log(f"backward {t_bwd * 1e3:.1f} us, forward {t_fwd * 1e3:.1f} us on {n_loc} rows")
    return sh, {"local_rows": n_loc, "backward_us": t_bwd * 1e3, "forward_us": t_fwd * 1e3,
                # executed MFMA work: dA 2, recomputed up-projection 4, dX 4, dW2 2, dW13 4 (x d F rows)
                "backward_tflops_executed": 16.0 * unit / (t_bwd * 1e-3) / 1e12,
                # the gradient products alone (twice the forward's 6 d F rows)
                "backward_tflops_gradients": 12.0 * unit / (t_bwd * 1e-3) / 1e12,
                "forward_tflops": 6.0 * unit / (t_fwd * 1e-3) / 1e12,
                "backward_frac_of_bf16_peak": 16.0 * unit / (t_bwd * 1e-3) / 1e12 / PEAK_BF16_TFLOPS}


def dense_ref_run(steps):
    """The DeepSeek-V3-shaped shared expert (8192 tokens, d = 7168, F = 2048) as a dense MLP: the
    library's grouped GEMMs on one group of 8192 rows (moe_grouped_ffn: W1/W3 + SwiGLU, then W2),
    next to the vendor GEMM library on the same two products (torch.nn.functional.linear, i.e.
    hipBLASLt; the SwiGLU between them is not timed).  A reference point for the grouped GEMM's
    efficiency; profile it with rocprofv3 counters to compare the kernels."""
    import torch
    import torch.nn.functional as tf

    from paper_2607_18631_amd import moe
    from paper_2607_18631_amd import workloads as wl
    inputs = wl.make_inputs("dsv3")
    full = inputs["shape"]
    T, d, F = full.T, full.d, full.F_shared
    sh = wl.MoEShape(T=T, d=d, E=1, top_k=1, F=F, E_local=1)
    dev = "cuda:0"
    x = moe.to_device_bf16(inputs["x"], dev)
    w13 = moe.to_device_bf16(inputs["ws13"], dev).reshape(1, 2 * F, d)
    w2 = moe.to_device_bf16(inputs["ws2"], dev).reshape(1, d, F)
    offsets = torch.tensor([0, T], dtype=torch.int32, device=dev)
    y = torch.empty((T, d), dtype=torch.bfloat16, device=dev)
    ws = moe.alloc_workspace(sh, moe.MOE_WS_FFN, dev)
    t_ours = timed_median(lambda: moe.moe_grouped_ffn(sh, x, offsets, w13, w2, y, ws), steps)
    w13_2d, w2_2d = w13[0], w2[0]
    h = tf.linear(x, w13_2d)
    act = (tf.silu(h[:, :F].float()) * h[:, F:].float()).to(torch.bfloat16)
    t_up = timed_median(lambda: tf.linear(x, w13_2d), steps)
    t_down = timed_median(lambda: tf.linear(act, w2_2d), steps)
    ref = tf.linear(act, w2_2d).float()
    err = float((y.float() - ref).norm() / ref.norm())
    up_f, down_f = 4.0 * T * d * F, 2.0 * T * d * F
    tfl = lambda f, ms: f / (ms * 1e-3) / 1e12
    log(f"dense shared expert: library {t_ours * 1e3:.1f} us, vendor up {t_up * 1e3:.1f} + down {t_down * 1e3:.1f} us")
    return {"T": T, "d": d, "F": F, "library_mlp_us": t_ours * 1e3, "library_mlp_tflops": tfl(up_f + down_f, t_ours),
            "vendor_up_us": t_up * 1e3, "vendor_up_tflops": tfl(up_f, t_up),
            "vendor_down_us": t_down * 1e3, "vendor_down_tflops": tfl(down_f, t_down),
            "vendor_mlp_tflops": tfl(up_f + down_f, t_up + t_down),
            "library_vs_vendor_rel_fro": err}


def layer_backward_run(workload, steps):
    """The whole layer backward (moe_layer_backward) after one forward of the workload: per-call
    time (warmup 10 calls and >= 0.1 s, median of 3 round medians of `steps` calls) next to the
    forward's, and the executed MFMA work: expert and shared MLP backward 16 d F rows each (dA 2,
    recomputed up-projection 4, dX 4, dW2 2, dW13 4), router 4 T E d (dx and dw_router)."""
    import numpy as np
    import torch

    from paper_2607_18631_amd import moe
    from paper_2607_18631_amd import workloads as wl
    inputs = wl.make_inputs(workload)
    sh = inputs["shape"]
    layer = moe.DeviceLayer(inputs, device="cuda:0")
    layer.forward()
    torch.cuda.synchronize()
    g = torch.Generator(device="cuda:0").manual_seed(9)
    dout = torch.randn((sh.T, sh.d), generator=g, device="cuda:0").to(torch.bfloat16)
    grads = layer.backward(dout)
    t_bwd = timed_median(lambda: layer.backward(dout), steps)
    t_fwd = timed_median(layer.forward, steps)
    assert bool(torch.isfinite(grads["dx"].float()).all()) and bool(torch.isfinite(grads["dw13"].float()).all())
    offsets = layer.region(moe.MOE_REGION_OFFSETS, torch.int32, (sh.E_local + 1,)).cpu().numpy()
    n_loc = int(offsets[-1]) if sh.expert_capacity == 0 else int(
        np.minimum(layer.region(moe.MOE_REGION_COUNTS, torch.int32, (sh.E_local,)).cpu().numpy(),
                   sh.expert_capacity).sum())
    d, F, Fs, T, E = sh.d, sh.F, sh.F_shared, sh.T, sh.E
    executed = 16.0 * d * (F * n_loc + Fs * T) + 4.0 * T * E * d
    fwd_flops = 6.0 * d * (F * n_loc + Fs * T) + 2.0 * T * E * d
    log(f"layer backward {t_bwd * 1e3:.1f} us, forward {t_fwd * 1e3:.1f} us on {n_loc} local rows")
    return sh, {"local_rows": n_loc, "backward_us": t_bwd * 1e3, "forward_us": t_fwd * 1e3,
                "backward_tokens_per_s": T / (t_bwd * 1e-3),
                "backward_tflops_executed": executed / (t_bwd * 1e-3) / 1e12,
                "backward_frac_of_bf16_peak": executed / (t_bwd * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
                "forward_tflops": fwd_flops / (t_fwd * 1e-3) / 1e12}


def all_workloads_run(steps):
    """Every workload of the metric's configuration list: per-call layer time (warmup 10 calls and
    >= 0.1 s, median of 3 round medians of `steps` calls), the per-step split from traced calls, tokens/s, the grouped
    GEMMs' TFLOP/s, the layer's algorithmic HBM bytes per second, and the layer's roofline floor
    max(FLOPs / bf16 peak, bytes / HBM peak) as a fraction of the measured time."""
    import numpy as np
    import torch

    from paper_2607_18631_amd import moe
    from paper_2607_18631_amd import workloads as wl
    ev = HipEvents()
    probe = ReadProbe()
    nstep = len(moe.MOE_STEP_NAMES)
    rows = []
    for name in wl.WORKLOADS:
        log(f"workload {name}: generating inputs")
        inputs = wl.make_inputs(name)
        sh = inputs["shape"]
        layer = moe.DeviceLayer(inputs, device="cuda:0")
        t = timed_median(layer.forward, steps)
        scrub = torch.ones(SCRUB_BYTES, dtype=torch.uint8, device="cuda:0")
        t_cold = cold_ms(layer.forward, lambda: probe.read(scrub), 20)
        del scrub
        events = [ev.create(nstep + 1) for _ in range(steps)]
        for i in range(steps):
            layer.forward_traced(events[i])
        torch.cuda.synchronize()
        split = np.array([[ev.elapsed_ms(e[j], e[j + 1]) for j in range(nstep)] for e in events]).mean(axis=0)
        for e in events:
            ev.destroy(e)
        offsets = layer.region(moe.MOE_REGION_OFFSETS, torch.int32, (sh.E_local + 1,)).cpu().numpy()
        n_loc = int(offsets[-1])
        active = int((np.diff(offsets) > 0).sum())
        d, F, Fs, T, k, E = sh.d, sh.F, sh.F_shared, sh.T, sh.top_k, sh.E
        gemm_flops = 6.0 * d * F * n_loc + 6.0 * d * Fs * T
        layer_flops = gemm_flops + 2.0 * T * d * E
        layer_bytes = (active * 3 * d * F * 2 + 3 * d * Fs * 2 + E * d * 2 + 2 * T * d * 2 + T * k * 8)
        s = {n: i for i, n in enumerate(moe.MOE_STEP_NAMES)}
        gemm_ms = sum(split[s[n]] for n in ("ffn_up", "ffn_down", "shared_up", "shared_down"))
        floor_ms = max(layer_flops / (PEAK_BF16_TFLOPS * 1e12), layer_bytes / (PEAK_HBM_GBS * 1e9)) * 1e3
        bound = "mfma" if layer_flops / (PEAK_BF16_TFLOPS * 1e12) >= layer_bytes / (PEAK_HBM_GBS * 1e9) else "hbm"
        rows.append({"workload": name, "T": T, "d": d, "E": E, "top_k": k, "E_local": sh.E_local, "F": F,
                     "F_shared": Fs, "local_rows": n_loc, "active_local_experts": active,
                     "layer_us": t * 1e3, "tokens_per_s": T / (t * 1e-3),
                     "gemm_us": float(gemm_ms * 1e3), "gemm_tflops": gemm_flops / (gemm_ms * 1e-3) / 1e12,
                     "gemm_frac_of_bf16_peak": gemm_flops / (gemm_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
                     "layer_hbm_gbs": layer_bytes / (t * 1e-3) / 1e9,
                     "layer_cold_us": t_cold * 1e3, "layer_hbm_gbs_cold": layer_bytes / (t_cold * 1e-3) / 1e9,
                     "layer_bound": bound, "layer_floor_us": floor_ms * 1e3,
                     "layer_frac_of_roofline": floor_ms / t,
                     "step_us": {n: round(float(split[i]) * 1e3, 2) for n, i in s.items()}})
        log(f"{name}: {t * 1e3:.1f} us per layer ({t_cold * 1e3:.1f} cold), {rows[-1]['tokens_per_s']:.3g} tokens/s, "
            f"GEMM {rows[-1]['gemm_tflops']:.0f} TFLOP/s, {rows[-1]['layer_hbm_gbs']:.0f} GB/s")
        del layer, inputs
        torch.cuda.empty_cache()
    return rows


def cpu_baseline(inputs, sample_tokens):
    """fp64 oracle (as it stands) on the first `sample_tokens` tokens: routing + expert MLPs + combine."""
    import numpy as np

    import oracle
    sh = inputs["shape"]
    n = min(sample_tokens, sh.T)
    blas = "unknown"
    try:
        from threadpoolctl import threadpool_info
        info = threadpool_info()
        cores = max([i.get("num_threads", 1) for i in info] or [1])
        blas = ", ".join(f"{i.get('internal_api')} {i.get('version')}" for i in info) or blas
    except Exception:  # pragma: no cover
        cores = len(os.sched_getaffinity(0))
    cpu_model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            cpu_model = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")), cpu_model)
    except OSError:  # pragma: no cover
        pass
    t0 = time.perf_counter()
    xd = oracle.bf16_to_f64(inputs["x"][:n])
    idx, w, _ = oracle.route(xd, oracle.bf16_to_f64(inputs["w_router"]), sh, inputs.get("bias"))
    out = oracle.expert_outputs_for_tokens(xd, idx, w, sh, inputs["w13"], inputs["w2"], inputs.get("ws13"),
                                           inputs.get("ws2"))
    dt = time.perf_counter() - t0
    assert np.isfinite(out).all()
    return {"value": n / dt, "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
            "cpu_model": cpu_model, "blas": blas, "host_cpus": len(os.sched_getaffinity(0)),
            "sample": f"first {n} of {sh.T} tokens of the same batch: fp64 routing, expert and shared SwiGLU "
                      f"MLPs and combine ({dt:.1f} s)"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    # an idle part needs ~30-40 DeepSeek-V3-sized layer steps (~50 ms of load) to reach its clock
    ap.add_argument("--warmup", type=int, default=40)
    ap.add_argument("--workload", default="dsv3")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-routed-gemm", action="store_true",
                    help="skip the routed-only grouped-MLP timing (it launches the layer's GEMM kernels "
                         "again, so kernel profiles of the layer pass this)")
    ap.add_argument("--cpu-sample", type=int, default=8192, help="tokens of the oracle CPU baseline sample")
    ap.add_argument("--crossover", action="store_true",
                    help="the paper's RQ4 kernel-crossover sweep (E=64, d=2048, F=1408, top-2, 8 local experts, "
                         "me = tokens per expert) instead of the layer benchmark")
    ap.add_argument("--masked-decode", action="store_true",
                    help="one decode step of --workload (default k2decode) in the offsets and the masked-decode "
                         "layout, eager and replayed from a HIP graph, instead of the layer benchmark")
    ap.add_argument("--fusion-matrix", action="store_true",
                    help="time the layer of --workload in the four fuse_gather x fuse_combine structures")
    ap.add_argument("--backward", action="store_true",
                    help="time the expert-MLP backward on one routed batch of --workload")
    ap.add_argument("--all-workloads", action="store_true",
                    help="time the layer on every workload (tiny, mixtral, dsv3, skewed, k2decode)")
    ap.add_argument("--dense-ref", action="store_true",
                    help="the DeepSeek-V3 shared expert as a dense MLP: the library's grouped GEMMs vs the vendor GEMM library")
    ap.add_argument("--layer-backward", action="store_true",
                    help="time the whole layer backward (moe_layer_backward) of --workload")
    ap.add_argument("--capacity", type=int, default=0,
                    help="expert capacity of --masked-decode (0: T, every slot kept)")
    ap.add_argument("--copy-ref-mib", type=int, default=0,
                    help="run one plain device copy of this many MiB first (reference dispatch for HBM counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this library runs one expert-parallel rank's share of the MoE layer on ONE "
                                   "GPU; --gpus must be 1 (the multi-GPU sharding is a design, not implemented)"}))
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2607_18631_amd import moe
    from paper_2607_18631_amd import workloads as wl

    torch.cuda.set_device(0)
    if args.crossover:
        rows = crossover_run()
        print(json.dumps({"metric": "per-token latency, kernel-crossover shape (E=64, d=2048, F=1408, top-2, "
                                    "8 local experts), 1 MI355X",
                          "unit": "us/token", "higher_is_better": False, "n_gpus": 1, "dtype": "bf16",
                          "data": "synthetic", "vs_baseline": None,
                          "protocol": "warmup 10 calls and >= 0.1 s; 200 calls per round for me < 16 else 50; median of 3 round "
                                      "medians; HIP events on the library's stream",
                          "rows": rows}), flush=True)
        return
    if args.masked_decode:
        workload = args.workload if args.workload != "dsv3" else "k2decode"
        sh0, C, rows, same = masked_decode_run(workload, args.capacity)
        print(json.dumps({"metric": "decode-step MoE-layer latency and HBM GB/s, offsets vs masked-decode layout, "
                                    "eager vs HIP-graph replay, 1 MI355X",
                          "unit": "us", "higher_is_better": False, "n_gpus": 1, "dtype": "bf16",
                          "data": "synthetic", "vs_baseline": None,
                          "config": {"workload": workload, "T": sh0.T, "d": sh0.d, "E": sh0.E, "top_k": sh0.top_k,
                                     "E_local": sh0.E_local, "F": sh0.F, "F_shared": sh0.F_shared,
                                     "expert_capacity": C},
                          "protocol": "warmup 10 calls and >= 0.1 s; 50 calls per round; median of 3 round medians; HIP events on "
                                      "the capturing stream",
                          "masked_equals_offsets_output": same,
                          "rows": rows}), flush=True)
        return
    if args.backward:
        sh, row = backward_run(args.workload, max(args.steps, 10))
        print(json.dumps({"metric": "expert-MLP backward (dX, dW13, dW2) latency and TFLOP/s, 1 MI355X",
                          "unit": "us", "higher_is_better": False, "n_gpus": 1, "dtype": "bf16",
                          "data": "synthetic", "vs_baseline": None,
                          "config": {"workload": args.workload, "T": sh.T, "d": sh.d, "E": sh.E, "top_k": sh.top_k,
                                     "E_local": sh.E_local, "F": sh.F},
                          "protocol": "warmup 10 calls and >= 0.1 s; median of 3 round medians of the per-call event times",
                          **row}), flush=True)
        return
    if args.all_workloads:
        rows = all_workloads_run(max(args.steps, 10))
        print(json.dumps({"metric": "MoE-layer tokens/s, grouped-GEMM TFLOP/s and layer HBM GB/s per workload, "
                                    "1 MI355X",
                          "unit": "tokens/s", "higher_is_better": True, "n_gpus": 1, "dtype": "bf16",
                          "data": "synthetic", "vs_baseline": None,
                          "protocol": "warmup 10 calls and >= 0.1 s; median of 3 round medians of the per-call event times; step "
                                      "split from traced calls; cold = median of 20 calls each right after a "
                                      "512 MiB read stream through the caches",
                          "peaks": {"bf16_tflops": PEAK_BF16_TFLOPS, "hbm_gbs": PEAK_HBM_GBS},
                          "rows": rows}), flush=True)
        return
    if args.dense_ref:
        row = dense_ref_run(max(args.steps, 10))
        print(json.dumps({"metric": "dense shared-expert MLP (DeepSeek-V3 shape): library grouped GEMMs vs vendor GEMM "
                                    "library, 1 MI355X", "unit": "TFLOP/s", "higher_is_better": True, "n_gpus": 1,
                          "dtype": "bf16", "data": "synthetic", "vs_baseline": None,
                          "protocol": "warmup 10 calls and >= 0.1 s; median of 3 round medians of the per-call event times", **row}),
              flush=True)
        return
    if args.layer_backward:
        sh, row = layer_backward_run(args.workload, max(args.steps, 10))
        print(json.dumps({"metric": "MoE-layer backward (dx, dw_router, expert and shared dW) latency and TFLOP/s, "
                                    "1 MI355X",
                          "unit": "us", "higher_is_better": False, "n_gpus": 1, "dtype": "bf16",
                          "data": "synthetic", "vs_baseline": None,
                          "config": {"workload": args.workload, "T": sh.T, "d": sh.d, "E": sh.E, "top_k": sh.top_k,
                                     "E_local": sh.E_local, "F": sh.F, "F_shared": sh.F_shared},
                          "protocol": "warmup 10 calls and >= 0.1 s; median of 3 round medians of the per-call event times",
                          **row}), flush=True)
        return
    if args.fusion_matrix:
        sh0, rows = fusion_matrix_run(args.workload, max(args.steps, 10))
        print(json.dumps({"metric": "MoE-layer latency per kernel structure (fuse_gather x fuse_combine), 1 MI355X",
                          "unit": "us", "higher_is_better": False, "n_gpus": 1, "dtype": "bf16",
                          "data": "synthetic", "vs_baseline": None,
                          "config": {"workload": args.workload, "T": sh0.T, "d": sh0.d, "E": sh0.E,
                                     "top_k": sh0.top_k, "E_local": sh0.E_local, "F": sh0.F,
                                     "F_shared": sh0.F_shared},
                          "protocol": "warmup 10 calls and >= 0.1 s; median of 3 round medians of the per-call event times; step "
                                      "split from traced calls",
                          "rows": rows}), flush=True)
        return
    log(f"generating inputs of workload {args.workload}")
    inputs = wl.make_inputs(args.workload)
    sh = inputs["shape"]
    layer = moe.DeviceLayer(inputs, device="cuda:0")
    torch.cuda.synchronize()
    if args.copy_ref_mib > 0:
        log(f"reference copy of {args.copy_ref_mib} MiB")
        src = torch.ones(args.copy_ref_mib << 20, dtype=torch.uint8, device="cuda:0")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    # The part's ceilings, measured before the layer (their ~0.5 s of load also brings an idle part
    # to its steady clock ahead of the warmup steps).  HBM: a 1 GiB device copy (bytes read +
    # written), a read-only stream (the probe kernel over 1 GiB) and a write-only stream (a 1 GiB fill)
    log("timing 1 GiB copy, read and fill streams")
    c_src = torch.ones(1 << 30, dtype=torch.uint8, device="cuda:0")
    c_dst = torch.empty_like(c_src)
    copy_ms = timed_median(lambda: c_dst.copy_(c_src), 10, warmup=3)
    probe = ReadProbe()
    read_ms = timed_median(lambda: probe.read(c_src), 10, warmup=3)
    fill_ms = timed_median(lambda: c_dst.zero_(), 10, warmup=3)
    del c_src, c_dst
    # practical MFMA ceiling: independent bf16 MFMAs on register operands on every SIMD (2 waves
    # each, as in the GEMM), a few ms per launch so that the clock settles under the load
    log("timing the MFMA loop probe")
    mfma_iters = 20000
    mfma_ms = timed_median(lambda: probe.mfma(mfma_iters), 5, warmup=2)
    mfma_tflops = probe.lib.probe_mfma_flops(mfma_iters) / (mfma_ms * 1e-3) / 1e12
    # LDS read ceiling: ds_read_b128 streams from LDS on every SIMD (2 waves each)
    log("timing the LDS read probe")
    lds_iters = 10000
    lds_ms = timed_median(lambda: probe.lds(lds_iters), 5, warmup=2)
    lds_tbs = probe.lib.probe_lds_bytes(lds_iters) / (lds_ms * 1e-3) / 1e12
    lds_clock = probe.lds_clock_ghz()

    ev = HipEvents()
    nstep = len(moe.MOE_STEP_NAMES)
    log(f"warmup {args.warmup} steps")
    for _ in range(args.warmup):
        layer.forward()
    torch.cuda.synchronize()

    # exactly K timed steps, bracketed by synchronisations.  Each recorded HIP event costs a few
    # microseconds of GPU time, so a timed step records only three, on the library's stream
    # (moe_layer_forward_traced with the other entries NULL): its start (the previous step's end)
    # and the two around the SwiGLU up-projection, the kernel the roofline object reports; one more
    # event closes the last step.
    # (A shared expert narrower or wider than the routed ones has an up-projection launch of its
    # own, bracketed the same way.)
    up_steps = [moe.MOE_STEP_NAMES.index("ffn_up")]
    if sh.F_shared > 0 and sh.F_shared != sh.F:
        up_steps.append(moe.MOE_STEP_NAMES.index("shared_up"))
    handles = [ev.create(1 + 2 * len(up_steps)) for _ in range(args.steps)]
    end_ev = ev.create(1)
    events = []
    for i in range(args.steps):
        arr = (ctypes.c_void_p * (nstep + 1))()
        arr[0] = handles[i][0]
        for u, j in enumerate(up_steps):
            arr[j], arr[j + 1] = handles[i][1 + 2 * u], handles[i][2 + 2 * u]
        if i == args.steps - 1:
            arr[nstep] = end_ev[0]
        events.append(arr)
    log(f"timing {args.steps} steps")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        layer.forward_traced(events[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    starts = [h[0] for h in handles] + [end_ev[0]]
    per_call = np.array([ev.elapsed_ms(starts[i], starts[i + 1]) for i in range(args.steps)])
    up_call = np.array([sum(ev.elapsed_ms(h[1 + 2 * u], h[2 + 2 * u]) for u in range(len(up_steps)))
                        for h in handles])
    for h in handles:
        ev.destroy(h)
    ev.destroy(end_ev)
    wall_ms_step = wall * 1e3 / args.steps
    # the paper's protocol on the timed steps: median over 3 rounds of each round's median
    rounds = np.array_split(np.arange(args.steps), min(3, args.steps))
    mrm = lambda v: float(np.median([np.median(v[r]) for r in rounds]))
    ms_step = mrm(per_call)

    # the split of a step into its launches, from separate fully traced steps after the timed ones
    # (every step boundary recorded; these steps run ~35 us longer than untraced ones at DSv3)
    log("tracing the step split")
    tr_events = [ev.create(nstep + 1) for _ in range(args.steps)]
    for i in range(args.steps):
        layer.forward_traced(tr_events[i])
    torch.cuda.synchronize()
    per_step = np.array([[ev.elapsed_ms(e[j], e[j + 1]) for j in range(nstep)] for e in tr_events])  # ms
    for e in tr_events:
        ev.destroy(e)
    step_med = np.array([mrm(per_step[:, j]) for j in range(nstep)])

    # standalone permutation (rank, placement and row copy), the form whose bytes the HBM figure
    # counts; inside the layer the row copy is folded into the up-projection
    log("timing the standalone permutation")
    T_, k_, cap_ = sh.T, sh.top_k, sh.capacity
    p_idx = layer.region(moe.MOE_REGION_TOPK_IDX, torch.int32, (T_, k_))
    p_counts = torch.empty(sh.E_local, dtype=torch.int32, device="cuda:0")
    p_offsets = torch.empty(sh.E_local + 1, dtype=torch.int32, device="cuda:0")
    p_row_token = torch.empty(cap_, dtype=torch.int32, device="cuda:0")
    p_slot_row = torch.empty((T_, k_), dtype=torch.int32, device="cuda:0")
    p_x_perm = torch.empty((cap_, sh.d), dtype=torch.bfloat16, device="cuda:0")
    p_ws = moe.alloc_workspace(sh, moe.MOE_WS_PERMUTE, "cuda:0")

    def permute_once():
        moe.moe_permute(sh, p_idx, layer.x, p_counts, p_offsets, p_row_token, p_slot_row, p_x_perm, p_ws)

    permute_ms = back_to_back_ms(permute_once, 50)
    # from HBM: back to back over rotating copies of the token rows and outputs (> the MALL)
    nrot = max(2, -(-ROTATE_BYTES // (2 * T_ * sh.d * 2)))
    r_x = [layer.x.clone() for _ in range(nrot)]
    r_xp = [torch.empty((cap_, sh.d), dtype=torch.bfloat16, device="cuda:0") for _ in range(nrot)]
    rot = [0]

    def permute_rot():
        i = rot[0] = (rot[0] + 1) % nrot
        moe.moe_permute(sh, p_idx, r_x[i], p_counts, p_offsets, p_row_token, p_slot_row, r_xp[i], p_ws)

    permute_hbm_ms = back_to_back_ms(permute_rot, 48)
    del r_x, r_xp

    # standalone combine on the layer's expert rows (warm: back to back; cold: after a scrub)
    log("timing the standalone combine")
    c_y = layer.region(moe.MOE_REGION_Y_PERM, torch.bfloat16, (cap_, sh.d))
    c_slot = layer.region(moe.MOE_REGION_SLOT_ROW, torch.int32, (T_, k_))
    c_w = layer.region(moe.MOE_REGION_TOPK_W, torch.float32, (T_, k_))
    c_sy = layer.region(moe.MOE_REGION_SHARED_Y, torch.bfloat16, (T_, sh.d)) if sh.F_shared > 0 else None
    c_out = torch.empty((T_, sh.d), dtype=torch.bfloat16, device="cuda:0")
    combine_once = lambda: moe.moe_combine(sh, c_y, c_slot, c_w, c_sy, c_out)
    combine_b2b_ms = back_to_back_ms(combine_once, 50)
    nrot_c = max(2, -(-ROTATE_BYTES // (3 * T_ * sh.d * 2)))
    r_y = [c_y.clone() for _ in range(nrot_c)]
    r_sy = [c_sy.clone() if c_sy is not None else None for _ in range(nrot_c)]
    r_out = [torch.empty((T_, sh.d), dtype=torch.bfloat16, device="cuda:0") for _ in range(nrot_c)]
    rot_c = [0]

    def combine_rot():
        i = rot_c[0] = (rot_c[0] + 1) % nrot_c
        moe.moe_combine(sh, r_y[i], c_slot, c_w, r_sy[i], r_out[i])

    combine_hbm_ms = back_to_back_ms(combine_rot, 48)
    del c_out, r_y, r_sy, r_out

    # the routed experts alone (moe_grouped_ffn on the permuted rows, no shared expert): the
    # routed-only grouped-GEMM figure; the shape describes exactly the batch's local rows
    n_routed = int(p_offsets[-1].item())
    routed_ms = None
    if n_routed > 0 and not args.no_routed_gemm:
        log("timing the routed grouped MLP alone")
        r_sh = sh.replace(T=n_routed, top_k=1, F_shared=0, fusion=0)
        r_y = torch.empty((n_routed, sh.d), dtype=torch.bfloat16, device="cuda:0")
        r_ws = moe.alloc_workspace(r_sh, moe.MOE_WS_FFN, "cuda:0")
        routed_ms = timed_median(lambda: moe.moe_grouped_ffn(r_sh, p_x_perm, p_offsets, layer.w13, layer.w2, r_y,
                                                             r_ws), 20)
        del r_y, r_ws
    del p_x_perm

    # algorithmic work of this batch (from the routing the GPU produced)
    offsets = layer.region(moe.MOE_REGION_OFFSETS, torch.int32, (sh.E_local + 1,)).cpu().numpy()
    slot_row = layer.region(moe.MOE_REGION_SLOT_ROW, torch.int32, (sh.T, sh.top_k)).cpu().numpy()
    out = layer.out.float()
    assert bool(torch.isfinite(out).all()), "non-finite layer output"
    n_loc = int(offsets[-1])
    tok_local = int((slot_row >= 0).any(axis=1).sum())
    d, F, Fs, T, k = sh.d, sh.F, sh.F_shared, sh.T, sh.top_k
    up_flops = 4.0 * d * F * n_loc + 4.0 * d * Fs * T
    gemm_flops = 6.0 * d * F * n_loc + 6.0 * d * Fs * T
    s = {name: i for i, name in enumerate(moe.MOE_STEP_NAMES)}
    # up-projection launch time(s) from the timed steps; a shared expert as wide as the routed ones
    # runs inside the routed launches
    up_ms = mrm(up_call)
    up_avg_ms = float(up_call.mean())
    up_launches = len(up_steps)
    gemm_ms = sum(step_med[s[n]] for n in ("ffn_up", "ffn_down", "shared_up", "shared_down"))
    perm_bytes = (tok_local + n_loc) * d * 2 + T * k * 8 + n_loc * 4
    comb_bytes = n_loc * d * 2 + (T * d * 2 if Fs > 0 else 0) + T * d * 2 + T * k * 8
    # whole-layer algorithmic HBM bytes (the decode-step figure): weights of the experts that
    # received rows, shared-expert and router weights, token rows in and out, routing arrays
    active = int((np.diff(offsets) > 0).sum())
    layer_bytes = (active * 3 * d * F * 2 + 3 * d * Fs * 2 + sh.E * d * 2 + 2 * T * d * 2
                   + T * k * 8)
    achieved = up_flops / (up_ms * 1e-3) / 1e12
    gbs = lambda by, ms: by / (ms * 1e-3) / 1e9
    res = {
        "metric": "MoE-layer tokens/s + grouped-GEMM TFLOP/s (% bf16 MFMA peak), 1 MI355X",
        "value": T / (ms_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": args.workload, "T": T, "d": d, "E": sh.E, "top_k": k, "E_local": sh.E_local,
                   "e_begin": sh.e_begin, "F": F, "F_shared": Fs, "gating": gating_desc(sh), "seed": inputs["seed"],
                   "local_rows": n_loc, "parallelism": "one expert-parallel rank's share on 1 GPU"},
        "protocol": (f"warmup {args.warmup} steps, then exactly {args.steps} timed steps recording HIP events "
                     "only at each step's start and around the up-projection launch; ms_per_step and the "
                     "roofline launch time = median over 3 rounds of the per-step medians; "
                     "wall_ms_per_step = synchronised wall clock of the timed steps / steps; step_ms from "
                     "separately traced steps after the timed ones (every step boundary recorded)"),
        "wall_ms_per_step": wall_ms_step,
        "gemm_tflops": gemm_flops / (gemm_ms * 1e-3) / 1e12,
        "gemm_frac_of_bf16_peak": gemm_flops / (gemm_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
        "routed_gemm_ms": routed_ms,
        "routed_gemm_tflops": (6.0 * d * F * n_loc / (routed_ms * 1e-3) / 1e12) if routed_ms else None,
        "permute_gbs": gbs(perm_bytes, permute_ms),
        "permute_ms": permute_ms,
        "permute_hbm_gbs": gbs(perm_bytes, permute_hbm_ms),
        "permute_in_layer": "row copy folded into the up-projection (token rows read through row_token)",
        "combine_gbs": gbs(comb_bytes, step_med[s["combine"]]),
        "combine_b2b_gbs": gbs(comb_bytes, combine_b2b_ms),
        "combine_hbm_gbs": gbs(comb_bytes, combine_hbm_ms),
        "hbm_bytes": {"permute": perm_bytes, "combine": comb_bytes, "layer": layer_bytes},
        "copy_gbs": 2.0 * (1 << 30) / (copy_ms * 1e-3) / 1e9,
        "read_gbs": (1 << 30) / (read_ms * 1e-3) / 1e9,
        "fill_gbs": (1 << 30) / (fill_ms * 1e-3) / 1e9,
        "mfma_loop_tflops": mfma_tflops,
        "mfma_loop_clock_ghz": mfma_tflops / PEAK_BF16_TFLOPS * 2.4,
        "lds_read_tbs": lds_tbs,
        "lds_read_bytes_per_clk_cu": lds_tbs * 1e12 / (256 * lds_clock * 1e9),
        "lds_probe_clock_ghz": lds_clock,
        "layer_hbm_gbs": layer_bytes / (ms_step * 1e-3) / 1e9,
        "active_local_experts": active,
        "step_ms": {n: round(float(step_med[i]), 5) for n, i in s.items()},
        "gpu_event_ms_per_step": float(per_call.mean()),
        "roofline": {
            "kernel": "k_grouped_gemm<EPI_SWIGLU> (W1/W3 GEMM + SwiGLU of the routed experts and the shared expert)",
            "bound": "mfma",
            "achieved": achieved,
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": achieved / PEAK_BF16_TFLOPS,
            "traffic": measured_traffic(args.workload),
            "launches_per_step": up_launches,
            "launch_ms": float(up_ms / up_launches),
            "avg_launch_ms": float(up_avg_ms / up_launches),
            "flops_per_step": up_flops,
        },
    }
    if not args.no_cpu_baseline:
        log(f"cpu baseline: oracle on {args.cpu_sample} tokens")
        res["cpu_baseline"] = cpu_baseline(inputs, args.cpu_sample)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
