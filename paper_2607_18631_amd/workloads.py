"""Seeded synthetic workloads for the MoE-layer forward.

This module only *describes* shapes and *draws* inputs.  It holds none of the
layer's arithmetic, so both the HIP path and the fp64 oracle can take their
inputs from it without sharing any computation.

Shapes follow the MoE-layer vocabulary of the paper's kernel study (hidden size,
expert count, top-k, local-expert slice, expert FFN width; Section 5, RQ4 and the
appendix's kernel-crossover protocol).  The five workloads are:

  tiny      T=256   d=512  E=8   top-2 softmax, F=1024, all local
  mixtral   T=4096  d=4096 E=8   top-2 softmax, F=14336, all local
  dsv3      T=8192  d=7168 E=256 top-8 sigmoid, 8 groups / top-4 groups,
            gates renormalised and scaled by 2.5, 32 local experts of F=2048
            plus one shared expert of width 2048 (one rank of an EP8 layout)
  skewed    T=16384 d=2048 E=128 top-8 softmax with a Zipf(1.2) router bias,
            F=768, all local
  k2decode  T=64    d=7168 E=384 top-8 sigmoid, 48 local experts of F=2048 plus
            one shared expert of width 2048 (one decode step of one EP8 rank)

The kernel-crossover workload of the paper's RQ4 figure (``crossover(me)``): E=64
experts of width F=1408 on hidden size d=2048, top-2 softmax gating (renormalised), one
rank holding 8 local experts (world size 8); ``me`` is the expert multiplicity (tokens per
expert), the batch has me * E / top_k tokens, and per-token latency is quoted over that
global token count.  ``CROSSOVER_ME`` lists the multiplicities the figure reports.

Input recipe (all seeded, synthetic):
  * every tensor is drawn as float32 N(0, std) from its own numpy PCG64 stream
    ``SeedSequence(seed, spawn_key=(tensor_id, index))`` and rounded to bf16 with
    round-to-nearest-even; expert tensors use one stream per expert, so one
    expert can be regenerated on its own;
  * x ~ N(0, 1); expert W1/W3 (and shared) ~ N(0, 1/sqrt(d)); W2 ~ N(0, 1/sqrt(F));
  * router ~ N(0, 0.02) for ``tiny``, N(0, 1/sqrt(d)) otherwise, except ``skewed``
    which uses N(0, 2/sqrt(d)) so that the Zipf bias gives a 10-50x hot/cold load
    ratio instead of a several-hundred-fold one;
  * the ``skewed`` bias is ``bias[e] = ln(w[pi(e)])`` with ``w[r] = (r+1)^-1.2`` and
    ``pi`` a seeded permutation of the experts.

bf16 tensors are returned as ``uint16`` bit patterns (row-major, contiguous).
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

GATE_SOFTMAX = 0
GATE_SIGMOID = 1
# kernel structure of the layer forward (values of the C ABI's MOE_FUSION_SET / MOE_FUSE_*)
FUSION_SET = 0x10
FUSE_GATHER = 0x1
FUSE_COMBINE = 0x2
FUSION_VARIANTS = {"unfused": FUSION_SET, "gather": FUSION_SET | FUSE_GATHER,
                   "combine": FUSION_SET | FUSE_COMBINE, "both": FUSION_SET | FUSE_GATHER | FUSE_COMBINE}

# stream ids of the per-tensor generators
_TID_X, _TID_ROUTER, _TID_W1, _TID_W3, _TID_W2 = 0, 1, 2, 3, 4
_TID_WS1, _TID_WS3, _TID_WS2, _TID_BIAS = 5, 6, 7, 8


@dataclasses.dataclass(frozen=True)
class MoEShape:
    """Shape and gating description of one MoE layer on one expert-parallel rank."""
    T: int                 # tokens
    d: int                 # hidden size (the GEMM K of the up projection)
    E: int                 # routed experts in the whole layer
    top_k: int             # experts per token
    F: int                 # routed expert FFN width
    E_local: int           # experts held by this rank: [e_begin, e_begin + E_local)
    e_begin: int = 0
    F_shared: int = 0      # shared-expert FFN width (0 = no shared expert)
    gate: int = GATE_SOFTMAX
    n_group: int = 1       # expert groups for group-limited routing (1 = off)
    topk_group: int = 1    # groups kept per token when n_group > 1
    renormalize: int = 1   # renormalise gates over the chosen experts
    routed_scale: float = 1.0
    expert_capacity: int = 0   # > 0: masked-decode layout, rows [e C, e C + C) per local expert
    fusion: int = 0        # kernel structure of the layer forward (0 = default; see FUSION_VARIANTS)

    def replace(self, **kw) -> "MoEShape":
        return dataclasses.replace(self, **kw)

    @property
    def capacity(self) -> int:
        """Rows of the permuted buffers: T * min(top_k, E_local), or E_local * expert_capacity."""
        if self.expert_capacity > 0:
            return self.E_local * self.expert_capacity
        return self.T * min(self.top_k, self.E_local)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    shape: MoEShape
    router_std: float
    x_std: float = 1.0
    zipf_s: float = 0.0    # > 0: router bias from Zipf(zipf_s) weights
    seed: int = 0


WORKLOADS = {
    "tiny": Workload("tiny", MoEShape(T=256, d=512, E=8, top_k=2, F=1024, E_local=8),
                     router_std=0.02),
    "mixtral": Workload("mixtral", MoEShape(T=4096, d=4096, E=8, top_k=2, F=14336, E_local=8),
                        router_std=4096 ** -0.5),
    "dsv3": Workload("dsv3", MoEShape(T=8192, d=7168, E=256, top_k=8, F=2048, E_local=32,
                                      F_shared=2048, gate=GATE_SIGMOID, n_group=8,
                                      topk_group=4, renormalize=1, routed_scale=2.5),
                     router_std=7168 ** -0.5),
    "skewed": Workload("skewed", MoEShape(T=16384, d=2048, E=128, top_k=8, F=768, E_local=128),
                       router_std=2.0 * 2048 ** -0.5, zipf_s=1.2),
    "k2decode": Workload("k2decode", MoEShape(T=64, d=7168, E=384, top_k=8, F=2048, E_local=48,
                                              F_shared=2048, gate=GATE_SIGMOID),
                         router_std=7168 ** -0.5),
}


# kernel-crossover workload (the paper's RQ4 figure; me = 512 is absent from its data)
CROSSOVER_ME = (2, 4, 8, 16, 32, 64, 128, 256, 1024)


def crossover(me: int) -> Workload:
    """The kernel-crossover shape at expert multiplicity ``me`` (me * 64 / 2 global tokens)."""
    E, top_k = 64, 2
    return Workload(f"crossover_me{me}", MoEShape(T=me * E // top_k, d=2048, E=E, top_k=top_k, F=1408,
                                                  E_local=8), router_std=2048 ** -0.5)


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (round to nearest, ties to even); returns uint16 bits.

    Inputs here are finite; NaN is not special-cased.
    """
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    return ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)


def _stream(seed: int, tid: int, index: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=(tid, index))))


def _normal_bf16(seed: int, tid: int, index: int, shape, std: float, out: np.ndarray | None = None):
    g = _stream(seed, tid, index)
    v = g.standard_normal(int(np.prod(shape)), dtype=np.float32)
    v *= np.float32(std)
    bits = f32_to_bf16_bits(v).reshape(shape)
    if out is not None:
        out[...] = bits
        return out
    return bits


def zipf_bias(E: int, s: float, seed: int) -> np.ndarray:
    """Per-expert router bias: log of Zipf(s) weights over a seeded expert order."""
    perm = _stream(seed, _TID_BIAS, 0).permutation(E)
    return (-s * np.log(perm.astype(np.float64) + 1.0)).astype(np.float32)


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def expert_tensors(wl: Workload | str, le: int, seed: int | None = None, out13=None, out2=None):
    """bf16 bits of local expert ``le``'s weights: ``w13 [2F, d]`` (rows [0,F) = W1 gate, rows
    [F,2F) = W3 up) and ``w2 [d, F]``, drawn from the streams of global expert e_begin + le."""
    if isinstance(wl, str):
        wl = WORKLOADS[wl]
    sh = wl.shape
    seed = wl.seed if seed is None else seed
    d, F = sh.d, sh.F
    ge = sh.e_begin + le
    w13 = np.empty((2 * F, d), np.uint16) if out13 is None else out13
    w2 = np.empty((d, F), np.uint16) if out2 is None else out2
    _normal_bf16(seed, _TID_W1, ge, (F, d), d ** -0.5, w13[:F])
    _normal_bf16(seed, _TID_W3, ge, (F, d), d ** -0.5, w13[F:])
    _normal_bf16(seed, _TID_W2, ge, (d, F), F ** -0.5, w2)
    return w13, w2


def shared_tensors(wl: Workload | str, seed: int | None = None):
    """bf16 bits of the shared expert's weights ``ws13 [2F_s, d]`` and ``ws2 [d, F_s]`` (None, None
    without a shared expert)."""
    if isinstance(wl, str):
        wl = WORKLOADS[wl]
    sh = wl.shape
    seed = wl.seed if seed is None else seed
    d, Fs = sh.d, sh.F_shared
    if Fs <= 0:
        return None, None
    ws13 = np.empty((2 * Fs, d), np.uint16)
    ws2 = np.empty((d, Fs), np.uint16)
    _normal_bf16(seed, _TID_WS1, 0, (Fs, d), d ** -0.5, ws13[:Fs])
    _normal_bf16(seed, _TID_WS3, 0, (Fs, d), d ** -0.5, ws13[Fs:])
    _normal_bf16(seed, _TID_WS2, 0, (d, Fs), Fs ** -0.5, ws2)
    return ws13, ws2


def make_inputs(wl: Workload | str, T: int | None = None, seed: int | None = None,
                with_experts: bool = True) -> dict:
    """Draw every input of workload ``wl`` (optionally with a different token count).

    Returns a dict with uint16 bf16 bit arrays ``x[T,d]``, ``w_router[E,d]``,
    ``w13[E_local,2F,d]`` (rows [0,F) = W1 gate, rows [F,2F) = W3 up),
    ``w2[E_local,d,F]``, ``ws13[2F_s,d]``/``ws2[d,F_s]`` (or None), the float32
    ``bias[E]`` (or None) and the shape under ``shape``.
    """
    if isinstance(wl, str):
        wl = WORKLOADS[wl]
    sh = wl.shape if T is None else wl.shape.replace(T=T)
    seed = wl.seed if seed is None else seed
    d, F = sh.d, sh.F
    out = {"shape": sh, "workload": wl.name, "seed": seed}
    jobs = []
    out["x"] = np.empty((sh.T, d), np.uint16)
    jobs.append(lambda: _normal_bf16(seed, _TID_X, 0, (sh.T, d), wl.x_std, out["x"]))
    out["w_router"] = np.empty((sh.E, d), np.uint16)
    jobs.append(lambda: _normal_bf16(seed, _TID_ROUTER, 0, (sh.E, d), wl.router_std, out["w_router"]))
    out["bias"] = zipf_bias(sh.E, wl.zipf_s, seed) if wl.zipf_s > 0 else None
    if with_experts:
        w13 = np.empty((sh.E_local, 2 * F, d), np.uint16)
        w2 = np.empty((sh.E_local, d, F), np.uint16)
        for le in range(sh.E_local):
            jobs.append(lambda le=le: expert_tensors(wl, le, seed, w13[le], w2[le]))
        out["w13"], out["w2"] = w13, w2
        shared = {}
        jobs.append(lambda: shared.update(zip(("ws13", "ws2"), shared_tensors(wl, seed))))
    with ThreadPoolExecutor(_threads()) as ex:
        for f in [ex.submit(j) for j in jobs]:
            f.result()
    if with_experts:
        out["ws13"], out["ws2"] = shared["ws13"], shared["ws2"]
    return out


def custom_inputs(shape: MoEShape, seed: int = 0, router_std: float | None = None,
                  zipf_s: float = 0.0) -> dict:
    """Inputs for an arbitrary shape (edge-case tests), with the default recipe."""
    wl = Workload("custom", shape, router_std=shape.d ** -0.5 if router_std is None else router_std,
                  zipf_s=zipf_s, seed=seed)
    return make_inputs(wl)
