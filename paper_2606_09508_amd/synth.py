"""Seeded synthetic single-layer prefill workloads.

This module only draws random bf16 tensors with planted structure; it holds
none of the method's arithmetic (no pooling, softmax, entropy, budget or
attention), so that the HIP path and the CPU oracle can both be fed the same
bytes from it.

Every tensor is drawn per (tensor, batch, head) from
``numpy.random.default_rng([seed, tensor_code, b, h])`` as float32 and rounded
to bf16 with round-to-nearest-even, so any head can be regenerated alone.

Planted structure uses the last three head dimensions:

* SINK (dim D-1): every key of key block 0 carries ``C_K = sqrt(D)`` there and
  every other key 0; a query of a *sink* region carries ``C_Q = 8``.  A sink
  query's raw dot product with each block-0 key therefore gains 8 sqrt(D),
  i.e. +8 after the 1/sqrt(D) attention scale.
* ROT (dims D-3, D-2): keys carry ``a (cos w t, sin w t)`` at position t; a
  *local* query carries the same pair, adding ``a^2 cos(w (i - t))`` to its
  raw dot products, a smooth local window.
* *diffuse* queries are the Gaussian part scaled by 0.25.

Workloads (shapes of the layers the paper evaluates, Section 5):

* ``c1`` tiny: B=1, Hq=4, Hkv=1, N=1024; heads 0-1 sink + local in every
  segment, heads 2-3 plain N(0, 1); L_S=128, L_B=64, B_h=256 (25% of blocks).
* ``c2`` Llama-3-8B layer at 32k: Hq=32, Hkv=8, N=32768; 2048-token regions;
  a quarter of the heads are sink in every region, the rest draw
  sink / local / diffuse per region with probabilities 0.2 / 0.4 / 0.4.
* ``c3`` the same layer at 131072 tokens with 8192-token regions.
* ``c4`` Qwen2.5-7B layer: Hq=28, Hkv=4 (GQA 7:1), N=65536; key rows scaled by
  LogNormal(0, 0.5); 10 retrieval spans (length U[32, 128], before the last
  segment) whose keys point along a per-group direction that the final
  segment's queries also carry.
* ``c5`` Llama-3-70B layer on one GPU: Hq=64, Hkv=8, N=131072; an eighth of
  the heads sink everywhere, the others drift between types over 8192-token
  regions as a Markov chain with stay probability 0.75.  The always-sink heads
  carry sink amplitudes spread evenly from 8.25 down to 7.25 (in head order),
  so that their largest segment entropies straddle the three entropy
  thresholds the workload is swept over (1e-6, 1e-5, 1e-4).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field, replace

import numpy as np


_T_Q, _T_K, _T_V, _T_PLAN, _T_SPAN = 1, 2, 3, 4, 5


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round to nearest even."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def from_bf16_bits(h: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> float32 (exact)."""
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclass
class Workload:
    name: str
    seed: int
    B: int
    Hq: int
    Hkv: int
    N: int
    D: int
    Ls: int
    Lb: int
    base_budget: int
    mult: int = 3
    e_t: float = 1e-5
    alpha: float = 0.5
    delta_t: float = 0.4
    probe_scale: float = 1.0
    recipe: str = "regions"
    region: int = 2048
    always_sink_frac: float = 0.25
    p_types: tuple = (0.2, 0.4, 0.4)
    markov_stay: float = 0.0
    key_lognormal: float = 0.0
    n_spans: int = 0
    sink_amp: tuple | None = None   # (first, last) C_Q of the always-sink heads
    q: np.ndarray | None = field(default=None, repr=False)
    k: np.ndarray | None = field(default=None, repr=False)
    v: np.ndarray | None = field(default=None, repr=False)
    plan: np.ndarray | None = field(default=None, repr=False)   # [B, Hq, n_regions] type codes
    spans: list = field(default_factory=list, repr=False)

    @property
    def softmax_scale(self) -> float:
        return 1.0 / math.sqrt(self.D)

    @property
    def CS(self) -> int:
        return -(-self.N // self.Ls)

    @property
    def CB(self) -> int:
        return -(-self.N // self.Lb)

    @property
    def kmax(self) -> int:
        return (self.mult * self.base_budget) // self.Lb + self.Ls // self.Lb

    def region_of_segment(self, s: int) -> int:
        return (s * self.Ls) // self.region


PRESETS = {
    "c1": dict(B=1, Hq=4, Hkv=1, N=1024, D=128, Ls=128, Lb=64, base_budget=256, recipe="c1",
               region=1024),
    "c2": dict(B=1, Hq=32, Hkv=8, N=32768, D=128, Ls=128, Lb=64, base_budget=2048,
               recipe="regions", region=2048),
    "c3": dict(B=1, Hq=32, Hkv=8, N=131072, D=128, Ls=128, Lb=64, base_budget=2048,
               recipe="regions", region=8192),
    "c4": dict(B=1, Hq=28, Hkv=4, N=65536, D=128, Ls=128, Lb=64, base_budget=2048,
               recipe="regions", region=2048, key_lognormal=0.5, n_spans=10),
    "c5": dict(B=1, Hq=64, Hkv=8, N=131072, D=128, Ls=128, Lb=64, base_budget=2048,
               recipe="regions", region=8192, always_sink_frac=0.125, markov_stay=0.75,
               sink_amp=(8.25, 7.25)),
}

# type codes used in Workload.plan
SINK, LOCAL, DIFFUSE, GAUSS = 0, 1, 2, 3

C_Q = 8.0
ROT_PERIOD = 512.0
A_LOCAL_C1 = 3.0      # a^2 = 9 raw: a local window well under the sink's 8 sqrt(D)
A_LOCAL = 6.0         # a^2 = 36 raw in the region workloads


def _rng(seed: int, code: int, b: int, h: int) -> np.random.Generator:
    return np.random.default_rng([int(seed), code, int(b), int(h)])


def _plan(w: Workload) -> np.ndarray:
    n_regions = -(-w.N // w.region)
    plan = np.empty((w.B, w.Hq, n_regions), np.int8)
    rng = _rng(w.seed, _T_PLAN, 0, 0)
    for b in range(w.B):
        if w.recipe == "c1":
            plan[b, :] = GAUSS
            plan[b, : min(2, w.Hq)] = SINK
            continue
        if w.recipe == "gauss":
            plan[b, :] = GAUSS
            continue
        n_sink = int(round(w.always_sink_frac * w.Hq))
        always = rng.permutation(w.Hq)[:n_sink]
        for h in range(w.Hq):
            if h in always:
                plan[b, h, :] = SINK
                continue
            if w.markov_stay > 0:
                t = rng.choice(3, p=np.asarray(w.p_types) / np.sum(w.p_types))
                for r in range(n_regions):
                    if r > 0 and rng.random() >= w.markov_stay:
                        t = rng.choice([x for x in range(3) if x != t])
                    plan[b, h, r] = t
            else:
                plan[b, h, :] = rng.choice(3, size=n_regions,
                                           p=np.asarray(w.p_types) / np.sum(w.p_types))
    return plan


def _rot(N: int, amp: float) -> np.ndarray:
    t = np.arange(N, dtype=np.float64)
    ang = 2.0 * math.pi * t / ROT_PERIOD
    return (amp * np.stack([np.cos(ang), np.sin(ang)], axis=1)).astype(np.float32)


def _span_plan(w: Workload):
    """Retrieval spans: (start, length) pairs and a unit direction per (b, g)."""
    if w.n_spans <= 0:
        return [], None
    rng = _rng(w.seed, _T_SPAN, 0, 0)
    spans = []
    hi = max(w.Lb + 1, w.N - w.Ls - 128)
    for _ in range(w.n_spans):
        ln = int(rng.integers(32, 129))
        st = int(rng.integers(w.Lb, max(w.Lb + 1, hi - ln)))
        spans.append((st, ln))
    dirs = rng.standard_normal((w.B, w.Hkv, w.D - 3)).astype(np.float32)
    dirs /= np.linalg.norm(dirs, axis=-1, keepdims=True)
    return spans, dirs


def sink_amplitudes(w: Workload) -> np.ndarray:
    """[B, Hq] query sink amplitude of every head (C_Q unless ``sink_amp``
    spreads the always-sink heads' amplitudes)."""
    amp = np.full((w.B, w.Hq), C_Q, np.float64)
    if w.sink_amp is None or w.plan is None:
        return amp
    for b in range(w.B):
        always = [h for h in range(w.Hq) if (w.plan[b, h] == SINK).all()]
        n = len(always)
        for i, h in enumerate(always):
            f = i / (n - 1) if n > 1 else 0.0
            amp[b, h] = w.sink_amp[0] + (w.sink_amp[1] - w.sink_amp[0]) * f
    return amp


def generate(w: Workload, heads_q=None) -> Workload:
    """Fill w.q, w.k, w.v (uint16 bf16 bits, [B, H, N, D]) in place and return w.

    heads_q: optional iterable of query heads to draw (others stay zero) for
    oracle-side sampling of very large workloads; keys and values are always
    drawn in full.
    """
    B, Hq, Hkv, N, D = w.B, w.Hq, w.Hkv, w.N, w.D
    G = Hq // Hkv
    w.plan = _plan(w)
    amp = sink_amplitudes(w)
    spans, dirs = _span_plan(w)
    w.spans = spans
    rot_c1 = _rot(N, A_LOCAL_C1)
    rot = _rot(N, A_LOCAL)
    c_k = float(np.sqrt(D))
    w.k = np.empty((B, Hkv, N, D), np.uint16)
    w.v = np.empty((B, Hkv, N, D), np.uint16)
    w.q = np.zeros((B, Hq, N, D), np.uint16)
    for b in range(B):
        for g in range(Hkv):
            x = _rng(w.seed, _T_K, b, g).standard_normal((N, D), dtype=np.float32)
            if w.key_lognormal > 0:
                s = _rng(w.seed, _T_K, b, g + 100000).lognormal(0.0, w.key_lognormal, size=(N, 1))
                x[:, : D - 3] *= s.astype(np.float32)
            x[:, D - 1] = 0.0
            x[: min(w.Lb, N), D - 1] = c_k
            x[:, D - 3: D - 1] = rot_c1 if w.recipe == "c1" else rot
            for (st, ln) in spans:
                e = min(N, st + ln)
                noise = _rng(w.seed, _T_SPAN, b, 1000 + g).standard_normal((e - st, D - 3))
                x[st:e, : D - 3] = 0.5 * noise.astype(np.float32) + 27.0 * dirs[b, g]
            w.k[b, g] = to_bf16_bits(x)
            w.v[b, g] = to_bf16_bits(_rng(w.seed, _T_V, b, g).standard_normal((N, D),
                                                                               dtype=np.float32))
        want = range(Hq) if heads_q is None else heads_q
        for h in want:
            x = _rng(w.seed, _T_Q, b, h).standard_normal((N, D), dtype=np.float32)
            x[:, D - 3:] = 0.0
            for r in range(w.plan.shape[2]):
                r0, r1 = r * w.region, min(N, (r + 1) * w.region)
                t = int(w.plan[b, h, r])
                if t == SINK:
                    x[r0:r1, D - 1] = amp[b, h]
                    if w.recipe == "c1":
                        x[r0:r1, D - 3: D - 1] = rot_c1[r0:r1]
                elif t == LOCAL:
                    x[r0:r1, D - 3: D - 1] = rot[r0:r1]
                elif t == DIFFUSE:
                    x[r0:r1, : D - 3] *= 0.25
            if spans:
                x[max(0, N - w.Ls):, : D - 3] += 2.5 * dirs[b, h // G]
            w.q[b, h] = to_bf16_bits(x)
    return w


def make(name: str, seed: int = 0, generate_tensors: bool = True, heads_q=None,
         **overrides) -> Workload:
    """A preset workload (``c1`` .. ``c5``), optionally with fields overridden."""
    if name not in PRESETS:
        raise KeyError(f"unknown workload {name!r}; presets: {sorted(PRESETS)}")
    params = dict(PRESETS[name])
    params.update(overrides)
    w = Workload(name=name, seed=seed, **params)
    if w.Hq % w.Hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    return generate(w, heads_q=heads_q) if generate_tensors else w


def with_fields(w: Workload, **kw) -> Workload:
    """A copy sharing the tensors with some scalar fields changed."""
    return replace(w, **kw)
