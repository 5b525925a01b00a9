"""Multi-layer prefill with the entropy-guided sparse attention as a drop-in.

A Llama-3-8B-shaped decoder (random bf16 weights, no checkpoint) runs its
prefill with the attention of every layer computed by this library: the
entropy probe, head classification / budgets / top-k selection and the
block-sparse kernel, in the library's one call (``attn="sparse"``), or the
dense causal kernel
(``attn="dense"``, the full-attention baseline).  Everything around the
attention is the ordinary decoder layer -- RMSNorm, the Q/K/V/O projections,
rotary position embedding, the SwiGLU MLP -- on PyTorch (the projections and
MLP are plain library GEMMs); it is the harness that gives time-to-first-token
(TTFT) against prompt length, the end-to-end setting of Section 5's latency
study, and carries no part of the method.

    python -m paper_2606_09508_amd.prefill --ttft      # markdown table on stdout
"""
from __future__ import annotations

import argparse
import math
import sys
import time
from dataclasses import dataclass

import torch

from . import binding as eb


@dataclass(frozen=True)
class DecoderShape:
    hidden: int = 4096
    n_q_heads: int = 32
    n_kv_heads: int = 8
    head_dim: int = 128
    intermediate: int = 14336
    n_layers: int = 32
    vocab: int = 128256
    rope_theta: float = 500000.0
    rms_eps: float = 1e-5


LLAMA3_8B = DecoderShape()


@dataclass
class SparseConfig:
    seg_len: int = 128
    block_len: int = 64
    base_budget: int = 2048
    entropy_threshold: float = 1e-5
    alpha: float = 0.5
    delta_t: float = 0.4
    mult: int = 3
    probe_scale: float = 1.0
    mode: int = eb.CLASSIFY_HEAD


def make_weights(shape: DecoderShape, n_layers: int, seed: int, device) -> list[dict]:
    """Random bf16 weights, N(0, 1/fan_in) so that activations keep their
    scale through the layers; norm gains are ones."""
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    H, D = shape.hidden, shape.head_dim

    def w(n_in, n_out):
        return (torch.randn((n_in, n_out), generator=g, device=device, dtype=torch.float32)
                * (1.0 / math.sqrt(n_in))).to(torch.bfloat16)

    layers = []
    for _ in range(n_layers):
        layers.append({
            "wq": w(H, shape.n_q_heads * D), "wk": w(H, shape.n_kv_heads * D),
            "wv": w(H, shape.n_kv_heads * D), "wo": w(shape.n_q_heads * D, H),
            "w_gate": w(H, shape.intermediate), "w_up": w(H, shape.intermediate),
            "w_down": w(shape.intermediate, H),
            "norm1": torch.ones(H, device=device, dtype=torch.bfloat16),
            "norm2": torch.ones(H, device=device, dtype=torch.bfloat16),
        })
    return layers


def rope_tables(N: int, D: int, theta: float, device):
    """cos / sin [N, D/2] (fp32) of the rotary embedding, half-split layout."""
    inv = 1.0 / (theta ** (torch.arange(0, D, 2, device=device, dtype=torch.float32) / D))
    ang = torch.arange(N, device=device, dtype=torch.float32)[:, None] * inv[None, :]
    return torch.cos(ang), torch.sin(ang)


def _rmsnorm(x, gain, eps):
    xf = x.float()
    return (xf * torch.rsqrt(xf.pow(2).mean(-1, keepdim=True) + eps) * gain.float()).to(x.dtype)


def _rope(x, cos, sin):
    """x [B, H, N, D] bf16 -> rotated bf16 (pairs (i, i + D/2))."""
    xf = x.float()
    h = xf.shape[-1] // 2
    a, b = xf[..., :h], xf[..., h:]
    return torch.cat([a * cos - b * sin, a * sin + b * cos], dim=-1).to(x.dtype)


class Attention:
    """The attention of one layer through the C ABI, with its buffers."""

    def __init__(self, shape: DecoderShape, B: int, N: int, kind: str, cfg: SparseConfig,
                 device):
        self.shape, self.kind, self.cfg = shape, kind, cfg
        self.scale = 1.0 / math.sqrt(shape.head_dim)
        self.out = torch.empty((B, shape.n_q_heads, N, shape.head_dim), dtype=torch.bfloat16,
                               device=device)
        self.bufs = {"out": self.out}   # buffers of the one-call sparse path
        self.sel = None                  # the last selection (sparse)
        if kind not in ("sparse", "dense"):
            raise ValueError("attention kind must be 'sparse' or 'dense'")

    def __call__(self, q, k, v):
        c = self.cfg
        if self.kind == "dense":
            return eb.dense_prefill_attn(q, k, v, self.scale, True, self.out)
        o, self.sel, _, _ = eb.entropy_guided_prefill(
            q, k, v, c.seg_len, c.block_len, c.base_budget, c.entropy_threshold, c.alpha,
            c.delta_t, c.mult, c.probe_scale, self.scale, bufs=self.bufs, mode=c.mode)
        return o


def layer_forward(x, w, shape: DecoderShape, attn: Attention, cos, sin, trace=None):
    """One decoder layer on x [B, N, hidden] bf16; returns the new hidden
    state.  trace (optional dict) receives the attention inputs and output."""
    B, N, _ = x.shape
    Hq, Hkv, D = shape.n_q_heads, shape.n_kv_heads, shape.head_dim
    h = _rmsnorm(x, w["norm1"], shape.rms_eps)
    q = (h @ w["wq"]).view(B, N, Hq, D).transpose(1, 2).contiguous()
    k = (h @ w["wk"]).view(B, N, Hkv, D).transpose(1, 2).contiguous()
    v = (h @ w["wv"]).view(B, N, Hkv, D).transpose(1, 2).contiguous()
    q, k = _rope(q, cos, sin), _rope(k, cos, sin)
    o = attn(q, k, v)
    if trace is not None:
        trace.update(q=q.clone(), k=k.clone(), v=v.clone(), o=o.clone())
    x = x + o.transpose(1, 2).reshape(B, N, Hq * D) @ w["wo"]
    h = _rmsnorm(x, w["norm2"], shape.rms_eps)
    x = x + (torch.nn.functional.silu(h @ w["w_gate"]) * (h @ w["w_up"])) @ w["w_down"]
    return x


def prefill(x, layers, shape: DecoderShape, attn: Attention, lm_head=None):
    """All layers over the prompt's hidden states x [B, N, hidden]; returns the
    final normed hidden state of the last token (and its logits when an LM
    head [hidden, vocab] is given) -- what the first generated token needs."""
    N = x.shape[1]
    cos, sin = rope_tables(N, shape.head_dim, shape.rope_theta, x.device)
    for w in layers:
        x = layer_forward(x, w, shape, attn, cos, sin)
    last = _rmsnorm(x[:, -1:], layers[-1]["norm2"], shape.rms_eps)
    return last, (last @ lm_head if lm_head is not None else None)


def ttft_table(lengths, shape: DecoderShape, n_layers: int, reps: int, cfg: SparseConfig,
               seed: int = 0, file=sys.stdout):
    """TTFT (ms) of sparse vs dense prefill for each prompt length."""
    dev = torch.device("cuda:0")
    layers = make_weights(shape, n_layers, seed, dev)
    g = torch.Generator(device=dev)
    g.manual_seed(seed + 1)
    lm_head = (torch.randn((shape.hidden, shape.vocab), generator=g, device=dev) /
               math.sqrt(shape.hidden)).to(torch.bfloat16)
    print(f"Decoder: {n_layers} layers, hidden {shape.hidden}, {shape.n_q_heads}/"
          f"{shape.n_kv_heads} heads of {shape.head_dim}, MLP {shape.intermediate}, random bf16 "
          f"weights; sparse: L_S = {cfg.seg_len}, L_B = {cfg.block_len}, B_h = "
          f"{cfg.base_budget}, e_t = {cfg.entropy_threshold}; {reps} timed runs after one "
          f"warm-up.\n", file=file)
    print("| prompt tokens | dense TTFT ms | sparse TTFT ms | speedup | dense attention share |",
          file=file)
    print("|---:|---:|---:|---:|---:|", file=file)
    for N in lengths:
        x0 = (torch.randn((1, N, shape.hidden), generator=g, device=dev)).to(torch.bfloat16)
        res = {}
        for kind in ("dense", "sparse"):
            attn = Attention(shape, 1, N, kind, cfg, dev)
            prefill(x0, layers, shape, attn, lm_head)
            torch.cuda.synchronize()
            e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            e[0].record()
            for _ in range(reps):
                prefill(x0, layers, shape, attn, lm_head)
            e[1].record()
            torch.cuda.synchronize()
            res[kind] = e[0].elapsed_time(e[1]) / reps
            # attention alone, one layer's inputs, for the share column
            if kind == "dense":
                cos, sin = rope_tables(N, shape.head_dim, shape.rope_theta, dev)
                tr = {}
                layer_forward(x0, layers[0], shape, attn, cos, sin, trace=tr)
                a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                torch.cuda.synchronize()
                a0.record()
                attn(tr["q"], tr["k"], tr["v"])
                a1.record()
                torch.cuda.synchronize()
                res["dense_attn_share"] = a0.elapsed_time(a1) * n_layers / res["dense"]
            del attn
        print(f"| {N} | {res['dense']:.1f} | {res['sparse']:.1f} | "
              f"{res['dense'] / res['sparse']:.2f} | {res['dense_attn_share']:.2f} |", file=file,
              flush=True)
        del x0
        torch.cuda.empty_cache()


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--ttft", action="store_true", help="time sparse vs dense prefill")
    ap.add_argument("--layers", type=int, default=LLAMA3_8B.n_layers)
    ap.add_argument("--reps", type=int, default=2)
    ap.add_argument("--lengths", default="4096,8192,16384,32768,65536,131072,143360")
    args = ap.parse_args()
    if not args.ttft:
        ap.print_help()
        return
    if not torch.cuda.is_available():
        print("a ROCm GPU is needed", file=sys.stderr)
        sys.exit(1)
    t0 = time.time()
    ttft_table([int(n) for n in args.lengths.split(",")], LLAMA3_8B, args.layers, args.reps,
               SparseConfig())
    print(f"\n(total wall time {time.time() - t0:.0f} s)", file=sys.stderr)


if __name__ == "__main__":
    main()
