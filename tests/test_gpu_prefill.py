"""The multi-layer prefill harness on the GPU, layer by layer, against an fp32
CPU decoder layer written out here: the projections + rotary embedding, the
attention (the oracle on the GPU's own block lists, or dense causal), and the
output projection + MLP.  Bars: Q/K/V within 4 bf16 ulps (2^-6) of the
rounded fp32 values, relative to max(|value|, RMS of the tensor) -- the rotary
embedding's differences of two products can cancel, so a one-ulp difference
before the rotation is measured against the tensor's scale; attention max-abs
2e-2 (as the kernel tests); layer output relative RMS error 1e-2."""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2606_09508_amd import prefill as pf

pytestmark = pytest.mark.gpu

SHAPE = pf.DecoderShape(hidden=512, n_q_heads=4, n_kv_heads=2, head_dim=128, intermediate=1024,
                        n_layers=2, vocab=1000)


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def _bf16(t):
    return t.to(torch.bfloat16).float()


def _rms(x, g, eps):
    return x * torch.rsqrt((x * x).mean(-1, keepdim=True) + eps) * g


def _rotary(x, N, D, theta):
    """x [B, H, N, D] fp32; pairs (i, i + D/2) rotated by position * theta^(-2i/D)."""
    i = torch.arange(D // 2, dtype=torch.float64)
    freq = theta ** (-2.0 * i / D)
    ang = torch.arange(N, dtype=torch.float64)[:, None] * freq[None, :]
    c, s = torch.cos(ang).float(), torch.sin(ang).float()
    a, b = x[..., : D // 2], x[..., D // 2:]
    return torch.cat([a * c - b * s, a * s + b * c], dim=-1)


def _cpu_w(w):
    return {k: v.float().cpu() for k, v in w.items()}


def _qkv_ref(x, w, N):
    B = x.shape[0]
    Hq, Hkv, D = SHAPE.n_q_heads, SHAPE.n_kv_heads, SHAPE.head_dim
    h = _bf16(_rms(x, w["norm1"], SHAPE.rms_eps))
    q = _bf16(h @ w["wq"]).view(B, N, Hq, D).transpose(1, 2)
    k = _bf16(h @ w["wk"]).view(B, N, Hkv, D).transpose(1, 2)
    v = _bf16(h @ w["wv"]).view(B, N, Hkv, D).transpose(1, 2)
    return _bf16(_rotary(q, N, D, SHAPE.rope_theta)), _bf16(_rotary(k, N, D, SHAPE.rope_theta)), v


def _rest_ref(x, o, w):
    B, N, _ = x.shape
    x = x + _bf16(o.transpose(1, 2).reshape(B, N, -1) @ w["wo"])
    h = _bf16(_rms(x, w["norm2"], SHAPE.rms_eps))
    g, u = _bf16(h @ w["w_gate"]), _bf16(h @ w["w_up"])
    m = _bf16(_bf16(g * torch.sigmoid(g)) * u)
    return x + _bf16(m @ w["w_down"])


def _u16(t):
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


@pytest.mark.parametrize("kind", ["sparse", "dense"])
def test_prefill_layers_match_cpu_layer(kind):
    dev = torch.device("cuda:0")
    N = 1024
    cfg = pf.SparseConfig(base_budget=256)
    layers = pf.make_weights(SHAPE, SHAPE.n_layers, seed=11, device=dev)
    g = torch.Generator(device=dev)
    g.manual_seed(12)
    x = torch.randn((1, N, SHAPE.hidden), generator=g, device=dev).to(torch.bfloat16)
    cos, sin = pf.rope_tables(N, SHAPE.head_dim, SHAPE.rope_theta, dev)
    attn = pf.Attention(SHAPE, 1, N, kind, cfg, dev)
    rows = np.array([[0, h, i] for h in range(SHAPE.n_q_heads) for i in range(N)], np.int32)
    for li, w in enumerate(layers):
        tr = {}
        x_next = pf.layer_forward(x, w, SHAPE, attn, cos, sin, trace=tr)
        torch.cuda.synchronize()
        wc = _cpu_w(w)
        xc = x.float().cpu()
        q_ref, k_ref, v_ref = _qkv_ref(xc, wc, N)
        for name, ref in (("q", q_ref), ("k", k_ref), ("v", v_ref)):
            got = tr[name].float().cpu()
            err = (got - ref).abs() / ref.abs().clamp_min(float(ref.pow(2).mean().sqrt()))
            assert float(err.max()) <= 2.0 ** -6, f"layer {li} {name}: rel {float(err.max()):.2e}"
        if kind == "sparse":
            idx = attn.sel["idx"].cpu().numpy()
            cnt = attn.sel["cnt"].cpu().numpy()
            ref_o = oracle.attention(_u16(tr["q"]), _u16(tr["k"]), _u16(tr["v"]), rows,
                                     1.0 / math.sqrt(SHAPE.head_dim), True, idx, cnt,
                                     cfg.seg_len, cfg.block_len)
        else:
            ref_o = oracle.attention(_u16(tr["q"]), _u16(tr["k"]), _u16(tr["v"]), rows,
                                     1.0 / math.sqrt(SHAPE.head_dim), True)
        got_o = tr["o"].float().cpu().numpy().astype(np.float64)[rows[:, 0], rows[:, 1],
                                                                  rows[:, 2]]
        aerr = np.abs(got_o - ref_o).max()
        assert aerr <= 2e-2, f"layer {li} attention max-abs {aerr:.3e}"
        ref_next = _rest_ref(xc, tr["o"].float().cpu(), wc)
        got_next = x_next.float().cpu()
        rel = float((got_next - ref_next).norm() / ref_next.norm())
        say(f"  [{kind}] layer {li}: attention max-abs {aerr:.2e}, layer rel-RMS {rel:.2e}")
        assert rel <= 1e-2, f"layer {li} output rel-RMS {rel:.3e}"
        x = x_next


def test_prefill_end_to_end_is_finite_and_deterministic():
    dev = torch.device("cuda:0")
    N = 2048
    layers = pf.make_weights(SHAPE, SHAPE.n_layers, seed=3, device=dev)
    head = torch.randn((SHAPE.hidden, SHAPE.vocab), device=dev).to(torch.bfloat16)
    x = torch.randn((1, N, SHAPE.hidden), device=dev).to(torch.bfloat16)
    attn = pf.Attention(SHAPE, 1, N, "sparse", pf.SparseConfig(base_budget=256), dev)
    h1, l1 = pf.prefill(x, layers, SHAPE, attn, head)
    h2, l2 = pf.prefill(x, layers, SHAPE, attn, head)
    torch.cuda.synchronize()
    assert l1.shape == (1, 1, SHAPE.vocab)
    assert torch.isfinite(l1.float()).all()
    assert torch.equal(l1, l2) and torch.equal(h1, h2)
