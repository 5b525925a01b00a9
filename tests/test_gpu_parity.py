"""HIP path vs the CPU oracle, element by element, through the C ABI.

Bars: entropy |dH| <= 1e-4 H + 1e-20; ln A_obs |dL| <= 1e-3 (+1e-6 |L|);
selection (rigid flags, budgets, block lists, counts) bit-exact given the
GPU's own fp32 scores; attention max-abs <= 2e-2 against fp64.
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2606_09508_amd import binding as eb
from paper_2606_09508_amd import synth

pytestmark = pytest.mark.gpu

H_REL, H_ABS = 1e-4, 1e-20
L_ABS = 1e-3
ATTN_ABS = 2e-2


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    eb.lib()
    return torch.device("cuda:0")


def to_dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()


def bf16_to_f64(t: torch.Tensor) -> np.ndarray:
    return t.float().cpu().numpy().astype(np.float64)


def run_path(w, base_budget=None):
    q, k, v = to_dev(w.q), to_dev(w.k), to_dev(w.v)
    bh = w.base_budget if base_budget is None else base_budget
    ls, en = eb.entropy_probe(q, k, w.Ls, w.Lb, w.probe_scale)
    sel = eb.select_blocks(ls, en, w.N, w.Ls, w.Lb, w.e_t, w.alpha, w.delta_t, bh, w.mult,
                           n_kv_heads=w.Hkv)
    o = eb.sparse_prefill_attn(q, k, v, sel["idx"], sel["cnt"], w.Ls, w.Lb, w.softmax_scale)
    torch.cuda.synchronize()
    return {"q": q, "k": k, "v": v, "ls": ls.cpu().numpy(), "en": en.cpu().numpy(),
            "sel": {kk: t.cpu().numpy() for kk, t in sel.items()}, "o": o, "bh": bh}


def check_probe(w, r, rows=None):
    """rows: optional [n, 3] (b, h, s) sample; default every row."""
    if rows is None:
        Lr, Hr = oracle.probe(w.q, w.k, w.Ls, w.Lb, w.probe_scale)
        Lr = Lr.reshape(-1, w.CB)
        Hr = Hr.reshape(-1)
        Lg = r["ls"].reshape(-1, w.CB)
        Hg = r["en"].reshape(-1)
        sidx = np.tile(np.arange(w.CS), w.B * w.Hq)
    else:
        Lr, Hr = oracle.probe(w.q, w.k, w.Ls, w.Lb, w.probe_scale, rows=rows)
        Lg = np.stack([r["ls"][b, h, s] for b, h, s in rows])
        Hg = np.array([r["en"][b, h, s] for b, h, s in rows])
        sidx = rows[:, 2]
    herr = np.abs(Hg.astype(np.float64) - Hr)
    assert (herr <= H_REL * Hr + H_ABS).all(), \
        f"entropy: worst rel {np.max(herr / np.maximum(Hr, 1e-300)):.3e}"
    r_ = w.Ls // w.Lb
    worst = 0.0
    cols = np.arange(w.CB)[None, :]
    for t0 in range(0, len(Hr), 2048):   # visible entries of 2048 rows at a time
        nv = np.minimum((sidx[t0:t0 + 2048].astype(np.int64) + 1) * r_, w.CB)[:, None]
        vis = cols < nv
        ref = Lr[t0:t0 + 2048]
        d = np.where(vis, np.abs(Lg[t0:t0 + 2048].astype(np.float64) - ref), 0.0)
        bad = vis & ~(d <= L_ABS + 1e-6 * np.abs(np.where(vis, ref, 0.0)))
        assert not bad.any(), f"log_scores rows {t0}+{np.nonzero(bad.any(1))[0][:4]}"
        worst = max(worst, float(d.max()))
    return float(np.max(herr / np.maximum(Hr, 1e-30))), worst


def check_select(w, r):
    ref = oracle.select(r["ls"], r["en"], w.N, w.Ls, w.Lb, w.e_t, w.alpha, w.delta_t, r["bh"],
                        w.mult)
    g = r["sel"]
    np.testing.assert_array_equal(g["rigid"], ref["rigid"])
    np.testing.assert_array_equal(g["budget"], ref["budget"])
    np.testing.assert_array_equal(g["cnt"], ref["cnt"])
    np.testing.assert_array_equal(g["idx"], ref["idx"])


def check_attention(w, r, rows=None):
    if rows is None:
        rows = np.array([[b, h, i] for b in range(w.B) for h in range(w.Hq) for i in range(w.N)],
                        np.int32)
    ref = oracle.attention(w.q, w.k, w.v, rows, w.softmax_scale, True, r["sel"]["idx"],
                           r["sel"]["cnt"], w.Ls, w.Lb)
    o = bf16_to_f64(r["o"])
    got = o[rows[:, 0], rows[:, 1], rows[:, 2]]
    err = np.abs(got - ref)
    assert err.max() <= ATTN_ABS, f"sparse attention max-abs {err.max():.3e}"
    return float(err.max()), float(err.mean())


C1_CASES = [
    dict(),                                           # the tiny workload itself
    dict(N=1000),                                     # ragged tail
    dict(N=1088),
    dict(N=128),                                      # a single segment
    dict(N=64),                                       # shorter than one segment
    dict(B=2, N=640),
    dict(Hq=4, Hkv=4),                                # MHA
    dict(Hq=7, Hkv=1, N=512),                         # G = 7
    dict(Hq=8, Hkv=2, N=768),
    dict(Ls=256, Lb=64, N=1280),
    dict(Ls=256, Lb=128, N=1280, base_budget=512),
    dict(Ls=2048, Lb=64, N=4096, base_budget=1024),
    dict(N=2048, base_budget=64),                     # k = 1 past block
    dict(N=2048, base_budget=0),                      # own blocks only
    dict(N=1),                                        # one token
    dict(N=65),                                       # one full block and one row
    dict(B=3, Hq=1, Hkv=1, N=200),                    # single head, batch of three
]


@pytest.mark.parametrize("case", C1_CASES, ids=lambda c: ",".join(f"{k}={v}" for k, v in c.items())
                         or "c1")
@pytest.mark.parametrize("seed", [0, 1])
def test_path_parity_small(case, seed):
    w = synth.make("c1", seed, **case)
    say(f"[small] seed={seed} {case}")
    r = run_path(w)
    hrel, lerr = check_probe(w, r)
    check_select(w, r)
    amax, amean = check_attention(w, r)
    say(f"  entropy rel {hrel:.2e}  logscore abs {lerr:.2e}  attn max {amax:.2e} mean {amean:.2e}")


def _span_inputs(N=1024, Hq=4, Hkv=1, seed=11):
    """Query / key elements far below each pooled vector's maximum, so that
    the probe's fixed-point grid (2^-13 of the maximum's binade) leaves
    residuals, plus bf16 subnormals, +-0 and all-zero query segments: dims
    0-3 scaled by 2^-20, 4-7 by 2^-128 (subnormal), 8-11 zero (negative
    zero in odd rows), 12-15 by 2^-8, dim 127 a +-6 sink on block 0 for
    heads 0-1; query segment 3 of head 2 is all zero."""
    rng = np.random.default_rng(seed)
    D = 128
    qf = rng.standard_normal((1, Hq, N, D)).astype(np.float32)
    kf = rng.standard_normal((1, Hkv, N, D)).astype(np.float32)
    for x in (qf, kf):
        x[..., 0:4] *= 2.0 ** -20
        x[..., 4:8] *= 2.0 ** -128
        x[..., 8:12] = 0.0
        x[..., 1::2, 8:12] = -0.0
        x[..., 12:16] *= 2.0 ** -8
        x[..., 127] = 0.0
    qf[:, :2, :, 127] = 6.0
    kf[:, :, :64, 127] = 6.0
    qf[:, 2, 3 * 128:4 * 128, :] = 0.0
    w = synth.make("c1", seed, Hq=Hq, Hkv=Hkv, N=N, generate_tensors=False)
    w.q, w.k = synth.to_bf16_bits(qf), synth.to_bf16_bits(kf)
    w.v = synth.to_bf16_bits(rng.standard_normal((1, Hkv, N, D)).astype(np.float32))
    return w


@pytest.mark.parametrize("probe_scale", [1.0, -1.0, 0.0, 1.0 / math.sqrt(128.0)])
def test_probe_residuals_subnormals_zeros(probe_scale):
    """Elements off the probe's fixed-point grid (its residual MFMA), bf16
    subnormals, +-0, all-zero segments and every sign of probe_scale: probe
    outputs against the oracle."""
    w = _span_inputs()
    say(f"[spans] probe_scale={probe_scale}")
    q, k = to_dev(w.q), to_dev(w.k)
    ls, en = eb.entropy_probe(q, k, w.Ls, w.Lb, probe_scale)
    torch.cuda.synchronize()
    r = {"ls": ls.cpu().numpy(), "en": en.cpu().numpy()}
    w.probe_scale = probe_scale
    hrel, lerr = check_probe(w, r)
    say(f"  entropy rel {hrel:.2e} L {lerr:.2e}")
    if probe_scale == 0.0:   # every logit 0: uniform rows, H = ln n_vis
        nv = np.minimum((np.arange(w.CS) + 1) * (w.Ls // w.Lb), w.CB)
        assert np.allclose(r["en"][0], np.log(nv)[None, :], rtol=1e-6)


def test_c1_labels_on_gpu():
    """The tiny workload's intended head types come out of the GPU path."""
    w = synth.make("c1", 0)
    r = run_path(w)
    assert list(r["sel"]["rigid"][0]) == [1, 1, 0, 0]


@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("case", [dict(), dict(N=1000), dict(B=2, Hq=8, Hkv=2, N=384),
                                  dict(N=64)])
def test_dense_parity(case, causal):
    w = synth.make("c1", 7, **case)
    say(f"[dense] causal={causal} {case}")
    q, k, v = to_dev(w.q), to_dev(w.k), to_dev(w.v)
    o = eb.dense_prefill_attn(q, k, v, w.softmax_scale, causal)
    torch.cuda.synchronize()
    rows = np.array([[b, h, i] for b in range(w.B) for h in range(w.Hq) for i in range(w.N)],
                    np.int32)
    ref = oracle.attention(w.q, w.k, w.v, rows, w.softmax_scale, causal)
    got = bf16_to_f64(o)[rows[:, 0], rows[:, 1], rows[:, 2]]
    assert np.abs(got - ref).max() <= ATTN_ABS


def test_full_budget_sparse_is_dense_bitwise():
    """With B_h >= N every visible block is selected; the sparse kernel then
    visits exactly the dense kernel's blocks in the same order."""
    w = synth.make("c1", 2, N=1280)
    r = run_path(w, base_budget=w.N)
    assert (r["sel"]["cnt"] == 2 * (np.arange(w.CS) + 1)[None, None, :]).all()
    od = eb.dense_prefill_attn(r["q"], r["k"], r["v"], w.softmax_scale, True)
    torch.cuda.synchronize()
    assert torch.equal(od, r["o"])


def _jump_inputs(N=1000, Hq=2, seed=5):
    """Scores that rise part way through each row: q_0 = 4 for every query,
    keys 320..383 carry k_0 = 80 (about 40 base-2 units over the earlier
    blocks' maximum), keys 640..703 k_0 = 400 (2^-x of the earlier maximum
    overflows fp32) and keys 900..909 k_0 = -400 (their probabilities
    underflow to zero)."""
    rng = np.random.default_rng(seed)
    D = 128
    qf = rng.standard_normal((1, Hq, N, D)).astype(np.float32)
    kf = rng.standard_normal((1, 1, N, D)).astype(np.float32)
    vf = rng.standard_normal((1, 1, N, D)).astype(np.float32)
    qf[..., 0] = 4.0
    kf[:, :, 320:384, 0] = 80.0
    kf[:, :, 640:704, 0] = 400.0
    kf[:, :, 900:910, 0] = -400.0
    w = synth.make("c1", seed, Hq=Hq, N=N, generate_tensors=False)
    w.q, w.k, w.v = (synth.to_bf16_bits(x) for x in (qf, kf, vf))
    return w


@pytest.mark.parametrize("causal", [True, False])
def test_dense_attention_running_max_jumps(causal):
    """The running maximum is left behind by more than the probabilities'
    2^32 limit, and by enough to overflow exp2, in the middle of rows: the
    kernel must take the row maxima and rescale; every row against the fp64
    oracle."""
    w = _jump_inputs()
    say(f"[dense jumps] causal={causal}")
    o = eb.dense_prefill_attn(to_dev(w.q), to_dev(w.k), to_dev(w.v), w.softmax_scale, causal)
    torch.cuda.synchronize()
    rows = np.array([[0, h, i] for h in range(w.Hq) for i in range(w.N)], np.int32)
    ref = oracle.attention(w.q, w.k, w.v, rows, w.softmax_scale, causal)
    got = bf16_to_f64(o)[rows[:, 0], rows[:, 1], rows[:, 2]]
    assert np.isfinite(got).all()
    assert np.abs(got - ref).max() <= ATTN_ABS


def test_sparse_attention_running_max_jumps():
    """The same inputs through probe, selection and sparse attention: every
    row against the oracle on the GPU's block lists."""
    w = _jump_inputs()
    say("[sparse jumps]")
    r = run_path(w)
    rows = np.array([[0, h, i] for h in range(w.Hq) for i in range(w.N)], np.int32)
    ref = oracle.attention(w.q, w.k, w.v, rows, w.softmax_scale, True, r["sel"]["idx"],
                           r["sel"]["cnt"], w.Ls, w.Lb)
    got = bf16_to_f64(r["o"])[rows[:, 0], rows[:, 1], rows[:, 2]]
    assert np.isfinite(got).all()
    assert np.abs(got - ref).max() <= ATTN_ABS


def test_deterministic():
    w = synth.make("c2", 3, N=4096)
    a = run_path(w)
    b = run_path(w)
    assert np.array_equal(a["en"], b["en"])
    assert np.array_equal(a["ls"][~np.isnan(a["ls"])], b["ls"][~np.isnan(a["ls"])])
    assert np.array_equal(a["sel"]["idx"], b["sel"]["idx"])
    assert torch.equal(a["o"], b["o"])


@pytest.mark.parametrize("wl,seed,case", [
    ("c1", 5, dict()),                                    # G = 4: two pairs
    ("c1", 5, dict(N=1000)),                              # ragged tail
    ("c1", 6, dict(Hq=7, Hkv=1, N=512)),                  # odd G: the last pair has one head
    ("c1", 6, dict(Hq=4, Hkv=4)),                         # G = 1: one head per workgroup
    ("c1", 7, dict(Ls=256, Lb=128, N=1280, base_budget=512)),   # two sub-blocks per block
    ("c1", 7, dict(B=2, Hq=8, Hkv=2, N=640)),
    ("c1", 8, dict(N=2048, base_budget=64)),              # short lists, large unions
    ("c1", 8, dict(N=65)),
    ("c2", 2, dict(N=16384)),
    ("c4", 1, dict(N=8192)),                              # G = 7 with real lists
], ids=lambda x: x if isinstance(x, str) else None)
def test_gqa_union_attention_equals_per_head(wl, seed, case):
    """GQA-union tiles (two heads of a KV group share each union block's copy)
    give bitwise the per-head kernel's output."""
    w = synth.make(wl, seed, **case)
    say(f"[union] {wl} seed={seed} {case}")
    q, k, v = to_dev(w.q), to_dev(w.k), to_dev(w.v)
    ls, en = eb.entropy_probe(q, k, w.Ls, w.Lb, w.probe_scale)
    sel = eb.select_blocks(ls, en, w.N, w.Ls, w.Lb, w.e_t, w.alpha, w.delta_t, w.base_budget,
                           w.mult, n_kv_heads=w.Hkv)
    o = eb.sparse_prefill_attn(q, k, v, sel["idx"], sel["cnt"], w.Ls, w.Lb, w.softmax_scale)
    ou = eb.sparse_prefill_attn(q, k, v, sel["idx"], sel["cnt"], w.Ls, w.Lb, w.softmax_scale,
                                gqa_union=True)
    torch.cuda.synchronize()
    assert torch.equal(ou, o)
    # and against the oracle on the GPU's lists: every row of the small cases,
    # a few thousand rows (every head, first and last rows of segments) else
    if w.N <= 2048:
        rows = np.array([[b, h, i] for b in range(w.B) for h in range(w.Hq) for i in range(w.N)],
                        np.int32)
    else:
        rows = _spread_query_rows(w, 3072, seed=seed)
    ref = oracle.attention(w.q, w.k, w.v, rows, w.softmax_scale, True, sel["idx"].cpu().numpy(),
                           sel["cnt"].cpu().numpy(), w.Ls, w.Lb)
    got = bf16_to_f64(ou)[rows[:, 0], rows[:, 1], rows[:, 2]]
    err = np.abs(got - ref)
    say(f"  union vs oracle: {len(rows)} rows, max-abs {err.max():.2e} mean {err.mean():.2e}")
    assert err.max() <= ATTN_ABS


@pytest.mark.parametrize("wl,seed,case", [
    ("c1", 3, dict()),                                    # one KV group: 8 XCDs share it
    ("c1", 3, dict(N=1000)),                              # ragged tail
    ("c1", 4, dict(B=2, Hq=8, Hkv=2, N=3072)),            # four groups, two XCDs each
    ("c1", 4, dict(B=2, Hq=16, Hkv=4, N=1024)),           # eight groups, one XCD each
    ("c1", 5, dict(B=4, Hq=8, Hkv=4, N=640)),             # sixteen groups, two per XCD
    ("c1", 5, dict(B=3, Hq=4, Hkv=1, N=384)),             # three groups: the static grid
    ("c1", 7, dict(B=2, Hq=4, Hkv=1, N=2560)),            # two groups, four XCDs each
    ("c1", 7, dict(B=3, Hq=16, Hkv=8, N=256)),            # 24 groups, three per XCD
    ("c1", 6, dict(Ls=256, Lb=128, N=1280, base_budget=512)),   # two sub-blocks per block
    ("c1", 6, dict(N=65)),
    ("c2", 2, dict(N=16384)),
    ("c4", 1, dict(N=8192)),                              # four KV groups, G = 7
], ids=lambda x: x if isinstance(x, str) else None)
def test_persistent_schedule_equals_static(wl, seed, case):
    """With a scheduling workspace the sparse kernel runs persistent
    workgroups over per-XCD queues with stealing; the output is bitwise the
    static grid's (no workspace), also on a second call into the same
    workspace (the counters are reset by each call)."""
    w = synth.make(wl, seed, **case)
    say(f"[persistent] {wl} seed={seed} {case}")
    q, k, v = to_dev(w.q), to_dev(w.k), to_dev(w.v)
    ls, en = eb.entropy_probe(q, k, w.Ls, w.Lb, w.probe_scale)
    sel = eb.select_blocks(ls, en, w.N, w.Ls, w.Lb, w.e_t, w.alpha, w.delta_t, w.base_budget,
                           w.mult, n_kv_heads=w.Hkv)
    o_static = eb.sparse_prefill_attn(q, k, v, sel["idx"], sel["cnt"], w.Ls, w.Lb,
                                      w.softmax_scale, persistent=False)
    ws = torch.empty((eb.ATTN_WORKSPACE_BYTES,), dtype=torch.uint8, device=q.device)
    for call in range(2):
        o = torch.full_like(q, float("nan"))
        eb.sparse_prefill_attn(q, k, v, sel["idx"], sel["cnt"], w.Ls, w.Lb, w.softmax_scale,
                               out=o, workspace=ws)
        torch.cuda.synchronize()
        assert torch.equal(o, o_static), f"call {call}"


def test_binding_refuses_mismatched_tensors():
    """k / v / score tensors that do not match q's sizes raise before any launch."""
    w = synth.make("c1", 4, N=512)
    q, k, v = to_dev(w.q), to_dev(w.k), to_dev(w.v)
    with pytest.raises(ValueError):
        eb.dense_prefill_attn(q, k[:, :, :256].contiguous(), v[:, :, :256].contiguous())
    with pytest.raises(ValueError):
        eb.entropy_probe(q, k[:, :, :256].contiguous(), w.Ls, w.Lb)
    ls, en = eb.entropy_probe(q, k, w.Ls, w.Lb, w.probe_scale)
    with pytest.raises(ValueError):
        eb.select_blocks(ls, en, 2 * w.N, w.Ls, w.Lb, n_kv_heads=w.Hkv)
    with pytest.raises(ValueError):
        eb.select_blocks(ls[:, :, :, :-1].contiguous(), en, w.N, w.Ls, w.Lb, n_kv_heads=w.Hkv)
    torch.cuda.synchronize()


def test_malformed_block_list_is_safe():
    """Out-of-range, descending and oversized counts stop the list walk."""
    w = synth.make("c1", 4, N=512)
    q, k, v = to_dev(w.q), to_dev(w.k), to_dev(w.v)
    km = w.kmax
    idx = torch.full((1, w.Hq, w.CS, km), -1, dtype=torch.int32)
    cnt = torch.zeros((1, w.Hq, w.CS), dtype=torch.int32)
    for s in range(w.CS):
        own = [2 * s, 2 * s + 1]
        idx[0, 0, s, :2] = torch.tensor(own)
        cnt[0, 0, s] = 2
        idx[0, 1, s, :3] = torch.tensor([10 ** 6] + own)         # out of range first
        cnt[0, 1, s] = 3
        idx[0, 2, s, :2] = torch.tensor(own)
        cnt[0, 2, s] = 10 ** 6                                    # count beyond kmax
        idx[0, 3, s, :3] = torch.tensor(own + [0])               # not ascending
        cnt[0, 3, s] = 3
    o = eb.sparse_prefill_attn(q, k, v, idx.cuda(), cnt.cuda(), w.Ls, w.Lb, w.softmax_scale)
    torch.cuda.synchronize()
    of = o.float().cpu()
    assert torch.isfinite(of).all()
    assert (of[0, 1] == 0).all()                                  # nothing visible -> zeros
    rows = np.array([[0, h, i] for h in (0, 2, 3) for i in range(w.N)], np.int32)
    ref_idx = idx.numpy().copy()
    ref_cnt = np.full((1, w.Hq, w.CS), 2, np.int32)
    ref = oracle.attention(w.q, w.k, w.v, rows, w.softmax_scale, True, ref_idx, ref_cnt, w.Ls,
                           w.Lb)
    got = of.numpy().astype(np.float64)[rows[:, 0], rows[:, 1], rows[:, 2]]
    assert np.abs(got - ref).max() <= ATTN_ABS


def _crafted_scores(CS, CB, Hq, seed=5):
    """Score rows that reach every branch of the GPU selector: exact ties,
    NaN / +-inf / +-0, rows of one value, a bucket of far more than 64 keys
    (two clusters that differ in one high mantissa bit), keys that differ
    only in their low 10 bits, and plain random rows."""
    rng = np.random.default_rng(seed)
    ls = np.empty((1, Hq, CS, CB), np.float32)
    shape = (CS, CB)
    ls[0, 0] = rng.choice(np.array([-1.5, -2.25, -3.0, -0.0, 0.0], np.float32), shape)
    x = rng.standard_normal(shape).astype(np.float32)
    u = rng.random(shape)
    x[u < 0.1] = np.nan
    x[(u >= 0.1) & (u < 0.15)] = -np.inf
    x[(u >= 0.15) & (u < 0.17)] = np.inf
    ls[0, 1] = x
    ls[0, 2] = -4.0
    bits = (0x3F800000 + rng.integers(0, 2, shape) * (1 << 20)
            + rng.integers(0, 512, shape)).astype(np.uint32)
    ls[0, 3] = bits.view(np.float32)
    ls[0, 4] = (0x3F800000 + rng.integers(0, 1024, shape)).astype(np.uint32).view(np.float32)
    ls[0, 5] = rng.standard_normal(shape).astype(np.float32)
    en = rng.uniform(0.5, 1.5, (1, Hq, CS)).astype(np.float32)
    en[0, 2] = 0.0                                               # a rigid head
    return ls, en


def test_select_crafted_scores():
    """Selection is bit-exact against the oracle on crafted score rows."""
    N, Ls, Lb, Hq = 32768, 128, 64, 6
    CS, CB = N // Ls, N // Lb
    ls, en = _crafted_scores(CS, CB, Hq)
    for bh, mult in ((2048, 3), (64, 3), (8192, 3)):
        sel = eb.select_blocks(torch.from_numpy(ls).cuda(), torch.from_numpy(en).cuda(), N, Ls,
                               Lb, 1e-5, 0.5, 0.4, bh, mult, n_kv_heads=Hq)
        torch.cuda.synchronize()
        g = {kk: t.cpu().numpy() for kk, t in sel.items()}
        ref = oracle.select(ls, en, N, Ls, Lb, 1e-5, 0.5, 0.4, bh, mult)
        for name in ("rigid", "budget", "cnt", "idx"):
            np.testing.assert_array_equal(g[name], ref[name], err_msg=f"{name} B_h={bh}")


def _crafted_large_scores(CS, CB, seed=7):
    """Rows for the wide selector instances (32 to 128 slots per lane): a
    cluster of 100 keys that share every bit above their low 12 (T's bucket
    then holds 65..128 keys: the two-per-lane compaction), a cluster of 300
    (more than 128: the resolution over all slots), 200 keys exactly equal
    to the row's maximum (ties at T: the index search), over a low random
    background; and a row type with NaN / +-inf / +-0."""
    rng = np.random.default_rng(seed)
    shape = (CS, CB)
    ls = np.empty((1, 4, CS, CB), np.float32)
    for h, n in ((0, 100), (1, 300)):
        x = (rng.standard_normal(shape) - 10.0).astype(np.float32)
        for s in range(CS):
            pos = rng.choice(CB, size=min(n, CB), replace=False)
            x[s, pos] = (0x3F800000 + rng.integers(0, 1 << 12, pos.size)).astype(
                np.uint32).view(np.float32)
        ls[0, h] = x
    x = (rng.standard_normal(shape) - 10.0).astype(np.float32)
    for s in range(CS):
        x[s, rng.choice(CB, size=min(200, CB), replace=False)] = 1.0
    ls[0, 2] = x
    x = rng.standard_normal(shape).astype(np.float32)
    u = rng.random(shape)
    x[u < 0.05] = np.nan
    x[(u >= 0.05) & (u < 0.1)] = -np.inf
    x[(u >= 0.1) & (u < 0.12)] = np.inf
    x[(u >= 0.12) & (u < 0.14)] = -0.0
    x[(u >= 0.14) & (u < 0.16)] = 0.0
    ls[0, 3] = x
    en = rng.uniform(0.5, 1.5, (1, 4, CS)).astype(np.float32)
    return ls, en


@pytest.mark.parametrize("N", [65472, 65536, 131008, 131072, 262144, 524288])
def test_select_crafted_large_rows(N):
    """The 16-, 32-, 64- and 128-slot selector instances, bit-exact against
    the oracle on crafted rows (large threshold buckets, ties at T, NaN / inf
    / +-0), with budgets that keep 32..96 and up to 384 past blocks.  C_B =
    1023 and 2047 (N not a multiple of 64 blocks' rows) make the long rows'
    slot groups reach past the row, where the loads are clamped."""
    Ls, Lb = 128, 64
    CS, CB = -(-N // Ls), -(-N // Lb)
    ls, en = _crafted_large_scores(CS, CB)
    for bh, mult in ((2048, 3), (8192, 3)):
        sel = eb.select_blocks(torch.from_numpy(ls).cuda(), torch.from_numpy(en).cuda(), N, Ls,
                               Lb, 1e-5, 0.5, 0.4, bh, mult, n_kv_heads=4)
        torch.cuda.synchronize()
        g = {kk: t.cpu().numpy() for kk, t in sel.items()}
        ref = oracle.select(ls, en, N, Ls, Lb, 1e-5, 0.5, 0.4, bh, mult)
        for name in ("rigid", "budget", "cnt", "idx"):
            np.testing.assert_array_equal(g[name], ref[name], err_msg=f"{name} N={N} B_h={bh}")
        del sel, g, ref


def test_budget_recurrence_across_chunks():
    """Alg. 3's recurrence over more segments than one pass of the budget
    kernel holds (1024): 2085 segments, so B is carried across two chunk
    boundaries into a ragged last chunk.  Dynamic heads only, with entropy
    runs that reach both clamps, x / 0 and 0 / 0; budgets, counts and lists
    bit-exact against the oracle."""
    Ls, Lb, Hq = 128, 64, 2
    CS = 2 * 1024 + 37
    N, CB = CS * Ls, 2 * CS
    rng = np.random.default_rng(11)
    en = rng.uniform(0.5, 1.5, (1, Hq, CS)).astype(np.float32)
    en[0, 0, 1000:1010] = 1.0                    # flat run: the budget decays to B_h
    en[0, 0, 1020:1030] = [1, 4, 16, 64, 256, 1, 1, 1, 1, 1]   # growth to the 3 B_h cap
    en[0, 1, 1023:1026] = [0.0, 0.0, 2.0]        # 0 / 0 -> 0, then x / 0 -> inf
    en[0, 1, 2047:2050] = [0.0, 1.0, 1.0]
    ls = rng.standard_normal((1, Hq, CS, CB)).astype(np.float32)
    sel = eb.select_blocks(torch.from_numpy(ls).cuda(), torch.from_numpy(en).cuda(), N, Ls, Lb,
                           1e-5, 0.5, 0.4, 2048, 3, n_kv_heads=1)
    torch.cuda.synchronize()
    g = {kk: t.cpu().numpy() for kk, t in sel.items()}
    ref = oracle.select(ls, en, N, Ls, Lb, 1e-5, 0.5, 0.4, 2048, 3)
    assert not ref["rigid"].any()
    b = ref["budget"][0]
    assert (b == 32).any() and (b == 96).any() and len(np.unique(b)) > 10
    for name in ("rigid", "budget", "cnt", "idx"):
        np.testing.assert_array_equal(g[name], ref[name], err_msg=name)


@pytest.mark.parametrize("mode", [eb.CLASSIFY_HEAD, eb.CLASSIFY_GQA_GROUP, eb.CLASSIFY_SEGMENT])
def test_budget_recurrence_off_the_clamps(mode):
    """Alg. 3's recurrence where the budget stays strictly between B_h and
    3 B_h for a whole chunk of segments (entropy ratios within 0.005 of
    Delta_t, so every increment is a few tokens), so no run of steps can be
    settled without the value carried into it and the kernel's evaluation
    degenerates to the sequential order; head 1 mixes such stretches with
    clamped ones.  1324 segments, so the unclamped value is also carried
    across a chunk boundary.  Budgets, counts and lists bit-exact against the
    oracle, under each classification rule (the GQA-group rule follows the
    two heads' mean)."""
    Ls, Lb, Hq = 128, 64, 2
    CS = 1024 + 300
    N, CB = CS * Ls, 2 * CS
    rng = np.random.default_rng(23)
    en = np.empty((1, Hq, CS), np.float64)
    for h, (ulo, uhi) in enumerate([(0.395, 0.405), (0.2, 0.6)]):
        e = [1.0, 3.4]                            # ratio 2.4: B_1 = B_h + 2 alpha B_h
        for _ in range(CS - 2):
            u = rng.uniform(ulo, uhi)
            e.append(e[-1] * (1.0 - u if e[-1] > 1.0 else 1.0 + u))
        en[0, h] = e
    en[0, 1, 700:720] = en[0, 1, 699]             # flat run: down to B_h
    en = en.astype(np.float32)
    ls = rng.standard_normal((1, Hq, CS, CB)).astype(np.float32)
    sel = eb.select_blocks(torch.from_numpy(ls).cuda(), torch.from_numpy(en).cuda(), N, Ls, Lb,
                           1e-5, 0.5, 0.4, 2048, 3, n_kv_heads=1, mode=mode)
    torch.cuda.synchronize()
    g = {kk: t.cpu().numpy() for kk, t in sel.items()}
    ref = oracle.select(ls, en, N, Ls, Lb, 1e-5, 0.5, 0.4, 2048, 3, mode=mode, n_kv_heads=1)
    b = ref["budget"][0]
    assert not ref["rigid"].any()
    if mode != eb.CLASSIFY_GQA_GROUP:
        assert (b[0, 48:] > 32).all() and (b[0, 48:] < 96).all()    # never clamped
        assert (b[1, 48:] == 32).any() and (b[1, 48:] == 96).any()
        assert len(np.unique(b[1, 48:])) > 20
    for name in ("rigid", "budget", "cnt", "idx"):
        np.testing.assert_array_equal(g[name], ref[name], err_msg=f"{name} mode={mode}")


@pytest.mark.parametrize("mode", [eb.CLASSIFY_HEAD, eb.CLASSIFY_GQA_GROUP, eb.CLASSIFY_SEGMENT])
@pytest.mark.parametrize("e_t", [1e-5, math.inf])
def test_select_modes_match_oracle(mode, e_t):
    """Every classification variant, bit-exact against the oracle on the GPU's
    own probe outputs (e_t = +inf: the uniform budget)."""
    w = synth.make("c2", 1, N=16384)
    q, k = to_dev(w.q), to_dev(w.k)
    ls, en = eb.entropy_probe(q, k, w.Ls, w.Lb, w.probe_scale)
    sel = eb.select_blocks(ls, en, w.N, w.Ls, w.Lb, e_t, w.alpha, w.delta_t, w.base_budget,
                           w.mult, n_kv_heads=w.Hkv, mode=mode)
    torch.cuda.synchronize()
    g = {kk: t.cpu().numpy() for kk, t in sel.items()}
    ref = oracle.select(ls.cpu().numpy(), en.cpu().numpy(), w.N, w.Ls, w.Lb, e_t, w.alpha,
                        w.delta_t, w.base_budget, w.mult, mode=mode, n_kv_heads=w.Hkv)
    for name in ("rigid", "budget", "cnt", "idx"):
        np.testing.assert_array_equal(g[name], ref[name], err_msg=f"{name} mode={mode}")
    if e_t == math.inf:
        assert g["rigid"].all()


def test_select_mode_worked_budgets_on_gpu():
    """The hand-worked variant budgets (see the oracle pins) on the GPU."""
    Ls, Lb = 4096, 64
    e = np.asarray([[2, 1, 1e-6, 1e-6, 3, 3]] * 2 + [[2, 1, 1e-6, 1e-6, 1e-6, 1e-6],
                                                    [2, 1, 1e-6, 1e-6, 1e-6, 3e-5]], np.float32)
    Hq, CS = e.shape
    N = CS * Ls
    ls = torch.zeros((1, Hq, CS, N // Lb), dtype=torch.float32, device="cuda")
    en = torch.from_numpy(e[None]).cuda()
    got = {}
    for mode in (eb.CLASSIFY_HEAD, eb.CLASSIFY_GQA_GROUP, eb.CLASSIFY_SEGMENT):
        sel = eb.select_blocks(ls, en, N, Ls, Lb, 1e-5, 0.5, 0.4, 2048, 3, n_kv_heads=2,
                               mode=mode)
        got[mode] = sel["budget"][0].cpu().numpy().tolist()
    assert got[eb.CLASSIFY_SEGMENT][0] == [0, 33, 32, 32, 96, 89]
    assert got[eb.CLASSIFY_HEAD][0] == [0, 33, 43, 36, 96, 89]
    assert got[eb.CLASSIFY_GQA_GROUP][0] == got[eb.CLASSIFY_HEAD][0]        # identical heads
    # group 1: heads 2 and 3 share the budgets of their mean entropy
    assert got[eb.CLASSIFY_GQA_GROUP][2] == got[eb.CLASSIFY_GQA_GROUP][3]


def _sample_rows(w, n_seg=48, seed=0):
    rng = np.random.default_rng(seed)
    segs = np.unique(np.concatenate([[0, 1, w.CS - 1], rng.integers(0, w.CS, n_seg)]))
    rows = []
    for s in segs:
        for h in rng.choice(w.Hq, size=min(3, w.Hq), replace=False):
            rows.append([0, int(h), int(s)])
    return np.array(rows, np.int32)


def _spread_query_rows(w, n, seed=0):
    """About n query rows over every (batch, head): the first and last row of
    randomly drawn segments plus uniformly drawn rows."""
    rng = np.random.default_rng(seed)
    per = max(2, n // (w.B * w.Hq))
    rows = set()
    for b in range(w.B):
        for h in range(w.Hq):
            for s in rng.integers(0, w.CS, per // 4 + 1):
                rows.add((b, h, int(s) * w.Ls))
                rows.add((b, h, min(w.N - 1, (int(s) + 1) * w.Ls - 1)))
            for i in rng.integers(0, w.N, per - 2 * (per // 4 + 1) + 2):
                rows.add((b, h, int(i)))
            rows.add((b, h, w.N - 1))
    return np.array(sorted(rows), np.int32)


def _sample_query_rows(w, n=96, seed=1):
    rng = np.random.default_rng(seed)
    idx = set()
    for i in list(rng.integers(0, w.N, n)) + [0, 1, w.Ls - 1, w.Ls, w.N - 1, w.N - 2]:
        idx.add(int(i))
    heads = rng.integers(0, w.Hq, len(idx))
    return np.array([[0, int(h), i] for h, i in zip(heads, sorted(idx))], np.int32)


def test_c2_llama8b_32k():
    w = synth.make("c2", 0)
    say("[c2] generated")
    r = run_path(w)
    hrel, lerr = check_probe(w, r)
    check_select(w, r)
    amax, amean = check_attention(w, r, _sample_query_rows(w))
    frac = float((r["en"] < w.e_t).mean())
    say(f"  entropy rel {hrel:.2e} L {lerr:.2e} attn {amax:.2e}/{amean:.2e} rigid-seg {frac:.3f}")
    assert 0.3 < frac < 0.5


@pytest.fixture(scope="module")
def c3():
    w = synth.make("c3", 0)
    say("[c3] generated")
    return w, run_path(w)


def test_c3_llama8b_128k(c3):
    """Bench workload, same launch configuration: every probe row (entropy
    and ln A of all 32768 (head, segment) rows), the full selection, and a
    few thousand attention rows over every head (first and last rows of
    segments among them)."""
    w, r = c3
    hrel, lerr = check_probe(w, r)
    say(f"  probe ok (all {w.B * w.Hq * w.CS} rows): entropy rel {hrel:.2e}, L {lerr:.2e}")
    check_select(w, r)
    say("  select bit-exact")
    rows = _spread_query_rows(w, 4096, seed=3)
    amax, amean = check_attention(w, r, rows)
    say(f"  attn ({len(rows)} rows) max {amax:.2e} mean {amean:.2e}")
    # the persistent schedule (the path's) against the static grid, whole layer
    sel = {kk: torch.from_numpy(t).to(r["q"].device) for kk, t in r["sel"].items()}
    o_static = eb.sparse_prefill_attn(r["q"], r["k"], r["v"], sel["idx"], sel["cnt"], w.Ls,
                                      w.Lb, w.softmax_scale, persistent=False)
    torch.cuda.synchronize()
    assert torch.equal(o_static, r["o"])
    say("  persistent schedule bitwise equal to the static grid")


def _fused_equals_path(w, r):
    """ei_probe_select_fused on a workload's inputs: bitwise the entropies and
    selections of the separate calls in r (which check_select holds to the
    oracle's selection on the same ln A)."""
    en2, sel2 = eb.probe_select_fused(r["q"], r["k"], w.Ls, w.Lb, w.e_t, w.alpha, w.delta_t,
                                      w.base_budget, w.mult, w.probe_scale)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(en2.cpu().numpy(), r["en"])
    for name in ("rigid", "budget", "idx", "cnt"):
        np.testing.assert_array_equal(sel2[name].cpu().numpy(), r["sel"][name], err_msg=name)
    say("  fused probe -> select bitwise equal to the separate calls")


def test_c3_fused_probe_select(c3):
    """The fused probe -> select at the 128k layer (the longest rows it
    supports, 2046 past blocks)."""
    w, r = c3
    _fused_equals_path(w, r)


def test_c3_dense_sampled(c3):
    w, r = c3
    od = eb.dense_prefill_attn(r["q"], r["k"], r["v"], w.softmax_scale, True)
    torch.cuda.synchronize()
    rows = _sample_query_rows(w, n=24, seed=5)
    ref = oracle.attention(w.q, w.k, w.v, rows, w.softmax_scale, True)
    got = bf16_to_f64(od)[rows[:, 0], rows[:, 1], rows[:, 2]]
    assert np.abs(got - ref).max() <= ATTN_ABS


def test_c4_qwen7b_64k_sampled():
    """Qwen2.5-7B layer shape (G = 7), 65536 tokens, lognormal key norms and
    retrieval spans: sampled probe rows and query rows, full selection."""
    w = synth.make("c4", 0)
    say("[c4] generated")
    r = run_path(w)
    hrel, lerr = check_probe(w, r, _sample_rows(w, n_seg=32, seed=2))
    check_select(w, r)
    amax, amean = check_attention(w, r, _sample_query_rows(w, n=48, seed=3))
    say(f"  entropy rel {hrel:.2e} L {lerr:.2e} attn {amax:.2e}/{amean:.2e}")
    # Retrieval-span recall of the final segment's selection: reported, not a
    # parity bar (the oracle's selection on the same scores is identical).
    span_blocks = sorted({j for st, ln in w.spans
                          for j in range(st // w.Lb, (st + ln - 1) // w.Lb + 1)})
    idx, cnt = r["sel"]["idx"], r["sel"]["cnt"]
    s_last = w.CS - 1
    rec = np.array([[np.isin(span_blocks, idx[b_, h, s_last, :cnt[b_, h, s_last]]).mean()
                     for h in range(w.Hq)] for b_ in range(w.B)])
    assert span_blocks and ((rec >= 0) & (rec <= 1)).all()
    say(f"  span-block recall in the last segment: mean {rec.mean():.3f}, min {rec.min():.3f} "
        f"over {w.B * w.Hq} heads ({len(span_blocks)} span blocks)")
    _fused_equals_path(w, r)   # G = 7, residual-heavy probe tiles


def test_c5_llama70b_128k_sampled():
    """Llama-3-70B layer on one GPU (64 query / 8 KV heads), 131072 tokens:
    sampled probe and attention rows; selection bit-exact at e_t = 1e-6,
    1e-5 and 1e-4."""
    w = synth.make("c5", 0)
    say("[c5] generated")
    r = run_path(w)
    hrel, lerr = check_probe(w, r, _sample_rows(w, n_seg=24, seed=4))
    check_select(w, r)
    # the three thresholds of the sweep classify 4, 6 and 7 heads as rigid
    # (the oracle's own counts, pinned on the CPU)
    counts = {e_t: int((r["en"].max(axis=2) < np.float32(e_t)).sum()) for e_t in (1e-6, 1e-5, 1e-4)}
    say(f"  rigid heads at e_t = 1e-6 / 1e-5 / 1e-4: {counts}")
    assert counts == {1e-6: 4, 1e-5: 6, 1e-4: 7}
    assert int(r["sel"]["rigid"].sum()) == counts[1e-5]
    for e_t in (1e-6, 1e-4):
        ls = torch.from_numpy(r["ls"]).cuda()
        en = torch.from_numpy(r["en"]).cuda()
        sel = eb.select_blocks(ls, en, w.N, w.Ls, w.Lb, e_t, w.alpha, w.delta_t, w.base_budget,
                               w.mult, n_kv_heads=w.Hkv)
        torch.cuda.synchronize()
        ref = oracle.select(r["ls"], r["en"], w.N, w.Ls, w.Lb, e_t, w.alpha, w.delta_t,
                            w.base_budget, w.mult)
        for name in ("rigid", "budget", "cnt", "idx"):
            np.testing.assert_array_equal(sel[name].cpu().numpy(), ref[name],
                                          err_msg=f"{name} e_t={e_t}")
        del ls, en, sel
    amax, amean = check_attention(w, r, _sample_query_rows(w, n=32, seed=6))
    say(f"  entropy rel {hrel:.2e} L {lerr:.2e} attn {amax:.2e}/{amean:.2e}")
    _fused_equals_path(w, r)


def test_maximum_block_count():
    """The largest C_B the selector supports (8192 key blocks: N = 524288 at
    L_B = 64), one head: probe rows up to 8192 visible blocks, the 128-slot
    selector, sampled attention rows."""
    w = synth.make("c1", 7, N=524288, Hq=1, Hkv=1, base_budget=2048)
    assert w.CB == 8192
    say("[max] generated")
    r = run_path(w)
    rows = np.array([[0, 0, s] for s in (0, 1, 2047, 4094, 4095)], np.int32)
    hrel, lerr = check_probe(w, r, rows)
    check_select(w, r)
    amax, amean = check_attention(w, r, _sample_query_rows(w, n=16, seed=8))
    say(f"  entropy rel {hrel:.2e} L {lerr:.2e} attn {amax:.2e}/{amean:.2e}")


@pytest.mark.parametrize("case,mode", [
    (dict(), eb.CLASSIFY_HEAD),
    (dict(B=2, N=640), eb.CLASSIFY_HEAD),
    (dict(Hq=7, Hkv=1, N=512), eb.CLASSIFY_GQA_GROUP),
    (dict(Ls=256, Lb=128, N=1280, base_budget=512), eb.CLASSIFY_SEGMENT),
    (dict(B=2, Hq=4, Hkv=2, N=16384 + 320), eb.CLASSIFY_HEAD),
    (dict(Hq=7, Hkv=1, N=16384 + 64), eb.CLASSIFY_GQA_GROUP),
    (dict(Hq=4, Hkv=2, Ls=256, Lb=128, N=16384 + 384, base_budget=512), eb.CLASSIFY_SEGMENT),
])
def test_one_call_prefill_equals_separate_calls(case, mode):
    """ei_entropy_guided_prefill gives bitwise the outputs of the three
    separate calls."""
    w = synth.make("c1", 6, **case)
    q, k, v = to_dev(w.q), to_dev(w.k), to_dev(w.v)
    ls, en = eb.entropy_probe(q, k, w.Ls, w.Lb, w.probe_scale)
    sel = eb.select_blocks(ls, en, w.N, w.Ls, w.Lb, w.e_t, w.alpha, w.delta_t, w.base_budget,
                           w.mult, n_kv_heads=w.Hkv, mode=mode)
    o = eb.sparse_prefill_attn(q, k, v, sel["idx"], sel["cnt"], w.Ls, w.Lb, w.softmax_scale)
    o2, sel2, ls2, en2 = eb.entropy_guided_prefill(q, k, v, w.Ls, w.Lb, w.base_budget, w.e_t,
                                                   w.alpha, w.delta_t, w.mult, w.probe_scale,
                                                   w.softmax_scale, mode=mode)
    torch.cuda.synchronize()
    assert torch.equal(en, en2)
    r = w.Ls // w.Lb
    for s in range(w.CS):   # ln A is defined on the visible blocks only
        nv = min((s + 1) * r, w.CB)
        assert torch.equal(ls[:, :, s, :nv], ls2[:, :, s, :nv])
    for name in ("rigid", "budget", "idx", "cnt"):
        assert torch.equal(sel[name], sel2[name]), name
    assert torch.equal(o, o2)


FUSED_CASES = [
    (dict(), eb.CLASSIFY_HEAD),
    (dict(N=1000), eb.CLASSIFY_HEAD),                    # ragged tail
    (dict(N=64), eb.CLASSIFY_HEAD),                      # no past blocks anywhere
    (dict(N=1), eb.CLASSIFY_HEAD),
    (dict(N=200, B=3, Hq=1, Hkv=1), eb.CLASSIFY_HEAD),
    (dict(B=2, N=640), eb.CLASSIFY_HEAD),
    (dict(Hq=7, Hkv=1, N=512), eb.CLASSIFY_GQA_GROUP),
    (dict(Ls=256, Lb=128, N=1280, base_budget=512), eb.CLASSIFY_SEGMENT),
    (dict(N=2048, base_budget=0), eb.CLASSIFY_HEAD),     # own blocks only
    (dict(N=2048, base_budget=64), eb.CLASSIFY_HEAD),    # k = 1
    (dict(B=2, Hq=4, Hkv=2, N=16384 + 320), eb.CLASSIFY_HEAD),
    (dict(Hq=7, Hkv=1, N=16384 + 64), eb.CLASSIFY_GQA_GROUP),
    (dict(Hq=4, Hkv=2, Ls=256, Lb=128, N=16384 + 384, base_budget=512), eb.CLASSIFY_SEGMENT),
    (dict(Hq=8, Hkv=2, N=40960), eb.CLASSIFY_HEAD),      # the 32-slot selector instance
]


def _check_fused(w, mode, ls, en, sel, en2, sel2):
    """The fused path against the separate calls (bitwise) and against the
    oracle's selection on the separate probe's ln A (bit-exact)."""
    assert torch.equal(en, en2), "entropy"
    for name in ("rigid", "budget", "idx", "cnt"):
        assert torch.equal(sel[name], sel2[name]), name
    ref = oracle.select(ls.cpu().numpy(), en.cpu().numpy(), w.N, w.Ls, w.Lb, w.e_t, w.alpha,
                        w.delta_t, w.base_budget, w.mult, mode=mode, n_kv_heads=w.Hkv)
    for name in ("rigid", "budget", "cnt", "idx"):
        np.testing.assert_array_equal(sel2[name].cpu().numpy(), ref[name], err_msg=name)


@pytest.mark.parametrize("case,mode", FUSED_CASES,
                         ids=lambda c: ",".join(f"{k}={v}" for k, v in c.items())
                         if isinstance(c, dict) else str(c))
def test_fused_probe_select_equals_separate_calls(case, mode):
    """ei_probe_select_fused (ln A never in memory) gives bitwise the
    entropies and selections of ei_entropy_probe + ei_select_blocks_mode, and
    they equal the oracle's selection on that ln A."""
    w = synth.make("c1", 9, **case)
    say(f"[fused] {case} mode={mode}")
    q, k = to_dev(w.q), to_dev(w.k)
    ls, en = eb.entropy_probe(q, k, w.Ls, w.Lb, w.probe_scale)
    sel = eb.select_blocks(ls, en, w.N, w.Ls, w.Lb, w.e_t, w.alpha, w.delta_t, w.base_budget,
                           w.mult, n_kv_heads=w.Hkv, mode=mode)
    bufs = {}
    for _ in range(2):   # a second call into the same buffers and workspace
        en2, sel2 = eb.probe_select_fused(q, k, w.Ls, w.Lb, w.e_t, w.alpha, w.delta_t,
                                          w.base_budget, w.mult, w.probe_scale, mode=mode,
                                          bufs=bufs)
        torch.cuda.synchronize()
        _check_fused(w, mode, ls, en, sel, en2, sel2)


def test_one_call_prefill_c2_repeated():
    """Repeated one-call runs on a 16k layer with reused buffers stay equal
    to the separate calls."""
    w = synth.make("c2", 2, N=16384)
    q, k, v = to_dev(w.q), to_dev(w.k), to_dev(w.v)
    ls, en = eb.entropy_probe(q, k, w.Ls, w.Lb)
    sel = eb.select_blocks(ls, en, w.N, w.Ls, w.Lb, n_kv_heads=w.Hkv)
    o = eb.sparse_prefill_attn(q, k, v, sel["idx"], sel["cnt"], w.Ls, w.Lb, w.softmax_scale)
    bufs = {}
    for _ in range(3):
        o2, sel2, _, en2 = eb.entropy_guided_prefill(q, k, v, w.Ls, w.Lb, bufs=bufs)
        torch.cuda.synchronize()
        assert torch.equal(o, o2) and torch.equal(en, en2)
        assert torch.equal(sel["idx"], sel2["idx"])


def _end_to_end_agreement(w, r):
    """Informational (not a parity bar): the oracle's own probe (binary64,
    rounded to binary32 as the GPU stores it) fed to the oracle's selection,
    against the GPU's selection.  Returns (fraction of (b, h, s) rows whose
    block list differs, fraction of heads whose rigid flag differs, fraction
    of rows whose budget differs)."""
    Lr, Hr = oracle.probe(w.q, w.k, w.Ls, w.Lb, w.probe_scale)
    ls = np.nan_to_num(Lr, nan=-np.inf).astype(np.float32)
    en = Hr.astype(np.float32)
    del Lr
    ref = oracle.select(ls, en, w.N, w.Ls, w.Lb, w.e_t, w.alpha, w.delta_t, w.base_budget,
                        w.mult)
    g = r["sel"]
    rows_diff = float(np.any(g["idx"] != ref["idx"], axis=-1).mean())
    rigid_diff = float((g["rigid"] != ref["rigid"]).mean())
    budget_diff = float((g["budget"] != ref["budget"]).mean())
    return rows_diff, rigid_diff, budget_diff


@pytest.mark.parametrize("wl", ["c2", "c3"])
def test_end_to_end_selection_agreement(wl, c3):
    """The selection the whole oracle path (probe -> select) makes against
    the GPU's, reported: rows whose block list differs, rigid flags and
    budgets.  Near-ties of fp32 scores can order differently after the
    probe's rounding, so this is not bit-exact by construction; the
    bit-exact bar is the selection on the GPU's own scores."""
    if wl == "c3":
        w, r = c3
    else:
        w = synth.make("c2", 0)
        r = run_path(w)
    rows_diff, rigid_diff, budget_diff = _end_to_end_agreement(w, r)
    say(f"  [{wl}] end-to-end: block lists differ on {rows_diff:.4%} of rows, rigid flags on "
        f"{rigid_diff:.4%} of heads, budgets on {budget_diff:.4%} of rows")
    assert rows_diff < 0.05 and rigid_diff == 0.0
