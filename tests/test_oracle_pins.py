"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

Each test names the passage it follows.  None of them re-types the oracle's
formulas: they use closed forms of hand-built inputs, invariants, brute force,
exact (Decimal) evaluation of the definitions and library routines.
"""
import itertools
import math
import os
from decimal import Decimal, getcontext
from fractions import Fraction

import numpy as np
import pytest
import torch

from paper_2606_09508_amd.synth import from_bf16_bits, make, to_bf16_bits


def bf(x):
    return to_bf16_bits(np.asarray(x, np.float32))


def qk_zero(B=1, Hq=1, Hkv=1, N=256, D=128):
    return (np.zeros((B, Hq, N, D), np.float32), np.zeros((B, Hkv, N, D), np.float32))


# --------------------------------------------------------------------------
# Algorithm 1 (representation vectors)
# --------------------------------------------------------------------------

def test_pool_matches_numpy_reduction_and_is_exact(orc):
    rng = np.random.default_rng(1)
    x = bf(rng.standard_normal((1000, 128)).astype(np.float32) * 3)
    for L in (64, 128, 1000, 7):
        mx, mn = orc.pool(x, L)
        xf = from_bf16_bits(x).astype(np.float64)
        pad = (-len(xf)) % L
        g = np.concatenate([xf, np.full((pad, 128), np.nan)]).reshape(-1, L, 128)
        np.testing.assert_array_equal(mx, np.nanmax(g, axis=1))
        np.testing.assert_array_equal(mn, np.nanmin(g, axis=1))
        # pooled values are input values, bit for bit
        assert set(bf(mx.astype(np.float32)).ravel()) <= set(x.ravel())


def test_pool_permutation_invariance(orc):
    rng = np.random.default_rng(2)
    x = bf(rng.standard_normal((512, 128)).astype(np.float32))
    mx, mn = orc.pool(x, 128)
    perm = np.concatenate([rng.permutation(128) + 128 * s for s in range(4)])
    mx2, mn2 = orc.pool(np.ascontiguousarray(x[perm]), 128)
    np.testing.assert_array_equal(mx, mx2)
    np.testing.assert_array_equal(mn, mn2)


# --------------------------------------------------------------------------
# Algorithm 2 + row entropy: closed forms
# --------------------------------------------------------------------------

@pytest.mark.parametrize("N,Ls,Lb", [(1024, 128, 64), (1000, 128, 64), (512, 256, 64),
                                     (768, 256, 128)])
def test_uniform_rows_entropy_is_ln_nvis(orc, N, Ls, Lb):
    """Q = 0 makes every logit 0, so every softmax is uniform over the visible
    blocks and A_obs = 1/n_vis: H = ln n_vis, ln A = -ln n_vis (Section 3's
    entropy of a uniform row)."""
    q, k = qk_zero(N=N)
    k[:] = np.random.default_rng(3).standard_normal(k.shape)
    L, H = orc.probe(bf(q), bf(k), Ls, Lb)
    r, CB = Ls // Lb, -(-N // Lb)
    for s in range(H.shape[2]):
        nvis = min((s + 1) * r, CB)
        assert H[0, 0, s] == pytest.approx(math.log(nvis), rel=1e-14, abs=1e-15)
        np.testing.assert_allclose(L[0, 0, s, :nvis], -math.log(nvis), rtol=1e-14, atol=1e-15)
        assert np.isnan(L[0, 0, s, nvis:]).all()   # block-causal: nothing past n_vis


def test_one_hot_rows_have_zero_entropy(orc):
    """A sink far above everything else gives one-hot softmaxes: H ~ 0."""
    q, k = qk_zero(N=512)
    q[..., 5] = 4.0
    k[:, :, :64, 5] = 64.0                       # logit gap 256 in every combo
    L, H = orc.probe(bf(q), bf(k), 128, 64)
    assert (H < 1e-90).all()
    np.testing.assert_allclose(L[0, 0, :, 0], 0.0, atol=1e-90)


@pytest.mark.parametrize("M", [0.5, 3.0, 40.0])
def test_pair_average_is_half_half(orc, M):
    """Qmax = Qmin; block 0 keys span [-M, M] at coordinate 0, block 1 keys are 0.
    S1 = S3 = (sigma(M), sigma(-M)) and S2 = S4 = (sigma(-M), sigma(M)), so
    (S1+S2)/2 = (1/2, 1/2) exactly (sigma(x) + sigma(-x) = 1): H = ln 2."""
    q, k = qk_zero(N=128)
    q[0, 0, :, 0] = 1.0
    k[0, 0, 0, 0] = M
    k[0, 0, 1, 0] = -M
    L, H = orc.probe(bf(q), bf(k), 128, 64)
    assert H[0, 0, 0] == pytest.approx(math.log(2), rel=1e-14)
    np.testing.assert_allclose(L[0, 0, 0, :2], -math.log(2), rtol=1e-14)


@pytest.mark.parametrize("c,M,scale", [(1.0, 2.0, 1.0), (2.0, 1.5, 1.0), (1.0, 8.0, 0.25)])
def test_max_combination_is_not_renormalised(orc, c, M, scale):
    """Qmax[0] = c, Qmin[0] = -c; block 0 keys all M, block 1 keys 0.  With
    x = scale c M: S1 = S2 = (sigma(x), sigma(-x)), S3 = S4 = (sigma(-x), sigma(x)),
    A = max of the pair averages = (sigma(x), sigma(x)) (sum > 1, used as is):
    H = -2 sigma(x) ln sigma(x)."""
    q, k = qk_zero(N=128)
    q[0, 0, 0, 0] = c
    q[0, 0, 1, 0] = -c
    k[0, 0, :64, 0] = M
    L, H = orc.probe(bf(q), bf(k), 128, 64, probe_scale=scale)
    x = scale * c * M
    sig = 1.0 / (1.0 + math.exp(-x))
    assert H[0, 0, 0] == pytest.approx(-2 * sig * math.log(sig), rel=1e-13)
    np.testing.assert_allclose(L[0, 0, 0, :2], math.log(sig), rtol=1e-13)


def test_max_picks_different_blocks_gives_zero_entropy(orc):
    """S1 = S2 one-hot at block a, S3 = S4 one-hot at block b: A = 1 at a and at
    b, H = 0 (a renormalised A would give ln 2).  Other blocks: ln A = -cM."""
    q, k = qk_zero(N=512)
    q[0, 0, 0, 0] = 1.0
    q[0, 0, 1, 0] = -1.0
    a, b = 1, 5
    k[0, 0, 64 * a: 64 * (a + 1), 0] = 100.0
    k[0, 0, 64 * b: 64 * (b + 1), 0] = -100.0
    L, H = orc.probe(bf(q), bf(k), 512, 64)       # one segment, 8 visible blocks
    assert H[0, 0, 0] < 1e-35
    assert abs(L[0, 0, 0, a]) < 1e-40 and abs(L[0, 0, 0, b]) < 1e-40
    others = [j for j in range(8) if j not in (a, b)]
    np.testing.assert_allclose(L[0, 0, 0, others], -100.0, rtol=1e-14)


def test_shift_invariance(orc):
    """Adding t to every logit of a row (a key coordinate equal to 1 for every
    key, a query coordinate t) changes neither ln A nor H."""
    rng = np.random.default_rng(4)
    q = rng.standard_normal((1, 2, 512, 128)).astype(np.float32)
    k = rng.standard_normal((1, 1, 512, 128)).astype(np.float32)
    q[..., 127] = 0.0
    k[..., 127] = 1.0
    L0, H0 = orc.probe(bf(q), bf(k), 128, 64)
    q[..., 127] = 37.0
    L1, H1 = orc.probe(bf(q), bf(k), 128, 64)
    np.testing.assert_allclose(H1, H0, rtol=1e-9, atol=1e-300)
    m = ~np.isnan(L0)
    np.testing.assert_allclose(L1[m], L0[m], rtol=1e-9, atol=1e-9)


def _exact_row(qrows, kblocks, scale):
    """Definition of Algorithms 1-2 and the entropy, evaluated exactly:
    logits as Fractions, softmax / log in 60-digit Decimal."""
    getcontext().prec = 60
    qf = [[Fraction(float(v)) for v in row] for row in qrows]
    D = len(qf[0])
    qmax = [max(r[d] for r in qf) for d in range(D)]
    qmin = [min(r[d] for r in qf) for d in range(D)]
    kreps = []
    for blk in kblocks:
        kf = [[Fraction(float(v)) for v in row] for row in blk]
        kreps.append(([max(r[d] for r in kf) for d in range(D)],
                      [min(r[d] for r in kf) for d in range(D)]))
    sc = Fraction(scale)

    def soft(qv, which):
        xs = [sc * sum(a * b for a, b in zip(qv, kr[which])) for kr in kreps]
        es = [Decimal(x.numerator) / Decimal(x.denominator) for x in xs]
        m = max(es)
        ex = [(e - m).exp() for e in es]
        tot = sum(ex)
        return [e / tot for e in ex]

    S1, S2, S3, S4 = soft(qmax, 0), soft(qmax, 1), soft(qmin, 0), soft(qmin, 1)
    A = [max((a + b) / 2, (c + d) / 2) for a, b, c, d in zip(S1, S2, S3, S4)]
    H = -sum(a * a.ln() for a in A if a > 0)
    return [float(a.ln()) for a in A], float(H)


@pytest.mark.parametrize("gap", [0.0, 5.0, 20.0, 28.0, 35.0])
def test_entropy_matches_exact_evaluation(orc, gap):
    """Near-one-hot rows (H down to ~1e-13) carry the rigid / dynamic decision
    (e_t = 1e-5); the fp64 oracle must match an exact evaluation to 1e-12."""
    rng = np.random.default_rng(int(gap * 10) + 5)
    D, N = 128, 256
    qf = np.zeros((1, 1, N, D), np.float32)
    kf = np.zeros((1, 1, N, D), np.float32)
    qf[0, 0, :, :8] = rng.standard_normal((N, 8))
    kf[0, 0, :, :8] = rng.standard_normal((N, 8))
    qf[0, 0, :, 9] = 1.0
    kf[0, 0, :64, 9] = gap                       # block 0 sink of size `gap`
    q, k = bf(qf), bf(kf)
    L, H = orc.probe(q, k, 128, 64)
    for s in range(2):
        nvis = 2 * (s + 1)
        qrows = from_bf16_bits(q[0, 0, 128 * s: 128 * (s + 1), :10])
        kblocks = [from_bf16_bits(k[0, 0, 64 * j: 64 * (j + 1), :10]) for j in range(nvis)]
        lnA, Hx = _exact_row(qrows, kblocks, 1.0)
        assert H[0, 0, s] == pytest.approx(Hx, rel=1e-12, abs=1e-300)
        np.testing.assert_allclose(L[0, 0, s, :nvis], lnA, rtol=1e-12, atol=1e-14)


def test_gqa_query_head_reads_its_group(orc):
    """Hq = 4, Hkv = 2: heads 0-1 read key head 0 and heads 2-3 key head 1;
    a G = 1 problem built from the same tensors gives the same rows."""
    rng = np.random.default_rng(6)
    q = bf(rng.standard_normal((1, 4, 512, 128)).astype(np.float32))
    k = bf(rng.standard_normal((1, 2, 512, 128)).astype(np.float32))
    L, H = orc.probe(q, k, 128, 64)
    for h in range(4):
        g = h // 2
        L1, H1 = orc.probe(np.ascontiguousarray(q[:, h:h + 1]), np.ascontiguousarray(k[:, g:g + 1]),
                           128, 64)
        np.testing.assert_array_equal(H1[0, 0], H[0, h])


def test_sampled_rows_equal_full_rows(orc):
    w = make("c1", 3)
    L, H = orc.probe(w.q, w.k, w.Ls, w.Lb)
    rows = np.array([[0, 2, 5], [0, 0, 7], [0, 3, 0]], np.int32)
    Ls_, Hs_ = orc.probe(w.q, w.k, w.Ls, w.Lb, rows=rows)
    for t, (b, h, s) in enumerate(rows):
        np.testing.assert_array_equal(Hs_[t], H[b, h, s])
        np.testing.assert_array_equal(Ls_[t], L[b, h, s])


# --------------------------------------------------------------------------
# Algorithm 3: hand-worked sequences (alpha = 0.5, Delta_t = 0.4, e_t = 1e-5)
# --------------------------------------------------------------------------

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _golden_lines(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return [ln.strip() for ln in f if ln.strip() and not ln.lstrip().startswith("#")]


def _alg3_cases():
    """(entropies, rigid, budgets in tokens worked by hand, k = floor(B / 64))
    from the golden file."""
    cases = []
    for ln in _golden_lines("algorithm3_worked_budgets.txt"):
        e, rg, Bx, kx = (part.split() for part in ln.split("|"))
        cases.append(([float(x) for x in e], rg == ["1"], [float(x) for x in Bx],
                      [int(x) for x in kx]))
    return cases


ALG3_CASES = _alg3_cases()
ALG3_CONST = {k: float(v) for k, v in (ln.split() for ln in _golden_lines("algorithm3_constants.txt"))}


def test_defaults_are_the_papers_constants(orc):
    """The oracle, the binding and the input generator default to the
    constants Algorithm 3 and the experimental setup state."""
    import inspect
    from paper_2606_09508_amd import binding, synth
    c = ALG3_CONST
    want = dict(e_t=c["e_t"], alpha=c["alpha"], delta_t=c["delta_t"],
                base_budget=c["base_budget_tokens"], mult=c["cap_multiplier"])
    for fn in (orc.budget, binding.budget_params):
        d = {k: v.default for k, v in inspect.signature(fn).parameters.items()
             if v.default is not inspect.Parameter.empty}
        for k, v in want.items():
            assert d[k] == v, (fn.__name__, k)
    w = synth.make("c3", 0, generate_tensors=False)
    assert (w.e_t, w.alpha, w.delta_t, w.base_budget, w.mult) == \
        (want["e_t"], want["alpha"], want["delta_t"], want["base_budget"], want["mult"])


@pytest.mark.parametrize("e,rigid,Bx,kx", ALG3_CASES)
def test_algorithm3_worked_sequences(orc, e, rigid, Bx, kx):
    c = ALG3_CONST
    rg, B = orc.budget(np.asarray(e, np.float32), c["e_t"], c["alpha"], c["delta_t"],
                       int(c["base_budget_tokens"]), int(c["cap_multiplier"]))
    assert rg == rigid
    np.testing.assert_allclose(B, Bx, rtol=0, atol=2e-3)
    assert [int(math.floor(b / 64)) for b in B] == kx


def test_algorithm3_small_budget_example(orc):
    """B_h = 256 (a quarter of 16 blocks): worked by hand,
    B = 256, 296.23, 693.03, 641.83, 675.96, 629.03, 656.28, 605.08."""
    e = np.asarray([0.7, 0.2, 0.9, 0.9, 0.3, 0.31, 0.5, 0.5], np.float32)
    rg, B = orc.budget(e, 1e-5, 0.5, 0.4, 256, 3)
    assert not rg
    np.testing.assert_allclose(B, [256, 296.23, 693.03, 641.83, 675.96, 629.03, 656.28, 605.08],
                               atol=0.02)
    assert [int(b // 64) for b in B] == [4, 4, 10, 10, 10, 9, 10, 9]


def test_algorithm3_nan_entropy_is_dynamic_and_clamps(orc):
    rg, B = orc.budget(np.asarray([1e-7, np.nan, 1e-7], np.float32))
    assert not rg
    assert np.isfinite(B).all() and (B >= 2048).all() and (B <= 6144).all()


# --------------------------------------------------------------------------
# Selection (Section 4.2, Eq. t_topk)
# --------------------------------------------------------------------------

def _keyed(v):
    """Rank of a float32 score: NaN lowest, -0 == +0."""
    return (-math.inf, 0) if math.isnan(v) else (1, float(v) + 0.0)


def _brute_topk(scores, k):
    """The unique k-subset whose members all beat every non-member under
    (score, index), found by enumerating every subset."""
    n = len(scores)
    key = [(_keyed(float(scores[j])), j) for j in range(n)]
    found = []
    for sub in itertools.combinations(range(n), k):
        inside = set(sub)
        if all(key[a] > key[b] for a in inside for b in range(n) if b not in inside):
            found.append(sub)
    assert len(found) == 1
    return sorted(found[0])


def _select_one_row(orc, scores, k_budget_blocks, s):
    """Drive orc.select on one head whose segment s has the given past scores."""
    Ls, Lb = 128, 64
    r = Ls // Lb
    CS = s + 1
    N = CS * Ls
    CB = N // Lb
    ls = np.full((1, 1, CS, CB), -1.0, np.float32)
    ls[0, 0, s, : s * r] = scores
    en = np.full((1, 1, CS), 1e-7, np.float32)   # rigid: B = B_h everywhere
    out = orc.select(ls, en, N, Ls, Lb, base_budget=k_budget_blocks * Lb, mult=3)
    c = out["cnt"][0, 0, s]
    return out, list(out["idx"][0, 0, s, :c])


@pytest.mark.parametrize("seed", range(6))
def test_topk_equals_exhaustive_enumeration(orc, seed):
    rng = np.random.default_rng(seed)
    s = 8                                       # 16 past blocks
    scores = rng.choice([-3.0, -1.5, -1.0, -0.5, 0.0, -0.0, -np.inf, np.nan],
                        size=16).astype(np.float32)
    if seed % 2:
        scores = rng.standard_normal(16).astype(np.float32)
    for k in (1, 3, 7, 12):
        out, idx = _select_one_row(orc, scores, k, s)
        want = _brute_topk(scores, k) + [16, 17]
        assert idx == want
        assert out["budget"][0, 0, s] == k
        assert (out["idx"][0, 0, s, len(idx):] == -1).all()


def test_uniform_scores_pick_most_recent_blocks(orc):
    """Equal scores: the tie rule keeps the most recent past blocks."""
    out, idx = _select_one_row(orc, np.zeros(20, np.float32), 5, 10)
    assert idx == [15, 16, 17, 18, 19, 20, 21]


def test_rigid_and_capped_budgets(orc):
    """A rigid head gets k = min(B_h / L_B, n_past(s)) in every segment."""
    w = make("c1", 0)
    L, H = orc.probe(w.q, w.k, w.Ls, w.Lb)
    out = orc.select(L.astype(np.float32), H.astype(np.float32), w.N, w.Ls, w.Lb,
                     base_budget=w.base_budget)
    assert list(out["rigid"][0]) == [1, 1, 0, 0]
    for h in (0, 1):
        assert list(out["budget"][0, h]) == [min(4, 2 * s) for s in range(8)]
    for h in range(4):
        for s in range(8):
            c = out["cnt"][0, h, s]
            idx = out["idx"][0, h, s, :c]
            assert c == out["budget"][0, h, s] + 2
            assert (np.diff(idx) > 0).all() and idx[-2:].tolist() == [2 * s, 2 * s + 1]


def test_work_count_bound(orc):
    """Appendix A, Eq. t_spa: computed query-key pairs per head are at most
    N (L_S + 1) / 2 + 3 B_h N (diagonal triangle + capped budget)."""
    w = make("c2", 1, N=8192)
    L, H = orc.probe(w.q, w.k, w.Ls, w.Lb)
    out = orc.select(L.astype(np.float32), H.astype(np.float32), w.N, w.Ls, w.Lb,
                     base_budget=512)
    for h in range(w.Hq):
        k = out["budget"][0, h].astype(np.int64)
        pairs = int(np.sum(w.Ls * (w.Ls + 1) // 2 + w.Ls * w.Lb * k))
        assert pairs <= w.N * (w.Ls + 1) // 2 + 3 * 512 * w.N
        assert (k <= 3 * 512 // w.Lb).all()


def test_full_budget_selects_every_visible_block(orc):
    w = make("c1", 1)
    L, H = orc.probe(w.q, w.k, w.Ls, w.Lb)
    out = orc.select(L.astype(np.float32), H.astype(np.float32), w.N, w.Ls, w.Lb,
                     base_budget=w.N)
    for s in range(w.CS):
        c = out["cnt"][0, :, s]
        assert (c == 2 * (s + 1)).all()
        np.testing.assert_array_equal(out["idx"][0, :, s, : 2 * (s + 1)],
                                      np.tile(np.arange(2 * (s + 1)), (w.Hq, 1)))


# --------------------------------------------------------------------------
# Attention (Section 2 definition; sparse key sets of Section 4.2)
# --------------------------------------------------------------------------

def _sdpa_fp64(w, mask_fn):
    q = torch.from_numpy(from_bf16_bits(w.q).astype(np.float64))
    k = torch.from_numpy(from_bf16_bits(w.k).astype(np.float64))
    v = torch.from_numpy(from_bf16_bits(w.v).astype(np.float64))
    G = w.Hq // w.Hkv
    k = k.repeat_interleave(G, dim=1)
    v = v.repeat_interleave(G, dim=1)
    mask = torch.from_numpy(mask_fn())
    return torch.nn.functional.scaled_dot_product_attention(
        q, k, v, attn_mask=mask, scale=w.softmax_scale).numpy()


def _all_rows(w):
    return np.array([[b, h, i] for b in range(w.B) for h in range(w.Hq) for i in range(w.N)],
                    np.int32)


def test_dense_causal_matches_library_sdpa(orc):
    w = make("c1", 2, N=512)
    rows = _all_rows(w)
    got = orc.attention(w.q, w.k, w.v, rows).reshape(w.B, w.Hq, w.N, w.D)
    ref = _sdpa_fp64(w, lambda: np.tril(np.ones((w.N, w.N), bool)))
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_sparse_matches_library_sdpa_with_block_mask(orc):
    w = make("c1", 4, N=768, Hq=4, Hkv=2)
    L, H = orc.probe(w.q, w.k, w.Ls, w.Lb)
    sel = orc.select(L.astype(np.float32), H.astype(np.float32), w.N, w.Ls, w.Lb,
                     base_budget=128)
    rows = _all_rows(w)
    got = orc.attention(w.q, w.k, w.v, rows, block_idx=sel["idx"], block_cnt=sel["cnt"],
                        Ls=w.Ls, Lb=w.Lb).reshape(w.B, w.Hq, w.N, w.D)

    def mask():
        m = np.zeros((w.B, w.Hq, w.N, w.N), bool)
        for h in range(w.Hq):
            for i in range(w.N):
                s = i // w.Ls
                for blk in sel["idx"][0, h, s, : sel["cnt"][0, h, s]]:
                    m[0, h, i, blk * w.Lb: (blk + 1) * w.Lb] = True
        return m & np.tril(np.ones((w.N, w.N), bool))

    ref = _sdpa_fp64(w, mask)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_full_budget_sparse_equals_dense(orc):
    w = make("c1", 5, N=640)
    L, H = orc.probe(w.q, w.k, w.Ls, w.Lb)
    sel = orc.select(L.astype(np.float32), H.astype(np.float32), w.N, w.Ls, w.Lb,
                     base_budget=w.N)
    rows = _all_rows(w)
    a = orc.attention(w.q, w.k, w.v, rows, block_idx=sel["idx"], block_cnt=sel["cnt"])
    d = orc.attention(w.q, w.k, w.v, rows)
    np.testing.assert_array_equal(a, d)


def test_attention_special_cases(orc):
    w = make("c1", 6, N=256)
    vv = w.v.copy()
    vv[0, 0, :] = vv[0, 0, 17]                   # constant value rows
    rows = _all_rows(w)
    out = orc.attention(w.q, w.k, vv, rows)
    np.testing.assert_allclose(out, np.tile(from_bf16_bits(vv[0, 0, 17]).astype(np.float64),
                                            (len(rows), 1)), rtol=1e-13)
    out0 = orc.attention(w.q, w.k, w.v, np.array([[0, h, 0] for h in range(4)], np.int32))
    for h in range(4):                            # query 0 sees only key 0
        np.testing.assert_array_equal(out0[h], from_bf16_bits(w.v[0, 0, 0]).astype(np.float64))


# --------------------------------------------------------------------------
# Classification variants (uniform budget, GQA-group mean, per-segment rule)
# --------------------------------------------------------------------------

def _select_k(orc, e, mode, n_kv=None, e_t=1e-5, Ls=4096, Lb=64):
    """k_s and rigid flags of orc.select for entropies e [Hq, C_S] (random
    scores; only the budgets are compared).  Ls = 4096 keeps n_past above
    every budget here."""
    e = np.asarray(e, np.float32)
    Hq, CS = e.shape
    N = CS * Ls
    rng = np.random.default_rng(0)
    ls = rng.standard_normal((1, Hq, CS, N // Lb)).astype(np.float32)
    r = orc.select(ls, e[None], N, Ls, Lb, e_t=e_t, base_budget=2048, mult=3, mode=mode,
                   n_kv_heads=n_kv)
    return r["budget"][0], r["rigid"][0]


def test_segment_rule_worked_sequence(orc):
    """B_h = 2048, alpha B_h = 1024, Delta_t = 0.4, cap 6144; worked by hand.
    e = [2, 1, 1e-6, 1e-6, 3, 3]:
      per segment: s1 |1-2|/2 = 0.5 -> +102.4 = 2150.4; s2, s3 below e_t -> 2048;
                   s4 ratio ~3e6 -> cap 6144; s5 ratio 0 -> -409.6 = 5734.4
      per head (dynamic): s2 |1e-6-1|/1 = 0.999999 -> +614.398976 = 2764.798976;
                   s3 -409.6 = 2355.198976; s4 cap 6144; s5 5734.4
    k = floor(B / 64), k_0 = 0 (no past block)."""
    e = np.asarray([2.0, 1.0, 1e-6, 1e-6, 3.0, 3.0], np.float32)
    rg, B = orc.budget_segment(e)
    assert not rg
    np.testing.assert_allclose(B, [2048, 2150.4, 2048, 2048, 6144, 5734.4], rtol=1e-12)
    rg, B = orc.budget(e)
    np.testing.assert_allclose(B, [2048, 2150.4, 2764.798976, 2355.198976, 6144, 5734.4],
                               rtol=1e-12)
    k, rigid = _select_k(orc, e[None], orc.CLASSIFY_SEGMENT)
    assert k.tolist() == [[0, 33, 32, 32, 96, 89]] and rigid.tolist() == [0]
    k, rigid = _select_k(orc, e[None], orc.CLASSIFY_HEAD)
    assert k.tolist() == [[0, 33, 43, 36, 96, 89]] and rigid.tolist() == [0]


def test_segment_rule_reduces_to_head_rule(orc):
    """All segments rigid, or none: the per-segment rule equals Algorithm 3."""
    rng = np.random.default_rng(7)
    for e in (rng.uniform(1e-9, 9e-6, 40), rng.uniform(1e-3, 5.0, 40)):
        e = e.astype(np.float32)
        a, Ba = orc.budget(e)
        b, Bb = orc.budget_segment(e)
        assert a == b
        assert np.array_equal(Ba, Bb)


def test_group_mean_entropy(orc):
    e = np.asarray([[1.0, 2.0, 0.5], [3.0, 2.0, 0.25]], np.float32)
    assert orc.group_entropy(e).tolist() == [2.0, 2.0, 0.375]
    x = np.random.default_rng(3).uniform(0, 4, 50).astype(np.float32)
    assert np.array_equal(orc.group_entropy(np.stack([x] * 7)), x)   # identical heads


def test_group_mode_worked_example(orc):
    """Two KV groups of two heads (e_t = 1e-5).  Group 0: both heads
    [2, 1, 1e-6] -> the mean is the same row: B = 2048, 2150.4, 2764.798976,
    k = 0, 33, 43.  Group 1: [1e-6]*3 and [1e-6, 1e-6, 3e-5] -> means
    [1e-6, 1e-6, 1.55e-5], dynamic (the last mean reaches e_t): s1 ratio 0 ->
    -409.6 -> clamp 2048; s2 |1.55e-5 - 1e-6| / 1e-6 = 14.5 -> cap 6144, so
    k = 0, 32, 96 for both heads.  Per head, head 2 would be rigid (k = 32)."""
    e = np.asarray([[2, 1, 1e-6], [2, 1, 1e-6], [1e-6, 1e-6, 1e-6], [1e-6, 1e-6, 3e-5]],
                   np.float32)
    k, rigid = _select_k(orc, e, orc.CLASSIFY_GQA_GROUP, n_kv=2)
    assert k.tolist() == [[0, 33, 43], [0, 33, 43], [0, 32, 96], [0, 32, 96]]
    assert rigid.tolist() == [0, 0, 0, 0]
    k, rigid = _select_k(orc, e, orc.CLASSIFY_HEAD)
    assert k.tolist() == [[0, 33, 43], [0, 33, 43], [0, 32, 32], [0, 32, 96]]
    assert rigid.tolist() == [0, 0, 1, 0]


def test_uniform_budget_is_infinite_threshold(orc):
    """e_t = +inf classifies every head rigid: k_s = min(B_h / L_B, n_past)
    for every head whatever its entropies (a fixed k shared by all heads)."""
    e = np.random.default_rng(9).uniform(0, 8, (4, 6)).astype(np.float32)
    k, rigid = _select_k(orc, e, orc.CLASSIFY_HEAD, e_t=np.inf, Ls=128)
    assert rigid.tolist() == [1, 1, 1, 1]
    assert k.tolist() == [[min(32, 2 * s) for s in range(6)]] * 4
