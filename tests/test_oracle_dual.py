"""A second, independent implementation of the probe (Algorithms 1-2 and the
row entropy, Section 4.2 / Section 3) in vectorised numpy on tiny inputs,
cross-checking the C oracle.  It restates the definitions, so it is a
cross-check of the C implementation (a dropped term, a wrong index or an
off-by-one in the visible range there would show), not a pin of the
definitions themselves; those are pinned in test_oracle_pins.py."""
import numpy as np
import pytest

import oracle
from paper_2606_09508_amd.synth import from_bf16_bits, make


def probe_numpy(q_bits, k_bits, Ls, Lb, scale=1.0):
    """ln A and entropy per (b, h, s), fp64, from bf16 bits."""
    q = from_bf16_bits(q_bits).astype(np.float64)
    k = from_bf16_bits(k_bits).astype(np.float64)
    B, Hq, N, D = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    CS, CB, r = -(-N // Ls), -(-N // Lb), Ls // Lb
    # Algorithm 1: per-segment / per-block max and min over the rows
    pad_q = np.full((B, Hq, CS * Ls, D), np.nan)
    pad_q[:, :, :N] = q
    pad_k = np.full((B, Hkv, CB * Lb, D), np.nan)
    pad_k[:, :, :N] = k
    qs = pad_q.reshape(B, Hq, CS, Ls, D)
    ks = pad_k.reshape(B, Hkv, CB, Lb, D)
    qmax, qmin = np.nanmax(qs, axis=3), np.nanmin(qs, axis=3)
    kmax, kmin = np.nanmax(ks, axis=3), np.nanmin(ks, axis=3)
    L = np.full((B, Hq, CS, CB), np.nan)
    H = np.zeros((B, Hq, CS))
    for b in range(B):
        for h in range(Hq):
            g = h // G
            # Algorithm 2: the four logit products of every (segment, block)
            x = [scale * (qa @ kb.T) for qa in (qmax[b, h], qmin[b, h])
                 for kb in (kmax[b, g], kmin[b, g])]          # S1 .. S4, [CS, CB]
            for s in range(CS):
                nv = min((s + 1) * r, CB)
                p = []
                for c in range(4):
                    z = x[c][s, :nv] - x[c][s, :nv].max()
                    e = np.exp(z)
                    p.append(e / e.sum())
                A = np.maximum((p[0] + p[1]) / 2, (p[2] + p[3]) / 2)
                L[b, h, s, :nv] = np.log(A)
                nz = A > 0
                H[b, h, s] = -(A[nz] * np.log(A[nz])).sum()
    return L, H


@pytest.mark.parametrize("seed,over", [
    (0, {}),
    (1, dict(N=1000)),                       # ragged tail segment and block
    (2, dict(Hq=6, Hkv=2, N=768, Ls=256, Lb=128, base_budget=512)),
    (3, dict(B=2, N=512)),
])
def test_probe_matches_numpy_implementation(seed, over):
    w = make("c1", seed, **over)
    L_c, H_c = oracle.probe(w.q, w.k, w.Ls, w.Lb, w.probe_scale)
    L_n, H_n = probe_numpy(w.q, w.k, w.Ls, w.Lb, w.probe_scale)
    vis = ~np.isnan(L_n)
    assert np.array_equal(vis, ~np.isnan(L_c))
    # ln A: the two sum the softmax in different orders; relative 1e-12 of
    # the row's scale, or 1e-9 absolute
    assert np.allclose(L_c[vis], L_n[vis], rtol=1e-10, atol=1e-9)
    assert np.allclose(H_c, H_n, rtol=1e-9, atol=1e-15)
