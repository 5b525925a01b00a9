"""The Llama-3-70B-shaped workload (64 query / 8 KV heads, 131072 tokens) is
swept over the entropy threshold e_t in {1e-6, 1e-5, 1e-4}.  Its always-sink
heads carry sink amplitudes spread so that their largest segment entropies
straddle those thresholds; through the oracle (its probe and Algorithm 3 on
its own entropies rounded to binary32) the three thresholds classify three
different numbers of heads as rigid, and no head of the drifting (Markov)
kind is rigid at any of them."""
import numpy as np
import pytest

import oracle
from paper_2606_09508_amd import synth

EXPECTED = {1e-6: 4, 1e-5: 6, 1e-4: 7}


@pytest.fixture(scope="module")
def c5_max_entropy():
    w = synth.make("c5", 0)
    L, H = oracle.probe(w.q, w.k, w.Ls, w.Lb, w.probe_scale)
    del L
    return w, H[0].astype(np.float32)            # [Hq, C_S]


def test_thresholds_give_three_rigid_counts(c5_max_entropy):
    w, H = c5_max_entropy
    always = [h for h in range(w.Hq) if (w.plan[0, h] == synth.SINK).all()]
    assert len(always) == 8
    counts = {}
    for e_t in EXPECTED:
        rigid = [oracle.budget(H[h], e_t, w.alpha, w.delta_t, w.base_budget, w.mult)[0]
                 for h in range(w.Hq)]
        counts[e_t] = sum(rigid)
        assert not any(rigid[h] for h in range(w.Hq) if h not in always)
    assert counts == EXPECTED
    assert len(set(counts.values())) == 3
