"""Pins of the oracle's FFN gates.  The paper runs the selected experts
without fixing how their outputs are weighted; the reading taken here is the
native probabilities of the selected experts renormalised to sum to one.
The checks below use properties of that reading, computed with fp64
arithmetic on the logits and not through the oracle's softmax: the gates sum
to one, a single selected expert gets weight one, the ratio of two gates is
exp of their logit difference, gates follow the selection order, and with
K = N they are the softmax itself."""
import numpy as np
import pytest

import oracle


def gates_of(zR, K):
    S, L, N = zR.shape
    run = oracle.Run(L, N, K, K, 0, S, oracle.MODE_TEMPORAL)
    out = run.step(zR, zR, None, want=("sel", "gate"))
    return out["sel"], out["gate"]


@pytest.mark.parametrize("N,K", [(16, 1), (16, 4), (128, 8), (100, 7), (32, 32)])
def test_gates_are_renormalised_selected_probabilities(N, K):
    rng = np.random.default_rng(N * 100 + K)
    S, L = 5, 3
    zR = (rng.normal(size=(S, L, N)) * 2.0).astype(np.float32)
    sel, gate = gates_of(zR, K)
    for s in range(S):
        for l in range(L):
            g, e = gate[s, l], sel[s, l]
            assert abs(g.sum() - 1.0) <= 1e-12
            if K == 1:
                assert g[0] == 1.0
            z = zR[s, l].astype(np.float64)
            ratio = np.exp(z[e] - z[e[0]])      # p_e / p_e0 in exact arithmetic
            assert np.allclose(g / g[0], ratio, rtol=2e-6, atol=0.0)
            assert np.all(np.diff(g) <= 0.0)    # selection order is descending logit
            if K == N:
                p = np.exp(z - z.max())
                p /= p.sum()
                assert np.allclose(g, p[e], rtol=2e-6, atol=1e-30)


def test_gates_do_not_depend_on_unselected_logits():
    # raising an unselected expert's logit (keeping it below the K-th) changes
    # every probability but not the renormalised gates of the selection
    rng = np.random.default_rng(11)
    N, K = 32, 4
    z = (rng.normal(size=(1, 1, N))).astype(np.float32)
    sel0, g0 = gates_of(z, K)
    kth = z[0, 0, sel0[0, 0, -1]]
    z2 = z.copy()
    other = [e for e in range(N) if e not in set(sel0[0, 0].tolist())][0]
    z2[0, 0, other] = np.float32(kth - 0.5)
    sel1, g1 = gates_of(z2, K)
    assert np.array_equal(sel0, sel1)
    assert np.allclose(g0, g1, rtol=2e-6, atol=0.0)
