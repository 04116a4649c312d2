"""Pins of the oracle's expert-use concentration metrics (Section 5: per-layer
effective experts exp(entropy), entropy, max frequency and top-8 mass of the
native selection frequencies, averaged over layers)."""
import json
import math
import os

import numpy as np
import pytest
import scipy.stats

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_concentration.json")


def test_uniform_and_one_hot_closed_forms():
    N = 128
    eff, H, fmax, top8 = oracle.concentration(np.full((1, N), 7), 8)
    assert H == pytest.approx(math.log(N), abs=1e-12)
    assert eff == pytest.approx(N, rel=1e-12)
    assert fmax == pytest.approx(1 / N, abs=1e-15) and top8 == pytest.approx(8 / N, abs=1e-15)
    c = np.zeros((1, N), np.int64)
    c[0, 17] = 42
    assert oracle.concentration(c, 8) == (1.0, 0.0, 1.0, 1.0)


def test_two_point_distribution():
    c = np.zeros((1, 16), np.int64)
    c[0, 3], c[0, 9] = 3, 1
    eff, H, fmax, top1 = oracle.concentration(c, 1)
    want = -(0.75 * math.log(0.75) + 0.25 * math.log(0.25))
    assert H == pytest.approx(want, abs=1e-15) and eff == pytest.approx(math.exp(want), rel=1e-15)
    assert fmax == 0.75 and top1 == 0.75


def test_matches_library_entropy_on_random_counts():
    rng = np.random.default_rng(0)
    for _ in range(20):
        L, N, m = int(rng.integers(1, 6)), int(rng.integers(2, 130)), int(rng.integers(1, 12))
        c = rng.integers(0, 50, size=(L, N)) * (rng.random((L, N)) < 0.7)
        c[:, 0] += 1                                   # every layer has a selection
        Hs = [scipy.stats.entropy(c[l]) for l in range(L)]
        f = c / c.sum(axis=1, keepdims=True)
        want = (np.mean(np.exp(Hs)), np.mean(Hs), f.max(axis=1).mean(),
                np.mean([np.sort(f[l])[::-1][:m].sum() for l in range(L)]))
        got = oracle.concentration(c, m)
        assert np.allclose(got, want, rtol=1e-12, atol=1e-15)


def test_layers_without_selections_are_skipped_and_means_are_per_layer():
    c = np.zeros((3, 8), np.int64)
    c[0, :2] = 5                     # uniform over 2: eff 2
    c[2, :] = 1                      # uniform over 8: eff 8
    eff, H, fmax, top2 = oracle.concentration(c, 2)
    assert eff == pytest.approx(5.0) and H == pytest.approx((math.log(2) + math.log(8)) / 2)
    assert fmax == pytest.approx((0.5 + 0.125) / 2) and top2 == pytest.approx((1.0 + 0.25) / 2)
    assert oracle.concentration(np.zeros((2, 4), np.int64), 2) == (0.0, 0.0, 0.0, 0.0)


def test_paper_figures_fix_natural_log_and_unit_sum_frequencies():
    """The printed layer means satisfy what the definitions force: the mean of
    exp(H) is at least exp(mean H) (Jensen) and close to it, which holds for
    natural-log entropy and fails for bits; frequencies sum to one, so
    max <= top-8 mass <= min(1, 8 max) and H <= ln N."""
    g = json.load(open(GOLDEN))
    N = g["experts_per_layer"]
    for r in g["rows"]:
        assert math.exp(r["entropy"]) <= r["effective_experts"] <= 1.05 * math.exp(r["entropy"]), r
        assert not (2 ** r["entropy"] <= r["effective_experts"] <= 1.05 * 2 ** r["entropy"])
        assert r["max_frequency"] <= r["top8_mass"] <= min(1.0, 8 * r["max_frequency"])
        assert r["entropy"] <= math.log(N)


def test_oracle_counts_native_selections_of_counted_tokens():
    rng = np.random.default_rng(4)
    S, L, N, K, T, warm = 3, 2, 16, 3, 9, 2
    run = oracle.Run(L, N, K, 5, 0, S, 0, warm)
    want = np.zeros((L, N), np.int64)
    for t in range(T):
        zR = rng.normal(size=(S, L, N)).astype(np.float32)
        out = run.step(zR, rng.normal(size=(S, L, N)).astype(np.float32))
        if t >= warm:
            for s in range(S):
                for l in range(L):
                    np.add.at(want[l], out["sel"][s, l], 1)
    assert np.array_equal(run.selcount, want)
    assert run.selcount.sum() == S * L * K * (T - warm)
