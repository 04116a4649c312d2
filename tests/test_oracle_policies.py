"""Pins of the oracle's classical retention policies (LRU, LFU, LRFU) and of
the Spatio-only mode.

The paper names the classical cache-update baselines (Section 4.1, Table 1
"Cache-Update Methods"; LRFU with lambda = 0.5) and the Spatio-only ablation
(Section 5 ablations, Appendix B.4) but prints no algorithm for them.  The
references here are written from the textbook definitions, in a different
form from the oracle's (an ordered recency list instead of time stamps, counts
recomputed from the whole selection history, the LRFU value summed directly
from its definition in fp64), plus a hand-worked sequence on which the three
policies disagree.
"""
import numpy as np
import pytest

import oracle
from oracle import (MODE_SPATIO_ONLY, MODE_TEMPORAL, POLICY_LFU, POLICY_LRFU, POLICY_LRU)
from test_oracle_replay import random_logits, ref_refine


def one_hot_logits(seq, N):
    """Native logits [T][1][1][N] whose Top-1 is seq[t]."""
    z = np.zeros((len(seq), 1, 1, N), np.float32)
    for t, e in enumerate(seq):
        z[t, 0, 0, e] = 1.0
    return z


def run_caches(z, L, N, K, C, policy, lam=0.5, R=0, mode=MODE_TEMPORAL, zS=None, S=1):
    run = oracle.Run(L, N, K, C, R, S, mode, policy=policy, lrfu_lambda=lam)
    caches, outs = [], []
    for t in range(z.shape[0]):
        out = run.step(z[t], None, None if zS is None else zS[t], want="all")
        caches.append(run.cache.copy())
        outs.append(out)
    return run, caches, outs


# ------------------------------------------------------------ hand-worked
# N = 4, K = 1, capacity 2, selections 0, 0, 1, 2, 3.
#   t = 3 (2 arrives, cache {0, 1} full):
#     LRU evicts 0 (last used at t = 1, 1 at t = 2)          -> {1, 2}
#     LFU evicts 1 (1 use against 2)                           -> {0, 2}
#     LRFU(0.5): C_0 = (1 w + 1) w^2 = 0.854, C_1 = w = 0.707 -> evicts 1 -> {0, 2}
#   t = 4 (3 arrives):
#     LRU evicts 1 (t = 2 against 3)                           -> {2, 3}
#     LFU evicts 2 (1 use against 2)                           -> {0, 3}
#     LRFU: C_0 = 0.854 w = 0.604, C_2 = w = 0.707            -> evicts 0 -> {2, 3}
HAND = {
    POLICY_LRU: ({1, 2}, {2, 3}),
    POLICY_LFU: ({0, 2}, {0, 3}),
    POLICY_LRFU: ({0, 2}, {2, 3}),
}


@pytest.mark.parametrize("policy", [POLICY_LRU, POLICY_LFU, POLICY_LRFU])
def test_hand_worked_sequence(policy):
    z = one_hot_logits([0, 0, 1, 2, 3], 4)
    run, caches, outs = run_caches(z, 1, 4, 1, 2, policy)
    at3 = set(np.nonzero(caches[3][0, 0])[0].tolist())
    at4 = set(np.nonzero(caches[4][0, 0])[0].tolist())
    assert (at3, at4) == HAND[policy]
    # misses: 0, then 1, 2, 3 -> 4 of 5 accesses
    t = run.totals()
    assert t["demand_misses"] == 4 and t["hits"] == 1


# ------------------------------------------------------------ independent forms
def selections(zR, K):
    """Top-K of native logits per token, ties to the lower index."""
    T, L, N = zR.shape
    out = np.empty((T, L, K), np.int64)
    for t in range(T):
        for l in range(L):
            out[t, l] = np.lexsort((np.arange(N), -zR[t, l].astype(np.float64)))[:K]
    return out


def ref_lru(sels, C):
    """Ordered recency list (least recent first); the experts used at the
    same token are ordered by index, lower first."""
    order, cache, hist = [], set(), []
    for S in sels:
        S = set(int(e) for e in S)
        for e in sorted(S - cache):
            if len(cache) < C:
                cache.add(e)
            else:
                v = next(u for u in order if u in cache and u not in S)
                cache.discard(v)
                cache.add(e)
        order = [u for u in order if u not in S] + sorted(S)
        hist.append(set(cache))
    return hist


def ref_lfu(sels, C):
    """Counts recomputed from the whole selection history at every token."""
    cache, hist = set(), []
    for t, S in enumerate(sels):
        S = set(int(e) for e in S)
        count = lambda u: sum(u in set(int(x) for x in sels[q]) for q in range(t + 1))
        for e in sorted(S - cache):
            if len(cache) < C:
                cache.add(e)
            else:
                v = min(cache - S, key=lambda u: (count(u), u))
                cache.discard(v)
                cache.add(e)
        hist.append(set(cache))
    return hist


def ref_lrfu(sels, C, lam):
    """CRF_e(t) = sum over uses t_i <= t of (1/2)^(lambda (t - t_i)), in fp64."""
    cache, hist = set(), []
    for t, S in enumerate(sels):
        S = set(int(e) for e in S)
        crf = lambda u: sum(0.5 ** (lam * (t - q)) for q in range(t + 1) if u in set(int(x) for x in sels[q]))
        for e in sorted(S - cache):
            if len(cache) < C:
                cache.add(e)
            else:
                v = min(cache - S, key=lambda u: (crf(u), u))
                cache.discard(v)
                cache.add(e)
        hist.append(set(cache))
    return hist


CASES = [(12, 3, 5, 30), (16, 4, 6, 40), (10, 2, 2, 30), (8, 2, 8, 25), (20, 1, 4, 30)]


def tie_logits(rng, T, L, N):
    zR = random_logits(rng, T, 1, L, N)[0][:, 0]
    return (np.round(zR * 2) / 2).astype(np.float32)     # frequent equal logits


@pytest.mark.parametrize("N,K,C,T", CASES)
@pytest.mark.parametrize("policy,ref", [(POLICY_LRU, ref_lru), (POLICY_LFU, ref_lfu),
                                        (POLICY_LRFU, lambda s, C: ref_lrfu(s, C, 0.5))])
def test_policy_matches_independent_form(N, K, C, T, policy, ref):
    rng = np.random.default_rng(N * 1000 + K * 10 + C)
    L = 2
    zR = tie_logits(rng, T, L, N)
    sels = selections(zR, K)
    _, caches, _ = run_caches(zR[:, None], L, N, K, C, policy)
    for l in range(L):
        want = ref(sels[:, l], C)
        for t in range(T):
            assert set(np.nonzero(caches[t][0, l])[0].tolist()) == want[t], (policy, l, t)


def test_lrfu_limits():
    """lambda = 0 weighs every use equally (LFU); lambda = 1 makes the most
    recent use dominate (LRU) when no two experts share their last use
    (K = 1) and before fp32 saturates (T <= 20)."""
    rng = np.random.default_rng(11)
    N, C, L = 10, 4, 3
    z = tie_logits(rng, 60, L, N)[:, None]
    _, c_lfu, _ = run_caches(z, L, N, 3, C, POLICY_LFU)
    _, c_l0, _ = run_caches(z, L, N, 3, C, POLICY_LRFU, lam=0.0)
    assert all(np.array_equal(a, b) for a, b in zip(c_lfu, c_l0))
    z = tie_logits(rng, 20, L, N)[:, None]
    _, c_lru, _ = run_caches(z, L, N, 1, C, POLICY_LRU)
    _, c_l1, _ = run_caches(z, L, N, 1, C, POLICY_LRFU, lam=1.0)
    assert all(np.array_equal(a, b) for a, b in zip(c_lru, c_l1))


def test_lrfu_values_follow_definition():
    """The fp32 incremental CRF stays within a few ulp of the fp64 sum."""
    rng = np.random.default_rng(3)
    N, K, C, T = 12, 3, 5, 40
    z = tie_logits(rng, T, 1, N)
    sels = selections(z, K)[:, 0]
    run = oracle.Run(1, N, K, C, 0, 1, MODE_TEMPORAL, policy=POLICY_LRFU, lrfu_lambda=0.5)
    for t in range(T):
        run.step(z[t][None, None], None)
        want = np.array([sum(0.5 ** (0.5 * (t - q)) for q in range(t + 1) if e in sels[q]) for e in range(N)])
        got = run.pol[0, 0].astype(np.float64)
        assert np.all(np.abs(got - want) <= 8 * 2.0 ** -24 * np.maximum(want, 1.0)), t


# ------------------------------------------------------------ Spatio-only
def test_spatio_only_without_refinement_is_update_only_lru():
    """R = 0 leaves only demand insertion with LRU eviction."""
    rng = np.random.default_rng(21)
    S, L, N, K, C, T = 3, 3, 16, 3, 6, 25
    zR, _, zS = random_logits(rng, T, S, L, N)
    zR = (np.round(zR * 2) / 2).astype(np.float32)
    a = oracle.Run(L, N, K, C, 0, S, MODE_SPATIO_ONLY, policy=POLICY_LRU)
    b = oracle.Run(L, N, K, C, 0, S, MODE_TEMPORAL, policy=POLICY_LRU)
    for t in range(T):
        oa = a.step(zR[t], None, zS[t], want="all")
        ob = b.step(zR[t], None, None, want="all")
        assert np.array_equal(a.cache, b.cache)
        assert np.array_equal(oa["nD"], ob["nD"]) and not oa["nP"].any()
    assert np.array_equal(a.ctr, b.ctr)


def spatio_only_replay(zR, zS, L, N, K, C, R):
    """Equation-level replay of one stream: s^S_{t,l} = p^R_{t-1,l} +
    p^S_rho(t,l) with rho(t,0) = (t-1, L-1), rho(t,l) = (t, l-1); refinement
    by Algorithm 2 (brute-force form); demand insertion with the recency list;
    a proactively inserted expert enters as the most recently used."""
    T = zR.shape[0]
    pR, pS = {}, {}
    cache = [set() for _ in range(L)]
    order = [[] for _ in range(L)]
    P = D = 0
    hist = []
    for t in range(T):
        for l in range(L):
            if t >= 1 and R > 0:
                pred = pS[(t - 1, L - 1)] if l == 0 else pS[(t, l - 1)]
                sS = (pR[(t - 1, l)] + pred).astype(np.float32)
                new = ref_refine(cache[l], sS, R, C)
                ins = new - cache[l]
                P += len(ins)
                order[l] = [u for u in order[l] if u not in ins] + sorted(ins)
                cache[l] = new
            pR[(t, l)] = oracle.softmax(zR[t, l])
            pS[(t, l)] = oracle.softmax(zS[t, l])
            sel = set(np.lexsort((np.arange(N), -zR[t, l].astype(np.float64)))[:K].tolist())
            for e in sorted(sel - cache[l]):
                D += 1
                if len(cache[l]) < C:
                    cache[l].add(e)
                else:
                    v = next(u for u in order[l] if u in cache[l] and u not in sel)
                    cache[l].discard(v)
                    cache[l].add(e)
            order[l] = [u for u in order[l] if u not in sel] + sorted(sel)
            hist.append(set(cache[l]))
    return hist, D, P


@pytest.mark.parametrize("N,K,C,R", [(12, 2, 4, 2), (16, 3, 5, 4), (10, 2, 6, 10)])
def test_spatio_only_matches_equation_replay(N, K, C, R):
    rng = np.random.default_rng(N + 7 * R)
    L, T = 3, 15
    zR, _, zS = random_logits(rng, T, 1, L, N)
    want, D, P = spatio_only_replay(zR[:, 0], zS[:, 0], L, N, K, C, R)
    run = oracle.Run(L, N, K, C, R, 1, MODE_SPATIO_ONLY, policy=POLICY_LRU)
    got = []
    for t in range(T):
        run.step(zR[t], None, zS[t])
        for l in range(L):
            got.append(set(np.nonzero(run.cache[0, l])[0].tolist()))
    assert got == want
    tot = run.totals()
    assert tot["demand_misses"] == D and tot["proactive_loads"] == P
    assert P > 0
    # one stream: physical fills are exactly the demand and proactive loads
    assert tot["phys_fills"] == D + P


def test_spatio_only_needs_spatio_logits():
    run = oracle.Run(2, 8, 2, 3, 2, 1, MODE_SPATIO_ONLY, policy=POLICY_LRU)
    with pytest.raises(ValueError):
        run.step(np.zeros((1, 2, 8), np.float32), None, None)
