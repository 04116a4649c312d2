"""Pins of the oracle's cache rules (Algorithm 1 and the refinement loop of
Algorithm 2) against closed forms and brute-force enumeration.

Algorithm 1 inserts each demand-loaded expert and, when the cache is full,
evicts the lowest-priority resident that is not selected now.  Closed form:
if |C u S| <= cap the result is C u S; otherwise it is S plus the
cap - |S| highest-priority members of C \\ S (equal priorities: the lower
index is evicted first).  Brute force: among all sets X with S <= X <= C u S
and |X| = min(cap, |C u S|), the result maximises the retained priority.

The refinement loop examines Top_R(s^ST) in descending order; a non-resident
candidate fills free room, else replaces the lowest resident if strictly
higher.  With distinct scores its result is: the first m = cap - |C|
non-resident candidates, plus the |C| best of C and the remaining candidates
(brute force over subsets).
"""
import itertools

import numpy as np
import pytest

import oracle


def subsets(items, k):
    return [set(c) for c in itertools.combinations(sorted(items), k)]


def mask(n, members):
    m = np.zeros(n, np.uint8)
    for e in members:
        m[e] = 1
    return m


def members(m):
    return set(int(e) for e in np.nonzero(m)[0])


# ------------------------------------------------------------ Algorithm 1
def closed_form_update(C, S, s, cap):
    U = C | S
    if len(U) <= cap:
        return U
    rest = sorted(C - S, key=lambda u: (s[u], u))    # eviction order
    return S | set(rest[len(U) - cap:])


def brute_force_update(C, S, s, cap):
    U = C | S
    size = min(cap, len(U))
    best, best_val = None, None
    for X in subsets(C - S, size - len(S)):
        val = sum(float(s[u]) for u in X)
        if best_val is None or val > best_val:
            best, best_val = X, val
    return S | best


@pytest.mark.parametrize("N", [4, 5, 6])
def test_update_cache_closed_form_exhaustive(N):
    rng = np.random.default_rng(N)
    score_sets = [rng.integers(0, 3, N).astype(np.float32) for _ in range(6)]   # heavy ties
    score_sets += [rng.random(N).astype(np.float32) for _ in range(4)]
    n_cases = 0
    for cap in range(1, N + 1):
        for K in range(1, cap + 1):
            for csize in range(0, cap + 1):
                for C in subsets(range(N), csize):
                    for S in subsets(range(N), K):
                        for s in score_sets:
                            Sl = sorted(S)
                            new, dem = oracle.update_cache(mask(N, C), Sl, s, cap)
                            got = members(new)
                            assert got == closed_form_update(C, S, s, cap)
                            # invariants: selected experts are resident, size
                            # is min(cap, |C u S|), only demanded experts enter
                            assert S <= got
                            assert len(got) == min(cap, len(C | S))
                            assert got - C <= set(dem.tolist())
                            assert list(dem) == sorted(S - C)
                            n_cases += 1
    assert n_cases > 1000


def test_update_cache_brute_force_optimal_retention():
    rng = np.random.default_rng(11)
    N = 7
    for _ in range(3000):
        cap = int(rng.integers(1, N + 1))
        K = int(rng.integers(1, cap + 1))
        C = set(rng.choice(N, size=int(rng.integers(0, cap + 1)), replace=False).tolist())
        S = set(rng.choice(N, size=K, replace=False).tolist())
        s = rng.random(N).astype(np.float32)           # distinct priorities
        got = members(oracle.update_cache(mask(N, C), sorted(S), s, cap)[0])
        assert got == brute_force_update(C, S, s, cap)


def test_update_cache_order_of_selected_list_is_irrelevant():
    rng = np.random.default_rng(12)
    N = 16
    for _ in range(500):
        cap, K = 6, 3
        C = set(rng.choice(N, size=cap, replace=False).tolist())
        S = rng.choice(N, size=K, replace=False)
        s = rng.integers(0, 4, N).astype(np.float32)
        a = oracle.update_cache(mask(N, C), S, s, cap)[0]
        b = oracle.update_cache(mask(N, C), S[::-1].copy(), s, cap)[0]
        assert np.array_equal(a, b)


def test_update_cache_capacity_equal_k_keeps_exactly_the_selection():
    rng = np.random.default_rng(13)
    N, K = 12, 4
    for _ in range(300):
        C = set(rng.choice(N, size=K, replace=False).tolist())
        S = set(rng.choice(N, size=K, replace=False).tolist())
        s = rng.random(N).astype(np.float32)
        assert members(oracle.update_cache(mask(N, C), sorted(S), s, K)[0]) == S


# ------------------------------------------------------------ refinement
def closed_form_refine(C, s, R, cap):
    """Distinct scores only."""
    A = sorted(range(len(s)), key=lambda e: -s[e])[:R]
    nonres = [e for e in A if e not in C]
    m = cap - len(C)
    if len(nonres) <= m:
        return C | set(nonres)
    forced = set(nonres[:m])
    pool = C | set(nonres[m:])
    best, best_val = None, None
    for Y in subsets(pool, len(C)):
        val = sum(float(s[u]) for u in Y)
        if best_val is None or val > best_val:
            best, best_val = Y, val
    return forced | best


def test_refine_brute_force_distinct_scores():
    rng = np.random.default_rng(21)
    for N in (5, 6, 7, 8):
        for _ in range(1500):
            cap = int(rng.integers(1, N + 1))
            C = set(rng.choice(N, size=int(rng.integers(0, cap + 1)), replace=False).tolist())
            R = int(rng.integers(0, N + 1))
            s = rng.random(N).astype(np.float32)
            new, loaded = oracle.refine(mask(N, C), s, R, cap)
            got = members(new)
            assert got == closed_form_refine(C, s, R, cap)
            # every insertion is one proactive load and none is undone
            assert set(loaded.tolist()) == got - C and len(loaded) == len(got - C)


def test_refine_invariants_with_ties():
    rng = np.random.default_rng(22)
    N = 8
    for _ in range(5000):
        cap = int(rng.integers(1, N + 1))
        C = set(rng.choice(N, size=int(rng.integers(0, cap + 1)), replace=False).tolist())
        R = int(rng.integers(0, N + 1))
        s = rng.integers(0, 4, N).astype(np.float32)
        new, loaded = oracle.refine(mask(N, C), s, R, cap)
        got = members(new)
        A = [int(e) for e in np.lexsort((np.arange(N), -s))[:R]]
        assert len(loaded) <= R                         # at most R proactive loads
        assert set(loaded.tolist()) <= set(A)           # only candidates enter
        assert got - C == set(loaded.tolist())
        assert len(got) <= cap
        assert len(got) == min(cap, len(C | set(A))) or len(got) == cap
        if got:
            floor = min(float(s[u]) for u in got)
            evicted = C - got
            rejected = set(A) - got
            # nothing dropped or rejected outranks what is kept
            assert all(float(s[v]) <= floor for v in evicted | rejected)
            # an eviction needs a strictly better replacement: incumbents win ties
            for v in evicted:
                assert all(float(s[e]) > float(s[v]) for e in loaded)


def test_refine_budget_zero_is_a_no_op():
    s = np.arange(6, dtype=np.float32)
    new, loaded = oracle.refine(mask(6, {0, 1}), s, 0, 3)
    assert members(new) == {0, 1} and len(loaded) == 0


# ------------------------------------------------------------ stepwise readings
def stepwise_update(C, S, s, cap):
    """Algorithm 1 read step by step: each demand-loaded expert (ascending) is
    inserted; when the cache is full the lowest-priority resident outside S
    leaves first (lower index on ties)."""
    C = set(C)
    for e in sorted(set(S) - C):
        if len(C) >= cap:
            v = min(C - set(S), key=lambda u: (s[u], u))
            C.remove(v)
        C.add(e)
    return C


def stepwise_refine(C, s, R, cap):
    """The refinement loop read step by step: candidates Top_R(s) from the
    highest score (lower index first on ties); a non-resident one enters while
    there is room, else replaces the weakest resident (lower index on ties)
    only if strictly higher.  Returns (cache, loaded in order)."""
    C = set(C)
    loaded = []
    for e in sorted(range(len(s)), key=lambda u: (-s[u], u))[:R]:
        if e in C:
            continue
        if len(C) < cap:
            C.add(e)
            loaded.append(e)
        else:
            v = min(C, key=lambda u: (s[u], u))
            if s[e] > s[v]:
                C.remove(v)
                C.add(e)
                loaded.append(e)
    return C, loaded


@pytest.mark.parametrize("N", [4, 5, 6])
def test_update_cache_equals_the_stepwise_reading_with_ties(N):
    rng = np.random.default_rng(100 + N)
    score_sets = [rng.integers(0, 3, N).astype(np.float32) for _ in range(8)]
    for cap in range(1, N + 1):
        for K in range(1, cap + 1):
            for csize in range(0, cap + 1):
                for C in subsets(range(N), csize):
                    for S in subsets(range(N), K):
                        for s in score_sets:
                            got = members(oracle.update_cache(mask(N, C), sorted(S), s, cap)[0])
                            assert got == stepwise_update(C, S, s, cap)


@pytest.mark.parametrize("N", [4, 5, 6, 7])
def test_refine_equals_the_stepwise_reading_with_ties(N):
    rng = np.random.default_rng(200 + N)
    score_sets = [rng.integers(0, 3, N).astype(np.float32) for _ in range(6)]
    score_sets += [rng.random(N).astype(np.float32) for _ in range(2)]
    n = 0
    for cap in range(1, N + 1):
        for csize in range(0, cap + 1):
            for C in subsets(range(N), csize):
                for R in range(0, N + 1):
                    for s in score_sets:
                        new, loaded = oracle.refine(mask(N, C), s, R, cap)
                        want, want_loaded = stepwise_refine(C, s, R, cap)
                        assert members(new) == want
                        assert loaded.tolist() == want_loaded
                        n += 1
    assert n > 1000
