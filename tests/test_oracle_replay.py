"""Pins of the oracle's whole decode replay (all layers, all tokens).

The reference replay here is written from the paper's equations, not from the
oracle's code: the causal predecessor rho(t, l) and the pre-access priority
a^T + p^S_rho are evaluated from stored per-(t, l) distributions exactly as
Section 3.3 writes them, and the two cache rules are replaced by their closed
forms / brute-force characterisations (pinned in test_oracle_cache.py).  The
special cases below are consequences the paper states or implies.
"""
import itertools

import numpy as np
import pytest

import oracle

TEMPORAL, FULL = 0, 1


def random_logits(rng, T, S, L, N, scale=2.0, rho=0.8):
    """AR(1)-correlated logits [T][S][L][N] per router, for temporal locality."""
    out = []
    for _ in range(3):
        z = np.empty((T, S, L, N), np.float32)
        prev = rng.normal(size=(S, L, N))
        for t in range(T):
            prev = rho * prev + np.sqrt(1 - rho * rho) * rng.normal(size=(S, L, N))
            z[t] = (prev * scale).astype(np.float32)
        out.append(z)
    return out


def ref_update(C, S, s, cap):
    U = C | S
    if len(U) <= cap:
        return U
    rest = sorted(C - S, key=lambda u: (s[u], u))
    return S | set(rest[len(U) - cap:])


def ref_refine(C, s, R, cap):
    A = sorted(range(len(s)), key=lambda e: (-s[e], e))[:R]
    nonres = [e for e in A if e not in C]
    m = cap - len(C)
    if len(nonres) <= m:
        return C | set(nonres)
    forced = set(nonres[:m])
    pool = sorted(C | set(nonres[m:]))
    best, best_val = None, None
    for Y in itertools.combinations(pool, len(C)):
        val = sum(float(s[u]) for u in Y)
        if best_val is None or val > best_val:
            best, best_val = set(Y), val
    return forced | best


def reference_replay(zR, zT, zS, L, N, K, C, R, mode, warmup=0):
    """Returns per-step caches and counters for one stream."""
    T = zR.shape[0]
    pR, pT, pS = {}, {}, {}
    cache = [set() for _ in range(L)]
    ctr = np.zeros((L, 5), np.int64)
    caches = []
    for t in range(T):
        for l in range(L):
            if mode == FULL and t >= 1 and R > 0:
                pred = pS[(t - 1, L - 1)] if l == 0 else pS[(t, l - 1)]       # rho(t, l)
                aT = (pR[(t - 1, l)] + pT[(t - 1, l)]).astype(np.float32)      # a^T_{t,l}
                sST = (aT + pred).astype(np.float32)                            # s^ST_{t,l}
                new = ref_refine(cache[l], sST, R, C)
                if t >= warmup:
                    ctr[l, 3] += len(new - cache[l])
                cache[l] = new
            pR[(t, l)] = oracle.softmax(zR[t, l])
            pT[(t, l)] = oracle.softmax(zT[t, l])
            if mode == FULL:
                pS[(t, l)] = oracle.softmax(zS[t, l])
            sel = set(np.lexsort((np.arange(N), -zR[t, l].astype(np.float64)))[:K].tolist())
            sT = (pR[(t, l)] + pT[(t, l)]).astype(np.float32)
            hits = len(sel & cache[l])
            if t >= warmup:
                ctr[l] += [K, hits, K - hits, 0, 1]
            cache[l] = ref_update(cache[l], sel, sT, C)
        caches.append([set(c) for c in cache])
    return caches, ctr


def run_oracle(zR, zT, zS, L, N, K, C, R, mode, S=1, warmup=0):
    run = oracle.Run(L, N, K, C, R, S, mode, warmup)
    caches = []
    outs = []
    for t in range(zR.shape[0]):
        outs.append(run.step(zR[t], zT[t], zS[t] if mode == FULL else None, want="all"))
        caches.append(run.cache.copy())
    return run, caches, outs


@pytest.mark.parametrize("mode,R", [(TEMPORAL, 0), (FULL, 1), (FULL, 2), (FULL, 5)])
def test_oracle_matches_equation_level_replay(mode, R):
    rng = np.random.default_rng(100 + 10 * mode + R)
    L, N, K, C, T = 3, 7, 2, 4, 40
    zR, zT, zS = random_logits(rng, T, 1, L, N)
    for warmup in (0, 5):
        run, caches, _ = run_oracle(zR, zT, zS, L, N, K, C, R, mode, warmup=warmup)
        ref_caches, ref_ctr = reference_replay(zR[:, 0], zT[:, 0], zS[:, 0], L, N, K, C, R, mode, warmup)
        for t in range(T):
            for l in range(L):
                assert set(np.nonzero(caches[t][0, l])[0].tolist()) == ref_caches[t][l], (t, l)
        assert np.array_equal(run.ctr[0], ref_ctr)


def test_update_only_issues_no_proactive_loads():
    rng = np.random.default_rng(1)
    L, N, K, C, T, S = 4, 16, 2, 6, 60, 3
    zR, zT, zS = random_logits(rng, T, S, L, N)
    run, _, outs = run_oracle(zR, zT, zS, L, N, K, C, 0, TEMPORAL, S=S)
    tot = run.totals()
    assert tot["proactive_loads"] == 0
    assert run.phys[:, 1].sum() == 0
    assert tot["accesses"] == T * S * L * K
    assert tot["hits"] + tot["demand_misses"] == tot["accesses"]
    h, adj, _ = oracle.metrics(tot["accesses"], tot["demand_misses"], 0, tot["tokens"], 1.0)
    assert h == pytest.approx(adj, abs=1e-15)


def test_full_mode_with_zero_budget_equals_update_only():
    rng = np.random.default_rng(2)
    L, N, K, C, T, S = 4, 16, 2, 6, 50, 2
    zR, zT, zS = random_logits(rng, T, S, L, N)
    a, ca, _ = run_oracle(zR, zT, zS, L, N, K, C, 0, TEMPORAL, S=S)
    b, cb, _ = run_oracle(zR, zT, zS, L, N, K, C, 0, FULL, S=S)
    assert all(np.array_equal(x, y) for x, y in zip(ca, cb))
    assert np.array_equal(a.ctr, b.ctr) and np.array_equal(a.phys, b.phys)


def test_capacity_equal_k_retains_exactly_the_last_selection():
    rng = np.random.default_rng(3)
    L, N, K, T = 3, 16, 3, 40
    zR, zT, zS = random_logits(rng, T, 1, L, N)
    run = oracle.Run(L, N, K, K, 0, 1, TEMPORAL)
    prev = None
    for t in range(T):
        o = run.step(zR[t], zT[t], want="all")
        sel = [set(o["sel"][0, l].tolist()) for l in range(L)]
        for l in range(L):
            assert set(np.nonzero(run.cache[0, l])[0].tolist()) == sel[l]
            if prev is not None:
                assert o["hits"][0, l] == len(prev[l] & sel[l])
        prev = sel


def test_capacity_n_only_compulsory_misses():
    rng = np.random.default_rng(4)
    L, N, K, T = 3, 16, 2, 80
    zR, zT, zS = random_logits(rng, T, 1, L, N)
    run = oracle.Run(L, N, K, N, 0, 1, TEMPORAL)
    seen = [set() for _ in range(L)]
    for t in range(T):
        o = run.step(zR[t], zT[t], want="all")
        for l in range(L):
            sel = set(o["sel"][0, l].tolist())
            assert o["nD"][0, l] == len(sel - seen[l])
            seen[l] |= sel


def test_temporal_router_equal_to_native_doubles_the_score():
    rng = np.random.default_rng(5)
    L, N, K, C, T = 2, 32, 4, 8, 10
    zR, _, _ = random_logits(rng, T, 1, L, N)
    run = oracle.Run(L, N, K, C, 0, 1, TEMPORAL)
    for t in range(T):
        o = run.step(zR[t], zR[t], want="all")
        assert np.array_equal(o["sT"], (2 * o["pR"]).astype(np.float32))


def test_single_stream_physical_fills_equal_logical_transfers():
    rng = np.random.default_rng(6)
    for mode, R in ((TEMPORAL, 0), (FULL, 2), (FULL, 6)):
        L, N, K, C, T = 4, 16, 2, 6, 60
        zR, zT, zS = random_logits(rng, T, 1, L, N)
        run, _, _ = run_oracle(zR, zT, zS, L, N, K, C, R, mode)
        tot = run.totals()
        assert tot["phys_fills"] == tot["demand_misses"] + tot["proactive_loads"]


def test_physical_residency_is_the_union_and_fills_are_bounded():
    rng = np.random.default_rng(7)
    L, N, K, C, R, T, S = 3, 16, 2, 4, 3, 40, 5
    zR, zT, zS = random_logits(rng, T, S, L, N)
    run = oracle.Run(L, N, K, C, R, S, FULL)
    for t in range(T):
        run.step(zR[t], zT[t], zS[t])
        for l in range(L):
            union = set(np.nonzero(run.cache[:, l].any(axis=0))[0].tolist())
            slots = run.slot_of[l]
            assert set(np.nonzero(slots >= 0)[0].tolist()) == union
            used = slots[slots >= 0]
            assert len(set(used.tolist())) == len(used)              # injective
            assert used.max(initial=-1) < min(N, S * C)
    tot = run.totals()
    assert tot["phys_fills"] <= tot["demand_misses"] + tot["proactive_loads"]


def test_slot_assignment_follows_the_lowest_free_slot_rule():
    """Update-only mode has one residency event per (token, layer), so the
    slot maps can be re-derived from the cache trajectory alone: a resident
    expert keeps its slot, experts that left every cache free theirs, and each
    newly needed expert, in ascending order, takes the lowest free slot."""
    rng = np.random.default_rng(17)
    L, N, K, C, T, S = 3, 16, 3, 4, 30, 3
    zR, zT, _ = random_logits(rng, T, S, L, N)
    run = oracle.Run(L, N, K, C, 0, S, TEMPORAL)
    n_slots = min(N, S * C)
    slot = [dict() for _ in range(L)]
    fills = 0
    for t in range(T):
        out = run.step(zR[t], zT[t], want="all")
        for l in range(L):
            union = set(np.nonzero(run.cache[:, l].any(axis=0))[0].tolist())
            for e in [e for e in slot[l] if e not in union]:
                del slot[l][e]
            new = sorted(union - set(slot[l]))
            free = sorted(set(range(n_slots)) - set(slot[l].values()))
            for e, q in zip(new, free):
                slot[l][e] = q
            assert len(new) <= len(free)
            assert out["fills"][l, 0] == len(new)
            fills += len(new)
            want = np.full(N, -1, np.int32)
            for e, q in slot[l].items():
                want[e] = q
            assert np.array_equal(run.slot_of[l], want), (t, l)
    assert run.totals()["phys_fills"] == fills


def test_refinement_loads_at_most_r_per_layer_step_and_starts_at_second_token():
    rng = np.random.default_rng(8)
    L, N, K, C, R, T, S = 4, 16, 2, 6, 3, 30, 2
    zR, zT, zS = random_logits(rng, T, S, L, N)
    run = oracle.Run(L, N, K, C, R, S, FULL)
    for t in range(T):
        o = run.step(zR[t], zT[t], zS[t], want="all")
        assert np.all(o["nP"] <= R)
        if t == 0:
            assert np.all(o["nP"] == 0)


def test_warmup_tokens_are_not_counted():
    rng = np.random.default_rng(9)
    L, N, K, C, R, T, S = 2, 16, 2, 6, 2, 20, 2
    zR, zT, zS = random_logits(rng, T, S, L, N)
    a, ca, _ = run_oracle(zR, zT, zS, L, N, K, C, R, FULL, S=S, warmup=0)
    b, cb, _ = run_oracle(zR, zT, zS, L, N, K, C, R, FULL, S=S, warmup=7)
    assert all(np.array_equal(x, y) for x, y in zip(ca, cb))      # same decisions
    assert b.totals()["tokens"] == S * (T - 7)
    assert b.totals()["accesses"] == S * L * K * (T - 7)
    assert b.totals()["demand_misses"] <= a.totals()["demand_misses"]
