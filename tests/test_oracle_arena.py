"""Pins of the oracle's capacity-limited arena: fewer HBM slots per layer than
the union of the streams' caches can reach (the paper's bounded device cache,
Section 3.1 and the Figure 1 caption, taken literally for many streams).

The arena is a second-level cache over the slots.  When the union of the
caches fits, every member is resident and new ones take the lowest free slot
(the unlimited arena).  When it does not, the experts the layer step executes
pass through the slots in rounds (resident ones first), each missing expert
taking the lowest free slot or evicting the least recently used expert no
remaining round needs (lower slot on equal recency); refinement only fills
free slots.  The pins below do not reuse the oracle's formulation: an ordered
recency list, the stack-distance characterisation of LRU (Mattson et al.
1970), and copy-count bounds that follow from the rules."""
import numpy as np
import pytest

import oracle
from test_oracle_replay import random_logits

TEMPORAL, FULL = 0, 1


def steps(run, zR, zT, zS, T):
    for t in range(T):
        yield t, run.step(zR[t], zT[t], zS[t] if run.mode else None, want="all")


def max_union(L, N, K, C, R, S, mode, zR, zT, zS, T):
    """The largest union of caches over every residency event (after the
    refinement and after the access) of an unlimited arena's run."""
    run = oracle.Run(L, N, K, C, R, S, mode)
    m = 0
    for t in range(T):
        before = run.cache.copy()
        out = run.step(zR[t], zT[t], zS[t] if mode else None, want="all")
        m = max(m, int(run.cache.any(axis=0).sum(axis=-1).max()))
        if mode == FULL and t >= 1 and R > 0:
            for l in range(L):
                m = max(m, len(refined_union(before[:, l], out, run, l)))
    return m


@pytest.mark.parametrize("mode", [TEMPORAL, FULL])
def test_an_arena_that_holds_every_union_is_the_unlimited_arena(mode):
    """With at least as many slots as the largest union of caches, the arena
    never overflows: slot maps and copies equal those of min(N, S C) slots."""
    rng = np.random.default_rng(31)
    L, N, K, C, R, S, T = 3, 32, 3, 6, 2, 5, 40
    zR, zT, zS = random_logits(rng, T, S, L, N)
    P = max_union(L, N, K, C, R, S, mode, zR, zT, zS, T)
    assert P < min(N, S * C)
    a = oracle.Run(L, N, K, C, R, S, mode)
    b = oracle.Run(L, N, K, C, R, S, mode, arena_slots=P)
    for t in range(T):
        oa = a.step(zR[t], zT[t], zS[t] if mode else None, want="all")
        ob = b.step(zR[t], zT[t], zS[t] if mode else None, want="all")
        assert np.array_equal(a.slot_of, b.slot_of), t
        assert np.array_equal(oa["fills"], ob["fills"]), t
    assert np.array_equal(a.ctr, b.ctr)


def lru_misses(seq, P):
    """Misses of an LRU cache of P entries on a reference string, from stack
    distances: a reference hits iff fewer than P distinct other items were
    referenced since its previous reference."""
    misses = 0
    for i, x in enumerate(seq):
        prev = [j for j in range(i) if seq[j] == x]
        if not prev or len(set(seq[prev[-1] + 1:i])) >= P:
            misses += 1
    return misses


@pytest.mark.parametrize("P", [1, 2, 3, 5])
def test_one_stream_one_expert_per_step_is_textbook_lru(P):
    """One stream, Top-1, a logical cache that keeps everything (C = N): the
    union only grows, each layer step executes one expert, and the arena of P
    slots is an LRU cache over the layer's sequence of selected experts, so
    its copies are the LRU misses of that sequence."""
    rng = np.random.default_rng(40 + P)
    L, N, T = 2, 12, 80
    zR, zT, _ = random_logits(rng, T, 1, L, N, rho=0.5)
    run = oracle.Run(L, N, 1, N, 0, 1, TEMPORAL, arena_slots=P)
    seqs = [[] for _ in range(L)]
    for t in range(T):
        out = run.step(zR[t], zT[t], want="all")
        for l in range(L):
            seqs[l].append(int(out["sel"][0, l, 0]))
    for l in range(L):
        assert run.phys[l, 0] == lru_misses(seqs[l], P), l
    assert run.phys[:, 1].sum() == 0


class RecencyListArena:
    """The arena of one layer as a set of slots plus a list of resident
    experts ordered from least to most recently used (experts used in the
    same round are appended in slot order, so the first of equally recent
    ones holds the lowest slot)."""

    def __init__(self, P):
        self.P = P
        self.slot = {}
        self.lru = []

    def _touch(self, experts):
        for e in sorted(experts, key=lambda e: self.slot[e]):
            if e in self.lru:
                self.lru.remove(e)
            self.lru.append(e)

    def _drop(self, e):
        del self.slot[e]
        self.lru.remove(e)

    def _free(self):
        taken = set(self.slot.values())
        return [q for q in range(self.P) if q not in taken]

    def event(self, union, executed):
        """Returns the number of copies."""
        for e in [e for e in self.slot if e not in union]:
            self._drop(e)
        copies = 0
        if len(union) <= self.P or executed is None:
            new = sorted(union - set(self.slot))
            touched = []
            for e in new:
                free = self._free()
                if not free:
                    break
                self.slot[e] = free[0]
                touched.append(e)
                copies += 1
            if executed is not None:
                touched += sorted(executed)
            self._touch(set(touched))
            return copies
        order = sorted(e for e in executed if e in self.slot) + sorted(e for e in executed if e not in self.slot)
        rounds = [order[i:i + self.P] for i in range(0, len(order), self.P)]
        for r, group in enumerate(rounds):
            later = set(x for g in rounds[r:] for x in g)
            for e in group:
                if e in self.slot:
                    continue
                free = self._free()
                if free:
                    q = free[0]
                else:
                    victim = next(v for v in self.lru if v not in later)
                    q = self.slot[victim]
                    self._drop(victim)
                self.slot[e] = q
                copies += 1
            self._touch(set(group))
        return copies


@pytest.mark.parametrize("mode,P,K,C,S", [(TEMPORAL, 4, 2, 4, 3), (TEMPORAL, 3, 3, 5, 4), (FULL, 5, 2, 4, 4),
                                          (FULL, 2, 3, 4, 3), (TEMPORAL, 1, 2, 3, 2), (FULL, 6, 4, 8, 5)])
def test_oracle_arena_matches_a_recency_list_model(mode, P, K, C, S):
    """Tie-heavy random traces (logits on a 1/2 grid), several tokens, every
    residency event of both kinds: the oracle's slot maps and copy counts
    equal those of the recency-list model."""
    rng = np.random.default_rng(100 * P + K + S)
    L, N, R, T = 2, 10, 2, 40
    zR, zT, zS = [np.round(z * 2) / 2 for z in random_logits(rng, T, S, L, N, rho=0.6)]
    run = oracle.Run(L, N, K, C, R, S, mode, arena_slots=P)
    model = [RecencyListArena(P) for _ in range(L)]
    overflow = {0: 0, 1: 0}   # events whose union does not fit, by kind
    for t in range(T):
        caches_before = run.cache.copy()
        out = run.step(zR[t], zT[t], zS[t] if mode else None, want="all")
        for l in range(L):
            union_after = set(np.nonzero(run.cache[:, l].any(axis=0))[0].tolist())
            executed = set(out["sel"][:, l].ravel().tolist())
            if mode == FULL and t >= 1 and R > 0:
                pre = refined_union(caches_before[:, l], out, run, l)
                overflow[1] += len(pre) > P
                assert model[l].event(pre, None) == out["fills"][l, 1], (t, l)
            overflow[0] += len(union_after) > P
            assert model[l].event(union_after, executed) == out["fills"][l, 0], (t, l)
            want = np.full(N, -1, np.int32)
            for e, q in model[l].slot.items():
                want[e] = q
            assert np.array_equal(run.slot_of[l], want), (t, l)
    assert overflow[0] > 0 and (mode == TEMPORAL or overflow[1] > 0), overflow


def refined_union(before, out, run, l):
    """Union over the streams of layer l's refined caches at this token: a
    layer's cache changes only at its own refinement and access, so its
    refined cache is the refinement rule (pinned on its own) applied to its
    cache after the previous token, with this token's s^ST."""
    caches = []
    for s in range(before.shape[0]):
        c1, _ = oracle.refine(before[s].astype(np.uint8), out["sST"][s, l], run.R, run.C)
        caches.append(c1.astype(bool))
    return set(np.nonzero(np.any(caches, axis=0))[0].tolist())


@pytest.mark.parametrize("P", [2, 5, 9])
def test_overflowing_layer_steps_copy_each_missing_expert_once(P):
    """Update-only, many streams, few slots: in a layer step whose union does
    not fit, exactly the executed experts that were not resident (after the
    experts outside the union left) are copied, each once; the arena never
    holds more than P experts, only members of the union, injectively."""
    rng = np.random.default_rng(60 + P)
    L, N, K, C, S, T = 2, 24, 3, 6, 6, 30
    zR, zT, _ = random_logits(rng, T, S, L, N)
    run = oracle.Run(L, N, K, C, 0, S, TEMPORAL, arena_slots=P)
    overflows = 0
    for t in range(T):
        before = run.slot_of.copy()
        out = run.step(zR[t], zT[t], want="all")
        for l in range(L):
            union = set(np.nonzero(run.cache[:, l].any(axis=0))[0].tolist())
            executed = set(out["sel"][:, l].ravel().tolist())
            resident = set(np.nonzero(before[l] >= 0)[0].tolist()) & union
            slots = run.slot_of[l]
            held = set(np.nonzero(slots >= 0)[0].tolist())
            assert held <= union and len(held) <= P
            assert len(set(slots[slots >= 0].tolist())) == len(held) and slots.max(initial=-1) < P
            if len(union) > P:
                overflows += 1
                assert out["fills"][l, 0] == len(executed - resident), (t, l)
            else:
                assert held == union
    assert overflows > 0
