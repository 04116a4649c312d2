"""Helpers shared by the GPU tests (not collected by pytest)."""
from __future__ import annotations

import copy
import sys
import zlib

import numpy as np

import oracle


def stable_seed(text: str) -> int:
    """A seed derived from a test-case name that is the same in every process
    (str hashes are salted per process, so hash() would draw new inputs on
    every run and a failing case could not be replayed from its ID)."""
    return zlib.crc32(text.encode("ascii"))


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def clone_run(run: oracle.Run) -> oracle.Run:
    r = copy.copy(run)
    r.cfg = oracle._Cfg(*[getattr(run.cfg, n) for n, _ in oracle._Cfg._fields_])
    for n in ("cache", "aT", "pS", "ctr", "slot_of", "phys", "pol", "selcount", "stamp", "clk"):
        setattr(r, n, getattr(run, n).copy())
    return r


def compare_step(eng, run: oracle.Run, out: dict, where: str):
    """Bit-exact comparison of every integer output of one token."""
    from paper_2609_04895_amd import cmoe as B
    sel = eng.cmoe_read(B.CMOE_VIEW_SELECTED)             # [L][S][K]
    assert np.array_equal(sel.transpose(1, 0, 2), out["sel"]), f"{where}: selected experts differ"
    gates = eng.cmoe_read(B.CMOE_VIEW_GATES).transpose(1, 0, 2)
    assert np.allclose(gates, out["gate"], rtol=2e-6, atol=1e-7), f"{where}: gates differ"
    cache = eng.cache_sets()
    assert np.array_equal(cache, run.cache.astype(bool)), f"{where}: cache sets differ"
    ev = eng.cmoe_read(B.CMOE_VIEW_EVENTS)                # [L][S][4]
    assert np.array_equal(ev[:, :, 0].T, out["hits"]), f"{where}: hits differ"
    assert np.array_equal(ev[:, :, 1].T, out["nD"]), f"{where}: demand misses differ"
    assert np.array_equal(ev[:, :, 2].T, out["nP"]), f"{where}: proactive loads differ"
    ctr = eng.cmoe_read(B.CMOE_VIEW_COUNTERS)
    assert np.array_equal(ctr, run.ctr), f"{where}: counters differ"
    slots = eng.cmoe_read(B.CMOE_VIEW_SLOTS)
    assert np.array_equal(slots, run.slot_of), f"{where}: slot maps differ"
    fills = eng.cmoe_read(B.CMOE_VIEW_FILLS)
    assert np.array_equal(fills, out["fills"]), f"{where}: physical fills differ"
    assert np.array_equal(eng.cmoe_read(B.CMOE_VIEW_PHYS), run.phys), f"{where}: physical counters differ"
    selcount = eng.cmoe_read(B.CMOE_VIEW_SELCOUNT)
    assert np.array_equal(selcount.astype(np.int64), run.selcount), f"{where}: selection counts differ"
    conc = eng.cmoe_concentration(8)
    assert np.allclose(conc, oracle.concentration(run.selcount, 8), rtol=1e-12, atol=1e-15), f"{where}: concentration"
    if run.policy != oracle.POLICY_ROUTER:
        pol = eng.cmoe_read(B.CMOE_VIEW_PRIORITY)
        assert np.array_equal(pol.view(np.uint32), run.pol.view(np.uint32)), f"{where}: priorities differ"
    # distinct experts selected per layer step, summed over the counted tokens
    # (what bench.py's roofline counts as expert weight reads); compare_step
    # runs after every token, so the sum is complete
    if not hasattr(run, "active_expected"):
        run.active_expected = np.zeros(run.L, np.int64)
    if run.t - 1 >= run.cfg.warmup_tokens:
        for l in range(run.L):
            run.active_expected[l] += np.unique(out["sel"][:, l, :]).size
    active = eng.cmoe_read(B.CMOE_VIEW_ACTIVE)
    assert np.array_equal(active, run.active_expected), f"{where}: distinct experts per layer differ"


def oracle_logits(w, WR, WT, WS, bias, H, t, streams):
    """The oracle's fp32 logits of token t, [len(streams)][L][n_r][N], router
    slots in the library's order (native, temporal if used, spatio if used)."""
    mats = [WR] + ([WT] if w.has_temporal else []) + ([WS] if w.has_spatio else [])
    z = np.empty((len(streams), w.L, len(mats), w.N), np.float32)
    for i, s in enumerate(streams):
        for l in range(w.L):
            h = H[(s, l)][t]
            for r, M in enumerate(mats):
                z[i, l, r] = oracle.logits(M[l], h, bias[l] if (r == 0 and bias is not None) else None)
    return z


def split_slots(w, z):
    """(zR, zT or None, zS or None) from [..][L][n_r][N] router-slot logits."""
    zT = z[:, :, 1] if w.has_temporal else None
    zS = z[:, :, -1] if w.has_spatio else None
    return z[:, :, 0], zT, zS


def host_routers(w):
    import synth
    WR = [synth.router_host(w, synth.KIND_ROUTER_NATIVE, l) for l in range(w.L)]
    WT = [synth.router_host(w, synth.KIND_ROUTER_TEMPORAL, l) for l in range(w.L)] if w.has_temporal else None
    WS = [synth.router_host(w, synth.KIND_ROUTER_SPATIO, l) for l in range(w.L)] if w.has_spatio else None
    return WR, WT, WS


def oracle_run(w, **kw):
    return oracle.Run(w.L, w.N, w.K, w.C, w.R, w.S, w.mode, policy=w.policy, lrfu_lambda=w.lrfu_lambda,
                      arena_slots=w.arena_slots, **kw)


def rel_err(y, ref):
    den = float(np.max(np.abs(ref)))
    return float(np.max(np.abs(np.asarray(y, np.float64) - ref))) / (den if den > 0 else 1.0)
