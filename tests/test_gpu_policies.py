"""Parity of the classical retention policies (LRU, LFU, LRFU; the paper's
cache-update baselines, Section 4.1 / Table 1) and of the Spatio-only mode
(Section 5, Appendix B.4) with the oracle.

- Cache path bit for bit from the same fp32 logits (cmoe_step_logits): the
  selections, caches, events, counters, slot maps, physical fills and the
  priority state itself (LRU time, LFU count, LRFU value).
- End to end (cmoe_step): the native router alone (one router slot) and
  native + Spatio routers, with the FFN.
- Full size in the bench launch configuration.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import compare_step, say
from test_gpu_cache_parity import logits_sequence
from test_gpu_e2e_parity import run_e2e
from test_gpu_full_size import run_full

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

LRU, LFU, LRFU = oracle.POLICY_LRU, oracle.POLICY_LFU, oracle.POLICY_LRFU
TEMPORAL, SPATIO_ONLY = oracle.MODE_TEMPORAL, oracle.MODE_SPATIO_ONLY


def make_engine(L, N, K, C, R, S, mode, policy, lam=0.5, warmup=0, side=True, d=64, F=64):
    from paper_2609_04895_amd import cmoe as B
    dev = torch.device("cuda", 0)
    w = torch.zeros((L, N, d), dtype=torch.float32, device=dev)
    pool = torch.arange(L * N * 3 * d * F, dtype=torch.float32, device=dev).reshape(L, N, 3 * d * F)
    cfg = B.make_config(L, N, K, d, F, C, R, S, mode, B.CMOE_F32, B.CMOE_POOL_DEVICE, warmup,
                        B.CMOE_FLAG_FILL_ON_SIDE if side else 0, policy, lam)
    eng = B.Engine(cfg, w, None, w if mode == SPATIO_ONLY else None, None, pool,
                   side_stream=torch.cuda.Stream() if side else None)
    return eng


CASES = [
    # L, N, K, C, R, S, mode, policy, lambda, warmup, ties, side
    (3, 16, 2, 6, 0, 3, TEMPORAL, LRU, 0.5, 0, True, True),
    (3, 16, 2, 6, 0, 3, TEMPORAL, LFU, 0.5, 0, True, True),
    (3, 16, 2, 6, 0, 3, TEMPORAL, LRFU, 0.5, 0, True, True),
    (2, 16, 3, 5, 0, 4, TEMPORAL, LRFU, 1.0, 0, False, True),   # w = 1/2
    (2, 16, 3, 5, 0, 4, TEMPORAL, LRFU, 0.0, 1, True, True),    # w = 1 (LFU)
    (2, 128, 8, 32, 0, 70, TEMPORAL, LRU, 0.5, 1, True, True),  # Qwen3-like shape
    (2, 128, 8, 32, 0, 9, TEMPORAL, LRFU, 0.5, 0, False, True),
    (3, 100, 7, 20, 5, 37, SPATIO_ONLY, LRU, 0.5, 2, True, True),   # ragged N and S
    (4, 32, 4, 8, 2, 5, SPATIO_ONLY, LRU, 0.5, 0, True, False),     # GPT-OSS-like, fills on main
    (2, 256, 8, 40, 12, 6, SPATIO_ONLY, LFU, 0.5, 0, True, True),   # four experts per lane
    (2, 64, 64, 64, 64, 2, SPATIO_ONLY, LRU, 0.5, 0, True, False),  # K = C = N = R
    (2, 1, 1, 1, 1, 2, SPATIO_ONLY, LRFU, 0.5, 0, False, True),     # a single expert
    (1, 16, 2, 4, 2, 3, SPATIO_ONLY, LRU, 0.5, 0, True, True),      # a single layer
]


def case_id(c):
    return f"L{c[0]}N{c[1]}K{c[2]}C{c[3]}R{c[4]}S{c[5]}m{c[6]}p{c[7]}lam{c[8]}"


@pytest.mark.parametrize("case", CASES, ids=[case_id(c) for c in CASES])
def test_policy_cache_path_bit_exact(case):
    L, N, K, C, R, S, mode, policy, lam, warmup, ties, side = case
    say(f"policy cache parity {case_id(case)}")
    T = 20
    rng = np.random.default_rng(abs(hash(case)) % (2 ** 32))
    z = logits_sequence(rng, T, S, L, N, ties)
    eng = make_engine(L, N, K, C, R, S, mode, policy, lam, warmup, side)
    run = oracle.Run(L, N, K, C, R, S, mode, warmup, policy=policy, lrfu_lambda=lam)
    dev = torch.device("cuda", 0)
    for t in range(T):
        zR = torch.from_numpy(z[t, 0]).to(dev)
        zS = torch.from_numpy(z[t, 2]).to(dev) if mode == SPATIO_ONLY else None
        eng.cmoe_step_logits(zR, None, zS)
        out = run.step(z[t, 0], None, z[t, 2] if mode == SPATIO_ONLY else None, want="all")
        compare_step(eng, run, out, f"case {case_id(case)} token {t}")
    total, per, phys = eng.cmoe_stats()
    ref = run.totals()
    for k in ("accesses", "hits", "demand_misses", "proactive_loads", "tokens", "phys_fills"):
        assert total[k] == ref[k], k
    if mode == TEMPORAL or R == 0:
        assert total["proactive_loads"] == 0
    eng.cmoe_destroy()


def test_spatio_only_budget_change_and_reset():
    L, N, K, C, S = 3, 32, 4, 8, 4
    rng = np.random.default_rng(9)
    z = logits_sequence(rng, 14, S, L, N, ties=True)
    eng = make_engine(L, N, K, C, 2, S, SPATIO_ONLY, LRU)
    run = oracle.Run(L, N, K, C, 2, S, SPATIO_ONLY, policy=LRU)
    dev = torch.device("cuda", 0)
    for t in range(14):
        if t == 4:
            eng.cmoe_set_R(6)
            run.set_R(6)
        if t == 9:
            eng.cmoe_set_R(0)
            run.set_R(0)
        eng.cmoe_step_logits(torch.from_numpy(z[t, 0]).to(dev), None, torch.from_numpy(z[t, 2]).to(dev))
        out = run.step(z[t, 0], None, z[t, 2], want="all")
        compare_step(eng, run, out, f"token {t}")
    eng.cmoe_reset()
    run = oracle.Run(L, N, K, C, 0, S, SPATIO_ONLY, policy=LRU)
    for t in range(3):
        eng.cmoe_step_logits(torch.from_numpy(z[t, 0]).to(dev), None, torch.from_numpy(z[t, 2]).to(dev))
        out = run.step(z[t, 0], None, z[t, 2], want="all")
        compare_step(eng, run, out, f"after reset, token {t}")
    eng.cmoe_destroy()


def test_lru_native_router_only_end_to_end():
    """One router slot: the GEMV, the cache path and the FFN with LRU."""
    w = synth.WORKLOADS["tiny"].replace(name="tiny_lru", policy=synth.POLICY_LRU)
    run_e2e(w, T=64, tol=1e-5)


def test_spatio_only_bf16_end_to_end():
    w = synth.WORKLOADS["qwen3_30b"].replace(name="bf16_spatio_only", L=3, d=256, F=128, S=20, C=24, R=4,
                                             mode=synth.MODE_SPATIO_ONLY, policy=synth.POLICY_LRU)
    run_e2e(w, T=10, tol=2e-2)


def test_lrfu_bf16_end_to_end():
    w = synth.WORKLOADS["qwen3_30b"].replace(name="bf16_lrfu", L=2, d=192, F=192, S=9, C=16,
                                             policy=synth.POLICY_LRFU)
    run_e2e(w, T=8, tol=2e-2)


def test_full_size_qwen3_30b_lru():
    run_full(synth.WORKLOADS["qwen3_30b"].replace(name="qwen3_30b_lru", policy=synth.POLICY_LRU), T=12,
             ffn_samples=4)


def test_full_size_qwen3_30b_zipf_spatio_only():
    w = synth.WORKLOADS["qwen3_30b_zipf"].replace(name="qwen3_30b_zipf_spatio_only", C=32, R=4,
                                                  mode=synth.MODE_SPATIO_ONLY, policy=synth.POLICY_LRU)
    run_full(w, T=8, ffn_samples=4)
