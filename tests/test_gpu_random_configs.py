"""Bit-exact parity of the cache path with the oracle over a seeded sweep of
random valid configurations: every mode and retention policy, ragged expert
and stream counts (1 to 256 experts, 1 to 90 streams), Top-K from 1 to 16,
any capacity from K to N, any refinement budget, warm-up tokens, tie-heavy
logits, and fills on the side or main stream.  Each case runs a few tokens
through cmoe_step_logits and compares every selection, cache, event,
counter and slot map with the oracle's.  A second sweep runs small random
shapes end to end (router, cache path, fills and expert FFN)."""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import compare_step, say, stable_seed
from test_gpu_cache_parity import logits_sequence

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

N_CHOICES = (1, 2, 3, 5, 8, 16, 17, 31, 32, 33, 63, 64, 65, 100, 127, 128, 129, 200, 255, 256)
POLICIES = (oracle.POLICY_ROUTER, oracle.POLICY_LRU, oracle.POLICY_LFU, oracle.POLICY_LRFU)


def random_cases(n, seed):
    rng = np.random.default_rng(seed)
    cases = []
    for _ in range(n):
        N = int(rng.choice(N_CHOICES))
        K = int(rng.integers(1, min(N, 16) + 1))
        C = int(rng.integers(K, N + 1))
        mode = int(rng.integers(0, 3))
        if mode == oracle.MODE_SPATIO_TEMPORAL:
            policy = oracle.POLICY_ROUTER
        elif mode == oracle.MODE_SPATIO_ONLY:
            policy = int(rng.choice(POLICIES[1:]))
        else:
            policy = int(rng.choice(POLICIES))
        R = int(rng.integers(0, N + 1)) if mode != oracle.MODE_TEMPORAL else 0
        cases.append(dict(L=int(rng.integers(1, 5)), N=N, K=K, C=C, R=R, S=int(rng.integers(1, 91)), mode=mode,
                          policy=policy, lam=float(rng.choice([0.0, 0.25, 0.5, 1.0, 2.0])),
                          warmup=int(rng.integers(0, 3)), ties=bool(rng.integers(0, 2)),
                          side=bool(rng.integers(0, 2))))
    return cases


CASES = random_cases(100, seed=2609)


def case_id(c):
    return "L{L}N{N}K{K}C{C}R{R}S{S}m{mode}p{policy}".format(**c)


@pytest.mark.parametrize("case", CASES, ids=[case_id(c) for c in CASES])
def test_random_config_cache_path_bit_exact(case):
    from paper_2609_04895_amd import cmoe as B
    c = case
    L, N, K, C, R, S, mode, policy = c["L"], c["N"], c["K"], c["C"], c["R"], c["S"], c["mode"], c["policy"]
    seed = stable_seed(case_id(c))
    say(f"random config {case_id(c)} seed={seed} lam={c['lam']} warmup={c['warmup']} ties={c['ties']} "
        f"side={c['side']}")
    T = 8
    rng = np.random.default_rng(seed)
    z = logits_sequence(rng, T, S, L, N, c["ties"])
    dev = torch.device("cuda", 0)
    d = F = 64
    w = torch.zeros((L, N, d), dtype=torch.float32, device=dev)
    pool = torch.arange(L * N * 3 * d * F, dtype=torch.float32, device=dev).reshape(L, N, 3 * d * F)
    cfg = B.make_config(L, N, K, d, F, C, R, S, mode, B.CMOE_F32, B.CMOE_POOL_DEVICE, c["warmup"],
                        B.CMOE_FLAG_FILL_ON_SIDE if c["side"] else 0, policy, c["lam"])
    has_t = policy == oracle.POLICY_ROUTER
    has_s = mode != oracle.MODE_TEMPORAL
    eng = B.Engine(cfg, w, w if has_t else None, w if has_s else None, None, pool,
                   side_stream=torch.cuda.Stream() if c["side"] else None)
    run = oracle.Run(L, N, K, C, R, S, mode, c["warmup"], policy=policy, lrfu_lambda=c["lam"])
    for t in range(T):
        zR = torch.from_numpy(z[t, 0]).to(dev)
        zT = torch.from_numpy(z[t, 1]).to(dev) if has_t else None
        zS = torch.from_numpy(z[t, 2]).to(dev) if has_s else None
        eng.cmoe_step_logits(zR, zT, zS)
        out = run.step(z[t, 0], z[t, 1] if has_t else None, z[t, 2] if has_s else None, want="all")
        compare_step(eng, run, out, f"{case_id(c)} token {t}")
    total, _, _ = eng.cmoe_stats()
    ref = run.totals()
    for k in ("accesses", "hits", "demand_misses", "proactive_loads", "tokens", "phys_fills"):
        assert total[k] == ref[k], k
    eng.cmoe_destroy()


def random_e2e_cases(n, seed):
    """Small random end-to-end shapes: d and F any multiple of 64 up to 384,
    bf16 or fp32, both bf16 FFN launch shapes, with and without Zipf bias."""
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        N = int(rng.choice((2, 8, 16, 24, 33, 64, 100, 128)))
        K = int(rng.integers(1, min(N, 10) + 1))
        mode = int(rng.integers(0, 3))
        if mode == synth.MODE_SPATIO_TEMPORAL:
            policy = synth.POLICY_ROUTER
        elif mode == synth.MODE_SPATIO_ONLY:
            policy = int(rng.integers(1, 4))
        else:
            policy = int(rng.integers(0, 4))
        cases.append(dict(name=f"rand_e2e_{i}", L=int(rng.integers(1, 4)), N=N, K=K,
                          C=int(rng.integers(K, N + 1)), R=int(rng.integers(0, N + 1)) if mode else 0,
                          S=int(rng.integers(1, 100)), d=64 * int(rng.integers(1, 7)), F=64 * int(rng.integers(1, 7)),
                          mode=mode, policy=policy, dtype=int(rng.integers(0, 2)),
                          zipf=float(rng.choice([0.0, 1.1])), shape=str(rng.choice(["single", "grouped"]))))
    return cases


E2E_CASES = random_e2e_cases(30, seed=4895)


@pytest.mark.parametrize("case", E2E_CASES, ids=[c["name"] for c in E2E_CASES])
def test_random_config_end_to_end(case):
    from test_gpu_e2e_parity import run_e2e
    c = dict(case)
    shape, zipf = c.pop("shape"), c.pop("zipf")
    w = synth.WORKLOADS["qwen3_30b"].replace(zipf=zipf or None, **c)
    say(f"random e2e {c} zipf={zipf} shape={shape}")
    run_e2e(w, T=4, tol=2e-2 if w.dtype == synth.DTYPE_BF16 else 1e-5, ffn_shape=shape)
