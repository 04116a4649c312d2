"""Bit-exact parity of the cache path (softmax, Top-K, refinement, access,
retention, counters, residency, fills) with the oracle, driven through
cmoe_step_logits with the same fp32 logits on both sides."""
import numpy as np
import pytest

import oracle
from gpu_util import compare_step, say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def make_engine(L, N, K, C, R, S, mode, warmup=0, side=True, d=64, F=64):
    from paper_2609_04895_amd import cmoe as B
    dev = torch.device("cuda", 0)
    # router weights are not read by cmoe_step_logits; the pool is (fills)
    w = torch.zeros((L, N, d), dtype=torch.float32, device=dev)
    pool = torch.arange(L * N * 3 * d * F, dtype=torch.float32, device=dev).reshape(L, N, 3 * d * F)
    cfg = B.make_config(L, N, K, d, F, C, R, S, mode, B.CMOE_F32, B.CMOE_POOL_DEVICE, warmup,
                        B.CMOE_FLAG_FILL_ON_SIDE if side else 0)
    eng = B.Engine(cfg, w, w, w if mode == 1 else None, None, pool,
                   side_stream=torch.cuda.Stream() if side else None)
    return eng, pool


def logits_sequence(rng, T, S, L, N, ties):
    """AR(1) logits [T][3][S][L][N]; with `ties` the values are rounded to
    multiples of 1/4 so that equal logits and equal scores are frequent."""
    z = np.empty((T, 3, S, L, N), np.float32)
    prev = rng.normal(size=(3, S, L, N))
    for t in range(T):
        prev = 0.85 * prev + np.sqrt(1 - 0.85 ** 2) * rng.normal(size=prev.shape)
        v = prev * 2.0
        if ties:
            v = np.round(v * 4) / 4
        z[t] = v.astype(np.float32)
    return z


CASES = [
    # L, N, K, C, R, S, mode, warmup, ties, side
    (3, 16, 2, 6, 0, 1, 0, 0, False, True),
    (3, 16, 2, 2, 0, 3, 0, 0, True, True),       # C = K: the cache is the last selection
    (2, 16, 2, 16, 0, 2, 0, 0, True, False),     # C = N: only compulsory misses
    (4, 32, 4, 8, 2, 5, 1, 0, True, True),       # GPT-OSS-like shape, full mode
    (3, 100, 7, 20, 5, 37, 1, 2, True, True),    # ragged N and S
    (3, 128, 8, 32, 0, 9, 1, 0, False, True),    # full mode with R = 0
    (2, 128, 8, 32, 0, 70, 0, 1, True, True),    # Qwen3-like shape, update-only
    (2, 256, 8, 40, 12, 6, 1, 0, True, True),    # N = 256 (four experts per lane)
    (2, 64, 64, 64, 64, 2, 1, 0, True, False),   # K = C = N = R
    (2, 1, 1, 1, 1, 2, 1, 0, False, True),       # a single expert
    (2, 256, 8, 16, 4, 300, 1, 0, True, True),   # 1200 cache words per layer: several per fill thread
    (1, 32, 4, 8, 3, 5, 1, 0, True, True),       # one layer: its causal predecessor is itself, one token back
    (2, 256, 64, 256, 256, 3, 1, 0, True, True),  # the largest N, K, C and R the kernels take
    (2, 8, 2, 3, 2, 1000, 1, 0, True, True),      # 1000 streams over 8 experts: buckets of ~250 tokens
]


@pytest.mark.parametrize("case", CASES, ids=[f"L{c[0]}N{c[1]}K{c[2]}C{c[3]}R{c[4]}S{c[5]}m{c[6]}" for c in CASES])
def test_cache_path_bit_exact(case):
    L, N, K, C, R, S, mode, warmup, ties, side = case
    say(f"cache parity case {case}")
    T = 20
    rng = np.random.default_rng(hash(case) % (2 ** 32))
    z = logits_sequence(rng, T, S, L, N, ties)
    eng, _ = make_engine(L, N, K, C, R, S, mode, warmup, side)
    run = oracle.Run(L, N, K, C, R, S, mode, warmup)
    dev = torch.device("cuda", 0)
    for t in range(T):
        zR, zT, zS = (torch.from_numpy(z[t, i]).to(dev) for i in range(3))
        eng.cmoe_step_logits(zR, zT, zS if mode == 1 else None)
        out = run.step(z[t, 0], z[t, 1], z[t, 2] if mode == 1 else None, want="all")
        compare_step(eng, run, out, f"case {case} token {t}")
    total, per, phys = eng.cmoe_stats()
    ref = run.totals()
    for k in ("accesses", "hits", "demand_misses", "proactive_loads", "tokens", "phys_fills"):
        assert total[k] == ref[k], k
    assert total["hits"] + total["demand_misses"] == total["accesses"]
    assert total["traffic_bytes"] == (total["demand_misses"] + total["proactive_loads"]) * 3 * 64 * 64 * 4
    if mode == 0 or R == 0:
        assert total["proactive_loads"] == 0
    eng.cmoe_destroy()


def test_refinement_budget_change_and_cache_set_replay():
    """R changes between tokens (no retraining needed, Section 3.3) and a
    cache set from the host are followed identically by both sides."""
    L, N, K, C, S = 3, 32, 4, 8, 4
    rng = np.random.default_rng(5)
    z = logits_sequence(rng, 16, S, L, N, ties=True)
    eng, _ = make_engine(L, N, K, C, 2, S, 1)
    run = oracle.Run(L, N, K, C, 2, S, 1)
    dev = torch.device("cuda", 0)
    for t in range(16):
        if t == 5:
            eng.cmoe_set_R(6)
            run.set_R(6)
        if t == 9:
            eng.cmoe_set_R(0)
            run.set_R(0)
        if t == 12:
            eng.cmoe_set_cache(1, 2, [3, 7, 30])
            run.cache[1, 2, :] = 0
            run.cache[1, 2, [3, 7, 30]] = 1
            assert eng.cmoe_get_cache(1, 2) == [3, 7, 30]
        zR, zT, zS = (torch.from_numpy(z[t, i]).to(dev) for i in range(3))
        eng.cmoe_step_logits(zR, zT, zS)
        out = run.step(z[t, 0], z[t, 1], z[t, 2], want="all")
        compare_step(eng, run, out, f"token {t}")
    for s in range(S):
        for l in range(L):
            assert eng.cmoe_get_cache(s, l) == sorted(np.nonzero(run.cache[s, l])[0].tolist())
    # reset returns to an empty state and a fresh replay matches again
    eng.cmoe_reset()
    run = oracle.Run(L, N, K, C, 0, S, 1)
    for t in range(4):
        zR, zT, zS = (torch.from_numpy(z[t, i]).to(dev) for i in range(3))
        eng.cmoe_step_logits(zR, zT, zS)
        out = run.step(z[t, 0], z[t, 1], z[t, 2], want="all")
        compare_step(eng, run, out, f"after reset, token {t}")
    eng.cmoe_destroy()


def test_fills_copy_the_right_expert_bytes():
    """Arena slots hold exactly the cold-pool values of the expert mapped
    there, each fp32 matrix transposed (W_gate^T, W_up^T [d][F], then
    W_down^T [F][d])."""
    L, N, K, C, S = 2, 16, 2, 4, 3
    rng = np.random.default_rng(8)
    z = logits_sequence(rng, 6, S, L, N, ties=False)
    eng, pool = make_engine(L, N, K, C, 2, S, 1)
    dev = torch.device("cuda", 0)
    for t in range(6):
        zR, zT, zS = (torch.from_numpy(z[t, i]).to(dev) for i in range(3))
        eng.cmoe_step_logits(zR, zT, zS)
    from paper_2609_04895_amd import cmoe as B
    slots = eng.cmoe_read(B.CMOE_VIEW_SLOTS)
    n_slots = min(N, S * C)
    per = 3 * 64 * 64
    arena = eng.arena[: L * n_slots * per * 4].view(torch.float32).reshape(L, n_slots, per)
    d = F = 64
    for l in range(L):
        for e in range(N):
            q = int(slots[l, e])
            if q >= 0:
                src = pool[l, e]
                want = torch.cat([src[:F * d].reshape(F, d).t().reshape(-1),
                                  src[F * d:2 * F * d].reshape(F, d).t().reshape(-1),
                                  src[2 * F * d:].reshape(d, F).t().reshape(-1)])
                assert torch.equal(arena[l, q], want), (l, e, q)
    eng.cmoe_destroy()


def packed_from_plain(plain_u16, d, F):
    """The packed slot order of a bf16 expert (see fill.hip), written out from
    its documented formula: 16-byte units of 8 bf16."""
    Wg = plain_u16[: F * d].reshape(F, d)
    Wu = plain_u16[F * d: 2 * F * d].reshape(F, d)
    Wd = plain_u16[2 * F * d:].reshape(d, F)
    units = []
    for ft in range(F // 16):
        for c in range(d // 64):
            for mat in (Wg, Wu):
                for half in range(2):
                    for lane in range(64):
                        row, col = 16 * ft + lane % 16, 64 * c + 32 * half + 8 * (lane // 16)
                        units.append(mat[row, col:col + 8])
    for dt in range(d // 32):
        for c in range(F // 64):
            for mt in range(2):
                for half in range(2):
                    for lane in range(64):
                        row, col = 32 * dt + 16 * mt + lane % 16, 64 * c + 32 * half + 8 * (lane // 16)
                        units.append(Wd[row, col:col + 8])
    return np.concatenate(units)


@pytest.mark.parametrize("pool_kind,d,F", [("device", 128, 128), ("host", 128, 128), ("device", 192, 320),
                                            ("host", 192, 320)])
def test_bf16_slots_hold_the_packed_expert(pool_kind, d, F):
    # the fill walks an HBM pool in packed-block order and a pinned host pool
    # in source order; both must leave the same packed bytes in the slots
    from paper_2609_04895_amd import cmoe as B
    L, N, K, C, S = 2, 8, 2, 3, 3
    say(f"packed slots, {pool_kind} pool, d={d} F={F}")
    dev = torch.device("cuda", 0)
    w = torch.zeros((L, N, d), dtype=torch.bfloat16, device=dev)
    per = 3 * d * F
    gen = torch.Generator().manual_seed(3)
    pool_cpu = torch.randint(0, 2 ** 16, (L, N, per), generator=gen, dtype=torch.int32).to(torch.int16)
    if pool_kind == "host":
        pool = pool_cpu.view(torch.bfloat16).pin_memory()
        kind = B.CMOE_POOL_HOST_PINNED
    else:
        pool = pool_cpu.view(torch.bfloat16).to(dev)
        kind = B.CMOE_POOL_DEVICE
    cfg = B.make_config(L, N, K, d, F, C, 0, S, 0, B.CMOE_BF16, kind)
    eng = B.Engine(cfg, w, w, None, None, pool)
    rng = np.random.default_rng(4)
    z = logits_sequence(rng, 5, S, L, N, ties=False)
    for t in range(5):
        eng.cmoe_step_logits(torch.from_numpy(z[t, 0]).to(dev), torch.from_numpy(z[t, 1]).to(dev))
    slots = eng.cmoe_read(B.CMOE_VIEW_SLOTS)
    n_slots = min(N, S * C)
    arena = eng.arena[: L * n_slots * per * 2].view(torch.int16).cpu().numpy().view(np.uint16).reshape(L, n_slots, per)
    plain = pool_cpu.numpy().view(np.uint16)
    checked = 0
    for l in range(L):
        for e in range(N):
            q = int(slots[l, e])
            if q >= 0:
                assert np.array_equal(arena[l, q], packed_from_plain(plain[l, e], d, F)), (l, e, q)
                checked += 1
    assert checked > 0
    eng.cmoe_destroy()
