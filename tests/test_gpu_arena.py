"""Parity of the capacity-limited arena (fewer HBM slots per layer than the
union of the streams' caches can reach) with the oracle: slot maps, physical
copies and every cache decision bit for bit on every token, through the cache
path alone and end to end, at small and full size.  When the union does not
fit, the layer step's FFN runs in rounds of at most arena_slots experts."""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import compare_step, host_routers, oracle_logits, oracle_run, rel_err, say, split_slots, stable_seed
from test_gpu_cache_parity import logits_sequence

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

M_T, M_F, M_SO = oracle.MODE_TEMPORAL, oracle.MODE_SPATIO_TEMPORAL, oracle.MODE_SPATIO_ONLY
P_R, P_LRU, P_LFU, P_LRFU = oracle.POLICY_ROUTER, oracle.POLICY_LRU, oracle.POLICY_LFU, oracle.POLICY_LRFU

CASES = [
    # L, N, K, C, R, S, mode, policy, P, warmup, ties, side
    (3, 16, 2, 6, 0, 4, M_T, P_R, 4, 0, False, True),
    (3, 16, 2, 6, 0, 4, M_T, P_R, 1, 0, True, False),       # a single slot
    (2, 32, 4, 8, 2, 8, M_F, P_R, 8, 0, True, True),
    (2, 32, 4, 8, 2, 8, M_F, P_R, 3, 0, True, True),        # fewer slots than Top-K
    (2, 128, 8, 32, 4, 64, M_F, P_R, 32, 0, False, True),   # 32 slots per layer, 64 streams
    (2, 128, 8, 32, 0, 64, M_T, P_R, 32, 0, True, False),
    (2, 100, 7, 20, 5, 37, M_F, P_R, 17, 2, True, True),    # ragged N and S, warm-up tokens
    (2, 256, 8, 40, 12, 20, M_F, P_R, 64, 0, True, True),   # four experts per lane
    (2, 256, 64, 256, 256, 3, M_F, P_R, 100, 0, True, True),  # the largest K, two rounds
    (2, 64, 8, 16, 4, 16, M_SO, P_LRU, 10, 0, True, True),
    (2, 64, 8, 16, 0, 16, M_T, P_LFU, 12, 0, True, False),
    (2, 64, 8, 16, 0, 16, M_T, P_LRFU, 9, 1, False, True),
    (3, 8, 2, 3, 2, 1000, M_F, P_R, 5, 0, True, True),      # 1000 streams through 5 slots
    (2, 33, 3, 5, 2, 9, M_F, P_R, 2, 2, True, False),
]


def case_id(c):
    return "L{}N{}K{}C{}R{}S{}m{}p{}P{}".format(*c[:9])


@pytest.mark.parametrize("case", CASES, ids=[case_id(c) for c in CASES])
def test_arena_cache_path_bit_exact(case):
    from paper_2609_04895_amd import cmoe as B
    L, N, K, C, R, S, mode, policy, P, warmup, ties, side = case
    seed = stable_seed(case_id(case))
    say(f"arena cache path {case_id(case)} seed={seed} warmup={warmup} ties={ties} side={side}")
    T = 10
    z = logits_sequence(np.random.default_rng(seed), T, S, L, N, ties)
    dev = torch.device("cuda", 0)
    d = F = 64
    w = torch.zeros((L, N, d), dtype=torch.float32, device=dev)
    pool = torch.arange(L * N * 3 * d * F, dtype=torch.float32, device=dev).reshape(L, N, 3 * d * F)
    cfg = B.make_config(L, N, K, d, F, C, R, S, mode, B.CMOE_F32, B.CMOE_POOL_DEVICE, warmup,
                        B.CMOE_FLAG_FILL_ON_SIDE if side else 0, policy, 0.5, P)
    has_t = policy == P_R
    has_s = mode != M_T
    eng = B.Engine(cfg, w, w if has_t else None, w if has_s else None, None, pool,
                   side_stream=torch.cuda.Stream() if side else None)
    run = oracle.Run(L, N, K, C, R, S, mode, warmup, policy=policy, lrfu_lambda=0.5, arena_slots=P)
    overflow = 0
    for t in range(T):
        zR = torch.from_numpy(z[t, 0]).to(dev)
        zT = torch.from_numpy(z[t, 1]).to(dev) if has_t else None
        zS = torch.from_numpy(z[t, 2]).to(dev) if has_s else None
        eng.cmoe_step_logits(zR, zT, zS)
        out = run.step(z[t, 0], z[t, 1] if has_t else None, z[t, 2] if has_s else None, want="all")
        compare_step(eng, run, out, f"{case_id(case)} token {t}")
        overflow += int((run.cache.any(axis=0).sum(axis=-1) > P).sum())
    total, _, _ = eng.cmoe_stats()
    ref = run.totals()
    for k in ("accesses", "hits", "demand_misses", "proactive_loads", "tokens", "phys_fills"):
        assert total[k] == ref[k], k
    say(f"{case_id(case)}: layer steps whose union overflowed the arena: {overflow}; copies {ref['phys_fills']}")
    eng.cmoe_destroy()


E2E = [
    ("update_only_bf16", "qwen3_30b", dict(L=2, N=32, K=4, C=8, S=16, d=256, F=128, arena_slots=8), "single"),
    ("update_only_bf16_grouped", "qwen3_30b", dict(L=2, N=32, K=4, C=8, S=16, d=256, F=128, arena_slots=6),
     "grouped"),
    ("update_only_fp32", "tiny", dict(L=3, N=16, K=2, C=6, S=5, d=128, F=64, arena_slots=3), None),
    ("full_bf16", "gptoss_20b", dict(L=3, N=32, K=4, C=8, R=2, S=24, d=256, F=128, arena_slots=6), None),
    ("heavy_buckets_bf16", "gptoss_20b", dict(L=2, N=16, K=4, C=8, R=2, S=200, d=128, F=128, arena_slots=4),
     "grouped"),
    ("heavy_buckets_single", "gptoss_20b", dict(L=2, N=16, K=4, C=8, R=2, S=200, d=128, F=128, arena_slots=5),
     "single"),
]


@pytest.mark.parametrize("name,base,repl,shape", E2E, ids=[e[0] for e in E2E])
def test_arena_end_to_end(name, base, repl, shape):
    from test_gpu_e2e_parity import run_e2e
    w = synth.WORKLOADS[base].replace(name=f"arena_{name}", **repl)
    say(f"arena end to end {name}: {repl} shape={shape}")
    run_e2e(w, T=5, tol=2e-2 if w.dtype == synth.DTYPE_BF16 else 1e-5, ffn_shape=shape)


def run_arena_full(w, T, ffn_samples, seed=0):
    """Full size: every stream's cache path replayed by the oracle from the
    GPU's logits (bit for bit, slot maps and copies included), the sampled
    streams' logits against the oracle's fp64 logits (one ulp), and sampled
    FFN outputs against the oracle's fp64 FFN."""
    from paper_2609_04895_amd import cmoe as B
    from paper_2609_04895_amd.workload import engine_for
    say(f"arena full size {w.name}: L={w.L} N={w.N} K={w.K} d={w.d} F={w.F} C={w.C} R={w.R} S={w.S} "
        f"slots={w.arena_slots}, {T} tokens")
    inp = synth.device_inputs(w, T=T)
    eng = engine_for(w, inp)
    y = torch.empty((w.S, w.L, w.d), dtype=torch.float32, device="cuda:0")
    streams = [0, w.S - 1]
    WR, WT, WS = host_routers(w)
    bias = synth.zipf_bias(w)
    H = {(s, l): synth.hidden_host(w, s, l, T=T) for s in streams for l in range(w.L)}
    run = oracle_run(w)
    rng = np.random.default_rng(seed)
    ffn_at = {(int(rng.integers(T)), int(rng.integers(len(streams))), int(rng.integers(w.L)))
              for _ in range(ffn_samples)}
    experts = {}
    overflow = 0
    for t in range(T):
        eng.cmoe_step(inp["hidden"][t], y)
        zg = eng.cmoe_read(B.CMOE_VIEW_LOGITS).transpose(1, 0, 2, 3)      # [S][L][n_r][N]
        ref = oracle_logits(w, WR, WT, WS, bias, H, t, streams)
        gap = np.abs(zg[streams].astype(np.float64) - ref)
        assert np.all(gap <= np.spacing(np.abs(ref))), f"token {t}: logit differs by more than one ulp"
        out = run.step(*split_slots(w, np.ascontiguousarray(zg)), want="all")
        compare_step(eng, run, out, f"{w.name} token {t}")
        overflow += int((run.cache.any(axis=0).sum(axis=-1) > w.arena_slots).sum())
        yg = None
        for (tt, i, l) in ffn_at:
            if tt != t:
                continue
            if yg is None:
                yg = y.cpu().numpy()
            s = streams[i]
            ex = []
            for e in out["sel"][s, l]:
                key = (l, int(e))
                if key not in experts:
                    experts[key] = synth.expert_host(w, l, int(e))
                ex.append(experts[key])
            r = oracle.moe_ffn(np.stack([a for a, _, _ in ex]), np.stack([b for _, b, _ in ex]),
                               np.stack([c for _, _, c in ex]), out["gate"][s, l], H[(s, l)][t])
            err = rel_err(yg[s, l], r)
            assert err <= 2e-2, f"token {t} stream {s} layer {l}: FFN relative error {err}"
    tot, _, _ = eng.cmoe_stats()
    ref_tot = run.totals()
    for k in ("accesses", "hits", "demand_misses", "proactive_loads", "tokens", "phys_fills"):
        assert tot[k] == ref_tot[k], k
    say(f"{w.name} with {w.arena_slots} slots: ok; overflowing layer steps {overflow} of {T * w.L}; "
        f"copies {tot['phys_fills']} ({tot['phys_bytes'] / 1e9:.1f} GB); logical loads "
        f"{tot['demand_misses'] + tot['proactive_loads']}")
    assert overflow > 0
    eng.cmoe_destroy()
    del inp, eng
    torch.cuda.empty_cache()


def test_arena_full_size_qwen3_30b_32_slots_hbm_pool():
    """The Qwen3 shape, 64 streams, 32 HBM slots per layer, pool in HBM."""
    run_arena_full(synth.WORKLOADS["qwen3_30b"].replace(arena_slots=32), T=6, ffn_samples=6)


def test_arena_full_size_qwen3_235b_slice_32_slots_host_pool():
    """The Qwen3-235B-A22B-shaped slice read literally: 32 HBM slots per
    layer, 256 streams, full mode, cold pool in pinned host memory (14 of its
    16 layers: the most one process can pin on the test machine)."""
    from test_gpu_full_size import PINNED_LIMIT_BYTES
    w = synth.WORKLOADS["qwen3_235b_slice"]
    L = min(w.L, PINNED_LIMIT_BYTES // (w.N * w.expert_bytes))
    run_arena_full(w.replace(L=L, arena_slots=32), T=3, ffn_samples=4, seed=3)
