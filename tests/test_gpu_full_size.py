"""Parity at the workloads' full sizes, in the launch configuration bench.py
times (all streams, all layers, proactive fills where the library puts them).

The oracle replays streams 0 and S-1 and two seeded streams between them
from the host twin's inputs (streams never interact in the logical cache
path, so a stream replayed alone is exact): logits within one ulp,
decisions, per-token events and the per-(stream, layer) counters bit for
bit, and FFN outputs of sampled (stream, token, layer) triples within the
bf16 tolerance.  For all streams the
invariants that hold at any size are checked on every token: hits + demand
misses = K, |C| <= capacity, proactive loads <= R (= 0 in update-only mode),
traffic = (D + P) x expert bytes, physical fills <= D + P.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import host_routers, oracle_logits, oracle_run, rel_err, say, split_slots, stable_seed

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def replay_streams(w, n_mid=2):
    """The streams the oracle replays: the first, the last and n_mid seeded
    ones between them (the same on every run)."""
    if w.S <= 2:
        return list(range(w.S))
    rng = np.random.default_rng(stable_seed(f"replay streams {w.name} S={w.S}"))
    mid = rng.choice(np.arange(1, w.S - 1), size=min(n_mid, w.S - 2), replace=False)
    return sorted({0, w.S - 1, *(int(s) for s in mid)})


def run_full(w, T, ffn_samples=8, seed=0, fills=None):
    from paper_2609_04895_amd import cmoe as B
    from paper_2609_04895_amd.workload import engine_for
    say(f"full-size parity {w.name}: L={w.L} (model layers {w.layer0}..{w.layer0 + w.L - 1}) N={w.N} K={w.K} "
        f"d={w.d} F={w.F} C={w.C} R={w.R} S={w.S}, {T} tokens")
    inp = synth.device_inputs(w, T=T)
    eng = engine_for(w, inp, fills=fills)
    y = torch.empty((w.S, w.L, w.d), dtype=torch.float32, device="cuda:0")
    streams = replay_streams(w)
    say(f"  replayed streams {streams}")
    WR, WT, WS = host_routers(w)
    bias = synth.zipf_bias(w)
    H = {(s, l): synth.hidden_host(w, s, l, T=T) for s in streams for l in range(w.L)}
    run = oracle_run(w.replace(S=len(streams)))
    rng = np.random.default_rng(seed)
    ffn_at = {(int(rng.integers(T)), int(rng.integers(len(streams))), int(rng.integers(w.L)))
              for _ in range(ffn_samples)}
    ulp_diffs = 0
    worst = 0.0
    max_abs64 = 0.0       # max |z_gpu - z_fp64| over all sampled logits
    max_ulp64 = 0.0       # the same in units of the fp32 ulp of z (0.5: correctly rounded)
    near_ties = 0         # (stream, token, layer) whose K-th / (K+1)-th native logit gap is < 1e-6
    mats = [WR] + ([WT] if w.has_temporal else []) + ([WS] if w.has_spatio else [])
    W64 = [[M[l].astype(np.float64) for l in range(w.L)] for M in mats]
    experts = {}
    for t in range(T):
        eng.cmoe_step(inp["hidden"][t], y)
        zg_all = eng.cmoe_read(B.CMOE_VIEW_LOGITS)               # [L][S][n_r][N]
        zg = zg_all[:, streams].transpose(1, 0, 2, 3)            # [streams][L][n_r][N]
        ref = oracle_logits(w, WR, WT, WS, bias, H, t, streams)   # [streams][L][n_r][N]
        d = zg != ref
        if d.any():
            gap = np.abs(zg.astype(np.float64) - ref)
            assert np.all(gap <= np.spacing(np.abs(ref))), f"token {t}: logit differs by more than one ulp"
            ulp_diffs += int(d.sum())
        # fp64 logits from numpy (independent of the oracle's C code)
        for i, s in enumerate(streams):
            for l in range(w.L):
                h64 = H[(s, l)][t].astype(np.float64)
                for r in range(len(mats)):
                    z64 = W64[r][l] @ h64
                    if r == 0 and bias is not None:
                        z64 = z64 + bias[l].astype(np.float64)
                    err = np.abs(zg[i, l, r].astype(np.float64) - z64)
                    max_abs64 = max(max_abs64, float(err.max()))
                    max_ulp64 = max(max_ulp64, float(np.max(err / np.spacing(np.abs(z64).astype(np.float32)))))
                    if r == 0 and w.K < w.N:
                        zs = np.sort(z64)[::-1]
                        near_ties += int(zs[w.K - 1] - zs[w.K] < 1e-6)
        out = run.step(*split_slots(w, zg), want="all")
        sel = eng.cmoe_read(B.CMOE_VIEW_SELECTED)                 # [L][S][K]
        assert np.array_equal(sel[:, streams].transpose(1, 0, 2), out["sel"]), f"token {t}: selections"
        cache = eng.cache_sets()                                   # [S][L][N]
        assert np.array_equal(cache[streams], run.cache.astype(bool)), f"token {t}: caches"
        ev = eng.cmoe_read(B.CMOE_VIEW_EVENTS)                    # [L][S][4]
        assert np.array_equal(ev[:, streams, 0].T, out["hits"])
        assert np.array_equal(ev[:, streams, 1].T, out["nD"])
        assert np.array_equal(ev[:, streams, 2].T, out["nP"])
        # invariants over all streams
        assert np.all(ev[:, :, 0] + ev[:, :, 1] == w.K), f"token {t}: hits + misses != K"
        assert np.all(cache.sum(axis=-1) <= w.C), f"token {t}: cache over capacity"
        assert np.all(ev[:, :, 2] <= (w.R if w.has_spatio else 0)), f"token {t}: too many proactive loads"
        for (tt, i, l) in ffn_at:
            if tt != t:
                continue
            s = streams[i]
            yg = y[s, l].cpu().numpy()
            ex = []
            for e in out["sel"][i, l]:
                key = (l, int(e))
                if key not in experts:
                    experts[key] = synth.expert_host(w, l, int(e))
                ex.append(experts[key])
            ref = oracle.moe_ffn(np.stack([a for a, _, _ in ex]), np.stack([b for _, b, _ in ex]),
                                 np.stack([c for _, _, c in ex]), out["gate"][i, l], H[(s, l)][t])
            err = rel_err(yg, ref)
            worst = max(worst, err)
            assert err <= 2e-2, f"token {t} stream {s} layer {l}: FFN relative error {err}"
    tot, per, phys = eng.cmoe_stats()
    assert np.array_equal(per[streams], run.ctr), "per-(stream, layer) counters"
    assert tot["accesses"] == w.S * w.L * T * w.K
    assert tot["hits"] + tot["demand_misses"] == tot["accesses"]
    assert tot["tokens"] == w.S * T
    assert tot["traffic_bytes"] == (tot["demand_misses"] + tot["proactive_loads"]) * w.expert_bytes
    if not w.arena_slots:   # an arena that holds the union copies each expert once per logical load at most
        assert tot["phys_fills"] <= tot["demand_misses"] + tot["proactive_loads"]
    if w.S == 1:   # the arena is the stream's own cache: every logical load is a copy
        assert tot["phys_fills"] == tot["demand_misses"] + tot["proactive_loads"]
    if not w.has_spatio or w.R == 0:
        assert tot["proactive_loads"] == 0
    assert max_ulp64 <= 1.0, f"max |z_gpu - z_fp64| = {max_ulp64} ulp"
    say(f"{w.name}: ok; one-ulp logit differences {ulp_diffs}; max |z_gpu - z_fp64| {max_abs64:.3g} "
        f"({max_ulp64:.3f} ulp); "
        f"Top-K near-tie opportunities (gap < 1e-6) {near_ties}; worst FFN error {worst:.3g}; "
        f"hit {1 - tot['demand_misses'] / tot['accesses']:.4f}; proactive {tot['proactive_loads']}; "
        f"physical fills {tot['phys_fills']}")
    eng.cmoe_destroy()
    del inp, eng
    torch.cuda.empty_cache()


def test_full_size_qwen3_30b_update_only():
    run_full(synth.WORKLOADS["qwen3_30b"], T=24)


@pytest.mark.parametrize("S", [16, 32])
def test_full_size_qwen3_30b_fewer_streams(S):
    # Fewer than 4 tokens per expert on average: the FFN grids spread every
    # work unit over all XCDs (80-110 units per layer step at full size).
    run_full(synth.WORKLOADS["qwen3_30b"].replace(S=S), T=12, ffn_samples=6)


def test_full_size_gptoss_20b_full_mode():
    run_full(synth.WORKLOADS["gptoss_20b"], T=24)


@pytest.mark.parametrize("C,R", [(C, R) for C in (16, 32, 64) for R in (0, 2, 4)])
def test_full_size_qwen3_30b_zipf_sweep_points(C, R):
    """Every (C, R) point of the Zipf workload's capacity x refinement-budget
    sweep (the stand-in for Table 3's sweep)."""
    run_full(synth.WORKLOADS["qwen3_30b_zipf"].replace(C=C, R=R), T=10, ffn_samples=4)


# Pinned host memory one process can hold on the test machine: about 64 GiB
# (measured with hipHostMalloc: one 64 GiB block, or 14 of the 4.83 GB
# per-layer pools at once, succeed, a 15th fails; memlock is unlimited and the
# host has 309 GB of RAM, so the limit is the driver's on device-mapped host
# memory).
PINNED_LIMIT_BYTES = 64 * 2 ** 30


def test_full_size_qwen3_235b_slice_host_pool():
    """Qwen3-235B-A22B-shaped slice with its cold pool in pinned host memory.

    The full 16-layer pool is 77.3 GB, above what one process can pin on the
    test machine, so the test keeps as many layers as fit (14: 67.6 GB), every
    other dimension at full size.  Proactive copies run on the side stream,
    overlapping the FFN (the default joins them to the demand fill)."""
    w = synth.WORKLOADS["qwen3_235b_slice"]
    L = min(w.L, PINNED_LIMIT_BYTES // (w.N * w.expert_bytes))
    assert L == 14
    run_full(w.replace(L=L), T=8, ffn_samples=4, fills="side")


def test_full_size_qwen3_235b_slice_last_layers_host_pool():
    """The two layers of the Qwen3-235B-A22B slice that do not fit next to the
    other 14 in pinned host memory (model layers 14 and 15: their own routers,
    experts and hidden states) as an engine of their own, so that every layer
    of the slice passes through the kernels at full size.  Its first layer is
    refined from its own last layer's prediction, not from model layer 13."""
    w = synth.WORKLOADS["qwen3_235b_slice"]
    first = min(w.L, PINNED_LIMIT_BYTES // (w.N * w.expert_bytes))
    assert first == 14
    run_full(w.replace(L=w.L - first, layer0=first), T=8, ffn_samples=4)


def test_full_size_qwen3_30b_single_stream_pinned_pool():
    """One decode stream at the Qwen3 shape with the cold pool in pinned host
    memory: the HBM arena holds exactly C = 32 slots per layer (the paper's
    per-layer capacity taken literally) and physical copies equal D + P."""
    run_full(synth.WORKLOADS["qwen3_30b_s1"], T=12, ffn_samples=6)
