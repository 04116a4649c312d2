"""End-to-end parity of cmoe_step (router GEMV, cache path, fills, expert FFN)
with the oracle on the same seeded inputs.

- The device generator reproduces the host twin's tensors bit for bit.
- Router logits: the GPU's fp32 logits equal the oracle's (fp64 sum rounded
  once) except possibly for sums within an fp32 rounding boundary; any
  difference is at most one ulp and is counted.
- Decisions: the oracle replayed on the GPU's own logits matches every
  selection, cache set and counter bit for bit; decisions from the oracle's
  own logits may differ only where a Top-K logit gap is below 1e-6.
- FFN outputs: max-norm relative error <= 1e-5 (fp32) or 2e-2 (bf16, fp32
  accumulation) against the oracle's fp64 SwiGLU on the same selection.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import (clone_run, compare_step, host_routers, oracle_logits, oracle_run, rel_err, say,
                      split_slots)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def bf16_bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def f32_of(w, t):
    """Device tensor -> float32 numpy of the stored values."""
    if w.dtype == synth.DTYPE_BF16:
        return (bf16_bits(t).astype(np.uint32) << 16).view(np.float32)
    return t.cpu().numpy()


def test_device_generator_matches_host_twin():
    for name, w in (("tiny", synth.WORKLOADS["tiny"]),
                    ("small_bf16", synth.WORKLOADS["gptoss_20b"].replace(L=2, S=3, d=256, F=128))):
        say(f"generator twin {name}")
        inp = synth.device_inputs(w, T=7)
        for kind, key in ((synth.KIND_ROUTER_NATIVE, "wR"), (synth.KIND_ROUTER_TEMPORAL, "wT")):
            for l in range(w.L):
                assert np.array_equal(f32_of(w, inp[key][l]), synth.router_host(w, kind, l))
        for l, e in ((0, 0), (w.L - 1, w.N - 1), (0, w.N // 2)):
            g, u, dn = synth.expert_host(w, l, e)
            dev = f32_of(w, inp["pool"][l, e])
            fd = w.F * w.d
            assert np.array_equal(dev[:fd], g.ravel()) and np.array_equal(dev[fd:2 * fd], u.ravel())
            assert np.array_equal(dev[2 * fd:], dn.ravel())
        for s in range(w.S):
            for l in range(w.L):
                ref = synth.hidden_host(w, s, l, T=7)
                assert np.array_equal(f32_of(w, inp["hidden"][:, s, l]), ref)
        del inp


def run_e2e(w, T, tol, check_ffn_every=1, samples=None, ffn_shape=None):
    from paper_2609_04895_amd import cmoe as B
    from paper_2609_04895_amd.workload import engine_for
    inp = synth.device_inputs(w, T=T)
    eng = engine_for(w, inp, ffn_shape=ffn_shape)
    dev = torch.device("cuda", 0)
    y = torch.empty((w.S, w.L, w.d), dtype=torch.float32, device=dev)
    # host copies of what the oracle needs
    WR, WT, WS = host_routers(w)
    bias = synth.zipf_bias(w)
    H = {(s, l): synth.hidden_host(w, s, l, T=T) for s in range(w.S) for l in range(w.L)}
    experts = {}

    def expert(l, e):
        l, e = int(l), int(e)
        if (l, e) not in experts:
            experts[(l, e)] = synth.expert_host(w, l, e)
        return experts[(l, e)]

    run = oracle_run(w)
    ulp_diffs = 0
    near_ties = 0
    worst_ffn = 0.0
    for t in range(T):
        eng.cmoe_step(inp["hidden"][t], y)
        z_gpu = eng.cmoe_read(B.CMOE_VIEW_LOGITS)      # [L][S][n_r][N]
        # oracle logits from the host twin's inputs
        z_orc = oracle_logits(w, WR, WT, WS, bias, H, t, range(w.S))
        zg = z_gpu.transpose(1, 0, 2, 3)
        diff = zg != z_orc
        if diff.any():
            gap = np.abs(zg.astype(np.float64) - z_orc.astype(np.float64))
            assert np.all(gap <= np.spacing(np.abs(z_orc)) * 1.0001), "logit differs by more than one ulp"
            ulp_diffs += int(diff.sum())
        # step-local: decisions from the oracle's own logits vs the GPU's
        own = clone_run(run).step(*split_slots(w, z_orc), want="all")
        out = run.step(*split_slots(w, zg), want="all")
        compare_step(eng, run, out, f"{w.name} token {t}")
        if not np.array_equal(own["sel"], out["sel"]):
            for s, l in zip(*np.nonzero((own["sel"] != out["sel"]).any(axis=-1))):
                zs = np.sort(z_orc[s, l, 0].astype(np.float64))[::-1]
                assert zs[w.K - 1] - zs[w.K] < 1e-6, "selection differs without a near tie"
                near_ties += 1
        # FFN
        if t % check_ffn_every == 0:
            yg = y.cpu().numpy()
            pairs = samples if samples is not None else [(s, l) for s in range(w.S) for l in range(w.L)]
            for s, l in pairs:
                sel = out["sel"][s, l]
                Wg = np.stack([expert(l, e)[0] for e in sel])
                Wu = np.stack([expert(l, e)[1] for e in sel])
                Wd = np.stack([expert(l, e)[2] for e in sel])
                ref = oracle.moe_ffn(Wg, Wu, Wd, out["gate"][s, l], H[(s, l)][t])
                err = rel_err(yg[s, l], ref)
                worst_ffn = max(worst_ffn, err)
                assert err <= tol, f"token {t} stream {s} layer {l}: FFN relative error {err}"
    say(f"{w.name}: logits differing by one ulp: {ulp_diffs}; near-tie selection flips: {near_ties}; "
        f"worst FFN error {worst_ffn:.3g}")
    tot, _, _ = eng.cmoe_stats()
    ref = run.totals()
    for k in ("accesses", "hits", "demand_misses", "proactive_loads", "tokens", "phys_fills"):
        assert tot[k] == ref[k], k
    eng.cmoe_destroy()
    del inp


def test_tiny_fp32_workload_end_to_end():
    """L=4, N=16, K=2, d=256, F=512, C=6, update-only, 1 stream x 256 tokens."""
    run_e2e(synth.WORKLOADS["tiny"], T=256, tol=1e-5)


def test_bf16_full_mode_small_shape():
    w = synth.WORKLOADS["qwen3_30b"].replace(name="bf16_small", L=3, d=256, F=128, S=20, C=32, R=4,
                                             mode=synth.MODE_SPATIO_TEMPORAL)
    run_e2e(w, T=10, tol=2e-2)


@pytest.mark.parametrize("shape", ["single", "grouped"])
def test_bf16_ragged_chunks_and_zipf_bias(shape):
    # d = 320 and F = 192 are not multiples of 256: exercises the chunk tails
    # (an odd number of 64-wide chunks; grouped down workgroups whose last
    # wavefronts have no d-tile); many tokens per expert (N = 16, S = 40)
    # exercises several token groups
    w = synth.WORKLOADS["qwen3_30b_zipf"].replace(name="bf16_ragged", L=2, N=16, K=4, d=320, F=192, S=40, C=6,
                                                  R=2)
    run_e2e(w, T=6, tol=2e-2, ffn_shape=shape)


@pytest.mark.parametrize("shape", ["single", "grouped"])
def test_bf16_hot_experts_span_several_ffn_units(shape):
    # 160 streams over 8 Zipf-biased experts: the hottest buckets hold well
    # over 64 tokens, so they are cut into several FFN work units, ranked by
    # size; every output is checked, with one-wavefront workgroups and with
    # grouped ones (activations of big units shared through LDS)
    w = synth.WORKLOADS["qwen3_30b_zipf"].replace(name="bf16_hot_units", L=2, N=8, K=2, d=256, F=128, S=160, C=4,
                                                  R=2)
    run_e2e(w, T=4, tol=2e-2, ffn_shape=shape)


def test_bf16_256_experts_full_mode():
    # four experts per lane in the cache kernel, sixteen expert tiles per router
    w = synth.WORKLOADS["qwen3_30b"].replace(name="bf16_n256", L=2, N=256, d=256, F=128, S=10, C=40, R=6,
                                             mode=synth.MODE_SPATIO_TEMPORAL)
    run_e2e(w, T=5, tol=2e-2)


def test_fp32_pool_in_pinned_host_memory():
    # plain fp32 expert copies read from pinned host memory by the fill kernel
    w = synth.WORKLOADS["tiny"].replace(name="tiny_host_pool", pool_kind=synth.POOL_HOST_PINNED, S=3, C=4)
    run_e2e(w, T=24, tol=1e-5)


def test_bf16_update_only_gptoss_like():
    w = synth.WORKLOADS["gptoss_20b"].replace(name="gptoss_small", L=2, d=192, F=192, S=7,
                                              mode=synth.MODE_TEMPORAL, R=0)
    run_e2e(w, T=8, tol=2e-2)


@pytest.mark.parametrize("dtype", [synth.DTYPE_BF16, synth.DTYPE_F32])
def test_single_layer_smallest_dims(dtype):
    # L = 1 (the refinement of each token reads the same layer's previous
    # prediction), d = F = 64 (one k chunk: every load block is a tail)
    w = synth.WORKLOADS["qwen3_30b"].replace(name=f"min_dims_{dtype}", L=1, N=8, K=2, d=64, F=64, S=5, C=3, R=2,
                                             mode=synth.MODE_SPATIO_TEMPORAL, dtype=dtype)
    run_e2e(w, T=8, tol=2e-2 if dtype == synth.DTYPE_BF16 else 1e-5)


def test_bf16_top11_output_combine():
    # K = 11: the output combine adds a full batch of eight gated outputs and
    # a clamped batch of three, in k order
    w = synth.WORKLOADS["qwen3_30b"].replace(name="bf16_top11", L=2, N=32, K=11, d=128, F=64, S=12, C=16)
    run_e2e(w, T=6, tol=2e-2)


def test_bf16_top64_largest_k():
    # K = 64 (the largest Top-K): eight full batches in the output combine,
    # 64 gated outputs per stream, every expert of a layer selected
    w = synth.WORKLOADS["qwen3_30b"].replace(name="bf16_top64", L=2, N=64, K=64, d=128, F=64, S=5, C=64)
    run_e2e(w, T=3, tol=2e-2)


@pytest.mark.parametrize("shape", ["single", "grouped"])
def test_bf16_buckets_of_hundreds_of_tokens(shape):
    # 600 streams over 4 experts, top-2: ~300 tokens per expert, so every
    # bucket is cut into about five 64-token work units
    w = synth.WORKLOADS["qwen3_30b"].replace(name="bf16_big_buckets", L=1, N=4, K=2, d=128, F=64, S=600, C=4, R=0)
    run_e2e(w, T=3, tol=2e-2, ffn_shape=shape)


@pytest.mark.parametrize("shape", ["single", "grouped"])
def test_bf16_multi_pass_units_with_ragged_expert_count(shape):
    # 37 experts (not a multiple of 4 or 16) under Zipf skew, 300 streams,
    # top-3: the hot experts' buckets take several work units, so the fill
    # kernel ranks all 37 bucket sizes (keys past N read as padding)
    w = synth.WORKLOADS["qwen3_30b_zipf"].replace(name="bf16_n37_multi", L=1, N=37, K=3, d=128, F=64, S=300, C=5,
                                                  R=2)
    run_e2e(w, T=3, tol=2e-2, ffn_shape=shape)


@pytest.mark.parametrize("base,N", [("qwen3_30b", 16), ("qwen3_30b_zipf", 64)])
def test_bf16_combine_in_the_next_cache_step_ragged_tail(base, N):
    # From the second layer on, the cache-step launch also combines the
    # previous layer's gated outputs in workgroups after the streams': 37
    # streams x d = 192 leave the last of them part-filled, K = 5 a part-filled
    # batch of outputs.  N = 16: 11.6 tokens per expert, each FFN work unit on
    # one XCD; N = 64 (full mode, with the refine-only launch of layer 0):
    # 2.9, units spread over all XCDs.
    w = synth.WORKLOADS[base].replace(name=f"bf16_combine_tail_{base}_{N}", L=3, N=N, K=5, d=192, F=128, S=37,
                                      C=6, R=2)
    run_e2e(w, T=3, tol=2e-2)


def test_profile_counts_one_combine_launch_per_token():
    from paper_2609_04895_amd.workload import engine_for
    w = synth.WORKLOADS["qwen3_30b"].replace(name="profile_counts", L=4, N=16, K=2, d=128, F=64, S=8, C=4, R=0)
    say(f"profile counts {w.name}")
    inp = synth.device_inputs(w, T=3)
    eng = engine_for(w, inp)
    y = torch.empty((w.S, w.L, w.d), dtype=torch.float32, device=torch.device("cuda", 0))
    eng.cmoe_step(inp["hidden"][0], y)
    eng.cmoe_profile_begin(2)
    for t in (1, 2):
        eng.cmoe_step(inp["hidden"][t], y)
    prof = eng.cmoe_profile_end()
    per_layer = {"router": 2 * w.L, "cache_step": 2 * w.L, "fill": 2 * w.L, "ffn_up": 2 * w.L, "ffn_down": 2 * w.L,
                 "combine": 2}
    for k, n in per_layer.items():
        assert prof[k][1] == n, (k, prof[k])
        assert prof[k][0] > 0, k
    eng.cmoe_destroy()
    del inp


def test_bf16_large_hidden_dims():
    # d = 8192, F = 4096: 201 MB per expert, 128 k chunks per gate/up tile,
    # router ranges at the largest split length
    w = synth.WORKLOADS["qwen3_30b"].replace(name="bf16_large_dims", L=1, N=8, K=2, d=8192, F=4096, S=3, C=3, R=1,
                                             mode=synth.MODE_SPATIO_TEMPORAL)
    run_e2e(w, T=3, tol=2e-2)


@pytest.mark.parametrize("shape", ["single", "grouped"])
def test_bf16_two_thousand_streams(shape):
    # 2048 streams over 16 experts, top-4: ~512 tokens per expert, eight work
    # units each; 2048 cache-step workgroups and 4096 cache words per fill
    w = synth.WORKLOADS["qwen3_30b"].replace(name="bf16_2048_streams", L=1, N=16, K=4, d=64, F=64, S=2048, C=6, R=2,
                                             mode=synth.MODE_SPATIO_TEMPORAL)
    run_e2e(w, T=3, tol=2e-2, ffn_shape=shape)

