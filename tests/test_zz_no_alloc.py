"""cmoe_step_noalloc (per-step buffers in the library's static scratch array,
no workspace, no allocation) against cmoe_step (the handle's workspace) on the
same inputs: outputs, logits, selections, gates, caches, events, counters and
slot maps identical, token after token.  Two calls in a row, the second with
fewer streams, so the second runs over what the first left in the scratch
array; a handle that switches between the two entry points; and a
configuration too large for the scratch array, which is refused."""
import numpy as np
import pytest

import synth
from gpu_util import say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

VIEWS = ("LOGITS", "SELECTED", "GATES", "CACHE", "COUNTERS", "PHYS", "SLOTS", "EVENTS", "FILLS", "ACTIVE",
         "SELCOUNT")


def compare(B, ea, eb, ya, yb, where):
    assert np.array_equal(ya.cpu().numpy().view(np.uint32), yb.cpu().numpy().view(np.uint32)), f"{where}: y"
    for v in VIEWS:
        va = ea.cmoe_read(getattr(B, "CMOE_VIEW_" + v))
        vb = eb.cmoe_read(getattr(B, "CMOE_VIEW_" + v))
        assert np.array_equal(va.view(np.uint8), vb.view(np.uint8)), f"{where}: view {v}"
    ta, _, _ = ea.cmoe_stats()
    tb, _, _ = eb.cmoe_stats()
    assert ta == tb, f"{where}: totals"


def small(S, full):
    base = synth.WORKLOADS["gptoss_20b" if full else "qwen3_30b"]
    return base.replace(name=f"noalloc_S{S}", L=3, N=32, K=4, C=8, d=256, F=128, S=S,
                        R=2 if full else 0)


@pytest.mark.parametrize("first,second", [((48, True), (12, False)), ((40, False), (9, True))],
                         ids=["full_then_update_only", "update_only_then_full"])
def test_noalloc_matches_step_two_calls_in_a_row(first, second):
    from paper_2609_04895_amd import cmoe as B
    from paper_2609_04895_amd.workload import engine_for
    for S, full in (first, second):
        w = small(S, full)
        T = 4
        say(f"no-alloc vs step: S={S} full={full} L={w.L} N={w.N} K={w.K} C={w.C} R={w.R}, {T} tokens")
        inp = synth.device_inputs(w, T=T)
        ea = engine_for(w, inp)
        eb = engine_for(w, inp, workspace=False)
        ya = torch.empty((w.S, w.L, w.d), dtype=torch.float32, device="cuda:0")
        yb = torch.full_like(ya, float("nan"))
        for t in range(T):
            ea.cmoe_step(inp["hidden"][t], ya)
            eb.cmoe_step_noalloc(inp["hidden"][t], yb)
            compare(B, ea, eb, ya, yb, f"S={S} token {t}")
        ea.cmoe_destroy()
        eb.cmoe_destroy()


def test_noalloc_with_a_capacity_limited_arena():
    """Six HBM slots per layer for a union of up to 32 experts: the FFN runs
    in rounds, whose plan and work units live in the scratch array too."""
    from paper_2609_04895_amd import cmoe as B
    from paper_2609_04895_amd.workload import engine_for
    w = small(24, True).replace(arena_slots=6)
    T = 4
    inp = synth.device_inputs(w, T=T)
    ea = engine_for(w, inp)
    eb = engine_for(w, inp, workspace=False)
    ya = torch.empty((w.S, w.L, w.d), dtype=torch.float32, device="cuda:0")
    yb = torch.empty_like(ya)
    for t in range(T):
        ea.cmoe_step(inp["hidden"][t], ya)
        eb.cmoe_step_noalloc(inp["hidden"][t], yb)
        compare(B, ea, eb, ya, yb, f"arena of 6 slots, token {t}")
    ea.cmoe_destroy()
    eb.cmoe_destroy()


def test_noalloc_and_step_interleaved_on_one_handle():
    """A handle with a workspace may take either entry point token by token
    (L = 3 is odd, so the bucket buffers change parity between tokens)."""
    from paper_2609_04895_amd import cmoe as B
    from paper_2609_04895_amd.workload import engine_for
    w = small(20, True)
    T = 5
    inp = synth.device_inputs(w, T=T)
    ea = engine_for(w, inp)
    eb = engine_for(w, inp)
    ya = torch.empty((w.S, w.L, w.d), dtype=torch.float32, device="cuda:0")
    yb = torch.empty_like(ya)
    for t in range(T):
        ea.cmoe_step(inp["hidden"][t], ya)
        if t % 2 == 0:
            eb.cmoe_step_noalloc(inp["hidden"][t], yb)
        else:
            eb.cmoe_step(inp["hidden"][t], yb)
        compare(B, ea, eb, ya, yb, f"interleaved token {t}")
    ea.cmoe_destroy()
    eb.cmoe_destroy()


def test_noalloc_refuses_a_configuration_beyond_the_scratch_array():
    from paper_2609_04895_amd import cmoe as B
    # gated expert outputs alone: S K d x 4 bytes = 20000 x 16 x 64 x 4 > 64 MiB
    cfg = B.make_config(1, 16, 16, 64, 64, 16, 0, 20000, B.CMOE_MODE_TEMPORAL, B.CMOE_F32)
    assert B.cmoe_query(cfg).workspace_bytes > 64 << 20
    dev = torch.device("cuda", 0)
    w = torch.zeros((1, 16, 64), dtype=torch.float32, device=dev)
    pool = torch.zeros((1, 16, 3 * 64 * 64), dtype=torch.float32, device=dev)
    with pytest.raises(B.CmoeError) as err:
        B.Engine(cfg, w, w, None, None, pool, workspace=False)
    assert err.value.status == B.CMOE_ERR_UNSUPPORTED
    eng = B.Engine(cfg, w, w, None, None, pool)
    h = torch.zeros((20000, 1, 64), dtype=torch.float32, device=dev)
    y = torch.empty((20000, 1, 64), dtype=torch.float32, device=dev)
    with pytest.raises(B.CmoeError) as err:
        eng.cmoe_step_noalloc(h, y)
    assert err.value.status == B.CMOE_ERR_UNSUPPORTED
    eng.cmoe_destroy()
