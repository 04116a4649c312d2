"""Run-to-run determinism: the same tokens after cmoe_reset give bit-identical
outputs, logits, selections and counters (no float atomics; every sum in a
fixed order; bucket positions from integer atomics do not change results)."""
import numpy as np
import pytest

import synth
from gpu_util import say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def run_tokens(eng, inp, w, T):
    from paper_2609_04895_amd import cmoe as B
    ys, zs, sels = [], [], []
    y = torch.empty((w.S, w.L, w.d), dtype=torch.float32, device="cuda:0")
    for t in range(T):
        eng.cmoe_step(inp["hidden"][t], y)
        torch.cuda.synchronize()
        ys.append(y.cpu().numpy().copy())
        zs.append(eng.cmoe_read(B.CMOE_VIEW_LOGITS).copy())
        sels.append(eng.cmoe_read(B.CMOE_VIEW_SELECTED).copy())
    tot, per, phys = eng.cmoe_stats()
    return ys, zs, sels, tot


@pytest.mark.parametrize("shape", ["single", "grouped"])
def test_repeat_after_reset_is_bit_identical(shape):
    from paper_2609_04895_amd.workload import engine_for
    # Zipf-skewed buckets over several work units, full mode with proactive
    # fills on the side stream
    w = synth.WORKLOADS["qwen3_30b_zipf"].replace(name="determinism", L=3, N=16, K=4, d=256, F=128, S=96, C=6,
                                                  R=2)
    T = 6
    say(f"determinism {shape}")
    inp = synth.device_inputs(w, T=T)
    eng = engine_for(w, inp, ffn_shape=shape)
    a = run_tokens(eng, inp, w, T)
    eng.cmoe_reset()
    b = run_tokens(eng, inp, w, T)
    eng.cmoe_destroy()
    for t in range(T):
        assert np.array_equal(a[0][t].view(np.uint32), b[0][t].view(np.uint32)), f"token {t}: outputs differ"
        assert np.array_equal(a[1][t].view(np.uint32), b[1][t].view(np.uint32)), f"token {t}: logits differ"
        assert np.array_equal(a[2][t], b[2][t]), f"token {t}: selections differ"
    assert a[3] == b[3], "counters differ"
