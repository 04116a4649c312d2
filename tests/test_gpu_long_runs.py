"""Full-size parity over longer token runs than test_gpu_full_size.py, in the
launch configuration bench.py times: caches reach their steady state, the
refinement runs for many tokens, and the Zipf and single-stream workloads
keep issuing physical fills.  Same checks as the full-size tests (logits
within one ulp, decisions and counters bit for bit for the replayed streams,
sampled FFN outputs within the bf16 bound)."""
import pytest

import synth
from test_gpu_full_size import run_full

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,repl,T,seed", [
    ("qwen3_30b", {}, 96, 5),
    ("qwen3_30b_zipf", {"C": 32, "R": 4}, 48, 6),
    ("gptoss_20b", {}, 64, 7),
    ("qwen3_30b_s1", {}, 96, 8),
], ids=["qwen3_30b", "qwen3_30b_zipf", "gptoss_20b", "qwen3_30b_s1"])
def test_long_run_full_size(name, repl, T, seed):
    run_full(synth.WORKLOADS[name].replace(**repl), T=T, ffn_samples=12, seed=seed)


def test_long_run_single_stream_side_stream_fills():
    """One stream with its pool in pinned host memory, every proactive load a
    real copy, the proactive copies on the side stream overlapping the FFN."""
    run_full(synth.WORKLOADS["qwen3_30b_s1"], T=64, ffn_samples=8, seed=9, fills="side")
