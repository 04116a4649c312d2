"""Synthetic workloads of the cache-aware MoE decode step.

Each workload has the layer/expert shapes of one of the paper's backbones
(Qwen3-30B-A3B: 48 MoE layers, 128 experts, top-8; GPT-OSS-20B: 24 layers, 32
experts, top-4; Section 4.1 "Backbone models") or of a larger Qwen3 slice, with
random-init weights N(0, 0.02) and AR(1) hidden states that give temporal
locality.  The paper's datasets (GSM8K, MATH, CommonsenseQA) are replaced by
these seeded synthetic streams; nothing here is taken from those datasets.

Names follow the paper's problem statement (Section 2): L MoE layers, N experts
per layer, native Top-K, per-layer cache capacity C (the paper's B), and the
pre-access refinement budget R (the paper's R, Appendix B.2), S independent
decode streams of T tokens each.
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Tuple

MODE_TEMPORAL = 0          # update-only Temporal Router (Section 3.2)
MODE_SPATIO_TEMPORAL = 1   # full mode with pre-access refinement (Section 3.3)
MODE_SPATIO_ONLY = 2       # Spatio-only ablation (Section 5, Appendix B.4)

POLICY_ROUTER = 0          # retention by the Temporal Router's s^T
POLICY_LRU = 1             # classical cache-update baselines (Section 4.1, Table 1)
POLICY_LFU = 2
POLICY_LRFU = 3

DTYPE_F32 = 0
DTYPE_BF16 = 1

POOL_DEVICE = 0
POOL_HOST_PINNED = 1


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    L: int
    N: int
    K: int
    d: int
    F: int
    C: int
    R: int
    S: int
    T: int
    mode: int
    dtype: int
    rho: float = 0.9
    sigma_w: float = 0.02
    zipf: Optional[float] = None      # exponent of the per-layer popularity bias
    pool_kind: int = POOL_DEVICE
    seed: int = 0
    sweep_C: Tuple[int, ...] = ()
    sweep_R: Tuple[int, ...] = ()
    policy: int = POLICY_ROUTER
    lrfu_lambda: float = 0.5
    arena_slots: int = 0              # HBM expert slots per layer (0: min(N, S C))
    layer0: int = 0                   # model layer of layer 0: a workload of L layers covers layers
                                      # layer0 .. layer0 + L - 1 of the model (their own weights and inputs)

    @property
    def elem_bytes(self) -> int:
        return 2 if self.dtype == DTYPE_BF16 else 4

    @property
    def expert_bytes(self) -> int:
        """Bytes of one expert: W_gate[F][d], W_up[F][d], W_down[d][F]."""
        return 3 * self.d * self.F * self.elem_bytes

    @property
    def has_temporal(self) -> bool:
        return self.policy == POLICY_ROUTER

    @property
    def has_spatio(self) -> bool:
        return self.mode in (MODE_SPATIO_TEMPORAL, MODE_SPATIO_ONLY)

    @property
    def n_routers(self) -> int:
        return 1 + int(self.has_temporal) + int(self.has_spatio)

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS = {
    # Tiny fp32 instance: L=4, N=16, K=2, d=256, SwiGLU 256->512->256, C=6,
    # update-only, 1 stream x 256 tokens, AR(1) rho=0.9, seed 0.
    "tiny": Workload("tiny", L=4, N=16, K=2, d=256, F=512, C=6, R=0, S=1, T=256,
                     mode=MODE_TEMPORAL, dtype=DTYPE_F32, rho=0.9),
    # Qwen3-30B-A3B-shaped bf16 slice, update-only, 64 streams x 512 tokens.
    "qwen3_30b": Workload("qwen3_30b", L=48, N=128, K=8, d=2048, F=768, C=32, R=0, S=64, T=512,
                          mode=MODE_TEMPORAL, dtype=DTYPE_BF16, rho=0.9),
    # GPT-OSS-20B-shaped bf16, full Spatio-Temporal mode, R=2, 64 x 512, rho=0.85.
    "gptoss_20b": Workload("gptoss_20b", L=24, N=32, K=4, d=2880, F=2880, C=8, R=2, S=64, T=512,
                           mode=MODE_SPATIO_TEMPORAL, dtype=DTYPE_BF16, rho=0.85),
    # Qwen3-30B shape in full mode with a Zipf(1.1) popularity bias on the native
    # logits, 256 x 256, swept over C in {16,32,64} and R in {0,2,4}.
    "qwen3_30b_zipf": Workload("qwen3_30b_zipf", L=48, N=128, K=8, d=2048, F=768, C=32, R=2, S=256,
                               T=256, mode=MODE_SPATIO_TEMPORAL, dtype=DTYPE_BF16, rho=0.9, zipf=1.1,
                               sweep_C=(16, 32, 64), sweep_R=(0, 2, 4)),
    # Qwen3-235B-A22B-shaped slice of 16 layers, full mode R=4, cold pool in
    # pinned host memory, 256 x 256.
    "qwen3_235b_slice": Workload("qwen3_235b_slice", L=16, N=128, K=8, d=4096, F=1536, C=32, R=4,
                                 S=256, T=256, mode=MODE_SPATIO_TEMPORAL, dtype=DTYPE_BF16, rho=0.9,
                                 pool_kind=POOL_HOST_PINNED),
    # One decode stream at the Qwen3-30B-A3B shape with the cold pool in
    # pinned host memory: every logical load is a physical copy over the host
    # link (the transfer-overlap study of Appendix B.3).
    "qwen3_30b_s1": Workload("qwen3_30b_s1", L=48, N=128, K=8, d=2048, F=768, C=32, R=4, S=1, T=256,
                             mode=MODE_SPATIO_TEMPORAL, dtype=DTYPE_BF16, rho=0.9, pool_kind=POOL_HOST_PINNED),
}
