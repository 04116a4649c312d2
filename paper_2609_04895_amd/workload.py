"""Runs a synthetic workload through the C ABI: maps a synth.Workload onto a
cmoe_config and binds the device-generated inputs to an Engine."""
from __future__ import annotations

from typing import Optional

from .cmoe import CMOE_FLAG_FFN_GROUPED, CMOE_FLAG_FFN_SINGLE, CMOE_FLAG_FILL_ON_MAIN, Engine, make_config

FFN_SHAPES = {None: 0, "auto": 0, "single": CMOE_FLAG_FFN_SINGLE, "grouped": CMOE_FLAG_FFN_GROUPED}


def config_for(w, C: Optional[int] = None, R: Optional[int] = None, warmup_tokens: int = 0,
               fill_on_main: bool = False, ffn_shape: Optional[str] = None):
    """ffn_shape: None or "auto" (the library's choice), "single" or "grouped"."""
    flags = (CMOE_FLAG_FILL_ON_MAIN if fill_on_main else 0) | FFN_SHAPES[ffn_shape]
    return make_config(w.L, w.N, w.K, w.d, w.F, w.C if C is None else C, w.R if R is None else R, w.S, w.mode,
                       w.dtype, w.pool_kind, warmup_tokens, flags, w.policy, w.lrfu_lambda, w.arena_slots)


def engine_for(w, inputs, C: Optional[int] = None, R: Optional[int] = None, warmup_tokens: int = 0,
               side_stream: bool = True, ffn_shape: Optional[str] = None, workspace: bool = True):
    import torch
    cfg = config_for(w, C, R, warmup_tokens, fill_on_main=not side_stream, ffn_shape=ffn_shape)
    side = torch.cuda.Stream() if side_stream else None
    return Engine(cfg, inputs["wR"], inputs.get("wT"), inputs.get("wS"), inputs.get("bias"), inputs["pool"],
                  side_stream=side, workspace=workspace)
