"""Runs a synthetic workload through the C ABI: maps a synth.Workload onto a
cmoe_config and binds the device-generated inputs to an Engine."""
from __future__ import annotations

from typing import Optional

from .cmoe import (CMOE_FLAG_FFN_GROUPED, CMOE_FLAG_FFN_SINGLE, CMOE_FLAG_FILL_ON_MAIN, CMOE_FLAG_FILL_ON_SIDE, Engine,
                   make_config)

FFN_SHAPES = {None: 0, "auto": 0, "single": CMOE_FLAG_FFN_SINGLE, "grouped": CMOE_FLAG_FFN_GROUPED}
FILLS = {None: 0, "auto": 0, "main": CMOE_FLAG_FILL_ON_MAIN, "side": CMOE_FLAG_FILL_ON_SIDE}


def config_for(w, C: Optional[int] = None, R: Optional[int] = None, warmup_tokens: int = 0,
               fills: Optional[str] = None, ffn_shape: Optional[str] = None):
    """ffn_shape: None or "auto" (the library's choice), "single" or "grouped".
    fills: where proactive fills run: None or "auto" (the library's choice:
    the side stream for a host pool, else with the demand fill), "main" or
    "side"."""
    flags = FILLS[fills] | FFN_SHAPES[ffn_shape]
    return make_config(w.L, w.N, w.K, w.d, w.F, w.C if C is None else C, w.R if R is None else R, w.S, w.mode,
                       w.dtype, w.pool_kind, warmup_tokens, flags, w.policy, w.lrfu_lambda, w.arena_slots)


def engine_for(w, inputs, C: Optional[int] = None, R: Optional[int] = None, warmup_tokens: int = 0,
               fills: Optional[str] = None, ffn_shape: Optional[str] = None, workspace: bool = True):
    import torch
    cfg = config_for(w, C, R, warmup_tokens, fills=fills, ffn_shape=ffn_shape)
    side = torch.cuda.Stream() if fills != "main" else None
    return Engine(cfg, inputs["wR"], inputs.get("wT"), inputs.get("wS"), inputs.get("bias"), inputs["pool"],
                  side_stream=side, workspace=workspace)
