"""ctypes binding of the CPU oracle (``oracle.c``).

TEST INFRASTRUCTURE: only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  It shares no code
with the GPU path; see ``oracle.c`` for what it computes and where the paper
defines each step.

Every function here is marshalling only; the arithmetic is in ``oracle.c``.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# ORACLE_LIBRARY lets the planted-mistake tests load a deliberately broken
# build of oracle.c; nothing else sets it.
LIB_PATH = os.environ.get("ORACLE_LIBRARY") or os.path.join(_HERE, "liboracle.so")

NCTR = 5  # A, hits, D, P, T
MODE_TEMPORAL, MODE_SPATIO_TEMPORAL, MODE_SPATIO_ONLY = 0, 1, 2
POLICY_ROUTER, POLICY_LRU, POLICY_LFU, POLICY_LRFU = 0, 1, 2, 3
CTR_A, CTR_HITS, CTR_D, CTR_P, CTR_T = range(NCTR)

_i32p = ctypes.POINTER(ctypes.c_int32)
_i64p = ctypes.POINTER(ctypes.c_int64)
_u8p = ctypes.POINTER(ctypes.c_uint8)
_f32p = ctypes.POINTER(ctypes.c_float)
_f64p = ctypes.POINTER(ctypes.c_double)


class _Cfg(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("L", "N", "K", "C", "R", "S", "mode", "warmup_tokens", "policy")] + \
        [("lrfu_w", ctypes.c_float)]


class _State(ctypes.Structure):
    _fields_ = [("cache", _u8p), ("aT", _f32p), ("pS", _f32p), ("ctr", _i64p), ("slot_of", _i32p),
                ("phys", _i64p), ("pol", _f32p), ("selcount", _i64p), ("stamp", _i64p), ("clk", _i64p),
                ("n_slots", ctypes.c_int32),
                ("t", ctypes.c_int32)]


class _Out(ctypes.Structure):
    _fields_ = [("sel", _i32p), ("gate", _f64p), ("pR", _f32p), ("sT", _f32p), ("sST", _f32p),
                ("hits", _i32p), ("nD", _i32p), ("nP", _i32p), ("fills", _i32p)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run oracle.build.build()")
        L = ctypes.CDLL(LIB_PATH)
        L.orc_exp.argtypes = [ctypes.c_float]
        L.orc_exp.restype = ctypes.c_float
        L.orc_exp_constants.argtypes = [_f32p]
        L.orc_softmax.argtypes = [_f32p, ctypes.c_int, _f32p]
        L.orc_topk.argtypes = [_f32p, ctypes.c_int, ctypes.c_int, _i32p]
        L.orc_update_cache.argtypes = [_u8p, ctypes.c_int, ctypes.c_int, _i32p, ctypes.c_int, _f32p, _i32p]
        L.orc_update_cache.restype = ctypes.c_int
        L.orc_refine.argtypes = [_u8p, ctypes.c_int, ctypes.c_int, _f32p, ctypes.c_int, _i32p]
        L.orc_refine.restype = ctypes.c_int
        L.orc_logits.argtypes = [_f32p, _f32p, _f32p, ctypes.c_int, ctypes.c_int, _f32p]
        L.orc_moe_ffn.argtypes = [_f32p, _f32p, _f32p, _f64p, ctypes.c_int, _f32p, ctypes.c_int,
                                  ctypes.c_int, _f64p]
        L.orc_metrics.argtypes = [ctypes.c_int64] * 4 + [ctypes.c_double, _f64p]
        L.orc_concentration.argtypes = [_i64p, ctypes.c_int, ctypes.c_int, ctypes.c_int, _f64p]
        L.orc_concentration.restype = ctypes.c_int
        L.orc_lrfu_weight.argtypes = [ctypes.c_float]
        L.orc_lrfu_weight.restype = ctypes.c_float
        L.orc_step.argtypes = [ctypes.POINTER(_Cfg), ctypes.POINTER(_State), _f32p, _f32p, _f32p,
                               ctypes.POINTER(_Out)]
        L.orc_step.restype = ctypes.c_int
        _lib = L
    return _lib


def _p(a: Optional[np.ndarray], t):
    if a is None:
        return ctypes.cast(None, t)
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(t)


# ---------------------------------------------------------------- primitives
def exp(x) -> np.ndarray:
    x = np.asarray(x, dtype=np.float32).ravel()
    f = lib().orc_exp
    return np.array([f(float(v)) for v in x], dtype=np.float32)


def exp_constants() -> np.ndarray:
    out = np.zeros(11, dtype=np.float32)
    lib().orc_exp_constants(_p(out, _f32p))
    return out


def softmax(z) -> np.ndarray:
    z = np.ascontiguousarray(z, dtype=np.float32)
    p = np.empty_like(z)
    lib().orc_softmax(_p(z, _f32p), z.size, _p(p, _f32p))
    return p


def topk(v, k: int) -> np.ndarray:
    v = np.ascontiguousarray(v, dtype=np.float32)
    out = np.empty(k, dtype=np.int32)
    lib().orc_topk(_p(v, _f32p), v.size, k, _p(out, _i32p))
    return out


def update_cache(cache, selected, score, cap: int):
    """Algorithm 1.  cache: bool/uint8 [N].  Returns (new cache, demand list)."""
    c = np.ascontiguousarray(cache, dtype=np.uint8).copy()
    sel = np.ascontiguousarray(selected, dtype=np.int32)
    s = np.ascontiguousarray(score, dtype=np.float32)
    dem = np.empty(max(1, sel.size), dtype=np.int32)
    n = lib().orc_update_cache(_p(c, _u8p), c.size, cap, _p(sel, _i32p), sel.size, _p(s, _f32p),
                               _p(dem, _i32p))
    return c, dem[:n].copy()


def refine(cache, score, R: int, cap: int):
    """Algorithm 2 refinement.  Returns (new cache, proactively loaded list)."""
    c = np.ascontiguousarray(cache, dtype=np.uint8).copy()
    s = np.ascontiguousarray(score, dtype=np.float32)
    loaded = np.empty(max(1, c.size), dtype=np.int32)
    n = lib().orc_refine(_p(c, _u8p), c.size, cap, _p(s, _f32p), R, _p(loaded, _i32p))
    return c, loaded[:n].copy()


def logits(W, h, bias=None) -> np.ndarray:
    """W: [N][d] float32, h: [d] -> fp32 logits (fp64 accumulation)."""
    W = np.ascontiguousarray(W, dtype=np.float32)
    h = np.ascontiguousarray(h, dtype=np.float32)
    b = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
    N, d = W.shape
    z = np.empty(N, dtype=np.float32)
    lib().orc_logits(_p(W, _f32p), _p(h, _f32p), _p(b, _f32p), N, d, _p(z, _f32p))
    return z


def logits_batch(W, H, bias=None) -> np.ndarray:
    """W: [N][d], H: [M][d] -> [M][N]."""
    return np.stack([logits(W, h, bias) for h in np.asarray(H)])


def moe_ffn(Wg, Wu, Wd, gates, x) -> np.ndarray:
    """Wg, Wu: [K][F][d]; Wd: [K][d][F]; gates [K]; x [d] -> y [d] in fp64."""
    Wg = np.ascontiguousarray(Wg, dtype=np.float32)
    Wu = np.ascontiguousarray(Wu, dtype=np.float32)
    Wd = np.ascontiguousarray(Wd, dtype=np.float32)
    g = np.ascontiguousarray(gates, dtype=np.float64)
    x = np.ascontiguousarray(x, dtype=np.float32)
    K, F, d = Wg.shape
    y = np.empty(d, dtype=np.float64)
    lib().orc_moe_ffn(_p(Wg, _f32p), _p(Wu, _f32p), _p(Wd, _f32p), _p(g, _f64p), K, _p(x, _f32p), d, F,
                      _p(y, _f64p))
    return y


def concentration(counts, top_m: int = 8):
    """Per-layer expert-use concentration of selection counts [L][N], averaged
    over layers: (effective experts exp(H), entropy H in nats, max frequency,
    top-m mass)."""
    c = np.ascontiguousarray(counts, dtype=np.int64)
    if c.ndim == 1:
        c = c[None]
    out = np.zeros(4, dtype=np.float64)
    lib().orc_concentration(_p(c, _i64p), c.shape[0], c.shape[1], int(top_m), _p(out, _f64p))
    return tuple(float(v) for v in out)


def metrics(A: int, D: int, P: int, T: int, expert_bytes: float):
    """(Hit, AdjHit, Load in MB per decode token)."""
    out = np.zeros(3, dtype=np.float64)
    lib().orc_metrics(int(A), int(D), int(P), int(T), float(expert_bytes), _p(out, _f64p))
    return float(out[0]), float(out[1]), float(out[2])


# ---------------------------------------------------------------- replay
def lrfu_weight(lam: float) -> float:
    """LRFU decay per token, fl32(2^-lambda)."""
    return float(lib().orc_lrfu_weight(float(lam)))


class Run:
    """State of all S streams; ``step`` advances one decode token.

    mode: MODE_TEMPORAL (update-only), MODE_SPATIO_TEMPORAL (full) or
    MODE_SPATIO_ONLY; policy: POLICY_ROUTER (s^T) or a classical retention
    priority (LRU, LFU, LRFU with ``lrfu_lambda``); arena_slots: physical
    slots per layer (0: min(N, S C), which always holds the union of the
    caches)."""

    def __init__(self, L, N, K, C, R, S, mode, warmup_tokens=0, policy=POLICY_ROUTER, lrfu_lambda=0.5,
                 arena_slots=0):
        self.cfg = _Cfg(L, N, K, C, R, S, mode, warmup_tokens, policy, lrfu_weight(lrfu_lambda))
        self.L, self.N, self.K, self.C, self.S, self.mode = L, N, K, C, S, mode
        self.policy = policy
        self.pol = np.zeros((S, L, N), dtype=np.float32)
        self.selcount = np.zeros((L, N), dtype=np.int64)
        self.cache = np.zeros((S, L, N), dtype=np.uint8)
        self.aT = np.zeros((S, L, N), dtype=np.float32)
        self.pS = np.zeros((S, N), dtype=np.float32)
        self.ctr = np.zeros((S, L, NCTR), dtype=np.int64)
        self.slot_of = np.full((L, N), -1, dtype=np.int32)
        self.phys = np.zeros((L, 2), dtype=np.int64)
        self.stamp = np.zeros((L, N), dtype=np.int64)
        self.clk = np.zeros(L, dtype=np.int64)
        self.n_slots = arena_slots if arena_slots else min(N, S * C)
        self.t = 0

    @property
    def R(self):
        return self.cfg.R

    def set_R(self, R: int):
        self.cfg.R = R

    def _state(self):
        return _State(_p(self.cache, _u8p), _p(self.aT, _f32p), _p(self.pS, _f32p), _p(self.ctr, _i64p),
                      _p(self.slot_of, _i32p), _p(self.phys, _i64p), _p(self.pol, _f32p), _p(self.selcount, _i64p),
                      _p(self.stamp, _i64p), _p(self.clk, _i64p), self.n_slots, self.t)

    def step(self, zR, zT=None, zS=None, want=("sel", "gate")):
        """zR, zT, zS: [S][L][N] float32 (zT only for the router policy in the
        Temporal / Spatio-Temporal modes, zS only in modes with a Spatio
        Router).  Returns a dict of per-token outputs."""
        S, L, N, K = self.S, self.L, self.N, self.K
        zR = np.ascontiguousarray(zR, dtype=np.float32).reshape(S, L, N)
        if self.policy == POLICY_ROUTER and zT is None:
            raise ValueError("the router policy needs Temporal Router logits")
        if self.mode in (MODE_SPATIO_TEMPORAL, MODE_SPATIO_ONLY) and zS is None:
            raise ValueError("this mode needs Spatio Router logits")
        zT = zR if zT is None else np.ascontiguousarray(zT, dtype=np.float32).reshape(S, L, N)
        zSa = zR if zS is None else np.ascontiguousarray(zS, dtype=np.float32).reshape(S, L, N)
        res = {
            "sel": np.zeros((S, L, K), np.int32), "gate": np.zeros((S, L, K), np.float64),
            "pR": np.zeros((S, L, N), np.float32), "sT": np.zeros((S, L, N), np.float32),
            "sST": np.zeros((S, L, N), np.float32), "hits": np.zeros((S, L), np.int32),
            "nD": np.zeros((S, L), np.int32), "nP": np.zeros((S, L), np.int32),
            "fills": np.zeros((L, 2), np.int32),
        }
        types = {"sel": _i32p, "gate": _f64p, "pR": _f32p, "sT": _f32p, "sST": _f32p, "hits": _i32p,
                 "nD": _i32p, "nP": _i32p, "fills": _i32p}
        out = _Out(*[_p(res[n], types[n]) if (n in want or want == "all") else ctypes.cast(None, types[n])
                     for n, _ in _Out._fields_])
        st = self._state()
        rc = lib().orc_step(ctypes.byref(self.cfg), ctypes.byref(st), _p(zR, _f32p), _p(zT, _f32p),
                            _p(zSa, _f32p), ctypes.byref(out))
        if rc != 0:
            raise RuntimeError("oracle invariant broken (hits + misses != K or |C| > capacity)")
        self.t = st.t
        return {n: v for n, v in res.items() if (n in want or want == "all")}

    def totals(self):
        c = self.ctr.sum(axis=(0, 1))
        return {"accesses": int(c[CTR_A]), "hits": int(c[CTR_HITS]), "demand_misses": int(c[CTR_D]),
                "proactive_loads": int(c[CTR_P]), "tokens": int(self.ctr[:, 0, CTR_T].sum()),
                "phys_fills": int(self.phys.sum())}
