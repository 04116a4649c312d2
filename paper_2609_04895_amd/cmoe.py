"""ctypes binding of libcmoe.so; the names are those of include/cmoe.h.

Argument marshalling only: every step of the decode path runs in the HIP
kernels behind the C ABI.  ``Engine`` is a convenience owner of the buffers the
library asks for (allocated with PyTorch, which serves here only as the device
memory and stream provider).
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcmoe.so")

CMOE_OK = 0
CMOE_ERR_INVALID_ARG = -1
CMOE_ERR_UNSUPPORTED = -2
CMOE_ERR_HIP = -3
CMOE_ERR_STATE = -4

CMOE_MODE_TEMPORAL = 0
CMOE_MODE_SPATIO_TEMPORAL = 1
CMOE_MODE_SPATIO_ONLY = 2
CMOE_POLICY_ROUTER = 0
CMOE_POLICY_LRU = 1
CMOE_POLICY_LFU = 2
CMOE_POLICY_LRFU = 3
CMOE_F32 = 0
CMOE_BF16 = 1
CMOE_POOL_DEVICE = 0
CMOE_POOL_HOST_PINNED = 1
CMOE_FLAG_FILL_ON_MAIN = 0x1
CMOE_FLAG_FFN_GROUPED = 0x2
CMOE_FLAG_FFN_SINGLE = 0x4
CMOE_FLAG_FILL_ON_SIDE = 0x8

CMOE_VIEW_LOGITS = 0
CMOE_VIEW_SELECTED = 1
CMOE_VIEW_GATES = 2
CMOE_VIEW_CACHE = 3
CMOE_VIEW_COUNTERS = 4
CMOE_VIEW_PHYS = 5
CMOE_VIEW_SLOTS = 6
CMOE_VIEW_EVENTS = 7
CMOE_VIEW_FILLS = 8
CMOE_VIEW_ACTIVE = 9
CMOE_VIEW_PRIORITY = 10
CMOE_VIEW_SELCOUNT = 11
CMOE_KERNEL_COUNT = 6
KERNEL_NAMES = ("router", "cache_step", "fill", "ffn_up", "ffn_down", "combine")

EXPORTED = ("cmoe_query", "cmoe_init", "cmoe_step", "cmoe_step_noalloc", "cmoe_step_logits", "cmoe_stats", "cmoe_get_cache",
            "cmoe_set_cache", "cmoe_set_R", "cmoe_reset", "cmoe_destroy", "cmoe_view_bytes", "cmoe_read",
            "cmoe_profile_begin", "cmoe_profile_end", "cmoe_concentration", "cmoe_read_probe", "cmoe_last_error")


class cmoe_config(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("L", "N", "K", "d", "F", "C", "R", "S", "mode", "dtype",
                                              "pool_kind", "warmup_tokens")] + \
        [("flags", ctypes.c_uint32), ("policy", ctypes.c_int32), ("lrfu_lambda", ctypes.c_float),
         ("arena_slots", ctypes.c_int32)]


class cmoe_weights(ctypes.Structure):
    _fields_ = [("w_router", ctypes.c_void_p), ("w_temporal", ctypes.c_void_p), ("w_spatio", ctypes.c_void_p),
                ("logit_bias", ctypes.c_void_p), ("cold_pool", ctypes.c_void_p)]


class cmoe_sizes(ctypes.Structure):
    _fields_ = [("arena_bytes", ctypes.c_size_t), ("state_bytes", ctypes.c_size_t),
                ("workspace_bytes", ctypes.c_size_t)]


class cmoe_buffers(ctypes.Structure):
    _fields_ = [("arena", ctypes.c_void_p), ("state", ctypes.c_void_p), ("workspace", ctypes.c_void_p)]


class cmoe_stats_t(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in ("accesses", "hits", "demand_misses", "proactive_loads", "tokens",
                                              "traffic_bytes", "phys_fills", "phys_bytes")]

    def as_dict(self):
        return {n: int(getattr(self, n)) for n, _ in self._fields_}


class CmoeError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"cmoe status {status}: {msg}")
        self.status = status


_lib = None


def lib():
    """Loads libcmoe.so; raises if it has not been built (there is no fallback)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with paper_2609_04895_amd.build.build()")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64p = ctypes.c_void_p, ctypes.c_int32, ctypes.POINTER(ctypes.c_int64)
        L.cmoe_query.argtypes = [ctypes.POINTER(cmoe_config), ctypes.POINTER(cmoe_sizes)]
        L.cmoe_init.argtypes = [ctypes.POINTER(cmoe_config), ctypes.POINTER(cmoe_weights),
                                ctypes.POINTER(cmoe_buffers), vp, vp, ctypes.POINTER(vp)]
        L.cmoe_step.argtypes = [vp, vp, vp]
        L.cmoe_step_noalloc.argtypes = [vp, vp, vp]
        L.cmoe_step_logits.argtypes = [vp, vp, vp, vp]
        L.cmoe_stats.argtypes = [vp, ctypes.POINTER(cmoe_stats_t), i64p, i64p]
        L.cmoe_get_cache.argtypes = [vp, i32, i32, ctypes.POINTER(i32), ctypes.POINTER(i32)]
        L.cmoe_set_cache.argtypes = [vp, i32, i32, ctypes.POINTER(i32), i32]
        L.cmoe_set_R.argtypes = [vp, i32]
        L.cmoe_reset.argtypes = [vp]
        L.cmoe_destroy.argtypes = [vp]
        L.cmoe_view_bytes.argtypes = [vp, i32]
        L.cmoe_view_bytes.restype = ctypes.c_size_t
        L.cmoe_read.argtypes = [vp, i32, vp, ctypes.c_size_t]
        L.cmoe_profile_begin.argtypes = [vp, i32, ctypes.c_uint32]
        L.cmoe_profile_end.argtypes = [vp, ctypes.POINTER(ctypes.c_double), i64p]
        L.cmoe_concentration.argtypes = [vp, i32, ctypes.POINTER(ctypes.c_double)]
        L.cmoe_read_probe.argtypes = [vp, ctypes.c_int64, i32, ctypes.POINTER(ctypes.c_double)]
        L.cmoe_last_error.argtypes = []
        L.cmoe_last_error.restype = ctypes.c_char_p
        for n in EXPORTED:
            if n not in ("cmoe_view_bytes", "cmoe_last_error"):
                getattr(L, n).restype = ctypes.c_int
        _lib = L
    return _lib


def _check(status: int):
    if status != CMOE_OK:
        raise CmoeError(status, lib().cmoe_last_error().decode())


def make_config(L, N, K, d, F, C, R, S, mode, dtype, pool_kind=CMOE_POOL_DEVICE, warmup_tokens=0, flags=0,
                policy=CMOE_POLICY_ROUTER, lrfu_lambda=0.5, arena_slots=0):
    return cmoe_config(L, N, K, d, F, C, R, S, mode, dtype, pool_kind, warmup_tokens, flags, policy, lrfu_lambda,
                       arena_slots)


def router_slots(cfg: cmoe_config):
    """Names of the router slots of the logits view, in order."""
    names = ["native"]
    if cfg.policy == CMOE_POLICY_ROUTER:
        names.append("temporal")
    if cfg.mode in (CMOE_MODE_SPATIO_TEMPORAL, CMOE_MODE_SPATIO_ONLY):
        names.append("spatio")
    return names


def cmoe_query(cfg: cmoe_config) -> cmoe_sizes:
    out = cmoe_sizes()
    _check(lib().cmoe_query(ctypes.byref(cfg), ctypes.byref(out)))
    return out


def cmoe_read_probe(buf, reps: int = 5) -> float:
    """GB/s of the device's streaming read of the device tensor buf (at
    least 64 MiB) with the expert weight loads' access pattern."""
    rate = ctypes.c_double()
    _check(lib().cmoe_read_probe(ctypes.c_void_p(buf.data_ptr()), buf.numel() * buf.element_size(), reps,
                                 ctypes.byref(rate)))
    return rate.value


def _ptr(t) -> Optional[int]:
    return None if t is None else int(t.data_ptr())


class Engine:
    """One handle plus the caller-owned buffers (torch tensors on cuda:0)."""

    def __init__(self, cfg: cmoe_config, w_router, w_temporal, w_spatio, logit_bias, cold_pool,
                 main_stream=None, side_stream=None, workspace=True):
        """workspace=False binds no workspace: every token then goes through
        cmoe_step_noalloc."""
        import torch
        self.torch = torch
        self.cfg = cfg
        sizes = cmoe_query(cfg)
        dev = torch.device("cuda", torch.cuda.current_device())

        def buf(n):
            # 256-byte aligned (the caching allocator aligns blocks to >= 512 bytes)
            return torch.empty(max(int(n), 256), dtype=torch.uint8, device=dev)

        self.arena = buf(sizes.arena_bytes)
        self.state = buf(sizes.state_bytes)
        self.workspace = buf(sizes.workspace_bytes) if workspace else None
        self._keep = (w_router, w_temporal, w_spatio, logit_bias, cold_pool)
        self.main_stream = main_stream if main_stream is not None else torch.cuda.current_stream()
        self.side_stream = side_stream
        wts = cmoe_weights(_ptr(w_router), _ptr(w_temporal), _ptr(w_spatio), _ptr(logit_bias), _ptr(cold_pool))
        bufs = cmoe_buffers(_ptr(self.arena), _ptr(self.state), _ptr(self.workspace) if workspace else None)
        h = ctypes.c_void_p()
        _check(lib().cmoe_init(ctypes.byref(cfg), ctypes.byref(wts), ctypes.byref(bufs),
                               ctypes.c_void_p(self.main_stream.cuda_stream),
                               ctypes.c_void_p(side_stream.cuda_stream if side_stream is not None else None),
                               ctypes.byref(h)))
        self.handle = h

    # -- the decode path
    def cmoe_step(self, h, y):
        _check(lib().cmoe_step(self.handle, ctypes.c_void_p(h.data_ptr()), ctypes.c_void_p(y.data_ptr())))

    def cmoe_step_noalloc(self, h, y):
        _check(lib().cmoe_step_noalloc(self.handle, ctypes.c_void_p(h.data_ptr()), ctypes.c_void_p(y.data_ptr())))

    def cmoe_step_logits(self, zR, zT=None, zS=None):
        _check(lib().cmoe_step_logits(self.handle, ctypes.c_void_p(zR.data_ptr()), ctypes.c_void_p(_ptr(zT)),
                                      ctypes.c_void_p(_ptr(zS))))

    # -- counters and state
    def cmoe_stats(self):
        c = self.cfg
        total = cmoe_stats_t()
        per = np.zeros((c.S, c.L, 5), np.int64)
        phys = np.zeros((c.L, 2), np.int64)
        _check(lib().cmoe_stats(self.handle, ctypes.byref(total), per.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                                phys.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))))
        return total.as_dict(), per, phys

    def cmoe_get_cache(self, stream: int, layer: int):
        out = (ctypes.c_int32 * self.cfg.C)()
        n = ctypes.c_int32()
        _check(lib().cmoe_get_cache(self.handle, stream, layer, out, ctypes.byref(n)))
        return [int(out[i]) for i in range(n.value)]

    def cmoe_set_cache(self, stream: int, layer: int, experts):
        arr = (ctypes.c_int32 * max(1, len(experts)))(*experts)
        _check(lib().cmoe_set_cache(self.handle, stream, layer, arr, len(experts)))

    def cmoe_set_R(self, R: int):
        _check(lib().cmoe_set_R(self.handle, R))

    def cmoe_reset(self):
        _check(lib().cmoe_reset(self.handle))

    def cmoe_read(self, view: int) -> np.ndarray:
        c = self.cfg
        n = lib().cmoe_view_bytes(self.handle, view)
        raw = np.empty(n, np.uint8)
        _check(lib().cmoe_read(self.handle, view, raw.ctypes.data_as(ctypes.c_void_p), n))
        n_r = len(router_slots(c))
        NW = (c.N + 63) // 64
        shapes = {
            CMOE_VIEW_LOGITS: (np.float32, (c.L, c.S, n_r, c.N)),
            CMOE_VIEW_SELECTED: (np.int32, (c.L, c.S, c.K)),
            CMOE_VIEW_GATES: (np.float32, (c.L, c.S, c.K)),
            CMOE_VIEW_CACHE: (np.uint64, (c.S, c.L, NW)),
            CMOE_VIEW_COUNTERS: (np.int64, (c.S, c.L, 5)),
            CMOE_VIEW_PHYS: (np.int64, (c.L, 2)),
            CMOE_VIEW_SLOTS: (np.int32, (c.L, c.N)),
            CMOE_VIEW_EVENTS: (np.int32, (c.L, c.S, 4)),
            CMOE_VIEW_FILLS: (np.int32, (c.L, 2)),
            CMOE_VIEW_ACTIVE: (np.int64, (c.L,)),
            CMOE_VIEW_PRIORITY: (np.float32, (c.S, c.L, c.N)),
            CMOE_VIEW_SELCOUNT: (np.uint64, (c.L, c.N)),
        }
        dt, shape = shapes[view]
        return raw.view(dt).reshape(shape)

    def cmoe_concentration(self, top_m: int = 8):
        """(effective experts, entropy in nats, max frequency, top-m mass),
        layer means of the native selection frequencies."""
        out = (ctypes.c_double * 4)()
        _check(lib().cmoe_concentration(self.handle, int(top_m), out))
        return tuple(float(v) for v in out)

    def cache_sets(self) -> np.ndarray:
        """Cache membership as a bool array [S][L][N]."""
        w = self.cmoe_read(CMOE_VIEW_CACHE)
        c = self.cfg
        bits = np.unpackbits(w.view(np.uint8).reshape(c.S, c.L, -1), axis=-1, bitorder="little")
        return bits[:, :, :c.N].astype(bool)

    # -- timing
    def cmoe_profile_begin(self, max_tokens: int, kernels=None):
        mask = 0 if kernels is None else sum(1 << KERNEL_NAMES.index(k) for k in kernels)
        _check(lib().cmoe_profile_begin(self.handle, max_tokens, mask))

    def cmoe_profile_end(self):
        ms = (ctypes.c_double * CMOE_KERNEL_COUNT)()
        n = (ctypes.c_int64 * CMOE_KERNEL_COUNT)()
        _check(lib().cmoe_profile_end(self.handle, ms, n))
        return {KERNEL_NAMES[i]: (float(ms[i]), int(n[i])) for i in range(CMOE_KERNEL_COUNT)}

    def cmoe_destroy(self):
        if self.handle is not None:
            _check(lib().cmoe_destroy(self.handle))
            self.handle = None

    def __del__(self):
        try:
            self.cmoe_destroy()
        except Exception:
            pass
