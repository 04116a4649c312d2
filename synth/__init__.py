"""Seeded synthetic inputs for the cache-aware MoE decode step.

This package is the only code shared by the oracle side and the GPU side of
the tests: it generates inputs and holds none of the method's arithmetic.  The
generator is defined in ``csrc/synth_cpu.c`` and implemented twice, once for
the host (``libsynth_cpu.so``) and once for the GPU (``libsynth_hip.so``); both
give bit-identical tensors.

Tensor identities (the ``tid`` fed to the counter-based generator):
  router weights  (kind << 56) + l, kind 1 = native W^R, 2 = temporal W^T,
                  3 = spatio W^S; tensor [N][d], element e*d + j
  expert weights  (4 << 56) + l*N + e; tensor W_gate[F][d] ++ W_up[F][d] ++
                  W_down[d][F] (the expert's bytes in the cold pool)
  hidden states   (5 << 56) + (s << 24) + l; innovation of token t, lane j is
                  element t*d + j
  Zipf ranks      (6 << 56) + l; Fisher-Yates draws
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional, Tuple

import numpy as np

from .workloads import (DTYPE_BF16, DTYPE_F32, MODE_SPATIO_ONLY, MODE_SPATIO_TEMPORAL,  # noqa: F401
                        MODE_TEMPORAL, POLICY_LFU, POLICY_LRFU, POLICY_LRU, POLICY_ROUTER, POOL_DEVICE,
                        POOL_HOST_PINNED, WORKLOADS, Workload)

_HERE = os.path.dirname(os.path.abspath(__file__))
CPU_LIB = os.path.join(_HERE, "libsynth_cpu.so")
HIP_LIB = os.path.join(_HERE, "libsynth_hip.so")

KIND_ROUTER_NATIVE = 1
KIND_ROUTER_TEMPORAL = 2
KIND_ROUTER_SPATIO = 3
KIND_EXPERT = 4
KIND_HIDDEN = 5
KIND_ZIPF = 6

_cpu = None
_hip = None


def _load_cpu():
    global _cpu
    if _cpu is None:
        if not os.path.exists(CPU_LIB):
            raise RuntimeError(f"{CPU_LIB} is not built; run synth.build.build()")
        lib = ctypes.CDLL(CPU_LIB)
        u64, i64, i32 = ctypes.c_uint64, ctypes.c_int64, ctypes.c_int32
        fp = ctypes.POINTER(ctypes.c_float)
        lib.syn_key.argtypes = [u64, u64]
        lib.syn_key.restype = u64
        lib.syn_draw.argtypes = [u64, u64]
        lib.syn_draw.restype = u64
        lib.syn_normal_f32.argtypes = [u64, u64, i64, ctypes.c_double, ctypes.c_int, fp]
        lib.syn_normal_f32.restype = None
        lib.syn_normal_bf16.argtypes = [u64, u64, i64, ctypes.c_double, ctypes.POINTER(ctypes.c_uint16)]
        lib.syn_normal_bf16.restype = None
        lib.syn_ar1_f32.argtypes = [u64, i32, i32, ctypes.c_float, ctypes.c_float, ctypes.c_double,
                                    ctypes.c_int, fp]
        lib.syn_ar1_f32.restype = None
        lib.syn_fnv1a.argtypes = [ctypes.c_void_p, i64, u64]
        lib.syn_fnv1a.restype = u64
        _cpu = lib
    return _cpu


def _load_hip():
    global _hip
    if _hip is None:
        if not os.path.exists(HIP_LIB):
            raise RuntimeError(f"{HIP_LIB} is not built; run synth.build.build()")
        lib = ctypes.CDLL(HIP_LIB)
        u64, i64, i32 = ctypes.c_uint64, ctypes.c_int64, ctypes.c_int32
        lib.syn_dev_fill.argtypes = [u64, u64, u64, i64, i64, ctypes.c_double, ctypes.c_int,
                                     ctypes.c_void_p, ctypes.c_void_p]
        lib.syn_dev_fill.restype = ctypes.c_int
        lib.syn_dev_ar1.argtypes = [u64, u64, u64, u64, i32, i32, i32, i32, ctypes.c_float,
                                    ctypes.c_float, ctypes.c_double, ctypes.c_int, ctypes.c_void_p,
                                    ctypes.c_void_p]
        lib.syn_dev_ar1.restype = ctypes.c_int
        lib.syn_host_alloc.argtypes = [i64, ctypes.POINTER(ctypes.c_void_p)]
        lib.syn_host_alloc.restype = ctypes.c_int
        lib.syn_host_free.argtypes = [ctypes.c_void_p]
        lib.syn_host_free.restype = ctypes.c_int
        _hip = lib
    return _hip


# ---------------------------------------------------------------- parameters
def weight_scale(w: Workload) -> float:
    """fp64 factor that maps the centred Irwin-Hall integer to N(0, sigma_w)."""
    return w.sigma_w * math.sqrt(3.0) / 65536.0


def unit_scale() -> float:
    return math.sqrt(3.0) / 65536.0


def ar1_params(w: Workload) -> Tuple[float, float]:
    """(rho, c0) as fp32 values: h_0 = e_0 * c0 with c0 = 1/sqrt(1 - rho^2)."""
    rho32 = float(np.float32(w.rho))
    c0 = float(np.float32(1.0 / math.sqrt(1.0 - rho32 * rho32)))
    return rho32, c0


def router_tid(kind: int, layer: int) -> int:
    return (int(kind) << 56) + int(layer)


def expert_tid(w: Workload, layer: int, expert: int) -> int:
    # Python ints throughout: numpy integer indices would overflow in 64-bit ids
    return (KIND_EXPERT << 56) + int(layer) * w.N + int(expert)


def hidden_tid(stream: int, layer: int) -> int:
    return (KIND_HIDDEN << 56) + (int(stream) << 24) + int(layer)


# ---------------------------------------------------------------- host twin
def _f32_ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_float))


def normal_host(seed: int, tid: int, n: int, scale: float, bf16: bool, first: int = 0) -> np.ndarray:
    lib = _load_cpu()
    out = np.empty(n, dtype=np.float32)
    lib.syn_normal_f32(lib.syn_key(seed, tid), first, n, scale, int(bf16), _f32_ptr(out))
    return out


def normal_host_bf16_bits(seed: int, tid: int, n: int, scale: float) -> np.ndarray:
    lib = _load_cpu()
    out = np.empty(n, dtype=np.uint16)
    lib.syn_normal_bf16(lib.syn_key(seed, tid), 0, n, scale,
                        out.ctypes.data_as(ctypes.POINTER(ctypes.c_uint16)))
    return out


def router_host(w: Workload, kind: int, layer: int) -> np.ndarray:
    """Router weights of one layer as stored values, float32 [N][d]."""
    v = normal_host(w.seed, router_tid(kind, w.layer0 + layer), w.N * w.d, weight_scale(w), w.dtype == DTYPE_BF16)
    return v.reshape(w.N, w.d)


def expert_host(w: Workload, layer: int, expert: int):
    """(W_gate[F][d], W_up[F][d], W_down[d][F]) of one expert as float32."""
    fd = w.F * w.d
    v = normal_host(w.seed, expert_tid(w, w.layer0 + layer, expert), 3 * fd, weight_scale(w),
                    w.dtype == DTYPE_BF16)
    return v[:fd].reshape(w.F, w.d), v[fd:2 * fd].reshape(w.F, w.d), v[2 * fd:].reshape(w.d, w.F)


def hidden_host(w: Workload, stream: int, layer: int, T: Optional[int] = None) -> np.ndarray:
    """AR(1) hidden states h_{t,l} of one stream, float32 [T][d] (stored values)."""
    lib = _load_cpu()
    T = w.T if T is None else T
    rho, c0 = ar1_params(w)
    out = np.empty(T * w.d, dtype=np.float32)
    lib.syn_ar1_f32(lib.syn_key(w.seed, hidden_tid(stream, w.layer0 + layer)), T, w.d, rho, c0, unit_scale(),
                    int(w.dtype == DTYPE_BF16), _f32_ptr(out))
    return out.reshape(T, w.d)


def zipf_bias(w: Workload) -> Optional[np.ndarray]:
    """Per-layer popularity bias [L][N] float32 added to the native logits.

    For each layer a seeded Fisher-Yates permutation assigns ranks r = 1..N to
    the experts; the bias is -a * ln(r) with a the Zipf exponent, so that the
    softmax weight of an expert is scaled by r^-a.  Computed once on the host
    in fp64 and handed to both sides as an input array.
    """
    if w.zipf is None:
        return None
    lib = _load_cpu()
    out = np.empty((w.L, w.N), dtype=np.float32)
    for l in range(w.L):
        key = lib.syn_key(w.seed, (KIND_ZIPF << 56) + w.layer0 + l)
        perm = list(range(w.N))
        for i in range(w.N - 1, 0, -1):
            j = int(lib.syn_draw(key, i) % (i + 1))
            perm[i], perm[j] = perm[j], perm[i]
        for pos, e in enumerate(perm):
            out[l, e] = np.float32(-w.zipf * math.log(pos + 1))
    return out


def fnv1a(buf: np.ndarray, h: int = 0xCBF29CE484222325) -> int:
    lib = _load_cpu()
    b = np.ascontiguousarray(buf)
    return int(lib.syn_fnv1a(b.ctypes.data_as(ctypes.c_void_p), b.nbytes, h))


# ---------------------------------------------------------------- device twin
def _check(rc: int, what: str):
    if rc != 0:
        raise RuntimeError(f"synth device generator failed in {what}: hipError {rc}")


def fill_router_dev(w: Workload, kind: int, out_ptr: int, stream: int = 0):
    """Fills [L][N][d] router weights of one kind at a device address."""
    _check(_load_hip().syn_dev_fill(w.seed, router_tid(kind, w.layer0), 1, w.L, w.N * w.d, weight_scale(w),
                                    int(w.dtype == DTYPE_BF16), out_ptr, stream), "router")


def fill_pool_dev(w: Workload, out_ptr: int, stream: int = 0, layers: Optional[Tuple[int, int]] = None):
    """Fills the cold expert pool [L][N] x (W_gate, W_up, W_down) at an address.

    `layers=(l0, l1)` fills only layers l0 <= l < l1 (into out_ptr, which then
    points at layer l0), so a pool in host memory can be built in chunks.
    """
    l0, l1 = (0, w.L) if layers is None else layers
    _check(_load_hip().syn_dev_fill(w.seed, expert_tid(w, w.layer0 + l0, 0), 1, (l1 - l0) * w.N,
                                    3 * w.F * w.d, weight_scale(w), int(w.dtype == DTYPE_BF16),
                                    out_ptr, stream), "pool")


def fill_hidden_dev(w: Workload, out_ptr: int, T: Optional[int] = None, stream: int = 0):
    """Fills AR(1) hidden states, token-major [T][S][L][d], at a device address."""
    T = w.T if T is None else T
    rho, c0 = ar1_params(w)
    _check(_load_hip().syn_dev_ar1(w.seed, hidden_tid(0, w.layer0), 1 << 24, 1, w.S, w.L, w.d, T, rho, c0,
                                   unit_scale(), int(w.dtype == DTYPE_BF16), out_ptr, stream), "hidden")


class _PinnedBlock:
    """hipHostMalloc memory of an exact size, freed with the last tensor that
    views it (torch's pinned allocator rounds sizes up, which on a host that
    limits the pinned memory of one process wastes most of that limit)."""

    def __init__(self, nbytes: int):
        p = ctypes.c_void_p()
        rc = _load_hip().syn_host_alloc(int(nbytes), ctypes.byref(p))
        if rc != 0 or not p.value:
            raise MemoryError(f"hipHostMalloc of {nbytes / 1e9:.1f} GB of pinned host memory failed (hipError {rc})")
        self.ptr = p.value
        self.nbytes = int(nbytes)

    def __del__(self):
        if getattr(self, "ptr", None):
            _load_hip().syn_host_free(ctypes.c_void_p(self.ptr))
            self.ptr = None


def pinned_host_tensor(shape, dtype):
    """A CPU tensor over pinned, device-mapped host memory of exactly its size."""
    import torch
    n = int(np.prod(shape)) * torch.empty((), dtype=dtype).element_size()
    block = _PinnedBlock(n)
    raw = np.ctypeslib.as_array((ctypes.c_uint8 * n).from_address(block.ptr))
    t = torch.from_numpy(raw).view(dtype).reshape(shape)
    t._pinned_block = block   # keeps the memory alive as long as the tensor
    return t


def device_inputs(w: Workload, T: Optional[int] = None, with_hidden: bool = True, stream: int = 0):
    """All inputs of a workload generated on the GPU (torch tensors on cuda:0).

    Returns a dict: wR, wT, wS ([L][N][d] or None), bias ([L][N] fp32 or None),
    pool ([L][N][3 d F] on the device, or in pinned host memory for a
    host-pool workload) and hidden ([T][S][L][d], token-major).  Values are
    bit-identical to the host twin's.
    """
    import torch
    dt = torch.bfloat16 if w.dtype == DTYPE_BF16 else torch.float32
    dev = torch.device("cuda", torch.cuda.current_device())
    out = {}
    out["wR"] = torch.empty((w.L, w.N, w.d), dtype=dt, device=dev)
    fill_router_dev(w, KIND_ROUTER_NATIVE, out["wR"].data_ptr(), stream)
    if w.has_temporal:
        out["wT"] = torch.empty((w.L, w.N, w.d), dtype=dt, device=dev)
        fill_router_dev(w, KIND_ROUTER_TEMPORAL, out["wT"].data_ptr(), stream)
    else:
        out["wT"] = None
    if w.has_spatio:
        out["wS"] = torch.empty((w.L, w.N, w.d), dtype=dt, device=dev)
        fill_router_dev(w, KIND_ROUTER_SPATIO, out["wS"].data_ptr(), stream)
    else:
        out["wS"] = None
    zb = zipf_bias(w)
    out["bias"] = None if zb is None else torch.from_numpy(zb).to(dev)
    per = 3 * w.F * w.d
    if w.pool_kind == POOL_HOST_PINNED:
        pool = pinned_host_tensor((w.L, w.N, per), dt)
        stage = torch.empty((1, w.N, per), dtype=dt, device=dev)
        for l in range(w.L):  # generate one layer on the device, copy it to host
            fill_pool_dev(w, stage.data_ptr(), stream, layers=(l, l + 1))
            pool[l].copy_(stage[0])
        del stage
    else:
        pool = torch.empty((w.L, w.N, per), dtype=dt, device=dev)
        fill_pool_dev(w, pool.data_ptr(), stream)
    out["pool"] = pool
    if with_hidden:
        T = w.T if T is None else T
        out["hidden"] = torch.empty((T, w.S, w.L, w.d), dtype=dt, device=dev)
        fill_hidden_dev(w, out["hidden"].data_ptr(), T, stream)
    torch.cuda.synchronize()
    return out
