"""The C-ABI library loads, exports every entry point the header declares, and
validates configurations on the host (no GPU needed for any of this)."""
import ctypes
import os
import re

import pytest

from paper_2609_04895_amd import cmoe as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cmoe.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(cmoe_[a-z_A-Z]+)\s*\(", text)))


def test_header_declares_the_binding_names():
    assert declared_functions() == sorted(B.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = B.lib()
    for name in declared_functions():
        assert hasattr(lib, name), name


def cfg(**kw):
    base = dict(L=4, N=16, K=2, d=256, F=512, C=6, R=0, S=1, mode=0, dtype=0)
    base.update(kw)
    return B.make_config(**base)


def query(**kw):
    out = B.cmoe_sizes()
    st = B.lib().cmoe_query(ctypes.byref(cfg(**kw)), ctypes.byref(out))
    return st, out


def test_query_sizes_of_tiny_workload():
    st, out = query()
    assert st == B.CMOE_OK
    # arena: L x min(N, S C) slots of 3 d F fp32 values
    assert out.arena_bytes == 4 * 6 * 3 * 256 * 512 * 4
    assert out.state_bytes > 0 and out.workspace_bytes > 0
    assert out.state_bytes % 256 == 0 and out.workspace_bytes % 256 == 0


def test_query_arena_is_capped_by_n_slots():
    st, out = query(S=64, C=6)      # S C > N: one slot per expert
    assert st == B.CMOE_OK and out.arena_bytes == 4 * 16 * 3 * 256 * 512 * 4


@pytest.mark.parametrize("kw,status", [
    (dict(K=7, C=6), B.CMOE_ERR_INVALID_ARG),          # capacity below Top-K
    (dict(C=17), B.CMOE_ERR_INVALID_ARG),              # capacity above N
    (dict(R=-1), B.CMOE_ERR_INVALID_ARG),
    (dict(R=17), B.CMOE_ERR_INVALID_ARG),
    (dict(L=0), B.CMOE_ERR_INVALID_ARG),
    (dict(S=0), B.CMOE_ERR_INVALID_ARG),
    (dict(mode=3), B.CMOE_ERR_INVALID_ARG),
    (dict(mode=2), B.CMOE_ERR_INVALID_ARG),            # Spatio-only has no Temporal Router
    (dict(policy=4), B.CMOE_ERR_INVALID_ARG),
    (dict(policy=-1), B.CMOE_ERR_INVALID_ARG),
    (dict(mode=1, R=2, policy=1), B.CMOE_ERR_UNSUPPORTED),   # full mode retains by s^T
    (dict(policy=3, lrfu_lambda=-0.5), B.CMOE_ERR_INVALID_ARG),
    (dict(policy=3, lrfu_lambda=float("nan")), B.CMOE_ERR_INVALID_ARG),
    (dict(policy=3, lrfu_lambda=float("inf")), B.CMOE_ERR_INVALID_ARG),
    (dict(dtype=5), B.CMOE_ERR_INVALID_ARG),
    (dict(flags=B.CMOE_FLAG_FFN_GROUPED | B.CMOE_FLAG_FFN_SINGLE), B.CMOE_ERR_INVALID_ARG),
    (dict(N=300, C=6), B.CMOE_ERR_UNSUPPORTED),
    (dict(d=200), B.CMOE_ERR_UNSUPPORTED),
    (dict(F=100), B.CMOE_ERR_UNSUPPORTED),
    (dict(N=128, K=65, C=70), B.CMOE_ERR_UNSUPPORTED),
])
def test_query_rejects_invalid_configs(kw, status):
    st, _ = query(**kw)
    assert st == status
    assert len(B.lib().cmoe_last_error()) > 0


@pytest.mark.parametrize("kw", [dict(policy=1), dict(policy=2), dict(policy=3, lrfu_lambda=0.0),
                                dict(mode=2, policy=1, R=3), dict(mode=2, policy=3, R=16),
                                dict(flags=B.CMOE_FLAG_FFN_GROUPED), dict(flags=B.CMOE_FLAG_FFN_SINGLE)])
def test_query_accepts_policy_configs(kw):
    st, out = query(**kw)
    assert st == B.CMOE_OK


def test_classical_policies_need_fewer_router_slots():
    # one router slot (native) instead of two: smaller partials and logits
    _, router = query(S=64, N=16, C=6)
    _, lru = query(S=64, N=16, C=6, policy=1)
    assert lru.workspace_bytes < router.workspace_bytes
    assert B.router_slots(cfg(policy=1)) == ["native"]
    assert B.router_slots(cfg(mode=2, policy=1)) == ["native", "spatio"]
    assert B.router_slots(cfg(mode=1)) == ["native", "temporal", "spatio"]


def test_spatio_only_needs_spatio_router_and_not_temporal():
    h = ctypes.c_void_p()
    bufs = B.cmoe_buffers(256, 512, 768)
    c = cfg(mode=2, policy=1, R=2)
    w = B.cmoe_weights(256, None, None, None, 1024)
    st = B.lib().cmoe_init(ctypes.byref(c), ctypes.byref(w), ctypes.byref(bufs), None, None, ctypes.byref(h))
    assert st == B.CMOE_ERR_INVALID_ARG and b"w_spatio" in B.lib().cmoe_last_error()
    c = cfg(policy=2)                         # LFU, update-only: W^T is not needed
    w = B.cmoe_weights(256, None, None, None, 1024)
    B.lib().cmoe_init(ctypes.byref(c), ctypes.byref(w), ctypes.byref(bufs), None, None, ctypes.byref(h))
    assert b"w_temporal" not in B.lib().cmoe_last_error()


def test_init_rejects_missing_pointers_before_touching_the_gpu():
    c = cfg()
    h = ctypes.c_void_p()
    w = B.cmoe_weights(None, None, None, None, None)
    bufs = B.cmoe_buffers(None, None, None)
    st = B.lib().cmoe_init(ctypes.byref(c), ctypes.byref(w), ctypes.byref(bufs), None, None, ctypes.byref(h))
    assert st == B.CMOE_ERR_INVALID_ARG and not h.value


def test_full_mode_needs_spatio_router():
    c = cfg(mode=1, R=2)
    h = ctypes.c_void_p()
    w = B.cmoe_weights(256, 512, None, None, 1024)
    bufs = B.cmoe_buffers(256, 512, 768)
    st = B.lib().cmoe_init(ctypes.byref(c), ctypes.byref(w), ctypes.byref(bufs), None, None, ctypes.byref(h))
    assert st == B.CMOE_ERR_INVALID_ARG
    assert b"w_spatio" in B.lib().cmoe_last_error()


def test_misaligned_buffers_rejected():
    c = cfg()
    h = ctypes.c_void_p()
    w = B.cmoe_weights(256, 512, None, None, 1024)
    bufs = B.cmoe_buffers(256 + 4, 512, 768)
    st = B.lib().cmoe_init(ctypes.byref(c), ctypes.byref(w), ctypes.byref(bufs), None, None, ctypes.byref(h))
    assert st == B.CMOE_ERR_INVALID_ARG


def test_null_handle_calls_fail_cleanly():
    L = B.lib()
    assert L.cmoe_step(None, None, None) == B.CMOE_ERR_INVALID_ARG
    assert L.cmoe_set_R(None, 1) == B.CMOE_ERR_INVALID_ARG
    assert L.cmoe_reset(None) == B.CMOE_ERR_INVALID_ARG
    assert L.cmoe_destroy(None) == B.CMOE_OK
    assert L.cmoe_view_bytes(None, 0) == 0


@pytest.mark.parametrize("src,nbytes,reps,out,msg", [
    (None, 1 << 30, 1, True, "required"),            # no buffer
    (1 << 20, 1 << 30, 1, False, "required"),        # no output
    (1 << 20, 1 << 30, 0, True, "reps"),             # no launch asked for
    (1 << 20, (64 << 20) - 1, 1, True, "64 MiB"),    # too small to occupy the device
])
def test_read_probe_rejects_bad_arguments_before_any_launch(src, nbytes, reps, out, msg):
    rate = ctypes.c_double(-1.0)
    st = B.lib().cmoe_read_probe(ctypes.c_void_p(src), nbytes, reps, ctypes.byref(rate) if out else None)
    assert st == B.CMOE_ERR_INVALID_ARG
    assert msg in B.lib().cmoe_last_error().decode()
    assert rate.value == -1.0
