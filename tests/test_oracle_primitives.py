"""Pins of the oracle's primitives against mathematics and independent routines.

Each check compares the oracle (C) with something other than itself: the fp64
exponential, closed forms, numpy's float64 linear algebra, or a numpy sort.
"""
import math
import struct

import numpy as np
import pytest

import oracle


def f32_bits(x):
    return struct.unpack("<I", struct.pack("<f", float(x)))[0]


def ulp32(x):
    x = abs(float(np.float32(x)))
    if x == 0:
        return 2.0 ** -149
    return float(np.spacing(np.float32(x)))


# ------------------------------------------------------------------ exp
def test_exp_constants_follow_their_definition():
    c = oracle.exp_constants()
    ln2_hi, ln2_lo, inv_ln2 = float(c[0]), float(c[1]), float(c[2])
    # the high part is fl32(ln 2) with the low 8 fraction bits cleared
    assert f32_bits(ln2_hi) == (f32_bits(math.log(2.0)) & ~0xFF)
    assert f32_bits(ln2_hi) & 0xFF == 0
    # hi + lo reconstructs ln 2 far below fp32 resolution
    assert abs((ln2_hi + ln2_lo) - math.log(2.0)) < 1e-13
    assert np.float32(inv_ln2) == np.float32(1.0 / math.log(2.0))
    for n in range(8):
        assert np.float32(c[3 + n]) == np.float32(1.0 / math.factorial(n))


def test_exp_special_values():
    e = oracle.exp([0.0, -0.0, -80.0, -80.5, -1000.0])
    assert e[0] == 1.0 and e[1] == 1.0          # exp(0) = 1 exactly
    assert e[2] > 0 and abs(e[2] - math.exp(-80.0)) <= 2 * ulp32(math.exp(-80.0))
    assert e[3] == 0.0 and e[4] == 0.0          # below -80 the result is +0


def test_exp_within_two_ulp_of_fp64_exp():
    rng = np.random.default_rng(1)
    xs = np.concatenate([-rng.uniform(0, 80, 20000), -rng.uniform(0, 1, 5000),
                         -np.arange(0, 80, 0.25)]).astype(np.float32)
    got = oracle.exp(xs)
    worst = 0.0
    for x, g in zip(xs, got):
        ref = math.exp(float(x))
        worst = max(worst, abs(float(g) - ref) / ulp32(ref))
    assert worst <= 2.0, worst


# ------------------------------------------------------------------ softmax
@pytest.mark.parametrize("n", [1, 2, 3, 16, 32, 100, 128, 256])
def test_softmax_matches_fp64_softmax(n):
    rng = np.random.default_rng(n)
    for scale in (0.1, 2.0, 8.0):
        z = (rng.normal(size=n) * scale).astype(np.float32)
        p = oracle.softmax(z)
        zz = z.astype(np.float64)
        ref = np.exp(zz - zz.max())
        ref /= ref.sum()
        # fp32 roundings: z - m (an argument error of |z - m| 2^-24, i.e. that
        # relative error after exp), exp (<= 2 ulp), the sum, the division
        tol = (4 + math.log2(max(n, 2)) + np.abs(zz - zz.max())) * 2.0 ** -24
        assert np.all(np.abs(p - ref) <= tol * ref + 1e-30), (n, scale)
        assert abs(float(np.sum(p.astype(np.float64))) - 1.0) <= n * 2.0 ** -23


def test_softmax_closed_forms():
    # all logits equal: u = 1 each, sum = n, p = fl32(1/n)
    for n in (1, 2, 5, 16, 128):
        p = oracle.softmax(np.full(n, 0.37, np.float32))
        assert np.all(p == np.float32(1.0 / n))
    # a dominant logit: the rest underflow to +0 (exp of < -80)
    z = np.array([0.0, -100.0, -200.0], np.float32)
    assert list(oracle.softmax(z)) == [1.0, 0.0, 0.0]
    # two logits differing by ln 3: p = (3/4, 1/4) to fp32 accuracy
    p = oracle.softmax(np.array([math.log(3.0), 0.0], np.float32))
    assert abs(p[0] - 0.75) < 3e-7 and abs(p[1] - 0.25) < 3e-7


def test_softmax_is_exactly_shift_invariant():
    # the max-shifted definition sees only z - max z; for logits on a 1/8 grid
    # adding c keeps z + c - (max z + c) exact in fp32, so the results agree
    # bit for bit (also where exp(z + c) itself would overflow)
    rng = np.random.default_rng(13)
    for n in (2, 5, 16, 128):
        z = (rng.integers(-32, 33, size=n) / 8.0).astype(np.float32)
        p = oracle.softmax(z)
        for c in (64.0, 1000.0, -1000.0):
            assert np.array_equal(oracle.softmax((z + np.float32(c)).astype(np.float32)), p), (n, c)


def test_softmax_is_monotone():
    rng = np.random.default_rng(7)
    z = np.sort(rng.normal(size=128).astype(np.float32) * 3)
    p = oracle.softmax(z)
    assert np.all(np.diff(p) >= 0)


# ------------------------------------------------------------------ Top-K
def _ref_topk(v, k):
    order = np.lexsort((np.arange(v.size), -v.astype(np.float64)))
    return order[:k]


@pytest.mark.parametrize("n,k", [(16, 2), (32, 4), (128, 8), (7, 7), (5, 1)])
def test_topk_matches_sorted_order_with_ties(n, k):
    rng = np.random.default_rng(n * 31 + k)
    for trial in range(200):
        if trial % 2:
            v = rng.integers(-3, 4, size=n).astype(np.float32)   # many ties
        else:
            v = rng.normal(size=n).astype(np.float32)
        assert list(oracle.topk(v, k)) == list(_ref_topk(v, k))


def test_topk_negative_zero_ties_with_positive_zero():
    v = np.array([-0.0, 0.0, -1.0, -0.0], np.float32)
    assert list(oracle.topk(v, 3)) == [0, 1, 3]


# ------------------------------------------------------------------ logits
def test_logits_equal_rounded_fp64_matvec():
    rng = np.random.default_rng(3)
    N, d = 64, 2048
    W = (rng.normal(size=(N, d)) * 0.02).astype(np.float32)
    h = rng.normal(size=d).astype(np.float32) * 2.3
    b = rng.normal(size=N).astype(np.float32)
    z = oracle.logits(W, h, b)
    ref = (W.astype(np.float64) @ h.astype(np.float64) + b.astype(np.float64))
    # both are fp64 sums rounded once; they may differ only by the rounding of
    # a sum that lands within ~1e-16 relative of an fp32 tie
    diff = np.abs(z.astype(np.float64) - ref.astype(np.float32).astype(np.float64))
    assert np.all(diff <= np.spacing(np.abs(ref).astype(np.float32)))
    assert np.mean(z == ref.astype(np.float32)) > 0.99


# ------------------------------------------------------------------ FFN
def test_moe_ffn_against_numpy_fp64():
    rng = np.random.default_rng(5)
    K, d, F = 3, 64, 96
    Wg = (rng.normal(size=(K, F, d)) * 0.1).astype(np.float32)
    Wu = (rng.normal(size=(K, F, d)) * 0.1).astype(np.float32)
    Wd = (rng.normal(size=(K, d, F)) * 0.1).astype(np.float32)
    g = np.array([0.5, 0.3, 0.2])
    x = rng.normal(size=d).astype(np.float32)
    y = oracle.moe_ffn(Wg, Wu, Wd, g, x)
    ref = np.zeros(d)
    for k in range(K):
        a = Wg[k].astype(np.float64) @ x
        b = Wu[k].astype(np.float64) @ x
        ref += g[k] * (Wd[k].astype(np.float64) @ (a / (1 + np.exp(-a)) * b))
    assert np.max(np.abs(y - ref)) <= 1e-12 * np.max(np.abs(ref))


def test_moe_ffn_one_hot_weights_route_each_activation():
    # x = e_2; row f of W_gate picks a_f, row f of W_up picks f + 1, and
    # W_down sends activation f to output perm[f] alone:
    # y[perm[f]] = g silu(a_f) (f + 1), every other output 0
    d, F, g = 6, 5, 0.75
    a = [0.5, -1.0, 2.0, 0.0, 1.5]
    perm = [4, 0, 5, 1, 3]
    x = np.zeros(d, np.float32)
    x[2] = 1.0
    Wg = np.zeros((1, F, d), np.float32)
    Wu = np.zeros((1, F, d), np.float32)
    Wd = np.zeros((1, d, F), np.float32)
    for f in range(F):
        Wg[0, f, 2] = a[f]
        Wu[0, f, 2] = f + 1
        Wd[0, perm[f], f] = 1.0
    y = oracle.moe_ffn(Wg, Wu, Wd, [g], x)
    expect = np.zeros(d)
    for f in range(F):
        expect[perm[f]] = g * a[f] / (1.0 + math.exp(-a[f])) * (f + 1)
    assert np.allclose(y, expect, rtol=1e-15, atol=1e-300)


def test_moe_ffn_closed_form_silu():
    # d = F = 1: W_gate = a, W_up = 1, W_down = 1, x = 1 -> y = g * silu(a)
    for a, silu in ((1.0, 0.7310585786300049), (-2.0, -0.2384058440442351), (0.0, 0.0)):
        y = oracle.moe_ffn(np.full((1, 1, 1), a, np.float32), np.ones((1, 1, 1), np.float32),
                           np.ones((1, 1, 1), np.float32), np.array([1.0]), np.ones(1, np.float32))
        assert abs(y[0] - silu) < 1e-15
    # gate weights scale linearly and two identical experts add
    rng = np.random.default_rng(9)
    Wg = rng.normal(size=(1, 8, 4)).astype(np.float32)
    Wu = rng.normal(size=(1, 8, 4)).astype(np.float32)
    Wd = rng.normal(size=(1, 4, 8)).astype(np.float32)
    x = rng.normal(size=4).astype(np.float32)
    y1 = oracle.moe_ffn(Wg, Wu, Wd, [1.0], x)
    y2 = oracle.moe_ffn(np.concatenate([Wg, Wg]), np.concatenate([Wu, Wu]), np.concatenate([Wd, Wd]),
                        [0.25, 0.75], x)
    assert np.allclose(y1, y2, rtol=1e-14, atol=1e-14)
