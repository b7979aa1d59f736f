"""Pins of the oracle's routing (O1-O4): exact logits against an independent
rational-arithmetic reference and closed forms, top-k against brute force,
softmax/renormalisation against scipy and invariants."""
import math
from fractions import Fraction

import numpy as np
import pytest
import scipy.special

import oracle
from paper_2609_11133_amd import synth


def bf16_to_f64(bits):
    return (np.asarray(bits, np.uint32) << 16).view(np.float32).astype(np.float64)


def rne_f32_of_fraction(q: Fraction) -> float:
    """Round an exact rational to fp32, nearest, ties to even -- integer arithmetic only."""
    if q == 0:
        return 0.0
    sign = -1.0 if q < 0 else 1.0
    a = abs(q)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    lsb = max(e - 23, -149)
    scaled = a / Fraction(2) ** lsb
    m = scaled.numerator // scaled.denominator
    rem = scaled - m
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and m % 2 == 1):
        m += 1
    return sign * math.ldexp(m, lsb)


def exact_logit(xv, wv, b=None):
    s = sum((Fraction(float(a)) * Fraction(float(c)) for a, c in zip(xv, wv)), Fraction(0))
    if b is not None:
        s += Fraction(float(b))
    return np.float32(rne_f32_of_fraction(s)) + np.float32(0.0)


def f32_bits(v):
    return int(np.array([v], np.float32).view(np.uint32)[0])


@pytest.mark.parametrize("H", [16, 64, 256])
def test_logit_matches_rational_reference_bf16(H):
    x = synth.x_bf16(11, 0, 24, H)
    w = synth.router_bf16(11, 0, 6, H)
    b = synth.bias_normal(11, 0, 6, 0.5)
    xf, wf = bf16_to_f64(x), bf16_to_f64(w)
    for t in range(x.shape[0]):
        for e in range(w.shape[0]):
            got = oracle.logit(x[t], w[e], float(b[e]))
            ref = exact_logit(xf[t], wf[e], b[e])
            assert f32_bits(got) == f32_bits(ref), (t, e, got, ref)


def test_logit_matches_rational_reference_f32():
    H = 256
    x = synth.x_f32(12, 0, 16, H)
    w = synth.router_f32(12, 0, 8, H)
    for t in range(16):
        for e in range(8):
            got = oracle.logit(x[t], w[e])
            ref = exact_logit(x[t].astype(np.float64), w[e].astype(np.float64))
            assert f32_bits(got) == f32_bits(ref)


def test_logit_one_hot_closed_form():
    H, E = 128, 10
    w = synth.router_bf16(3, 0, E, H)
    for h in [0, 5, 127]:
        x = np.zeros(H, np.uint16)
        x[h] = 0x3F80  # 1.0 in bf16
        for e in range(E):
            assert f32_bits(oracle.logit(x, w[e])) == f32_bits(np.float32(bf16_to_f64(w[e, h])))


def test_logit_small_integers_exact():
    rng = np.random.default_rng(1)
    xi = rng.integers(-20, 21, 200).astype(np.float32)
    wi = rng.integers(-20, 21, 200).astype(np.float32)
    assert oracle.logit(xi, wi) == float(np.dot(xi.astype(np.int64), wi.astype(np.int64)))


def test_logit_cancellation_is_exact():
    # 2^80 + 2^-80 - 2^80: any fp64 running sum loses the middle term.
    x = np.ones(3, np.float32)
    w = np.array([2.0**80, 2.0**-80, -(2.0**80)], np.float32)
    assert oracle.logit(x, w) == 2.0**-80


def test_logit_ties_and_sticky():
    x = np.ones(2, np.float32)
    # 1 + 2^-24 is the midpoint of 1 and 1 + 2^-23: ties to even -> 1.
    assert oracle.logit(x, np.array([1.0, 2.0**-24], np.float32)) == 1.0
    # (1 + 2^-23) + 2^-24: midpoint of 1+2^-23 (odd) and 1+2^-22 (even) -> 1+2^-22.
    assert oracle.logit(x, np.array([1.0 + 2.0**-23, 2.0**-24], np.float32)) == np.float32(1.0 + 2.0**-22)
    # just above the midpoint -> rounds up
    x3 = np.ones(3, np.float32)
    assert oracle.logit(x3, np.array([1.0, 2.0**-24, 2.0**-60], np.float32)) == np.float32(1.0 + 2.0**-23)
    # subnormal results: exact, and rounded on the fixed 2^-149 grid
    assert oracle.logit(x[:1], np.array([2.0**-140], np.float32)) == np.float32(2.0**-140)
    tiny = np.array([2.0**-75, 2.0**-76], np.float32)  # 2^-150 + 2^-152 -> 2^-149
    assert oracle.logit(tiny, tiny) == np.float32(2.0**-149)
    tiny2 = np.array([2.0**-75], np.float32)  # 2^-150 alone: a tie between 0 and 2^-149 -> 0
    assert oracle.logit(tiny2, tiny2) == 0.0


def test_logit_negative_zero_canonical():
    x = np.zeros(8, np.float32)
    w = -np.ones(8, np.float32)
    assert f32_bits(oracle.logit(x, w)) == 0
    assert f32_bits(oracle.logit(x, w, -0.0)) == 0
    xb = np.full(4, 0x8000, np.uint16)  # -0 in bf16
    wb = np.full(4, 0x3F80, np.uint16)
    assert f32_bits(oracle.logit(xb, wb)) == 0


def brute_topk(l, k):
    return sorted(range(len(l)), key=lambda e: (-float(l[e]), e))[:k]


@pytest.mark.parametrize("E,k", [(8, 2), (16, 4), (40, 8), (5, 5), (7, 1)])
def test_topk_matches_brute_force(E, k):
    H = 64
    x = synth.x_bf16(21, 0, 40, H)
    w = synth.router_bf16(21, 0, E, H)
    b = synth.bias_normal(21, 0, E, 0.5)
    for t in range(x.shape[0]):
        l, ids, wts, p = oracle.route_token(x[t], w, b, k)
        assert list(ids) == brute_topk(l, k)


def test_topk_duplicate_rows_prefer_lower_index():
    H, E, k = 64, 12, 4
    w = synth.router_bf16(5, 0, E, H)
    w[9] = w[2]
    w[7] = w[2]
    x = synth.x_bf16(5, 0, 30, H)
    seen = 0
    for t in range(x.shape[0]):
        l, ids, _, _ = oracle.route_token(x[t], w, None, k)
        assert l[2] == l[7] == l[9]
        ids = list(ids)
        if 2 in ids:
            seen += 1
            pos = ids.index(2)
            assert ids[pos:pos + 3] == [2, 7, 9][: len(ids[pos:pos + 3])]
        assert 7 not in ids or 2 in ids
    assert seen > 0


def test_zero_input_routes_to_first_k_equally():
    H, E, k = 64, 16, 5
    w = synth.router_bf16(6, 0, E, H)
    x = np.zeros(H, np.uint16)
    l, ids, wts, p = oracle.route_token(x, w, None, k)
    assert list(ids) == list(range(k))
    assert np.all(wts == 1.0 / k)
    assert np.all(l == 0)


def test_softmax_and_renormalisation():
    H, E = 128, 24
    x = synth.x_bf16(8, 0, 30, H)
    w = synth.router_bf16(8, 0, E, H)
    b = synth.bias_normal(8, 0, E, 0.5)
    for t in range(30):
        for k in [1, 3, 8, E]:
            l, ids, wts, p = oracle.route_token(x[t], w, b, k)
            ref_p = scipy.special.softmax(l.astype(np.float64))
            np.testing.assert_allclose(p, ref_p, rtol=1e-12, atol=0)
            assert abs(wts.sum() - 1.0) <= 1e-12
            np.testing.assert_allclose(wts, scipy.special.softmax(l[ids].astype(np.float64)), rtol=1e-12)
            if k == 1:
                assert wts[0] == 1.0
            if k == E:
                np.testing.assert_allclose(wts, ref_p[ids], rtol=1e-12)
            assert np.all(np.diff(l[ids]) <= 0)


def test_bias_shift_invariance():
    """Adding one constant to every bias leaves the selection unchanged (away from
    near-ties, which these draws do not contain) and the weights equal up to the
    fp32 rounding of the shifted logits (softmax is shift invariant)."""
    H, E, k = 64, 16, 4
    x = synth.x_bf16(9, 0, 20, H)
    w = synth.router_bf16(9, 0, E, H)
    b = synth.bias_normal(9, 0, E, 0.5)
    for t in range(20):
        _, ids0, w0, _ = oracle.route_token(x[t], w, b, k)
        _, ids1, w1, _ = oracle.route_token(x[t], w, (b + np.float32(0.25)).astype(np.float32), k)
        assert list(ids0) == list(ids1)
        np.testing.assert_allclose(w0, w1, rtol=1e-5)
