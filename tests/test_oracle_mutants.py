"""Each plausible mistake planted in a copy of the oracle's source must fail at
least one of the pins (which compare the oracle with independent references).
The mutants are built and run on the CPU only."""
import importlib.util
import math
import os
import subprocess
from fractions import Fraction

import numpy as np
import pytest
import scipy.special
import torch

from paper_2609_11133_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "moe_oracle.c")
ATTN_SRC = os.path.join(ROOT, "oracle", "attn_oracle.c")  # linked unchanged: the loader binds its symbol too
INIT = os.path.join(ROOT, "oracle", "__init__.py")

MUTANTS = {
    "swap_gate_up": ("a[i] = g / (1.0 + exp(-g)) * u;", "a[i] = u / (1.0 + exp(-u)) * g;"),
    "silu_sign": ("a[i] = g / (1.0 + exp(-g)) * u;", "a[i] = g / (1.0 + exp(g)) * u;"),
    "drop_bias": ("if (bias) acc_add(&acc, (double)*bias);", "(void)bias;"),
    "tie_to_higher_index": ("(l[f] == l[e] && f < e)", "(l[f] == l[e] && f > e)"),
    "transposed_down": ("acc += weight(X, e, 2, n, i) * a[i];", "acc += weight(X, e, 2, i, n) * a[i];"),
    "transposed_scale_block": ("sc[(n / 128) * (K / 128) + c / 128]", "sc[(c / 128) * (K / 128) + n / 128]"),
    "renorm_over_all": ("for (int j = 0; j < k; j++) zk += pe[ids[j]];", "for (int j = 0; j < E; j++) zk += pe[j];"),
    "round_half_up": ("if (rnd && (sticky || (mant & 1))) mant++;", "if (rnd) mant++;"),
    "combine_unweighted": ("acc += w[s * k + j] * o[(s * k + j) * H + n];", "acc += o[(s * k + j) * H + n];"),
    "nibble_order": ("(c % 2 == 0) ? (byte & 15) : (byte >> 4)", "(c % 2 == 0) ? (byte >> 4) : (byte & 15)"),
    "e4m3_bias": ("ldexp((double)(8 + m), e - 10)", "ldexp((double)(8 + m), e - 9)"),
    "acc_drops_sign": ("a->d[off / 32 + i] += q < 0 ? -dig : dig;", "a->d[off / 32 + i] += dig;"),
    "subnormal_grid": ("if (lsb < -149) lsb = -149;", "if (lsb < -150) lsb = -150;"),
    "e8m0_bias": ("ldexp(1.0, (int)c - 127)", "ldexp(1.0, (int)c - 128)"),
    "nvfp4_block_32": ("sb[n * (K / 16) + c / 16]", "sb[n * (K / 16) + c / 32]"),
    "nvfp4_no_matrix_scale": ("oracle_dec_e4m3(sb[n * (K / 16) + c / 16]) * (double)ts;",
                              "oracle_dec_e4m3(sb[n * (K / 16) + c / 16]);"),
    "nvfp4_gate_scale_for_all": ("memcpy(&ts, s + 4 * mat, 4);", "memcpy(&ts, s, 4);"),
    "nvfp4_scale_bytes_skip_header": ("const uint8_t *sb = s + 16 + (int64_t)mat * I * H / 16;",
                                      "const uint8_t *sb = s + (int64_t)mat * I * H / 16;"),
    "softmax_without_bias_in_weights": ("pe[e] = exp((double)l[e] - m);", "pe[e] = exp((double)l[e] - m - (bias ? bias[e] : 0));"),
}


def build_variant(tmp_path, name, old, new):
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation site for {name} not unique"
    path = tmp_path / f"{name}.c"
    path.write_text(src.replace(old, new))
    so = tmp_path / f"lib{name}.so"
    subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-std=c11", "-pthread", "-ffp-contract=off", "-o",
                           str(so), str(path), ATTN_SRC, "-lm"])
    spec = importlib.util.spec_from_file_location(f"oracle_{name}", INIT)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    mod._LIB = str(so)
    mod._lib = None
    return mod


# ---------------------------------------------------------------- pins (compact)

def bf16_f64(b):
    return (np.asarray(b, np.uint32) << 16).view(np.float32).astype(np.float64)


def rne_f32(q):
    if q == 0:
        return 0.0
    sign, a = (-1.0 if q < 0 else 1.0), abs(q)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    lsb = max(e - 23, -149)
    sc = a / Fraction(2) ** lsb
    m = sc.numerator // sc.denominator
    rem = sc - m
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and m % 2):
        m += 1
    return sign * math.ldexp(m, lsb)


def bits(v):
    return int(np.array([v], np.float32).view(np.uint32)[0])


def pin_formats(o):
    ref = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    for c in range(256):
        a, b = o.dec_e4m3(c), float(ref[c])
        if not ((math.isnan(a) and math.isnan(b)) or a == b):
            return False
    ref = torch.arange(255, dtype=torch.uint8).view(torch.float8_e8m0fnu).to(torch.float64).numpy()
    return all(o.dec_e8m0(c) == ref[c] for c in range(255))


def pin_rational_logits(o):
    H = 64
    x = synth.x_bf16(11, 0, 6, H)
    w = synth.router_bf16(11, 0, 4, H)
    b = synth.bias_normal(11, 0, 4, 0.5)
    for t in range(6):
        for e in range(4):
            s = sum((Fraction(float(p)) * Fraction(float(q)) for p, q in zip(bf16_f64(x[t]), bf16_f64(w[e]))),
                    Fraction(0)) + Fraction(float(b[e]))
            if bits(o.logit(x[t], w[e], float(b[e]))) != bits(np.float32(rne_f32(s)) + np.float32(0)):
                return False
    one = np.ones(2, np.float32)
    if o.logit(one, np.array([1.0 + 2.0**-23, 2.0**-24], np.float32)) != np.float32(1.0 + 2.0**-22):
        return False
    if o.logit(one, np.array([1.0, 2.0**-24], np.float32)) != 1.0:
        return False
    if o.logit(one[:1], np.array([2.0**-140], np.float32)) != np.float32(2.0**-140):
        return False
    tiny = np.array([2.0**-75, 2.0**-76], np.float32)  # products 2^-150 + 2^-152 round to 2^-149
    if o.logit(tiny, tiny) != np.float32(2.0**-149):
        return False
    return bits(o.logit(np.zeros(4, np.float32), -np.ones(4, np.float32))) == 0


def pin_topk_and_weights(o):
    H, E = 64, 12
    x = synth.x_bf16(21, 0, 12, H)
    w = synth.router_bf16(21, 0, E, H)
    w[9] = w[2]
    b = synth.bias_normal(21, 0, E, 0.5)
    b[9] = b[2]
    for t in range(12):
        for k in (1, 4, E):
            l, ids, wts, p = o.route_token(x[t], w, b, k)
            if list(ids) != sorted(range(E), key=lambda e: (-float(l[e]), e))[:k]:
                return False
            if not np.allclose(wts, scipy.special.softmax(l[ids].astype(np.float64)), rtol=1e-12, atol=0):
                return False
    l, ids, wts, _ = o.route_token(np.zeros(H, np.uint16), w, None, 3)
    return list(ids) == [0, 1, 2] and np.all(wts == 1 / 3)


def pin_dense(o):
    import test_oracle_layer as L  # independent numpy/torch dequantisers

    H, I = 256, 128
    x = synth.x_bf16(31, 0, 3, H)
    rw = synth.router_bf16(31, 0, 1, H)
    for wfmt in (0, 1, 2):
        w, s = synth.experts(31, 0, wfmt, 1, H, I)
        _, _, _, y = o.forward(x, rw, None, w, s, 1, I, wfmt)
        g, u, d = L.SPLIT[wfmt](w[0], s[0], H, I)
        ref = L.dense_swiglu(bf16_f64(x), g, u, d)
        if not np.allclose(y, ref, rtol=1e-11, atol=1e-13 * np.abs(ref).max()):
            return False
    return True


def pin_multi_expert(o):
    """k=E layer against the dense reference weighted by the scipy softmax."""
    import test_oracle_layer as L

    E, H, I, T = 4, 256, 128, 3
    x = synth.x_bf16(41, 0, T, H)
    rw = synth.router_bf16(41, 0, E, H)
    b = synth.bias_normal(41, 0, E, 0.5)
    w, s = synth.experts(41, 0, 0, E, H, I)
    for k in (E, 2):
        l, ids, wts, y = o.forward(x, rw, b, w, s, k, I, 0)
        xf = bf16_f64(x)
        for t in range(T):
            ref = np.zeros(H)
            sel = sorted(range(E), key=lambda e: (-float(l[t, e]), e))[:k]
            p = scipy.special.softmax(l[t, sel].astype(np.float64))
            for j, e in enumerate(sel):
                g, u, d = L.split_fp8_expert(w[e], s[e], H, I)
                ref += p[j] * L.dense_swiglu(xf[t:t + 1], g, u, d)[0]
            if not np.allclose(y[t], ref, rtol=1e-10, atol=1e-12 * np.abs(ref).max()):
                return False
    return True


PINS = [pin_formats, pin_rational_logits, pin_topk_and_weights, pin_dense, pin_multi_expert]


def test_unmutated_oracle_passes_every_pin(tmp_path):
    o = build_variant(tmp_path, "original", "return r + 0.0f; /* -0 -> +0 */", "return r + 0.0f; /* -0 -> +0 */")
    for pin in PINS:
        assert pin(o), pin.__name__


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(tmp_path, name):
    old, new = MUTANTS[name]
    o = build_variant(tmp_path, name, old, new)
    failed = [pin.__name__ for pin in PINS if not pin(o)]
    assert failed, f"mutant {name} passed every pin"
