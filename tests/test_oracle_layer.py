"""Pins of the oracle's expert FFN and combine (O5-O7): the dense-SwiGLU reduction
against numpy with torch's independent FP8 decoder, an identity closed form,
MXFP4 against the OCP table, and layer invariants."""
import os
import time

import numpy as np
import pytest
import torch

import oracle
from paper_2609_11133_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def bf16_to_f64(bits):
    return (np.asarray(bits, np.uint32) << 16).view(np.float32).astype(np.float64)


def e2m1_table():
    vals = {}
    for line in open(os.path.join(GOLDEN, "e2m1_ocp_mx.txt")):
        if line.strip() and not line.startswith("#"):
            c, v = line.split()
            vals[int(c, 16)] = float(v)
    return np.array([vals[c] for c in range(16)])


def dequant_fp8_numpy(wq, sc, N, K):
    """Independent dequantisation: torch's float8_e4m3fn decoder + numpy block scales."""
    q = torch.from_numpy(np.ascontiguousarray(wq).reshape(N, K)).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    s = np.asarray(sc, np.float64).reshape(N // 128, K // 128)
    return q * np.kron(s, np.ones((128, 128)))


def split_fp8_expert(w, s, H, I):
    g = dequant_fp8_numpy(w[: I * H], s[: (I // 128) * (H // 128)], I, H)
    u = dequant_fp8_numpy(w[I * H: 2 * I * H], s[(I // 128) * (H // 128): 2 * (I // 128) * (H // 128)], I, H)
    d = dequant_fp8_numpy(w[2 * I * H:], s[2 * (I // 128) * (H // 128):], H, I)
    return g, u, d


def dequant_mxfp4_numpy(wq, sc, N, K):
    tab = e2m1_table()
    b = np.asarray(wq, np.uint8).reshape(N, K // 2)
    codes = np.empty((N, K), np.int64)
    codes[:, 0::2] = b & 15
    codes[:, 1::2] = b >> 4
    scale = np.exp2(np.asarray(sc, np.float64).reshape(N, K // 32) - 127.0)
    return tab[codes] * np.repeat(scale, 32, axis=1)


def split_mxfp4_expert(w, s, H, I):
    g = dequant_mxfp4_numpy(w[: I * H // 2], s[: I * H // 32], I, H)
    u = dequant_mxfp4_numpy(w[I * H // 2: I * H], s[I * H // 32: 2 * I * H // 32], I, H)
    d = dequant_mxfp4_numpy(w[I * H:], s[2 * I * H // 32:], H, I)
    return g, u, d


def dequant_nvfp4_numpy(wq, sb, ts, N, K):
    """Independent NVFP4 dequantisation: the OCP E2M1 table, torch's float8_e4m3fn
    decoder for the per-16 block scales, and the fp32 matrix scale."""
    tab = e2m1_table()
    b = np.asarray(wq, np.uint8).reshape(N, K // 2)
    codes = np.empty((N, K), np.int64)
    codes[:, 0::2] = b & 15
    codes[:, 1::2] = b >> 4
    s = torch.from_numpy(np.ascontiguousarray(sb).reshape(N, K // 16)).view(torch.float8_e4m3fn)
    s = s.to(torch.float64).numpy()
    return tab[codes] * np.repeat(s, 16, axis=1) * float(ts)


def split_nvfp4_expert(w, s, H, I):
    ts = np.ascontiguousarray(s[:16]).view(np.float32)
    blk = s[16:]
    g = dequant_nvfp4_numpy(w[: I * H // 2], blk[: I * H // 16], ts[0], I, H)
    u = dequant_nvfp4_numpy(w[I * H // 2: I * H], blk[I * H // 16: 2 * I * H // 16], ts[1], I, H)
    d = dequant_nvfp4_numpy(w[I * H:], blk[2 * I * H // 16:], ts[2], H, I)
    return g, u, d


SPLIT = {0: split_fp8_expert, 1: split_mxfp4_expert, 2: split_nvfp4_expert}


def dense_swiglu(x, g, u, d):
    a = x @ g.T
    return ((a / (1.0 + np.exp(-a))) * (x @ u.T)) @ d.T


@pytest.mark.parametrize("wfmt", [0, 1, 2])
def test_single_expert_is_dense_swiglu(wfmt):
    H, I, T = 256, 128, 6
    x = synth.x_bf16(31, 0, T, H)
    rw = synth.router_bf16(31, 0, 1, H)
    w, s = synth.experts(31, 0, wfmt, 1, H, I)
    _, ids, wts, y = oracle.forward(x, rw, None, w, s, 1, I, wfmt)
    assert np.all(ids == 0) and np.all(wts == 1.0)
    g, u, d = SPLIT[wfmt](w[0], s[0], H, I)
    ref = dense_swiglu(bf16_to_f64(x), g, u, d)
    np.testing.assert_allclose(y, ref, rtol=1e-11, atol=1e-13 * np.abs(ref).max())


def test_expert_ffn_direct_matches_dense():
    H, I = 256, 256
    w, s = synth.experts(32, 0, 0, 3, H, I)
    rng = np.random.default_rng(3)
    xv = rng.standard_normal(H)
    for e in range(3):
        g, u, d = split_fp8_expert(w[e], s[e], H, I)
        ref = dense_swiglu(xv[None, :], g, u, d)[0]
        o = oracle.expert_ffn(w, s, e, xv, H, I, 0)
        np.testing.assert_allclose(o, ref, rtol=1e-11, atol=1e-13 * np.abs(ref).max())


def test_identity_expert_closed_form():
    """gate = c [I|0], up = [I|0], down = [I;0] with unit scales:
    y[h] = silu(c x_h) x_h for h < I and 0 above."""
    H, I, E, k, T = 256, 128, 4, 2, 5
    c_code, c = 0x30, 0.5  # 0x30 = 0.5 in E4M3
    w = np.zeros((E, 3 * H * I), np.uint8)
    for e in range(E):
        gate = np.zeros((I, H), np.uint8)
        up = np.zeros((I, H), np.uint8)
        down = np.zeros((H, I), np.uint8)
        for i in range(I):
            gate[i, i] = c_code
            up[i, i] = 0x38
            down[i, i] = 0x38
        w[e] = np.concatenate([gate.ravel(), up.ravel(), down.ravel()])
    s = np.ones((E, 3 * (H // 128) * (I // 128)), np.float32)
    x = synth.x_bf16(33, 0, T, H)
    rw = synth.router_bf16(33, 0, E, H)
    _, ids, wts, y = oracle.forward(x, rw, None, w, s, k, I, 0)
    xf = bf16_to_f64(x)
    ref = np.zeros((T, H))
    ref[:, :I] = (c * xf[:, :I]) / (1.0 + np.exp(-c * xf[:, :I])) * xf[:, :I]
    np.testing.assert_allclose(y, ref, rtol=1e-14, atol=1e-15)
    assert np.all(y[:, I:] == 0.0)


def _layer(E=8, H=256, I=128, k=2, T=6, wfmt=0, seed=41, bias=True):
    x = synth.x_bf16(seed, 0, T, H)
    rw = synth.router_bf16(seed, 0, E, H)
    b = synth.bias_normal(seed, 0, E, 0.5) if bias else None
    w, s = synth.experts(seed, 0, wfmt, E, H, I)
    return x, rw, b, w, s


@pytest.mark.parametrize("wfmt", [0, 1, 2])
def test_relabel_experts_invariance(wfmt):
    E, H, I, k = 8, 256, 128, 3
    x, rw, b, w, s = _layer(E=E, k=k, wfmt=wfmt)
    _, ids, wts, y = oracle.forward(x, rw, b, w, s, k, I, wfmt)
    perm = np.random.default_rng(4).permutation(E)  # new label of old expert e is perm[e]
    inv = np.argsort(perm)
    _, ids2, wts2, y2 = oracle.forward(x, rw[inv], b[inv], w[inv], s[inv], k, I, wfmt)
    assert np.array_equal(ids2, perm[ids])
    np.testing.assert_allclose(wts2, wts, rtol=1e-14)
    np.testing.assert_allclose(y2, y, rtol=1e-12, atol=1e-14 * np.abs(y).max())


def test_token_permutation_and_batch_independence():
    E, H, I, k, T = 8, 256, 128, 2, 7
    x, rw, b, w, s = _layer(E=E, k=k, T=T)
    l, ids, wts, y = oracle.forward(x, rw, b, w, s, k, I, 0)
    perm = np.random.default_rng(5).permutation(T)
    l2, ids2, wts2, y2 = oracle.forward(x[perm], rw, b, w, s, k, I, 0)
    assert np.array_equal(y2, y[perm]) and np.array_equal(ids2, ids[perm]) and np.array_equal(l2, l[perm])
    sub = [5, 1]
    _, ids3, _, y3 = oracle.forward(x, rw, b, w, s, k, I, 0, tokens=sub)
    assert np.array_equal(y3, y[sub]) and np.array_equal(ids3, ids[sub])
    _, _, _, y4 = oracle.forward(x[[3]], rw, b, w, s, k, I, 0)
    assert np.array_equal(y4[0], y[3])


@pytest.mark.parametrize("wfmt", [0, 1, 2])
def test_doubling_down_scales_doubles_output(wfmt):
    E, H, I, k = 8, 256, 128, 2
    x, rw, b, w, s = _layer(E=E, k=k, wfmt=wfmt)
    _, _, _, y = oracle.forward(x, rw, b, w, s, k, I, wfmt)
    s2 = s.copy()
    if wfmt == 0:
        nsg = 2 * (I // 128) * (H // 128)
        s2[:, nsg:] *= 2
    elif wfmt == 1:
        s2[:, 2 * I * H // 32:] += 1
    else:
        s2[:, 8:12] = (s2[:, 8:12].copy().view(np.float32) * 2).view(np.uint8)  # the down matrix scale
    _, _, _, y2 = oracle.forward(x, rw, b, w, s2, k, I, wfmt)
    assert np.array_equal(y2, 2 * y)


def test_threads_do_not_change_result():
    x, rw, b, w, s = _layer(T=9, k=3)
    r1 = oracle.forward(x, rw, b, w, s, 3, 128, 0, threads=1)
    r4 = oracle.forward(x, rw, b, w, s, 3, 128, 0, threads=4)
    for a, c in zip(r1, r4):
        assert np.array_equal(a, c)


def test_all_experts_selected_k_equals_e():
    E, H, I = 4, 256, 128
    x, rw, b, w, s = _layer(E=E, k=E, T=3)
    _, ids, wts, y = oracle.forward(x, rw, b, w, s, E, I, 0)
    assert all(sorted(r) == list(range(E)) for r in ids)
    # y = sum over all experts, weighted by the full softmax
    xf = bf16_to_f64(x)
    ref = np.zeros_like(y)
    for t in range(3):
        for j in range(E):
            g, u, d = split_fp8_expert(w[ids[t, j]], s[ids[t, j]], H, I)
            ref[t] += wts[t, j] * dense_swiglu(xf[t:t + 1], g, u, d)[0]
    np.testing.assert_allclose(y, ref, rtol=1e-11, atol=1e-13 * np.abs(ref).max())


def test_nvfp4_block_scale_closed_form():
    """One NVFP4 expert with hand-set codes: gate row i holds code c_i at input i and
    block scale S_i, up row i holds 1.0 with scale 1, down row i holds 1.0 at input i,
    and matrix scales tg, tu, td: y[h] = td * silu(tg * e2m1(c_h) * S_h * x_h) * tu * x_h
    for h < I, 0 above.  Block scales differ in their mantissa bits, so a scale applied
    per 32 inputs or without its mantissa fails."""
    H, I, E = 256, 128, 1
    codes = [0x2, 0x3, 0x5, 0x7, 0x9, 0xB, 0xD, 0xF]  # 1, 1.5, 3, 6 and their negatives
    scodes = [0x38, 0x39, 0x3A, 0x3B, 0x3C, 0x3D, 0x3E, 0x3F, 0x30, 0x41, 0x2B]  # 1 .. 1.875, 0.5, 2.25, 0.34375
    tg, tu, td = np.float32(0.75), np.float32(1.25), np.float32(0.5)
    gate = np.zeros((I, H), np.uint8)
    up = np.zeros((I, H), np.uint8)
    down = np.zeros((H, I), np.uint8)
    sg = np.zeros((I, H // 16), np.uint8)
    su = np.full((I, H // 16), 0x38, np.uint8)
    sd = np.full((H, I // 16), 0x38, np.uint8)
    for i in range(I):
        gate[i, i] = codes[i % len(codes)]
        sg[i, i // 16] = scodes[i % len(scodes)]
        up[i, i] = 0x2
        down[i, i] = 0x2

    def pack(m):
        return (m[:, 0::2] | (m[:, 1::2] << 4)).astype(np.uint8).ravel()

    w = np.concatenate([pack(gate), pack(up), pack(down)])[None, :]
    ts = np.array([tg, tu, td, 0], np.float32).view(np.uint8)
    s = np.concatenate([ts, sg.ravel(), su.ravel(), sd.ravel()])[None, :]
    T = 4
    x = synth.x_bf16(34, 0, T, H)
    rw = synth.router_bf16(34, 0, E, H)
    _, _, _, y = oracle.forward(x, rw, None, w, s, 1, I, 2)
    tab = e2m1_table()
    s_of = lambda c: torch.tensor([c], dtype=torch.uint8).view(torch.float8_e4m3fn).double().item()
    xf = bf16_to_f64(x)
    ref = np.zeros((T, H))
    for h in range(I):
        gv = float(tg) * tab[codes[h % len(codes)]] * s_of(scodes[h % len(scodes)]) * xf[:, h]
        ref[:, h] = float(td) * gv / (1.0 + np.exp(-gv)) * float(tu) * xf[:, h]
    np.testing.assert_allclose(y, ref, rtol=1e-14, atol=1e-16)
    assert np.all(y[:, I:] == 0.0)


def test_tiny_config_under_one_second():
    """The 4-token tiny layer (hidden 256, 8 experts, top-2, intermediate 128, fp32
    activations) runs through the oracle in well under a second."""
    H, E, k, I, T = 256, 8, 2, 128, 4
    x = synth.x_f32(1234, 0, T, H)
    rw = synth.router_f32(1234, 0, E, H)
    w, s = synth.experts(1234, 0, 0, E, H, I)
    t0 = time.perf_counter()
    _, ids, wts, y = oracle.forward(x, rw, None, w, s, k, I, 0)
    assert time.perf_counter() - t0 < 1.0
    assert y.shape == (T, H) and np.all(np.isfinite(y))
