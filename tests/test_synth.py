"""The seeded input generator: determinism, distribution, and its quantisers
checked against torch's conversions and the OCP rounding rules."""
import numpy as np
import torch

import oracle
from paper_2609_11133_amd import synth


def test_deterministic_and_stream_separated():
    a = synth.x_bf16(1234, 0, 4, 64)
    b = synth.x_bf16(1234, 0, 4, 64)
    c = synth.x_bf16(1234, 1, 4, 64)
    assert np.array_equal(a, b) and not np.array_equal(a, c)
    # prefix property: token t of a batch does not depend on the batch size
    assert np.array_equal(synth.x_bf16(1234, 0, 9, 64)[:4], a)
    w1, s1 = synth.experts(7, 0, 0, 4, 256, 128)
    w2, s2 = synth.experts(7, 0, 0, 4, 256, 128, e0=2, e1=4)
    assert np.array_equal(w1[2:], w2) and np.array_equal(s1[2:], s2)


def test_normal_moments():
    v = synth.normal(5, "x", 0, 0, 0, 400_000)
    assert abs(v.mean()) < 0.01 and abs(v.var() - 1.0) < 0.01
    assert abs((v**4).mean() - 2.9) < 0.05  # Irwin-Hall(12) kurtosis 2.9
    assert v.min() >= -6 and v.max() <= 6


def test_e4m3_encoder_matches_torch_rne():
    rng = np.random.default_rng(0)
    vals = np.concatenate([rng.standard_normal(3000) * 30, rng.standard_normal(1000) * 0.01, [0.0, -0.0, 448.0]])
    vals = vals[np.abs(vals) <= 448]
    ref = torch.from_numpy(vals).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    got = np.array([synth.e4m3_from_f64(float(v)) for v in vals], np.uint8)
    assert np.array_equal(got, ref)
    assert synth.e4m3_from_f64(1e6) == 0x7E and synth.e4m3_from_f64(-500.0) == 0xFE  # saturation


def test_e4m3_encoder_roundtrip_all_codes():
    for c in range(256):
        v = oracle.dec_e4m3(c)
        if v == v:  # not NaN
            assert synth.e4m3_from_f64(v) == c


def test_e2m1_encoder_rne_and_saturation():
    cases = {0.25: 0x0, 0.3: 0x1, 0.75: 0x2, 1.25: 0x2, 1.75: 0x4, 2.5: 0x4, 3.5: 0x6, 5.0: 0x6, 5.5: 0x7,
             7.0: 0x7, 100.0: 0x7, -0.75: 0xA, -6.0: 0xF}
    for v, c in cases.items():
        assert synth.e2m1_from_f64(v) == c, v
    for c in range(16):
        assert synth.e2m1_from_f64(oracle.dec_e2m1(c)) == c


def test_bf16_encoder_single_rounding():
    rng = np.random.default_rng(1)
    vals = rng.standard_normal(2000)
    ref = torch.from_numpy(vals.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().astype(np.uint16)
    got = np.array([synth.bf16_from_f64(float(v)) for v in vals], np.uint16)
    # the generator rounds fp64 straight to bf16; torch rounds the fp32 value.  They can
    # differ only where fp64 -> fp32 -> bf16 double-rounds, which these draws never hit.
    assert (got != ref).sum() == 0
    # a double-rounding case: 1 + 2^-8 + 2^-30 rounds up directly, but to 1 via fp32
    assert synth.bf16_from_f64(1.0 + 2.0**-8 + 2.0**-30) == 0x3F81


def test_fp8_blocks_use_full_range():
    H, I = 256, 256
    w, s = synth.experts(9, 0, 0, 1, H, I)
    gate = w[0, : I * H].reshape(I, H)
    for rb in range(I // 128):
        for cb in range(H // 128):
            blk = gate[rb * 128:(rb + 1) * 128, cb * 128:(cb + 1) * 128]
            assert (blk & 0x7F).max() == 0x7E  # the block's absolute max maps to 448


def test_mxfp4_groups_scale():
    H, I = 256, 128
    w, s = synth.experts(10, 0, 1, 1, H, I)
    g = w[0, : I * H // 2].reshape(I, H // 2)
    codes = np.stack([g & 15, g >> 4], axis=-1).reshape(I, H)
    mags = (codes & 7).reshape(I, H // 32, 32).max(axis=-1)
    # amax / 2^(floor(log2 amax) - 2) lies in [4, 8): the largest code is 4.0, 6.0 (or saturates to 6)
    assert np.all(mags >= 6)


def test_nvfp4_two_level_scales():
    """NVFP4 recipe: the matrix scale maps the matrix maximum to 6 x 448, every block's
    E4M3 scale is positive and maps its block maximum onto the top E2M1 code (6), and
    the block holding the matrix maximum gets the largest scale code (448)."""
    H, I = 256, 128
    w, s = synth.experts(12, 0, 2, 1, H, I)
    ts = s[0, :16].copy().view(np.float32)
    assert ts[3] == 0.0 and np.all(ts[:3] > 0)
    g = w[0, : I * H // 2].reshape(I, H // 2)
    codes = np.stack([g & 15, g >> 4], axis=-1).reshape(I, H)
    sg = s[0, 16: 16 + I * H // 16].reshape(I, H // 16)
    assert np.all(sg < 0x80)  # positive scales
    assert np.all((codes & 7).reshape(I, H // 16, 16).max(axis=-1) == 7)
    assert sg.max() == 0x7E
    v = synth.normal(12, "gate", 0, 0, 0, I * H, 1.0 / np.sqrt(H))
    assert np.float32(np.abs(v).max() / (6 * 448)) == ts[0]
