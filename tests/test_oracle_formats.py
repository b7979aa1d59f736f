"""Pins of the oracle's number-format decoders (O5) against the OCP format tables
and against torch's independent CPU conversions."""
import math
import os

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _read_golden(name, base):
    rows = []
    for line in open(os.path.join(GOLDEN, name)):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        c, v = line.split()
        rows.append((int(c, base), float(v)))
    return rows


def _same(a, b):
    if math.isnan(b):
        return math.isnan(a)
    return a == b and math.copysign(1.0, a) == math.copysign(1.0, b)


def test_e4m3_spec_table():
    for c, v in _read_golden("e4m3_ocp_special.txt", 16):
        assert _same(oracle.dec_e4m3(c), v), hex(c)


def test_e4m3_all_codes_match_torch():
    codes = torch.arange(256, dtype=torch.uint8)
    ref = codes.view(torch.float8_e4m3fn).to(torch.float64).numpy()
    for c in range(256):
        assert _same(oracle.dec_e4m3(c), float(ref[c])), hex(c)


def test_e4m3_monotone_and_count():
    pos = [oracle.dec_e4m3(c) for c in range(0x7F)]
    assert all(b > a for a, b in zip(pos, pos[1:]))  # strictly increasing over 0x00..0x7E
    assert len(set(pos)) == 127


def test_e2m1_spec_table():
    rows = _read_golden("e2m1_ocp_mx.txt", 16)
    assert len(rows) == 16
    for c, v in rows:
        assert _same(oracle.dec_e2m1(c), v), hex(c)


def test_e8m0_spec_table_and_torch():
    for c, v in _read_golden("e8m0_ocp_mx.txt", 10):
        assert _same(oracle.dec_e8m0(c), v), c
    ref = torch.arange(256, dtype=torch.uint8).view(torch.float8_e8m0fnu).to(torch.float64).numpy()
    for c in range(256):
        assert _same(oracle.dec_e8m0(c), float(ref[c])), c


def test_bf16_matches_torch():
    rng = np.random.default_rng(0)
    bits = np.concatenate([rng.integers(0, 1 << 16, 4000), [0, 0x8000, 0x3F80, 0xBF80, 0x0001, 0x7F7F]])
    bits = bits[((bits >> 7) & 0xFF) != 0xFF]  # finite only
    ref = torch.from_numpy(bits.astype(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    for b, r in zip(bits, ref):
        assert _same(oracle.dec_bf16(int(b)), float(r)), hex(int(b))
