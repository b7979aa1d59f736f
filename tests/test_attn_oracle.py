"""Pins of the decode-attention oracle (``oracle/attn_oracle.c``), on the CPU.

Each pin compares the oracle with something that does not share its arithmetic:
closed forms (one token, identical keys, a zero query, a value constant per key/value
head), torch's float64 scaled-dot-product attention on the gathered dense cache, and
invariants (page relabelling, bytes past the context, scale folded into the query).
Planted mistakes in a copy of the oracle must each fail at least one pin."""
import importlib.util
import os
import subprocess

import numpy as np
import pytest
import torch

import oracle
from paper_2609_11133_amd import synth
from paper_2609_11133_amd.attn_workload import NAN_BF16

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ATTN_SRC = os.path.join(ROOT, "oracle", "attn_oracle.c")
MOE_SRC = os.path.join(ROOT, "oracle", "moe_oracle.c")
INIT = os.path.join(ROOT, "oracle", "__init__.py")
D, P = 128, 16


def bf16_f64(b):
    return (np.asarray(b, np.uint32) << 16).view(np.float32).astype(np.float64)


def f64_bf16(v):
    """Round-to-nearest-even fp64 -> bf16 bits (values well inside range)."""
    f = np.asarray(v, np.float32).view(np.uint32).astype(np.uint64)
    return ((f + 0x7FFF + ((f >> 16) & 1)) >> 16).astype(np.uint16)


def case(seed, B, Hq, Hkv, lens, max_pages=None, garbage=True):
    """Random scattered paged cache for context lengths `lens`."""
    rng = np.random.default_rng(seed)
    lens = np.asarray(lens, np.int32)
    pages = (lens.astype(np.int64) + P - 1) // P
    mp = max(1, int(pages.max())) if max_pages is None else max_pages
    used = int(pages.sum())
    n_pages = used + 3
    perm = rng.permutation(n_pages).astype(np.int32)
    bt = np.full((B, mp), -7, np.int32)  # entries past the context are never read
    o = 0
    for b in range(B):
        bt[b, : pages[b]] = perm[o: o + pages[b]]
        o += pages[b]
    q = synth.normal_bf16(seed, "q", 0, 0, B * Hq * D).reshape(B, Hq, D)
    kc = synth.normal_bf16(seed, "k", 0, 0, n_pages * Hkv * P * D).reshape(n_pages, Hkv, P, D)
    vc = synth.normal_bf16(seed, "v", 0, 0, n_pages * Hkv * D * P).reshape(n_pages, Hkv, D, P)
    if garbage:
        kc[perm[used:]] = NAN_BF16
        vc[perm[used:]] = NAN_BF16
        for b in range(B):
            if pages[b] and lens[b] % P:
                last = bt[b, pages[b] - 1]
                kc[last, :, lens[b] % P:, :] = NAN_BF16
                vc[last, :, :, lens[b] % P:] = NAN_BF16
    return q, kc, vc, bt, lens


def dense(kc, vc, bt, b, L, g):
    """Keys [L, D] and values [L, D] of sequence b, head g, gathered token by token."""
    K = np.stack([kc[bt[b, j // P], g, j % P, :] for j in range(L)]) if L else np.zeros((0, D), np.uint16)
    V = np.stack([vc[bt[b, j // P], g, :, j % P] for j in range(L)]) if L else np.zeros((0, D), np.uint16)
    return bf16_f64(K), bf16_f64(V)


# ---------------------------------------------------------------- pins (each returns a bool)

def pin_single_token(o):
    q, kc, vc, bt, L = case(1, 3, 8, 2, [1, 1, 1])
    out = o.attn_decode(q, kc, vc, bt, L, 0.088)
    for b in range(3):
        for h in range(8):
            if not np.array_equal(out[b, h], bf16_f64(vc[bt[b, 0], h // 4, :, 0])):
                return False
    return True


def pin_identical_keys(o):
    q, kc, vc, bt, L = case(2, 2, 4, 1, [37, 300], garbage=False)
    kc[:] = kc[0, 0, 0]
    out = o.attn_decode(q, kc, vc, bt, L, 0.3)
    for b in range(2):
        _, V = dense(kc, vc, bt, b, int(L[b]), 0)
        if not np.allclose(out[b], V.mean(axis=0)[None, :], rtol=1e-12, atol=1e-15):
            return False
    return True


def pin_zero_query(o):
    q, kc, vc, bt, L = case(3, 2, 6, 3, [5, 90])
    q[:] = 0
    out = o.attn_decode(q, kc, vc, bt, L, 0.088)
    for b in range(2):
        for h in range(6):
            _, V = dense(kc, vc, bt, b, int(L[b]), h // 2)
            if not np.allclose(out[b, h], V.mean(axis=0), rtol=1e-12, atol=1e-15):
                return False
    return True


def pin_value_per_head(o):
    """V constant g + 1 on key/value head g: query head h must read head h // G."""
    q, kc, vc, bt, L = case(4, 2, 12, 3, [17, 64])
    for g in range(3):
        vc[:, g] = f64_bf16(g + 1.0)
    out = o.attn_decode(q, kc, vc, bt, L, 0.088)
    return all(np.allclose(out[b, h], h // 4 + 1.0, rtol=1e-12, atol=0) for b in range(2) for h in range(12))


def pin_torch_sdpa(o):
    B, Hq, Hkv = 4, 8, 2
    q, kc, vc, bt, L = case(5, B, Hq, Hkv, [1, 16, 33, 250])
    scale = 1 / np.sqrt(D)
    out = o.attn_decode(q, kc, vc, bt, L, scale)
    for b in range(B):
        Ks, Vs = zip(*(dense(kc, vc, bt, b, int(L[b]), g) for g in range(Hkv)))
        k = torch.from_numpy(np.stack(Ks)).repeat_interleave(Hq // Hkv, dim=0)[None]  # [1, Hq, L, D]
        v = torch.from_numpy(np.stack(Vs)).repeat_interleave(Hq // Hkv, dim=0)[None]
        qq = torch.from_numpy(bf16_f64(q[b]))[None, :, None, :]
        ref = torch.nn.functional.scaled_dot_product_attention(qq, k, v, scale=scale)[0, :, 0, :].numpy()
        if not np.allclose(out[b], ref, rtol=1e-10, atol=1e-13):
            return False
    return True


def pin_page_relabelling(o):
    q, kc, vc, bt, L = case(6, 3, 4, 2, [20, 47, 100])
    out = o.attn_decode(q, kc, vc, bt, L, 0.1)
    rng = np.random.default_rng(66)
    pi = rng.permutation(kc.shape[0])  # new page index of old page p: pi[p]
    kc2, vc2 = np.empty_like(kc), np.empty_like(vc)
    kc2[pi], vc2[pi] = kc, vc
    bt2 = np.where(bt >= 0, pi[np.clip(bt, 0, None)], bt).astype(np.int32)
    return np.array_equal(out, o.attn_decode(q, kc2, vc2, bt2, L, 0.1))


def pin_past_context(o):
    """Bytes past a context (slots of its last page, unused pages) do not matter."""
    q, kc, vc, bt, L = case(7, 2, 4, 1, [21, 50])
    out = o.attn_decode(q, kc, vc, bt, L, 0.1)
    _, kz, vz, _, _ = case(7, 2, 4, 1, [21, 50], garbage=False)
    mask_k, mask_v = kc == NAN_BF16, vc == NAN_BF16
    kz[mask_k], vz[mask_v] = 0, 0
    return np.all(np.isfinite(out)) and np.array_equal(out, o.attn_decode(q, kz, vz, bt, L, 0.1))


def pin_scale_into_query(o):
    """scale 2s with q equals scale s with 2q (both exact doublings in fp64)."""
    q, kc, vc, bt, L = case(8, 2, 4, 2, [30, 77])
    q2 = f64_bf16(2.0 * bf16_f64(q))
    return np.array_equal(o.attn_decode(q, kc, vc, bt, L, 0.2), o.attn_decode(q2, kc, vc, bt, L, 0.1))


def pin_empty_context(o):
    q, kc, vc, bt, L = case(9, 2, 4, 2, [0, 5])
    out = o.attn_decode(q, kc, vc, bt, L, 0.1)
    return np.all(out[0] == 0) and np.all(np.isfinite(out[1])) and np.any(out[1] != 0)


PINS = [pin_single_token, pin_identical_keys, pin_zero_query, pin_value_per_head, pin_torch_sdpa,
        pin_page_relabelling, pin_past_context, pin_scale_into_query, pin_empty_context]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_attn_oracle_pin(pin):
    assert pin(oracle)


# ---------------------------------------------------------------- planted mistakes

MUTANTS = {
    "head_modulo": ("const int g = h / G;", "const int g = h % Hkv;"),
    "no_scale": ("                s *= scale;\n", "                s *= 1.0;\n"),
    "drop_last_token": ("for (int j = 0; j < L; j++) {\n                const int64_t pg = block_table[(int64_t)b * max_pages + j / P];\n                const uint16_t *kv = kc + ((pg * Hkv + g) * P + j % P) * (int64_t)D;\n                double s = 0.0;\n                for (int d = 0; d < D; d++) s += attn_dec_bf16(qv[d]) * attn_dec_bf16(kv[d]);\n                const double e",
                        "for (int j = 0; j < L - 1; j++) {\n                const int64_t pg = block_table[(int64_t)b * max_pages + j / P];\n                const uint16_t *kv = kc + ((pg * Hkv + g) * P + j % P) * (int64_t)D;\n                double s = 0.0;\n                for (int d = 0; d < D; d++) s += attn_dec_bf16(qv[d]) * attn_dec_bf16(kv[d]);\n                const double e"),
    "values_token_major": ("ov[d] += e * attn_dec_bf16(vp[(int64_t)d * P + j % P]);",
                           "ov[d] += e * attn_dec_bf16(vp[(int64_t)(j % P) * D + d]);"),
    "whole_last_page": ("        const int L = ctx[b];\n", "        const int L = (ctx[b] + P - 1) / P * P;\n"),
    "no_normalise": ("for (int d = 0; d < D; d++) ov[d] /= den;", "(void)den;"),
    "key_slot_by_page": ("(pg * Hkv + g) * P + j % P) * (int64_t)D;\n                double s = 0.0;\n                for (int d = 0; d < D; d++) s += attn_dec_bf16(qv[d]) * attn_dec_bf16(kv[d]);\n                const double e",
                         "(pg * Hkv + g) * P + j / P) * (int64_t)D;\n                double s = 0.0;\n                for (int d = 0; d < D; d++) s += attn_dec_bf16(qv[d]) * attn_dec_bf16(kv[d]);\n                const double e"),
}


def build_variant(tmp_path, name, old, new):
    src = open(ATTN_SRC).read()
    assert src.count(old) == 1, f"mutation site for {name} not unique"
    path = tmp_path / f"{name}.c"
    path.write_text(src.replace(old, new))
    so = tmp_path / f"lib{name}.so"
    subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-std=c11", "-pthread", "-ffp-contract=off", "-o",
                           str(so), MOE_SRC, str(path), "-lm"])
    spec = importlib.util.spec_from_file_location(f"oracle_attn_{name}", INIT)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    mod._LIB = str(so)
    mod._lib = None
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_attn_mutant_is_caught(tmp_path, name):
    old, new = MUTANTS[name]
    mod = build_variant(tmp_path, name, old, new)
    failed = []
    for pin in PINS:
        try:
            ok = pin(mod)
        except Exception:  # noqa: BLE001 -- a crash or a rejected input also catches it
            ok = False
        if not ok:
            failed.append(pin.__name__)
    assert failed, f"mutant {name} passes every pin"
