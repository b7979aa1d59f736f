"""TEST INFRASTRUCTURE -- numpy front end of the fp64 CPU oracles (``moe_oracle.c``, the MoE
decode layer; ``attn_oracle.c``, decode attention over a paged KV cache).

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the HIP library and
never imports it.  See the C files for the definitions they implement.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRCS = [os.path.join(_HERE, "moe_oracle.c"), os.path.join(_HERE, "attn_oracle.c")]
_LIB = os.path.join(_HERE, "liboracle.so")

DT_F32, DT_BF16 = 0, 1
WF_FP8, WF_MXFP4, WF_NVFP4 = 0, 1, 2


def build(force: bool = True) -> str:
    """Compile ``liboracle.so`` with gcc: plain -O2, no fast-math, no FMA contraction."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(
            ["gcc", "-O2", "-fPIC", "-shared", "-std=c11", "-pthread", "-ffp-contract=off", "-o", tmp, *_SRCS, "-lm"]
        )
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        p, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
        lib.oracle_dec_e4m3.restype = ctypes.c_double
        lib.oracle_dec_e4m3.argtypes = [ctypes.c_uint8]
        lib.oracle_dec_e2m1.restype = ctypes.c_double
        lib.oracle_dec_e2m1.argtypes = [ctypes.c_uint8]
        lib.oracle_dec_e8m0.restype = ctypes.c_double
        lib.oracle_dec_e8m0.argtypes = [ctypes.c_uint8]
        lib.oracle_dec_bf16.restype = ctypes.c_double
        lib.oracle_dec_bf16.argtypes = [ctypes.c_uint16]
        lib.oracle_logit.restype = ctypes.c_float
        lib.oracle_logit.argtypes = [p, i32, p, i32, i64, p]
        lib.oracle_route_token.restype = None
        lib.oracle_route_token.argtypes = [p, i32, p, i32, p, i64, i32, i32, p, p, p, p]
        lib.oracle_forward.restype = ctypes.c_int
        lib.oracle_forward.argtypes = [
            i64, i32, i64, i32, i32, i32, p, i64, p, p, p, p, i32, p, i64, i32, p, p, p, p
        ]
        lib.oracle_attn_decode.restype = ctypes.c_int
        lib.oracle_attn_decode.argtypes = [i32, i32, i32, i32, i32, p, p, p, i64, p, i32, p, ctypes.c_double, p]
        lib.oracle_expert_ffn.restype = ctypes.c_int
        lib.oracle_expert_ffn.argtypes = [i64, i32, i64, i32, p, p, i32, p, p]
        _lib = lib
    return _lib


def _ptr(a):
    if a is None:
        return None
    assert isinstance(a, np.ndarray) and a.flags["C_CONTIGUOUS"], "oracle inputs must be C-contiguous numpy arrays"
    return a.ctypes.data


def _dtype_of(a: np.ndarray) -> int:
    if a.dtype == np.uint16:
        return DT_BF16
    if a.dtype == np.float32:
        return DT_F32
    raise TypeError(f"activations/router weights must be bf16 bits (uint16) or float32, got {a.dtype}")


def dec_e4m3(c: int) -> float:
    return _load().oracle_dec_e4m3(c)


def dec_e2m1(c: int) -> float:
    return _load().oracle_dec_e2m1(c)


def dec_e8m0(c: int) -> float:
    return _load().oracle_dec_e8m0(c)


def dec_bf16(c: int) -> float:
    return _load().oracle_dec_bf16(c)


def logit(x_row: np.ndarray, w_row: np.ndarray, bias: float | None = None) -> float:
    """Canonical router logit (O1) of one token row against one router row."""
    x_row = np.ascontiguousarray(x_row)
    w_row = np.ascontiguousarray(w_row)
    b = None if bias is None else np.array([bias], np.float32)
    return float(
        _load().oracle_logit(_ptr(x_row), _dtype_of(x_row), _ptr(w_row), _dtype_of(w_row), x_row.shape[-1], _ptr(b))
    )


def route_token(x_row, router_w, bias, k):
    """O1-O4 for one token: (logits f32 [E], ids int32 [k], w f64 [k], p f64 [E])."""
    x_row = np.ascontiguousarray(x_row)
    router_w = np.ascontiguousarray(router_w)
    E, H = router_w.shape
    l = np.empty(E, np.float32)
    ids = np.empty(k, np.int32)
    w = np.empty(k, np.float64)
    p = np.empty(E, np.float64)
    b = None if bias is None else np.ascontiguousarray(bias, np.float32)
    _load().oracle_route_token(
        _ptr(x_row), _dtype_of(x_row), _ptr(router_w), _dtype_of(router_w), _ptr(b), H, E, k,
        _ptr(l), _ptr(ids), _ptr(w), _ptr(p)
    )
    return l, ids, w, p


def forward(x, router_w, bias, expert_w, scales, k, inter, wfmt, tokens=None, threads=1):
    """The whole layer (O1-O7) for ``tokens`` (all tokens if None).

    ``x`` [T,H] bf16 bits (uint16) or float32; ``router_w`` [E,H] likewise; ``bias`` [E]
    float32 or None; ``expert_w`` uint8 [E, expert bytes]; ``scales`` [E, ...] (float32
    for FP8, uint8 for MXFP4 and NVFP4).  Returns ``(logits f32 [n,E], ids int32 [n,k], w f64 [n,k],
    y f64 [n,H])``.
    """
    x = np.ascontiguousarray(x)
    router_w = np.ascontiguousarray(router_w)
    expert_w = np.ascontiguousarray(expert_w)
    scales = np.ascontiguousarray(scales)
    T, H = x.shape
    E = router_w.shape[0]
    tok = None if tokens is None else np.ascontiguousarray(np.asarray(tokens, np.int64))
    n = T if tok is None else tok.shape[0]
    logits = np.empty((n, E), np.float32)
    ids = np.empty((n, k), np.int32)
    w = np.empty((n, k), np.float64)
    y = np.empty((n, H), np.float64)
    b = None if bias is None else np.ascontiguousarray(bias, np.float32)
    rc = _load().oracle_forward(
        H, E, inter, _dtype_of(x), _dtype_of(router_w), wfmt, _ptr(x), T, _ptr(router_w), _ptr(b),
        _ptr(expert_w), _ptr(scales), k, _ptr(tok), n, threads, _ptr(logits), _ptr(ids), _ptr(w), _ptr(y)
    )
    if rc != 0:
        raise ValueError("oracle_forward rejected its arguments")
    return logits, ids, w, y


def expert_ffn(expert_w, scales, e, xv, hidden, inter, wfmt):
    """O6 alone: one fp64 token vector through expert ``e``; returns o [H] fp64."""
    expert_w = np.ascontiguousarray(expert_w)
    scales = np.ascontiguousarray(scales)
    xv = np.ascontiguousarray(xv, np.float64)
    o = np.empty(hidden, np.float64)
    rc = _load().oracle_expert_ffn(hidden, expert_w.shape[0], inter, wfmt, _ptr(expert_w), _ptr(scales), e,
                                   _ptr(xv), _ptr(o))
    if rc != 0:
        raise ValueError("oracle_expert_ffn rejected its arguments")
    return o


def attn_decode(q, k_cache, v_cache, block_table, ctx, scale):
    """Decode attention over a paged KV cache (``attn_oracle.c``), fp64.

    q [B, Hq, D] bf16 bits (uint16); k_cache [n_pages, Hkv, P, D] and v_cache
    [n_pages, Hkv, D, P] bf16 bits; block_table [B, max_pages] int32; ctx [B] int32;
    returns o [B, Hq, D] float64."""
    q = np.ascontiguousarray(q, np.uint16)
    k_cache = np.ascontiguousarray(k_cache, np.uint16)
    v_cache = np.ascontiguousarray(v_cache, np.uint16)
    block_table = np.ascontiguousarray(block_table, np.int32)
    ctx = np.ascontiguousarray(ctx, np.int32)
    B, Hq, D = q.shape
    n_pages, Hkv, P, D2 = k_cache.shape
    assert D2 == D and v_cache.shape == (n_pages, Hkv, D, P)
    assert block_table.shape[0] == B and ctx.shape == (B,)
    o = np.empty((B, Hq, D), np.float64)
    rc = _load().oracle_attn_decode(B, Hq, Hkv, D, P, _ptr(q), _ptr(k_cache), _ptr(v_cache), n_pages,
                                    _ptr(block_table), block_table.shape[1], _ptr(ctx), float(scale), _ptr(o))
    if rc != 0:
        raise ValueError("oracle_attn_decode: inconsistent sizes or page index out of range")
    return o
