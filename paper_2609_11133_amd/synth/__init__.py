"""Seeded synthetic inputs for the MoE decode layer (numpy front end of ``synth.c``).

Every tensor is a pure function of ``(seed, tag, layer/batch, index)``: the same
bytes come out on any machine and any slice can be regenerated on its own.  The
module holds no arithmetic of the layer itself; it only draws Gaussian values and
quantises weights into the formats the layer consumes (FP8-E4M3 with 128x128 fp32
block scales, MXFP4 = E2M1 with one E8M0 scale per 32 inputs, or NVFP4 = E2M1 with
one E4M3 scale per 16 inputs and one fp32 scale per matrix).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "synth.c")
_LIB = os.path.join(_HERE, "libsynth.so")

WFMT_FP8 = 0
WFMT_MXFP4 = 1
WFMT_NVFP4 = 2


def build(force: bool = True) -> str:
    """Compile ``libsynth.so`` with gcc (OpenMP)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(
            ["gcc", "-O2", "-msse4.1", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off", "-std=c11", "-o", tmp, _SRC, "-lm"]
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
        u64, u32, i64, p = ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int64, ctypes.c_void_p
        lib.synth_stream_key.restype = u64
        lib.synth_stream_key.argtypes = [u64, u32, u32, u32]
        lib.synth_normal_f64.argtypes = [u64, u64, u64, ctypes.c_double, p]
        lib.synth_bf16_from_f64.restype = ctypes.c_uint16
        lib.synth_bf16_from_f64.argtypes = [ctypes.c_double]
        lib.synth_e4m3_from_f64.restype = ctypes.c_uint8
        lib.synth_e4m3_from_f64.argtypes = [ctypes.c_double]
        lib.synth_e2m1_from_f64.restype = ctypes.c_uint8
        lib.synth_e2m1_from_f64.argtypes = [ctypes.c_double]
        lib.synth_x_bf16.argtypes = [u64, u32, i64, i64, p]
        lib.synth_normal_bf16.argtypes = [u64, u64, i64, ctypes.c_double, p]
        lib.synth_x_f32.argtypes = [u64, u32, i64, i64, p]
        lib.synth_router_bf16.argtypes = [u64, u32, i64, i64, p]
        lib.synth_router_f32.argtypes = [u64, u32, i64, i64, p]
        lib.synth_bias_normal.argtypes = [u64, u32, i64, ctypes.c_double, p]
        lib.synth_bias_zipf.argtypes = [u64, u32, i64, ctypes.c_double, p]
        lib.synth_expert_bytes.restype = i64
        lib.synth_expert_bytes.argtypes = [ctypes.c_int, i64, i64]
        lib.synth_expert_scale_bytes.restype = i64
        lib.synth_expert_scale_bytes.argtypes = [ctypes.c_int, i64, i64]
        lib.synth_experts.argtypes = [u64, u32, ctypes.c_int, i64, i64, i64, i64, p, p]
        _lib = lib
    return _lib


def _ptr(a: np.ndarray) -> int:
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data


TAGS = dict(x=1, router=2, bias=3, gate=4, up=5, down=6, perm=7, q=8, k=9, v=10)


def stream_key(seed: int, tag: str, layer: int, sub: int = 0) -> int:
    return int(_load().synth_stream_key(seed, TAGS[tag], layer, sub))


def normal(seed: int, tag: str, layer: int, sub: int, start: int, n: int, sigma: float = 1.0) -> np.ndarray:
    """Raw Gaussian draws (Irwin-Hall(12)) of one stream, as fp64."""
    out = np.empty(n, np.float64)
    _load().synth_normal_f64(stream_key(seed, tag, layer, sub), start, n, sigma, _ptr(out))
    return out


def normal_bf16(seed: int, tag: str, layer: int, sub: int, n: int, sigma: float = 1.0) -> np.ndarray:
    """n Gaussian draws of one stream times sigma, rounded to bf16 (uint16 bit patterns)."""
    out = np.empty(n, np.uint16)
    _load().synth_normal_bf16(stream_key(seed, tag, layer, sub), 0, n, sigma, _ptr(out))
    return out


def bf16_from_f64(v: float) -> int:
    return int(_load().synth_bf16_from_f64(v))


def e4m3_from_f64(v: float) -> int:
    return int(_load().synth_e4m3_from_f64(v))


def e2m1_from_f64(v: float) -> int:
    return int(_load().synth_e2m1_from_f64(v))


def x_bf16(seed: int, batch: int, T: int, H: int) -> np.ndarray:
    """Activations x[T,H] ~ N(0,1) rounded to bf16 (returned as uint16 bit patterns)."""
    out = np.empty((T, H), np.uint16)
    _load().synth_x_bf16(seed, batch, T, H, _ptr(out))
    return out


def x_f32(seed: int, batch: int, T: int, H: int) -> np.ndarray:
    out = np.empty((T, H), np.float32)
    _load().synth_x_f32(seed, batch, T, H, _ptr(out))
    return out


def router_bf16(seed: int, layer: int, E: int, H: int) -> np.ndarray:
    """Router weights W_r[E,H] ~ N(0, 1/sqrt(H)) rounded to bf16 (uint16 bit patterns)."""
    out = np.empty((E, H), np.uint16)
    _load().synth_router_bf16(seed, layer, E, H, _ptr(out))
    return out


def router_f32(seed: int, layer: int, E: int, H: int) -> np.ndarray:
    out = np.empty((E, H), np.float32)
    _load().synth_router_f32(seed, layer, E, H, _ptr(out))
    return out


def bias_normal(seed: int, layer: int, E: int, sd: float) -> np.ndarray:
    out = np.empty(E, np.float32)
    _load().synth_bias_normal(seed, layer, E, sd, _ptr(out))
    return out


def bias_zipf(seed: int, layer: int, E: int, s: float) -> np.ndarray:
    out = np.empty(E, np.float32)
    _load().synth_bias_zipf(seed, layer, E, s, _ptr(out))
    return out


def expert_bytes(wfmt: int, H: int, I: int) -> int:
    return int(_load().synth_expert_bytes(wfmt, H, I))


def expert_scale_bytes(wfmt: int, H: int, I: int) -> int:
    return int(_load().synth_expert_scale_bytes(wfmt, H, I))


def experts(seed: int, layer: int, wfmt: int, E: int, H: int, I: int, e0: int = 0, e1: int | None = None):
    """Quantised expert weights for experts [e0, e1) of one layer.

    Returns ``(w, s)``: ``w`` uint8 [n, expert_bytes], ``s`` [n, ...] float32 block
    scales (FP8), uint8 E8M0 scales (MXFP4), or uint8 bytes holding four fp32 matrix
    scales followed by E4M3 block scales (NVFP4), packed as the library expects.
    """
    if e1 is None:
        e1 = E
    n = e1 - e0
    w = np.empty((n, expert_bytes(wfmt, H, I)), np.uint8)
    sb = expert_scale_bytes(wfmt, H, I)
    s = np.empty((n, sb // 4), np.float32) if wfmt == WFMT_FP8 else np.empty((n, sb), np.uint8)
    _load().synth_experts(seed, layer, wfmt, e0, e1, H, I, _ptr(w), _ptr(s))
    return w, s
