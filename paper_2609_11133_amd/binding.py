"""ctypes binding of ``libmoe_decode.so`` (C ABI in ``include/moe_decode.h`` and
``include/attn_decode.h``).

Argument marshalling only: every step of the decode layer runs in the library's HIP
kernels.  Functions carry the C names; pointer arguments accept a torch tensor
(its ``data_ptr()``), a plain integer address or ``None`` (NULL).  A non-OK status
raises :class:`MoEDecodeError` with the library's message.  Loading fails loudly when
the library has not been built.
"""
from __future__ import annotations

import ctypes
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("MOE_DECODE_LIB") or os.path.join(_PKG, "libmoe_decode.so")

MOE_OK, MOE_ERR_INVALID, MOE_ERR_UNSUPPORTED, MOE_ERR_WORKSPACE, MOE_ERR_HIP = 0, -1, -2, -3, -4
MOE_DTYPE_F32, MOE_DTYPE_BF16 = 0, 1
MOE_WFMT_FP8_E4M3_B128, MOE_WFMT_MXFP4_E2M1_B32, MOE_WFMT_NVFP4_E2M1_B16 = 0, 1, 2
MOE_STAGE_ROUTE, MOE_STAGE_W13, MOE_STAGE_W2, MOE_STAGE_COMBINE, MOE_N_STAGES = 0, 1, 2, 3, 4
MOE_WLAYOUT_ROW_MAJOR, MOE_WLAYOUT_TILED16 = 0, 1
STAGE_NAMES = ["route", "w13", "w2", "combine"]


class moe_decode_config(ctypes.Structure):
    _fields_ = [
        ("hidden", ctypes.c_int32),
        ("n_experts", ctypes.c_int32),
        ("inter", ctypes.c_int32),
        ("max_topk", ctypes.c_int32),
        ("max_tokens", ctypes.c_int32),
        ("act_dtype", ctypes.c_int32),
        ("router_dtype", ctypes.c_int32),
        ("wfmt", ctypes.c_int32),
        ("mfma_min_tokens", ctypes.c_int32),
        ("weight_layout", ctypes.c_int32),
        ("screen_min_tokens", ctypes.c_int32),
        ("reserved", ctypes.c_int32 * 5),
    ]


class moe_decode_stats(ctypes.Structure):
    _fields_ = [
        ("n_tokens", ctypes.c_int32),
        ("n_active", ctypes.c_int32),
        ("n_active_mfma", ctypes.c_int32),
        ("n_fallback", ctypes.c_int32),
        ("n_exact_logits", ctypes.c_int32),
        ("route_screened", ctypes.c_int32),
        ("active_weight_bytes", ctypes.c_int64),
    ]


class attn_decode_config(ctypes.Structure):
    _fields_ = [
        ("n_q_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("page_size", ctypes.c_int32),
        ("max_batch", ctypes.c_int32),
        ("max_pages_per_seq", ctypes.c_int32),
        ("fused_merge_max_splits", ctypes.c_int32),
        ("reserved", ctypes.c_int32 * 3),
    ]


class MoEDecodeError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{message} (status {status})")
        self.status = status


_lib = None


def lib():
    """The loaded library; raises if it is missing (no fallback path exists)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is not built: the MoE decode layer has no CPU or Python fallback. "
                "Build it with `python -c 'import __graft_entry__ as g; g.build()'`."
            )
        L = ctypes.CDLL(LIB_PATH)
        P, I32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        cfgp = ctypes.POINTER(moe_decode_config)
        L.moe_decode_workspace_bytes.restype = SZ
        L.moe_decode_workspace_bytes.argtypes = [cfgp]
        L.moe_decode_expert_weight_bytes.restype = SZ
        L.moe_decode_expert_weight_bytes.argtypes = [cfgp]
        L.moe_decode_expert_scale_bytes.restype = SZ
        L.moe_decode_expert_scale_bytes.argtypes = [cfgp]
        L.moe_decode_init.restype = ctypes.c_int
        L.moe_decode_init.argtypes = [cfgp, P, SZ, ctypes.POINTER(P)]
        L.moe_decode_forward.restype = ctypes.c_int
        L.moe_decode_forward.argtypes = [P, P, P, I32, P, P, P, P, I32, P, P, P]
        L.moe_decode_forward_noalloc.restype = ctypes.c_int
        L.moe_decode_forward_noalloc.argtypes = [cfgp, P, P, I32, P, P, P, P, I32, P, P, P]
        L.moe_decode_pack_weights.restype = ctypes.c_int
        L.moe_decode_pack_weights.argtypes = [cfgp, P, P, P, P, P, I32]
        L.moe_decode_route.restype = ctypes.c_int
        L.moe_decode_route.argtypes = [P, P, P, I32, P, P, I32, P, P, P]
        L.moe_decode_get_stats.restype = ctypes.c_int
        L.moe_decode_get_stats.argtypes = [P, ctypes.POINTER(moe_decode_stats), P]
        L.moe_decode_profile_enable.restype = ctypes.c_int
        L.moe_decode_profile_enable.argtypes = [P, I32]
        L.moe_decode_profile_read.restype = ctypes.c_int
        L.moe_decode_profile_read.argtypes = [P, P, ctypes.POINTER(I32)]
        L.moe_decode_free.restype = None
        L.moe_decode_free.argtypes = [P]
        L.moe_decode_status_string.restype = ctypes.c_char_p
        L.moe_decode_status_string.argtypes = [ctypes.c_int]
        L.moe_decode_last_error.restype = ctypes.c_char_p
        L.moe_decode_last_error.argtypes = [P]
        acfgp = ctypes.POINTER(attn_decode_config)
        L.attn_decode_workspace_bytes.restype = SZ
        L.attn_decode_workspace_bytes.argtypes = [acfgp]
        L.attn_decode_workspace_init.restype = ctypes.c_int
        L.attn_decode_workspace_init.argtypes = [acfgp, P, SZ, P]
        L.attn_decode_forward.restype = ctypes.c_int
        L.attn_decode_forward.argtypes = [acfgp, P, SZ, P, P, P, P, ctypes.c_int64, P, P, I32, ctypes.c_float, P]
        L.attn_decode_last_error.restype = ctypes.c_char_p
        L.attn_decode_last_error.argtypes = []
        _lib = L
    return _lib


def _addr(p):
    if p is None:
        return None
    if isinstance(p, int):
        return p
    return p.data_ptr()


def _check(status: int, handle=None):
    if status != MOE_OK:
        msg = lib().moe_decode_last_error(handle).decode()
        raise MoEDecodeError(status, msg or lib().moe_decode_status_string(status).decode())


def make_config(hidden, n_experts, inter, max_topk, max_tokens, act_dtype=MOE_DTYPE_BF16,
                router_dtype=MOE_DTYPE_BF16, wfmt=MOE_WFMT_FP8_E4M3_B128, mfma_min_tokens=0,
                screen_min_tokens=0, weight_layout=0) -> moe_decode_config:
    c = moe_decode_config()
    c.hidden, c.n_experts, c.inter, c.max_topk, c.max_tokens = hidden, n_experts, inter, max_topk, max_tokens
    c.act_dtype, c.router_dtype, c.wfmt, c.mfma_min_tokens = act_dtype, router_dtype, wfmt, mfma_min_tokens
    c.screen_min_tokens = screen_min_tokens
    c.weight_layout = weight_layout
    return c


def moe_decode_workspace_bytes(cfg: moe_decode_config) -> int:
    return int(lib().moe_decode_workspace_bytes(ctypes.byref(cfg)))


def moe_decode_expert_weight_bytes(cfg: moe_decode_config) -> int:
    return int(lib().moe_decode_expert_weight_bytes(ctypes.byref(cfg)))


def moe_decode_expert_scale_bytes(cfg: moe_decode_config) -> int:
    return int(lib().moe_decode_expert_scale_bytes(ctypes.byref(cfg)))


def moe_decode_init(cfg: moe_decode_config, workspace, workspace_bytes: int) -> int:
    h = ctypes.c_void_p()
    _check(lib().moe_decode_init(ctypes.byref(cfg), _addr(workspace), workspace_bytes, ctypes.byref(h)))
    return h.value


def moe_decode_forward(h, stream, x, n_tokens, router_w, router_bias, expert_w, scales, topk, y,
                       topk_ids=None, topk_weights=None):
    _check(lib().moe_decode_forward(h, stream, _addr(x), n_tokens, _addr(router_w), _addr(router_bias),
                                    _addr(expert_w), _addr(scales), topk, _addr(y), _addr(topk_ids),
                                    _addr(topk_weights)), h)


def moe_decode_forward_noalloc(cfg: moe_decode_config, stream, x, n_tokens, router_w, router_bias, expert_w, scales,
                               topk, y, topk_ids=None, topk_weights=None):
    """One decode step on the library's static device scratch array (no handle, no
    workspace, no allocation)."""
    _check(lib().moe_decode_forward_noalloc(ctypes.byref(cfg), stream, _addr(x), n_tokens, _addr(router_w),
                                            _addr(router_bias), _addr(expert_w), _addr(scales), topk, _addr(y),
                                            _addr(topk_ids), _addr(topk_weights)))


def moe_decode_pack_weights(cfg: moe_decode_config, stream, src, dst, n_experts: int, src_scales=None,
                            dst_scales=None):
    """Enqueue the row-major -> packed 16-row tile conversion of n_experts experts
    (scales too for MXFP4 and NVFP4 weights)."""
    _check(lib().moe_decode_pack_weights(ctypes.byref(cfg), stream, _addr(src), _addr(dst), _addr(src_scales),
                                         _addr(dst_scales), n_experts))


def moe_decode_route(h, stream, x, n_tokens, router_w, router_bias, topk, logits=None, topk_ids=None,
                     topk_weights=None):
    _check(lib().moe_decode_route(h, stream, _addr(x), n_tokens, _addr(router_w), _addr(router_bias), topk,
                                  _addr(logits), _addr(topk_ids), _addr(topk_weights)), h)


def moe_decode_get_stats(h, n_experts: int | None = None):
    """Returns (stats, counts list or None)."""
    st = moe_decode_stats()
    counts = (ctypes.c_int32 * n_experts)() if n_experts else None
    _check(lib().moe_decode_get_stats(h, ctypes.byref(st), counts), h)
    return st, (list(counts) if counts is not None else None)


def moe_decode_profile_enable(h, max_calls: int):
    _check(lib().moe_decode_profile_enable(h, max_calls), h)


def moe_decode_profile_read(h, max_calls: int):
    """Returns a list of per-call [route, w13, w2, combine] stage times in ms."""
    buf = (ctypes.c_float * (max(max_calls, 1) * MOE_N_STAGES))()
    n = ctypes.c_int32()
    _check(lib().moe_decode_profile_read(h, buf, ctypes.byref(n)), h)
    return [list(buf[c * MOE_N_STAGES:(c + 1) * MOE_N_STAGES]) for c in range(n.value)]


def moe_decode_free(h):
    lib().moe_decode_free(h)


def moe_decode_status_string(status: int) -> str:
    return lib().moe_decode_status_string(status).decode()


def moe_decode_last_error(h) -> str:
    return lib().moe_decode_last_error(h).decode()


class MoEDecode:
    """A handle plus its device workspace (a torch uint8 tensor on ``device``).

    ``forward`` enqueues one decode step on torch's current stream of that device.
    """

    def __init__(self, cfg: moe_decode_config, device="cuda"):
        import torch

        self.cfg = cfg
        self.nbytes = moe_decode_workspace_bytes(cfg)
        if self.nbytes == 0:
            _check(lib().moe_decode_init(ctypes.byref(cfg), None, 0, ctypes.byref(ctypes.c_void_p())))
        self.workspace = torch.empty(self.nbytes + 256, dtype=torch.uint8, device=device)
        base = self.workspace.data_ptr()
        self._ws_addr = (base + 255) // 256 * 256
        self.handle = moe_decode_init(cfg, self._ws_addr, self.nbytes)
        self.device = self.workspace.device

    def stream(self):
        import torch

        return torch.cuda.current_stream(self.device).cuda_stream

    def forward(self, x, n_tokens, router_w, router_bias, expert_w, scales, topk, y, topk_ids=None,
                topk_weights=None):
        moe_decode_forward(self.handle, self.stream(), x, n_tokens, router_w, router_bias, expert_w, scales, topk,
                           y, topk_ids, topk_weights)

    def route(self, x, n_tokens, router_w, router_bias, topk, logits=None, topk_ids=None, topk_weights=None):
        moe_decode_route(self.handle, self.stream(), x, n_tokens, router_w, router_bias, topk, logits, topk_ids,
                         topk_weights)

    def stats(self):
        return moe_decode_get_stats(self.handle, self.cfg.n_experts)

    def close(self):
        if getattr(self, "handle", None):
            moe_decode_free(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ---------------------------------------------------------------- decode attention


def make_attn_config(n_q_heads, n_kv_heads, max_batch, max_pages_per_seq, head_dim=128, page_size=16,
                     fused_merge_max_splits=0):
    return attn_decode_config(n_q_heads, n_kv_heads, head_dim, page_size, max_batch, max_pages_per_seq,
                              fused_merge_max_splits)


def attn_decode_workspace_init(cfg, workspace, workspace_bytes, stream):
    st = lib().attn_decode_workspace_init(ctypes.byref(cfg), _addr(workspace), workspace_bytes, stream)
    if st != 0:
        raise MoEDecodeError(st, lib().attn_decode_last_error().decode() or "attn_decode_workspace_init failed")


def attn_decode_workspace_bytes(cfg: attn_decode_config) -> int:
    return int(lib().attn_decode_workspace_bytes(ctypes.byref(cfg)))


def attn_decode_forward(cfg, workspace, workspace_bytes, stream, q, k_cache, v_cache, n_pages, block_table, ctx_lens,
                        batch, scale, out):
    st = lib().attn_decode_forward(ctypes.byref(cfg), _addr(workspace), workspace_bytes, stream, _addr(q),
                                   _addr(k_cache), _addr(v_cache), n_pages, _addr(block_table), _addr(ctx_lens),
                                   batch, scale, _addr(out))
    if st != MOE_OK:
        raise MoEDecodeError(st, lib().attn_decode_last_error().decode() or "attn_decode_forward failed")


class AttnDecode:
    """A configuration plus its device workspace (a torch uint8 tensor on ``device``);
    ``forward`` enqueues one decode step of attention on torch's current stream."""

    def __init__(self, cfg: attn_decode_config, device="cuda"):
        import torch

        self.cfg = cfg
        self.nbytes = attn_decode_workspace_bytes(cfg)
        if self.nbytes == 0:
            raise MoEDecodeError(MOE_ERR_INVALID, "invalid attention configuration")
        self.workspace = torch.empty(self.nbytes + 256, dtype=torch.uint8, device=device)
        self._ws_addr = (self.workspace.data_ptr() + 255) // 256 * 256
        self.device = self.workspace.device
        attn_decode_workspace_init(cfg, self._ws_addr, self.nbytes, torch.cuda.current_stream(self.device).cuda_stream)

    def forward(self, q, k_cache, v_cache, n_pages, block_table, ctx_lens, batch, scale, out):
        import torch

        stream = torch.cuda.current_stream(self.device).cuda_stream
        attn_decode_forward(self.cfg, self._ws_addr, self.nbytes, stream, q, k_cache, v_cache, n_pages, block_table,
                            ctx_lens, batch, scale, out)
