"""The C-ABI library loads, exports every symbol of include/moe_decode.h, and rejects
invalid arguments before enqueuing anything (runs without a GPU: nothing here
reaches a HIP call)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "moe_decode.h")


@pytest.fixture(scope="module")
def B():
    from paper_2609_11133_amd import binding

    if not os.path.exists(binding.LIB_PATH):
        from paper_2609_11133_amd import build

        build.build(force=True)
    binding.lib()
    return binding


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(moe_decode_\w+)\s*\(", src)))


def test_every_declared_symbol_is_exported(B):
    names = declared_functions()
    assert len(names) >= 10
    lib = ctypes.CDLL(B.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


def test_no_oracle_or_generator_symbols_in_library(B):
    out = os.popen(f"nm -D --defined-only {B.LIB_PATH}").read()
    assert "oracle_" not in out and "synth_" not in out


def cfg(B, **kw):
    base = dict(hidden=512, n_experts=16, inter=256, max_topk=4, max_tokens=32)
    base.update(kw)
    return B.make_config(**base)


def test_workspace_bytes_and_sizes(B):
    c = cfg(B)
    assert B.moe_decode_workspace_bytes(c) > 0
    assert B.moe_decode_expert_weight_bytes(c) == 3 * 512 * 256
    assert B.moe_decode_expert_scale_bytes(c) == 4 * 3 * 4 * 2
    c4 = cfg(B, wfmt=B.MOE_WFMT_MXFP4_E2M1_B32)
    assert B.moe_decode_expert_weight_bytes(c4) == 3 * 512 * 256 // 2
    assert B.moe_decode_expert_scale_bytes(c4) == 3 * 512 * 256 // 32
    c5 = cfg(B, wfmt=B.MOE_WFMT_NVFP4_E2M1_B16)
    assert B.moe_decode_expert_weight_bytes(c5) == 3 * 512 * 256 // 2
    assert B.moe_decode_expert_scale_bytes(c5) == 16 + 3 * 512 * 256 // 16
    assert B.moe_decode_workspace_bytes(c5) > 0


@pytest.mark.parametrize(
    "kw,code",
    [
        (dict(hidden=500), -1),
        (dict(hidden=0), -1),
        (dict(inter=100), -1),
        (dict(hidden=128, wfmt=1), -1),  # MXFP4 needs multiples of 256
        (dict(n_experts=0), -1),
        (dict(n_experts=2000), -1),
        (dict(max_topk=17), -1),
        (dict(max_topk=0), -1),
        (dict(max_tokens=0), -1),
        (dict(max_tokens=4096), -1),
        (dict(act_dtype=7), -1),
        (dict(wfmt=3), -1),
        (dict(hidden=128, wfmt=2), -1),  # NVFP4 needs multiples of 256
        (dict(wfmt=2, act_dtype=0), -2),  # NVFP4 needs bf16 activations
    ],
)
def test_invalid_configs_rejected(B, kw, code):
    c = cfg(B, **kw)
    assert B.moe_decode_workspace_bytes(c) == 0
    with pytest.raises(B.MoEDecodeError) as ei:
        B.moe_decode_init(c, 1 << 20, 1 << 30)
    assert ei.value.status == code
    assert B.moe_decode_last_error(None)


def test_reserved_must_be_zero(B):
    c = cfg(B)
    c.reserved[3] = 1
    assert B.moe_decode_workspace_bytes(c) == 0


def test_workspace_checks(B):
    c = cfg(B)
    need = B.moe_decode_workspace_bytes(c)
    for ws, nb in [(None, need), (4096 + 16, need), (4096, need - 1)]:
        with pytest.raises(B.MoEDecodeError) as ei:
            B.moe_decode_init(c, ws, nb)
        assert ei.value.status == B.MOE_ERR_WORKSPACE


FAKE = 1 << 32  # a 256-aligned address; nothing dereferences it in these tests


def make_handle(B):
    c = cfg(B)
    return B.moe_decode_init(c, FAKE, B.moe_decode_workspace_bytes(c))


@pytest.mark.parametrize(
    "change,needle",
    [
        (dict(n_tokens=33), "n_tokens"),
        (dict(n_tokens=-1), "n_tokens"),
        (dict(topk=5), "topk"),
        (dict(topk=0), "topk"),
        (dict(x=None), "x is NULL"),
        (dict(x=FAKE + 8), "x is not 16-byte aligned"),
        (dict(router_w=FAKE + 4), "router_w"),
        (dict(expert_w=None), "expert_w"),
        (dict(scales=FAKE + 2), "scales"),
        (dict(y=None), "y is NULL"),
        (dict(y=FAKE), "alias"),
        (dict(router_bias=FAKE + 1), "router_bias"),
        (dict(topk_ids=FAKE + 2), "topk_ids"),
    ],
)
def test_forward_validates_before_launch(B, change, needle):
    h = make_handle(B)
    args = dict(stream=None, x=FAKE, n_tokens=4, router_w=FAKE + 4096, router_bias=None, expert_w=FAKE + 8192,
                scales=FAKE + 12288, topk=2, y=FAKE + 16384, topk_ids=None, topk_weights=None)
    args.update(change)
    with pytest.raises(B.MoEDecodeError) as ei:
        B.moe_decode_forward(h, **args)
    assert ei.value.status == B.MOE_ERR_INVALID
    assert needle in str(ei.value)
    B.moe_decode_free(h)


def test_zero_tokens_is_a_no_op(B):
    h = make_handle(B)
    B.moe_decode_forward(h, None, FAKE, 0, FAKE + 4096, None, FAKE + 8192, FAKE + 12288, 2, FAKE + 16384)
    st, counts = B.moe_decode_get_stats(h, 16)
    assert st.n_tokens == 0 and st.n_active == 0 and counts == [0] * 16
    B.moe_decode_free(h)


def test_stats_before_forward_is_an_error(B):
    h = make_handle(B)
    with pytest.raises(B.MoEDecodeError):
        B.moe_decode_get_stats(h, 16)
    B.moe_decode_free(h)


def test_status_strings(B):
    for s in (0, -1, -2, -3, -4):
        assert B.moe_decode_status_string(s)
    B.lib().moe_decode_free(None)  # NULL is ignored


# ---------------------------------------------------------------- decode attention (include/attn_decode.h)

ATTN_HEADER = os.path.join(ROOT, "include", "attn_decode.h")


def test_every_attention_symbol_is_exported(B):
    src = re.sub(r"/\*.*?\*/", "", open(ATTN_HEADER).read(), flags=re.S)
    names = sorted(set(re.findall(r"\b(attn_decode_\w+)\s*\(", src)))
    assert names == ["attn_decode_forward", "attn_decode_last_error", "attn_decode_workspace_bytes",
                     "attn_decode_workspace_init"]
    lib = ctypes.CDLL(B.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


def test_attention_workspace_bytes(B):
    c = B.make_attn_config(64, 4, 24, 128)  # 2048 tokens: 8 splits of 256
    parts = 24 * 4 * 8 * 16
    rnd = lambda n: (n + 255) // 256 * 256  # noqa: E731
    assert B.attn_decode_workspace_bytes(c) == rnd(parts * 128 * 4) + rnd(parts * 8) + 24 * 4 * 4


@pytest.mark.parametrize(
    "kw,code",
    [
        (dict(n_q_heads=64, n_kv_heads=3), -1),  # not a multiple
        (dict(n_q_heads=68, n_kv_heads=2), -2),  # 34 query heads per key/value head
        (dict(n_q_heads=8, n_kv_heads=0), -1),
        (dict(head_dim=64), -2),
        (dict(page_size=32), -2),
        (dict(max_batch=0), -1),
        (dict(max_batch=5000), -1),
        (dict(max_pages_per_seq=0), -1),
        (dict(fused_merge_max_splits=17), -1),
    ],
)
def test_attention_invalid_configs_rejected(B, kw, code):
    base = dict(n_q_heads=64, n_kv_heads=4, max_batch=8, max_pages_per_seq=16)
    base.update(kw)
    c = B.make_attn_config(**base)
    assert B.attn_decode_workspace_bytes(c) == 0
    with pytest.raises(B.MoEDecodeError) as e:
        B.attn_decode_forward(c, 256, 1 << 20, None, 16, 32, 48, 1, 64, 64, 1, 0.1, 80)
    assert e.value.status == code


@pytest.mark.parametrize(
    "change,needle",
    [
        (dict(batch=9), "batch"),
        (dict(scale=0.0), "scale"),
        (dict(scale=float("nan")), "scale"),
        (dict(n_pages=0), "n_pages"),
        (dict(q=0), "q is NULL"),
        (dict(k_cache=24), "k_cache must be 16-byte aligned"),
        (dict(out=16), "alias"),
        (dict(block_table=0), "block_table"),
        (dict(ctx_lens=2), "ctx_lens"),
        (dict(workspace=0), "workspace"),
        (dict(workspace_bytes=100), "workspace of 100 bytes"),
    ],
)
def test_attention_forward_validates_before_launch(B, change, needle):
    """Every check fails before a launch: no GPU is touched (the pointers are fake)."""
    c = B.make_attn_config(64, 4, 8, 16)
    args = dict(workspace=256, workspace_bytes=B.attn_decode_workspace_bytes(c), q=16, k_cache=32, v_cache=48,
                n_pages=4, block_table=64, ctx_lens=68, batch=8, scale=0.1, out=80)
    args.update(change)
    with pytest.raises(B.MoEDecodeError) as e:
        B.attn_decode_forward(c, args["workspace"], args["workspace_bytes"], None, args["q"], args["k_cache"],
                              args["v_cache"], args["n_pages"], args["block_table"], args["ctx_lens"], args["batch"],
                              args["scale"], args["out"])
    assert needle in str(e.value)


@pytest.mark.parametrize(
    "change,needle",
    [
        (dict(workspace=0), "workspace"),
        (dict(workspace=300), "workspace"),
        (dict(workspace_bytes=100), "workspace of 100 bytes"),
    ],
)
def test_attention_workspace_init_validates(B, change, needle):
    c = B.make_attn_config(64, 4, 8, 16)
    args = dict(workspace=256, workspace_bytes=B.attn_decode_workspace_bytes(c))
    args.update(change)
    with pytest.raises(B.MoEDecodeError) as e:
        B.attn_decode_workspace_init(c, args["workspace"], args["workspace_bytes"], None)
    assert needle in str(e.value)


def test_attention_config_struct(B):
    assert ctypes.sizeof(B.attn_decode_config) == 40
    c = B.make_attn_config(64, 4, 8, 16, fused_merge_max_splits=-1)
    assert B.attn_decode_workspace_bytes(c) > 0
    c.reserved[2] = 1
    assert B.attn_decode_workspace_bytes(c) == 0


def test_attention_zero_batch_is_a_no_op(B):
    c = B.make_attn_config(64, 4, 8, 16)
    B.attn_decode_forward(c, 256, B.attn_decode_workspace_bytes(c), None, 16, 32, 48, 4, 64, 68, 0, 0.1, 80)


def test_struct_sizes_match_header(B):
    """The ctypes mirrors of the C structs: 16 int32 config words, stats of 6 int32 + int64."""
    import ctypes

    assert ctypes.sizeof(B.moe_decode_config) == 64
    assert ctypes.sizeof(B.moe_decode_stats) == 32
    assert B.moe_decode_stats.active_weight_bytes.offset == 24
    c = cfg(B)
    c.screen_min_tokens = -1
    assert B.moe_decode_workspace_bytes(c) > 0
    c.screen_min_tokens = 7
    assert B.moe_decode_workspace_bytes(c) > 0


# ---------------------------------------------------------------- packed 16-row tile layout

@pytest.mark.parametrize(
    "kw,code",
    [
        (dict(weight_layout=2), -1),
        (dict(weight_layout=1, mfma_min_tokens=-1), -2),  # the GEMV path reads row-major weights
        (dict(weight_layout=1, mfma_min_tokens=4), -2),
    ],
)
def test_weight_layout_checks(B, kw, code):
    c = cfg(B, **kw)
    assert B.moe_decode_workspace_bytes(c) == 0
    with pytest.raises(B.MoEDecodeError) as e:
        B.moe_decode_init(c, 256, 1 << 30)
    assert e.value.status == code


def test_weight_layout_accepted(B):
    for wfmt in (0, 1, 2):
        for mm in (0, 1):
            assert B.moe_decode_workspace_bytes(cfg(B, weight_layout=1, wfmt=wfmt, mfma_min_tokens=mm)) > 0


@pytest.mark.parametrize(
    "change,needle",
    [
        (dict(n_experts=0), "n_experts"),
        (dict(n_experts=17), "n_experts"),
        (dict(src=0), "NULL"),
        (dict(dst=8), "aligned"),
        (dict(dst=256 + 1024), "overlap"),
        (dict(ssrc=1 << 31), "keep their layout"),  # FP8 scales are not converted
        (dict(wfmt=1), "need src_scales"),
        (dict(wfmt=2), "need src_scales"),
        (dict(wfmt=2, ssrc=1 << 31, sdst=(1 << 31) + 2), "4-byte aligned"),
        (dict(wfmt=2, ssrc=1 << 31, sdst=(1 << 31) + 64), "scales overlap"),
    ],
)
def test_pack_validates_before_launch(B, change, needle):
    """Every check of moe_decode_pack_weights fails before a launch (fake pointers)."""
    args = dict(n_experts=2, src=256, dst=1 << 30, wfmt=0, ssrc=None, sdst=None)
    args.update(change)
    c = cfg(B, wfmt=args["wfmt"])
    with pytest.raises(B.MoEDecodeError) as e:
        B.moe_decode_pack_weights(c, None, args["src"], args["dst"], args["n_experts"], args["ssrc"], args["sdst"])
    assert needle in str(e.value)
