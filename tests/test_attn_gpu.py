"""Parity of the HIP decode attention (through the C ABI) with the fp64 oracle.

Tolerance, per output row (sequence, query head): max|err| <= 1e-2 * max|ref row|.  It
is derived from the arithmetic: the output is rounded once to bf16 (2^-9 relative) and
the probabilities enter the P.V product rounded to bf16 (2^-9 relative each, averaging
out over the context), with fp32 accumulation; 1e-2 leaves about a fivefold margin.
Small cases cover every split/page boundary and ragged tail, empty contexts, group
sizes 1-16, bytes past the contexts holding NaN, and page indices outside the cache,
with the splits merged inside the split kernel and by the second kernel (the two give
the same bits when each split is one 256-token piece), and with several pieces per split
(online softmax inside a workgroup); the full-size agentic steps of both models are
compared on every row, the 32K-token long-context step on sampled sequences."""
import sys

import numpy as np
import pytest

import oracle
from paper_2609_11133_amd import attn_workload as A

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

TOL = 1e-2


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_11133_amd import binding as B

    B.lib()  # fails loudly if the library is missing
    return torch.device("cuda:0")


def bf16_to_f64(t):
    return (t.cpu().numpy().view(np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def run_gpu(cfg, h, dev, scale, max_pages=None, fused=0):
    from paper_2609_11133_amd import binding as B

    mp = h.block_table.shape[1] if max_pages is None else max_pages
    acfg = B.make_attn_config(cfg.n_q_heads, cfg.n_kv_heads, cfg.batch, mp, fused_merge_max_splits=fused)
    m = B.AttnDecode(acfg, device=dev)
    d = A.to_device(h, dev)
    out = torch.full((cfg.batch, cfg.n_q_heads, 128), 0x7FC1, dtype=torch.int16, device=dev)
    say(f"[attn] {cfg.name} B={cfg.batch} Hq={cfg.n_q_heads} Hkv={cfg.n_kv_heads} max_pages={mp} "
        f"L=[{int(h.ctx.min())}, {int(h.ctx.max())}] fused_merge_max_splits={fused}")
    m.forward(d["q"], d["k_cache"], d["v_cache"], h.n_pages, d["block_table"], d["ctx"], cfg.batch, scale, out)
    torch.cuda.synchronize(dev)
    return out, m, d


def check(got, ref, rows=None, label=""):
    rows = range(ref.shape[0]) if rows is None else rows
    worst = 0.0
    for i, b in enumerate(rows):
        for hh in range(ref.shape[1]):
            r, g = ref[i, hh], got[b, hh]
            assert np.all(np.isfinite(g)), f"{label} b={b} h={hh}: non-finite output"
            mr = np.abs(r).max()
            err = np.abs(g - r).max()
            if mr == 0:
                assert err == 0, f"{label} b={b} h={hh}: expected zeros"
                continue
            worst = max(worst, err / mr)
            assert err <= TOL * mr, f"{label} b={b} h={hh}: max err {err:.3g} > {TOL} * {mr:.3g}"
    say(f"[attn] {label}: worst max|err|/max|ref| per row {worst:.3g}")


SMALL_LENS = [0, 1, 15, 16, 17, 63, 64, 65, 255, 256, 257, 511, 700, 1025]


@pytest.mark.parametrize("hq,hkv", [(64, 4), (24, 2), (8, 8), (4, 1), (32, 2)])
def test_small_cases(dev, hq, hkv):
    cfg = A.AttnConfig(f"small-{hq}x{hkv}", hq, hkv, len(SMALL_LENS), "standard")
    h = A.host_attn(cfg, seed=301 + hq, ctx=np.array(SMALL_LENS, np.int32))
    scale = 1 / np.sqrt(128)
    out, _, _ = run_gpu(cfg, h, dev, scale)  # 5 splits at most: merged in the split kernel
    ref = oracle.attn_decode(h.q, h.k_cache, h.v_cache, h.block_table, h.ctx, scale)
    check(bf16_to_f64(out), ref, label=cfg.name)
    out2, _, _ = run_gpu(cfg, h, dev, scale, fused=-1)  # merged by the second kernel
    assert torch.equal(out, out2), "the two merges differ"
    for lim in (2, 1):  # 5 pieces: 3 per split (2 splits), or all 5 in one workgroup
        out3, _, _ = run_gpu(cfg, h, dev, scale, fused=lim)
        check(bf16_to_f64(out3), ref, label=f"{cfg.name} at most {lim} splits")


@pytest.mark.parametrize("name", ["qwen3-235b-a22b-attn-agentic", "qwen3-coder-480b-a35b-tp4-attn-agentic"])
def test_fused_merge_matches_two_kernels(dev, name):
    """Full-size steps: the in-kernel merge (last workgroup per sequence and key/value
    head) and the second kernel give the same bits; two further steps on the same
    workspace, the second with fewer sequences, reuse the counters the first left at
    zero."""
    cfg = A.ATTN_BY_NAME[name]
    h = A.host_attn(cfg, draw=4)
    scale = 1 / np.sqrt(128)
    out, m, d = run_gpu(cfg, h, dev, scale)
    out2, _, _ = run_gpu(cfg, h, dev, scale, fused=-1)
    assert torch.equal(out, out2)
    out3 = torch.empty_like(out)
    m.forward(d["q"], d["k_cache"], d["v_cache"], h.n_pages, d["block_table"], d["ctx"], cfg.batch, scale, out3)
    nb = cfg.batch // 3
    out4 = torch.full_like(out, 0x7FC1)
    m.forward(d["q"], d["k_cache"], d["v_cache"], h.n_pages, d["block_table"], d["ctx"], nb, scale, out4)
    torch.cuda.synchronize(dev)
    assert torch.equal(out3, out) and torch.equal(out4[:nb], out[:nb])
    assert torch.all(out4[nb:] == 0x7FC1)  # rows past the batch untouched


def test_block_table_wider_than_contexts(dev):
    """A block-table row longer than any context: more splits than any sequence uses."""
    cfg = A.AttnConfig("wide-table", 16, 2, 5, "standard")
    h = A.host_attn(cfg, seed=311, ctx=np.array([3, 40, 300, 0, 17], np.int32), max_pages=200)
    scale = 0.05
    out, _, _ = run_gpu(cfg, h, dev, scale)
    ref = oracle.attn_decode(h.q, h.k_cache, h.v_cache, h.block_table, h.ctx, scale)
    check(bf16_to_f64(out), ref, label=cfg.name)


def test_page_outside_cache_reads_zeros(dev):
    """A page index outside [0, n_pages) reads as a page of zeros, with no fault."""
    cfg = A.AttnConfig("bad-page", 8, 2, 3, "standard")
    h = A.host_attn(cfg, seed=321, ctx=np.array([40, 70, 33], np.int32))
    h.block_table[0, 1] = h.n_pages + 5
    h.block_table[2, 0] = -3
    scale = 0.09
    out, _, _ = run_gpu(cfg, h, dev, scale)
    # the oracle's view: those pages replaced by an appended zero page
    zk = np.zeros((1,) + h.k_cache.shape[1:], np.uint16)
    zv = np.zeros((1,) + h.v_cache.shape[1:], np.uint16)
    bt = h.block_table.copy()
    bt[0, 1] = bt[2, 0] = h.n_pages
    ref = oracle.attn_decode(h.q, np.concatenate([h.k_cache, zk]), np.concatenate([h.v_cache, zv]), bt, h.ctx, scale)
    check(bf16_to_f64(out), ref, label=cfg.name)


def test_bitwise_repeatable(dev):
    cfg = A.ATTN_BY_NAME["qwen3-235b-a22b-attn-standard"]
    h = A.host_attn(cfg, draw=3)
    out, m, d = run_gpu(cfg, h, dev, 1 / np.sqrt(128))
    out2 = torch.empty_like(out)
    m.forward(d["q"], d["k_cache"], d["v_cache"], h.n_pages, d["block_table"], d["ctx"], cfg.batch, 1 / np.sqrt(128),
              out2)
    torch.cuda.synchronize(dev)
    assert torch.equal(out, out2)


@pytest.mark.parametrize("name", ["qwen3-235b-a22b-attn-agentic", "qwen3-coder-480b-a35b-tp4-attn-agentic",
                                  "qwen3-235b-a22b-attn-standard"])
def test_full_size_step(dev, name):
    cfg = A.ATTN_BY_NAME[name]
    h = A.host_attn(cfg, draw=1)
    scale = 1 / np.sqrt(128)
    out, _, _ = run_gpu(cfg, h, dev, scale)
    ref = oracle.attn_decode(h.q, h.k_cache, h.v_cache, h.block_table, h.ctx, scale)
    check(bf16_to_f64(out), ref, label=name)


def test_long_context_sampled(dev):
    """32K-token contexts (128 pieces per sequence), checked on three sampled sequences:
    8 splits of 16 pieces merged in the split kernel (the default on 256 compute units:
    at most three workgroups per unit), and 128 one-piece splits merged by the second
    kernel; a call with fewer sequences on the same workspace repeats their rows bitwise."""
    cfg = A.ATTN_BY_NAME["qwen3-235b-a22b-attn-long32k"]
    h = A.host_attn(cfg, draw=2)
    scale = 1 / np.sqrt(128)
    rows = [0, 11, cfg.batch - 1]
    ref = oracle.attn_decode(h.q[rows], h.k_cache, h.v_cache, h.block_table[rows], h.ctx[rows], scale)
    for fused in (0, -1):
        out, m, d = run_gpu(cfg, h, dev, scale, fused=fused)
        check(bf16_to_f64(out), ref, rows=rows, label=f"{cfg.name} fused_merge_max_splits={fused}")
        if fused == 0:
            # the split count follows the configuration, not the call: a call with the first
            # 12 sequences on the same workspace gives their rows bit for bit
            nb = 12
            out2 = torch.full_like(out, 0x7FC1)
            m.forward(d["q"], d["k_cache"], d["v_cache"], h.n_pages, d["block_table"], d["ctx"], nb, scale, out2)
            torch.cuda.synchronize(dev)
            assert torch.equal(out2[:nb], out[:nb]) and torch.all(out2[nb:] == 0x7FC1)


def test_capacity_sized_config_short_contexts(dev):
    """The agentic step on a configuration sized for 32K-token contexts (2048-page rows,
    so the grid has 8 splits of up to 16 pieces): every sequence spreads its own 3-8
    pieces one per split, matches the oracle per row, and a call with fewer sequences on
    the same workspace repeats their rows bit for bit."""
    cfg = A.ATTN_BY_NAME["qwen3-235b-a22b-attn-agentic-cap32k"]
    h = A.host_attn(cfg, draw=5)
    assert h.block_table.shape[1] == 2048
    scale = 1 / np.sqrt(128)
    out, m, d = run_gpu(cfg, h, dev, scale)
    ref = oracle.attn_decode(h.q, h.k_cache, h.v_cache, h.block_table, h.ctx, scale)
    check(bf16_to_f64(out), ref, label=cfg.name)
    nb = 7
    out2 = torch.full_like(out, 0x7FC1)
    m.forward(d["q"], d["k_cache"], d["v_cache"], h.n_pages, d["block_table"], d["ctx"], nb, scale, out2)
    torch.cuda.synchronize(dev)
    assert torch.equal(out2[:nb], out[:nb]) and torch.all(out2[nb:] == 0x7FC1)

