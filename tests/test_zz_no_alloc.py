"""moe_decode_forward_noalloc (workspace in the library's static device array) against
moe_decode_forward (caller workspace), both through the C ABI: two calls in a row on
the static array, the second with fewer tokens, and a change of configuration in
between; selection, routing weights and outputs must be bitwise equal to the handle
path's, which the parity tests check against the oracle (checked here too on a small
layer)."""
import sys

import numpy as np
import pytest

import oracle
from paper_2609_11133_amd import configs as C
from paper_2609_11133_amd import workload as W
from paper_2609_11133_amd.configs import LayerConfig

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_11133_amd import binding as B

    B.lib()
    return torch.device("cuda:0")


class Layer:
    def __init__(self, cfg, dev, max_tokens, layout, seed=1234):
        from paper_2609_11133_amd import binding as B

        self.cfg, self.dev = cfg, dev
        self.hl = W.host_layer(cfg, seed=seed)
        self.bc = W.binding_config(cfg, max_tokens, 0, 0, layout)
        self.rw = W.to_device(self.hl.router_w, dev)
        self.bias = W.to_device(self.hl.bias, dev)
        self.ew = W.to_device(self.hl.expert_w, dev)
        self.sc = W.to_device(self.hl.scales, dev)
        if layout == 1:
            packed = torch.empty_like(self.ew)
            nv = cfg.wfmt != "fp8"
            psc = torch.empty_like(self.sc) if nv else None
            B.moe_decode_pack_weights(self.bc, torch.cuda.current_stream(dev).cuda_stream, self.ew, packed,
                                      cfg.n_experts, self.sc if nv else None, psc)
            torch.cuda.synchronize(dev)
            self.ew = packed
            if nv:
                self.sc = psc
        self.m = B.MoEDecode(self.bc, device=dev)

    def outputs(self, T):
        k = self.cfg.topk
        return (W.empty_y(self.cfg, T, self.dev), torch.full((T, k), -1, dtype=torch.int32, device=self.dev),
                torch.zeros((T, k), dtype=torch.float32, device=self.dev))

    def handle_path(self, xd, T):
        y, ids, wts = self.outputs(T)
        self.m.forward(xd, T, self.rw, self.bias, self.ew, self.sc, self.cfg.topk, y, ids, wts)
        return y, ids, wts

    def noalloc_path(self, xd, T):
        from paper_2609_11133_amd import binding as B

        y, ids, wts = self.outputs(T)
        B.moe_decode_forward_noalloc(self.bc, torch.cuda.current_stream(self.dev).cuda_stream, xd, T, self.rw,
                                     self.bias, self.ew, self.sc, self.cfg.topk, y, ids, wts)
        return y, ids, wts


def same(a, b, label):
    ya, ia, wa = a
    yb, ib, wb = b
    assert torch.equal(ia, ib), f"{label}: expert selection differs"
    assert torch.equal(wa.view(torch.int32), wb.view(torch.int32)), f"{label}: routing weights differ"
    assert torch.equal(ya.view(torch.int16) if ya.dtype == torch.bfloat16 else ya.view(torch.int32),
                       yb.view(torch.int16) if yb.dtype == torch.bfloat16 else yb.view(torch.int32)), \
        f"{label}: outputs differ"


SMALL = LayerConfig("noalloc-small", 512, 16, 4, 256, "bf16", "bf16", "fp8", "normal:0.5", [])


def test_noalloc_matches_forward(dev):
    """235B-shaped layer on packed weights (the benchmark's launch configuration,
    max_tokens 64): T = 64, then T = 8 on the same static array; then a small layer
    of another configuration (T = 13, then 5), checked against the oracle too; then
    the 235B layer again at T = 33."""
    big = Layer(C.QWEN3_235B, dev, 64, 1)
    small = Layer(SMALL, dev, 16, 1, seed=77)
    plan = [(big, 64, 11), (big, 8, 12), (small, 13, 13), (small, 5, 14), (big, 33, 15)]
    for lay, T, batch in plan:
        label = f"{lay.cfg.name} T={T}"
        say(f"[noalloc] {label}")
        x = W.host_x(lay.cfg, T, batch=batch)
        xd = W.to_device(x, dev)
        ref = lay.handle_path(xd, T)
        got = lay.noalloc_path(xd, T)
        torch.cuda.synchronize(dev)
        same(got, ref, label)
        if lay is small:
            _, io, wo, yo = oracle.forward(x, lay.hl.router_w, lay.hl.bias, lay.hl.expert_w, lay.hl.scales,
                                           lay.cfg.topk, lay.cfg.inter, lay.cfg.wfmt_id, threads=4)
            assert np.array_equal(got[1].cpu().numpy(), io)
            err = np.abs(W.y_to_f64(got[0]) - yo).max()
            assert err <= 2e-2 * np.abs(yo).max(), f"{label}: max|err| {err}"
        say(f"[noalloc] {label}: bitwise equal to moe_decode_forward")


def test_noalloc_rejects_oversized(dev):
    """A configuration whose workspace exceeds the static array is refused before
    anything is enqueued (the 480B-shaped layer at max_tokens 256 needs about 92 MiB)."""
    from paper_2609_11133_amd import binding as B

    bc = W.binding_config(C.QWEN3_480B, 256)
    assert B.moe_decode_workspace_bytes(bc) > 64 << 20
    dummy = torch.zeros(1 << 16, dtype=torch.uint8, device=dev)
    with pytest.raises(B.MoEDecodeError) as ei:
        B.moe_decode_forward_noalloc(bc, torch.cuda.current_stream(dev).cuda_stream, dummy, 1, dummy, None, dummy,
                                     dummy, 8, dummy)
    assert ei.value.status == B.MOE_ERR_WORKSPACE
    assert "static scratch" in str(ei.value)
