"""Benchmark of the MoE decode layer on one MI355X.

A step is one decode step of one MoE layer (router, top-k, grouping, grouped
experts, combine) over one batch of T synthetic tokens, with all inputs resident in
HBM.  The headline workload is the Qwen3-Coder-480B-A35B-shaped layer (hidden 6144,
160 experts, top-8, SwiGLU intermediate 2560, FP8-E4M3 weights with 128x128 fp32
block scales, bf16 activations, router bias N(0, 0.5)) at T = 64, the largest batch
of its sweep at or below 64 tokens.  The same run times, and reports beside it, the
other workloads: the Qwen3-235B-A22B-shaped layer (hidden 4096, 128 experts, top-8,
I 1536) swept over T = 1/8/32/64, one GPU's TP4 share of the 480B-shaped layer, the
235B-shaped layer with MXFP4 and with NVFP4 weights (the Zipf-skewed batch of 256
tokens for both, and the NVFP4 sweep), the stack of 12 distinct 480B-shaped layers
decoded back to back over T = 1..256, and the decode-attention steps over a paged KV
cache (--no-stack, --no-attn and --also '' leave them out).

Cold-cache protocol: steps cycle over L copies of the layer's expert weights at
distinct HBM addresses and over a pool of 16 token batches, so consecutive steps
stream weights that are not resident in the 256 MB MALL or the L2s, as in a model
whose layers follow each other.

Printed: one JSON line with tokens/s (value), the layer-level HBM rate of the
unique activated-expert bytes, the sweep over the layer's batch sizes, the roofline
of the dominant kernel (gate/up projection, from HIP events around it on the
launch stream over a second timed region of K steps: events between kernels add a
launch gap at every boundary, so the headline steps are timed without them), board
power where readable, and the fp64 CPU oracle timed on this host's cores on a
bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import math
import os
import statistics
import sys
import threading
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0  # MI355X HBM3E, published
METRIC = "MoE decode-layer tokens/s and achieved HBM GB/s (% of peak) vs batch size"
CSRC = os.path.join(ROOT, "paper_2609_11133_amd", "csrc")
# sources the gate/up MFMA kernel is compiled from: a counter profile is valid only
# for the kernel it was taken on
W13_SOURCES = ["mfma.hip", "fp8split.h", "moe_internal.h"]


def w13_source_hash() -> str:
    h = hashlib.sha256()
    for f in W13_SOURCES:
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def w13_traffic(cfg, T):
    """HBM bytes per launch of the gate/up MFMA kernel from the committed counter
    profile of this workload (FETCH_SIZE + WRITE_SIZE, each scaled by what the same
    counter reads for a copy kernel of known size); None if there is no profile or
    the kernel sources changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"w13_mfma_{cfg.name}_T{T}_traffic.txt")
    if not os.path.exists(path):
        return None, "no counter profile for this workload"
    kv = {}
    with open(path) as fh:
        for line in fh:
            if ":" in line and not line.startswith((" ", "#")):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
    if kv.get("kernel_source_sha256") != w13_source_hash():
        return None, f"{os.path.relpath(path, ROOT)} was taken on an older kernel"
    return float(kv["traffic_bytes_per_launch"]), os.path.relpath(path, ROOT)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", default="qwen3-coder-480b-a35b", help="layer of the headline line")
    ap.add_argument("--also", default="qwen3-235b-a22b,qwen3-coder-480b-a35b-tp4,qwen3-235b-a22b-mxfp4-zipf,"
                                      "qwen3-235b-a22b-nvfp4,qwen3-235b-a22b-nvfp4-zipf",
                    help="comma-separated further layer configurations swept in the same run and reported under "
                         "other_layers ('' for none)")
    ap.add_argument("--no-attn", action="store_true", help="leave the decode-attention steps out of the default run")
    ap.add_argument("--no-stack", action="store_true", help="leave the 12-layer stack out of the default run")
    ap.add_argument("--tokens", type=int, default=None, help="T of the headline line (default: largest T <= 64)")
    ap.add_argument("--copies", type=int, default=0, help="weight copies cycled (0: enough for 8 GB)")
    ap.add_argument("--no-sweep", action="store_true",
                    help="the headline T only (no sweep, no stack, no attention steps)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-power", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target CPU work of the oracle sample")
    ap.add_argument("--attn", action="store_true",
                    help="decode attention over a paged KV cache instead of the MoE layer: one JSON line per "
                         "workload of attn_workload.ATTN_CONFIGS")
    ap.add_argument("--attn-merge-max-splits", type=int, default=0,
                    help="with --attn: at most this many splits per sequence, each walking one or more 256-token "
                         "pieces and merged inside the split kernel (0: library default 16, -1: one piece per split, "
                         "merged by a second kernel)")
    ap.add_argument("--stack", action="store_true",
                    help="time the stack of 12 distinct 480B-shaped layers decoded back to back, T = 1..256, also "
                         "with --no-sweep (the default run times it unless --no-stack)")
    ap.add_argument("--stack-steps", type=int, default=20)
    ap.add_argument("--layout", choices=["packed", "row-major"], default=None,
                    help="expert weight layout: packed 16-row tiles (default; converted once at setup by "
                         "moe_decode_pack_weights) or row-major")
    ap.add_argument("--screen-min-tokens", type=int, default=0,
                    help="tokens per step from which routing screens the logits (0: library default, -1: never)")
    ap.add_argument("--power-cap-probe", action="store_true",
                    help="read the board power cap, its range, the clocks and who may write the cap, then exit")
    ap.add_argument("--mstar", type=int, default=0,
                    help="tokens per expert from which MFMA tiles are used (0: library default, -1: GEMV only)")
    return ap.parse_args()


class PowerSampler:
    """Board power via amdsmi every 100 ms (None where unreadable)."""

    def __init__(self):
        self.samples = []
        self.ok = False
        try:
            import amdsmi

            amdsmi.amdsmi_init()
            self.amdsmi = amdsmi
            self.h = amdsmi.amdsmi_get_processor_handles()[0]
            self.read()
            self.ok = True
        except Exception as e:  # noqa: BLE001
            self.err = repr(e)

    def read(self):
        info = self.amdsmi.amdsmi_get_power_info(self.h)
        for key in ("socket_power", "current_socket_power", "average_socket_power"):
            v = info.get(key)
            if isinstance(v, (int, float)) and v > 0:
                return float(v)
        raise RuntimeError(f"no power field in {info}")

    def run(self, stop: threading.Event):
        while not stop.is_set():
            try:
                self.samples.append((time.perf_counter(), self.read()))
            except Exception:  # noqa: BLE001
                pass
            stop.wait(0.1)


def power_cap_probe():
    """The board power cap as this process sees it, read only: amdsmi's cap and
    range, the GPU and memory clocks, and the driver's sysfs cap files with their
    owner, mode and whether this user may write them.  A cap sweep needs a writable
    cap; the job pool these runs use allows no power-cap or clock setting at all."""
    rec = dict(euid=os.geteuid())
    try:
        import amdsmi

        amdsmi.amdsmi_init()
        h = amdsmi.amdsmi_get_processor_handles()[0]
    except Exception as e:  # noqa: BLE001
        rec["error"] = "amdsmi unavailable: " + repr(e)
        return rec

    def clocks():
        out = {}
        for name in ("GFX", "MEM"):
            try:
                out[name.lower()] = amdsmi.amdsmi_get_clock_info(h, getattr(amdsmi.AmdSmiClkType, name))
            except Exception as e:  # noqa: BLE001
                out[name.lower()] = repr(e)
        return out

    try:
        rec["cap_uW"] = amdsmi.amdsmi_get_power_cap_info(h, 0)
    except Exception as e:  # noqa: BLE001
        rec["cap_uW"] = repr(e)
    rec["clocks"] = clocks()
    files = []
    for p in sorted(glob.glob("/sys/class/drm/card*/device/hwmon/hwmon*/power1_cap")):
        try:
            st = os.stat(p)
            files.append(dict(path=p, mode=oct(st.st_mode & 0o777), uid=st.st_uid,
                              writable_by_this_user=os.access(p, os.W_OK)))
        except OSError as e:
            files.append(dict(path=p, error=repr(e)))
    rec["sysfs_power_cap_files"] = files
    try:
        amdsmi.amdsmi_shut_down()
    except Exception:  # noqa: BLE001
        pass
    return rec


def settle_hbm(dev, reserve_bytes=int(32e9), wait_s=3.0):
    """Reserve and release a large device block, then wait, before any weights are
    placed.  Right after a process that freed some 100 GB of mixed-size buffers (the
    GPU test suite), weight copies allocated at once streamed about 3% slower for the
    whole run (235B-shaped layer at T=64: 136k against 140k tokens/s); after this
    step, or after half a minute of idle, they run at the rate of a quiet device.
    Outside every timed region."""
    import torch

    block = torch.empty(reserve_bytes, dtype=torch.uint8, device=dev)
    torch.cuda.synchronize(dev)
    del block
    torch.cuda.empty_cache()
    time.sleep(wait_s)


def run_stack(args, dev):
    """Decode steps through a stack of distinct 480B-shaped layers (one handle, one
    stream, layer after layer with its own input batch), swept over T.  Weights are
    generated layer by layer on the host and kept on the device (about 90 GB), so no
    step finds its experts in the MALL."""
    import statistics

    import torch

    from paper_2609_11133_amd import binding as B
    from paper_2609_11133_amd import configs as C
    from paper_2609_11133_amd import workload as W

    cfg = C.QWEN3_480B_X12
    layout = 0 if args.layout == "row-major" else 1
    bcfg = W.binding_config(cfg, max(cfg.tokens), args.mstar, args.screen_min_tokens, layout)
    t0 = time.time()
    layers = []
    for li in range(cfg.layers):
        hl = W.host_layer(cfg, layer=li)
        ew = W.to_device(hl.expert_w, dev)
        if layout:  # converted once per layer, as at load time
            packed = torch.empty_like(ew)
            B.moe_decode_pack_weights(bcfg, torch.cuda.current_stream(dev).cuda_stream, ew, packed, cfg.n_experts)
            torch.cuda.synchronize(dev)
            ew = packed
        layers.append((W.to_device(hl.router_w, dev), W.to_device(hl.bias, dev), ew, W.to_device(hl.scales, dev)))
        del hl
        print(f"[stack] layer {li} resident ({time.time() - t0:.0f} s)", file=sys.stderr, flush=True)
    m = B.MoEDecode(bcfg, device=dev)
    stream = torch.cuda.current_stream(dev)
    Be = cfg.expert_bytes()
    out = {}
    for T in cfg.tokens:
        xs = [W.to_device(W.host_x(cfg, T, batch=li), dev) for li in range(cfg.layers)]
        ys = [W.empty_y(cfg, T, dev) for _ in range(2)]
        n_act = []
        for li, (rw, bias, ew, sc) in enumerate(layers):
            m.forward(xs[li], T, rw, bias, ew, sc, cfg.topk, ys[0])
            n_act.append(m.stats()[0].n_active)

        def step():
            for li, (rw, bias, ew, sc) in enumerate(layers):
                m.forward(xs[li], T, rw, bias, ew, sc, cfg.topk, ys[li & 1])

        for _ in range(2):
            step()
        torch.cuda.synchronize(dev)
        start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record(stream)
        for _ in range(args.stack_steps):
            step()
        end.record(stream)
        torch.cuda.synchronize(dev)
        ms = start.elapsed_time(end) / args.stack_steps
        bytes_step = sum(n_act) * Be
        out[str(T)] = [round(T / (ms * 1e-3), 1), round(ms * 1e3, 1),
                       round(bytes_step / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)]
        print(f"[stack] T={T}: {T / (ms * 1e-3):.0f} tok/s, {ms * 1e3:.0f} us per 12-layer step "
              f"({ms * 1e3 / cfg.layers:.1f} us per layer), {bytes_step / (ms * 1e-3) / 1e9:.0f} GB/s, "
              f"n_active {statistics.mean(n_act):.1f}", file=sys.stderr, flush=True)
        del xs, ys
    m.close()
    del layers
    torch.cuda.empty_cache()
    return dict(workload=f"{cfg.layers} distinct {cfg.name[:-4]}-shaped fp8 layers back to back, "
                         f"{cfg.layers * cfg.n_experts * Be / 1e9:.1f} GB of expert weights",
                steps=args.stack_steps, fields=["tokens_per_s", "us_per_stack_step", "frac_of_peak"], **out)


def run_attn(args, dev, emit=True):
    """Decode attention: per workload, B sequences' step time between HIP events over K
    steps that cycle KV-cache copies (>= 1 GB, so no step finds its cache in the MALL)
    and 4 length draws; GB/s = the context's K and V bytes per step / step time.
    Returns one record per workload; with `emit`, also prints each as a JSON line."""
    import numpy as np
    import torch

    from paper_2609_11133_amd import attn_workload as A
    from paper_2609_11133_amd import binding as B

    lines = []
    for cfg in A.ATTN_CONFIGS:
        draws = [A.host_attn(cfg, draw=d, garbage=False) for d in range(4)]
        mp = max(h.block_table.shape[1] for h in draws)
        nbytes = max(h.k_cache.nbytes + h.v_cache.nbytes for h in draws)
        copies = max(1, math.ceil(1e9 / nbytes))
        dd = []
        for h in draws:
            bt = np.zeros((cfg.batch, mp), np.int32)
            bt[:, : h.block_table.shape[1]] = h.block_table
            h.block_table = bt
            d0 = A.to_device(h, dev)
            dd.append([d0] + [dict(d0, k_cache=d0["k_cache"].clone(), v_cache=d0["v_cache"].clone())
                              for _ in range(copies - 1)])
        m = B.AttnDecode(B.make_attn_config(cfg.n_q_heads, cfg.n_kv_heads, cfg.batch, mp,
                                            fused_merge_max_splits=args.attn_merge_max_splits), device=dev)
        out = torch.empty((cfg.batch, cfg.n_q_heads, 128), dtype=torch.int16, device=dev)
        scale = 1 / math.sqrt(128)

        def step(i):
            h, d = draws[i % 4], dd[i % 4][(i // 4) % copies]
            m.forward(d["q"], d["k_cache"], d["v_cache"], h.n_pages, d["block_table"], d["ctx"], cfg.batch, scale, out)

        for i in range(args.warmup):
            step(i)
        stream = torch.cuda.current_stream(dev)
        start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize(dev)
        start.record(stream)
        for i in range(args.steps):
            step(i)
        end.record(stream)
        torch.cuda.synchronize(dev)
        ms = start.elapsed_time(end) / args.steps
        kv = statistics.mean(draws[i % 4].kv_bytes(cfg.n_kv_heads) for i in range(args.steps))
        ctx_mean = statistics.mean(float(h.ctx.mean()) for h in draws)
        gbs = kv / (ms * 1e-3) / 1e9
        line = {
            "metric": "decode attention steps: sequences/s and achieved HBM GB/s (% of peak)",
            "value": cfg.batch / (ms * 1e-3), "unit": "sequences/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": f"{cfg.name}: {cfg.batch} sequences, {cfg.n_q_heads} query / {cfg.n_kv_heads} "
                                   f"key-value heads, head dim 128, 16-token pages, {cfg.mix} context lengths "
                                   f"(mean {ctx_mean:.0f} tokens), block-table rows of {mp} pages",
                       "cold_cache": f"{copies} KV-cache copies x 4 draws"},
            "roofline": {"kernel": "attn_split_kernel + attn_combine_kernel (one step)", "bound": "hbm",
                         "achieved": gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": gbs / PEAK_HBM_GBS,
                         "bytes_per_step": kv},
        }
        print(f"[attn] {cfg.name}: {ms * 1e3:.1f} us/step, {gbs:.0f} GB/s ({gbs / PEAK_HBM_GBS:.3f} of peak), "
              f"mean context {ctx_mean:.0f}", file=sys.stderr, flush=True)
        if emit:
            print(json.dumps(line), flush=True)
        lines.append(line)
        del dd, m
        torch.cuda.empty_cache()
    return lines


def cpu_info():
    """Host cores the oracle may use: the affinity mask, the CPU share of this host's
    GPU jobs (OMP_NUM_THREADS where the job scheduler sets it) and the CPU model."""
    affinity = len(os.sched_getaffinity(0))
    share = os.environ.get("OMP_NUM_THREADS")
    share = int(share) if share and share.isdigit() and int(share) > 0 else None
    model = None
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return affinity, share, model


def bench_layer(args, dev, cfg, sweep_T, T_main, pool=16):
    """Time one layer configuration over its T sweep: tokens/s from an event-free
    region of K steps (plus five repetitions), per-kernel durations from a second
    region with the library's stage events, and board power over a steady loop at
    every T.  Returns (results by T, layout, copies, setup seconds, host layer)."""
    import torch

    from paper_2609_11133_amd import binding as B
    from paper_2609_11133_amd import workload as W

    Tmax = max(sweep_T)
    layer_bytes = cfg.n_experts * (cfg.expert_weight_bytes() + cfg.expert_scale_bytes())
    copies = args.copies or max(2, math.ceil(8e9 / layer_bytes))

    t0 = time.time()
    hl = W.host_layer(cfg)
    xs = {T: [W.to_device(W.host_x(cfg, T, batch=b), dev) for b in range(pool)] for T in sweep_T}
    rw, bias = W.to_device(hl.router_w, dev), W.to_device(hl.bias, dev)
    ew0, sc0 = W.to_device(hl.expert_w, dev), W.to_device(hl.scales, dev)
    layout = 0 if args.layout == "row-major" else 1
    bcfg = W.binding_config(cfg, Tmax, args.mstar, args.screen_min_tokens, layout)
    if layout:  # weights (and E2M1 scales) converted once, as at load time
        packed = torch.empty_like(ew0)
        nv = cfg.wfmt != "fp8"
        psc = torch.empty_like(sc0) if nv else None
        B.moe_decode_pack_weights(bcfg, torch.cuda.current_stream(dev).cuda_stream, ew0, packed, cfg.n_experts,
                                  sc0 if nv else None, psc)
        torch.cuda.synchronize(dev)
        ew0 = packed
        if nv:
            sc0 = psc
    ews = [ew0] + [ew0.clone() for _ in range(copies - 1)]
    scs = [sc0] + [sc0.clone() for _ in range(copies - 1)]
    setup_s = time.time() - t0

    m = B.MoEDecode(bcfg, device=dev)
    stream = torch.cuda.current_stream(dev)
    Be = cfg.expert_bytes()
    results = {}

    for T in sweep_T:
        ys = [W.empty_y(cfg, T, dev) for _ in range(2)]
        # unique activated experts of each pooled batch (deterministic per batch)
        n_act = []
        for b in range(pool):
            m.forward(xs[T][b], T, rw, bias, ews[0], scs[0], cfg.topk, ys[0])
            n_act.append(m.stats()[0].n_active)

        def step(i):
            c = i % copies
            m.forward(xs[T][i % pool], T, rw, bias, ews[c], scs[c], cfg.topk, ys[i & 1])

        for i in range(args.warmup):
            step(i)
        torch.cuda.synchronize(dev)
        # timed region: K steps between two events on the launch stream (events
        # between the kernels would add a launch gap at every boundary)
        start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize(dev)
        start.record(stream)
        for i in range(args.steps):
            step(i)
        end.record(stream)
        torch.cuda.synchronize(dev)
        ms = start.elapsed_time(end) / args.steps
        # repetitions: five more timed regions of K steps each (median and spread)
        reps = []
        for _ in range(5):
            r0, r1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            r0.record(stream)
            for i in range(args.steps):
                step(i)
            r1.record(stream)
            torch.cuda.synchronize(dev)
            reps.append(r0.elapsed_time(r1) / args.steps)
        # per-kernel durations: K more steps with the library's stage events recording
        # each kernel on the same stream
        B.moe_decode_profile_enable(m.handle, args.steps)
        for i in range(args.steps):
            step(i)
        torch.cuda.synchronize(dev)
        stages = B.moe_decode_profile_read(m.handle, args.steps)
        B.moe_decode_profile_enable(m.handle, 0)
        acts = [n_act[i % pool] for i in range(args.steps)]
        bytes_step = statistics.mean(acts) * Be
        st_ms = [statistics.mean(s[j] for s in stages) for j in range(B.MOE_N_STAGES)]
        w13_bytes = statistics.mean(a * cfg.w13_bytes() for a in acts)
        w2_bytes = statistics.mean(a * cfg.w2_bytes() for a in acts)
        w13_gbs = w13_bytes / (st_ms[B.MOE_STAGE_W13] * 1e-3) / 1e9
        w2_gbs = w2_bytes / (st_ms[B.MOE_STAGE_W2] * 1e-3) / 1e9
        exp_gbs = (w13_bytes + w2_bytes) / ((st_ms[1] + st_ms[2]) * 1e-3) / 1e9
        results[T] = dict(
            tokens_per_s=T / (ms * 1e-3),
            ms_per_step=ms,
            reps_ms_per_step=dict(n=len(reps), median=statistics.median(reps), stdev=statistics.stdev(reps)),
            n_active_mean=statistics.mean(acts),
            bytes_per_step=bytes_step,
            layer_GBs=bytes_step / (ms * 1e-3) / 1e9,
            layer_frac=bytes_step / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS,
            stage_ms={n: v for n, v in zip(B.STAGE_NAMES, st_ms)},
            w13_GBs=w13_gbs,
            w2_GBs=w2_gbs,
            experts_GBs=exp_gbs,
            experts_frac=exp_gbs / PEAK_HBM_GBS,
            w13_bytes_per_launch=w13_bytes,
        )
        print(f"[bench] {cfg.name} T={T}: {results[T]['tokens_per_s']:.0f} tok/s, {ms * 1e3:.1f} us/step "
              f"(5 reps: median {statistics.median(reps) * 1e3:.1f} +- {statistics.stdev(reps) * 1e3:.1f}), layer "
              f"{results[T]['layer_GBs']:.0f} GB/s, experts {exp_gbs:.0f} GB/s, stages(us) "
              + " ".join(f"{n}={v * 1e3:.1f}" for n, v in zip(B.STAGE_NAMES, st_ms)), file=sys.stderr, flush=True)

    # board power over a steady loop at each batch size (4 s at the headline one), and
    # over 2 s of an idle device (after 3 s of rest) for context
    if not args.no_power:
        ps = PowerSampler()
        if ps.ok:

            def sample(seconds, work):
                ps.samples = []
                stop = threading.Event()
                th = threading.Thread(target=ps.run, args=(stop,), daemon=True)
                th.start()
                n, tp0 = 0, time.perf_counter()
                while time.perf_counter() - tp0 < seconds:
                    n += work()
                dt = time.perf_counter() - tp0
                stop.set()
                th.join()
                watts = [w for _, w in ps.samples]
                return (statistics.mean(watts) if watts else None), len(watts), n, dt

            def loop_at(T):
                ys = [W.empty_y(cfg, T, dev) for _ in range(2)]
                ctr = [0]

                def work():
                    for _ in range(50):
                        n = ctr[0]
                        c = n % copies
                        m.forward(xs[T][n % pool], T, rw, bias, ews[c], scs[c], cfg.topk, ys[n & 1])
                        ctr[0] += 1
                    torch.cuda.synchronize(dev)
                    return 50

                return work

            torch.cuda.synchronize(dev)
            time.sleep(3.0)  # the board sensor averages over about a second
            idle_W, _, _, _ = sample(2.0, lambda: (time.sleep(0.05), 0)[1])
            for T in sweep_T:
                pw, ns, n, dt = sample(4.0 if T == T_main else 3.0, loop_at(T))
                if pw:
                    results[T]["power"] = dict(board_W=pw, samples=ns, tokens_per_J=(n * T / dt) / pw,
                                               idle_board_W=idle_W)
                    print(f"[power] {cfg.name} T={T}: {pw:.0f} W board (idle {idle_W or 0:.0f} W), "
                          f"{results[T]['power']['tokens_per_J']:.1f} tokens/J", file=sys.stderr, flush=True)
        else:
            for T in sweep_T:
                results[T]["power"] = dict(board_W=None, note="amdsmi power unreadable: " + getattr(ps, "err", "?"))
    m.close()
    del ews, scs, xs, ew0, sc0
    torch.cuda.empty_cache()
    return results, layout, copies, setup_s, hl


SWEEP_FIELDS = ["tokens_per_s", "us_per_step", "n_active_mean", "layer_frac", "w13_frac", "experts_frac",
                "route_us", "w13_us", "w2_us", "combine_us", "board_W", "tokens_per_J"]
OTHER_FIELDS = ["tokens_per_s", "us_per_step", "w13_frac", "experts_frac", "tokens_per_J"]


def sweep_row(r, fields):
    """One T of a layer as a list in the order of `fields`: the JSON line carries every
    workload of the run, so each T is a short row and the full per-T records go to stderr."""
    pw = r.get("power") or {}
    v = dict(tokens_per_s=round(r["tokens_per_s"], 1), us_per_step=round(r["ms_per_step"] * 1e3, 2),
             n_active_mean=round(r["n_active_mean"], 1), layer_frac=round(r["layer_frac"], 4),
             w13_frac=round(r["w13_GBs"] / PEAK_HBM_GBS, 4), experts_frac=round(r["experts_frac"], 4),
             board_W=round(pw["board_W"], 1) if pw.get("board_W") else None,
             tokens_per_J=round(pw["tokens_per_J"], 2) if pw.get("board_W") else None)
    for n in ("route", "w13", "w2", "combine"):
        v[n + "_us"] = round(r["stage_ms"][n] * 1e3, 1)
    return [v[f] for f in fields]


def sweep_json(results, fields=SWEEP_FIELDS):
    out = {"fields": fields}
    out.update({str(T): sweep_row(r, fields) for T, r in results.items()})
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "the benchmark runs on one GPU: the layer is measured at one GPU's share "
                                   "(the TP4 shard configuration); the library has no multi-GPU path",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    import torch

    from paper_2609_11133_amd import binding as B
    from paper_2609_11133_amd import configs as C
    from paper_2609_11133_amd import workload as W

    if not os.path.exists(B.LIB_PATH):
        import __graft_entry__

        __graft_entry__.build()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    settle_hbm(dev)
    if args.attn:
        run_attn(args, dev)
        return
    if args.power_cap_probe:
        print(json.dumps(power_cap_probe()), flush=True)
        return
    cfg = C.BY_NAME[args.config]
    small = [t for t in cfg.tokens if t <= 64]
    T_main = args.tokens or (max(small) if small else min(cfg.tokens))
    sweep_T = sorted(set(cfg.tokens) | {T_main}) if not args.no_sweep else [T_main]
    results, layout, copies, setup_s, hl = bench_layer(args, dev, cfg, sweep_T, T_main)

    # further layer configurations, timed the same way and reported beside the headline
    others = {}
    for name in [n for n in (args.also or "").split(",") if n and n != cfg.name]:
        ocfg = C.BY_NAME[name]
        ores, _, ocopies, osetup, _ = bench_layer(args, dev, ocfg, sorted(ocfg.tokens), max(ocfg.tokens))
        others[name] = dict(
            layer=f"H {ocfg.hidden}, E {ocfg.n_experts}, top-{ocfg.topk}, I {ocfg.inter}, {ocfg.wfmt}"
                  + (f", bias {ocfg.bias}" if ocfg.bias else ""),
            copies=ocopies, **{str(T): sweep_row(r, OTHER_FIELDS) for T, r in ores.items()})

    # the fp64 oracle on this host's cores, on a bounded sample of the headline batch
    cpu = None
    if not args.no_cpu_baseline:
        import oracle

        affinity, share, model = cpu_info()
        threads = min(affinity, share) if share else affinity
        x_host = W.host_x(cfg, T_main, batch=0)
        tp = time.perf_counter()
        oracle.forward(x_host, hl.router_w, hl.bias, hl.expert_w, hl.scales, cfg.topk, cfg.inter, cfg.wfmt_id,
                       tokens=[0], threads=threads)
        t1 = time.perf_counter() - tp
        # one token keeps at most k threads busy: with more threads and tokens a token
        # costs about t1 * min(threads, k) / threads of wall time
        per_tok = max(t1 * min(threads, cfg.topk) / threads, 1e-3)
        n_tok = max(1, min(T_main, int(args.cpu_seconds / per_tok)))
        tokens = list(range(n_tok))
        tp = time.perf_counter()
        oracle.forward(x_host, hl.router_w, hl.bias, hl.expert_w, hl.scales, cfg.topk, cfg.inter, cfg.wfmt_id,
                       tokens=tokens, threads=threads)
        dt = time.perf_counter() - tp
        cpu = dict(value=n_tok / dt, unit="tokens/s", cores=threads, kind="oracle",
                   sample=f"first {n_tok} of the {T_main} tokens of batch 0: full layer in fp64 (exact router "
                          f"logits, top-{cfg.topk}, {cfg.topk} dequantised experts per token, combine); "
                          f"{dt:.1f} s wall",
                   affinity_cpus=affinity, cpu_share=share, cpu_model=model,
                   threads_rule="the affinity mask's CPUs, capped at this host's per-GPU CPU share "
                                "(OMP_NUM_THREADS) where it is set")
        print(f"[cpu] oracle {n_tok} tokens in {dt:.1f} s on {threads} threads (affinity {affinity}, share {share}, "
              f"{model})", file=sys.stderr, flush=True)

    R = results[T_main]
    traffic, traffic_src = w13_traffic(cfg, T_main)
    # the 12-layer stack and the decode-attention steps: in the default run, or on request
    stack = None
    if args.stack or not (args.no_stack or args.no_sweep):
        stack = run_stack(args, dev)
    attention = None
    if not (args.no_attn or args.no_sweep):
        attention = {"fields": ["us_per_step", "frac_of_peak"]}
        attention.update({a["config"]["workload"].split(":")[0]: [round(a["ms_per_step"] * 1e3, 2),
                                                                  round(a["roofline"]["frac"], 4)]
                          for a in run_attn(args, dev, emit=False)})
    power = R.get("power")
    line = {
        "metric": METRIC,
        "value": R["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": R["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp8" if cfg.wfmt == "fp8" else "fp4",
        "data": "synthetic",
        "config": {
            "workload": f"{cfg.name} MoE decode layer: hidden {cfg.hidden}, {cfg.n_experts} experts, top-{cfg.topk}, "
                        f"SwiGLU intermediate {cfg.inter}, {cfg.wfmt} weights, {cfg.act} activations"
                        + (f", router bias {cfg.bias}" if cfg.bias else "") + f", T={T_main} tokens per step",
            "tokens_per_step": T_main,
            "weights": {"fp8": "fp8-e4m3, fp32 scale per 128x128 block", "mxfp4": "mxfp4 (e2m1 + e8m0/32)",
                        "nvfp4": "nvfp4 (e2m1 + e4m3/16 + fp32/matrix)"}[cfg.wfmt]
                       + (", packed 16-row tiles" if layout else ", row-major"),
            "activations": cfg.act,
            "cold_cache": f"{copies} weight copies x 16 token batches cycled",
        },
        "hbm": {
            "bytes_per_step": R["bytes_per_step"],
            "layer_GBs": R["layer_GBs"],
            "layer_frac_of_peak": R["layer_frac"],
            "experts_GBs": R["experts_GBs"],
            "experts_frac_of_peak": R["experts_frac"],
            "n_active_mean": R["n_active_mean"],
        },
        "roofline": {
            "kernel": (("w13_nvfp4_kernel (grouped gate/up + SiLU-gate, weights dequantised to bf16 in registers, "
                        "bf16 MFMA)" if cfg.wfmt == "nvfp4" else
                        "w13_mfma_lds_kernel (grouped gate/up + SiLU-gate, activations staged in LDS, MFMA for every "
                        "expert)") if args.mstar in (0, 1) else "w13 stage (GEMV and MFMA kernels)"),
            "bound": "hbm",
            "achieved": R["w13_GBs"],
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": R["w13_GBs"] / PEAK_HBM_GBS,
            "traffic": traffic,
            "traffic_source": traffic_src,
            "avg_launch_us": R["stage_ms"]["w13"] * 1e3,
            "bytes_per_launch": R["w13_bytes_per_launch"],
        },
        "sweep": sweep_json(results),
        "other_layers": {"fields": OTHER_FIELDS, **others} if others else None,
        "power": power,
        "cpu_baseline": cpu,
        "stack": stack,
        "attention": attention,
        "setup_s": round(setup_s, 1),
    }
    print(json.dumps(line))


if __name__ == "__main__":
    main()
