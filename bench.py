"""Benchmark of the Forcing-KV hot path on one MI355X.

One step = one AR step of one attention layer (a "unit"): segment scoring and
BottomK selection for the dynamic heads, the static heads' structural pruning,
then chunk attention of all heads over their retained history -- the C-ABI
calls, on the 480P Wan-1.3B-style layer (12 heads, d = 128, 1560
tokens/frame, 21-frame history, 3-frame chunk, heads 0-5 static with sink + 6
recent frames, heads 6-11 dynamic with sink + 10 of 20 frames).

Inputs are seeded synthetic tensors already resident in HBM.  The step
rotates through several independent copies of the layer's buffers (as the
layers of a real rollout would), so a step never finds its cache in the
256 MB last-level cache from the previous step.

Prints ONE JSON line on stdout (progress lines go to stderr).  `value` is
the wall-clock ms per step (one layer, one AR step) over the timed steps,
lower is better.  The timed step is the layer driver's default step
(CompressedLayer.step, "paged"): one launch scores the dynamic heads'
segments and selects the kept ones, then one attention launch covers all 12
heads, every retained history read in place from the cache (no compaction,
no gather).  Before the timed steps a serial pass of the compacting path's
four calls with HIP events between them gives the per-stage breakdown (and
brings the clock up).  During the timed steps HIP
events on each launch's own stream time every attention launch the step
makes; `roofline` reports the longest of them (MFMA-bound), `roofline_launches`
all of them.  `cpu_baseline` times the CPU oracle on the host cores on a
bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "ms per AR chunk (score+compact+attn) and attn TFLOP/s, 480P/1080P shapes"
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_FP8_TFLOPS = 5000.0      # MI355X dense FP8 MFMA
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E
EXTRAS = ("parts", "fp8", "scoring", "uncompressed", "sweep", "1080p")


def log(msg):
    """A progress line on stderr (stdout carries only the JSON line)."""
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=100)
    p.add_argument("--resolution", default="480p", choices=["480p", "1080p"])
    p.add_argument("--copies", type=int, default=4, help="independent layer buffers rotated per step")
    p.add_argument("--breakdown-reps", type=int, default=50,
                   help="serial units of the per-stage pass ahead of the timed steps")
    p.add_argument("--cpu-rows", type=int, default=4680,
                   help="query rows per head in the 480P CPU oracle sample (4680 = every row)")
    p.add_argument("--cpu-rows-1080p", type=int, default=2048,
                   help="query rows per head in the 1080P CPU oracle sample (extrapolated to 24480)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--step", default="paged", choices=["paged", "paged2", "compact", "serial"],
                   help="timed step: paged (score + select in one launch, then one attention launch over "
                        "every head read in place), paged2 (the same with the static heads on a side "
                        "stream), compact (static heads on a side stream, dynamic heads scored, compacted "
                        "and attended), or serial (the four calls of the compacting path on one stream)")
    p.add_argument("--static", default="in_place", choices=["in_place", "gather"],
                   help="compact step: static heads attended in place from the cache, or gathered "
                        "into the compressed buffers first")
    p.add_argument("--no-rollout", action="store_true",
                   help="skip the measured 30-layer x 4-step rollouts (10 and 60 chunks)")
    p.add_argument("--no-extras", action="store_true",
                   help="skip the extra measurements (1080P, sweep, FP8, proxy, uncompressed attention)")
    p.add_argument("--extras", default="all",
                   help="comma-separated subset of the extra measurements: " + ",".join(EXTRAS) + " (or all)")
    p.add_argument("--schedule", default="balanced", choices=["balanced", "per-item"],
                   help="attention work schedule (balanced needs the attention workspace)")
    p.add_argument("--traffic-json", default=os.path.join(ROOT, "profiles", "attention_traffic.json"),
                   help="HBM bytes per attention launch measured with rocprofv3 counters")
    p.add_argument("--copy-calibration", action="store_true",
                   help="only run a plain 256 MiB device-to-device copy three times (the known-size "
                        "kernel that FETCH_SIZE / WRITE_SIZE are scaled by) and exit")
    p.add_argument("--read-reference", action="store_true",
                   help="only time the runtime's own reductions and copy over the bytes the scoring "
                        "reads at 480P and 1080P (52.7 and 275.7 MB of bf16), as a reference for what "
                        "one pass over that many bytes reaches, and exit")
    return p.parse_args()


def copy_calibration():
    import torch
    n = 256 << 20
    a = torch.ones(n // 4, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": n, "launches": 3}), flush=True)


def read_reference():
    """torch's sum (fp32 accumulation) and copy over 52.7 MB and 275.7 MB of
    bf16 -- the scoring's reads at 480P and 1080P -- rotating enough buffers
    that each pass misses the 256 MB MALL; HIP events, mean of 50 calls."""
    import torch
    out = []
    for mb, nbuf in ((52.7, 8), (275.7, 3)):
        n = int(mb * 1e6 / 2)
        bufs = [torch.randn(n, device="cuda").to(torch.bfloat16) for _ in range(nbuf)]
        k = [0]

        def nxt():
            k[0] += 1
            return bufs[k[0] % nbuf]
        for name, fn in (("sum_fp32", lambda: torch.sum(nxt(), dtype=torch.float32)),
                         ("copy", lambda: nxt().clone())):
            ms = _time_ms(fn, 50, torch.cuda.current_stream(), warm=5)
            moved = mb * 1e6 * (2 if name == "copy" else 1)
            out.append({"MB_read": mb, "op": name, "us": round(ms * 1e3, 1),
                        "GB_s_moved": round(moved / (ms * 1e-3) / 1e9, 1),
                        "frac_of_hbm_peak": round(moved / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 3)})
            log(f"read reference {mb} MB {name}: {ms * 1e3:.1f} us")
        del bufs
        torch.cuda.empty_cache()
    print(json.dumps({"read_reference": out}), flush=True)


def to_dev(a, dtype):
    import numpy as np
    import torch
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host_bits(t):
    """A bf16 device tensor as its uint16 bit pattern on the host."""
    import numpy as np
    import torch
    return t.cpu().view(torch.int16).numpy().view(np.uint16)


def device_layer_inputs(cfg, seed):
    """The layer's tensors generated on the device from a seed (the 1080P
    cache is too large to draw quickly on the host): keys an AR(1) chain over
    the H history frames and the chunk's frames (rho = 0.9, elementwise, fp32,
    each frame rounded to bf16), values and queries N(0,1); logical frame t in
    slot t."""
    import torch
    g = torch.Generator(device="cuda").manual_seed(seed)
    h, d, F, H, C = cfg.n_heads, cfg.head_dim, cfg.frame_tokens, cfg.hist_frames, cfg.chunk_frames
    rho = 0.9
    a = math.sqrt(1 - rho * rho)
    K_hist = torch.empty(h, cfg.cap_frames, F, d, dtype=torch.bfloat16, device="cuda")
    K_cur = torch.empty(h, C * F, d, dtype=torch.bfloat16, device="cuda")
    k = torch.randn(h, F, d, device="cuda", generator=g)
    for t in range(H + C):
        if t > 0:
            k = rho * k + a * torch.randn(h, F, d, device="cuda", generator=g)
        if t < H:
            K_hist[:, t] = k.to(torch.bfloat16)
        else:
            K_cur[:, (t - H) * F:(t - H + 1) * F] = k.to(torch.bfloat16)
    V_hist = torch.randn(h, cfg.cap_frames, F, d, device="cuda", generator=g).to(torch.bfloat16)
    V_cur = torch.randn(h, C * F, d, device="cuda", generator=g).to(torch.bfloat16)
    Q = torch.randn(h, C * F, d, device="cuda", generator=g).to(torch.bfloat16)
    return dict(K_hist=K_hist, V_hist=V_hist, K_cur=K_cur, V_cur=V_cur, Q=Q)


def attention_flop(cfg, kv_len, heads=None):
    """4 * Lq * d * (kv_len + Lq) summed over the given heads (QK^T and PV only)."""
    idx = range(cfg.n_heads) if heads is None else heads
    return float(sum(4.0 * cfg.lq * cfg.head_dim * (int(kv_len[h]) + cfg.lq) for h in idx))


def static_kv_len(cfg, heads):
    """Retained history tokens of every head whose kept set follows from its
    budget alone (static heads: |kept frames| * F); None for dynamic heads."""
    import workloads as W
    H = cfg.hist_frames
    out = []
    for b in heads:
        if b.type != W.STATIC:
            out.append(None)
            continue
        a = min(b.sink_frames, H)
        lo = max(H - b.recent_frames, 0)
        out.append((H if lo <= a else a + (H - lo)) * cfg.frame_tokens)
    return out


def _time_ms(fn, reps, stream, warm=3):
    """Mean ms of fn() over reps launches, HIP events on the launch stream."""
    import torch
    for _ in range(warm):
        fn()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(reps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def staged_breakdown(layers, bufs, slots, reps, stream, warm=10):
    """The four calls one after another on one stream with HIP events between
    them, rotating over the buffer copies.  Returns [reps][4] ms (score,
    select_compact, compress_static, attention)."""
    import numpy as np
    import torch
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(reps)]

    def staged(i, e):
        L, b = layers[i % len(layers)], bufs[i % len(layers)]
        e[0].record(stream)
        L.score(b["K_hist"], slots, b["K_cur"])
        e[1].record(stream)
        L.select_compact(b["K_hist"], b["V_hist"], slots)
        e[2].record(stream)
        L.compress_static(b["K_hist"], b["V_hist"], slots)
        e[3].record(stream)
        L.attention(b["Q"], b["K_cur"], b["V_cur"], b["O"])
        e[4].record(stream)

    for i in range(warm):
        staged(i, ev[0])
    torch.cuda.synchronize()
    for i in range(reps):
        staged(i, ev[i])
    torch.cuda.synchronize()
    return np.array([[e[j].elapsed_time(e[j + 1]) for j in range(4)] for e in ev])


def stage_report(cfg, layer, stage_ms):
    """Per-kernel ms, achieved GB/s (algorithmic bytes) and fraction of peak."""
    import numpy as np
    import workloads as W
    kv = layer.kv_len.cpu().numpy().astype(np.int64)
    d, e, F, H = cfg.head_dim, cfg.esize, cfg.frame_tokens, cfg.hist_frames
    dyn = np.array([b.type == W.DYNAMIC for b in layer_budgets(layer)])
    score_bytes = int(dyn.sum()) * (H + 1) * F * d * e
    dyn_bytes = 4 * d * e * int(kv[dyn].sum())
    st_bytes = 4 * d * e * int(kv[~dyn].sum())
    flop = attention_flop(cfg, kv)
    mean = stage_ms.mean(axis=0)
    p10, p50, p90 = np.percentile(stage_ms, [10, 50, 90], axis=0)
    names = ("score_segments", "select_compact", "compress_static", "chunk_attention")
    gbs = lambda b, ms: b / (ms * 1e-3) / 1e9
    rep = {
        "ms": {k: round(float(mean[j]), 4) for j, k in enumerate(names)},
        "ms_p10_p50_p90": {k: [round(float(p10[j]), 4), round(float(p50[j]), 4), round(float(p90[j]), 4)]
                           for j, k in enumerate(names)},
        "algorithmic_bytes": {"score_segments": score_bytes, "select_compact": dyn_bytes,
                              "compress_static": st_bytes},
        "GB_s": {"score_segments": round(gbs(score_bytes, mean[0]), 1),
                 "select_compact": round(gbs(dyn_bytes, mean[1]), 1),
                 "compress_static": round(gbs(st_bytes, mean[2]), 1)},
        "frac_of_hbm_peak": {"score_segments": round(gbs(score_bytes, mean[0]) / PEAK_HBM_GBS, 3),
                             "select_compact": round(gbs(dyn_bytes, mean[1]) / PEAK_HBM_GBS, 3),
                             "compress_static": round(gbs(st_bytes, mean[2]) / PEAK_HBM_GBS, 3)},
        "attention_algorithmic_flop": flop,
        "attention_TFLOP_s": round(flop / (mean[3] * 1e-3) / 1e12, 1),
        "attention_frac_of_bf16_peak": round(flop / (mean[3] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        "serial_unit_ms": round(float(mean.sum()), 4),
    }
    return rep


def layer_budgets(layer):
    import workloads as W
    return [W.HeadBudget(int(h.type), int(h.sink_frames), int(h.recent_frames), int(h.keep_k), int(h.scope))
            for h in layer.heads]


def step_mode_of(args, cfg):
    """The layer's step mode for the timed step (the paged modes fall back to
    the compacting step where the shape does not allow them)."""
    from paper_2605_09681_amd.layer import paged_supported
    if args.step in ("paged", "paged2") and paged_supported(cfg.dtype, cfg.frame_tokens, cfg.seg_tokens,
                                                           cfg.cap_frames):
        return args.step
    return "compact"


def make_layers(cfg, n, args, budgets=None):
    from paper_2605_09681_amd.layer import CompressedLayer
    mode = step_mode_of(args, cfg)
    return [CompressedLayer(cfg.n_heads, cfg.head_dim, cfg.frame_tokens, cfg.hist_frames, cfg.cap_frames,
                            cfg.chunk_frames, cfg.seg_tokens, cfg.dtype, cfg.heads if budgets is None else budgets,
                            balanced=args.schedule == "balanced",
                            in_place=args.static == "in_place" if mode == "compact" else None, step_mode=mode)
            for _ in range(n)]


def timed_steps(cfg, layers, bufs, slots, args, mode):
    """W warm-up steps, then exactly K timed steps bracketed by device
    synchronisation; HIP events around every attention launch of the timed
    steps, on the stream that launch runs on."""
    import numpy as np
    import torch
    stream = torch.cuda.current_stream()
    names = ("attention",) if mode in ("paged", "serial") else ("static_attention", "dynamic_attention")
    events = [{n: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for n in names}
              for _ in range(args.steps)]

    def step(i, ev=None):
        L, b = layers[i % len(layers)], bufs[i % len(layers)]
        if mode != "serial":
            L.step(b["K_hist"], b["V_hist"], slots, b["Q"], b["K_cur"], b["V_cur"], b["O"], events=ev)
            return
        L.score(b["K_hist"], slots, b["K_cur"])
        L.select_compact(b["K_hist"], b["V_hist"], slots)
        L.compress_static(b["K_hist"], b["V_hist"], slots)
        if ev is not None:
            ev["attention"][0].record(stream)
        L.attention(b["Q"], b["K_cur"], b["V_cur"], b["O"])
        if ev is not None:
            ev["attention"][1].record(stream)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(i, events[i])
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) * 1e3 / args.steps
    launch_ms = {n: np.array([e[n][0].elapsed_time(e[n][1]) for e in events]) for n in names}
    return wall_ms, launch_ms


def launch_rooflines(cfg, layer, launch_ms, traffic, mode):
    """Per attention launch of the timed step: algorithmic FLOP, mean ms,
    achieved TFLOP/s and fraction of the bf16 peak."""
    import numpy as np
    import workloads as W
    budgets = layer_budgets(layer)
    kv = layer.kv_len.cpu().numpy().astype(np.int64)
    st = static_kv_len(cfg, budgets)
    kv_all = [st[h] if st[h] is not None else int(kv[h]) for h in range(cfg.n_heads)]
    groups = {"static_attention": [h for h, b in enumerate(budgets) if b.type == W.STATIC],
              "dynamic_attention": [h for h, b in enumerate(budgets) if b.type == W.DYNAMIC],
              "attention": list(range(cfg.n_heads))}
    # cut items are merged inside the bf16 kernel: one kernel per launch
    paged = "attn_bf16_kernel<128, balanced, paged>"
    plain = "attn_bf16_kernel<128, balanced>"
    kernels = {
        "paged": {"attention": f"fkv_chunk_attention_paged: {paged} (all heads, every kept history read in "
                               "place from the cache)"},
        "paged2": {"static_attention": f"fkv_chunk_attention_paged: {paged} (static heads, in place)",
                   "dynamic_attention": f"fkv_chunk_attention_paged: {paged} (dynamic heads, kept segments "
                                        "read in place)"},
        "compact": {"static_attention": f"fkv_chunk_attention_static: {paged} (static heads, in place)",
                    "dynamic_attention": f"fkv_chunk_attention_heads: {plain} (dynamic heads, compacted "
                                         "history)"},
        "serial": {"attention": f"fkv_chunk_attention: {plain} (all heads, compacted history)"},
    }[mode]
    out = []
    for name, ms in launch_ms.items():
        flop = attention_flop(cfg, kv_all, groups[name])
        avg = float(ms.mean())
        tf = flop / (avg * 1e-3) / 1e12
        out.append({"launch": name, "kernel": kernels[name], "bound": "mfma", "achieved": round(tf, 1),
                    "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": round(tf / PEAK_BF16_TFLOPS, 4),
                    "traffic": (traffic or {}).get(name), "algorithmic_flop_per_launch": flop,
                    "avg_launch_ms": round(avg, 4),
                    "launch_ms_p10_p50_p90": [round(float(v), 4) for v in np.percentile(ms, [10, 50, 90])]})
    return out


def measure_step_parts(cfg, layers, bufs, slots, stream, mode, reps=50):
    """The paged step's two launches one after another with HIP events between
    them: fkv_score_select (per-frame sums, the per-head reduction and the
    BottomK selection in one kernel; algorithmic bytes = the dynamic heads'
    keys of frames 0..H) and fkv_chunk_attention_paged over all heads."""
    import numpy as np
    import torch
    import workloads as W
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(reps)]
    for i in range(reps + 5):
        L, b = layers[i % len(layers)], bufs[i % len(layers)]
        e = ev[i - 5] if i >= 5 else None
        if e:
            e[0].record(stream)
        L.score_select(b["K_hist"], slots, b["K_cur"])
        if e:
            e[1].record(stream)
        L.attention_paged(b["K_hist"], b["V_hist"], slots, b["Q"], b["K_cur"], b["V_cur"], b["O"])
        if e:
            e[2].record(stream)
    torch.cuda.synchronize()
    t = np.array([[e[0].elapsed_time(e[1]), e[1].elapsed_time(e[2])] for e in ev])
    n_dyn = sum(1 for b in cfg.heads if b.type == W.DYNAMIC)
    score_bytes = n_dyn * (cfg.hist_frames + 1) * cfg.frame_tokens * cfg.head_dim * cfg.esize
    sm, am = float(t[:, 0].mean()), float(t[:, 1].mean())
    kv = layers[0].kv_len.cpu().numpy().astype(np.int64)
    st = static_kv_len(cfg, layer_budgets(layers[0]))
    flop = attention_flop(cfg, [st[h] if st[h] is not None else int(kv[h]) for h in range(cfg.n_heads)])
    return {"score_select_ms": round(sm, 4),
            "score_select_GB_s": round(score_bytes / (sm * 1e-3) / 1e9, 1),
            "score_select_frac_of_hbm_peak": round(score_bytes / (sm * 1e-3) / 1e9 / PEAK_HBM_GBS, 3),
            "score_select_algorithmic_bytes": score_bytes,
            "attention_paged_ms": round(am, 4),
            "attention_paged_TFLOP_s": round(flop / (am * 1e-3) / 1e12, 1),
            "attention_paged_frac_of_bf16_peak": round(flop / (am * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
            "serial_sum_ms": round(sm + am, 4),
            "ms_p10_p50_p90": {"score_select": [round(float(v), 4) for v in np.percentile(t[:, 0], [10, 50, 90])],
                               "attention_paged": [round(float(v), 4) for v in np.percentile(t[:, 1], [10, 50, 90])]},
            "note": "HIP events between the two launches on one stream, rotating buffer copies"}


def load_traffic(path, workload):
    """HBM bytes per launch from the committed rocprofv3 counter summary, only
    while the attention sources are the ones the counters were taken on."""
    try:
        with open(path) as f:
            tj = json.load(f)
    except (OSError, ValueError):
        return None
    if tj.get("kernel_source_sha") != _kernel_sha():
        return None
    return (tj.get("workloads") or {}).get(workload, {}).get("bytes_per_launch_by_launch")


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE {world}); "
              "this build runs on a single GPU.  The Forcing-KV hot path shards by head with no "
              "exchange, so N GPUs would run N independent head subsets of this step.", file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration()
        return
    if args.read_reference:
        read_reference()
        return

    import numpy as np
    import torch

    import workloads as W
    import paper_2605_09681_amd as fkv

    fkv.lib()  # fail loudly if the HIP library is missing
    torch.cuda.set_device(0)
    extras_on = set() if args.no_extras else (set(EXTRAS) if args.extras == "all" else set(args.extras.split(",")))
    unknown = extras_on - set(EXTRAS)
    if unknown:
        sys.exit(f"unknown --extras {sorted(unknown)}; choose from {','.join(EXTRAS)}")
    log(f"{args.resolution} layer: inputs and {args.copies} buffer copies")
    cfg = W.wan_layer_config(args.resolution)
    x = None
    if args.resolution == "480p":
        x = W.make_layer_inputs(cfg, seed=0)
        base = {k: to_dev(getattr(x, k), cfg.dtype) for k in ("K_hist", "V_hist", "K_cur", "V_cur", "Q")}
    else:
        base = device_layer_inputs(cfg, seed=0)
    slots = np.arange(cfg.hist_frames, dtype=np.int32) if x is None else x.frame_slot
    bufs = []
    for c in range(args.copies):
        b = base if c == 0 else {k: v.clone() for k, v in base.items()}
        b["O"] = torch.empty_like(b["Q"])
        bufs.append(b)
    layers = make_layers(cfg, args.copies, args)
    stream = torch.cuda.current_stream()

    # per-stage breakdown first: it also brings the clock up before the timed steps
    log("per-stage breakdown (serial compacting path)")
    # (50 serial units, ~30 ms at 480P: long enough for the clock to come up; a
    # longer pass, 200 units, measurably slowed the timed steps that follow --
    # sustained MFMA load lowers the clock the part holds)
    stage = staged_breakdown(layers, bufs, slots, max(args.breakdown_reps, 1), stream)
    breakdown = stage_report(cfg, layers[0], stage)

    traffic = load_traffic(args.traffic_json, cfg.name)
    mode = args.step if args.step == "serial" else step_mode_of(args, cfg)
    log(f"timed steps ({mode}): {args.warmup} warm-up + {args.steps}")
    wall_ms, launch_ms = timed_steps(cfg, layers, bufs, slots, args, mode)
    launches = launch_rooflines(cfg, layers[0], launch_ms, traffic, mode)
    dominant = max(launches, key=lambda r: r["avg_launch_ms"])
    step_parts = measure_step_parts(cfg, layers, bufs, slots, stream, mode) if mode == "paged" else None

    d, F, H, Lq = cfg.head_dim, cfg.frame_tokens, cfg.hist_frames, cfg.lq
    out = {
        "metric": METRIC,
        "value": round(wall_ms, 4),
        "unit": "ms",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall_ms, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic: seeded AR(1) keys (rho 0.9) across frames, N(0,1) queries/values",
        "config": {
            "workload": (f"{cfg.name}: one layer, one AR step; {cfg.n_heads} heads x d{d}, "
                         f"{F} tokens/frame, {H}-frame history, {cfg.chunk_frames}-frame chunk "
                         f"(Lq {Lq}); heads 0-5 static (sink 1 + recent 6), heads 6-11 dynamic "
                         f"(sink 1 + 10 of 20 frame segments)"),
            "value_is": "ms per layer per AR step (one unit); the measured 30-layer x 4-step ms per chunk "
                        "is rollout_480p",
            "rotating_copies": args.copies,
            "attention_schedule": args.schedule,
            "step": {"paged": "fkv_score_select (dynamic heads: scores + kept segments, one launch), then one "
                              "fkv_chunk_attention_paged launch over all 12 heads with every kept history read "
                              "in place from the cache (no compaction, no gather)",
                     "paged2": "static heads' in-place attention on a side stream; dynamic heads: "
                               "fkv_score_select, then in-place attention",
                     "compact": ("static heads (attention read in place from the cache" if args.static ==
                                 "in_place" else "static heads (gather + attention") +
                                ") on a side stream, dynamic heads (score + select/compact + attention) on the "
                                "main stream",
                     "serial": "the four calls of the compacting path one after another on one stream"}[mode],
        },
        "roofline": {k: v for k, v in dominant.items() if k != "launch_ms_p10_p50_p90"},
        "roofline_launches": launches,
        "breakdown_serial": breakdown,
        "attn_tflops": dominant["achieved"],
    }
    if step_parts is not None:
        out["step_parts"] = step_parts
    extras = None
    if extras_on & {"parts", "fp8", "scoring", "uncompressed"}:
        extras = measure_extras(args, cfg, slots, bufs, layers, stream, extras_on)
        ua = extras.get("uncompressed_attention")
        if ua is not None:
            ua["speedup_of_compressed"] = round(ua["ms"] / breakdown["ms"]["chunk_attention"], 3)
        out["extras"] = extras
    if extras_on & {"sweep", "1080p"} and args.resolution == "480p":
        out.setdefault("extras", {})
        for b in bufs[1:]:
            b.clear()
        del layers
        torch.cuda.empty_cache()
        if "sweep" in extras_on:
            log("extras: keep-fraction x segment-length sweep")
            out["extras"]["sweep_480p"] = measure_sweep(args, bufs[0], stream)
        if "1080p" in extras_on:
            log("extras: 1080P unit")
            out["extras"]["unit_1080p"] = measure_1080p(args, stream)
    if not args.no_rollout and not args.no_extras:
        for b in bufs:   # free the single-layer buffers before the 30-layer caches
            b.clear()
        torch.cuda.empty_cache()
        log("rollout: 30 layers x 4 steps x 10 chunks, three scoring modes")
        out["rollout_480p"] = measure_rollouts({"per_layer_scoring": (False, False),
                                                "per_layer_incremental_rescoring": (False, True),
                                                "pooled_first_block_proxy": (True, False)})
        log("rollout: 60 chunks")
        out["rollout_480p_60_chunks"] = measure_rollouts({"per_layer_scoring": (False, False)}, n_chunks=60,
                                                         reps=1)
    if not args.no_cpu_baseline and args.resolution == "480p":
        log("cpu_baseline: the oracle on the host cores (480P unit, then the 1080P sample)")
        out["cpu_baseline"] = cpu_baseline(cfg, x, args.cpu_rows)
        out["cpu_baseline"]["leg_1080p"] = cpu_baseline_1080p(args.cpu_rows_1080p)
    print(json.dumps(out), flush=True)


_pair_counter = [0]


def _next_pair(layers, bufs):
    """The next (layer, buffers) copy in rotation."""
    i = _pair_counter[0] % len(layers)
    _pair_counter[0] += 1
    return layers[i], bufs[i]


def measure_extras(args, cfg, slots, bufs, layers, stream, which):
    """Measurements outside the step (each selected by name in `which`):
    parts -- the compacting two-stream step's attention launches, each alone;
    fp8 -- the FP8 variant (packing + attention); scoring -- incremental
    rescoring and the first-block proxy (scores pooled over all heads, once per
    chunk, shared by every layer); uncompressed -- the same attention kernel on
    the uncompressed cache (every head keeps all H frames), for the
    kernel-level speedup of the compression."""
    import numpy as np
    import torch
    import workloads as W
    import paper_2605_09681_amd as fkv
    from paper_2605_09681_amd.layer import CompressedLayer

    d, F, H, Lq = cfg.head_dim, cfg.frame_tokens, cfg.hist_frames, cfg.lq
    L0, b = layers[0], bufs[0]
    out = {}
    if "scoring" in which:
        log("extras: incremental rescoring and the pooled proxy")
        pooled = torch.empty((L0.n_seg,), dtype=torch.float32, device="cuda")
        ws = torch.zeros(max(fkv.fkv_score_pooled_workspace_size(L0.shape), 1), dtype=torch.uint8, device="cuda")
        pooled_ms = _time_ms(lambda: fkv.fkv_score_pooled(L0.shape, b["K_hist"], slots, b["K_cur"], pooled, ws),
                             20, stream)
        pooled_bytes = cfg.n_heads * (H + 1) * F * d * 2
        stats = torch.empty(fkv.fkv_score_stats_size(L0.shape, L0.heads) // 8, dtype=torch.float64,
                            device="cuda")
        hist_ms = _time_ms(lambda: fkv.fkv_score_history(L0.shape, L0.heads, b["K_hist"], slots, stats,
                                                         L0.workspace), 20, stream)
        cached_ms = _time_ms(lambda: fkv.fkv_score_segments_cached(L0.shape, L0.heads, b["K_hist"], slots,
                                                                   b["K_cur"], stats, L0.scores, L0.workspace),
                             20, stream)
        n_dyn = sum(1 for t in L0.types if t == W.DYNAMIC)
        out["incremental_score"] = {
            "history_ms": round(hist_ms, 4), "step_ms": round(cached_ms, 4),
            "step_GB_s": round(n_dyn * 2 * F * d * 2 / (cached_ms * 1e-3) / 1e9, 1),
            "note": "history statistics once per chunk, then per AR step the scores from them plus frames "
                    "H-1 and H (2 of the 22 frames per dynamic head)"}
        out["pooled_proxy_score"] = {
            "ms": round(pooled_ms, 4), "GB_s": round(pooled_bytes / (pooled_ms * 1e-3) / 1e9, 1),
            "frac_of_hbm_peak": round(pooled_bytes / (pooled_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 3),
            "note": "all 12 heads pooled, once per AR step for all layers (not part of the step)"}

    if "parts" in which:
        # the compacting two-stream step's launches: each attention launch
        # alone, the one 12-head launch, and the step without the dynamic
        # compression (its attention then reads the compacted cache of the
        # previous step)
        log("extras: the compacting step's launches")

        def rot(fn):
            return lambda: fn(*_next_pair(layers, bufs))

        def static_only(L, bb):
            L.attention_static(bb["K_hist"], bb["V_hist"], slots, bb["Q"], bb["K_cur"], bb["V_cur"], bb["O"],
                               None, L.attn_workspace)

        def dynamic_only(L, bb):
            fkv.fkv_chunk_attention_heads(L.shape, L.dynamic_heads, bb["Q"], L.Kc, L.Vc, L.kv_len, bb["K_cur"],
                                          bb["V_cur"], L.scale, bb["O"], None, L.attn_workspace)

        def all_heads(L, bb):
            L.attention(bb["Q"], bb["K_cur"], bb["V_cur"], bb["O"])

        def step_nocomp(L, bb):
            main = torch.cuda.current_stream()
            L.side.wait_stream(main)
            with torch.cuda.stream(L.side):
                static_only(L, bb)
            dynamic_only(L, bb)
            main.wait_stream(L.side)

        parts = {name: round(_time_ms(rot(fn), 50, stream), 4)
                 for name, fn in (("static_heads_in_place_ms", static_only), ("dynamic_heads_ms", dynamic_only),
                                  ("all_heads_one_launch_ms", all_heads),
                                  ("step_without_compression_ms", step_nocomp))}
        out["compact_step_launches"] = dict(parts, note="the compacting two-stream step's launches, each timed "
                                                        "alone over the rotated buffer copies")

    if "fp8" in which:
        log("extras: FP8 packing + attention")
        O8 = torch.empty_like(b["Q"])
        pack_ms = _time_ms(lambda: L0.pack_fp8(b["Q"], b["K_cur"], b["V_cur"]), 20, stream)
        fp8_ms = _time_ms(lambda: L0.attention_fp8_packed(O8), 20, stream)
        kv_len = L0.kv_len.cpu().numpy().astype(np.int64)
        attn_flop = attention_flop(cfg, kv_len)
        # the FP8 step with nothing compacted (scores + kept segments, packing
        # read in place from the cache, FP8 attention) against the bf16 default
        # step, both over the rotated buffer copies
        outs8 = [torch.empty_like(bb["Q"]) for bb in bufs]

        def step8(i):
            L, bb = layers[i % len(layers)], bufs[i % len(layers)]
            L.step_fp8(bb["K_hist"], bb["V_hist"], slots, bb["Q"], bb["K_cur"], bb["V_cur"], outs8[i % len(layers)])

        def step16(i):
            L, bb = layers[i % len(layers)], bufs[i % len(layers)]
            L.step(bb["K_hist"], bb["V_hist"], slots, bb["Q"], bb["K_cur"], bb["V_cur"], bb["O"])

        ctr = [0]

        def nxt(fn):
            def f():
                fn(ctr[0])
                ctr[0] += 1
            return f
        steps = {}
        for name, fn in (("fp8", step8), ("bf16", step16), ("fp8_again", step8), ("bf16_again", step16)):
            steps[name] = _time_ms(nxt(fn), 50, stream)
        fp8_step = (steps["fp8"] + steps["fp8_again"]) / 2
        bf16_step = (steps["bf16"] + steps["bf16_again"]) / 2
        out["fp8_attention"] = {
            "attention_ms": round(fp8_ms, 4), "TFLOP_s": round(attn_flop / (fp8_ms * 1e-3) / 1e12, 1),
            "peak_TFLOP_s": PEAK_FP8_TFLOPS,
            "frac_of_fp8_peak": round(attn_flop / (fp8_ms * 1e-3) / 1e12 / PEAK_FP8_TFLOPS, 4),
            "pack_ms": round(pack_ms, 4), "pack_plus_attention_ms": round(pack_ms + fp8_ms, 4),
            "step_fp8_in_place_ms": round(fp8_step, 4), "step_bf16_in_place_ms": round(bf16_step, 4),
            "step_speedup_fp8": round(bf16_step / fp8_step, 3),
            "note": "E4M3 Q/K/V/P on gfx950 FP8 MFMA; pack = statistics + quantise + transpose (over the "
                    "compacted history); the FP8 step = fkv_score_select + fkv_fp8_pack_paged (history read in "
                    "place) + fkv_chunk_attention_fp8, against the bf16 step (fkv_score_select + "
                    "fkv_chunk_attention_paged), alternating, 50 steps each twice"}

    if "uncompressed" in which:
        log("extras: uncompressed attention")
        full_heads = tuple(W.HeadBudget(W.STATIC, 0, H) for _ in range(cfg.n_heads))
        full = CompressedLayer(cfg.n_heads, d, F, H, cfg.cap_frames, cfg.chunk_frames, cfg.seg_tokens, cfg.dtype,
                               full_heads, balanced=args.schedule == "balanced", step_mode="compact")
        full.compress_static(b["K_hist"], b["V_hist"], slots)
        O = torch.empty_like(b["Q"])
        full_ms = _time_ms(lambda: full.attention(b["Q"], b["K_cur"], b["V_cur"], O), 10, stream)
        full_flop = 4.0 * Lq * d * cfg.n_heads * (H * F + Lq)
        del full
        out["uncompressed_attention"] = {"ms": round(full_ms, 4),
                                         "TFLOP_s": round(full_flop / (full_ms * 1e-3) / 1e12, 1),
                                         "kv_len": H * F}
    return out


def measure_sweep(args, b, stream, reps=30):
    """The keep-fraction x segment-length sweep at 480P: per point the four
    calls of the compacting path one after another (score, select + compact,
    static gather, 12-head attention), mean ms per kernel over `reps` units
    with HIP events, achieved GB/s of the HBM kernels and attention TFLOP/s;
    and, where the shape allows it, the paged step (score + select, then one
    in-place attention launch).  Keep 100% also keeps every frame of the
    static heads (full-attention equivalence)."""
    import numpy as np
    import workloads as W
    out = []
    slots = np.arange(21, dtype=np.int32)
    for L in (390, 1560, 4680):
        for frac in (0.25, 0.5, 0.75, 1.0):
            cfg = W.wan_layer_config("480p", keep_fraction=frac, seg_tokens=L,
                                     static_recent=21 if frac == 1.0 else 6)
            layer = make_layers(cfg, 1, args)[0]
            stage = staged_breakdown([layer], [b], slots, reps, stream, warm=3)
            rep = stage_report(cfg, layer, stage)
            rec = {"seg_tokens": L, "keep_fraction": frac, "unit_ms_compact_serial": rep["serial_unit_ms"],
                   "ms": rep["ms"], "GB_s": rep["GB_s"], "frac_of_hbm_peak": rep["frac_of_hbm_peak"],
                   "attention_TFLOP_s": rep["attention_TFLOP_s"],
                   "attention_frac_of_bf16_peak": rep["attention_frac_of_bf16_peak"],
                   "kv_len_dynamic": int(layer.kv_len[6].item())}
            if layer.step_mode == "paged":
                parts = measure_step_parts(cfg, [layer], [b], slots, stream, "paged", reps=reps)
                rec["paged_unit_ms"] = parts["serial_sum_ms"]
                rec["paged"] = {k: parts[k] for k in ("score_select_ms", "score_select_GB_s",
                                                      "attention_paged_ms", "attention_paged_TFLOP_s",
                                                      "attention_paged_frac_of_bf16_peak")}
            out.append(rec)
            del layer
    return {"points": out,
            "note": "one buffer set (cache 202 MB: the rotating copies are freed first), serial calls"}


def measure_1080p(args, stream):
    """The 1080P layer (68x120 patches per frame): the default step, the four
    calls with a per-kernel breakdown, and each launch of the step, with
    device-generated inputs and one buffer set (the 1.05 GB cache far exceeds
    the 256 MB MALL)."""
    import numpy as np
    import torch
    import workloads as W
    c10 = W.wan_layer_config("1080p")
    b = device_layer_inputs(c10, seed=1)
    b["O"] = torch.empty_like(b["Q"])
    slots10 = np.arange(c10.hist_frames, dtype=np.int32)
    layer = make_layers(c10, 1, args)[0]
    stage = staged_breakdown([layer], [b], slots10, 6, stream, warm=2)
    rep = stage_report(c10, layer, stage)
    a10 = argparse.Namespace(**vars(args))
    a10.steps, a10.warmup = 6, 2
    mode = step_mode_of(args, c10)
    wall, launch_ms = timed_steps(c10, [layer], [b], slots10, a10, mode)
    launches = launch_rooflines(c10, layer, launch_ms, None, mode)
    parts = measure_step_parts(c10, [layer], [b], slots10, stream, mode, reps=6) if mode == "paged" else None
    del layer, b
    torch.cuda.empty_cache()
    return {"step_ms": round(wall, 3), "step_mode": mode, "step_parts": parts, "breakdown_serial": rep,
            "step_launches": launches,
            "workload": "wan1.3b-1080p-layer: 12 heads x d128, 8160 tokens/frame, 21-frame history, "
                        "3-frame chunk; heads 0-5 static (sink 1 + recent 6), 6-11 dynamic (sink 1 + 10 of 20)",
            "note": "device-generated inputs, one buffer set"}


def measure_rollouts(modes, n_chunks: int = 10, n_steps: int = 4, n_layers: int = 30, reps: int = 3):
    """The metric measured rather than extrapolated: the 30-layer stack of the
    480P layer, 4 denoising steps per chunk, `n_chunks` chunks, each layer with
    its own rolling 21-frame cache (sink pinned, 3-frame chunks written back
    after each chunk) and its own seeded head mask (6 of 12 heads dynamic).
    modes maps a name to (pooled, incremental): every step re-scores and
    compacts every layer (pooled=False), or scores once per step from the first
    layer's keys pooled over all heads and reuses that row in every layer
    (pooled=True, the first-block proxy); incremental=True computes each
    layer's history statistics once per chunk and then scores each step from
    them plus the pair touching the chunk.  All modes run on one stack (one
    allocation: a re-allocated 6 GB stack has measured up to 8% slower) in
    `reps` rounds, each round one pass per mode from empty caches; the pass
    with the median full-window time is reported.  Inputs are device-generated
    N(0,1) tensors (values do not change the work)."""
    import torch
    import workloads as W
    from paper_2605_09681_amd.layer import RolloutStack
    nh, d, F, window, C = 12, 128, 1560, 21, 3
    masks = W.rollout_head_masks(0, n_layers=n_layers, n_heads=nh, n_dynamic=6)
    stack = RolloutStack(n_layers, nh, d, F, window, C, F)
    g = torch.Generator(device="cuda").manual_seed(3)
    sets = [tuple(torch.randn(nh, C * F, d, device="cuda", dtype=torch.bfloat16, generator=g) for _ in range(3))
            for _ in range(2)]
    O = torch.empty_like(sets[0][0])

    def budgets(layer, H):
        k = (H - 1) // 2 if H > 1 else 0       # dynamic: sink frame + half of the other frames
        return tuple(W.HeadBudget(W.DYNAMIC, 1, 0, k, W.SCOPE_GLOBAL) if m == W.DYNAMIC else
                     W.HeadBudget(W.STATIC, 1, 6) for m in masks[layer])

    def chunk(i, pooled, incremental):
        slots = W.ring_frame_slots(i, C, window)
        H = len(slots)
        if incremental and H > 0:
            if pooled:
                stack.history(0, None, slots, pooled=True)
            else:
                for layer in range(n_layers):
                    stack.history(layer, budgets(layer, H), slots)
        for step in range(n_steps):
            Q, Kq, Vq = sets[step % 2]
            row = stack.score_pooled(0, slots, Kq, incremental=incremental) if pooled and H > 0 else None
            for layer in range(n_layers):
                stack.run_layer(layer, budgets(layer, H), slots, Q, Kq, Vq, O, pooled=row, incremental=incremental)
        dst = W.chunk_write_slots(i, C, window).tolist()
        for layer in range(n_layers):
            stack.append(layer, Kq, Vq, dst)

    def run(pooled, incremental):
        for layer in range(n_layers):
            stack.K_hist[layer].zero_()
            stack.V_hist[layer].zero_()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(n_chunks + 1)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ev[0].record()
        for i in range(n_chunks):
            chunk(i, pooled, incremental)
            ev[i + 1].record()
        torch.cuda.synchronize()
        wall = (time.perf_counter() - t0) * 1e3
        per_chunk = [ev[i].elapsed_time(ev[i + 1]) for i in range(n_chunks)]
        full = [t for i, t in enumerate(per_chunk) if len(W.ring_frame_slots(i, C, window)) == window]
        return (sum(full) / len(full) if full else wall / n_chunks, wall / n_chunks, per_chunk)

    if reps > 1:
        for pooled, incremental in modes.values():    # untimed: fills the caches, warms the clock
            run(pooled, incremental)
    runs = {name: [] for name in modes}
    for _ in range(reps):
        for name, (pooled, incremental) in modes.items():
            runs[name].append(run(pooled, incremental))
    del stack
    torch.cuda.empty_cache()
    out = {}
    for name, rs in runs.items():
        rs.sort(key=lambda r: r[0])
        full_ms, chunk_ms, per_chunk = rs[len(rs) // 2]
        rec = {"ms_per_chunk": round(chunk_ms, 2), "ms_per_chunk_full_window": round(full_ms, 2),
               "full_window_ms_of_each_pass": [round(r[0], 2) for r in rs]}
        if n_chunks <= 12:
            rec["per_chunk_ms"] = [round(t, 2) for t in per_chunk]
        else:
            full = [t for i, t in enumerate(per_chunk) if len(W.ring_frame_slots(i, C, window)) == window]
            rec["full_window_chunks"] = len(full)
            rec["full_window_ms_p10_p50_p90"] = [round(float(v), 2) for v in
                                                 __import__("numpy").percentile(full, [10, 50, 90])]
            rec["ring_wraps"] = round((n_chunks * C - window) / (window - 1), 2)
        out[name] = rec
    out["workload"] = (f"{n_layers} layers x {n_steps} steps x {n_chunks} chunks, rolling {window}-frame cache "
                       "(sink pinned), 3-frame chunks appended, seeded masks with 6 of 12 heads dynamic; "
                       f"wall-clock including the chunk writes; median of {reps} passes per mode"
                       + (", modes interleaved on one stack" if len(modes) > 1 else ""))
    return out


def cpu_baseline(cfg, x, rows_per_head):
    """Time the CPU oracle on the host cores: full compression of every head
    and attention for a seeded sample of query rows per head, scaled to one
    unit (the attention time is multiplied by Lq / rows_per_head)."""
    import numpy as np
    import oracle
    import workloads as W
    oracle.lib()
    rng = np.random.default_rng(0)
    rows = np.sort(rng.choice(cfg.lq, size=min(rows_per_head, cfg.lq), replace=False)).astype(np.int32)
    t0 = time.perf_counter()
    res = oracle.run_layer(cfg, x, attention=False)
    t1 = time.perf_counter()
    scale = 1.0 / math.sqrt(cfg.head_dim)
    for h in range(cfg.n_heads):
        oracle.attention_rows(x.Q[h], res.Kc[h], res.Vc[h], x.K_cur[h], x.V_cur[h], scale, rows)
    t2 = time.perf_counter()
    per_unit_s = (t1 - t0) + (t2 - t1) * cfg.lq / len(rows)
    # the tiny fp32 configuration in full on one thread, for reference
    threads = oracle.max_threads()
    tiny = W.tiny_config()
    xt = W.make_layer_inputs(tiny, seed=0)
    oracle.set_threads(1)
    t3 = time.perf_counter()
    oracle.run_layer(tiny, xt)
    t4 = time.perf_counter()
    oracle.set_threads(threads)
    cpu_model = ""
    try:
        with open("/proc/cpuinfo") as f:
            cpu_model = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")), "")
    except OSError:
        pass
    return {
        "value": round(per_unit_s * 1e3, 1),
        "unit": "ms",
        "cores": oracle.max_threads(),
        "kind": "oracle",
        "sample": (f"480P layer unit: fp64 C oracle, scoring+selection+compaction of all {cfg.n_heads} heads "
                   f"in full ({t1 - t0:.2f} s) + attention of {len(rows)} of {cfg.lq} query rows per head "
                   f"({t2 - t1:.2f} s), attention scaled x{cfg.lq / len(rows):.1f} to one unit"),
        "measured_s": round(t2 - t0, 2),
        "cpu_model": cpu_model,
        "nproc": os.cpu_count(),
        "omp_num_threads": os.environ.get("OMP_NUM_THREADS"),
        "tiny_f32_unit_1thread_ms": round((t4 - t3) * 1e3, 2),
    }


def cpu_baseline_1080p(rows_per_head):
    """The oracle on the 1080P layer: scoring, selection and compaction of all
    heads in full, attention on a seeded sample of query rows per head,
    extrapolated to all 24480 rows (labelled so).  Inputs are generated on the
    device and copied to the host (the same bits on both sides)."""
    import numpy as np
    import torch
    import oracle
    import workloads as W
    c10 = W.wan_layer_config("1080p")
    b = device_layer_inputs(c10, seed=1)
    x = W.LayerInputs(c10, host_bits(b["K_hist"]), host_bits(b["V_hist"]), host_bits(b["K_cur"]),
                      host_bits(b["V_cur"]), host_bits(b["Q"]), np.arange(c10.hist_frames, dtype=np.int32))
    del b
    torch.cuda.empty_cache()
    rng = np.random.default_rng(1)
    rows = np.sort(rng.choice(c10.lq, size=min(rows_per_head, c10.lq), replace=False)).astype(np.int32)
    t0 = time.perf_counter()
    res = oracle.run_layer(c10, x, attention=False)
    t1 = time.perf_counter()
    scale = 1.0 / math.sqrt(c10.head_dim)
    for h in range(c10.n_heads):
        oracle.attention_rows(x.Q[h], res.Kc[h], res.Vc[h], x.K_cur[h], x.V_cur[h], scale, rows)
    t2 = time.perf_counter()
    per_unit_s = (t1 - t0) + (t2 - t1) * c10.lq / len(rows)
    return {"value": round(per_unit_s * 1e3, 1), "unit": "ms", "cores": oracle.max_threads(), "kind": "oracle",
            "extrapolated": True,
            "sample": (f"1080P layer unit: scoring+selection+compaction of all 12 heads in full ({t1 - t0:.2f} s) "
                       f"+ attention of {len(rows)} of {c10.lq} query rows per head ({t2 - t1:.2f} s), "
                       f"attention extrapolated x{c10.lq / len(rows):.1f} to one unit"),
            "measured_s": round(t2 - t0, 2)}


# the sources the attention kernel is compiled from
ATTN_SOURCES = ("k_attn.hip", "attn_common.h", "attn_merge.h", "handover.h")


def _kernel_sha():
    """sha256 (first 16 hex digits) over the attention kernel's sources, in order."""
    import hashlib
    h = hashlib.sha256()
    for name in ATTN_SOURCES:
        with open(os.path.join(ROOT, "paper_2605_09681_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


if __name__ == "__main__":
    main()
