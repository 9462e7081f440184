"""Benchmark of the per-chunk stream step on one MI355X: score -> select -> compact -> attend.

Workload: the 80K-token history (81,920-slot bf16 pool, 30% of units already evicted, 32 query /
8 KV heads, d = 128, budget 16,384, a 665-token chunk).  Inputs are seeded synthetic streams
resident in HBM; ``--copies`` distinct copies of the inputs are rotated so that no step finds its
inputs in the 256 MB last-level (Infinity) cache.  Each of the K timed steps runs the whole path.

Prints one JSON line.  ``value`` is attention TFLOP/s over the whole step (attention work of a
step / step time); per-kernel rates and roofline fractions are in ``kernels`` and ``roofline``.
``cpu_baseline`` times the CPU oracle on one step of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import streamgen as sg  # noqa: E402

HBM_PEAK_GBPS = 8000.0
BF16_PEAK_TFLOPS = 2516.6
WORKLOAD = "history_80k"
CSRC = os.path.join(ROOT, "paper_2609_34653_amd", "csrc")

# HBM traffic of one call of each stage on the default workload, from two rocprofv3 --pmc passes
# over `bench.py --steps 5 --warmup 1 --no-cpu-baseline --no-graph --loop-steps 0 --no-ceilings
# --no-other-configs --copy-calibration-mb 1024` (FETCH_SIZE, then WRITE_SIZE; KiB per dispatch,
# summed over the stage's kernels).  Scaled by what the same
# counters read for the calibration copy (1 GiB read + 1 GiB written by one elementwise kernel):
# FETCH_SIZE reads 524,297 KiB for 1,048,576 KiB fetched (x2.000), WRITE_SIZE reads 1,048,576 KiB
# (x1.000).  Each entry carries a hash of the sources of its kernels and is reported only while
# they are unchanged (otherwise null: the counters describe other code).
FETCH_SCALE, WRITE_SCALE = 2.000, 1.000
COUNTER_TRAFFIC = {
    "score": (("score.hip", "common.h"), "8b69f17ec98290ac", 57031.8, 161.3),
    "select": (("select.hip", "common.h"), "3b421e2e735569a4", 20.6, 3.0),
    "compact": (("compact.hip", "common.h"), "edffe68dcca4279a", 34169.7, 68113.6),
    "attend": (("attention.hip", "combine.h", "common.h"), "6a3ec62fcf042dfe", 54348.0, 43058.8),
    "compact_rope": (("compact.hip", "common.h"), "edffe68dcca4279a", 34232.0, 68041.7),
    "decode": (("decode.hip", "combine.h", "common.h"), "2ec842b1862a6e13", 34325.6, 536.0),
}


# Matrix-core busy fraction of the chunk attention kernel from rocprofv3 counters over
# `bench.py --steps 5 --warmup 1 --no-cpu-baseline --no-graph --loop-steps 0 --no-other-configs`:
# SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / 8 XCDs x 1,024 SIMDs) per dispatch (the MFMA-only
# probe reads 0.97 with this normalisation); keyed by the kernel's sources like COUNTER_TRAFFIC.
MFMA_BUSY = (("attention.hip", "combine.h", "common.h"), "6a3ec62fcf042dfe", 0.549)


def mfma_busy(config):
    """Counter-measured MFMA busy fraction of attn_kernel, or None if not measured on this
    code/config."""
    import hashlib
    srcs, digest, frac = MFMA_BUSY
    if config != WORKLOAD:
        return None
    h = hashlib.sha256()
    for f in srcs:
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    return frac if h.hexdigest()[:16] == digest else None


def graph_time(fn, reps, dev, use_graph=True, replays=5):
    """GPU time of fn() over `reps` calls, captured in one HIP graph and replayed (the calls are
    too short for host-side launches to keep the GPU busy); if capture fails, or use_graph is
    False, timed with events around host launches instead.  After one untimed replay (or loop),
    `replays` replays are timed one by one: returns {"us": mean per call over all of them,
    "us_p10"/"us_p50"/"us_p90": percentiles of the per-replay means, "timing": method,
    "replays", "calls_per_replay"}."""
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(run):
        run()
        torch.cuda.synchronize()
        per = []
        for _ in range(replays):
            e0.record()
            run()
            e1.record()
            torch.cuda.synchronize()
            per.append(e0.elapsed_time(e1) / reps * 1e3)
        return per

    how = "graph replay"
    try:
        if not use_graph:
            raise RuntimeError("graph capture disabled")
        side = torch.cuda.Stream(device=dev)
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            fn(0)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for i in range(reps):
                fn(i)
        per = timed(g.replay)
        del g
    except Exception:  # pragma: no cover - capture unsupported or disabled
        torch.cuda.synchronize()
        how = "events around host launches"

        def loop():
            for i in range(reps):
                fn(i)
        per = timed(loop)
    p10, p50, p90 = np.percentile(per, [10, 50, 90])
    return {"us": float(np.mean(per)), "us_p10": float(p10), "us_p50": float(p50),
            "us_p90": float(p90), "timing": how, "replays": replays, "calls_per_replay": reps}


def graph_time_us(fn, reps, dev, use_graph=True):
    """(mean GPU time per call in us, method): graph_time without the distribution."""
    r = graph_time(fn, reps, dev, use_graph)
    return r["us"], r["timing"]


def counter_traffic(stage, config):
    """Calibrated HBM bytes per call of `stage`, or None if not measured on this code/config."""
    import hashlib
    srcs, digest, fetch_kib, write_kib = COUNTER_TRAFFIC[stage]
    if config != WORKLOAD:
        return None
    h = hashlib.sha256()
    for f in srcs:
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    if h.hexdigest()[:16] != digest:
        return None
    return int(round((fetch_kib * FETCH_SCALE + write_kib * WRITE_SCALE) * 1024))


def attn_flops(L, kept, Hq, d):
    return 4.0 * Hq * d * (L * kept + L * (L + 1) / 2)


def score_bytes(lay, H, d, elt, U):
    live = int((lay.unit_id >= 0).sum())
    return live * H * d * elt + lay.n_slots * 5 + U * 24


def compact_bytes(kept, L, H, d, elt, cap, U):
    row = H * d * elt
    return 2 * row * (2 * kept + 2 * L) + kept * 9 + L * 5 + cap * 13 + U * 13


def progress(msg):
    """One line on stderr as each part of the run finishes (the JSON result goes to stdout)."""
    print(f"bench: {msg}", file=sys.stderr, flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--copies", type=int, default=4)
    ap.add_argument("--config", default=WORKLOAD)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="run a plain elementwise copy kernel (reads and writes this many MiB) "
                         "three times before the warmup: a known-size reference for hardware "
                         "byte counters")
    ap.add_argument("--no-ceilings", dest="ceilings", action="store_false",
                    help="skip the measured-ceiling probes (library GEMM, device copy)")
    ap.add_argument("--loop-steps", type=int, default=64,
                    help="steps of the stream-loop layout comparison (0 = skip)")
    ap.add_argument("--no-other-configs", dest="other_configs", action="store_false",
                    help="skip the single-layer 8K and 36-layer 32K measurements")
    ap.add_argument("--no-graph", action="store_true",
                    help="time the standalone calls with events around host launches instead of "
                         "one captured HIP graph (for counter passes)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}): the stream step "
              "has no multi-GPU path.", file=sys.stderr)
        sys.exit(2)

    from paper_2609_34653_amd import omnitide as ot
    from paper_2609_34653_amd.step import StreamStep
    ot.lib()
    dev = torch.device("cuda:0")
    cfg = sg.CONFIG_BY_NAME[args.config]
    stream = sg.make_stream(cfg)
    lay, seg = stream.layout, stream.segment(0)
    H, d, Hq, L = cfg.n_kv_heads, cfg.head_dim, cfg.n_q_heads, lay.chunk_len
    elt = 2 if cfg.dtype == "bf16" else 4
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)  # noqa: E731
    copies = []
    for _ in range(args.copies):
        copies.append(dict(
            k=seg.k_hist.to(dev)[None].contiguous(), v=seg.v_hist.to(dev)[None].contiguous(),
            uid=t(lay.unit_id), mod=t(lay.modality), pos=t(lay.pos),
            kc=seg.k_chunk.to(dev)[None].contiguous(), vc=seg.v_chunk.to(dev)[None].contiguous(),
            cm=t(lay.chunk_modality), cu=t(lay.chunk_unit), q=seg.q.to(dev)[None].contiguous()))
    st = StreamStep(n_seg=1, n_slots=lay.n_slots, n_units=lay.n_units, n_q_heads=Hq,
                    n_kv_heads=H, head_dim=d, chunk_len=L, budget=cfg.budget, recent=cfg.recent,
                    page_size=cfg.page_size, weights=cfg.weights, device=dev)
    s = torch.cuda.current_stream()

    def step(i, ev=None):
        c = copies[i % len(copies)]
        if ev is not None:
            ev[0].record(s)
        st.score(c["k"], c["uid"], c["mod"])
        if ev is not None:
            ev[1].record(s)
        st.select()
        if ev is not None:
            ev[2].record(s)
        st.compact(c["k"], c["v"], c["uid"], c["mod"], c["pos"], c["kc"], c["vc"], c["cm"],
                   c["cu"])
        if ev is not None:
            ev[3].record(s)
        st.attend(c["q"], cfg.scale)
        if ev is not None:
            ev[4].record(s)

    if args.copy_calibration_mb:
        # torch.neg is one elementwise kernel dispatch (a same-dtype copy_ would go to a runtime
        # blit instead): exactly n bytes read and n bytes written per launch.
        n = (args.copy_calibration_mb << 20) // 4
        a = torch.ones(n, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        for _ in range(3):
            torch.neg(a, out=b)
        torch.cuda.synchronize()
        del a, b
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    status = int(st.d_status.item())
    if status != 0:
        raise RuntimeError(f"device status {status}: {ot.status_string(status)}")
    kept = int(st.kept_tokens.item())
    n_ctx = int(st.n_ctx.item())

    # Per-call times: events around each call of K host-launched steps.
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(s)
    for i in range(args.steps):
        step(args.warmup + i, evs[i])
    end.record(s)
    torch.cuda.synchronize()
    launched_ms_per_step = start.elapsed_time(end) / args.steps
    per = np.array([[e[j].elapsed_time(e[j + 1]) for j in range(4)] for e in evs])  # ms

    # Whole-step time: the K timed steps (all four calls each, no host synchronisation, input
    # copies rotating) captured in one HIP graph; three untimed replays warm the graph (and let
    # the clocks settle under this load), then one replay is timed.  The last step's output is
    # checked bitwise against the same step launched from the host.
    step_timing = "one HIP graph of the K steps"
    try:
        if args.no_graph:
            raise RuntimeError("graph capture disabled")
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for i in range(args.steps):
                step(args.warmup + i)
        torch.cuda.synchronize()
        for _ in range(3):
            g.replay()
        torch.cuda.synchronize()
        wall0 = time.perf_counter()
        start.record(s)
        g.replay()
        end.record(s)
        torch.cuda.synchronize()
        wall = time.perf_counter() - wall0
        ms_per_step = start.elapsed_time(end) / args.steps
        # the spread: four more replays of the same K steps, each timed on its own
        step_replays = [ms_per_step]
        for _ in range(4):
            start.record(s)
            g.replay()
            end.record(s)
            torch.cuda.synchronize()
            step_replays.append(start.elapsed_time(end) / args.steps)
        out_graph = st.out.clone()
        step(args.warmup + args.steps - 1)
        torch.cuda.synchronize()
        if not torch.equal(out_graph, st.out):
            raise RuntimeError("graph replay differs from the launched step")
        del g
    except RuntimeError as exc:
        if not args.no_graph and "differs" in str(exc):
            raise
        step_timing = "host launches"
        step_replays = None
        wall0 = time.perf_counter()
        start.record(s)
        for i in range(args.steps):
            step(args.warmup + i)
        end.record(s)
        torch.cuda.synchronize()
        wall = time.perf_counter() - wall0
        ms_per_step = start.elapsed_time(end) / args.steps
    status = int(st.d_status.item())
    if status != 0:
        raise RuntimeError(f"device status {status}: {ot.status_string(status)}")
    avg = per.mean(axis=0)
    names = ["score", "select", "compact", "attend"]

    # Per-call times as the step runs them back to back: each call captured `4 * steps` times
    # in one HIP graph (rotating the input copies) and replayed; the host-launched event times
    # above are kept beside them (they include launch gaps on calls of a few microseconds).
    def call(name):
        def f(i):
            c = copies[i % len(copies)]
            if name == "score":
                st.score(c["k"], c["uid"], c["mod"])
            elif name == "select":
                st.select()
            elif name == "compact":
                st.compact(c["k"], c["v"], c["uid"], c["mod"], c["pos"], c["kc"], c["vc"],
                           c["cm"], c["cu"])
            else:
                st.attend(c["q"], cfg.scale)
        return f
    progress(f"step: {ms_per_step:.4f} ms per step ({step_timing})")
    us, dist = {}, {}
    for j, n in enumerate(names):
        dist[n] = graph_time(call(n), 4 * args.steps, dev, not args.no_graph)
        us[n] = dist[n]["us"]
    torch.cuda.synchronize()

    flops = attn_flops(L, kept, Hq, d)
    sbytes = score_bytes(lay, H, d, elt, lay.n_units)
    cbytes = compact_bytes(kept, L, H, d, elt, st.cap_dst, lay.n_units)
    sel_bytes = lay.n_units * (8 + 4 * 4) + lay.n_units * 9 + 4
    attn_tflops = flops / (us["attend"] * 1e-6) / 1e12
    kernels = {
        "score": {"us": us["score"], "bytes": sbytes,
                  "GBps": sbytes / (us["score"] * 1e-6) / 1e9},
        "select": {"us": us["select"], "bytes": sel_bytes,
                   "GBps": sel_bytes / (us["select"] * 1e-6) / 1e9},
        "compact": {"us": us["compact"], "bytes": cbytes,
                    "GBps": cbytes / (us["compact"] * 1e-6) / 1e9},
        "attend": {"us": us["attend"], "flops": flops, "TFLOPs": attn_tflops},
    }
    for j, n in enumerate(names):
        for key in ("us_p10", "us_p50", "us_p90", "timing", "replays", "calls_per_replay"):
            kernels[n][key] = dist[n][key]
        kernels[n]["us_host_launched"] = avg[j] * 1e3
    for k in ("score", "compact"):
        kernels[k]["frac_hbm"] = kernels[k]["GBps"] / HBM_PEAK_GBPS
    # Minimum movement: kept history rows whose slot changes (the rest could stay in place), read
    # and written once each for K and V -- the figure a selective migration would move.
    src = st.src_of_dst[:kept].cpu().numpy()
    moved = int(np.count_nonzero(src != np.arange(kept)))
    kernels["compact"]["moved_rows"] = moved
    kernels["compact"]["min_move_bytes"] = 2 * moved * 2 * H * d * elt
    kernels["attend"]["frac_mfma"] = attn_tflops / BF16_PEAK_TFLOPS
    for k in kernels:
        kernels[k]["traffic"] = counter_traffic(k, cfg.name)
    for k in kernels:
        kernels[k] = {a: (round(b, 4) if isinstance(b, float) else b) for a, b in kernels[k].items()}

    # Compaction with rotary re-encoding of the moved keys (base 1e6, all 128 dims, split-halves
    # pairing), timed on its own after the step loop: same rows moved, so the same algorithmic
    # bytes; not part of the step.
    c = copies[0]
    rope = (1.0e6, d, 0)
    st.compact(c["k"], c["v"], c["uid"], c["mod"], c["pos"], c["kc"], c["vc"], c["cm"], c["cu"],
               rope=rope)
    def rope_call(i):
        c = copies[i % len(copies)]
        st.compact(c["k"], c["v"], c["uid"], c["mod"], c["pos"], c["kc"], c["vc"], c["cm"],
                   c["cu"], rope=rope)
    rope_us, rope_how = graph_time_us(rope_call, args.steps, dev, not args.no_graph)
    kernels["compact_rope"] = {"us": round(rope_us, 4), "bytes": cbytes, "timing": rope_how,
                               "GBps": round(cbytes / (rope_us * 1e-6) / 1e9, 4),
                               "frac_hbm": round(cbytes / (rope_us * 1e-6) / 1e9 / HBM_PEAK_GBPS,
                                                 4),
                               "traffic": counter_traffic("compact_rope", cfg.name),
                               "in_step": False}

    # Decode attention of one new token (all 32 query heads) over the compacted pool of this
    # workload (n_ctx rows), timed on its own: four copies of the pool are rotated so that the
    # reads come from HBM, not the 256 MB last-level cache.
    pools = [(st.k_dst.clone(), st.v_dst.clone()) for _ in range(4)]
    qd = torch.randn(1, 1, Hq, d, device=dev).to(torch.bfloat16)
    od = torch.empty(1, 1, Hq, d, device=dev)
    nbd = ot.omnitide_decode_workspace_bytes(1, st.cap_dst, 1, Hq, H, d)
    wsd = torch.zeros(max(nbd, 1), dtype=torch.uint8, device=dev)
    def dec_call(i):
        kp, vp = pools[i % len(pools)]
        ot.omnitide_decode_attn(qd, kp, vp, st.n_ctx, cfg.scale, od, wsd, st.d_status)
    dec_us, dec_how = graph_time_us(dec_call, 4 * args.steps, dev, not args.no_graph)
    dbytes = n_ctx * H * d * elt * 2 + Hq * d * (2 + 4)
    kernels["decode"] = {"us": round(dec_us, 4), "bytes": dbytes, "timing": dec_how,
                         "GBps": round(dbytes / (dec_us * 1e-6) / 1e9, 4),
                         "frac_hbm": round(dbytes / (dec_us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
                         "traffic": counter_traffic("decode", cfg.name), "n_ctx": n_ctx,
                         "in_step": False}
    del pools

    # Span plan (recent units whole; older units keep their markers, 256 leading tokens of each
    # video span and 16 of each audio span, and 1,024 text tokens oldest first; trimmed toward
    # the budget) and compaction of its kept slots, each timed on its own after the step loop
    # on the same pool.
    sp = dict(low=cfg.budget, high=cfg.budget, recent=cfg.recent, sink_video=256, sink_audio=16,
              text_budget=1024)
    c = copies[0]
    st.score(c["k"], c["uid"], c["mod"])
    def plan_call(i):
        c = copies[i % len(copies)]
        st.plan_spans(c["uid"], c["mod"], sp["low"], sp["high"], sp["recent"], sp["sink_video"],
                      sp["sink_audio"], sp["text_budget"])
    plan_us, plan_how = graph_time_us(plan_call, args.steps, dev, not args.no_graph)
    torch.cuda.synchronize()
    kept_sp = int(st.kept_tokens.item())
    def span_compact_call(i):
        c = copies[i % len(copies)]
        st.compact_spans(c["k"], c["v"], c["uid"], c["mod"], c["pos"], c["kc"], c["vc"],
                         c["cm"], c["cu"])
    sc_us, sc_how = graph_time_us(span_compact_call, args.steps, dev, not args.no_graph)
    torch.cuda.synchronize()
    status = int(st.d_status.item())
    if status != 0:
        raise RuntimeError(f"device status {status}: {ot.status_string(status)}")
    # tags in (unit id, modality), the slot mask out, per-unit structure in, keep_len out
    plan_bytes = lay.n_slots * (4 + 1 + 1) + lay.n_units * (4 * 4 + 4) + 4
    sbytes_c = compact_bytes(kept_sp, L, H, d, elt, st.cap_dst, lay.n_units)
    kernels["span_plan"] = {"us": round(plan_us, 4), "bytes": plan_bytes, "timing": plan_how,
                            "GBps": round(plan_bytes / (plan_us * 1e-6) / 1e9, 4),
                            "params": sp, "kept_tokens": kept_sp, "in_step": False}
    kernels["compact_spans"] = {"us": round(sc_us, 4), "bytes": sbytes_c, "timing": sc_how,
                                "GBps": round(sbytes_c / (sc_us * 1e-6) / 1e9, 4),
                                "frac_hbm": round(sbytes_c / (sc_us * 1e-6) / 1e9 / HBM_PEAK_GBPS,
                                                  4),
                                "kept_tokens": kept_sp, "in_step": False}

    progress("per-call timings done")
    kernels["layouts"] = layout_ablation(ot, st, copies[0], lay, cfg, L, H, Hq, d, dev,
                                         args.steps, n_ctx, not args.no_graph)

    progress("layout comparison done")
    if args.loop_steps > 0:
        kernels["stream_loop_layouts"] = stream_loop_ablation(ot, dev, args.loop_steps)
        progress("stream loop done")
    if args.other_configs:
        kernels["other_configs"] = other_configs(dev, args.steps, not args.no_graph)
        progress("other workloads done")

    value = flops / (ms_per_step * 1e-3) / 1e12
    result = {
        "metric": "chunk-attn TFLOP/s + score/compact GB/s (% roofline), 80K-token history, 1 GPU",
        "value": round(value, 3), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "step_timing": step_timing,
        "ms_per_step_host_launched": round(launched_ms_per_step, 4), "higher_is_better": True,
        "ms_per_step_replays": (None if step_replays is None else
                                {"timed_replay_and_4_more": [round(x, 4) for x in step_replays],
                                 "p10": round(float(np.percentile(step_replays, 10)), 4),
                                 "p50": round(float(np.percentile(step_replays, 50)), 4),
                                 "p90": round(float(np.percentile(step_replays, 90)), 4)}),
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {cfg.description}", "history_slots": lay.n_slots,
                   "live_tokens": int((lay.unit_id >= 0).sum()), "units": lay.n_units,
                   "budget": cfg.budget, "chunk_len": L, "n_q_heads": Hq, "n_kv_heads": H,
                   "head_dim": d, "page_size": cfg.page_size, "kept_tokens": kept,
                   "n_ctx": n_ctx, "input_copies": args.copies},
        "kernels": kernels,
        "roofline": {"bound": "mfma",
                     "kernel": "chunk attention call (attn_kernel + attn_combine_kernel)",
                     "timing": kernels["attend"]["timing"],
                     "achieved": round(attn_tflops, 3), "peak": BF16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(attn_tflops / BF16_PEAK_TFLOPS, 4),
                     "traffic": kernels["attend"]["traffic"],
                     "mfma_busy_counter": mfma_busy(cfg.name)},
        "wall_s_timed_region": round(wall, 4),
    }
    if args.ceilings:
        result["measured_ceilings"] = measured_ceilings(dev)
        c = result["measured_ceilings"]
        result["roofline"]["frac_of_measured_mfma"] = round(attn_tflops / c["mfma_bf16_tflops"], 4)
        result["roofline"]["frac_of_measured_mfma_randn"] = round(
            attn_tflops / c["mfma_bf16_randn_8w_tflops"], 4)
        for k in ("score", "compact"):
            kernels[k]["frac_of_measured_copy"] = round(kernels[k]["GBps"] / 1e3 /
                                                        c["copy_tbps"], 4)
    if not args.no_cpu_baseline:
        progress("CPU oracle baseline ...")
        result["cpu_baseline"] = cpu_baseline(cfg, stream, seg, flops)
    print(json.dumps(result), flush=True)


def measured_ceilings(dev):
    """What this chip sustains right now, beside the published peaks: a large bf16 GEMM through
    the vendor library (torch.matmul; 8192^3, fp32 accumulate), an elementwise copy of 1 GiB in /
    1 GiB out (torch.neg), each the best of 5 timed launches, and an MFMA-only probe with the
    shader clock it ran at."""
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def best(fn, reps=5):
        fn()
        torch.cuda.synchronize()
        t = []
        for _ in range(reps):
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            t.append(e0.elapsed_time(e1))
        return min(t) * 1e-3
    n = 8192
    a = torch.randn(n, n, device=dev).to(torch.bfloat16)
    b = torch.randn(n, n, device=dev).to(torch.bfloat16)
    gemm_s = best(lambda: torch.matmul(a, b))
    del a, b
    x = torch.ones((1 << 30) // 4, dtype=torch.float32, device=dev)
    y = torch.empty_like(x)
    copy_s = best(lambda: torch.neg(x, out=y))
    del x, y
    out = {"gemm_bf16_tflops": round(2.0 * n ** 3 / gemm_s / 1e12, 1),
           "copy_tbps": round(2.0 * (1 << 30) / copy_s / 1e12, 3),
           "method": "torch.matmul bf16 8192^3 and torch.neg over 1 GiB, best of 5"}
    # Matrix-core probe (libomnitide_probe.so): 1,024 workgroups x 4 waves, each wave four
    # independent 32x32x16 bf16 MFMA chains; shader clock from wave 0's counters.
    import ctypes
    from paper_2609_34653_amd import build as b
    probe = ctypes.CDLL(b.PROBE_PATH)
    probe.omnitide_probe_mfma.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                          ctypes.c_void_p, ctypes.c_void_p]
    n_wg, iters = 1024, 20000
    sink = torch.empty(n_wg * 256, device=dev)
    clocks = torch.zeros(2, dtype=torch.int64, device=dev)
    stream = torch.cuda.current_stream().cuda_stream

    def run_probe():
        if probe.omnitide_probe_mfma(n_wg, iters, ctypes.c_void_p(sink.data_ptr()),
                                     ctypes.c_void_p(clocks.data_ptr()), stream) != 0:
            raise RuntimeError("probe launch failed")
    probe_s = best(run_probe, 3)
    cyc, ticks = (int(x) for x in clocks.cpu())
    out["mfma_bf16_tflops"] = round(n_wg * 4 * iters * 4 * 32768 / probe_s / 1e12, 1)
    out["sclk_ghz_under_mfma"] = round(cyc / (ticks / 100e6) / 1e9, 3) if ticks else None
    # The same with N(0,1) operands rounded to bf16 (the attention inputs' statistics): the
    # matrix cores draw more power on such bits and the clock drops.  Run at 1,024 workgroups
    # (16 waves per CU) and at 512 (8 per CU, the chunk attention's occupancy).
    probe.omnitide_probe_mfma_ops.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                              ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    gen = torch.Generator(device=dev).manual_seed(1)
    ops = torch.randn(64 * 8 * 64 * 8, generator=gen, device=dev).to(torch.bfloat16)
    for wg, key in ((1024, "mfma_bf16_randn_tflops"), (512, "mfma_bf16_randn_8w_tflops")):
        it_ops = iters // 2

        def run_ops():
            if probe.omnitide_probe_mfma_ops(wg, it_ops, ctypes.c_void_p(ops.data_ptr()),
                                             ctypes.c_void_p(sink.data_ptr()),
                                             ctypes.c_void_p(clocks.data_ptr()), stream) != 0:
                raise RuntimeError("probe launch failed")
        ops_s = best(run_ops, 3)
        out[key] = round(wg * 4 * it_ops * 8 * 32768 / ops_s / 1e12, 1)
        if wg == 1024:
            cyc, ticks = (int(x) for x in clocks.cpu())
            out["sclk_ghz_under_mfma_randn"] = (round(cyc / (ticks / 100e6) / 1e9, 3)
                                                if ticks else None)
    out["method"] += ("; an MFMA-only probe (1,024 x 4 waves x 20,000 x 4 independent "
                      "32x32x16 bf16 MFMAs) with the shader clock of its first wave, and the "
                      "same with N(0,1) bf16 operands at 1,024 and 512 workgroups")
    return out


def layout_ablation(ot, st, c, lay, cfg, L, H, Hq, d, dev, reps, n_ctx, use_graph=True):
    """The same retention plan (the step's whole-unit selection) under three physical layouts:
    native (logical eviction, the chunk in the lowest empty run, attention over the holey span),
    ordered-suffix packing (eviction, then the suffix whose packing saves >= 1 page of 256
    slots, then the chunk) and eager compaction (the step's own compact + attend).  Each
    maintenance call is timed from its layout's state before it: `reps` repetitions of
    [restore the tags from a snapshot, call] in one captured graph, minus the same graph without
    the call; attention is `reps` calls over the final layout.  `evict_rope_us` is the eviction
    with the rotary adjustment of the keys that stay (base 1e6, 128 dims, split halves; on a copy
    of the keys), the native counterpart of the eager path's rotary compaction
    (kernels.compact_rope)."""
    cap = lay.n_slots + L
    pad = cap - lay.n_slots
    i32 = dict(dtype=torch.int32, device=dev)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)  # noqa: E731
    tags0 = (t(np.concatenate([lay.unit_id, np.full(pad, -1)]).astype(np.int32)),
             t(np.concatenate([lay.pos, np.full(pad, -1)]).astype(np.int32)),
             t(np.concatenate([lay.modality, np.full(pad, 1)]).astype(np.uint8)))
    k = torch.cat([c["k"][0], torch.zeros(pad, H, d, dtype=c["k"].dtype, device=dev)])[None]
    v = torch.cat([c["v"][0], torch.zeros(pad, H, d, dtype=c["v"].dtype, device=dev)])[None]
    k, v = k.contiguous(), v.contiguous()
    uid, pos, mod = (x.clone() for x in tags0)
    remap = torch.zeros(lay.n_units, **i32)
    kept, nku, span, slot, cut, moved = (torch.zeros(1, **i32) for _ in range(6))
    ws_e = torch.zeros(ot.omnitide_evict_native_workspace_bytes(1, lay.n_units),
                       dtype=torch.uint8, device=dev)
    ws_er = torch.zeros(ot.omnitide_evict_native_rope_workspace_bytes(1, lay.n_units, cap),
                        dtype=torch.uint8, device=dev)
    k_rope = k.clone()
    ws_p = torch.zeros(ot.omnitide_pack_suffix_workspace_bytes(0, 1, cap, H, d),
                       dtype=torch.uint8, device=dev)
    ws_a = torch.zeros(ot.omnitide_span_attn_workspace_bytes(1, cap, L, Hq, H, d),
                       dtype=torch.uint8, device=dev)
    ws_c = torch.zeros(ot.omnitide_place_chunk_workspace_bytes(1, cap), dtype=torch.uint8,
                       device=dev)
    out = torch.zeros(1, L, Hq, d, device=dev)

    def restore(snap):
        for dst, src in zip((uid, pos, mod), snap):
            dst.copy_(src)

    def evict():
        ot.omnitide_evict_native(uid, pos, 1, lay.n_units, st.unit_len, remap, kept, nku, span,
                                 ws_e, keep=st.keep, d_status=st.d_status)

    def evict_rope():
        ot.omnitide_evict_native_rope(uid, pos, k_rope, 1, lay.n_units, st.unit_len, remap, kept,
                                      nku, span, ws_er, 1.0e6, 128, ot.ROPE_HALF, keep=st.keep,
                                      d_status=st.d_status)

    def pack():
        ot.omnitide_pack_suffix(k, v, 256, 1, uid, mod, pos, span, cut, moved, ws_p)

    def place():
        ot.omnitide_place_chunk(k, v, uid, mod, pos, c["kc"], c["vc"], c["cm"], c["cu"], kept,
                                nku, slot, span, ws_c, d_status=st.d_status)

    def attend(position_order=False):
        ot.omnitide_span_attn(c["q"], k, v, pos, span, kept, cfg.scale, out, ws_a, st.d_status,
                              position_order=position_order)

    def staged(snap, call):
        """(us per call, method): graph of [restore, call] minus graph of [restore]."""
        span0 = span.clone()
        def with_call(i):
            restore(snap)
            span.copy_(span0)
            call()
        def without(i):
            restore(snap)
            span.copy_(span0)
        t1, how = graph_time_us(with_call, reps, dev, use_graph)
        t0, _ = graph_time_us(without, reps, dev, use_graph)
        return max(t1 - t0, 0.0), how

    res = {}
    for name, packed in (("native", False), ("ordered_suffix", True)):
        restore(tags0)
        evict()
        snap_ev = tuple(x.clone() for x in (uid, pos, mod))
        span_ev = span.clone()
        if packed:
            pack()
        snap_pk = tuple(x.clone() for x in (uid, pos, mod))
        span_pk = span.clone()
        place()
        torch.cuda.synchronize()
        status = int(st.d_status.item())
        if status != 0:
            raise RuntimeError(f"device status {status}: {ot.status_string(status)}")
        u = uid.cpu().numpy()
        occ = np.nonzero(u >= 0)[0]
        sp = int(span.item())
        r = {"span": sp, "pages_256": -(-sp // 256),
             "active_pages_256": int(len(np.unique(occ // 256))),
             "active_tiles_64": int(len(np.unique(occ // 64))),
             "chunk_slot": int(slot.item())}
        if packed:
            r.update(cut=int(cut.item()), moved_rows=int(moved.item()))
        attn_us, how = graph_time_us(lambda i: attend(), reps, dev, use_graph)
        r["attend_position_order_us"], _ = graph_time_us(lambda i: attend(True), reps, dev,
                                                         use_graph)
        final = tuple(x.clone() for x in (uid, pos, mod))
        span_final = span.clone()
        span.copy_(torch.zeros_like(span))
        r["evict_us"], _ = staged(tags0, evict)
        span.copy_(torch.zeros_like(span))
        r["evict_rope_us"], _ = staged(tags0, evict_rope)
        span.copy_(span_ev)
        if packed:
            r["pack_us"], _ = staged(snap_ev, pack)
        span.copy_(span_pk)
        r["place_us"], _ = staged(snap_pk, place)
        restore(final)
        span.copy_(span_final)
        r["attend_us"] = attn_us
        r["timing"] = how
        r = {a: (round(b, 3) if isinstance(b, float) else b) for a, b in r.items()}
        res[name] = r
    res["eager"] = {"span": n_ctx, "pages_256": -(-n_ctx // 256),
                    "active_pages_256": -(-n_ctx // 256), "active_tiles_64": -(-n_ctx // 64),
                    "note": "the step's compact + attend (kernels.compact, kernels.attend)"}
    return res


def stream_loop_ablation(ot, dev, steps, page=64, suffix_pages=(1, 11)):
    """The 64-step stream loop (prefill 16,384 tokens, then 665-token chunks, budget 16,384)
    with the same selections under three layouts: eager (the step: compact + chunk attention,
    ping-pong pools), native (logical eviction, the chunk in the lowest empty run, attention
    over the holey span) and ordered-suffix packing (native plus, after each eviction, the
    suffix whose packing saves >= T pages of `page` slots, for each T in `suffix_pages`).  The
    eager path's score + select decide each step's plan; the native pools apply the same keep
    flags (their unit ids and positions coincide with the eager pool's).  Attention over a
    native pool runs twice per step: skipping empty 64-slot tiles, and traversing the whole
    span (as kernels without tile skipping do).  Each step then decodes the chunk's last token
    over each layout (the eager pool's rows [0, n_ctx); a native pool's span, with and without
    tile skipping), as the decode half of the paper's layout ablation.  A third attention over
    each native pool takes its entries in position order through a position -> slot index (the
    compacted pool's tiles, gathered), and so does a third decode.  Attention, decode and
    maintenance are timed with events around their launches (the per-step latency percentiles
    come from the same events); spans and active pages are recorded per step."""
    from paper_2609_34653_amd.step import StreamStep
    cfg = sg.CONFIG_BY_NAME["stream_loop_64x665"]
    stream = sg.make_stream(cfg)
    lay, seg0 = stream.layout, stream.segment(0)
    U, L = 512, 665
    H, d, Hq = cfg.n_kv_heads, cfg.head_dim, cfg.n_q_heads
    cap_e, cap_n = cfg.budget + L, 131072
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)  # noqa: E731
    chunks = []
    for i in range(steps):
        clay, cseg = sg.loop_chunk(cfg, i)
        chunks.append(dict(kc=cseg.k_chunk.to(dev)[None].contiguous(),
                           vc=cseg.v_chunk.to(dev)[None].contiguous(),
                           q=cseg.q.to(dev)[None].contiguous(), cm=t(clay.chunk_modality),
                           cu=t(clay.chunk_unit)))
    mk = lambda n: StreamStep(n_seg=1, n_slots=n, n_units=U, n_q_heads=Hq, n_kv_heads=H,  # noqa
                              head_dim=d, chunk_len=L, budget=cfg.budget, recent=cfg.recent,
                              page_size=cfg.page_size, weights=cfg.weights, cap_dst=cap_e,
                              device=dev)
    st_first, st_a, st_b = mk(lay.n_slots), mk(cap_e), mk(cap_e)
    src = dict(k=seg0.k_hist.to(dev)[None].contiguous(), v=seg0.v_hist.to(dev)[None].contiguous(),
               uid=t(lay.unit_id), mod=t(lay.modality), pos=t(lay.pos))
    i32 = dict(dtype=torch.int32, device=dev)
    pad = cap_n - lay.n_slots

    def native_pool(min_pages):
        k = torch.zeros(1, cap_n, H, d, dtype=torch.bfloat16, device=dev)
        v = torch.zeros_like(k)
        k[0, :lay.n_slots] = src["k"][0]
        v[0, :lay.n_slots] = src["v"][0]
        return dict(k=k, v=v, min_pages=min_pages,
                    uid=t(np.concatenate([lay.unit_id, np.full(pad, -1)]).astype(np.int32)),
                    pos=t(np.concatenate([lay.pos, np.full(pad, -1)]).astype(np.int32)),
                    mod=t(np.concatenate([lay.modality, np.full(pad, 1)]).astype(np.uint8)),
                    remap=torch.zeros(U, **i32), kept=torch.zeros(1, **i32),
                    nku=torch.zeros(1, **i32), span=torch.zeros(1, **i32),
                    slot=torch.zeros(1, **i32), cut=torch.zeros(1, **i32),
                    moved=torch.zeros(1, **i32), out=torch.zeros(1, L, Hq, d, device=dev),
                    moved_sum=torch.zeros(1, **i32), migrations=torch.zeros(1, **i32))
    pools = {"native": native_pool(0)}
    for T in suffix_pages:
        pools[f"ordered_suffix_T{T}"] = native_pool(T)
    ws_e = torch.zeros(ot.omnitide_evict_native_workspace_bytes(1, U), dtype=torch.uint8,
                       device=dev)
    ws_p = torch.zeros(ot.omnitide_pack_suffix_workspace_bytes(0, 1, cap_n, H, d),
                       dtype=torch.uint8, device=dev)
    ws_c = torch.zeros(ot.omnitide_place_chunk_workspace_bytes(1, cap_n), dtype=torch.uint8,
                       device=dev)
    ws_a = torch.zeros(ot.omnitide_span_attn_workspace_bytes(1, cap_n, L, Hq, H, d),
                       dtype=torch.uint8, device=dev)
    ws_d = torch.zeros(max(1, ot.omnitide_decode_workspace_bytes(1, cap_e, 1, Hq, H, d)),
                       dtype=torch.uint8, device=dev)
    ws_ds = torch.zeros(ot.omnitide_decode_span_workspace_bytes(1, cap_n, 1, Hq, H, d),
                        dtype=torch.uint8, device=dev)
    dec_e = torch.zeros(1, 1, Hq, d, device=dev)
    for pl in pools.values():
        pl["dec"] = torch.zeros(1, 1, Hq, d, device=dev)
        pl["qpos"] = torch.zeros(1, **i32)
    names = ["eager"] + list(pools)
    ev = {n: [[torch.cuda.Event(enable_timing=True) for _ in range(11)] for _ in range(steps)]
          for n in names}
    spans = {n: torch.zeros(steps, **i32) for n in names}
    active = {n: torch.zeros(steps, **i32) for n in names}
    diff = torch.zeros(len(pools), device=dev)
    diff_dec = torch.zeros(len(pools), device=dev)
    diff_pos = torch.zeros(len(pools), device=dev)
    diff_dec_pos = torch.zeros(len(pools), device=dev)
    s = torch.cuda.current_stream()
    d_status = st_first.d_status
    for i in range(steps):
        c = chunks[i]
        st = st_first if i == 0 else (st_a if i % 2 else st_b)
        st.d_status = d_status
        e = ev["eager"][i]
        e[4].record(s)
        st.score(src["k"], src["uid"], src["mod"])
        st.select()
        e[0].record(s)
        st.compact(src["k"], src["v"], src["uid"], src["mod"], src["pos"], c["kc"], c["vc"],
                   c["cm"], c["cu"])
        e[1].record(s)
        st.attend(c["q"], cfg.scale)
        e[2].record(s)
        qd = c["q"][:, L - 1:L]                      # the chunk's last token decodes
        ot.omnitide_decode_attn(qd, st.k_dst, st.v_dst, st.n_ctx, cfg.scale, dec_e, ws_d,
                                d_status)
        e[5].record(s)
        spans["eager"][i:i + 1].copy_(st.n_ctx)
        active["eager"][i:i + 1].copy_((st.n_ctx + page - 1) // page)
        for j, (n, pl) in enumerate(pools.items()):
            e = ev[n][i]
            e[0].record(s)
            ot.omnitide_evict_native(pl["uid"], pl["pos"], 1, U, st.unit_len, pl["remap"],
                                     pl["kept"], pl["nku"], pl["span"], ws_e, keep=st.keep,
                                     d_status=d_status)
            if pl["min_pages"] > 0:
                ot.omnitide_pack_suffix(pl["k"], pl["v"], page, pl["min_pages"], pl["uid"],
                                        pl["mod"], pl["pos"], pl["span"], pl["cut"],
                                        pl["moved"], ws_p)
                pl["moved_sum"] += pl["moved"]
                pl["migrations"] += (pl["cut"] >= 0).to(torch.int32)
            ot.omnitide_place_chunk(pl["k"], pl["v"], pl["uid"], pl["mod"], pl["pos"], c["kc"],
                                    c["vc"], c["cm"], c["cu"], pl["kept"], pl["nku"], pl["slot"],
                                    pl["span"], ws_c, d_status=d_status)
            e[1].record(s)
            ot.omnitide_span_attn(c["q"], pl["k"], pl["v"], pl["pos"], pl["span"], pl["kept"],
                                  cfg.scale, pl["out"], ws_a, d_status, skip_empty_tiles=True)
            e[2].record(s)
            ot.omnitide_span_attn(c["q"], pl["k"], pl["v"], pl["pos"], pl["span"], pl["kept"],
                                  cfg.scale, pl["out"], ws_a, d_status, skip_empty_tiles=False)
            e[3].record(s)
            torch.add(pl["kept"], L - 1, out=pl["qpos"])   # position of the decoding token
            e[5].record(s)
            ot.omnitide_decode_span_attn(qd, pl["k"], pl["v"], pl["pos"], pl["span"],
                                         pl["qpos"], cfg.scale, pl["dec"], ws_ds, d_status,
                                         skip_empty_tiles=True)
            e[6].record(s)
            ot.omnitide_decode_span_attn(qd, pl["k"], pl["v"], pl["pos"], pl["span"],
                                         pl["qpos"], cfg.scale, pl["dec"], ws_ds, d_status,
                                         skip_empty_tiles=False)
            e[7].record(s)
            diff_dec[j] = torch.maximum(diff_dec[j], (pl["dec"] - dec_e).abs().max())
            diff[j] = torch.maximum(diff[j], (pl["out"] - st.out).abs().max())
            e[8].record(s)
            ot.omnitide_span_attn(c["q"], pl["k"], pl["v"], pl["pos"], pl["span"], pl["kept"],
                                  cfg.scale, pl["out"], ws_a, d_status, position_order=True)
            e[9].record(s)
            ot.omnitide_decode_span_attn(qd, pl["k"], pl["v"], pl["pos"], pl["span"],
                                         pl["qpos"], cfg.scale, pl["dec"], ws_ds, d_status,
                                         position_order=True)
            e[10].record(s)
            diff_pos[j] = torch.maximum(diff_pos[j], (pl["out"] - st.out).abs().max())
            diff_dec_pos[j] = torch.maximum(diff_dec_pos[j], (pl["dec"] - dec_e).abs().max())
            spans[n][i:i + 1].copy_(pl["span"])
            occ = (pl["uid"] >= 0).view(-1, page).any(dim=1)
            active[n][i:i + 1].copy_(occ.sum().view(1).to(torch.int32))
        src = dict(k=st.k_dst, v=st.v_dst, uid=st.unit_id_dst, mod=st.modality_dst,
                   pos=st.pos_dst)
    torch.cuda.synchronize()
    status = int(d_status.item())
    if status != 0:
        raise RuntimeError(f"device status {status}: {ot.status_string(status)}")
    res = {"steps": steps, "page_size": page,
           "max_abs_diff_vs_eager": round(float(diff.max().item()), 6),
           "position_order_max_abs_diff_vs_eager": round(float(diff_pos.max().item()), 6),
           "decode_max_abs_diff_vs_eager": round(float(diff_dec.max().item()), 8),
           "decode_position_order_max_abs_diff_vs_eager": round(float(diff_dec_pos.max().item()),
                                                                8)}
    for n in names:
        ms = lambda a, b: sum(ev[n][i][a].elapsed_time(ev[n][i][b]) for i in range(steps))  # noqa
        sp = spans[n].cpu().numpy()
        ac = active[n].cpu().numpy()
        r = {"maintenance_ms_total": round(ms(0, 1), 3), "mean_span": round(float(sp.mean()), 1),
             "max_span": int(sp.max()), "final_span": int(sp[-1]),
             "mean_active_pages": round(float(ac.mean()), 1)}
        # per-step latency: eager = score + select + compact + attention; native layouts =
        # eviction (+ packing) + placement + attention with tile skipping
        a = 4 if n == "eager" else 0
        per_step = lambda x, y: np.array([ev[n][i][x].elapsed_time(ev[n][i][y])  # noqa: E731
                                          for i in range(steps)])
        pct = lambda arr: {"p50": round(float(np.percentile(arr, 50)), 4),  # noqa: E731
                           "p99": round(float(np.percentile(arr, 99)), 4)}
        lat = per_step(a, 2)
        r["step_ms_p50"] = round(float(np.percentile(lat, 50)), 4)
        r["step_ms_p99"] = round(float(np.percentile(lat, 99)), 4)
        r["step_ms_max"] = round(float(lat.max()), 4)
        if n != "eager":
            # maintenance + attention in position order
            lat_p = per_step(0, 1) + per_step(8, 9)
            r["step_position_order_ms_p50"] = round(float(np.percentile(lat_p, 50)), 4)
            r["step_position_order_ms_p99"] = round(float(np.percentile(lat_p, 99)), 4)
        # the same per call: eager score + select, compaction, attention; native maintenance
        # (eviction, packing, placement), attention with and without tile skipping
        if n == "eager":
            r["per_call_ms"] = {"score_select": pct(per_step(4, 0)),
                                "compact": pct(per_step(0, 1)), "attend": pct(per_step(1, 2)),
                                "decode": pct(per_step(2, 5))}
        else:
            r["per_call_ms"] = {"maintenance": pct(per_step(0, 1)),
                                "attend_skip": pct(per_step(1, 2)),
                                "attend_full_span": pct(per_step(2, 3)),
                                "attend_position_order": pct(per_step(8, 9)),
                                "decode_skip": pct(per_step(5, 6)),
                                "decode_full_span": pct(per_step(6, 7)),
                                "decode_position_order": pct(per_step(9, 10))}
        if n == "eager":
            r["attend_ms_total"] = round(ms(1, 2), 3)
            r["decode_ms_total"] = round(ms(2, 5), 3)
        else:
            r["attend_skip_ms_total"] = round(ms(1, 2), 3)
            r["attend_full_span_ms_total"] = round(ms(2, 3), 3)
            r["attend_position_order_ms_total"] = round(ms(8, 9), 3)
            r["decode_skip_ms_total"] = round(ms(5, 6), 3)
            r["decode_full_span_ms_total"] = round(ms(6, 7), 3)
            r["decode_position_order_ms_total"] = round(ms(9, 10), 3)
            if pools[n]["min_pages"] > 0:
                r["min_pages"] = pools[n]["min_pages"]
                r["moved_rows_total"] = int(pools[n]["moved_sum"].item())
                r["migrations"] = int(pools[n]["migrations"].item())
        res[n] = r
    nat = res["native"]
    for n in names[1:]:
        for mode in ("skip", "full_span"):
            res[n][f"attend_{mode}_reduction_vs_native"] = round(
                1 - res[n][f"attend_{mode}_ms_total"] / nat[f"attend_{mode}_ms_total"], 4)
            res[n][f"decode_{mode}_reduction_vs_native"] = round(
                1 - res[n][f"decode_{mode}_ms_total"] / nat[f"decode_{mode}_ms_total"], 4)
    for n in names[1:]:
        res[n]["attend_position_order_vs_eager"] = round(
            res[n]["attend_position_order_ms_total"] / res["eager"]["attend_ms_total"], 4)
        res[n]["decode_position_order_vs_eager"] = round(
            res[n]["decode_position_order_ms_total"] / res["eager"]["decode_ms_total"], 4)
    for mode in ("skip", "full_span"):
        res["eager"][f"attend_reduction_vs_native_{mode}"] = round(
            1 - res["eager"]["attend_ms_total"] / nat[f"attend_{mode}_ms_total"], 4)
        res["eager"][f"decode_reduction_vs_native_{mode}"] = round(
            1 - res["eager"]["decode_ms_total"] / nat[f"decode_{mode}_ms_total"], 4)
    return res


def device_segments(cfg, lay, dev):
    """All layers of a multi-layer workload drawn on the device with the host generator's
    recipe (N(0,1) keys, values and queries plus per-unit offsets drawn from N(0, 0.5^2), stored
    as bf16), each layer from its own seeded device generator: [n_layers, ...] tensors.  The
    values differ from the host generator's (a different random stream); the shapes, the
    distribution and the tags are the same."""
    H, d, Hq, L, n = cfg.n_kv_heads, cfg.head_dim, cfg.n_q_heads, lay.chunk_len, lay.n_slots
    orig = torch.from_numpy(lay.orig_unit.astype(np.int64)).to(dev)
    cu = torch.from_numpy(lay.chunk_unit.astype(np.int64)).to(dev) + lay.n_orig_units
    nu = lay.n_orig_units + lay.n_chunk_units
    out = {key: [] for key in ("k", "v", "kc", "vc", "q")}
    for layer in range(cfg.n_layers):
        g = torch.Generator(device=dev)
        g.manual_seed(cfg.seed * 1000 + layer)
        off_k = torch.randn(nu, generator=g, device=dev) * 0.5
        off_v = torch.randn(nu, generator=g, device=dev) * 0.5
        rn = lambda *shape: torch.randn(*shape, generator=g, device=dev)  # noqa: E731
        out["k"].append((rn(n, H, d) + off_k[orig][:, None, None]).to(torch.bfloat16))
        out["v"].append((rn(n, H, d) + off_v[orig][:, None, None]).to(torch.bfloat16))
        out["kc"].append((rn(L, H, d) + off_k[cu][:, None, None]).to(torch.bfloat16))
        out["vc"].append((rn(L, H, d) + off_v[cu][:, None, None]).to(torch.bfloat16))
        out["q"].append(rn(L, Hq, d).to(torch.bfloat16))
    return {key: torch.stack(val) for key, val in out.items()}


def other_configs(dev, steps, use_graph=True):
    """The four step calls on the single-layer 8K case (host-generated, the parity tests'
    inputs; input copies rotated so that 512 MB pass between reuses) and on the 36-layer 32K
    case (all 36 layers in one multi-segment call of each entry point, device-generated with the
    same recipe).  Rates are algorithmic bytes or flops summed over segments per call time."""
    from paper_2609_34653_amd.step import StreamStep
    res = {}
    for name in ("single_layer_8k", "hires_32k_36layer"):
        cfg = sg.CONFIG_BY_NAME[name]
        stream = sg.make_stream(cfg)
        lay = stream.layout
        H, d, Hq, L, n_seg = cfg.n_kv_heads, cfg.head_dim, cfg.n_q_heads, lay.chunk_len, \
            cfg.n_layers
        elt = 2
        t = lambda a: torch.from_numpy(np.ascontiguousarray(np.tile(a, n_seg))).to(dev)  # noqa
        tags = dict(uid=t(lay.unit_id), mod=t(lay.modality), pos=t(lay.pos),
                    cm=torch.from_numpy(lay.chunk_modality).to(dev),
                    cu=torch.from_numpy(lay.chunk_unit).to(dev))
        if n_seg == 1:
            seg = stream.segment(0)
            one = dict(k=seg.k_hist.to(dev)[None], v=seg.v_hist.to(dev)[None],
                       kc=seg.k_chunk.to(dev)[None], vc=seg.v_chunk.to(dev)[None],
                       q=seg.q.to(dev)[None])
            per_copy = 2 * one["k"].numel() * elt
            n_copies = max(1, -(-(512 << 20) // per_copy))
            copies = [one] + [{k_: v_.clone() for k_, v_ in one.items()}
                              for _ in range(n_copies - 1)]
            data = "host generator (the parity tests' inputs)"
        else:
            copies = [device_segments(cfg, lay, dev)]
            data = "device generator, same recipe, one seed per layer"
        st = StreamStep(n_seg=n_seg, n_slots=lay.n_slots, n_units=lay.n_units, n_q_heads=Hq,
                        n_kv_heads=H, head_dim=d, chunk_len=L, budget=cfg.budget,
                        recent=cfg.recent, page_size=cfg.page_size, weights=cfg.weights,
                        device=dev)

        def calls(name_):
            def f(i):
                c = copies[i % len(copies)]
                if name_ == "score":
                    st.score(c["k"], tags["uid"], tags["mod"])
                elif name_ == "select":
                    st.select()
                elif name_ == "compact":
                    st.compact(c["k"], c["v"], tags["uid"], tags["mod"], tags["pos"], c["kc"],
                               c["vc"], tags["cm"], tags["cu"])
                else:
                    st.attend(c["q"], cfg.scale)
            return f
        for nm in ("score", "select", "compact", "attend"):
            calls(nm)(0)
        torch.cuda.synchronize()
        status = int(st.d_status.item())
        if status != 0:
            raise RuntimeError(f"{name}: device status {status}")
        kept = [int(x) for x in st.kept_tokens.cpu().tolist()]
        reps = 4 * steps if n_seg == 1 else 4
        tm = {nm: graph_time(calls(nm), reps, dev, use_graph, replays=3)
              for nm in ("score", "select", "compact", "attend")}
        flops = sum(attn_flops(L, kp, Hq, d) for kp in kept)
        sb = score_bytes(lay, H, d, elt, lay.n_units) * n_seg
        cb = sum(compact_bytes(kp, L, H, d, elt, st.cap_dst, lay.n_units) for kp in kept)
        r = {"segments": n_seg, "history_slots": lay.n_slots, "units": lay.n_units,
             "chunk_len": L, "budget": cfg.budget, "kept_tokens": kept if n_seg <= 4 else
             {"min": min(kept), "max": max(kept)}, "data": data,
             "input_copies": len(copies)}
        for nm in ("score", "select", "compact", "attend"):
            e = {"us": round(tm[nm]["us"], 3), "us_p10": round(tm[nm]["us_p10"], 3),
                 "us_p90": round(tm[nm]["us_p90"], 3), "timing": tm[nm]["timing"]}
            sec = tm[nm]["us"] * 1e-6
            if nm == "score":
                e.update(bytes=sb, GBps=round(sb / sec / 1e9, 2),
                         frac_hbm=round(sb / sec / 1e9 / HBM_PEAK_GBPS, 4))
            elif nm == "compact":
                e.update(bytes=cb, GBps=round(cb / sec / 1e9, 2),
                         frac_hbm=round(cb / sec / 1e9 / HBM_PEAK_GBPS, 4))
            elif nm == "attend":
                e.update(flops=flops, TFLOPs=round(flops / sec / 1e12, 2),
                         frac_mfma=round(flops / sec / 1e12 / BF16_PEAK_TFLOPS, 4))
            r[nm] = e
        res[name] = r
        del copies, st
        torch.cuda.empty_cache()
    return res


def cpu_model():
    """The host CPU's model name (first 'model name' line of /proc/cpuinfo), or None."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(cfg, stream, seg, flops):
    """The CPU oracle (exact integers + float64 attention) on one step of the same workload."""
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = len(os.sched_getaffinity(0))
    lay = stream.layout
    bits = lambda x: x.contiguous().view(torch.int16).numpy().view(np.uint16)  # noqa: E731
    k, v = bits(seg.k_hist), bits(seg.v_hist)
    t0 = time.perf_counter()
    sc = oracle.score_units(k, cfg.dtype, lay.unit_id, lay.modality, cfg.weights, lay.n_units)
    t1 = time.perf_counter()
    _, keep, kept = oracle.select_units(sc["wsum"], sc["len"], sc["first"], sc["last"],
                                        sc["flags"], cfg.budget, cfg.recent)
    t2 = time.perf_counter()
    cp = oracle.compact_kv(k, v, lay.unit_id, lay.modality, lay.pos, keep, lay.n_units,
                           bits(seg.k_chunk), bits(seg.v_chunk), lay.chunk_modality,
                           lay.chunk_unit, cfg.budget + lay.chunk_len, cfg.page_size)
    t3 = time.perf_counter()
    oracle.chunk_attention(oracle.to_f64(bits(seg.q), "bf16"), oracle.to_f64(cp["k"], "bf16"),
                           oracle.to_f64(cp["v"], "bf16"), cfg.scale)
    t4 = time.perf_counter()
    step_s = t4 - t0
    res = {"value": round(flops / step_s / 1e12, 5), "unit": "TFLOP/s", "cores": int(threads),
           "kind": "oracle",
           "sample": "one full step of the same workload (score, select, compact, float64 "
                     "attention of all 665 queries x 32 heads)",
           "stage_s": {"score": round(t1 - t0, 3), "select": round(t2 - t1, 3),
                       "compact": round(t3 - t2, 3), "attend": round(t4 - t3, 3)},
           "step_s": round(step_s, 3), "cpu_model": cpu_model()}
    # The same oracle on one thread: score, select and compact as above, attention for the
    # first KV head's group of query heads only (1/H_kv of the flops); the rate is scaled from
    # that group's flops.
    try:
        from threadpoolctl import threadpool_limits
    except Exception:  # pragma: no cover
        return res
    G = cfg.n_q_heads // cfg.n_kv_heads
    with threadpool_limits(limits=1):
        u0 = time.perf_counter()
        sc = oracle.score_units(k, cfg.dtype, lay.unit_id, lay.modality, cfg.weights,
                                lay.n_units)
        _, keep, kept = oracle.select_units(sc["wsum"], sc["len"], sc["first"], sc["last"],
                                            sc["flags"], cfg.budget, cfg.recent)
        cp = oracle.compact_kv(k, v, lay.unit_id, lay.modality, lay.pos, keep, lay.n_units,
                               bits(seg.k_chunk), bits(seg.v_chunk), lay.chunk_modality,
                               lay.chunk_unit, cfg.budget + lay.chunk_len, cfg.page_size)
        u1 = time.perf_counter()
        oracle.chunk_attention(oracle.to_f64(bits(seg.q)[:, :G], "bf16"),
                               oracle.to_f64(cp["k"][:, :1], "bf16"),
                               oracle.to_f64(cp["v"][:, :1], "bf16"), cfg.scale)
        u2 = time.perf_counter()
    one_s = (u1 - u0) + (u2 - u1) * cfg.n_kv_heads
    res["single_thread"] = {
        "value": round(flops / one_s / 1e12, 6), "unit": "TFLOP/s", "cores": 1,
        "sample": f"score + select + compact of the step, then attention of query heads 0..{G - 1} "
                  f"(KV head 0) timed and multiplied by {cfg.n_kv_heads}",
        "stage_s": {"score_select_compact": round(u1 - u0, 3),
                    "attend_one_kv_head": round(u2 - u1, 3)},
        "step_s_estimated": round(one_s, 3)}
    return res


if __name__ == "__main__":
    main()
