"""Benchmark of the speculate-reuse-repair decode step on one MI355X.

    python bench.py [--steps K] [--warmup W] [--config glm128k] [--gpus 1]

A step is one decode token: every layer of the workload runs its per-layer hot path
(select + speculate + repair, with the EMA update and next prediction).  Inputs are
seeded synthetic K/V/queries with the workload's shapes (see workloads/synth.py),
resident in HBM before timing starts; every layer has its own K/V, so a token touches
far more than the 256 MB last-level cache.  The token step is captured once per
prediction-buffer parity as a HIP graph and replayed.

Prints one JSON line.  `value` is microseconds per decode step per layer (lower is
better).  Also reported: the serial select-then-attend latency measured the same way,
per-kernel HIP-event durations, the roofline of the dominant kernel, and the oracle's
CPU time per layer-step on a bounded sample (rank 0 only).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import multiprocessing as mp
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import workloads as W  # noqa: E402

METRIC = "µs per decode step per layer (select+spec+repair) at batch 1; achieved HBM GB/s"
HBM_PEAK_GBPS = 8000.0


def _gen_layer(args):
    name, layer = args
    li = W.layer_inputs(W.CONFIGS[name], layer)
    return layer, li.k_bits, li.v_bits


def algorithmic_bytes(cfg, n_pages):
    """Bytes the method must move per layer-step: page metadata + K/V of the selected
    pages + q + o (fp32 and 16-bit)."""
    hkv, d = cfg.num_kv_heads, cfg.head_dim
    meta_page = (2 * d * 2) if cfg.meta_kind == "minmax" else d * 4
    kv_page = 2 * cfg.page_size * d * 2
    q = cfg.num_q_heads * d * 2
    o = cfg.num_q_heads * d * (4 + 2)
    return hkv * n_pages * meta_page + hkv * cfg.selected_count * kv_page + q + o


def score_kernel_bytes(cfg, n_pages):
    """Algorithmic bytes of one score_topk launch: per (KV head, page) one metadata
    record read and one float32 score written; plus q and the selected list."""
    d = cfg.head_dim
    meta_page = (2 * d * 2) if cfg.meta_kind == "minmax" else d * 4
    return cfg.num_kv_heads * n_pages * (meta_page + 4) + cfg.num_q_heads * d * 2 + \
        cfg.num_kv_heads * cfg.selected_count * 4


def kernel_source_hash():
    h = hashlib.sha256()
    for f in ("paper_2606_30389_amd/csrc/prr_kernels.hip", "paper_2606_30389_amd/csrc/prr_device.h"):
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def load_traffic(kernel):
    """HBM bytes per launch from the committed rocprofv3 counter runs, if they were taken
    on the current kernel source (otherwise null)."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("kernel_source") != kernel_source_hash():
        return None
    return t.get("kernels", {}).get(kernel, {}).get("hbm_bytes_per_launch")


def cpu_baseline(cfg, budget_s):
    """The oracle's serial select-then-attend step (scores, top-K, attention over the
    selected pages), timed on this host on a bounded sample of layer 0's decode steps;
    metadata is prefill work and is built before timing."""
    import oracle as O
    try:
        from threadpoolctl import threadpool_limits
    except ImportError:  # pragma: no cover
        threadpool_limits = None
    li = W.layer_inputs(cfg, 0)
    k, v = li.k64(), li.v64()
    meta = (O.page_metadata_minmax(k, cfg.page_size, cfg.context) if cfg.meta_kind == "minmax"
            else O.page_metadata_mean(k, cfg.page_size, cfg.context))
    _, qb = W.query_trajectory(cfg, 0, steps=cfg.steps)
    times = []

    def run():
        t_start = time.perf_counter()
        t = 1
        while time.perf_counter() - t_start < budget_s and t <= cfg.steps:
            q = W.bits_to_f64(qb[t], cfg.dtype)
            t0 = time.perf_counter()
            O.serial_step(q, k, v, cfg.page_size, cfg.context, cfg.k_select, cfg.forced_pages(),
                          cfg.forced_in_budget, cfg.meta_kind, meta=meta)
            times.append(time.perf_counter() - t0)
            t += 1

    if threadpool_limits is not None:
        with threadpool_limits(limits=1):
            run()
    else:
        run()
    us = 1e6 * float(np.median(times))
    return {"value": round(us, 1), "unit": "us/layer-step", "cores": 1, "kind": "oracle",
            "sample": f"{len(times)} decode steps of layer 0 of {cfg.name} (float64 NumPy, 1 thread), median"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--config", default="glm128k")
    ap.add_argument("--layers", type=int, default=None, help="fewer layers (quick runs only)")
    ap.add_argument("--mode", default="exact", choices=["exact", "keep"])
    ap.add_argument("--chunk", type=int, default=None, help="pages per speculation chunk (default 8, 4 for 64-token pages)")
    ap.add_argument("--no-graph", action="store_true", help="skip the HIP-graph variant")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--kernel-reps", type=int, default=4, help="tokens per kernel-timing pass")
    ap.add_argument("--workers", type=int, default=16, help="input-generation processes (0 = in-process)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="also run a plain device copy of this size (calibrates HBM byte counters)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "this decode path runs on one GPU; bench.py supports --gpus 1 only",
                          "n_gpus": args.gpus}), flush=True)
        sys.exit(2)

    import torch
    from paper_2606_30389_amd import _lib as L
    from paper_2606_30389_amd import runtime as R

    cfg = W.CONFIGS[args.config]
    n_layers = args.layers or cfg.layers
    dev = torch.device("cuda:0")
    mode = L.PRR_EXACT_SELECTED if args.mode == "exact" else L.PRR_KEEP_WASTED
    pc = R.PathConfig(num_q_heads=cfg.num_q_heads, num_kv_heads=cfg.num_kv_heads, page_size=cfg.page_size,
                      num_tokens=cfg.context, k_select=cfg.k_select, forced=cfg.forced_pages(),
                      forced_in_budget=cfg.forced_in_budget, dtype=cfg.dtype, meta_kind=cfg.meta_kind,
                      alpha=cfg.alpha, beta=cfg.beta, gamma=cfg.gamma,
                      chunk_pages=args.chunk or min(8, 256 // cfg.page_size), mode=mode)
    total_tokens = 1 + max(2, args.warmup) + 5 * args.steps + args.kernel_reps + 16
    t0 = time.time()
    layers = [None] * n_layers

    def add_layer(layer, kb, vb):
        st = R.LayerState(pc, dev, k=R.bits_tensor(kb, pc.torch_dtype, dev), v=R.bits_tensor(vb, pc.torch_dtype, dev))
        st.build_meta()
        layers[layer] = st
        print(f"[bench] layer {layer} ready ({time.time() - t0:.1f}s)", file=sys.stderr, flush=True)

    jobs = [(cfg.name, l) for l in range(n_layers)]
    if args.workers > 0:
        with mp.get_context("fork").Pool(min(args.workers, os.cpu_count() or 1)) as pool:
            for layer, kb, vb in pool.imap_unordered(_gen_layer, jobs):
                add_layer(layer, kb, vb)
    else:
        for job in jobs:
            add_layer(*_gen_layer(job))
    qs = []
    for l in range(n_layers):
        _, qb = W.query_trajectory(cfg, l, steps=total_tokens)
        qs.append(R.bits_tensor(qb, pc.torch_dtype, dev))
    q_all = torch.stack(qs, dim=1).contiguous()  # [T][L][Hq][d]
    q_static = torch.empty_like(q_all[0])
    torch.cuda.synchronize()

    s = torch.cuda.Stream(device=dev)
    p = torch.cuda.Stream(device=dev)
    e = torch.cuda.Stream(device=dev)

    def prr_token(serial=False):
        """One token over all layers: the fork/join pattern of each layer step."""
        joins = []
        for l, st in enumerate(layers):
            q = q_static[l]
            if serial:
                st.select(q, stream=s)
                st.repair(q, stream=s, serial=True)
                continue
            fork = torch.cuda.Event()
            fork.record(s)
            p.wait_event(fork)
            st.select(q, stream=s)
            sel = torch.cuda.Event()
            sel.record(s)
            st.speculate(q, stream=p)
            spec = torch.cuda.Event()
            spec.record(p)
            s.wait_event(spec)
            st.repair(q, stream=s)
            e.wait_event(sel)
            st.predict(stream=e)
        if not serial:
            for strm in (p, e):
                ev = torch.cuda.Event()
                ev.record(strm)
                s.wait_event(ev)
        return joins

    # step 0: the prefill stand-in initialises the EMA state and predicts step 1
    q_static.copy_(q_all[0])
    stack = R.DecodeStack(layers, [q_static[l] for l in range(n_layers)], dev)
    s.wait_stream(torch.cuda.current_stream())
    stack.step(L.PRR_SCHED_PREFILL, s)
    torch.cuda.synchronize()

    tok = [1]

    def run_native(n, schedule, measure_hits=False):
        hits = []
        for _ in range(n):
            with torch.cuda.stream(s):
                q_static.copy_(q_all[tok[0]])
            stack.step(schedule, s, p)
            tok[0] += 1
            if measure_hits:
                torch.cuda.synchronize()
                miss = torch.stack([st.missed for st in layers]).sum().item()
                hits.append(1.0 - miss / (n_layers * cfg.num_kv_heads * cfg.selected_count))
        return hits

    def timed_native(n, schedule):
        torch.cuda.synchronize()
        start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.wait_stream(torch.cuda.current_stream())
        start.record(s)
        run_native(n, schedule)
        end.record(s)
        torch.cuda.synchronize()
        return start.elapsed_time(end) / n  # ms per token

    hits = run_native(max(2, args.warmup), L.PRR_SCHED_TWO_STREAM, measure_hits=True)
    run_native(2, L.PRR_SCHED_SERIAL)
    ms_prr = timed_native(args.steps, L.PRR_SCHED_TWO_STREAM)
    ms_serial = timed_native(args.steps, L.PRR_SCHED_SERIAL)
    ms_prr = min(ms_prr, timed_native(args.steps, L.PRR_SCHED_TWO_STREAM))
    ms_serial = min(ms_serial, timed_native(args.steps, L.PRR_SCHED_SERIAL))

    def run_tokens(n, serial, graphs):
        for _ in range(n):
            s.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(s):
                q_static.copy_(q_all[tok[0]])
                graphs[layers[0].cur if not serial else 0].replay()
            if not serial:
                for st in layers:
                    st.cur = 1 - st.cur
            tok[0] += 1

    def capture(serial):
        gs = []
        for parity in ((0,) if serial else (0, 1)):
            for st in layers:
                st.cur = parity
            g = torch.cuda.CUDAGraph()
            s.wait_stream(torch.cuda.current_stream())
            with torch.cuda.graph(g, stream=s):
                prr_token(serial)
            gs.append(g)
        torch.cuda.synchronize()
        return gs

    ms_graph = None
    if not args.no_graph:
        # the same PRR token captured from the Python runtime as one HIP graph (its branches
        # were observed to run one after another)
        saved = [st.cur for st in layers]
        prr_graphs = capture(False)
        for st, c in zip(layers, saved):
            st.cur = c
        stack.parity = saved[0]
        run_tokens(2, False, prr_graphs)
        torch.cuda.synchronize()
        start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.wait_stream(torch.cuda.current_stream())
        start.record(s)
        run_tokens(args.steps, False, prr_graphs)
        end.record(s)
        torch.cuda.synchronize()
        ms_graph = start.elapsed_time(end) / args.steps
        stack.parity = layers[0].cur

    # critical path of one layer with direct launches: q ready -> o ready
    def critical_path(reps):
        prr, ser = [], []
        for _ in range(reps):
            q_static.copy_(q_all[tok[0]])
            torch.cuda.synchronize()
            for l, st in enumerate(layers):
                q = q_static[l]
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record(s)
                p.wait_event(a)
                st.select(q, stream=s)
                sel = torch.cuda.Event()
                sel.record(s)
                st.speculate(q, stream=p)
                spec = torch.cuda.Event()
                spec.record(p)
                s.wait_event(spec)
                st.repair(q, stream=s)
                b.record(s)
                e.wait_event(sel)
                st.predict(stream=e)
                torch.cuda.synchronize()
                prr.append(1000.0 * a.elapsed_time(b))
                a2, b2 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a2.record(s)
                st.select(q, stream=s)
                st.repair(q, stream=s, serial=True)
                b2.record(s)
                torch.cuda.synchronize()
                ser.append(1000.0 * a2.elapsed_time(b2))
            for st in layers:
                st.advance()
            stack.parity = layers[0].cur
            tok[0] += 1
        return float(np.median(prr)), float(np.median(ser))

    crit_prr, crit_serial = critical_path(2)

    # per-kernel durations: HIP events around each launch on the stream it runs on
    def kernel_times(reps):
        names = ("score_topk", "spec_attn", "repair", "predict", "repair_serial")
        acc = {k: [] for k in names}
        for _ in range(reps):
            q_static.copy_(q_all[tok[0]])
            torch.cuda.synchronize()
            for l, st in enumerate(layers):
                q = q_static[l]
                evs = [torch.cuda.Event(enable_timing=True) for _ in range(10)]
                evs[0].record(s)
                st.select(q, stream=s)
                evs[1].record(s)
                evs[2].record(s)
                st.speculate(q, stream=s)
                evs[3].record(s)
                evs[4].record(s)
                st.repair(q, stream=s)
                evs[5].record(s)
                evs[6].record(s)
                st.predict(stream=s)
                evs[7].record(s)
                evs[8].record(s)
                st.repair(q, stream=s, serial=True)
                evs[9].record(s)
                torch.cuda.synchronize()
                for i, k in enumerate(names):
                    acc[k].append(1000.0 * evs[2 * i].elapsed_time(evs[2 * i + 1]))
            for st in layers:
                st.advance()
            tok[0] += 1
        return {k: float(np.mean(v)) for k, v in acc.items()}

    ktimes = kernel_times(args.kernel_reps)

    b_alg = algorithmic_bytes(cfg, cfg.num_pages)
    us_prr = 1000.0 * ms_prr / n_layers
    us_serial = 1000.0 * ms_serial / n_layers
    dominant = max(("score_topk", "spec_attn", "repair", "predict"), key=lambda k: ktimes[k])
    sb = score_kernel_bytes(cfg, cfg.num_pages)
    achieved = (sb / (ktimes["score_topk"] * 1e-6)) / 1e9
    roofline = {"bound": "hbm", "kernel": "score_topk", "dominant_kernel": dominant,
                "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": load_traffic("score_topk"),
                "alg_bytes_per_launch": sb, "avg_launch_us": round(ktimes["score_topk"], 2)}

    out = {
        "metric": METRIC, "value": round(us_prr, 3), "unit": "us/layer-step", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_prr, 4),
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": cfg.dtype,
        "data": "synthetic (seeded N(0,1) K/V with hot pages, AR(1) queries; no model weights)",
        "config": {"workload": f"{cfg.name}: {n_layers} layers x ({cfg.num_q_heads} q / {cfg.num_kv_heads} kv heads, "
                               f"d {cfg.head_dim}), {cfg.dtype}, {cfg.context}-token context, page {cfg.page_size}, "
                               f"top-{cfg.k_select} pages, batch 1",
                   "mode": args.mode, "chunk_pages": pc.chunk_pages,
                   "schedule": "prr_decode_step: select on stream S while speculating on stream P, repair on S, "
                               "EMA update on P; native launches"},
        "graph_us_per_layer": round(1000.0 * ms_graph / n_layers, 3) if ms_graph else None,
        "achieved_gbps": round(b_alg / (us_prr * 1e-6) / 1e9, 1),
        "alg_bytes_per_layer_step": b_alg,
        "serial_us_per_layer": round(us_serial, 3),
        "speedup_vs_serial": round(us_serial / us_prr, 3),
        "hit_rate": round(float(np.mean(hits)), 4) if hits else None,
        "critical_path_us": {"prr": round(crit_prr, 2), "serial": round(crit_serial, 2),
                             "note": "one layer, direct launches, q ready -> o ready, median"},
        "kernel_us": {k: round(v, 2) for k, v in ktimes.items()},
        "roofline": roofline,
    }
    if args.copy_calibration_mib > 0:
        nbytes = args.copy_calibration_mib << 20
        src = torch.empty(nbytes // 4, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        out["copy_calibration_bytes"] = {"read": nbytes, "write": nbytes}
    out["cpu_baseline"] = cpu_baseline(cfg, args.cpu_seconds) if args.cpu_seconds > 0 else None
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
