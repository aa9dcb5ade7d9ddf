"""Benchmark of the speculate-reuse-repair decode step on one MI355X.

    python bench.py [--steps K] [--warmup W] [--config glm128k] [--gpus 1]

A step is one decode token: every layer of the workload runs its per-layer hot path
(select + speculate + repair, with the EMA update and next prediction), layer after
layer on one stream.  Inputs are seeded synthetic K/V/queries with the workload's
shapes (see workloads/synth.py), resident in HBM before timing starts; every layer has
its own K/V, so a token touches far more than the 256 MB last-level cache.

Schedules timed (all launched natively by prr_decode_step):
  fused_prr     one launch per layer: select while speculating over P, repair, EMA update
  fused_serial  one launch per layer: select, then attend every page of A
  two_stream    separate kernels, selection and speculation on two streams (event fork/join)
  two_stream_mem  the same, the streams ordered by stream memory writes and waits
  serial        separate kernels on one stream: select, then attend A

Prints one JSON line.  `value` is microseconds per decode step per layer of fused_prr
(lower is better).  Also reported: the other schedules, per-kernel HIP-event durations
of the separate kernels, the roofline of the fused kernel, and the oracle's CPU time per
layer-step on a bounded sample (rank 0 only).
"""
from __future__ import annotations

import argparse
import dataclasses
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


def load_traffic(kernel, config):
    """HBM bytes per launch from the committed rocprofv3 counter runs, if they were taken
    on the current kernel source and this workload (otherwise null)."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    from paper_2606_30389_amd.profile_summary import kernel_source_hash
    if t.get("kernel_source") != kernel_source_hash() or t.get("config") != config:
        return None
    return t.get("kernels", {}).get(kernel, {}).get("hbm_bytes_per_launch")


def host_info():
    """The host the CPU baseline runs on."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        affinity = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        affinity = os.cpu_count()
    blas = None
    try:
        from threadpoolctl import threadpool_info
        blas = [{"api": i.get("internal_api"), "threads": i.get("num_threads")} for i in threadpool_info()]
    except ImportError:  # pragma: no cover
        pass
    return {"cpu_model": model, "cpu_count": os.cpu_count(), "affinity": affinity, "blas": blas}


def cpu_baseline(cfg, budget_s, threads=1):
    """The oracle's serial select-then-attend step (scores, top-K, attention over the
    selected pages), timed on this host on a bounded sample of layer 0's decode steps;
    metadata is prefill work and is built before timing.  `threads`: BLAS / OpenMP threads
    of the numpy oracle (the oracle itself is not changed)."""
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
        i = 0
        while time.perf_counter() - t_start < budget_s:
            q = W.bits_to_f64(qb[1 + i % cfg.steps], cfg.dtype)
            t0 = time.perf_counter()
            O.serial_step(q, k, v, cfg.page_size, cfg.context, cfg.k_select, cfg.forced_pages(),
                          cfg.forced_in_budget, cfg.meta_kind, meta=meta)
            times.append(time.perf_counter() - t0)
            i += 1

    if threadpool_limits is not None:
        with threadpool_limits(limits=threads):
            run()
    else:
        run()
    us = 1e6 * float(np.median(times))
    return {"value": round(us, 1), "unit": "us/layer-step", "cores": threads, "kind": "oracle",
            "sample": f"{len(times)} decode steps of layer 0 of {cfg.name} (float64 NumPy, {threads} BLAS "
                      f"thread(s); the {cfg.steps}-step query trajectory repeats), median"}


def kernel_sweep(args):
    """Section 5.4's kernel comparison shape: 32 query / 8 KV heads, head_dim 128, a
    131072-token fp16 cache, blocks (pages) of 16 to 256 tokens, budgets of 1K to 8K tokens
    (a random sorted set of budget / page pages per KV head).  Times attention over the set
    two ways -- the serial repair call (attend every page, merge: one launch) and the
    speculation kernel alone (partial states per chunk) -- and reports microseconds per
    call and GB/s of selected K/V."""
    import torch
    from paper_2606_30389_amd import runtime as R
    dev = torch.device("cuda:0")
    hq, hkv, d, ctx = 32, 8, 128, 131072
    gen = torch.Generator(device="cpu").manual_seed(2606)
    k = torch.randn(hkv * ctx * d, generator=gen, dtype=torch.float32).to(torch.float16).to(dev)
    v = torch.randn(hkv * ctx * d, generator=gen, dtype=torch.float32).to(torch.float16).to(dev)
    q = torch.randn(hq * d, generator=gen, dtype=torch.float32).to(torch.float16).to(dev)
    s = torch.cuda.Stream(device=dev)
    rows = []

    def timed(fn, n=50):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(s)
        for _ in range(n):
            fn()
        b.record(s)
        torch.cuda.synchronize()
        return 1000.0 * a.elapsed_time(b) / n

    for ps in (16, 32, 64, 128, 256):
        npg = ctx // ps
        for budget in (1024, 2048, 4096, 6144, 8192):
            kk = budget // ps
            sel = np.stack([np.sort(np.random.default_rng(7 + h).choice(npg, kk, replace=False)) for h in range(hkv)])
            best = None
            # the pages per workgroup (chunk) is a launch parameter: every allowed value is
            # timed and the fastest kept (small budgets want more, smaller chunks)
            for chunk in (c for c in (1, 2, 4, 8, 16) if c * ps <= 256 and c <= kk):
                pc = R.PathConfig(num_q_heads=hq, num_kv_heads=hkv, page_size=ps, num_tokens=ctx, k_select=kk,
                                  forced=[], forced_in_budget=True, dtype="f16", meta_kind="minmax", chunk_pages=chunk)
                st = R.LayerState(pc, dev, k=k.view(hkv, npg, ps, d), v=v.view(hkv, npg, ps, d))
                st.sel[:, :kk].copy_(torch.from_numpy(sel.astype(np.int32)))
                st.sel_count.fill_(kk)
                us = timed(lambda: st.repair(q, stream=s, serial=True))
                spec_us = timed(lambda: st.speculate(q, stream=s, pages=st.sel, counts=st.sel_count))
                if best is None:
                    best = dict(chunk_us=chunk, us=us, chunk_spec=chunk, spec_us=spec_us)
                if us < best["us"]:
                    best.update(chunk_us=chunk, us=us)
                if spec_us < best["spec_us"]:
                    best.update(chunk_spec=chunk, spec_us=spec_us)
                del st
            kv_bytes = hkv * budget * d * 2 * 2
            rows.append({"page": ps, "budget_tokens": budget, "us": round(best["us"], 2),
                         "gbps": round(kv_bytes / (best["us"] * 1e-6) / 1e9, 1), "chunk": best["chunk_us"],
                         "spec_us": round(best["spec_us"], 2),
                         "spec_gbps": round(kv_bytes / (best["spec_us"] * 1e-6) / 1e9, 1),
                         "spec_chunk": best["chunk_spec"]})
            print(f"[kernel-sweep] {rows[-1]}", file=sys.stderr, flush=True)
    print(json.dumps({"sweep": "sparse attention over a selected set (Section 5.4 shape)", "table": rows}), flush=True)


LUT_PATH = os.path.join(ROOT, "paper_2606_30389_amd", "delta_lut.json")

# Pages per attending workgroup of the fused step, measured best per page size:
# (speculation schedules, serial schedule).  128 tokens per speculation workgroup either
# way; the serial step prefers 64 tokens at 16-token pages and 128 at 64-token pages.
BEST_CHUNK = {16: (8, 4), 64: (2, 2)}


def best_chunk(page_size, serial=False):
    spec, ser = BEST_CHUNK.get(page_size, (max(1, 128 // page_size), max(1, 64 // page_size)))
    return ser if serial else spec


def delta_sweep(args, cfg):
    """Section 4.4's offline profiling on the fused PRR step (with late speculation): for
    each context length (a prefix of the layers' caches) and budget delta = |P| / |A|, the
    selection window (launch start to the threshold's publication, as the select
    workgroup stamps it) and the speculation latency (launch start to the last
    speculation workgroup holding its pages' states), both from the launch's phase
    timestamps, medians over layers and tokens; plus the step's latency from HIP events.
    Four layers with caches of their own are stepped in turn, so that, as in a model, a
    layer's K/V is not still in the memory-side cache from its previous step."""
    import torch
    from paper_2606_30389_amd import _lib as L
    from paper_2606_30389_amd import runtime as R
    from paper_2606_30389_amd.profile_summary import kernel_source_hash
    dev = torch.device("cuda:0")
    n_lay = 4
    tdt = {"bf16": torch.bfloat16, "f16": torch.float16}[cfg.dtype]
    kv = []
    for layer in range(n_lay):
        li = W.layer_inputs(cfg, layer)
        kv.append((R.bits_tensor(li.k_bits, tdt, dev), R.bits_tensor(li.v_bits, tdt, dev)))
        del li
    n_tok = 24
    _, qb = W.query_trajectory(cfg, 0, steps=8 + 2 * n_tok + 40)
    rows = []
    s = torch.cuda.Stream(device=dev)
    stamps = torch.zeros(n_lay, 16, 1024, dtype=torch.int64, device=dev)
    contexts = [c for c in (4096, 8192, 16384, 32768, 65536, 131072) if c <= cfg.context]
    serial_us = {}

    def make_stack(ctx, **kw):
        npg = ctx // cfg.page_size
        pc = R.PathConfig(num_q_heads=cfg.num_q_heads, num_kv_heads=cfg.num_kv_heads, page_size=cfg.page_size,
                          num_tokens=ctx, k_select=cfg.k_select, forced=cfg.forced_pages(npg),
                          forced_in_budget=cfg.forced_in_budget, dtype=cfg.dtype, meta_kind=cfg.meta_kind,
                          alpha=cfg.alpha, beta=cfg.beta, gamma=cfg.gamma, **kw)
        pc.max_pages = cfg.num_pages
        sts = []
        for k, v in kv:
            st = R.LayerState(pc, dev, k=k, v=v)
            st.build_meta()
            sts.append(st)
        qs = R.bits_tensor(qb, pc.torch_dtype, dev)
        q = qs[0].clone()
        return R.DecodeStack(sts, [q] * n_lay, dev), sts, qs, q

    for ctx in contexts:
        for delta in (1.0, 1.25, 1.5, 2.0):
            npg = ctx // cfg.page_size
            p_sel = int(round(delta * cfg.k_select))
            stack, sts, qs, q = make_stack(ctx, chunk_pages=best_chunk(cfg.page_size), p_select=p_sel)
            st = sts[0]
            stack.params.late_spec = 1
            t = [0]

            def step():
                q.copy_(qs[t[0]])
                stack.step(L.PRR_SCHED_FUSED_PRR if t[0] else L.PRR_SCHED_FUSED_PREFILL, s)
                t[0] += 1

            with torch.cuda.stream(s):
                for _ in range(8):
                    step()
                # roles in grid order: score, select, predict, speculation, late, missed, merge
                H, nsc = cfg.num_kv_heads, -(-npg // 128)
                nspec = -(-st.cap // st.cfg.chunk_pages)
                sel0, spec0 = H * nsc, H * (nsc + 2)
                win, spec, hits = [], [], []
                stack.params.phase_stamps = stamps.data_ptr()
                for _ in range(n_tok):
                    stamps.zero_()
                    step()
                    torch.cuda.synchronize()
                    for a in stamps.cpu().numpy():
                        t0 = a[0][a[0] > 0].min()
                        thr = a[4, sel0:sel0 + H]
                        att = a[13, spec0:spec0 + H * nspec]
                        win.append((thr.max() - t0) / 100.0)
                        spec.append((att[att > 0].max() - t0) / 100.0 if (att > 0).any() else 0.0)
                    hits.append(1.0 - sum(x.missed.sum().item() for x in sts) / (n_lay * H * cfg.selected_count))
                stack.params.phase_stamps = None
                torch.cuda.synchronize()
                a_ev, b_ev = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a_ev.record(s)
                for _ in range(n_tok):
                    step()
                b_ev.record(s)
            torch.cuda.synchronize()
            rows.append({"context": ctx, "delta": delta, "select_us": round(float(np.median(win)), 2),
                         "spec_us": round(float(np.median(spec)), 2),
                         "fused_prr_late_us": round(1000.0 * a_ev.elapsed_time(b_ev) / (n_tok * n_lay), 2),
                         "hit_rate": round(float(np.mean(hits)), 4)})
            print(f"[sweep] {rows[-1]}", file=sys.stderr, flush=True)
            del stack, sts, st
        # the select-then-attend step at this context (no speculation), for comparison
        stack, sts, qs, q = make_stack(ctx, chunk_pages=best_chunk(cfg.page_size, serial=True))
        with torch.cuda.stream(s):
            for i in range(8):
                q.copy_(qs[i])
                stack.step(L.PRR_SCHED_FUSED_SERIAL, s)
            a_ev, b_ev = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a_ev.record(s)
            for i in range(n_tok):
                q.copy_(qs[8 + i])
                stack.step(L.PRR_SCHED_FUSED_SERIAL, s)
            b_ev.record(s)
        torch.cuda.synchronize()
        serial_us[ctx] = round(1000.0 * a_ev.elapsed_time(b_ev) / (n_tok * n_lay), 2)
        print(f"[sweep] context {ctx}: fused serial {serial_us[ctx]} us", file=sys.stderr, flush=True)
        del stack, sts
    pick = {c: R.pick_delta(rows, c) for c in contexts}
    out = {"sweep": "speculation budget (Section 4.4) on the fused PRR step with late speculation",
           "config": cfg.name, "workload": f"{cfg.name} layer 0, context prefixes", "kernel_source": kernel_source_hash(),
           "table": rows, "picked_delta": pick, "fused_serial_us": serial_us}
    if args.write_lut:
        with open(args.write_lut, "w") as f:
            json.dump({k: out[k] for k in ("sweep", "config", "workload", "kernel_source", "table")}, f, indent=1)
            f.write("\n")
    print(json.dumps(out), flush=True)


def auto_delta(cfg, how):
    """delta from the committed profile of this workload at its full context: "rule" is
    Section 4.4's rule (the largest budget whose speculation fits the selection window),
    "auto" the fitting budget with the shortest profiled step.  1 when there is no profile.
    Returns (delta, source, the rule's choice or None)."""
    from paper_2606_30389_amd import runtime as R
    if os.path.exists(LUT_PATH):
        with open(LUT_PATH) as f:
            lut = json.load(f)
        if lut.get("config") == cfg.name and lut.get("table"):
            rule = R.pick_delta(lut["table"], cfg.context)
            if how == "rule":
                return rule, f"Section 4.4 rule over {os.path.basename(LUT_PATH)}", rule
            d, _ = R.pick_delta_step(lut["table"], cfg.context)
            return d, f"fitting budget with the shortest profiled step ({os.path.basename(LUT_PATH)})", rule
    return 1.0, "default (no profile of this workload)", None


def causal_calibration(args, cfg, pc, layers, s, dev, L, R, torch):
    """Section 4.2 on a causal prefill trajectory, per layer, overlapped with the GPU.

    Rows are the last ROWS prefill tokens STRIDE tokens apart (args.calibrate_stride; 1 =
    consecutive tokens, like decode steps; page_size = one block forms per row), each
    scoring only the blocks formed by its position; the scores come
    from the library's selection kernel on the GPU (the prefill stand-in), are copied to
    pinned host memory, and each layer's grid search (prr_calibrate, all host threads)
    starts as soon as that layer's rows are on the host, while the GPU scores the next
    layers.  The search of the last layer cannot overlap with prefill: its time is the
    non-overlapped tail (the appendix "Search and Prediction Cost")."""
    import threading
    rows, stride, nb, ps = args.calibrate, args.calibrate_stride, cfg.num_pages, cfg.page_size
    hkv, n_layers = cfg.num_kv_heads, len(layers)
    pos = [cfg.context - (rows - 1 - r) * stride for r in range(rows)]  # tokens up to and incl. row r
    formed = [min(nb, p // ps) for p in pos]
    # the row at which each block forms (rows: never, within the trajectory)
    born = np.array([next(r for r in range(rows) if formed[r] > b) if b < formed[-1] else rows
                     for b in range(nb)], dtype=np.int32)
    grid = np.asarray(R.THETA_GRID, dtype=np.float32)
    host = torch.zeros((n_layers, hkv, rows, nb), dtype=torch.float32, pin_memory=True)
    dev_scores = torch.zeros((rows, hkv, layers[0].dims.max_pages), dtype=torch.float32, device=dev)
    sel = torch.zeros((hkv, layers[0].cap), dtype=torch.int32, device=dev)
    sel_n = torch.zeros(hkv, dtype=torch.int32, device=dev)
    qs = [R.bits_tensor(W.prefill_trajectory(cfg, l, rows, stride), pc.torch_dtype, dev) for l in range(n_layers)]
    events = [torch.cuda.Event() for _ in range(n_layers)]
    ready, done, gpu_ms = [0.0] * n_layers, [0.0] * n_layers, []
    thetas, objective = [None] * n_layers, [0.0] * n_layers
    nthreads = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)

    failure = []

    def search():
        try:
            for l in range(n_layers):
                events[l].synchronize()
                ready[l] = time.perf_counter()
                traj = host[l].numpy()
                best, obj = L.prr_calibrate(traj, cfg.k_select, grid, p_select=pc.p_select or cfg.k_select,
                                            n_threads=nthreads, form_row=born)
                thetas[l], objective[l] = tuple(float(x) for x in best), float(obj.max())
                done[l] = time.perf_counter()
        except BaseException as e:  # (re-raised by the main thread after the join)
            failure.append(e)

    worker = threading.Thread(target=search)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    worker.start()
    for l, st in enumerate(layers):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(s):
            a.record(s)
            for r in range(rows):
                fc = cfg.forced_pages(formed[r])
                L.prr_score_topk(st.dims, qs[l][r], st.meta, formed[r], cfg.k_select, fc, cfg.forced_in_budget,
                                 dev_scores[r], sel, sel_n, st.cap, st.workspace, st.ws_bytes, s)
            b.record(s)
            host[l].copy_(dev_scores[:, :, :nb].transpose(0, 1), non_blocking=True)
            events[l].record(s)
        gpu_ms.append((a, b))
    events[-1].synchronize()
    t_gpu = time.perf_counter()
    worker.join()
    if failure:
        raise failure[0]
    t_end = time.perf_counter()
    per_layer_gpu = [a.elapsed_time(b) for a, b in gpu_ms]
    search_ms = [1000.0 * (done[l] - max(ready[l], done[l - 1] if l else 0.0)) for l in range(n_layers)]
    hist = {}
    for th in thetas:
        key = ",".join(f"{x:.2f}" for x in th)
        hist[key] = hist.get(key, 0) + 1
    return {
        "rows": rows, "row_stride_tokens": stride, "layers": n_layers, "blocks_forming_in_trajectory": int(nb - formed[0]),
        "host_threads": nthreads, "grid_points": len(grid),
        "search_ms_per_layer": {"median": round(float(np.median(search_ms)), 2), "max": round(max(search_ms), 2)},
        "gpu_prefill_standin_ms_per_layer": round(float(np.median(per_layer_gpu)), 3),
        "non_overlapped_tail_ms": round(search_ms[-1], 2),
        "search_total_ms": round(sum(search_ms), 1),
        "wall_ms_after_gpu_done": round(1000.0 * (t_end - t_gpu), 1),
        "wall_ms": round(1000.0 * (t_end - t0), 1),
        "objective_median": round(float(np.median(objective)), 5),
        "theta_histogram": dict(sorted(hist.items(), key=lambda kv: -kv[1])),
        "_thetas": thetas,
    }


# phase-stamp slots (prr_step_params.phase_stamps) read for each workgroup role
STAMP_SLOTS = {"start": 0, "scores": 1, "candidates_stored": 2, "candidates_gathered": 3, "threshold": 4,
               "missed_count": 5, "spec_state": 6, "late_state": 7, "miss_state": 8, "merge_done": 9,
               "select_done": 10, "predict_done": 11, "end": 12, "attended": 13, "late_list": 14}
ROLE_PHASES = {
    "score": ["scores", "candidates_stored", "end"],
    "select": ["candidates_gathered", "threshold", "missed_count", "miss_state", "select_done", "end"],
    # (predict: "missed_count" / "select_done" mark its middle path / full gather)
    "predict": ["candidates_gathered", "threshold", "missed_count", "select_done", "predict_done", "end"],
    "spec": ["attended", "spec_state", "end"],
    "late": ["late_list", "attended", "late_state", "end"],
    "miss": ["miss_state", "end"],
    "merge": ["merge_done", "end"],
}


def role_ranges(H, n_score, nchunks, group, schedule, late, n_late, n_miss):
    """Workgroup index ranges of each role in a fused launch's grid (role-major: every KV
    head's score workgroups, then every head's select workgroup, ...)."""
    roles = [("score", H * n_score), ("select", H)]
    if schedule != 0:
        roles.append(("predict", H))
    if schedule == 1:
        roles += [("spec", H * nchunks), ("late", H * n_late if late else 0)]
    if schedule != 2:
        roles += [("miss", H * n_miss), ("merge", H * group)]
    out, b = {}, 0
    for name, n in roles:
        if n:
            out[name] = (b, b + n)
        b += n
    return out


def phase_table(args, cfg, layers, stack, stack_serial, cur, run, torch, dev, L, n_layers):
    """Per-role phase times of the fused launches (device clock, 100 MHz), in us from the
    launch's first workgroup start: for each role and phase, the median over launches (tokens
    x layers) of [median over the role's workgroups, latest workgroup], and the share of
    launches in which some workgroup of the role reached the phase."""
    stamps = torch.zeros(n_layers, 16, 1024, dtype=torch.int64, device=dev)
    out = {}
    for label, sched, late, stk in (("fused_prr_late", L.PRR_SCHED_FUSED_PRR, 1, stack),
                                    ("fused_serial", L.PRR_SCHED_FUSED_SERIAL, 0, stack_serial)):
        cur[0] = stk
        stk.params.late_spec = late
        st0 = stk.layers[0]
        nchunks = -(-st0.cap // st0.cfg.chunk_pages)
        n_score = -(-cfg.num_pages // 128)
        schedule = 1 if sched == L.PRR_SCHED_FUSED_PRR else 0
        # the missed-list workgroups per KV head (four take the chunks in turn with late
        # speculation at one page per wave), and the late ones: what the grid holds beyond
        # the other roles
        n_miss = min(nchunks, 4) if schedule == 1 and late and st0.cfg.chunk_pages <= 8 else nchunks
        grid = L.prr_fused_grid(stk.dims, stk.params, sched)
        per = grid // cfg.num_kv_heads
        n_late = per - (n_score + 2 + nchunks + n_miss + cfg.group) if schedule == 1 and late else 0
        ranges = role_ranges(cfg.num_kv_heads, n_score, nchunks, cfg.group, schedule, late, n_late, n_miss)
        acc = {(r, p): [] for r in ranges for p in ROLE_PHASES[r]}
        ends = []
        stk.params.phase_stamps = stamps.data_ptr()
        for _ in range(args.phases):
            stamps.zero_()
            torch.cuda.synchronize()
            run(1, sched)
            torch.cuda.synchronize()
            a = stamps.cpu().numpy()
            for l in range(n_layers):
                st = a[l, 0][a[l, 0] > 0]
                t0 = st.min()
                e = a[l, STAMP_SLOTS["end"]]
                ends.append((e[e > 0].max() - t0) / 100.0)
                for (r, p), lst in acc.items():
                    lo, hi = ranges[r]
                    v = a[l, STAMP_SLOTS[p], lo:hi]
                    v = v[v > 0]
                    if v.size:
                        lst.append(((np.median(v) - t0) / 100.0, (v.max() - t0) / 100.0))
        stk.params.phase_stamps = None
        if args.phases_raw:
            raw = stamps.cpu().numpy()[0]
            t0 = raw[0][raw[0] > 0].min()
            out[label + "_raw_layer0"] = [[int((x - t0) // 10) if x > 0 else -1 for x in raw[k][:1024]]
                                          for k in range(15)]
        tab = {}
        for (r, p), lst in acc.items():
            if lst:
                # [median workgroup, latest workgroup, share of launches in which the phase occurred]
                arr = np.asarray(lst)
                tab.setdefault(r, {})[p] = [round(float(np.median(arr[:, 0])), 2), round(float(np.median(arr[:, 1])), 2),
                                            round(len(lst) / len(ends), 3)]
        tab["launch_end"] = round(float(np.median(ends)), 2)
        tab["workgroups"] = {r: hi - lo for r, (lo, hi) in ranges.items()}
        out[label] = tab
    return out


def late_spec_of(schedule):
    """prr_step_params.late_spec of a schedule label: fused_prr_late* speculate late pages
    (with the read-ahead; *_nora without it)."""
    if not schedule.startswith("fused_prr_late"):
        return 0
    return 2 if "nora" in schedule else 1


def _timed_ms(torch, stream, fn, n):
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(n):
        fn()
    b.record(stream)
    torch.cuda.synchronize()
    return a.elapsed_time(b) / n


def extra_measurements(args, cfg, pc, layers, stack, s, dev, L, R, torch, n_layers):
    """Launch floor of the fused grid, measured HBM peaks, and the metadata build (a
    prefill step, not part of the decode step)."""
    out = {}
    grid = L.prr_fused_grid(stack.dims, stack.params, L.PRR_SCHED_FUSED_PRR)
    stack.params.late_spec = 1
    grid_late = L.prr_fused_grid(stack.dims, stack.params, L.PRR_SCHED_FUSED_PRR)
    stack.params.late_spec = 0
    floor = {"grid": grid_late, "threads": 512}
    floor["direct_us"] = round(1000.0 * _timed_ms(torch, s, lambda: L.prr_empty_launch(grid_late, 512, s), 400), 3)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        for _ in range(n_layers):
            L.prr_empty_launch(grid_late, 512, s)
    with torch.cuda.stream(s):
        floor["graph_us"] = round(1000.0 * _timed_ms(torch, s, g.replay, 20) / n_layers, 3)
    floor["fused_prr_grid_without_late"] = grid
    # a dependency between two streams: a chain of empty one-workgroup kernels on one stream,
    # against the same chain alternating between two streams with a dependency per hop (an
    # event, or a stream memory write and wait); the library enqueues each chain in one call,
    # so the host's enqueue cost stays out of the per-hop time
    p2 = torch.cuda.Stream(device=dev)
    n_hop = 200
    chain = {}
    for name, mode in (("one", L.PRR_CHAIN_ONE_STREAM), ("events", L.PRR_CHAIN_EVENTS),
                       ("memory", L.PRR_CHAIN_STREAM_MEMORY)):
        L.prr_stream_chain(n_hop, mode, s, p2)  # (first use makes the events and words)
        chain[name] = 1000.0 * _timed_ms(torch, s, lambda: L.prr_stream_chain(n_hop, mode, s, p2), 5) / n_hop
    floor["one_stream_chain_us"] = round(chain["one"], 3)
    floor["two_stream_chain_us"] = round(chain["events"], 3)
    floor["cross_stream_dependency_us"] = round(chain["events"] - chain["one"], 3)
    floor["stream_memory_dependency_us"] = round(chain["memory"] - chain["one"], 3)
    out["launch_floor"] = floor
    # HBM: a plain device copy (read + write) and a read-only reduction of 2 GiB
    nbytes = 2 << 30
    src = torch.empty(nbytes // 4, dtype=torch.float32, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    with torch.cuda.stream(s):
        cp_ms = _timed_ms(torch, s, lambda: dst.copy_(src), 10)
        rd_ms = _timed_ms(torch, s, lambda: src.sum(), 10)
        # the library's read-stream kernel (16-byte loads, eight in flight per thread):
        # the best over a few grid sizes
        sink = torch.empty(16384, dtype=torch.int32, device=dev)
        rs = {}
        for grid in (2048, 4096, 8192, 16384):
            rs[grid] = _timed_ms(torch, s, lambda: L.prr_read_stream(src, nbytes, sink, grid, s), 10)
    del src, dst
    torch.cuda.empty_cache()
    best_grid = min(rs, key=rs.get)
    out["hbm_measured"] = {"copy_gbps": round(2 * nbytes / (cp_ms * 1e-3) / 1e9, 1),
                           "torch_sum_read_gbps": round(nbytes / (rd_ms * 1e-3) / 1e9, 1),
                           "read_gbps": round(nbytes / (rs[best_grid] * 1e-3) / 1e9, 1),
                           "read_grid": best_grid,
                           "kind": "2 GiB buffer: torch copy_ (read + write), torch sum (read), prr_read_stream (read)"}
    # page metadata (a1): every layer's K read once, metadata written
    def build_all():
        for st in layers:
            st.build_meta(stream=s)
    meta_ms = _timed_ms(torch, s, build_all, 3) / n_layers
    kv_bytes = cfg.num_kv_heads * cfg.num_pages * cfg.page_size * cfg.head_dim * 2
    meta_bytes = cfg.num_kv_heads * cfg.num_pages * ((2 * cfg.head_dim * 2) if cfg.meta_kind == "minmax" else cfg.head_dim * 4)
    out["metadata_build"] = {"us_per_layer": round(1000.0 * meta_ms, 2), "bytes_per_layer": kv_bytes + meta_bytes,
                             "gbps": round((kv_bytes + meta_bytes) / (meta_ms * 1e-3) / 1e9, 1)}
    return out


def other_workload(args, name, L, R, torch, dev, pool):
    """The fused PRR step with late speculation and the fused serial step on another
    workload: microseconds per layer-step and per token."""
    cfg = W.CONFIGS[name]
    pc = R.PathConfig(num_q_heads=cfg.num_q_heads, num_kv_heads=cfg.num_kv_heads, page_size=cfg.page_size,
                      num_tokens=cfg.context, k_select=cfg.k_select, forced=cfg.forced_pages(),
                      forced_in_budget=cfg.forced_in_budget, dtype=cfg.dtype, meta_kind=cfg.meta_kind,
                      alpha=cfg.alpha, beta=cfg.beta, gamma=cfg.gamma, chunk_pages=best_chunk(cfg.page_size))
    layers = [None] * cfg.layers
    t0 = time.time()
    jobs = [(name, l) for l in range(cfg.layers)]
    for layer, kb, vb in (pool.imap_unordered(_gen_layer, jobs) if pool is not None else map(_gen_layer, jobs)):
        st = R.LayerState(pc, dev, k=R.bits_tensor(kb, pc.torch_dtype, dev), v=R.bits_tensor(vb, pc.torch_dtype, dev))
        st.build_meta()
        layers[layer] = st
    print(f"[bench] {name}: {cfg.layers} layers ready ({time.time() - t0:.1f}s)", file=sys.stderr, flush=True)
    steps = max(args.steps // 2, 8)
    qs = torch.stack([R.bits_tensor(W.query_trajectory(cfg, l, steps=2 * steps + 16)[1], pc.torch_dtype, dev)
                      for l in range(cfg.layers)], dim=1).contiguous()
    q_static = torch.empty_like(qs[0])
    stack = R.DecodeStack(layers, [q_static[l] for l in range(cfg.layers)], dev)
    # the serial step at its own best chunk, on layer states that share the K/V and metadata
    pc_s = dataclasses.replace(pc, chunk_pages=best_chunk(cfg.page_size, serial=True))
    layers_s = []
    for st in layers:
        st2 = R.LayerState(pc_s, dev, k=st.k, v=st.v, page_table=st.page_table)
        st2.meta.copy_(st.meta)
        layers_s.append(st2)
    stack_serial = R.DecodeStack(layers_s, [q_static[l] for l in range(cfg.layers)], dev)
    s = torch.cuda.Stream(device=dev)
    tok = [0]
    cur = [stack]

    def step(schedule):
        with torch.cuda.stream(s):
            q_static.copy_(qs[tok[0]])
        cur[0].step(schedule, s)
        tok[0] += 1

    s.wait_stream(torch.cuda.current_stream())
    step(L.PRR_SCHED_FUSED_PREFILL)
    res = {"layers": cfg.layers, "chunk_pages": pc.chunk_pages, "serial_chunk_pages": pc_s.chunk_pages}
    for label, sched, late in (("fused_prr_late", L.PRR_SCHED_FUSED_PRR, 1), ("fused_serial", L.PRR_SCHED_FUSED_SERIAL, 0)):
        cur[0] = stack_serial if sched == L.PRR_SCHED_FUSED_SERIAL else stack
        cur[0].params.late_spec = late
        for _ in range(4):
            step(sched)
        ms = _timed_ms(torch, s, lambda: step(sched), steps)
        res[label] = {"us_per_layer": round(1000.0 * ms / cfg.layers, 3), "us_per_token": round(1000.0 * ms, 1)}
        flags = [int(st.workspace[:1].cpu()[0]) for st in cur[0].layers]
        if any(flags):
            res[label]["error_flags"] = flags
    b_alg = algorithmic_bytes(cfg, cfg.num_pages)
    res["alg_bytes_per_layer_step"] = b_alg
    res["roofline_frac"] = round(b_alg / (res["fused_prr_late"]["us_per_layer"] * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4)
    res["speedup_vs_serial"] = round(res["fused_serial"]["us_per_layer"] / res["fused_prr_late"]["us_per_layer"], 3)
    del stack, stack_serial, layers, layers_s
    torch.cuda.empty_cache()
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--config", default="glm128k")
    ap.add_argument("--layers", type=int, default=None, help="fewer layers (quick runs only)")
    ap.add_argument("--mode", default="exact", choices=["exact", "keep", "recompute"])
    ap.add_argument("--theta", default=None, help="EMA alpha,beta,gamma (default: the workload's)")
    ap.add_argument("--delta-sweep", action="store_true",
                    help="only the offline speculation-budget sweep (Section 4.4): selection and speculation "
                         "latency per context length and delta, and the fused PRR step; prints the table")
    ap.add_argument("--write-lut", default=None, metavar="PATH", help="with --delta-sweep: also write the table as JSON")
    ap.add_argument("--kernel-sweep", action="store_true",
                    help="only the sparse-attention kernel sweep (the shape of Section 5.4's kernel table: 32 q / 8 kv "
                         "heads, d 128, 128K context, pages of 16-256 tokens, budget 1K-8K tokens): microseconds and GB/s")
    ap.add_argument("--calibrate", type=int, default=64, metavar="ROWS",
                    help="calibrate theta per layer (Section 4.2) on a causal prefill trajectory of ROWS rows, "
                         "overlapped with the GPU; then compare hit rate and step time with the default theta "
                         "(0 = skip)")
    ap.add_argument("--calibrate-stride", type=int, default=1, metavar="TOKENS",
                    help="tokens between the calibration rows (1: consecutive, as decode steps are)")
    ap.add_argument("--ablation", action="store_true",
                    help="also time the ablation stages S1 (reuse the previous top-K, recompute on a miss), "
                         "S2 (reuse + repair) and S3 (EMA + repair) with the fused PRR schedule")
    ap.add_argument("--no-extras", dest="extras", action="store_false",
                    help="skip the launch floor, HBM peak, metadata build and other-workload measurements")
    ap.add_argument("--other-workloads", default="llama64k,infllm128k",
                    help="workloads whose per-layer and per-token latency are also measured (comma list, '' = none)")
    ap.add_argument("--phases", type=int, default=0, metavar="TOKENS",
                    help="also record the fused launches' phase timestamps over TOKENS tokens (medians, us from start)")
    ap.add_argument("--phases-raw", action="store_true", help=argparse.SUPPRESS)
    ap.add_argument("--chunk", type=int, default=None, help="pages per speculation chunk (default 8, 4 for 64-token pages)")
    ap.add_argument("--delta", default="auto",
                    help="|P| / |A| (speculation budget); 'rule': Section 4.4's rule over the profiled table; "
                         "'auto': of the budgets that rule allows, the one with the shortest profiled step")
    ap.add_argument("--schedules", default="fused_prr,fused_prr_late,fused_prr_late_nora,fused_serial,fused_prr_late_graph,"
                                           "two_stream,two_stream_mem,serial")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--kernel-reps", type=int, default=2, help="batches of 20 back-to-back calls per separate kernel (kernel_us)")
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
    if args.delta_sweep:
        delta_sweep(args, cfg)
        return
    if args.kernel_sweep:
        kernel_sweep(args)
        return
    n_layers = args.layers or cfg.layers
    dev = torch.device("cuda:0")
    mode = {"exact": L.PRR_EXACT_SELECTED, "keep": L.PRR_KEEP_WASTED, "recompute": L.PRR_RECOMPUTE_ON_MISS}[args.mode]
    theta = tuple(float(x) for x in args.theta.split(",")) if args.theta else (cfg.alpha, cfg.beta, cfg.gamma)
    if args.delta in ("auto", "rule"):
        delta, delta_source, delta_rule = auto_delta(cfg, args.delta)
    else:
        delta, delta_source, delta_rule = float(args.delta), "--delta", None
    p_select = int(round(delta * cfg.k_select))
    pc = R.PathConfig(num_q_heads=cfg.num_q_heads, num_kv_heads=cfg.num_kv_heads, page_size=cfg.page_size,
                      num_tokens=cfg.context, k_select=cfg.k_select, forced=cfg.forced_pages(),
                      forced_in_budget=cfg.forced_in_budget, dtype=cfg.dtype, meta_kind=cfg.meta_kind,
                      alpha=theta[0], beta=theta[1], gamma=theta[2],
                      chunk_pages=args.chunk or best_chunk(cfg.page_size), mode=mode, p_select=p_select)
    schedules = [x for x in args.schedules.split(",") if x]
    sched_id = {"fused_prr": L.PRR_SCHED_FUSED_PRR, "fused_prr_late": L.PRR_SCHED_FUSED_PRR,
                "fused_prr_late_nora": L.PRR_SCHED_FUSED_PRR,
                "fused_serial": L.PRR_SCHED_FUSED_SERIAL, "two_stream": L.PRR_SCHED_TWO_STREAM,
                "two_stream_mem": L.PRR_SCHED_TWO_STREAM,
                "serial": L.PRR_SCHED_SERIAL, "fused_prr_late_graph": L.PRR_SCHED_FUSED_PRR}
    n_abl = (3 if args.ablation else 0) + (2 if args.calibrate > 1 else 0)
    total_tokens = 2 + max(2, args.warmup) + 2 * (len(schedules) + n_abl) * (args.steps + 2) + \
        n_abl * (1 + max(2, args.warmup)) + args.kernel_reps + 2 * args.phases + max(2, args.warmup) + 8
    t0 = time.time()
    layers = [None] * n_layers

    def add_layer(layer, kb, vb):
        st = R.LayerState(pc, dev, k=R.bits_tensor(kb, pc.torch_dtype, dev), v=R.bits_tensor(vb, pc.torch_dtype, dev))
        st.build_meta()
        layers[layer] = st
        print(f"[bench] layer {layer} ready ({time.time() - t0:.1f}s)", file=sys.stderr, flush=True)

    jobs = [(cfg.name, l) for l in range(n_layers)]
    # input generators are forked before anything initialises the GPU, and kept for the
    # other workloads measured at the end
    pool = mp.get_context("fork").Pool(min(args.workers, os.cpu_count() or 1)) if args.workers > 0 else None
    if pool is not None:
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
    stack = R.DecodeStack(layers, [q_static[l] for l in range(n_layers)], dev)
    # The serial baseline runs at its own best chunk (4 pages: twice the attending
    # workgroups, measured faster for it; speculation is fastest at 8), on layer states of
    # its own that share the K/V cache and metadata.
    serial_chunk = pc.chunk_pages
    stack_serial = stack
    if "fused_serial" in args.schedules.split(",") and args.chunk is None:
        serial_chunk = best_chunk(cfg.page_size, serial=True)
        if serial_chunk != pc.chunk_pages:
            pc_s = dataclasses.replace(pc, chunk_pages=serial_chunk)
            layers_s = []
            for st in layers:
                st2 = R.LayerState(pc_s, dev, k=st.k, v=st.v, page_table=st.page_table)
                st2.meta.copy_(st.meta)
                layers_s.append(st2)
            stack_serial = R.DecodeStack(layers_s, [q_static[l] for l in range(n_layers)], dev)
    cur = [stack]
    tok = [0]

    def run(n, schedule, measure_hits=False, tag=None):
        hits = []
        for _ in range(n):
            with torch.cuda.stream(s):
                q_static.copy_(q_all[tok[0]])
            if tag is None:
                cur[0].step(schedule, s, p)
            else:
                cur[0].replay(schedule, s, tag)
            tok[0] += 1
            if measure_hits:
                torch.cuda.synchronize()
                miss = torch.stack([st.missed for st in layers]).sum().item()
                hits.append(1.0 - miss / (n_layers * cfg.num_kv_heads * cfg.selected_count))
        return hits

    def timed(n, schedule, tag=None):
        torch.cuda.synchronize()
        start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.wait_stream(torch.cuda.current_stream())
        start.record(s)
        run(n, schedule, tag=tag)
        end.record(s)
        torch.cuda.synchronize()
        return start.elapsed_time(end) / n  # ms per token

    # step 0: the prefill stand-in selects and initialises the EMA state (predicts step 1)
    s.wait_stream(torch.cuda.current_stream())
    run(1, L.PRR_SCHED_FUSED_PREFILL)
    torch.cuda.synchronize()
    hits = run(max(2, args.warmup), L.PRR_SCHED_FUSED_PRR, measure_hits=True)
    # how much of A the headline schedule attends before the threshold is known: P and the
    # late pages (measured over warm-up tokens with late speculation)
    coverage = []
    stack.params.late_spec = next((late_spec_of(x) for x in schedules if late_spec_of(x)), 1)
    for _ in range(max(2, args.warmup)):
        run(1, L.PRR_SCHED_FUSED_PRR)
        torch.cuda.synchronize()
        miss = torch.stack([st.missed for st in layers]).sum().item()
        cov = torch.stack([st.covered for st in layers]).sum().item()
        coverage.append(1.0 - (miss - cov) / (n_layers * cfg.num_kv_heads * cfg.selected_count))
    stack.params.late_spec = 0
    ms = {}
    for name in schedules:  # warm each schedule, then two timed passes (the better one counts)
        cur[0] = stack_serial if name == "fused_serial" else stack
        stack.params.late_spec = late_spec_of(name)
        stack.two_stream_events = name != "two_stream_mem"
        run(2, sched_id[name])
        # *_graph: the token's launches are captured as HIP graphs (one per parity of the
        # prediction buffers) and replayed; otherwise launched directly
        tag = None
        if name.endswith("_graph"):
            torch.cuda.synchronize()
            stack.capture(sched_id[name], s, tag=name)
            tag = name
            run(2, sched_id[name], tag=tag)
        ms[name] = min(timed(args.steps, sched_id[name], tag), timed(args.steps, sched_id[name], tag))
    cur[0] = stack
    stack.params.late_spec = 0
    ablation = None
    if args.ablation:
        # Section 5.3: S1 reuses the previous step's top-K (theta = (1, .5, 0)) and
        # recomputes attention over A on any miss; S2 repairs instead; S3 is the EMA
        # predictor with repair.  Every stage restarts from a fresh prefill.
        ablation = {}
        stages = {"S1": ((1.0, 0.5, 0.0), L.PRR_RECOMPUTE_ON_MISS), "S2": ((1.0, 0.5, 0.0), L.PRR_EXACT_SELECTED),
                  "S3": ((cfg.alpha, cfg.beta, cfg.gamma), L.PRR_EXACT_SELECTED)}
        saved = (stack.params.alpha, stack.params.beta, stack.params.gamma, stack.params.mode)
        for name, (th, md) in stages.items():
            stack.params.alpha, stack.params.beta, stack.params.gamma = th
            stack.params.mode = md
            for st in layers:
                st.init_bits.zero_()
            torch.cuda.synchronize()
            run(1, L.PRR_SCHED_FUSED_PREFILL)
            h = run(max(2, args.warmup), L.PRR_SCHED_FUSED_PRR, measure_hits=True)
            t_ms = min(timed(args.steps, L.PRR_SCHED_FUSED_PRR), timed(args.steps, L.PRR_SCHED_FUSED_PRR))
            ablation[name] = {"theta": list(th), "mode": {0: "repair", 2: "recompute on miss"}[md],
                              "us_per_layer": round(1000.0 * t_ms / n_layers, 3),
                              "hit_rate": round(float(np.mean(h)), 4)}
        stack.params.alpha, stack.params.beta, stack.params.gamma, stack.params.mode = saved
        for st in layers:
            st.init_bits.zero_()
        run(1, L.PRR_SCHED_FUSED_PREFILL)
    calibration = None
    if args.calibrate > 1:
        calibration = causal_calibration(args, cfg, pc, layers, s, dev, L, R, torch)
        thetas = calibration.pop("_thetas")
        default_theta = (stack.params.alpha, stack.params.beta, stack.params.gamma)
        for name, th in (("default", None), ("calibrated", thetas)):
            stack.set_layer_theta(th)
            for st in layers:
                st.init_bits.zero_()
            torch.cuda.synchronize()
            run(1, L.PRR_SCHED_FUSED_PREFILL)
            h = run(max(4, args.warmup), L.PRR_SCHED_FUSED_PRR, measure_hits=True)
            calibration[f"hit_rate_{name}"] = round(float(np.mean(h)), 4)
            stack.params.late_spec = 1
            calibration[f"us_per_layer_{name}"] = round(
                1000.0 * timed(args.steps, L.PRR_SCHED_FUSED_PRR) / n_layers, 3)
            stack.params.late_spec = 0
        calibration["default_theta"] = [round(float(x), 3) for x in default_theta]
        stack.set_layer_theta(None)
        for st in layers:
            st.init_bits.zero_()
        run(1, L.PRR_SCHED_FUSED_PREFILL)
    phases = None
    if args.phases > 0:
        phases = phase_table(args, cfg, layers, stack, stack_serial, cur, run, torch, dev, L, n_layers)
        cur[0] = stack
        stack.params.late_spec = 0
    flags = [int(st.workspace[:1].cpu()[0]) for st in layers]
    if any(flags):
        print(json.dumps({"error": f"device error flags {flags}"}), flush=True)
        sys.exit(3)

    # per-call time of each separate kernel: back-to-back calls on one stream between two HIP
    # events (an event pair around a single launch adds several microseconds of its own), on
    # layer 0 after one full separate-kernel step of the current token
    def kernel_times(reps):
        n = 20 * reps
        st, q = layers[0], q_static[0]
        q_static.copy_(q_all[tok[0]])
        torch.cuda.synchronize()
        st.select(q, stream=s)
        st.speculate(q, stream=s)
        st.repair(q, stream=s)
        calls = {"score_topk": lambda: st.select(q, stream=s), "spec_attn": lambda: st.speculate(q, stream=s),
                 "repair": lambda: st.repair(q, stream=s), "predict": lambda: st.predict(stream=s),
                 "repair_serial": lambda: st.repair(q, stream=s, serial=True)}
        out = {}
        for name, fn in calls.items():
            fn()
            a_ev, b_ev = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a_ev.record(s)
            for _ in range(n):
                fn()
            b_ev.record(s)
            torch.cuda.synchronize()
            out[name] = 1000.0 * a_ev.elapsed_time(b_ev) / n
        return out

    ktimes = kernel_times(args.kernel_reps) if args.kernel_reps > 0 else {}

    b_alg = algorithmic_bytes(cfg, cfg.num_pages)
    us = {k: 1000.0 * v / n_layers for k, v in ms.items()}
    main_sched = next((k for k in ("fused_prr_late", "fused_prr") if k in us), schedules[0])
    us_prr = us[main_sched]
    # the fused PRR step is one kernel per layer: its average launch duration is the
    # timed region divided by the launches in it
    achieved = b_alg / (us_prr * 1e-6) / 1e9
    roofline = {"bound": "hbm", "kernel": f"fused_step_kernel ({main_sched})", "achieved": round(achieved, 1),
                "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                "traffic": load_traffic(main_sched, cfg.name), "alg_bytes_per_launch": b_alg,
                "traffic_over_alg": None,
                "avg_launch_us": round(us_prr, 3)}
    if roofline["traffic"]:
        roofline["traffic_over_alg"] = round(roofline["traffic"] / b_alg, 3)
    best_serial = min(us[k] for k in ("fused_serial", "serial") if k in us) if any(
        k in us for k in ("fused_serial", "serial")) else None
    out = {
        "metric": METRIC, "value": round(us_prr, 3), "unit": "us/layer-step", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms[main_sched], 4),
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": cfg.dtype,
        "data": "synthetic (seeded N(0,1) K/V with hot pages, AR(1) queries; no model weights)",
        "config": {"workload": f"{cfg.name}: {n_layers} layers x ({cfg.num_q_heads} q / {cfg.num_kv_heads} kv heads, "
                               f"d {cfg.head_dim}), {cfg.dtype}, {cfg.context}-token context, page {cfg.page_size}, "
                               f"top-{cfg.k_select} pages, batch 1",
                   "mode": args.mode, "chunk_pages": pc.chunk_pages, "serial_chunk_pages": serial_chunk, "p_select": p_select, "delta": delta,
                   "delta_source": delta_source, "delta_rule": delta_rule, "theta": list(theta),
                   "schedule": main_sched},
        "us_per_layer": {k: round(v, 3) for k, v in us.items()},
        "achieved_gbps": round(achieved, 1),
        "alg_bytes_per_layer_step": b_alg,
        "serial_us_per_layer": round(best_serial, 3) if best_serial else None,
        "speedup_vs_serial": round(best_serial / us_prr, 3) if best_serial else None,
        "hit_rate": round(float(np.mean(hits)), 4) if hits else None,
        "coverage_before_threshold": round(float(np.mean(coverage)), 4) if coverage else None,
        "kernel_us": {k: round(v, 2) for k, v in ktimes.items()},
        "ablation": ablation,
        "calibration": calibration,
        "phases_us": phases,
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
    if args.extras:
        out.update(extra_measurements(args, cfg, pc, layers, stack, s, dev, L, R, torch, n_layers))
        # the same achieved rate against the read rate this chip reaches in practice
        roofline["measured_read_peak"] = out["hbm_measured"]["read_gbps"]
        roofline["frac_of_measured_read"] = round(achieved / out["hbm_measured"]["read_gbps"], 4)
        if args.other_workloads:
            del stack, stack_serial, cur
            layers.clear()
            torch.cuda.empty_cache()
            out["other_workloads"] = {name: other_workload(args, name, L, R, torch, dev, pool)
                                      for name in args.other_workloads.split(",") if name}
    if pool is not None:
        pool.close()
        pool.join()
    if args.cpu_seconds > 0:
        out["host"] = host_info()
        out["cpu_baseline"] = cpu_baseline(cfg, args.cpu_seconds, threads=out["host"]["affinity"] or 1)
        out["cpu_baseline_1core"] = cpu_baseline(cfg, args.cpu_seconds, threads=1)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
