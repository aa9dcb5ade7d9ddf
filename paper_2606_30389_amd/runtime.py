"""Two-stream decode-step runtime over the C ABI (device memory and streams via torch).

Per layer and decode step t (Fig. 1; Section 4):

    stream S (critical):    score_topk(q_t) -> IS^t, A^t   | repair(A^t, P^t, spec) -> o_t
    stream P (speculation): spec_attn(q_t, P^t)            | predict(IS^t) -> P^{t+1}

spec_attn needs only q_t and P^t (predicted at the end of step t-1), so it runs while
the selection is in flight; repair waits for both; the EMA update and the next
prediction wait for the selection only and are off the critical path.  The serial
baseline is score_topk followed by repair with no prediction, on one stream.

All arithmetic happens in libprr.so; this module only allocates, uploads and orders.
"""
from __future__ import annotations

import ctypes
import dataclasses
from typing import List, Optional, Sequence

import numpy as np
import torch

from . import _lib as L


@dataclasses.dataclass
class PathConfig:
    num_q_heads: int
    num_kv_heads: int
    page_size: int
    num_tokens: int
    k_select: int
    forced: Sequence[int] = ()
    forced_in_budget: bool = True
    dtype: str = "bf16"  # "bf16" | "f16"
    meta_kind: str = "minmax"  # "minmax" | "mean"
    alpha: float = 0.5
    beta: float = 0.5
    gamma: float = 0.0
    p_select: Optional[int] = None  # |P| budget; default = k_select (delta = 1)
    chunk_pages: int = 8
    mode: int = L.PRR_EXACT_SELECTED
    max_pages: Optional[int] = None

    @property
    def group(self):
        return self.num_q_heads // self.num_kv_heads

    @property
    def num_pages(self):
        return (self.num_tokens + self.page_size - 1) // self.page_size

    @property
    def torch_dtype(self):
        return torch.bfloat16 if self.dtype == "bf16" else torch.float16

    def dims(self):
        return L.make_dims(self.num_q_heads, self.num_kv_heads, self.page_size, self.max_pages or self.num_pages,
                           L.PRR_BF16 if self.dtype == "bf16" else L.PRR_F16,
                           L.PRR_META_MEAN if self.meta_kind == "mean" else L.PRR_META_MINMAX)

    def list_cap(self):
        nf = len(self.forced)
        def size(k):
            return min(self.num_pages, max(k, nf) if self.forced_in_budget else k + nf)
        return max(1, size(self.k_select), size(self.p_select if self.p_select is not None else self.k_select))


def bits_tensor(bits: np.ndarray, dtype: torch.dtype, device) -> torch.Tensor:
    """Upload 16-bit storage patterns as a tensor of the given 16-bit dtype."""
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.to(device).view(dtype)


class LayerState:
    """Device memory of one layer: KV cache, metadata, EMA state, lists, partials, outputs."""

    def __init__(self, cfg: PathConfig, device, k=None, v=None, page_table=None):
        self.cfg = cfg
        self.dims = cfg.dims()
        hkv, g, d = cfg.num_kv_heads, cfg.group, 128
        mp = self.dims.max_pages
        dev = device
        self.cap = cfg.list_cap()
        f32 = dict(dtype=torch.float32, device=dev)
        i32 = dict(dtype=torch.int32, device=dev)
        self.k = k if k is not None else torch.zeros(hkv, mp, cfg.page_size, d, dtype=cfg.torch_dtype, device=dev)
        self.v = v if v is not None else torch.zeros_like(self.k)
        self.page_table = page_table
        if cfg.meta_kind == "mean":
            self.meta = torch.zeros(hkv, mp, d, **f32)
        else:
            self.meta = torch.zeros(hkv, mp, 2, d, dtype=cfg.torch_dtype, device=dev)
        self.scores = torch.zeros(hkv, mp, **f32)
        self.level = torch.zeros(hkv, mp, **f32)
        self.trend = torch.zeros(hkv, mp, **f32)
        self.init_bits = torch.zeros(hkv, (mp + 31) // 32, **i32)
        self.sel = torch.zeros(hkv, self.cap, **i32)
        self.sel_count = torch.zeros(hkv, **i32)
        self.pred = [torch.zeros(hkv, self.cap, **i32) for _ in range(2)]
        self.pred_count = [torch.zeros(hkv, **i32) for _ in range(2)]
        _, po, pml, pm = L.prr_spec_state_floats(self.dims, self.cap, cfg.chunk_pages)
        self.part_o = torch.zeros(po, **f32)
        self.part_m = torch.zeros(pml, **f32)
        self.part_l = torch.zeros(pml, **f32)
        self.page_m = torch.zeros(pm, **f32)
        self.out_o32 = torch.zeros(cfg.num_q_heads, d, **f32)
        self.out_o = torch.zeros(cfg.num_q_heads, d, dtype=cfg.torch_dtype, device=dev)
        self.out_m = torch.zeros(cfg.num_q_heads, **f32)
        self.out_l = torch.zeros(cfg.num_q_heads, **f32)
        self.missed = torch.zeros(hkv, **i32)
        self.wasted = torch.zeros(hkv, **i32)
        self.covered = torch.zeros(hkv, **i32)
        self.ws_bytes = L.prr_workspace_size(self.dims, self.cap, cfg.chunk_pages)
        self.workspace = torch.empty(self.ws_bytes // 4 + 64, dtype=torch.int32, device=dev)
        L.prr_workspace_init(self.workspace, self.ws_bytes)
        self.cur = 0  # which predicted-list buffer holds P^t
        self.theta = None  # this layer's (alpha, beta, gamma), host float32 [3], or None (the step's)

    # --------------------------------------------------------------- steps
    def build_meta(self, stream=None, page_begin=0, page_end=None):
        cfg = self.cfg
        L.prr_build_page_meta(self.dims, self.k, self.page_table, cfg.num_tokens, page_begin,
                              cfg.num_pages if page_end is None else page_end, self.meta, stream)

    def select(self, q, stream=None):
        cfg = self.cfg
        L.prr_score_topk(self.dims, q, self.meta, cfg.num_pages, cfg.k_select, cfg.forced, cfg.forced_in_budget,
                         self.scores, self.sel, self.sel_count, self.cap, self.workspace, self.ws_bytes, stream)

    def predict(self, with_scores=True, stream=None):
        """EMA update with this step's scores, then P for the next step (into the other buffer)."""
        cfg = self.cfg
        nxt = 1 - self.cur
        L.prr_predict(self.dims, self.level, self.trend, self.init_bits, self.scores if with_scores else None,
                      cfg.num_pages, cfg.alpha, cfg.beta, cfg.gamma,
                      cfg.k_select if cfg.p_select is None else cfg.p_select, cfg.forced, cfg.forced_in_budget,
                      self.pred[nxt], self.pred_count[nxt], self.cap, stream)

    def advance(self):
        self.cur = 1 - self.cur

    def speculate(self, q, stream=None, pages=None, counts=None):
        cfg = self.cfg
        L.prr_spec_attn(self.dims, q, self.k, self.v, self.page_table, cfg.num_tokens,
                        self.pred[self.cur] if pages is None else pages,
                        self.pred_count[self.cur] if counts is None else counts,
                        self.cap, cfg.chunk_pages, self.part_o, self.part_m, self.part_l, self.page_m, stream)

    def repair(self, q, stream=None, serial=False, mode=None, pages=None, counts=None):
        cfg = self.cfg
        pred = None if serial else (self.pred[self.cur] if pages is None else pages)
        cnt = None if serial else (self.pred_count[self.cur] if counts is None else counts)
        L.prr_repair(self.dims, q, self.k, self.v, self.page_table, cfg.num_tokens, cfg.num_pages, self.sel,
                     self.sel_count, pred, cnt, self.cap, cfg.chunk_pages, self.part_o, self.part_m, self.part_l,
                     self.page_m, cfg.mode if mode is None else mode, self.out_o32, self.out_o, self.out_m,
                     self.out_l, self.missed, self.wasted, self.workspace, self.ws_bytes, stream)


    def io(self, q):
        """This layer's buffers as the C ABI's prr_layer_io (q: the layer's query tensor)."""
        def ptr(t):
            return None if t is None else t.data_ptr()
        y = L.prr_layer_io()
        y.q, y.k_cache, y.v_cache, y.page_table, y.meta = ptr(q), ptr(self.k), ptr(self.v), ptr(self.page_table), ptr(self.meta)
        y.scores, y.ema_level, y.ema_trend, y.ema_init_bits = ptr(self.scores), ptr(self.level), ptr(self.trend), ptr(self.init_bits)
        y.selected, y.selected_count = ptr(self.sel), ptr(self.sel_count)
        y.predicted[0], y.predicted[1] = ptr(self.pred[0]), ptr(self.pred[1])
        y.predicted_count[0], y.predicted_count[1] = ptr(self.pred_count[0]), ptr(self.pred_count[1])
        y.part_o, y.part_m, y.part_l, y.page_m = ptr(self.part_o), ptr(self.part_m), ptr(self.part_l), ptr(self.page_m)
        y.out_o32, y.out_o, y.out_m, y.out_l = ptr(self.out_o32), ptr(self.out_o), ptr(self.out_m), ptr(self.out_l)
        y.missed_count, y.wasted_count = ptr(self.missed), ptr(self.wasted)
        y.covered_count = ptr(self.covered)
        y.workspace, y.ws_bytes = ptr(self.workspace), self.ws_bytes
        y.theta = None if self.theta is None else self.theta.ctypes.data
        return y


# Section 4.2: the calibration grid, alpha in 0.2..0.8 step 0.2, beta in 0.1..0.5 step 0.1,
# gamma in 0..0.75 step 0.25 (80 candidates).
THETA_GRID = [(a, b, c) for a in (0.2, 0.4, 0.6, 0.8) for b in (0.1, 0.2, 0.3, 0.4, 0.5)
              for c in (0.0, 0.25, 0.5, 0.75)]


def pick_delta(lut, context, degree=2):
    """Section 4.4's speculation budget for this context length, decided by the library
    (prr_pick_delta) from the profiled table `lut` (rows with "context", "delta",
    "select_us", "spec_us").  Returns the chosen delta."""
    return L.prr_pick_delta(lut, context, degree)[0]


def pick_delta_step(lut, context, degree=2):
    """The budget among those whose speculation fits the selection window (the test of
    pick_delta, per delta) with the shortest profiled step ("fused_prr_late_us") at this
    context; pick_delta's choice when the context was not profiled or the rows carry no
    step latency.  Returns (delta, step latency or None)."""
    rows = [r for r in lut if r["context"] == context and r.get("fused_prr_late_us") is not None]
    if not rows:
        return pick_delta(lut, context, degree), None
    fits = [r for r in rows if r["delta"] == 1.0 or
            L.prr_pick_delta([x for x in lut if x["delta"] == r["delta"]], context, degree)[0] == r["delta"]]
    best = min(fits, key=lambda r: (r["fused_prr_late_us"], r["delta"]))
    return best["delta"], best["fused_prr_late_us"]


_epoch = [0]


def next_epoch():
    """A process-wide increasing value: the fused schedules need a new one for every call
    on a workspace (the device-side hand-offs of a call are tagged with it)."""
    _epoch[0] += 1
    assert _epoch[0] < GRAPH_EPOCH_BASE
    return _epoch[0]


# Captured fused steps read their epoch from one device word per device, advanced by
# every replay; it counts up from 2^30, above every epoch the host hands out.
GRAPH_EPOCH_BASE = 1 << 30
_device_epoch = {}


def device_epoch(device) -> torch.Tensor:
    dev = torch.device(device)
    key = (dev.type, dev.index if dev.index is not None else torch.cuda.current_device())
    if key not in _device_epoch:
        _device_epoch[key] = torch.full((1,), GRAPH_EPOCH_BASE, dtype=torch.int32, device=dev)
    return _device_epoch[key]


class DecodeStack:
    """A stack of layers whose decode step is launched natively by prr_decode_step:
    the two-stream PRR schedule, the serial select-then-attend schedule, or the step-0
    select + EMA initialisation."""

    def __init__(self, layers: List[LayerState], queries, device):
        self.layers = layers
        self.cfg = layers[0].cfg
        self.dims = layers[0].dims
        cfg = self.cfg
        self.io = (L.prr_layer_io * len(layers))(*[st.io(q) for st, q in zip(layers, queries)])
        self.forced = (ctypes.c_int32 * max(1, len(cfg.forced)))(*cfg.forced)
        p = L.prr_step_params()
        p.num_tokens, p.num_pages, p.k_select = cfg.num_tokens, cfg.num_pages, cfg.k_select
        p.p_select = cfg.k_select if cfg.p_select is None else cfg.p_select
        p.cap, p.chunk_pages, p.mode = layers[0].cap, cfg.chunk_pages, cfg.mode
        p.forced_in_budget, p.n_forced = int(bool(cfg.forced_in_budget)), len(cfg.forced)
        p.forced = ctypes.cast(self.forced, ctypes.POINTER(ctypes.c_int32))
        p.alpha, p.beta, p.gamma = cfg.alpha, cfg.beta, cfg.gamma
        self.params = p
        self.events = L.hip_events(3 * len(layers) + 1)
        # the two-stream schedule's fork/join: the caller's events, or (False) the library's
        # stream-memory words
        self.two_stream_events = True

    def set_layer_theta(self, thetas):
        """Per-layer EMA parameters (Section 4.2 calibrates one per layer): a sequence of
        (alpha, beta, gamma) per layer, or None to use the step's for every layer."""
        for i, st in enumerate(self.layers):
            st.theta = None if thetas is None else np.asarray(thetas[i], dtype=np.float32).copy()
            self.io[i].theta = None if st.theta is None else st.theta.ctypes.data

    def _parity(self):
        parity = self.layers[0].cur
        assert all(st.cur == parity for st in self.layers), "layers disagree on the current prediction buffer"
        return parity

    def _advance(self, schedule, parity):
        if schedule not in (L.PRR_SCHED_SERIAL, L.PRR_SCHED_FUSED_SERIAL):
            for st in self.layers:
                st.cur = 1 - parity

    def step(self, schedule, stream, spec_stream=None):
        """One decode step of every layer; P^t is in each layer's predicted[cur]."""
        parity = self._parity()
        self.params.epoch = next_epoch()
        self.params.epoch_dev = None
        events = self.events if (schedule != L.PRR_SCHED_TWO_STREAM or self.two_stream_events) else None
        L.prr_decode_step(self.dims, self.params, self.io, parity, schedule, stream, spec_stream, events)
        self._advance(schedule, parity)

    def capture(self, schedule, stream, tag=None):
        """Capture one fused decode step of every layer as a HIP graph per parity of the
        prediction buffers: an advance of the device epoch word, then the layers' launches
        (which read it).  The step parameters are those of this moment; `tag` names the
        capture when several are kept for one schedule."""
        assert schedule in (L.PRR_SCHED_FUSED_SERIAL, L.PRR_SCHED_FUSED_PRR), "fused steps only"
        if not hasattr(self, "graphs"):
            self.graphs = {}
        ep = device_epoch(self.layers[0].k.device)
        self.params.epoch = 0
        self.params.epoch_dev = ep.data_ptr()
        for parity in (0, 1):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=stream):
                L.prr_epoch_advance(ep, stream)
                L.prr_decode_step(self.dims, self.params, self.io, parity, schedule, stream, None, self.events)
            self.graphs[(schedule, tag, parity)] = g
        self.params.epoch_dev = None

    def replay(self, schedule, stream, tag=None):
        """One decode step of every layer by replaying the captured graph (see capture)."""
        parity = self._parity()
        with torch.cuda.stream(stream):
            self.graphs[(schedule, tag, parity)].replay()
        self._advance(schedule, parity)


class TwoStream:
    """Fork/join orchestration of one layer step on two HIP streams (default priority)."""

    def __init__(self, device):
        self.s = torch.cuda.Stream(device=device)
        self.p = torch.cuda.Stream(device=device)
        self._events = []

    def _ev(self):
        return torch.cuda.Event()

    def prr_layer(self, st: LayerState, q, mode=None):
        s, p = self.s, self.p
        fork = self._ev()
        fork.record(s)
        p.wait_event(fork)
        st.select(q, stream=s)
        sel = self._ev()
        sel.record(s)
        st.speculate(q, stream=p)
        spec = self._ev()
        spec.record(p)
        s.wait_event(spec)
        st.repair(q, stream=s, mode=mode)
        p.wait_event(sel)
        st.predict(stream=p)
        done = self._ev()
        done.record(p)
        return done

    def serial_layer(self, st: LayerState, q):
        st.select(q, stream=self.s)
        st.repair(q, stream=self.s, serial=True)

    def join(self, events: List[torch.cuda.Event]):
        for e in events:
            self.s.wait_event(e)
