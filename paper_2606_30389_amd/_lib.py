"""ctypes binding of libprr.so: the C ABI of include/prr.h with the same names.

Argument marshalling only: every step of the decode path runs in the HIP kernels of
the shared library.  Pointer arguments accept a torch tensor (its data_ptr), a plain
integer address, or None (NULL).  Every call raises PrrError when the library returns
a status other than PRR_OK.  Importing this module fails loudly when the library has
not been built.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libprr.so")

PRR_OK = 0
PRR_ERR_INVALID_ARG = 1
PRR_ERR_UNSUPPORTED = 2
PRR_ERR_WORKSPACE = 3
PRR_ERR_HIP = 4
PRR_F16 = 0
PRR_BF16 = 1
PRR_META_MINMAX = 0
PRR_META_MEAN = 1
PRR_EXACT_SELECTED = 0
PRR_KEEP_WASTED = 1
PRR_RECOMPUTE_ON_MISS = 2
PRR_MAX_PAGES = 16384
PRR_MAX_CAP = 1024
PRR_MAX_FORCED = 64
PRR_STATIC_MAX_KV_HEADS = 256

PRR_SCHED_SERIAL = 0
PRR_SCHED_TWO_STREAM = 1
PRR_SCHED_PREFILL = 2
PRR_SCHED_FUSED_SERIAL = 3
PRR_SCHED_FUSED_PRR = 4
PRR_SCHED_FUSED_PREFILL = 5

# every function declared in include/prr.h
EXPORTED = (
    "prr_status_string", "prr_last_error", "prr_workspace_size", "prr_workspace_init",
    "prr_spec_state_floats", "prr_build_page_meta", "prr_score_topk", "prr_predict",
    "prr_spec_attn", "prr_repair", "prr_merge_states", "prr_decode_step", "prr_calibrate",
    "prr_epoch_advance", "prr_pick_delta", "prr_score_topk_static", "prr_empty_launch", "prr_fused_grid",
    "prr_read_stream", "prr_stream_chain",
)


class PrrError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{status_string(status)}: {message}")
        self.status = status


class prr_dims(ctypes.Structure):
    _fields_ = [(name, ctypes.c_int32) for name in
                ("num_q_heads", "num_kv_heads", "head_dim", "page_size", "max_pages", "dtype", "meta_kind")]


class prr_layer_io(ctypes.Structure):
    _fields_ = [
        ("q", ctypes.c_void_p), ("k_cache", ctypes.c_void_p), ("v_cache", ctypes.c_void_p),
        ("page_table", ctypes.c_void_p), ("meta", ctypes.c_void_p), ("scores", ctypes.c_void_p),
        ("ema_level", ctypes.c_void_p), ("ema_trend", ctypes.c_void_p), ("ema_init_bits", ctypes.c_void_p),
        ("selected", ctypes.c_void_p), ("selected_count", ctypes.c_void_p),
        ("predicted", ctypes.c_void_p * 2), ("predicted_count", ctypes.c_void_p * 2),
        ("part_o", ctypes.c_void_p), ("part_m", ctypes.c_void_p), ("part_l", ctypes.c_void_p),
        ("page_m", ctypes.c_void_p), ("out_o32", ctypes.c_void_p), ("out_o", ctypes.c_void_p),
        ("out_m", ctypes.c_void_p), ("out_l", ctypes.c_void_p), ("missed_count", ctypes.c_void_p),
        ("wasted_count", ctypes.c_void_p), ("workspace", ctypes.c_void_p), ("ws_bytes", ctypes.c_size_t),
        ("covered_count", ctypes.c_void_p),
        ("theta", ctypes.c_void_p),
    ]


class prr_step_params(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("num_tokens", "num_pages", "k_select", "p_select", "cap",
                                               "chunk_pages", "mode", "forced_in_budget", "n_forced")] + [
        ("forced", ctypes.POINTER(ctypes.c_int32)), ("alpha", ctypes.c_float), ("beta", ctypes.c_float),
        ("gamma", ctypes.c_float), ("epoch", ctypes.c_uint32), ("epoch_dev", ctypes.c_void_p),
        ("late_spec", ctypes.c_int32), ("phase_stamps", ctypes.c_void_p)]


if not os.path.exists(LIB_PATH):
    raise ImportError(f"libprr.so is not built ({LIB_PATH}); run __graft_entry__.build() first")
_lib = ctypes.CDLL(LIB_PATH)

_P = ctypes.c_void_p
_I = ctypes.c_int32
_F = ctypes.c_float
_S = ctypes.c_size_t
_DIMS = ctypes.POINTER(prr_dims)

_SIGS = {
    "prr_status_string": (ctypes.c_char_p, [_I]),
    "prr_last_error": (ctypes.c_char_p, []),
    "prr_workspace_size": (_S, [_DIMS, _I, _I]),
    "prr_workspace_init": (_I, [_P, _S, _P]),
    "prr_spec_state_floats": (_S, [_DIMS, _I, _I, ctypes.POINTER(_S), ctypes.POINTER(_S), ctypes.POINTER(_S)]),
    "prr_build_page_meta": (_I, [_DIMS, _P, _P, _I, _I, _I, _P, _P]),
    "prr_score_topk": (_I, [_DIMS, _P, _P, _I, _I, _P, _I, _I, _P, _P, _P, _I, _P, _S, _P]),
    "prr_score_topk_static": (_I, [_DIMS, _P, _P, _I, _I, _P, _I, _I, _P, _P, _P, _I, _P]),
    "prr_predict": (_I, [_DIMS, _P, _P, _P, _P, _I, _F, _F, _F, _I, _P, _I, _I, _P, _P, _I, _P]),
    "prr_spec_attn": (_I, [_DIMS, _P, _P, _P, _P, _I, _P, _P, _I, _I, _P, _P, _P, _P, _P]),
    "prr_repair": (_I, [_DIMS, _P, _P, _P, _P, _I, _I, _P, _P, _P, _P, _I, _I, _P, _P, _P, _P, _I,
                        _P, _P, _P, _P, _P, _P, _P, _S, _P]),
    "prr_merge_states": (_I, [_I, _I, _I, _P, _P, _P, _P, _P, _P, _P]),
    "prr_decode_step": (_I, [_DIMS, ctypes.POINTER(prr_step_params), ctypes.POINTER(prr_layer_io), _I, _I, _I, _P,
                             _P, ctypes.POINTER(ctypes.c_void_p)]),
    "prr_calibrate": (_I, [_P, _I, _I, _I, _P, _I, _I, _P, _I, _I, _P, _P]),
    "prr_epoch_advance": (_I, [_P, _P]),
    "prr_empty_launch": (_I, [_I, _I, _P]),
    "prr_read_stream": (_I, [_P, _S, _P, _I, _P]),
    "prr_stream_chain": (_I, [_I, _I, _P, _P]),
    "prr_fused_grid": (_I, [_DIMS, _P, _I]),
    "prr_pick_delta": (_I, [_P, _P, _P, _P, _I, _I, _I, _P, _P, _P]),
}
for _name, (_res, _args) in _SIGS.items():
    _fn = getattr(_lib, _name)
    _fn.restype = _res
    _fn.argtypes = _args


def status_string(status: int) -> str:
    return _lib.prr_status_string(status).decode()


def last_error() -> str:
    return _lib.prr_last_error().decode()


def _ptr(x) -> Optional[int]:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        if torch.cuda.is_available():
            return torch.cuda.current_stream().cuda_stream
        return None
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(status: int):
    if status != PRR_OK:
        raise PrrError(status, last_error())


def _forced(forced: Optional[Sequence[int]]):
    if not forced:
        return None, 0
    arr = (ctypes.c_int32 * len(forced))(*[int(x) for x in forced])
    return arr, len(forced)


def make_dims(num_q_heads, num_kv_heads, page_size, max_pages, dtype, meta_kind=PRR_META_MINMAX, head_dim=128):
    return prr_dims(num_q_heads, num_kv_heads, head_dim, page_size, max_pages, dtype, meta_kind)


def prr_workspace_size(dims: prr_dims, cap: int, chunk_pages: int) -> int:
    return int(_lib.prr_workspace_size(ctypes.byref(dims), cap, chunk_pages))


def prr_workspace_init(workspace, nbytes: int, stream=None):
    _check(_lib.prr_workspace_init(_ptr(workspace), nbytes, _stream(stream)))


def prr_spec_state_floats(dims: prr_dims, cap: int, chunk_pages: int):
    po, pml, pm = _S(), _S(), _S()
    total = _lib.prr_spec_state_floats(ctypes.byref(dims), cap, chunk_pages, ctypes.byref(po), ctypes.byref(pml),
                                       ctypes.byref(pm))
    return int(total), int(po.value), int(pml.value), int(pm.value)


def prr_build_page_meta(dims, k_cache, page_table, num_tokens, page_begin, page_end, meta, stream=None):
    _check(_lib.prr_build_page_meta(ctypes.byref(dims), _ptr(k_cache), _ptr(page_table), num_tokens, page_begin,
                                    page_end, _ptr(meta), _stream(stream)))


def prr_score_topk(dims, q, meta, num_pages, k_select, forced, forced_in_budget, scores, selected, selected_count,
                   cap, workspace, ws_bytes, stream=None):
    farr, nf = _forced(forced)
    _check(_lib.prr_score_topk(ctypes.byref(dims), _ptr(q), _ptr(meta), num_pages, k_select,
                               ctypes.cast(farr, _P) if farr is not None else None, nf, int(bool(forced_in_budget)),
                               _ptr(scores), _ptr(selected), _ptr(selected_count), cap, _ptr(workspace), ws_bytes,
                               _stream(stream)))


def prr_score_topk_static(dims, q, meta, num_pages, k_select, forced, forced_in_budget, scores, selected,
                          selected_count, cap, stream=None):
    farr, nf = _forced(forced)
    _check(_lib.prr_score_topk_static(ctypes.byref(dims), _ptr(q), _ptr(meta), num_pages, k_select,
                                      ctypes.cast(farr, _P) if farr is not None else None, nf,
                                      int(bool(forced_in_budget)), _ptr(scores), _ptr(selected), _ptr(selected_count),
                                      cap, _stream(stream)))


def prr_predict(dims, ema_level, ema_trend, ema_init_bits, scores, num_pages, alpha, beta, gamma, p_select, forced,
                forced_in_budget, predicted, predicted_count, cap, stream=None):
    farr, nf = _forced(forced)
    _check(_lib.prr_predict(ctypes.byref(dims), _ptr(ema_level), _ptr(ema_trend), _ptr(ema_init_bits), _ptr(scores),
                            num_pages, alpha, beta, gamma, p_select,
                            ctypes.cast(farr, _P) if farr is not None else None, nf, int(bool(forced_in_budget)),
                            _ptr(predicted), _ptr(predicted_count), cap, _stream(stream)))


def prr_spec_attn(dims, q, k_cache, v_cache, page_table, num_tokens, pages, page_count, cap, chunk_pages, part_o,
                  part_m, part_l, page_m, stream=None):
    _check(_lib.prr_spec_attn(ctypes.byref(dims), _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(page_table), num_tokens,
                              _ptr(pages), _ptr(page_count), cap, chunk_pages, _ptr(part_o), _ptr(part_m),
                              _ptr(part_l), _ptr(page_m), _stream(stream)))


def prr_repair(dims, q, k_cache, v_cache, page_table, num_tokens, num_pages, selected, selected_count, predicted,
               predicted_count, cap, chunk_pages, part_o, part_m, part_l, page_m, mode, out_o32, out_o, out_m, out_l,
               missed_count, wasted_count, workspace, ws_bytes, stream=None):
    _check(_lib.prr_repair(ctypes.byref(dims), _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(page_table), num_tokens,
                           num_pages, _ptr(selected), _ptr(selected_count), _ptr(predicted), _ptr(predicted_count),
                           cap, chunk_pages, _ptr(part_o), _ptr(part_m), _ptr(part_l), _ptr(page_m), mode,
                           _ptr(out_o32), _ptr(out_o), _ptr(out_m), _ptr(out_l), _ptr(missed_count),
                           _ptr(wasted_count), _ptr(workspace), ws_bytes, _stream(stream)))


def prr_merge_states(n_states, rows, d, o, m, l, out_o, out_m, out_l, stream=None):
    _check(_lib.prr_merge_states(n_states, rows, d, _ptr(o), _ptr(m), _ptr(l), _ptr(out_o), _ptr(out_m), _ptr(out_l),
                                 _stream(stream)))


def prr_epoch_advance(epoch_dev, stream=None):
    _check(_lib.prr_epoch_advance(_ptr(epoch_dev), _stream(stream)))


def prr_calibrate(scores, k_select, grid, p_select=0, n_threads=0, form_row=None):
    """scores: host float32 array [n_traj][n_rows][n_blocks]; grid: host float32 [n_grid][3];
    form_row: host int32 [n_blocks] (the row at which each block forms) or None.
    Returns (best theta as a tuple, objective per grid point as a float64 array)."""
    import numpy as np
    sc = np.ascontiguousarray(scores, dtype=np.float32)
    if sc.ndim == 2:
        sc = sc[None]
    g = np.ascontiguousarray(grid, dtype=np.float32).reshape(-1, 3)
    best = np.zeros(3, dtype=np.float32)
    obj = np.zeros(len(g), dtype=np.float64)
    fr = None if form_row is None else np.ascontiguousarray(form_row, dtype=np.int32)
    if fr is not None and fr.shape != (sc.shape[2],):
        raise ValueError(f"form_row has shape {fr.shape}, expected ({sc.shape[2]},)")
    _check(_lib.prr_calibrate(sc.ctypes.data, sc.shape[0], sc.shape[1], sc.shape[2],
                              None if fr is None else fr.ctypes.data, k_select, p_select,
                              g.ctypes.data, len(g), n_threads, best.ctypes.data, obj.ctypes.data))
    return tuple(float(x) for x in best), obj


def prr_pick_delta(rows, query_context, degree=2):
    """rows: the profiled table, dicts with "context", "delta", "select_us", "spec_us".
    Returns (delta, select_us estimate, spec_us estimate) at query_context."""
    import numpy as np
    ctx = np.ascontiguousarray([int(r["context"]) for r in rows], dtype=np.int32)
    dl = np.ascontiguousarray([float(r["delta"]) for r in rows], dtype=np.float32)
    se = np.ascontiguousarray([float(r["select_us"]) for r in rows], dtype=np.float32)
    sp = np.ascontiguousarray([float(r["spec_us"]) for r in rows], dtype=np.float32)
    out = (ctypes.c_float * 3)()
    n = len(rows)
    _check(_lib.prr_pick_delta(ctx.ctypes.data if n else None, dl.ctypes.data if n else None,
                               se.ctypes.data if n else None, sp.ctypes.data if n else None, n, int(query_context),
                               int(degree), ctypes.addressof(out), ctypes.addressof(out) + 4,
                               ctypes.addressof(out) + 8))
    return float(out[0]), float(out[1]), float(out[2])


def prr_empty_launch(grid, threads, stream=None):
    _check(_lib.prr_empty_launch(int(grid), int(threads), _stream(stream)))


def prr_read_stream(buf, nbytes, sink, grid, stream=None):
    _check(_lib.prr_read_stream(_ptr(buf), int(nbytes), _ptr(sink), int(grid), _stream(stream)))


PRR_CHAIN_ONE_STREAM = 0
PRR_CHAIN_EVENTS = 1
PRR_CHAIN_STREAM_MEMORY = 2


def prr_stream_chain(n_hops, mode, a=None, b=None):
    _check(_lib.prr_stream_chain(int(n_hops), int(mode), _stream(a), _stream(b) if b is not None else None))


def prr_fused_grid(dims, params, schedule):
    return int(_lib.prr_fused_grid(ctypes.byref(dims), ctypes.byref(params), int(schedule)))


def prr_decode_step(dims, params, layers, parity, schedule, stream=None, spec_stream=None, events=None):
    """layers: a ctypes array of prr_layer_io; events: a ctypes array of hipEvent_t (3 per layer + 1)."""
    _check(_lib.prr_decode_step(ctypes.byref(dims), ctypes.byref(params), layers, len(layers), parity, schedule,
                                _stream(stream), _stream(spec_stream) if spec_stream is not None else None,
                                events))


_hip = None


def hip_events(n):
    """n HIP events without timing (for prr_decode_step's fork/join), from the HIP runtime."""
    global _hip
    if _hip is None:
        _hip = ctypes.CDLL("libamdhip64.so")
        _hip.hipEventCreateWithFlags.restype = ctypes.c_int
        _hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
    arr = (ctypes.c_void_p * n)()
    for i in range(n):
        h = ctypes.c_void_p()
        err = _hip.hipEventCreateWithFlags(ctypes.byref(h), 0x2)  # hipEventDisableTiming
        if err != 0:
            raise PrrError(PRR_ERR_HIP, f"hipEventCreateWithFlags failed ({err})")
        arr[i] = h
    return arr


def library():
    """The loaded ctypes.CDLL (for symbol checks)."""
    return _lib
