"""Host-side tests of the C ABI (no GPU needed): the library loads, exports every
function include/prr.h declares, and rejects invalid arguments before any launch."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def P():
    import paper_2606_30389_amd as P
    return P


def declared_functions():
    src = open(os.path.join(ROOT, "include", "prr.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(prr_[a-z_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported(P):
    names = declared_functions()
    assert len(names) >= 11
    lib = P.library()
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(P.EXPORTED) == names


def test_status_strings(P):
    assert P.status_string(0) == "PRR_OK"
    assert P.status_string(P.PRR_ERR_INVALID_ARG) == "PRR_ERR_INVALID_ARG"
    assert P.status_string(99) == "PRR_ERR_UNKNOWN"


def test_workspace_and_spec_state_sizes(P):
    d = P.make_dims(32, 2, 16, 8192, P.PRR_BF16)
    ws = P.prr_workspace_size(d, 256, 8)
    nch = 32
    # flags + counters + per-work-unit partial states (2 * 32 units, 16 heads, 130 floats)
    assert ws >= 2 * 2 * nch * 16 * 130 * 4 and ws % 256 == 0
    tot, po, pml, pm = P.prr_spec_state_floats(d, 256, 8)
    assert (po, pml, pm) == (2 * nch * 16 * 128, 2 * nch * 16, 2 * 256 * 16)
    assert tot == po + 2 * pml + pm
    assert P.prr_workspace_size(d, 0, 8) == 0
    assert P.prr_workspace_size(d, 256, 17) == 0
    d64 = P.make_dims(32, 2, 64, 2048, P.PRR_BF16, P.PRR_META_MEAN)
    assert P.prr_workspace_size(d64, 67, 4) > 0 and P.prr_workspace_size(d64, 67, 5) == 0
    bad = P.make_dims(32, 2, 16, 8192, P.PRR_BF16, head_dim=64)
    assert P.prr_workspace_size(bad, 256, 8) == 0


FAKE = 0x10000  # an aligned non-null address; every case below fails validation before use


def _expect(P, status, fn, *args, **kwargs):
    with pytest.raises(P.PrrError) as ei:
        fn(*args, **kwargs)
    assert ei.value.status == status, str(ei.value)
    assert P.last_error()


@pytest.mark.parametrize("field,value,status", [
    ("head_dim", 64, 2), ("page_size", 48, 2), ("page_size", 512, 2), ("num_kv_heads", 0, 1), ("num_q_heads", 33, 1),
    ("num_q_heads", 34, 2), ("max_pages", 0, 1), ("dtype", 5, 1), ("meta_kind", 3, 1)])
def test_bad_dims(P, field, value, status):
    kw = dict(num_q_heads=32, num_kv_heads=2, page_size=16, max_pages=100, dtype=P.PRR_BF16)
    d = P.make_dims(**kw)
    setattr(d, field, value)
    _expect(P, status, P.prr_build_page_meta, d, FAKE, None, 1600, 0, 100, FAKE, None)


def test_bad_meta_args(P):
    d = P.make_dims(32, 2, 16, 100, P.PRR_BF16)
    _expect(P, 1, P.prr_build_page_meta, d, None, None, 1600, 0, 100, FAKE, None)
    _expect(P, 1, P.prr_build_page_meta, d, FAKE + 2, None, 1600, 0, 100, FAKE, None)
    _expect(P, 1, P.prr_build_page_meta, d, FAKE, None, 0, 0, 1, FAKE, None)
    _expect(P, 1, P.prr_build_page_meta, d, FAKE, None, 1601, 0, 100, FAKE, None)
    _expect(P, 1, P.prr_build_page_meta, d, FAKE, None, 1600, 0, 101, FAKE, None)
    _expect(P, 1, P.prr_build_page_meta, d, FAKE, None, 1600, 5, 4, FAKE, None)


def test_bad_score_topk_args(P):
    d = P.make_dims(32, 2, 16, 100, P.PRR_BF16)
    ws = P.prr_workspace_size(d, 16, 8)
    args = dict(q=FAKE, meta=FAKE, num_pages=100, k=16, forced=[], fib=True, scores=FAKE, sel=FAKE, cnt=FAKE,
                cap=16, ws=FAKE, wsb=ws)

    def call(**over):
        a = dict(args, **over)
        P.prr_score_topk(d, a["q"], a["meta"], a["num_pages"], a["k"], a["forced"], a["fib"], a["scores"], a["sel"],
                         a["cnt"], a["cap"], a["ws"], a["wsb"])

    _expect(P, 1, call, num_pages=0)
    _expect(P, 1, call, num_pages=101)
    _expect(P, 1, call, k=-1)
    _expect(P, 1, call, k=17)  # |A| exceeds cap
    _expect(P, 1, call, forced=[3, 3])
    _expect(P, 1, call, forced=[100])
    _expect(P, 1, call, forced=[1], fib=False)  # 16 + 1 > cap
    _expect(P, 1, call, forced=list(range(65)))
    _expect(P, 1, call, cap=0)
    _expect(P, 1, call, cap=2000)
    _expect(P, 1, call, q=FAKE + 8)
    _expect(P, 3, call, wsb=16)
    _expect(P, 1, call, ws=FAKE + 64)


def test_bad_predict_args(P):
    d = P.make_dims(4, 1, 16, 128, P.PRR_F16)

    def call(alpha=0.5, beta=0.5, gamma=0.0, p=16, cap=16, n=128):
        P.prr_predict(d, FAKE, FAKE, FAKE, None, n, alpha, beta, gamma, p, [], True, FAKE, FAKE, cap)

    _expect(P, 1, call, alpha=0.0)
    _expect(P, 1, call, alpha=1.5)
    _expect(P, 1, call, beta=0.0)
    _expect(P, 1, call, gamma=-0.1)
    _expect(P, 1, call, gamma=1.1)
    _expect(P, 1, call, p=-1)
    _expect(P, 1, call, p=17)
    _expect(P, 1, call, n=129)


def test_bad_spec_and_repair_args(P):
    d = P.make_dims(32, 2, 16, 100, P.PRR_BF16)
    ws = P.prr_workspace_size(d, 16, 8)
    _expect(P, 1, P.prr_spec_attn, d, FAKE, FAKE, FAKE, None, 1600, FAKE, FAKE, 16, 0, FAKE, FAKE, FAKE, None)
    _expect(P, 1, P.prr_spec_attn, d, FAKE, FAKE, FAKE, None, 1600, FAKE, FAKE, 16, 17, FAKE, FAKE, FAKE, None)
    _expect(P, 1, P.prr_spec_attn, d, FAKE, FAKE, FAKE, None, 0, FAKE, FAKE, 16, 8, FAKE, FAKE, FAKE, None)
    _expect(P, 1, P.prr_spec_attn, d, FAKE, FAKE, FAKE, None, 1600, FAKE, FAKE, 16, 8, FAKE + 4, FAKE, FAKE, None)

    def rep(pred=FAKE, pcnt=FAKE, mode=0, nt=1600, npg=100, wsb=ws, chunk=8):
        P.prr_repair(d, FAKE, FAKE, FAKE, None, nt, npg, FAKE, FAKE, pred, pcnt, 16, chunk, FAKE, FAKE, FAKE, None,
                     mode, FAKE, None, FAKE, FAKE, None, None, FAKE, wsb)

    _expect(P, 1, rep, pcnt=None)
    _expect(P, 1, rep, mode=2)
    _expect(P, 1, rep, npg=101)
    _expect(P, 1, rep, nt=1500)  # num_pages exceeds ceil(num_tokens / page_size)
    _expect(P, 3, rep, wsb=ws - 256)
    _expect(P, 3, rep, chunk=4)  # workspace sized for chunk 8 is too small for chunk 4
    _expect(P, 1, P.prr_merge_states, 1, 1, 2000, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE)
    _expect(P, 1, P.prr_workspace_init, FAKE + 16, 256)


def test_stream_chain_rejects_bad_arguments(P):
    # (fake stream handles: every case fails before the HIP runtime is called)
    for n_hops, mode, a, b in ((3, P.PRR_CHAIN_EVENTS, 16, 32), (0, P.PRR_CHAIN_EVENTS, 16, 32),
                               (258, P.PRR_CHAIN_ONE_STREAM, 16, 32), (4, 3, 16, 32),
                               (4, P.PRR_CHAIN_EVENTS, 16, 16), (4, P.PRR_CHAIN_STREAM_MEMORY, 16, 16)):
        with pytest.raises(P.PrrError) as e:
            P.prr_stream_chain(n_hops, mode, a, b)
        assert e.value.status == P.PRR_ERR_INVALID_ARG, (n_hops, mode)


def test_last_error_is_thread_local(P):
    import threading
    d = P.make_dims(32, 2, 16, 100, P.PRR_BF16)
    with pytest.raises(P.PrrError):
        P.prr_build_page_meta(d, None, None, 1600, 0, 100, FAKE, None)
    msg = []
    t = threading.Thread(target=lambda: msg.append(P.last_error()))
    t.start()
    t.join()
    assert msg == [""] and "k_cache" in P.last_error()


def test_fused_step_rejects_bad_stamps_and_epoch(P):
    """Fused schedules: a misaligned phase-stamp buffer and the reserved epoch 0 are rejected
    before any launch."""
    d = P.make_dims(32, 2, 16, 100, P.PRR_BF16)
    ws = P.prr_workspace_size(d, 16, 8)
    y = P.prr_layer_io()
    for name, _ in P.prr_layer_io._fields_:
        if name in ("predicted", "predicted_count"):
            getattr(y, name)[0] = FAKE
            getattr(y, name)[1] = FAKE
        elif name == "ws_bytes":
            y.ws_bytes = ws
        elif name in ("page_table", "out_o", "missed_count", "wasted_count", "covered_count", "theta"):
            setattr(y, name, None)
        else:
            setattr(y, name, FAKE)
    layers = (P.prr_layer_io * 1)(y)

    def params(stamps=None, epoch=1):
        p = P.prr_step_params()
        p.num_tokens, p.num_pages, p.k_select, p.p_select, p.cap = 1600, 100, 16, 16, 16
        p.chunk_pages, p.mode, p.forced_in_budget, p.n_forced = 8, 0, 1, 0
        p.alpha, p.beta, p.gamma, p.epoch, p.late_spec = 0.5, 0.5, 0.0, epoch, 1
        p.phase_stamps = stamps
        return p

    _expect(P, 1, P.prr_decode_step, d, params(stamps=FAKE + 4), layers, 0, P.PRR_SCHED_FUSED_PRR)
    _expect(P, 1, P.prr_decode_step, d, params(epoch=0), layers, 0, P.PRR_SCHED_FUSED_PRR)
    bad_late = params()
    bad_late.late_spec = 3
    _expect(P, 1, P.prr_decode_step, d, bad_late, layers, 0, P.PRR_SCHED_FUSED_PRR)
    # a layer's own (alpha, beta, gamma) out of range (host memory, read at the call)
    import numpy as np
    for bad in ((0.0, 0.5, 0.0), (0.5, 1.5, 0.0), (0.5, 0.5, -0.25)):
        th = np.asarray(bad, dtype=np.float32)
        layers[0].theta = th.ctypes.data
        for sched in (P.PRR_SCHED_FUSED_PRR, P.PRR_SCHED_FUSED_PREFILL):
            _expect(P, 1, P.prr_decode_step, d, params(), layers, 0, sched)
            assert "alpha" in P.last_error()
    layers[0].theta = None
    assert P.prr_fused_grid(d, params(), P.PRR_SCHED_FUSED_PRR) > 0


def test_fused_step_page_cap(P):
    """The fused schedules take at most 8192 pages per KV head (the select workgroup's
    fallback holds every score of a KV head); a longer context is PRR_ERR_UNSUPPORTED before
    any launch, while the separate kernels' workspace still covers it."""
    d = P.make_dims(32, 2, 16, 16384, P.PRR_BF16)
    assert P.prr_workspace_size(d, 256, 8) > 0
    y = P.prr_layer_io()
    for name, _ in P.prr_layer_io._fields_:
        if name in ("predicted", "predicted_count"):
            getattr(y, name)[0] = FAKE
            getattr(y, name)[1] = FAKE
        elif name == "ws_bytes":
            y.ws_bytes = P.prr_workspace_size(d, 256, 8)
        elif name in ("page_table", "out_o", "missed_count", "wasted_count", "covered_count", "theta"):
            setattr(y, name, None)
        else:
            setattr(y, name, FAKE)
    layers = (P.prr_layer_io * 1)(y)
    for npages, status in ((8193, 2), (16384, 2)):
        p = P.prr_step_params()
        p.num_tokens, p.num_pages, p.k_select, p.p_select, p.cap = 16 * npages, npages, 256, 256, 256
        p.chunk_pages, p.alpha, p.beta, p.epoch, p.late_spec = 8, 0.5, 0.5, 1, 1
        for sched in (P.PRR_SCHED_FUSED_SERIAL, P.PRR_SCHED_FUSED_PRR, P.PRR_SCHED_FUSED_PREFILL):
            _expect(P, status, P.prr_decode_step, d, p, layers, 0, sched)
            assert "8192" in P.last_error()


@pytest.mark.parametrize("ps", [32, 128, 256])
def test_fused_schedules_need_page_16_or_64(P, ps):
    """The separate kernels take pages of 16 to 256 tokens; the fused schedules only 16
    and 64 (PRR_ERR_UNSUPPORTED before any launch)."""
    d = P.make_dims(32, 8, ps, 64, P.PRR_F16)
    assert P.prr_workspace_size(d, 8, 1) > 0
    p = P.prr_step_params()
    p.num_tokens, p.num_pages, p.k_select, p.p_select, p.cap, p.chunk_pages, p.epoch = 64 * ps, 64, 8, 8, 8, 1, 1
    layers = (P.prr_layer_io * 1)()
    for sched in (P.PRR_SCHED_FUSED_SERIAL, P.PRR_SCHED_FUSED_PRR, P.PRR_SCHED_FUSED_PREFILL):
        _expect(P, 2, P.prr_decode_step, d, p, layers, 0, sched)
        assert P.prr_fused_grid(d, p, sched) == 0


def test_fused_grid_counts_the_roles(P):
    """prr_fused_grid: per KV head, the score workgroups (128 pages each), the select, the
    predict (PRR and prefill), the speculation and late workgroups (PRR, one per chunk of the
    list capacity), the missed-page workgroups (one per chunk, or four taking the chunks in
    turn with late speculation at one page per wave) and the merge (one per query head)."""
    d = P.make_dims(32, 2, 16, 8192, P.PRR_BF16)
    p = P.prr_step_params()
    p.num_tokens, p.num_pages, p.k_select, p.p_select, p.cap, p.chunk_pages, p.epoch = 131072, 8192, 256, 256, 256, 8, 1
    p.alpha, p.beta, p.gamma = 0.5, 0.5, 0.0
    n_score, nch, g = 64, 32, 16
    p.late_spec = 1
    assert P.prr_fused_grid(d, p, P.PRR_SCHED_FUSED_PRR) == 2 * (n_score + 2 + 2 * nch + 4 + g)
    p.chunk_pages = 16  # (two pages per wave: a missed-page workgroup per chunk)
    assert P.prr_fused_grid(d, p, P.PRR_SCHED_FUSED_PRR) == 2 * (n_score + 2 + 3 * 16 + g)
    p.chunk_pages = 8
    p.late_spec = 0
    assert P.prr_fused_grid(d, p, P.PRR_SCHED_FUSED_PRR) == 2 * (n_score + 2 + 2 * nch + g)
    assert P.prr_fused_grid(d, p, P.PRR_SCHED_FUSED_PREFILL) == 2 * (n_score + 2)
    p.chunk_pages = 4
    assert P.prr_fused_grid(d, p, P.PRR_SCHED_FUSED_SERIAL) == 2 * (n_score + 1 + 64 + g)
    p.chunk_pages = 17  # (invalid: the helper returns 0)
    assert P.prr_fused_grid(d, p, P.PRR_SCHED_FUSED_SERIAL) == 0
