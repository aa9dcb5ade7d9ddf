"""Parity of the HIP path (through the C ABI) with the fp64 oracle, on the GPU.

Every case prints its name, workload, shape and seed before touching the GPU.
"""
import zlib

import numpy as np
import pytest

import oracle as O
import workloads as W
from tests import gpu_support as S

pytestmark = pytest.mark.gpu

# (workload, pages per KV head or None = full size)
FULL = [("tiny", None), ("glm32k", None), ("glm128k", None), ("llama64k", None), ("infllm128k", None)]
REDUCED = [("tiny", None), ("glm32k", 300), ("glm128k", 777), ("llama64k", 129), ("infllm128k", 150)]


@pytest.fixture(scope="module")
def torch():
    import torch as _t
    assert _t.cuda.is_available(), "no GPU visible"
    import paper_2606_30389_amd  # noqa: F401  (fails loudly when libprr.so is missing)
    return _t


def _setup(name, npages, **kw):
    cfg = W.CONFIGS[name]
    pc = S.path_config(cfg, num_pages=npages, **kw)
    S.log(f"setup {name}: pages={pc.num_pages} tokens={pc.num_tokens} Hq={pc.num_q_heads} Hkv={pc.num_kv_heads} "
          f"dtype={pc.dtype} meta={pc.meta_kind} chunk={pc.chunk_pages}")
    st, li = S.make_layer(cfg, pc)
    return cfg, pc, st, li


# ----------------------------------------------------------------------------- metadata

@pytest.mark.parametrize("name,npages", FULL + [("glm32k", 77)])
def test_meta_parity(torch, name, npages):
    cfg, pc, st, li = _setup(name, npages)
    st.build_meta()
    torch.cuda.synchronize()
    ref = S.oracle_meta(li, pc)
    if pc.meta_kind == "mean":
        got = S.to_np(st.meta)[:, :pc.num_pages]
        assert np.allclose(got, ref, rtol=2e-6, atol=2e-7), np.abs(got - ref).max()
    else:
        got = S.to_np(st.meta)[:, :pc.num_pages]
        assert np.array_equal(got[:, :, 0], ref[0]) and np.array_equal(got[:, :, 1], ref[1])


def test_meta_partial_last_page_and_range(torch):
    cfg = W.CONFIGS["glm32k"]
    for nt in (64 * 16 - 5, 64 * 16 - 15, 63 * 16 + 1):
        pc = S.path_config(cfg, num_pages=64, num_tokens=nt)
        S.log(f"meta partial page: tokens={nt}")
        st, li = S.make_layer(cfg, pc)
        st.build_meta(page_begin=0, page_end=pc.num_pages)
        torch.cuda.synchronize()
        ref = S.oracle_meta(li, pc)
        got = S.to_np(st.meta)[:, :pc.num_pages]
        assert np.array_equal(got[:, :, 0], ref[0]) and np.array_equal(got[:, :, 1], ref[1])
    # a sub-range leaves the other pages untouched
    pc = S.path_config(cfg, num_pages=64)
    st, li = S.make_layer(cfg, pc)
    st.meta.fill_(7)
    st.build_meta(page_begin=10, page_end=20)
    torch.cuda.synchronize()
    got = S.to_np(st.meta)
    ref = S.oracle_meta(li, pc)
    assert np.array_equal(got[:, 10:20, 0], ref[0][:, 10:20])
    assert np.all(got[:, :10] == 7) and np.all(got[:, 20:64] == 7)


def test_meta_mean_page16_and_minmax_page64(torch):
    # the other (meta kind, page size) pairings compile and match too
    for name, kind in (("glm32k", "mean"), ("infllm128k", "minmax")):
        cfg = W.CONFIGS[name]
        pc = S.path_config(cfg, num_pages=40)
        pc.meta_kind = kind
        S.log(f"meta {kind} on {name} pages")
        st, li = S.make_layer(cfg, pc)
        st.build_meta()
        torch.cuda.synchronize()
        ref = S.oracle_meta(li, pc)
        got = S.to_np(st.meta)[:, :pc.num_pages]
        if kind == "mean":
            assert np.allclose(got, ref, rtol=2e-6, atol=2e-7)
        else:
            assert np.array_equal(got[:, :, 0], ref[0]) and np.array_equal(got[:, :, 1], ref[1])


# ----------------------------------------------------------------------------- score + top-K

@pytest.mark.parametrize("name,npages", FULL + REDUCED[1:])
def test_score_topk_parity(torch, name, npages):
    cfg, pc, st, li = _setup(name, npages)
    st.build_meta()
    meta = S.oracle_meta(li, pc)
    _, qb = W.query_trajectory(cfg, 0, steps=3)
    for t in range(4):
        S.log(f"score_topk {name} step {t}")
        st.select(S.q_tensor(qb[t], pc))
        torch.cuda.synchronize()
        ref = S.oracle_scores(W.bits_to_f64(qb[t], cfg.dtype), meta, pc)
        got = S.to_np(st.scores)[:, :pc.num_pages]
        assert np.all(np.abs(got - ref) <= 1e-5 * np.maximum(1.0, np.abs(ref))), np.abs(got - ref).max()
        S.check_selection(S.lists(st), ref, pc.k_select, list(pc.forced), pc.forced_in_budget)


@pytest.mark.parametrize("k,forced,fib", [(0, [], True), (1, [], True), (5, [3, 0], True), (5, [3, 0], False),
                                          (2, [7, 1, 4], True), (299, [], True), (400, [], True), (40, [299], False)])
def test_topk_budgets_and_forced(torch, k, forced, fib):
    cfg = W.CONFIGS["glm32k"]
    pc = S.path_config(cfg, num_pages=300)
    pc.k_select, pc.forced, pc.forced_in_budget = k, forced, fib
    S.log(f"top-k budget k={k} forced={forced} in_budget={fib}")
    st, li = S.make_layer(cfg, pc)
    st.build_meta()
    _, qb = W.query_trajectory(cfg, 0, steps=0)
    st.select(S.q_tensor(qb[0], pc))
    torch.cuda.synchronize()
    ref = S.oracle_scores(W.bits_to_f64(qb[0], cfg.dtype), S.oracle_meta(li, pc), pc)
    S.check_selection(S.lists(st), ref, k, forced, fib)


def test_topk_exact_ties(torch):
    """All pages identical -> all scores equal -> the lowest page indices win."""
    torch_ = torch
    cfg = W.CONFIGS["glm32k"]
    pc = S.path_config(cfg, num_pages=200)
    S.log("top-k ties")
    st, li = S.make_layer(cfg, pc)
    st.k[:] = st.k[:, :1].clone()
    st.build_meta()
    _, qb = W.query_trajectory(cfg, 0, steps=0)
    st.select(S.q_tensor(qb[0], pc))
    torch_.cuda.synchronize()
    for h, lst in enumerate(S.lists(st)):
        want = sorted({0, 199} | set(range(1, 1 + pc.k_select - 2)))
        assert list(np.sort(lst)) == want


# ----------------------------------------------------------------------------- predictor

@pytest.mark.parametrize("name,npages", REDUCED + [("glm128k", None)])
def test_predict_parity(torch, name, npages):
    cfg, pc, st, li = _setup(name, npages)
    st.build_meta()
    meta = S.oracle_meta(li, pc)
    steps = 6
    _, qb = W.query_trajectory(cfg, 0, steps=steps)
    forced = list(pc.forced)
    level = trend = None
    for t in range(steps + 1):
        S.log(f"predict {name} step {t}")
        st.select(S.q_tensor(qb[t], pc))
        st.predict()
        torch.cuda.synchronize()
        s64 = S.oracle_scores(W.bits_to_f64(qb[t], cfg.dtype), meta, pc)
        if level is None:
            level, trend = O.ema_init(s64)
        else:
            level, trend = O.ema_update(level, trend, s64, cfg.alpha, cfg.beta)
        scale = max(1.0, np.abs(s64).max())
        gl = S.to_np(st.level)[:, :pc.num_pages]
        gt = S.to_np(st.trend)[:, :pc.num_pages]
        assert np.abs(gl - level).max() <= 1e-5 * scale
        assert np.abs(gt - trend).max() <= 1e-5 * scale
        pred = O.ema_predict(level, trend, cfg.gamma)
        S.check_selection(S.lists(st, 1 - st.cur), pred, pc.k_select, forced, pc.forced_in_budget, what="P")
        st.advance()


def test_predict_trend_and_uninitialised_pages(torch):
    """gamma > 0 exercises the trend; pages without state are never predicted unless forced;
    the predict-only call (no scores) leaves the state unchanged."""
    cfg = W.CONFIGS["glm32k"]
    pc = S.path_config(cfg, num_pages=256)
    pc.alpha, pc.beta, pc.gamma = 0.6, 0.3, 0.75
    S.log("predict with trend")
    st, li = S.make_layer(cfg, pc)
    st.build_meta()
    meta = S.oracle_meta(li, pc)
    _, qb = W.query_trajectory(cfg, 0, steps=4)
    level = trend = None
    for t in range(5):
        st.select(S.q_tensor(qb[t], pc))
        st.predict()
        torch.cuda.synchronize()
        s64 = S.oracle_scores(W.bits_to_f64(qb[t], cfg.dtype), meta, pc)
        level, trend = (O.ema_init(s64) if level is None else O.ema_update(level, trend, s64, 0.6, 0.3))
        pred = O.ema_predict(level, trend, 0.75)
        S.check_selection(S.lists(st, 1 - st.cur), pred, pc.k_select, list(pc.forced), True, what="P")
        st.advance()
    lv0 = st.level.clone()
    st.predict(with_scores=False)
    torch.cuda.synchronize()
    assert torch.equal(lv0, st.level)
    # half of the pages lose their state: only initialised or forced pages may be predicted
    st.init_bits[:, :4] = 0
    st.predict(with_scores=False)
    torch.cuda.synchronize()
    for lst in S.lists(st, 1 - st.cur):
        assert all(p >= 128 or p in pc.forced for p in lst)


def _select_values(dist, n, rng):
    """float32 keys of one KV head with the structure `dist` asks for."""
    f32 = np.float32
    if dist == "gauss":
        return rng.standard_normal(n).astype(f32)
    if dist == "extreme":  # the range overflows float32: the key-space select
        return rng.uniform(-3.0e38, 3.0e38, n).astype(f32)
    if dist == "inf":
        v = rng.standard_normal(n).astype(f32)
        v[rng.choice(n, 7, replace=False)] = np.inf
        v[rng.choice(n, 5, replace=False)] = -np.inf
        return v
    if dist == "equal_at_threshold":  # rank K falls inside a group of 500 equal keys
        v = np.where(rng.random(n) < 0.5, rng.uniform(2.0, 3.0, n), rng.uniform(-3.0, 0.5, n)).astype(f32)
        grp = rng.choice(n, 500, replace=False)
        v[grp] = 1.0
        return v
    if dist == "dense_bin":  # 600 distinct keys inside one of the 2048 value bins
        v = rng.uniform(-1000.0, 1000.0, n).astype(f32)
        grp = rng.choice(n, 600, replace=False)
        v[grp] = (1.0 + rng.random(600) * 1e-4).astype(f32)
        v[rng.choice(np.setdiff1d(np.arange(n), grp), 40, replace=False)] = 2000.0
        return v
    if dist == "constant":  # every key equal: the lowest page indices win
        return np.full(n, -0.75, dtype=f32)
    if dist == "tiny":  # normal floats so close together that 2048 / span overflows
        mag = 1e-36 * (1.0 + np.abs(rng.standard_normal(n)))
        return np.where(rng.random(n) < 0.5, -mag, mag).astype(f32)
    if dist == "negative_zero":  # -0.0 and +0.0 are the same key
        v = np.zeros(n, dtype=f32)
        v[rng.random(n) < 0.5] = -0.0
        v[rng.choice(n, 30, replace=False)] = 1.0
        return v
    raise ValueError(dist)


SELECT_DISTS = ["gauss", "extreme", "inf", "equal_at_threshold", "dense_bin", "constant", "tiny", "negative_zero"]


@pytest.mark.parametrize("dist", SELECT_DISTS)
@pytest.mark.parametrize("n,k", [(8192, 256), (3001, 1000), (16384, 1024), (700, 900)])
def test_predict_select_key_structures(torch, dist, n, k):
    """The separate kernels' top-K (shared by prr_score_topk and prr_predict) on keys set
    directly (gamma = 0, so the predicted key is the level): every path of the select
    (value bins, a crowded boundary bin, the key-space fallback for non-finite or
    underflowing spans, ties cut by page index) against the oracle's ranking, exactly."""
    from paper_2606_30389_amd import runtime as R
    S.log(f"select structure {dist}: n={n} k={k}")
    pc = R.PathConfig(num_q_heads=8, num_kv_heads=2, page_size=16, num_tokens=n * 16, k_select=k,
                      forced=[0, n - 1], forced_in_budget=True, dtype="bf16")
    st = R.LayerState(pc, torch.device("cuda:0"))
    rng = np.random.default_rng(zlib.crc32(f"{dist}/{n}".encode()))
    vals = np.stack([_select_values(dist, n, rng) for _ in range(2)])
    st.level[:, :n].copy_(torch.from_numpy(vals))
    st.trend.zero_()
    st.init_bits.fill_(-1)
    st.predict(with_scores=False)
    torch.cuda.synchronize()
    for h, got in enumerate(S.lists(st, 1 - st.cur)):
        want = O.select_topk(vals[h].astype(np.float64), k, [0, n - 1], True)
        assert np.array_equal(np.sort(got), want), f"head {h}: {len(set(got) ^ set(want))} pages differ"


# ----------------------------------------------------------------------------- attention

def _upload_lists(torch, lists, cap):
    hkv = len(lists)
    arr = np.full((hkv, cap), -7, dtype=np.int32)
    cnt = np.zeros(hkv, dtype=np.int32)
    for h, l in enumerate(lists):
        arr[h, :len(l)] = l
        cnt[h] = len(l)
    dev = torch.device("cuda:0")
    return torch.from_numpy(arr).to(dev), torch.from_numpy(cnt).to(dev)


def _run_spec_repair(torch, st, q, A, P, mode):
    cap = st.cap
    a_t, a_c = _upload_lists(torch, A, cap)
    st.sel.copy_(a_t)
    st.sel_count.copy_(a_c)
    for buf in (st.out_o32, st.out_m, st.out_l):
        buf.fill_(float("nan"))
    if P is None:
        st.repair(q, serial=True)
    else:
        p_t, p_c = _upload_lists(torch, P, cap)
        st.speculate(q, pages=p_t, counts=p_c)
        st.repair(q, mode=mode, pages=p_t, counts=p_c)
    torch.cuda.synchronize()
    return S.to_np(st.out_o32), S.to_np(st.out_o), S.to_np(st.out_m), S.to_np(st.out_l)


SPLITS = ["serial", "empty", "equal", "disjoint", "superset", "random", "subset"]


@pytest.mark.parametrize("name,npages", [("tiny", None), ("glm32k", 300), ("llama64k", 200), ("infllm128k", 90)])
@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("split", SPLITS)
def test_speculate_repair_any_split(torch, name, npages, mode, split):
    """Host-chosen A and P (every kind of misprediction): the output is attention over
    exactly A (exact mode) or over P u A (keep-wasted mode)."""
    cfg, pc, st, li = _setup(name, npages)
    rng = np.random.default_rng(zlib.crc32(f"{name}/{split}/{mode}".encode()))
    n = pc.num_pages
    ka = min(pc.k_select - 5, n // 2)
    A, P = [], []
    for h in range(pc.num_kv_heads):
        a = np.sort(rng.choice(n, ka, replace=False))
        rest = np.setdiff1d(np.arange(n), a)
        if split == "empty":
            p = np.array([], dtype=np.int64)
        elif split in ("equal", "serial"):
            p = a.copy()
        elif split == "disjoint":
            p = np.sort(rng.choice(rest, min(ka, len(rest)), replace=False))
        elif split == "superset":
            p = np.sort(np.concatenate([a, rng.choice(rest, min(5, len(rest)), replace=False)]))[:st.cap]
        elif split == "subset":
            p = np.sort(rng.choice(a, ka // 2, replace=False))
        else:
            keep = a[rng.random(len(a)) < 0.7]
            p = np.sort(np.concatenate([keep, rng.choice(rest, ka - len(keep), replace=False)]))
        A.append(a)
        P.append(p)
    _, qb = W.query_trajectory(cfg, 0, steps=1)
    q = S.q_tensor(qb[1], pc)
    q64 = W.bits_to_f64(qb[1], cfg.dtype)
    S.log(f"spec+repair {name} split={split} mode={mode}")
    o32, od, m, l = _run_spec_repair(torch, st, q, A, None if split == "serial" else P, mode)
    k64, v64 = li.k64(), li.v64()
    target = A if (mode == 0 or split == "serial") else [np.union1d(a, p) for a, p in zip(A, P)]
    ref = O.attend(q64, k64, v64, target, pc.page_size, pc.num_tokens)
    S.check_attention(o32, m, l, ref, od, dtype=pc.dtype)
    if split != "serial":
        mc, wc = S.to_np(st.missed), S.to_np(st.wasted)
        for h in range(pc.num_kv_heads):
            mm, ww = O.missed_and_wasted(A[h], P[h])
            assert mc[h] == len(mm) and wc[h] == len(ww)


def _page_masses(q64, k64, pages, page_size, num_tokens, g):
    """Per (query head, page): the page's softmax mass sum_t exp(q.k_t / sqrt(d)) (fp64)."""
    out = np.zeros((q64.shape[0], len(pages)))
    for i, p in enumerate(pages):
        toks = O.page_tokens([p], page_size, num_tokens) - p * page_size
        for j in range(q64.shape[0]):
            out[j, i] = np.exp(k64[j // g, p, toks] @ q64[j] / np.sqrt(q64.shape[1])).sum()
    return out


@pytest.mark.parametrize("band", [(0.80, 0.875), (0.876, 0.95)], ids=["subtract", "reattend"])
def test_repair_wasted_share_near_the_limit(torch, band):
    """Exact-mode repair of a speculation chunk whose wasted pages carry a share of the
    chunk's softmax mass just below the 7/8 limit for every query head (the wasted part is
    subtracted, the largest cancellation allowed) and just above it for some head (the
    chunk's pages of A are attended afresh).  The chunk is chosen on the CPU from the
    oracle's per-page masses."""
    cfg, pc, st, li = _setup("glm32k", 300)
    _, qb = W.query_trajectory(cfg, 0, steps=1)
    q64 = W.bits_to_f64(qb[1], cfg.dtype)
    k64, v64 = li.k64(), li.v64()
    g = pc.group
    rng = np.random.default_rng(42)
    pool = rng.choice(300, 120, replace=False)
    masses = _page_masses(q64, k64, pool, 16, pc.num_tokens, g)
    lo, hi = band
    found = None
    for _ in range(200000):
        pick = rng.choice(len(pool), 8, replace=False)
        wasted, clean = pick[:6], pick[6:]
        tot = [masses[h * g:(h + 1) * g][:, pick].sum(axis=1) for h in range(2)]
        share = [masses[h * g:(h + 1) * g][:, wasted].sum(axis=1) / tot[h] for h in range(2)]
        top = max(float(share[0].max()), float(share[1].max()))
        if lo <= top < hi:
            found = (pool[wasted], pool[clean], top)
            break
    assert found is not None, "no chunk with the wanted wasted share"
    wasted, clean, top = found
    S.log(f"wasted share {top:.4f} in band {band}")
    chunk = np.sort(np.concatenate([wasted, clean]))
    extra = np.setdiff1d(pool, chunk)[:20]
    A = [np.sort(np.concatenate([clean, extra])) for _ in range(2)]
    P = [chunk for _ in range(2)]
    o32, od, m, l = _run_spec_repair(torch, st, S.q_tensor(qb[1], pc), A, P, 0)
    S.check_attention(o32, m, l, O.attend(q64, k64, v64, A, 16, pc.num_tokens), od, dtype=pc.dtype)


@pytest.mark.parametrize("chunk", [1, 3, 8, 16])
def test_chunk_sizes(torch, chunk):
    cfg, pc, st, li = _setup("glm32k", 500, chunk_pages=chunk)
    rng = np.random.default_rng(chunk)
    A = [np.sort(rng.choice(500, 128, replace=False)) for _ in range(2)]
    P = [np.sort(np.concatenate([a[:90], rng.choice(np.setdiff1d(np.arange(500), a), 38, replace=False)])) for a in A]
    _, qb = W.query_trajectory(cfg, 0, steps=1)
    q64 = W.bits_to_f64(qb[1], cfg.dtype)
    S.log(f"chunk={chunk}")
    o32, od, m, l = _run_spec_repair(torch, st, S.q_tensor(qb[1], pc), A, P, 0)
    S.check_attention(o32, m, l, O.attend(q64, li.k64(), li.v64(), A, 16, pc.num_tokens), od, dtype=pc.dtype)


def test_all_pages_is_dense_attention(torch):
    """K = N: the sparse output equals dense attention over the whole context."""
    cfg = W.CONFIGS["tiny"]
    pc = S.path_config(cfg)
    pc.k_select = pc.num_pages
    S.log("all pages selected")
    st, li = S.make_layer(cfg, pc)
    _, qb = W.query_trajectory(cfg, 0, steps=1)
    q = S.q_tensor(qb[1], pc)
    st.build_meta()
    st.select(q)
    st.repair(q, serial=True)
    torch.cuda.synchronize()
    q64 = W.bits_to_f64(qb[1], cfg.dtype)
    ref = O.attend(q64, li.k64(), li.v64(), [range(pc.num_pages)], 16, pc.num_tokens)
    S.check_attention(S.to_np(st.out_o32), S.to_np(st.out_m), S.to_np(st.out_l), ref, S.to_np(st.out_o), dtype=pc.dtype)


@pytest.mark.parametrize("poison", [False, True], ids=["clean-tail", "nan-tail"])
@pytest.mark.parametrize("name", ["glm32k", "infllm128k"])
def test_partial_last_page(torch, name, poison):
    """A partial last page; with `poison` the tokens past num_tokens hold NaN and Inf in K
    and V (an unwritten cache tail), which must not reach the metadata or the output."""
    cfg = W.CONFIGS[name]
    npg = 100
    nt = npg * cfg.page_size - (5 if cfg.page_size == 16 else 37)
    pc = S.path_config(cfg, num_pages=npg, num_tokens=nt)
    S.log(f"partial last page {name} tokens={nt} poison={poison}")
    st, li = S.make_layer(cfg, pc)
    if poison:
        valid = nt - (npg - 1) * cfg.page_size
        st.v[:, npg - 1, valid:] = float("nan")
        st.k[:, npg - 1, valid:] = float("inf")
        st.k[:, npg - 1, valid::3] = float("nan")
    st.build_meta()
    _, qb = W.query_trajectory(cfg, 0, steps=1)
    q = S.q_tensor(qb[1], pc)
    st.select(q)
    st.predict()
    st.advance()
    st.select(q)
    st.speculate(q)
    st.repair(q)
    torch.cuda.synchronize()
    q64 = W.bits_to_f64(qb[1], cfg.dtype)
    meta = S.oracle_meta(li, pc)
    A = S.check_selection(S.lists(st), S.oracle_scores(q64, meta, pc), pc.k_select, list(pc.forced), pc.forced_in_budget)
    assert all(npg - 1 in a for a in A)  # forced pages include the partial last page
    ref = O.attend(q64, li.k64(), li.v64(), A, pc.page_size, nt)
    S.check_attention(S.to_np(st.out_o32), S.to_np(st.out_m), S.to_np(st.out_l), ref, S.to_np(st.out_o), dtype=pc.dtype)


def test_page_table_indirection(torch):
    cfg = W.CONFIGS["glm32k"]
    pc = S.path_config(cfg, num_pages=256)
    ptab = W.page_table_permutation(256, 300, seed=5)
    S.log("page table")
    st, li = S.make_layer(cfg, pc, page_table=ptab, num_physical=300)
    st.build_meta()
    meta = S.oracle_meta(li, pc)
    got = S.to_np(st.meta)[:, :256]
    assert np.array_equal(got[:, :, 0], meta[0]) and np.array_equal(got[:, :, 1], meta[1])
    _, qb = W.query_trajectory(cfg, 0, steps=2)
    st.select(S.q_tensor(qb[0], pc))
    st.predict()
    st.advance()
    q = S.q_tensor(qb[1], pc)
    st.select(q)
    st.speculate(q)
    st.repair(q)
    torch.cuda.synchronize()
    q64 = W.bits_to_f64(qb[1], cfg.dtype)
    A = S.check_selection(S.lists(st), S.oracle_scores(q64, meta, pc), pc.k_select, list(pc.forced), True)
    ref = O.attend(q64, li.k64(), li.v64(), A, 16, pc.num_tokens)
    S.check_attention(S.to_np(st.out_o32), S.to_np(st.out_m), S.to_np(st.out_l), ref, S.to_np(st.out_o), dtype=pc.dtype)


def test_out_of_range_list_entries_are_skipped(torch):
    cfg, pc, st, li = _setup("glm32k", 200)
    A = [np.array([1, 5, 9, 13]), np.array([2, 4])]
    A_bad = [np.array([1, 5, -3, 9, 13, 200]), np.array([2, 4, 999])]
    P_bad = [np.array([5, 9, 250, 17]), np.array([-1, 4])]
    _, qb = W.query_trajectory(cfg, 0, steps=1)
    q64 = W.bits_to_f64(qb[1], cfg.dtype)
    S.log("out-of-range entries")
    o32, od, m, l = _run_spec_repair(torch, st, S.q_tensor(qb[1], pc), A_bad, P_bad, 0)
    S.check_attention(o32, m, l, O.attend(q64, li.k64(), li.v64(), A, 16, pc.num_tokens), od, dtype=pc.dtype)
    flags = int(st.workspace[0].item())
    assert flags & 1


def test_empty_selection_gives_empty_state(torch):
    cfg, pc, st, li = _setup("glm32k", 100)
    _, qb = W.query_trajectory(cfg, 0, steps=1)
    S.log("empty A")
    o32, od, m, l = _run_spec_repair(torch, st, S.q_tensor(qb[1], pc), [np.array([], int)] * 2,
                                     [np.array([3, 4]), np.array([], int)], 0)
    assert np.all(o32 == 0) and np.all(np.isneginf(m)) and np.all(l == 0)


# ----------------------------------------------------------------------------- whole steps

@pytest.mark.parametrize("name,npages,steps", [("tiny", None, 16), ("glm32k", None, 8), ("glm128k", None, 4),
                                               ("llama64k", None, 4), ("infllm128k", None, 4)])
@pytest.mark.parametrize("mode", [0, 1])
def test_decode_steps_parity(torch, name, npages, steps, mode):
    """The full PRR step (select, speculate over the prediction, repair, predict) over
    several decode steps at the workload's full size, against the oracle's selections,
    predictions and direct attention; the serial path is checked on the same steps."""
    cfg, pc, st, li = _setup(name, npages, mode=mode)
    st.build_meta()
    meta = S.oracle_meta(li, pc)
    k64, v64 = li.k64(), li.v64()
    _, qb = W.query_trajectory(cfg, 0, steps=steps)
    forced = list(pc.forced)
    st.select(S.q_tensor(qb[0], pc))
    st.predict()
    st.advance()
    s0 = S.oracle_scores(W.bits_to_f64(qb[0], cfg.dtype), meta, pc)
    level, trend = O.ema_init(s0)
    hits = []
    for t in range(1, steps + 1):
        S.log(f"step {name} t={t} mode={mode}")
        q = S.q_tensor(qb[t], pc)
        q64 = W.bits_to_f64(qb[t], cfg.dtype)
        pred64 = O.ema_predict(level, trend, cfg.gamma)
        P = S.check_selection(S.lists(st, st.cur), pred64, pc.k_select, forced, pc.forced_in_budget, what="P")
        st.select(q)
        st.speculate(q)
        st.repair(q)
        torch.cuda.synchronize()
        s64 = S.oracle_scores(q64, meta, pc)
        A = S.check_selection(S.lists(st), s64, pc.k_select, forced, pc.forced_in_budget)
        target = A if mode == 0 else [np.union1d(a, p) for a, p in zip(A, P)]
        ref = O.attend(q64, k64, v64, target, pc.page_size, pc.num_tokens)
        S.check_attention(S.to_np(st.out_o32), S.to_np(st.out_m), S.to_np(st.out_l), ref, S.to_np(st.out_o), dtype=pc.dtype)
        hits.append(np.mean([O.hit_rate(a, p) for a, p in zip(A, P)]))
        if mode == 0:
            st.repair(q, serial=True)
            torch.cuda.synchronize()
            S.check_attention(S.to_np(st.out_o32), S.to_np(st.out_m), S.to_np(st.out_l),
                              O.attend(q64, k64, v64, A, pc.page_size, pc.num_tokens), S.to_np(st.out_o),
                              what="serial", dtype=pc.dtype)
        st.predict()
        st.advance()
        level, trend = O.ema_update(level, trend, s64, cfg.alpha, cfg.beta)
    S.log(f"{name}: mean hit rate {np.mean(hits):.3f}")


def test_two_stream_step_and_determinism(torch):
    """The two-stream fork/join step gives the single-stream result, bit for bit, twice."""
    from paper_2606_30389_amd import runtime as R
    cfg, pc, st, li = _setup("glm32k", None)
    st.build_meta()
    _, qb = W.query_trajectory(cfg, 0, steps=2)
    st.select(S.q_tensor(qb[0], pc))
    st.predict()
    st.advance()
    q = S.q_tensor(qb[1], pc)
    ts = R.TwoStream(torch.device("cuda:0"))
    outs = []
    for rep in range(2):
        S.log(f"two-stream rep {rep}")
        torch.cuda.synchronize()
        ts.s.wait_stream(torch.cuda.current_stream())
        done = ts.prr_layer(st, q)
        ts.join([done])
        torch.cuda.synchronize()
        outs.append((st.out_o32.clone(), st.out_m.clone(), st.out_l.clone(), st.pred[1 - st.cur].clone()))
        # undo the EMA update so the second repetition starts from the same state
        st.level.zero_()
        st.trend.zero_()
        st.init_bits.zero_()
        st.select(S.q_tensor(qb[0], pc))
        st.predict()
        torch.cuda.synchronize()
    for a, b in zip(outs[0], outs[1]):
        assert torch.equal(a, b)
    st.select(q)
    st.speculate(q)
    st.repair(q)
    torch.cuda.synchronize()
    assert torch.equal(st.out_o32, outs[0][0])


def test_merge_states(torch):
    rng = np.random.default_rng(0)
    ns, rows, d = 5, 7, 96
    o = rng.standard_normal((ns, rows, d))
    m = rng.standard_normal((ns, rows)) * 3
    l = np.exp(rng.standard_normal((ns, rows)))
    l[2, 3] = 0.0  # an empty state
    m[2, 3] = -np.inf
    dev = torch.device("cuda:0")
    tt = lambda x: torch.tensor(x, dtype=torch.float32, device=dev)  # noqa: E731
    out_o, out_m, out_l = torch.zeros(rows, d, device=dev), torch.zeros(rows, device=dev), torch.zeros(rows, device=dev)
    import paper_2606_30389_amd as P
    S.log("merge_states")
    P.prr_merge_states(ns, rows, d, tt(o), tt(m), tt(l), out_o, out_m, out_l)
    torch.cuda.synchronize()
    ref = O.merge_states([(o[s].astype(np.float32).astype(np.float64), m[s].astype(np.float32).astype(np.float64),
                           l[s].astype(np.float32).astype(np.float64)) for s in range(ns)])
    assert np.abs(S.to_np(out_o) - ref[0]).max() < 1e-5
    assert np.abs(S.to_np(out_m) - ref[1]).max() < 1e-6
    assert np.allclose(S.to_np(out_l), ref[2], rtol=1e-5)


@pytest.mark.parametrize("sync", ["events", "memory"])
@pytest.mark.parametrize("name,npages,mode", [("glm32k", 512, 0), ("llama64k", 300, 1), ("infllm128k", 200, 0)])
def test_native_decode_step(torch, name, npages, mode, sync):
    """prr_decode_step over a stack of layers: step 0 (select + EMA init), then the
    two-stream PRR schedule (its streams ordered by the caller's events, or by the library's
    stream-memory words) and the serial schedule, every layer against the oracle."""
    from paper_2606_30389_amd import _lib as L
    from paper_2606_30389_amd import runtime as R
    cfg = W.CONFIGS[name]
    n_layers, steps = 3, 3
    layers, inputs, metas, qs, queries = [], [], [], [], []
    for layer in range(n_layers):
        pc = S.path_config(cfg, num_pages=npages, mode=mode)
        S.log(f"native step {name} layer {layer} pages={npages} mode={mode}")
        st, li = S.make_layer(cfg, pc, layer=layer)
        st.build_meta()
        layers.append(st)
        inputs.append(li)
        metas.append(S.oracle_meta(li, pc))
        _, qb = W.query_trajectory(cfg, layer, steps=steps)
        qs.append(qb)
        queries.append(S.q_tensor(qb[0], pc))
    pc = layers[0].cfg
    stack = R.DecodeStack(layers, queries, torch.device("cuda:0"))
    stack.two_stream_events = sync == "events"
    s, p = torch.cuda.Stream(), torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    stack.step(L.PRR_SCHED_PREFILL, s)
    torch.cuda.synchronize()
    forced = list(pc.forced)
    state = []
    for layer in range(n_layers):
        s64 = S.oracle_scores(W.bits_to_f64(qs[layer][0], cfg.dtype), metas[layer], pc)
        state.append(O.ema_init(s64))
    for t in range(1, steps + 1):
        for layer in range(n_layers):
            queries[layer].copy_(S.q_tensor(qs[layer][t], pc))
        torch.cuda.synchronize()
        preds = [S.lists(st, st.cur) for st in layers]
        S.log(f"native two-stream step {t} ({sync})")
        s.wait_stream(torch.cuda.current_stream())
        stack.step(L.PRR_SCHED_TWO_STREAM, s, p)
        torch.cuda.synchronize()
        for layer, st in enumerate(layers):
            q64 = W.bits_to_f64(qs[layer][t], cfg.dtype)
            level, trend = state[layer]
            P = S.check_selection(preds[layer], O.ema_predict(level, trend, cfg.gamma), pc.k_select, forced,
                                  pc.forced_in_budget, what="P")
            s64 = S.oracle_scores(q64, metas[layer], pc)
            A = S.check_selection(S.lists(st), s64, pc.k_select, forced, pc.forced_in_budget)
            target = A if mode == 0 else [np.union1d(a, b) for a, b in zip(A, P)]
            ref = O.attend(q64, inputs[layer].k64(), inputs[layer].v64(), target, pc.page_size, pc.num_tokens)
            S.check_attention(S.to_np(st.out_o32), S.to_np(st.out_m), S.to_np(st.out_l), ref, S.to_np(st.out_o),
                              dtype=pc.dtype, what=f"layer {layer}")
            state[layer] = O.ema_update(level, trend, s64, cfg.alpha, cfg.beta)
        S.log(f"native serial step {t}")
        stack.step(L.PRR_SCHED_SERIAL, s)
        torch.cuda.synchronize()
        for layer, st in enumerate(layers):
            q64 = W.bits_to_f64(qs[layer][t], cfg.dtype)
            A = S.check_selection(S.lists(st), S.oracle_scores(q64, metas[layer], pc), pc.k_select, forced,
                                  pc.forced_in_budget)
            ref = O.attend(q64, inputs[layer].k64(), inputs[layer].v64(), A, pc.page_size, pc.num_tokens)
            S.check_attention(S.to_np(st.out_o32), S.to_np(st.out_m), S.to_np(st.out_l), ref, S.to_np(st.out_o),
                              dtype=pc.dtype, what=f"serial layer {layer}")


FUSED_CASES = [
    # name, pages, mode, chunk, |P|/|A|, k_select override, layers, steps
    ("tiny", None, 0, None, 1, None, 2, 4),
    ("tiny", None, 1, None, 1, None, 1, 3),
    ("tiny", None, 0, 3, 1, 6, 1, 4),        # |A| <= 8: the select workgroup attends itself
    ("glm32k", 512, 0, 16, 1, None, 2, 3),   # two pages per wave
    ("glm32k", 512, 0, 8, 2, None, 1, 3),    # |P| = 2|A|
    ("llama64k", 300, 1, None, 1, None, 2, 3),
    ("infllm128k", 200, 0, None, 1, None, 1, 3),
    ("glm128k", None, 0, None, 1, None, 1, 2),  # full size: 8192 pages, top-256
    ("glm128k", None, 0, 4, 1, None, 1, 2),     # full size at chunk 4 (the serial baseline's)
    # ablation stages: theta = (1, 0.5, 0) predicts the previous step's top-K; with a
    # recompute on any miss (S1) and with repair (S2)
    ("glm32k", 512, 2, None, 1, None, 1, 3, (1.0, 0.5, 0.0)),
    ("glm32k", 512, 0, None, 1, None, 1, 3, (1.0, 0.5, 0.0)),
    ("tiny", None, 2, None, 1, 6, 1, 4, (1.0, 0.5, 0.0)),
    # late speculation over the pages just above the threshold that P missed
    ("glm32k", 512, 0, None, 1, None, 2, 4, None, True),
    ("glm128k", None, 0, None, 1, None, 1, 4, None, True),
    ("llama64k", 300, 1, None, 1, None, 1, 3, None, True),
    ("infllm128k", 200, 0, None, 1, None, 1, 3, None, True),
    ("tiny", None, 0, 3, 1, 6, 1, 4, None, True),
    # scores in 12 tied groups of ~43 pages: the threshold falls inside a group, so the
    # select ranks a small bin of equal keys and cuts the tie by page index
    ("glm32k", 512, 0, None, 1, None, 1, 3, None, False, 12),
    ("glm32k", 512, 0, None, 1, None, 1, 3, None, True, 12),
]


@pytest.mark.parametrize("case", FUSED_CASES,
                         ids=lambda c: f"{c[0]}-p{c[1]}-m{c[2]}-c{c[3]}-d{c[4]}-k{c[5]}"
                         + ("-reuse" if len(c) > 8 and c[8] is not None else "")
                         + ("-late" if len(c) > 9 and c[9] else "")
                         + (f"-lv{c[10]}" if len(c) > 10 else ""))
def test_fused_decode_step(torch, case):
    """The fused schedules of prr_decode_step (one launch per layer): step-0 select + EMA
    initialisation, then per step the PRR launch and the serial launch, every layer
    against the oracle (A, P, output, missed and wasted counts)."""
    from paper_2606_30389_amd import _lib as L
    from paper_2606_30389_amd import runtime as R
    name, npages, mode, chunk, delta, kover, n_layers, steps = case[:8]
    cfg = W.CONFIGS[name]
    theta = case[8] if len(case) > 8 and case[8] is not None else (cfg.alpha, cfg.beta, cfg.gamma)
    late = bool(case[9]) if len(case) > 9 else False
    levels = case[10] if len(case) > 10 else None
    layers, inputs, metas, qs, queries = [], [], [], [], []
    for layer in range(n_layers):
        pc = S.path_config(cfg, num_pages=npages, mode=mode, chunk_pages=chunk)
        if kover is not None:
            pc.k_select = kover
        pc.p_select = delta * pc.k_select
        pc.alpha, pc.beta, pc.gamma = theta
        S.log(f"fused {name} layer {layer} pages={pc.num_pages} mode={mode} chunk={pc.chunk_pages} "
              f"K={pc.k_select} |P|={pc.p_select}")
        st, li = S.make_layer(cfg, pc, layer=layer, levels=levels)
        st.build_meta()
        layers.append(st)
        inputs.append(li)
        metas.append(S.oracle_meta(li, pc))
        _, qb = W.query_trajectory(cfg, layer, steps=steps)
        qs.append(qb)
        queries.append(S.q_tensor(qb[0], pc))
    pc = layers[0].cfg
    forced = list(pc.forced)
    stack = R.DecodeStack(layers, queries, torch.device("cuda:0"))
    stack.params.late_spec = int(late)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    stack.step(L.PRR_SCHED_FUSED_PREFILL, s)
    torch.cuda.synchronize()
    state = []
    for layer, st in enumerate(layers):
        s64 = S.oracle_scores(W.bits_to_f64(qs[layer][0], cfg.dtype), metas[layer], pc)
        S.check_selection(S.lists(st), s64, pc.k_select, forced, pc.forced_in_budget, what="A0")
        state.append(O.ema_init(s64))
    for t in range(1, steps + 1):
        for layer in range(n_layers):
            queries[layer].copy_(S.q_tensor(qs[layer][t], pc))
        torch.cuda.synchronize()
        preds = [S.lists(st, st.cur) for st in layers]
        S.log(f"fused PRR step {t}")
        s.wait_stream(torch.cuda.current_stream())
        stack.step(L.PRR_SCHED_FUSED_PRR, s)
        torch.cuda.synchronize()
        for layer, st in enumerate(layers):
            q64 = W.bits_to_f64(qs[layer][t], cfg.dtype)
            level, trend = state[layer]
            P = S.check_selection(preds[layer], O.ema_predict(level, trend, theta[2]), pc.p_select, forced,
                                  pc.forced_in_budget, what="P")
            s64 = S.oracle_scores(q64, metas[layer], pc)
            A = S.check_selection(S.lists(st), s64, pc.k_select, forced, pc.forced_in_budget)
            target = A if mode != 1 else [np.union1d(x, y) for x, y in zip(A, P)]
            ref = O.attend(q64, inputs[layer].k64(), inputs[layer].v64(), target, pc.page_size, pc.num_tokens)
            S.check_attention(S.to_np(st.out_o32), S.to_np(st.out_m), S.to_np(st.out_l), ref, S.to_np(st.out_o),
                              dtype=pc.dtype, what=f"PRR layer {layer} step {t}")
            mc, wc = S.to_np(st.missed), S.to_np(st.wasted)
            for h in range(pc.num_kv_heads):
                mm, ww = O.missed_and_wasted(A[h], P[h])
                assert (mc[h], wc[h]) == (len(mm), len(ww)), f"layer {layer} head {h}: missed/wasted counts"
            state[layer] = O.ema_update(level, trend, s64, theta[0], theta[1])
        S.log(f"fused serial step {t}")
        stack.step(L.PRR_SCHED_FUSED_SERIAL, s)
        torch.cuda.synchronize()
        for layer, st in enumerate(layers):
            q64 = W.bits_to_f64(qs[layer][t], cfg.dtype)
            A = S.check_selection(S.lists(st), S.oracle_scores(q64, metas[layer], pc), pc.k_select, forced,
                                  pc.forced_in_budget)
            ref = O.attend(q64, inputs[layer].k64(), inputs[layer].v64(), A, pc.page_size, pc.num_tokens)
            S.check_attention(S.to_np(st.out_o32), S.to_np(st.out_m), S.to_np(st.out_l), ref, S.to_np(st.out_o),
                              dtype=pc.dtype, what=f"serial layer {layer} step {t}")
    for st in layers:
        fl = int(st.workspace[:4].view(torch.int32).cpu()[0])
        assert fl == 0, f"workspace error flags {fl:#x}"


@pytest.mark.parametrize("late", [False, True], ids=["spec", "late"])
def test_fused_graph_replay(torch, late):
    """Fused PRR steps captured once as HIP graphs (the launches read a device epoch word
    that each replay advances) and replayed with eager work and synchronisations in
    between: every replay equals the eager launch of the same step on a twin stack bit for
    bit, and the oracle."""
    from paper_2606_30389_amd import _lib as L
    from paper_2606_30389_amd import runtime as R
    cfg = W.CONFIGS["glm32k"]
    n_layers, steps = 2, 5
    stacks, inputs, metas, qs, queries = [], [], [[], []], [], [[], []]
    for twin in range(2):
        layers = []
        for layer in range(n_layers):
            pc = S.path_config(cfg, num_pages=512, mode=0)
            st, li = S.make_layer(cfg, pc, layer=layer)
            st.build_meta()
            layers.append(st)
            if twin == 0:
                inputs.append(li)
                metas[0].append(S.oracle_meta(li, pc))
                _, qb = W.query_trajectory(cfg, layer, steps=steps)
                qs.append(qb)
            queries[twin].append(S.q_tensor(qs[layer][0], pc))
        stack = R.DecodeStack(layers, queries[twin], torch.device("cuda:0"))
        stack.params.late_spec = int(late)
        stacks.append(stack)
    pc = stacks[0].layers[0].cfg
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    for stack in stacks:
        stack.step(L.PRR_SCHED_FUSED_PREFILL, s)
    torch.cuda.synchronize()
    S.log(f"capturing fused PRR graphs (late={late})")
    stacks[1].capture(L.PRR_SCHED_FUSED_PRR, s)
    torch.cuda.synchronize()
    for t in range(1, steps + 1):
        for twin in range(2):
            for layer in range(n_layers):
                queries[twin][layer].copy_(S.q_tensor(qs[layer][t], pc))
        torch.cuda.synchronize()
        S.log(f"graph replay step {t}")
        s.wait_stream(torch.cuda.current_stream())
        stacks[0].step(L.PRR_SCHED_FUSED_PRR, s)
        torch.cuda.synchronize()
        junk = torch.randn(1 << 16, device="cuda:0").sum().item()  # eager work between replays
        assert junk == junk
        s.wait_stream(torch.cuda.current_stream())
        stacks[1].replay(L.PRR_SCHED_FUSED_PRR, s)
        torch.cuda.synchronize()
        for layer in range(n_layers):
            a, b = stacks[0].layers[layer], stacks[1].layers[layer]
            for name in ("out_o32", "out_m", "out_l", "out_o", "sel", "sel_count", "missed", "wasted"):
                x, y = getattr(a, name), getattr(b, name)
                assert torch.equal(x.view(torch.uint8), y.view(torch.uint8)) if x.dtype.is_floating_point else \
                    torch.equal(x, y), f"step {t} layer {layer}: {name} differs between eager and graph replay"
            assert torch.equal(a.pred[a.cur], b.pred[b.cur]) and torch.equal(a.pred_count[a.cur], b.pred_count[b.cur]), \
                f"step {t} layer {layer}: next prediction"
            q64 = W.bits_to_f64(qs[layer][t], cfg.dtype)
            A = S.check_selection(S.lists(b), S.oracle_scores(q64, metas[0][layer], pc), pc.k_select, list(pc.forced),
                                  pc.forced_in_budget)
            ref = O.attend(q64, inputs[layer].k64(), inputs[layer].v64(), A, pc.page_size, pc.num_tokens)
            S.check_attention(S.to_np(b.out_o32), S.to_np(b.out_m), S.to_np(b.out_l), ref, S.to_np(b.out_o),
                              dtype=pc.dtype, what=f"graph layer {layer} step {t}")
    for stack in stacks:
        for st in stack.layers:
            fl = int(st.workspace[:4].view(torch.int32).cpu()[0])
            assert fl == 0, f"workspace error flags {fl:#x}"
