"""The separate kernels at every compiled page (block) size, 16 to 256 tokens, on the
kernel-comparison shape of Section 5.4 (32 query / 8 KV heads, d 128, fp16): page
metadata (min/max and mean), scores + top-K, and speculation + repair over host-chosen
A and P, each against the fp64 oracle, with a ragged last page."""
import dataclasses
import zlib

import numpy as np
import pytest

import oracle as O
import workloads as W
from tests import gpu_support as S

pytestmark = pytest.mark.gpu

SIZES = [16, 32, 64, 128, 256]


@pytest.fixture(scope="module")
def torch():
    import torch as _t
    assert _t.cuda.is_available(), "no GPU visible"
    import paper_2606_30389_amd  # noqa: F401  (fails loudly when libprr.so is missing)
    return _t


def _cfg(ps, meta="minmax"):
    # a 2048-token budget at every page size; hot pages cover about 1300 tokens
    base = W.CONFIGS["llama64k"]
    return dataclasses.replace(base, name=f"kernel_p{ps}", page_size=ps, k_select=2048 // ps, meta_kind=meta,
                               drift_every=0, hot_count=max(2, 1312 // ps))


def _setup(ps, meta="minmax", tail=7):
    cfg = _cfg(ps, meta)
    n = 6144 // ps + 3
    pc = S.path_config(cfg, num_pages=n, num_tokens=n * ps - tail)
    S.log(f"page size {ps}: pages={n} tokens={pc.num_tokens} K={pc.k_select} meta={meta} chunk={pc.chunk_pages}")
    st, li = S.make_layer(cfg, pc)
    return cfg, pc, st, li


@pytest.mark.parametrize("meta", ["minmax", "mean"])
@pytest.mark.parametrize("ps", SIZES)
def test_meta_and_scores(torch, ps, meta):
    cfg, pc, st, li = _setup(ps, meta)
    st.build_meta()
    torch.cuda.synchronize()
    ref = S.oracle_meta(li, pc)
    got = S.to_np(st.meta)[:, :pc.num_pages]
    if meta == "mean":
        assert np.allclose(got, ref, rtol=2e-6, atol=2e-7), np.abs(got - ref).max()
    else:
        assert np.array_equal(got[:, :, 0], ref[0]) and np.array_equal(got[:, :, 1], ref[1])
    _, qb = W.query_trajectory(cfg, 0, steps=2)
    for t in range(3):
        st.select(S.q_tensor(qb[t], pc))
        torch.cuda.synchronize()
        s64 = S.oracle_scores(W.bits_to_f64(qb[t], cfg.dtype), ref, pc)
        got_s = S.to_np(st.scores)[:, :pc.num_pages]
        assert np.all(np.abs(got_s - s64) <= 1e-5 * np.maximum(1.0, np.abs(s64))), np.abs(got_s - s64).max()
        S.check_selection(S.lists(st), s64, pc.k_select, list(pc.forced), pc.forced_in_budget)


def _upload(torch, lists, cap):
    arr = np.full((len(lists), cap), -7, dtype=np.int32)
    cnt = np.zeros(len(lists), dtype=np.int32)
    for h, x in enumerate(lists):
        arr[h, :len(x)] = x
        cnt[h] = len(x)
    return torch.from_numpy(arr).cuda(), torch.from_numpy(cnt).cuda()


# (the serial call has no P, so it runs in the exact mode only)
_SPLITS = [(0, "serial"), (0, "random"), (0, "disjoint"), (1, "random"), (1, "disjoint")]


@pytest.mark.parametrize("mode,split", _SPLITS)
@pytest.mark.parametrize("ps", SIZES)
def test_speculate_repair(torch, ps, mode, split):
    """Attention over exactly A (exact mode) or P u A (keep-wasted mode) after speculating
    over P and repairing; "serial" attends A in one call.  The last page is partial and
    is in A for every head."""
    cfg, pc, st, li = _setup(ps)
    rng = np.random.default_rng(zlib.crc32(f"{ps}/{mode}/{split}".encode()))
    n, ka = pc.num_pages, pc.k_select
    A, P = [], []
    for _ in range(pc.num_kv_heads):
        a = np.sort(np.concatenate([rng.choice(n - 1, ka - 1, replace=False), [n - 1]]))
        rest = np.setdiff1d(np.arange(n), a)
        if split == "disjoint":
            p = np.sort(rng.choice(rest, min(ka, len(rest)), replace=False))
        else:
            keep = a[rng.random(len(a)) < 0.7]
            p = np.sort(np.concatenate([keep, rng.choice(rest, ka - len(keep), replace=False)]))
        A.append(a)
        P.append(p)
    _, qb = W.query_trajectory(cfg, 0, steps=1)
    q = S.q_tensor(qb[1], pc)
    q64 = W.bits_to_f64(qb[1], cfg.dtype)
    a_t, a_c = _upload(torch, A, st.cap)
    st.sel.copy_(a_t)
    st.sel_count.copy_(a_c)
    for buf in (st.out_o32, st.out_m, st.out_l):
        buf.fill_(float("nan"))
    S.log(f"spec+repair page {ps} mode {mode} split {split}")
    if split == "serial":
        st.repair(q, serial=True)
    else:
        p_t, p_c = _upload(torch, P, st.cap)
        st.speculate(q, pages=p_t, counts=p_c)
        st.repair(q, mode=mode, pages=p_t, counts=p_c)
    torch.cuda.synchronize()
    target = A if (mode == 0 or split == "serial") else [np.union1d(a, p) for a, p in zip(A, P)]
    ref = O.attend(q64, li.k64(), li.v64(), target, pc.page_size, pc.num_tokens)
    S.check_attention(S.to_np(st.out_o32), S.to_np(st.out_m), S.to_np(st.out_l), ref, S.to_np(st.out_o),
                      dtype=pc.dtype, what=f"page {ps}")
