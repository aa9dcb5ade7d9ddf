"""Shared helpers of the GPU parity tests: set up a layer from a seeded workload, run
the library's calls, and compare with the oracle (near-tie rule, tolerances)."""
from __future__ import annotations

import math
import sys

import numpy as np

import oracle as O
import workloads as W

# Judged bound on attention outputs (fp16/bf16 inputs, fp32 accumulation) and the
# stricter internal bounds used on every parity case.
O_JUDGED = 2e-3
O_INTERNAL = 1e-4
M_REL = 1e-5
L_REL = 1e-4
NEAR_TIE_REL = 1e-5


def log(*a):
    print("[gpu-test]", *a, flush=True)
    sys.stdout.flush()


def torch_and_lib():
    import torch
    import paper_2606_30389_amd as P
    from paper_2606_30389_amd import runtime as R
    return torch, P, R


def path_config(cfg: W.Config, num_pages=None, chunk_pages=None, mode=0, num_tokens=None):
    _, P, R = torch_and_lib()
    if chunk_pages is None:
        chunk_pages = max(1, 128 // cfg.page_size)  # (128 tokens per attending workgroup, as the bench runs it)
    n = cfg.num_pages if num_pages is None else num_pages
    nt = n * cfg.page_size if num_tokens is None else num_tokens
    return R.PathConfig(num_q_heads=cfg.num_q_heads, num_kv_heads=cfg.num_kv_heads, page_size=cfg.page_size,
                        num_tokens=nt, k_select=cfg.k_select, forced=cfg.forced_pages(n),
                        forced_in_budget=cfg.forced_in_budget, dtype=cfg.dtype, meta_kind=cfg.meta_kind,
                        alpha=cfg.alpha, beta=cfg.beta, gamma=cfg.gamma, chunk_pages=chunk_pages, mode=mode)


def make_layer(cfg: W.Config, pc, layer=0, epoch=0, page_table=None, num_physical=None, levels=None):
    """Upload one layer's keys and values; returns (LayerState, LayerInputs).  levels: page p
    takes the keys of page p mod levels, so that scores come in `levels` tied groups."""
    torch, P, R = torch_and_lib()
    li = W.layer_inputs(cfg, layer, epoch, num_pages=pc.num_pages)
    if levels:
        li.k_bits[:] = li.k_bits[:, np.arange(li.k_bits.shape[1]) % levels]
    dev = torch.device("cuda:0")
    if page_table is not None:
        kb = W.to_physical(li.k_bits, page_table, num_physical)
        vb = W.to_physical(li.v_bits, page_table, num_physical)
        pc.max_pages = num_physical
        ptab = torch.from_numpy(page_table.astype(np.int32)).to(dev)
    else:
        kb, vb, ptab = li.k_bits, li.v_bits, None
    k = R.bits_tensor(kb, pc.torch_dtype, dev)
    v = R.bits_tensor(vb, pc.torch_dtype, dev)
    st = R.LayerState(pc, dev, k=k, v=v, page_table=ptab)
    return st, li


def q_tensor(qbits, pc):
    torch, _, R = torch_and_lib()
    return R.bits_tensor(qbits, pc.torch_dtype, torch.device("cuda:0"))


def oracle_meta(li, pc):
    k = li.k64()
    if pc.meta_kind == "mean":
        return O.page_metadata_mean(k, pc.page_size, pc.num_tokens)
    return O.page_metadata_minmax(k, pc.page_size, pc.num_tokens)


def oracle_scores(q64, meta, pc):
    qbar = O.representative_query(q64, pc.num_kv_heads)
    if pc.meta_kind == "mean":
        return O.criticality_mean(qbar, meta)
    return O.criticality_minmax(qbar, *meta)


def check_selection(got_lists, scores64, k, forced, fib, what="A"):
    """Compare per-head selections with the oracle's under the near-tie rule.
    Returns the selection to use for downstream comparisons (the GPU's, once validated)."""
    out = []
    for h, got in enumerate(got_lists):
        want = O.select_topk(scores64[h], k, forced, fib)
        got = np.sort(np.asarray(got, dtype=np.int64))
        assert len(got) == len(want), f"{what}[{h}]: size {len(got)} != {len(want)}"
        assert len(set(got.tolist())) == len(got), f"{what}[{h}] has duplicates"
        diff = set(got.tolist()) ^ set(want.tolist())
        if diff:
            keys = O.decision_keys(scores64[h]).astype(np.float64)
            cand = [p for p in range(len(keys)) if p not in set(forced)]
            extra = max(0, k - len(forced)) if fib else k
            kth = sorted((keys[p] for p in cand), reverse=True)[extra - 1]
            for p in diff:
                assert abs(scores64[h][p] - kth) <= NEAR_TIE_REL * abs(kth) + 1e-30, (
                    f"{what}[{h}]: page {p} (score {scores64[h][p]!r}) differs and is not a near-tie of "
                    f"the threshold {kth!r}")
            log(f"{what}[{h}]: {len(diff)} near-tie difference(s) excused")
        out.append(got)
    return out


def dtype_ulp(x, dtype):
    """Spacing of the 16-bit format at |x| (normal range)."""
    mant = 7 if dtype == "bf16" else 10
    e = np.floor(np.log2(np.maximum(np.abs(x), 2.0 ** -14)))
    return 2.0 ** (e - mant)


def check_attention(o32, m, l, ref, o_dtype=None, tol=O_INTERNAL, what="out", dtype=None):
    """fp32 output within `tol` (<= the judged 2e-3) of the fp64 reference; the 16-bit
    output is the round-to-nearest-even of the fp32 output (bit-exact) and so within one
    unit in the last place of the reference (its own rounding dominates any 2e-3 bound
    once |o| > 0.5 in bfloat16)."""
    o_ref, m_ref, l_ref = ref
    assert tol <= O_JUDGED
    err = np.abs(o32 - o_ref).max() if o32.size else 0.0
    log(f"{what}: max |o - o_ref| = {err:.2e}")
    assert err <= tol, f"{what}: max |o - o_ref| = {err:.3e} > {tol:.1e}"
    if o_dtype is not None and o_dtype.size:
        assert dtype in ("bf16", "f16"), "pass the 16-bit output's dtype"
        dt = dtype
        rne = W.bits_to_f64(W.f32_to_dtype_bits(o32.astype(np.float32), dt), dt)
        assert np.array_equal(rne, o_dtype), f"{what}: 16-bit output is not the rounded fp32 output"
        assert np.all(np.abs(o_dtype - o_ref) <= dtype_ulp(o_ref, dt)), f"{what}: 16-bit output off by > 1 ulp"
    fin = np.isfinite(m_ref)
    assert np.array_equal(np.isfinite(m), fin), f"{what}: empty rows differ"
    if fin.any():
        em = np.abs(m[fin] - m_ref[fin]) / np.maximum(np.abs(m_ref[fin]), 1.0)
        el = np.abs(l[fin] - l_ref[fin]) / np.abs(l_ref[fin])
        assert em.max() <= M_REL, f"{what}: m rel err {em.max():.3e}"
        assert el.max() <= L_REL, f"{what}: l rel err {el.max():.3e}"
    assert np.all(l[~fin] == 0) and np.all(o32[~fin] == 0), f"{what}: empty rows not (0, -inf, 0)"
    return err


def to_np(t):
    import torch
    if t.dtype in (torch.bfloat16, torch.float16):
        return t.float().cpu().numpy().astype(np.float64)
    return t.cpu().numpy()


def lists(st, which="sel"):
    if which == "sel":
        cnt, arr = to_np(st.sel_count), to_np(st.sel)
    else:
        cnt, arr = to_np(st.pred_count[which]), to_np(st.pred[which])
    return [arr[h, :cnt[h]] for h in range(len(cnt))]


def dense_ok(x):
    return np.all(np.isfinite(x))


def hkv_of(pc):
    return pc.num_kv_heads


def rel_err(a, b):
    return np.abs(a - b).max() / max(1.0, np.abs(b).max())


def sqrtd():
    return math.sqrt(128)
