"""Parity of the fused one-launch step (the measured path) with the fp64 oracle, on the GPU,
at the workloads' full sizes: selections A and P, the EMA state (level and trend), the
output, and the missed / wasted counts, every step.

Cases cover what the launch learns or reads across steps and what a real cache holds:
paged layouts (a permuted page table), a partial last page whose unwritten tail holds NaN
and Inf, the select workgroup's fallback paths (forced by re-zeroing the workspace, which
resets the candidate windows learned from earlier steps), long runs, and the Llama-shaped
workload's drifting hot set with the touched pages' metadata rebuilt between steps.
"""
import dataclasses

import numpy as np
import pytest

import oracle as O
import workloads as W
from tests import gpu_support as S

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch as _t
    assert _t.cuda.is_available(), "no GPU visible"
    import paper_2606_30389_amd  # noqa: F401  (fails loudly when libprr.so is missing)
    return _t


@dataclasses.dataclass
class Case:
    name: str
    npages: int = None          # pages per KV head (None = the workload's)
    tail: int = 0               # tokens missing from the last page
    mode: int = 0
    chunk: int = None
    delta: float = 1.0
    layers: int = 1
    steps: int = 4
    late: bool = False
    nora: bool = False          # late speculation without the read-ahead (late_spec 2)
    page_table: bool = False
    nan_tail: bool = False
    reinit: tuple = ()          # steps before which the workspace is zeroed again
    drift: bool = False
    serial: bool = True         # also run the fused serial step after each PRR step
    thetas: tuple = ()          # per-layer (alpha, beta, gamma) in place of the workload's

    def id(self):
        bits = [self.name, f"p{self.npages}" if self.npages else "full", f"m{self.mode}", f"s{self.steps}"]
        for flag in ("late", "nora", "page_table", "nan_tail", "drift"):
            if getattr(self, flag):
                bits.append(flag)
        if self.tail:
            bits.append(f"tail{self.tail}")
        if self.chunk:
            bits.append(f"c{self.chunk}")
        if self.delta != 1.0:
            bits.append(f"d{self.delta}")
        if self.reinit:
            bits.append("reinit" + "-".join(map(str, self.reinit)))
        if self.thetas:
            bits.append(f"theta{self.layers}l")
        return "_".join(bits)


CASES = [
    # the workloads at full size, with and without late speculation
    Case("glm32k", steps=4), Case("glm32k", steps=4, late=True), Case("glm32k", steps=4, late=True, nora=True),
    Case("llama64k", steps=3), Case("llama64k", steps=3, late=True), Case("llama64k", mode=1, steps=2, late=True),
    Case("infllm128k", steps=4), Case("infllm128k", steps=4, late=True),
    # paged layout and a partial last page whose unwritten tail holds NaN / Inf
    Case("glm32k", page_table=True, late=True, steps=3),
    Case("glm32k", tail=5, nan_tail=True, late=True, steps=3),
    Case("glm32k", page_table=True, tail=11, nan_tail=True, steps=3, chunk=16),
    Case("infllm128k", page_table=True, tail=37, nan_tail=True, late=True, steps=3),
    Case("infllm128k", chunk=4, late=True, steps=3),
    Case("glm128k", page_table=True, tail=3, nan_tail=True, late=True, steps=2),
    # the select's fallback paths in PRR steps: all 2048 pages of glm32k become candidates
    # (the one-workgroup middle path), all 4096 / 8192 of llama64k / glm128k (full gather)
    Case("glm32k", reinit=(2, 3), late=True, steps=4),
    Case("llama64k", reinit=(2,), late=True, steps=3),
    Case("glm128k", reinit=(2,), steps=3, late=True),
    # the other output modes at full size: attention over P u A, and recomputation of A on any miss
    Case("glm128k", mode=1, steps=3, late=True), Case("glm128k", mode=2, steps=3),
    Case("infllm128k", mode=1, steps=3, late=True),
    # long runs: candidate windows and the late bound are learned across steps
    Case("glm128k", steps=12, late=True, serial=False),
    Case("glm32k", steps=64, late=True, serial=False),
    Case("glm32k", steps=24, delta=1.5, late=True, serial=False),
    # the Llama-shaped workload's hot set re-drawn every 16 steps
    Case("llama64k", steps=20, drift=True, late=True, serial=False),
    # a calibrated (alpha, beta, gamma) per layer (Section 4.2), two layers that differ
    # (values exact in float32, so that both sides rank the same predictions)
    Case("glm32k", layers=2, steps=6, late=True, serial=False, thetas=((0.75, 0.375, 0.75), (0.25, 0.125, 0.5))),
]


def _poison_tail(torch, st, pc, li, ptab):
    """NaN / Inf in K and V of the tokens past num_tokens on the last page (as an unwritten
    cache tail may hold)."""
    last = pc.num_pages - 1
    phys = int(ptab[last]) if ptab is not None else last
    valid = pc.num_tokens - last * pc.page_size
    with torch.no_grad():
        st.v[:, phys, valid:] = float("nan")
        st.k[:, phys, valid:] = float("inf")
        st.k[:, phys, valid::2] = float("nan")


def _upload_kv(torch, st, pc, li, ptab, num_physical):
    from paper_2606_30389_amd import runtime as R
    dev = torch.device("cuda:0")
    kb, vb = li.k_bits, li.v_bits
    if ptab is not None:
        kb, vb = W.to_physical(kb, ptab, num_physical), W.to_physical(vb, ptab, num_physical)
    st.k.copy_(R.bits_tensor(kb, pc.torch_dtype, dev))
    st.v.copy_(R.bits_tensor(vb, pc.torch_dtype, dev))


def _check_state(st, level, trend, pc, what):
    n = pc.num_pages
    got_l, got_v = S.to_np(st.level)[:, :n], S.to_np(st.trend)[:, :n]
    scale = max(1.0, float(np.abs(level).max()))
    el = np.abs(got_l - level).max() / scale
    ev = np.abs(got_v - trend).max() / scale
    assert el <= 1e-5 and ev <= 1e-5, f"{what}: EMA level err {el:.2e}, trend err {ev:.2e} (relative to {scale:.3g})"


@pytest.mark.parametrize("case", CASES, ids=lambda c: c.id())
def test_fused_full_size(torch, case):
    from paper_2606_30389_amd import _lib as L
    from paper_2606_30389_amd import runtime as R
    cfg = W.CONFIGS[case.name]
    n = case.npages or cfg.num_pages
    nt = n * cfg.page_size - case.tail
    layers, inputs, metas, qs, queries, ptabs, kv64 = [], [], [], [], [], [], []
    for layer in range(case.layers):
        pc = S.path_config(cfg, num_pages=n, mode=case.mode, chunk_pages=case.chunk, num_tokens=nt)
        pc.p_select = int(round(case.delta * pc.k_select))
        S.log(f"fused {case.id()} layer {layer}: pages={pc.num_pages} tokens={nt} K={pc.k_select} "
              f"|P|={pc.p_select} chunk={pc.chunk_pages}")
        ptab = W.page_table_permutation(n, n + 37, seed=11 + layer) if case.page_table else None
        st, li = S.make_layer(cfg, pc, layer=layer, page_table=ptab, num_physical=n + 37 if case.page_table else None)
        if case.nan_tail:
            _poison_tail(torch, st, pc, li, ptab)
        st.build_meta()
        layers.append(st)
        inputs.append(li)
        ptabs.append(ptab)
        metas.append(S.oracle_meta(li, pc))
        kv64.append((li.k64(), li.v64()))
        _, qb = W.query_trajectory(cfg, layer, steps=case.steps)
        qs.append(qb)
        queries.append(S.q_tensor(qb[0], pc))
    pc = layers[0].cfg
    forced = list(pc.forced)
    stack = R.DecodeStack(layers, queries, torch.device("cuda:0"))
    stack.params.late_spec = (2 if case.nora else 1) if case.late else 0
    thetas = list(case.thetas) if case.thetas else [(pc.alpha, pc.beta, pc.gamma)] * case.layers
    if case.thetas:
        stack.set_layer_theta(case.thetas)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    stack.step(L.PRR_SCHED_FUSED_PREFILL, s)
    torch.cuda.synchronize()
    state = []
    for layer, st in enumerate(layers):
        s64 = S.oracle_scores(W.bits_to_f64(qs[layer][0], cfg.dtype), metas[layer], pc)
        S.check_selection(S.lists(st), s64, pc.k_select, forced, pc.forced_in_budget, what="A0")
        state.append(O.ema_init(s64))
        _check_state(st, *state[-1], pc, f"layer {layer} step 0")
    epoch = 0
    for t in range(1, case.steps + 1):
        if case.drift and cfg.drift_every and t % cfg.drift_every == 0:
            epoch = t // cfg.drift_every
            for layer, st in enumerate(layers):
                old = inputs[layer].hot
                li = W.layer_inputs(cfg, layer, epoch, num_pages=n)
                touched = np.unique(np.concatenate([old.ravel(), li.hot.ravel()]))
                S.log(f"drift epoch {epoch} layer {layer}: {len(touched)} pages rewritten and re-described")
                _upload_kv(torch, st, pc, li, ptabs[layer], st.dims.max_pages)
                for p in touched:
                    st.build_meta(page_begin=int(p), page_end=int(p) + 1)
                inputs[layer] = li
                metas[layer] = S.oracle_meta(li, pc)
                kv64[layer] = (li.k64(), li.v64())
            torch.cuda.synchronize()
        if t in case.reinit:
            S.log(f"workspace zeroed before step {t} (candidate windows reset)")
            for st in layers:
                L.prr_workspace_init(st.workspace, st.ws_bytes)
        for layer in range(case.layers):
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
            al, be, ga = thetas[layer]
            P = S.check_selection(preds[layer], O.ema_predict(level, trend, ga), pc.p_select, forced,
                                  pc.forced_in_budget, what=f"P step {t}")
            s64 = S.oracle_scores(q64, metas[layer], pc)
            got_s = S.to_np(st.scores)[:, :n]
            assert np.all(np.abs(got_s - s64) <= 1e-5 * np.maximum(1.0, np.abs(s64))), f"scores step {t}"
            A = S.check_selection(S.lists(st), s64, pc.k_select, forced, pc.forced_in_budget, what=f"A step {t}")
            target = A if case.mode != 1 else [np.union1d(x, y) for x, y in zip(A, P)]
            ref = O.attend(q64, *kv64[layer], target, pc.page_size, nt)
            S.check_attention(S.to_np(st.out_o32), S.to_np(st.out_m), S.to_np(st.out_l), ref, S.to_np(st.out_o),
                              dtype=pc.dtype, what=f"PRR layer {layer} step {t}")
            mc, wc, cc = S.to_np(st.missed), S.to_np(st.wasted), S.to_np(st.covered)
            for h in range(pc.num_kv_heads):
                mm, ww = O.missed_and_wasted(A[h], P[h])
                assert (mc[h], wc[h]) == (len(mm), len(ww)), f"layer {layer} head {h} step {t}: missed/wasted"
                # pages of A outside P that late speculation attended: none without it
                assert 0 <= cc[h] <= (mc[h] if case.late else 0), f"layer {layer} head {h} step {t}: covered {cc[h]}"
            state[layer] = O.ema_update(level, trend, s64, al, be)
            _check_state(st, *state[layer], pc, f"layer {layer} step {t}")
        if case.serial:
            S.log(f"fused serial step {t}")
            stack.step(L.PRR_SCHED_FUSED_SERIAL, s)
            torch.cuda.synchronize()
            for layer, st in enumerate(layers):
                q64 = W.bits_to_f64(qs[layer][t], cfg.dtype)
                A = S.check_selection(S.lists(st), S.oracle_scores(q64, metas[layer], pc), pc.k_select, forced,
                                      pc.forced_in_budget, what=f"serial A step {t}")
                ref = O.attend(q64, *kv64[layer], A, pc.page_size, nt)
                S.check_attention(S.to_np(st.out_o32), S.to_np(st.out_m), S.to_np(st.out_l), ref, S.to_np(st.out_o),
                                  dtype=pc.dtype, what=f"serial layer {layer} step {t}")
    for st in layers:
        fl = int(st.workspace[:4].view(torch.int32).cpu()[0])
        assert fl == 0, f"workspace error flags {fl:#x}"
