"""prr_score_topk_static (the selection entry point that allocates nothing, its scratch a
static device array) against prr_score_topk with a caller-owned workspace, through the C
ABI: two calls in a row, the second on a smaller input, each bit for bit equal to the
workspace call on the same inputs (same kernel), and the selections equal to the oracle's
under the near-tie rule."""
import numpy as np
import pytest

import workloads as W
from tests import gpu_support as S

pytestmark = pytest.mark.gpu


def _run_both(torch, name, npages):
    from paper_2606_30389_amd import _lib as L
    cfg = W.CONFIGS[name]
    pc = S.path_config(cfg, num_pages=npages)
    S.log(f"static-scratch selection {name} pages={pc.num_pages} Hkv={pc.num_kv_heads}")
    st, li = S.make_layer(cfg, pc)
    st.build_meta()
    _, qb = W.query_trajectory(cfg, 0, steps=1)
    q = S.q_tensor(qb[1], pc)
    st.select(q)  # the workspace call
    torch.cuda.synchronize()
    want = (st.scores.clone(), st.sel.clone(), st.sel_count.clone())
    st.scores.fill_(float("nan"))
    st.sel.fill_(-5)
    st.sel_count.fill_(-5)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    L.prr_score_topk_static(st.dims, q, st.meta, pc.num_pages, pc.k_select, pc.forced, pc.forced_in_budget,
                            st.scores, st.sel, st.sel_count, st.cap, s)
    torch.cuda.synchronize()
    assert torch.equal(st.scores.view(torch.int32), want[0].view(torch.int32)), "scores differ"
    assert torch.equal(st.sel_count, want[2]), "selected counts differ"
    for h in range(pc.num_kv_heads):
        n = int(want[2][h])
        assert torch.equal(st.sel[h, :n], want[1][h, :n]), f"head {h}: selected pages differ"
    meta = S.oracle_meta(li, pc)
    ref = S.oracle_scores(W.bits_to_f64(qb[1], cfg.dtype), meta, pc)
    S.check_selection(S.lists(st), ref, pc.k_select, list(pc.forced), pc.forced_in_budget)


def test_static_scratch_selection_twice():
    import torch
    assert torch.cuda.is_available(), "no GPU visible"
    import paper_2606_30389_amd  # noqa: F401
    _run_both(torch, "glm128k", None)    # 2 KV heads x 8192 pages
    _run_both(torch, "glm32k", 300)      # then a smaller input


def test_static_scratch_rejects_too_many_heads():
    from paper_2606_30389_amd import _lib as L
    d = L.make_dims(2 * 300, 300, 16, 64, L.PRR_BF16)
    fake = 0x10000
    with pytest.raises(L.PrrError) as ei:
        L.prr_score_topk_static(d, fake, fake, 64, 8, [], True, fake, fake, fake, 16)
    assert ei.value.status == L.PRR_ERR_INVALID_ARG and "static scratch" in str(ei.value)
