"""The native EMA calibration (Section 4.2, Eqs. (4)-(5)) against the oracle's, on the CPU:
the library's prr_calibrate runs on host cores, so these tests need no GPU."""
from __future__ import annotations

import numpy as np
import pytest

import oracle as O



def _lib():
    try:
        from paper_2606_30389_amd import _lib as L
    except ImportError as e:  # the library is built by __graft_entry__.build()
        pytest.skip(f"libprr not built: {e}")
    return L


def _trajectory(seed, rows, blocks, drift=0.15, growing=0):
    """Positive AR(1)-drifting scores; with `growing`, the last rows gain blocks one by one
    (blocks not formed yet score 0)."""
    rng = np.random.default_rng(seed)
    base = rng.gamma(2.0, 1.0, size=blocks)
    out = np.empty((rows, blocks), dtype=np.float32)
    cur = base.copy()
    for r in range(rows):
        cur = np.abs(cur + drift * rng.normal(size=blocks))
        out[r] = cur
        if growing:
            formed = blocks - growing + min(r, growing)
            out[r, formed:] = 0.0
    return out


@pytest.mark.parametrize("seed,rows,blocks,k,p", [(1, 10, 96, 8, 0), (2, 14, 200, 16, 24), (3, 6, 40, 40, 0),
                                                  (4, 9, 128, 12, 12)])
def test_calibrate_matches_oracle(seed, rows, blocks, k, p):
    L = _lib()
    grid = np.asarray(O.THETA_GRID, dtype=np.float32)
    trajs = np.stack([_trajectory(seed, rows, blocks), _trajectory(seed + 100, rows, blocks)])
    best, obj = L.prr_calibrate(trajs, k, grid, p_select=p, n_threads=4)
    ref = np.array([np.mean([O.calibration_objective(t.astype(np.float64), k, tuple(float(x) for x in th),
                                                     p or None) for t in trajs]) for th in grid])
    np.testing.assert_allclose(obj, ref, rtol=0, atol=1e-12)
    want = int(np.argmax(ref))  # the first grid point on ties, as in Eq. (5) of the oracle
    assert np.allclose(best, grid[want]) or abs(ref[want] - ref[int(np.argmax(obj))]) <= 1e-12


def test_calibrate_growing_blocks_and_threads():
    L = _lib()
    grid = np.asarray(O.THETA_GRID, dtype=np.float32)
    traj = _trajectory(7, 12, 150, growing=10)
    b1, o1 = L.prr_calibrate(traj, 10, grid, n_threads=1)
    b8, o8 = L.prr_calibrate(traj, 10, grid, n_threads=8)
    assert b1 == b8 and np.array_equal(o1, o8)
    t64 = traj.astype(np.float64)
    ref = np.array([O.calibration_objective(t64, 10, tuple(float(x) for x in th)) for th in grid])
    np.testing.assert_allclose(o1, ref, rtol=0, atol=1e-12)


def test_calibrate_invalid_arguments():
    L = _lib()
    grid = np.asarray([[0.5, 0.5, 0.0]], dtype=np.float32)
    traj = _trajectory(1, 4, 16)
    with pytest.raises(L.PrrError):
        L.prr_calibrate(traj[:1], 4, grid)  # one row: no prediction to score
    with pytest.raises(L.PrrError):
        L.prr_calibrate(traj, 4, np.asarray([[0.0, 0.5, 0.0]], dtype=np.float32))  # alpha = 0
    with pytest.raises(L.PrrError):
        L.prr_calibrate(traj, -1, grid)


def test_runtime_grid_is_the_papers():
    """The product's calibration grid (Section 4.2) equals the oracle's pinned grid."""
    try:
        from paper_2606_30389_amd import runtime as R
    except ImportError as e:
        pytest.skip(f"libprr not built: {e}")
    assert [tuple(map(float, t)) for t in R.THETA_GRID] == [tuple(map(float, t)) for t in O.THETA_GRID]


def test_pick_delta():
    """The largest budget whose speculation fits in the selection window, interpolated in
    log2(context) between profiled contexts."""
    try:
        from paper_2606_30389_amd import runtime as R
    except ImportError as e:
        pytest.skip(f"libprr not built: {e}")
    lut = []
    for ctx, sel in ((4096, 10.0), (16384, 20.0)):
        for d, spec in ((1.0, 5.0), (1.5, 9.0), (2.0, 12.0 if ctx == 4096 else 19.0)):
            lut.append({"context": ctx, "delta": d, "select_us": sel, "spec_us": spec})
    assert R.pick_delta(lut, 4096) == 1.5       # 12 > 10
    assert R.pick_delta(lut, 16384) == 2.0      # 19 <= 20
    assert R.pick_delta(lut, 8192) == 1.5       # midway: spec 15.5 > select 15
    assert R.pick_delta(lut, 1024) == 1.5       # clamped to the smallest context
    assert R.pick_delta([], 4096) == 1.0
    lut_bad = [{"context": 4096, "delta": 2.0, "select_us": 1.0, "spec_us": 5.0}]
    assert R.pick_delta(lut_bad, 4096) == 1.0
