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
    (entries of blocks not formed yet hold junk that must never be read)."""
    rng = np.random.default_rng(seed)
    base = rng.gamma(2.0, 1.0, size=blocks)
    out = np.empty((rows, blocks), dtype=np.float32)
    cur = base.copy()
    for r in range(rows):
        cur = np.abs(cur + drift * rng.normal(size=blocks))
        out[r] = cur
        if growing:
            formed = blocks - growing + min(r, growing)
            out[r, formed:] = 1e6
    return out


def _form_rows(rows, blocks, growing):
    """Row at which each block of a `growing` trajectory forms."""
    return np.array([max(0, b - (blocks - growing)) if b >= blocks - growing else 0 for b in range(blocks)],
                    dtype=np.int32)


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
    fr = _form_rows(12, 150, 10)
    b1, o1 = L.prr_calibrate(traj, 10, grid, n_threads=1, form_row=fr)
    b8, o8 = L.prr_calibrate(traj, 10, grid, n_threads=8, form_row=fr)
    assert b1 == b8 and np.array_equal(o1, o8)
    t64 = traj.astype(np.float64)
    ref = np.array([O.calibration_objective(t64, 10, tuple(float(x) for x in th), None, fr) for th in grid])
    np.testing.assert_allclose(o1, ref, rtol=0, atol=1e-12)
    assert int(np.argmax(ref)) == int(np.argmax(o1)) and b1 == tuple(float(x) for x in grid[int(np.argmax(ref))])


def test_calibrate_formation_pins_natively():
    """The library's calibration on the hand-worked trajectories that pin the oracle."""
    from tests import oracle_pins as pins
    L = _lib()
    grid = [tuple(float(x) for x in t) for t in O.THETA_GRID]

    def objective(traj, k, theta, p_select=None, form_row=None):
        g = np.asarray([theta], dtype=np.float32)
        return float(L.prr_calibrate(np.asarray(traj, np.float32), k, g, p_select=p_select or 0,
                                     form_row=form_row)[1][0])

    def calibrate(traj, k, grid_):
        best, obj = L.prr_calibrate(np.asarray(traj, np.float32), k, np.asarray(grid_, np.float32))
        return tuple(round(x, 6) for x in best), float(obj.max())

    assert pins.check_calibrate_closed_form(objective, calibrate, grid)
    assert pins.check_calibrate_all_tied(calibrate, grid)
    assert pins.check_calibration_formation(objective, grid)


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
    with pytest.raises(L.PrrError):
        L.prr_calibrate(traj, 4, grid, form_row=np.full(16, -1, dtype=np.int32))


def test_runtime_grid_is_the_papers():
    """The product's calibration grid (Section 4.2) equals the oracle's pinned grid."""
    try:
        from paper_2606_30389_amd import runtime as R
    except ImportError as e:
        pytest.skip(f"libprr not built: {e}")
    assert [tuple(map(float, t)) for t in R.THETA_GRID] == [tuple(map(float, t)) for t in O.THETA_GRID]


def test_pick_delta():
    """Section 4.4 in the library: the largest delta whose speculation fits in the selection
    window.  The profiled latencies are exact polynomials of x = log2(context) of degree
    <= 2, so the degree-2 regression recovers them at unprofiled contexts and the pick
    follows by hand: select(x) = 2 + x; delta 1 and 1.5 always fit (1 + x/2 and 1 + x);
    delta 2 (0.25 (x - 14)^2 + 12) fits iff x^2 - 32 x + 236 <= 0, i.e. for x in
    [16 - 2 sqrt(5), 16 + 2 sqrt(5)]."""
    L = _lib()
    rows = []
    for ctx in (4096, 8192, 16384, 32768, 65536):
        x = np.log2(ctx)
        for d, spec in ((1.0, 1 + x / 2), (1.5, 1.0 + x), (2.0, 0.25 * (x - 14) ** 2 + 12)):
            rows.append({"context": ctx, "delta": d, "select_us": 2 + x, "spec_us": spec})
    lo, hi = 16 - 2 * np.sqrt(5), 16 + 2 * np.sqrt(5)
    for ctx in (5000, 12000, 20000, 100000, 131072, 2 ** 20, 2 ** 22):
        x = np.log2(ctx)
        want = 2.0 if lo <= x <= hi else 1.5
        d, se, sp = L.prr_pick_delta(rows, ctx, degree=2)
        assert d == want, (ctx, d, want)
        assert abs(se - (2 + x)) < 1e-3
    # a profiled context uses its own row: make delta 2 fit only there
    rows2 = [dict(r) for r in rows]
    for r in rows2:
        if r["delta"] == 2.0:
            r["spec_us"] = 100.0 if r["context"] != 16384 else 1.0
    assert L.prr_pick_delta(rows2, 16384)[0] == 2.0
    assert L.prr_pick_delta(rows2, 16000)[0] == 1.5
    # degree 0 averages: a constant fit
    d0 = L.prr_pick_delta([{"context": 4096, "delta": 2.0, "select_us": 10.0, "spec_us": 9.0},
                           {"context": 8192, "delta": 2.0, "select_us": 10.0, "spec_us": 12.0}], 6000, degree=0)
    assert d0[0] == 1.0 and abs(d0[2] - 10.5) < 1e-5
    # no table: delta 1; nothing fits: delta 1
    assert L.prr_pick_delta([], 4096)[0] == 1.0
    assert L.prr_pick_delta([{"context": 4096, "delta": 2.0, "select_us": 1.0, "spec_us": 5.0}], 4096)[0] == 1.0
    with pytest.raises(L.PrrError):
        L.prr_pick_delta(rows, 0)
    with pytest.raises(L.PrrError):
        L.prr_pick_delta(rows, 4096, degree=4)
    with pytest.raises(L.PrrError):
        L.prr_pick_delta([{"context": 4096, "delta": 0.5, "select_us": 1.0, "spec_us": 0.5}], 4096)


def test_runtime_pick_delta_is_the_library_call():
    try:
        from paper_2606_30389_amd import runtime as R
    except ImportError as e:
        pytest.skip(f"libprr not built: {e}")
    L = _lib()
    lut = [{"context": c, "delta": d, "select_us": 10.0, "spec_us": 5.0 * d} for c in (4096, 65536) for d in (1.0, 2.0, 3.0)]
    assert R.pick_delta(lut, 16384) == L.prr_pick_delta(lut, 16384)[0] == 2.0


def test_pick_delta_step_takes_the_fastest_fitting_budget():
    """Of the budgets whose speculation fits the selection window, the one with the
    shortest profiled step; a budget that does not fit is never taken, however fast; an
    unprofiled context falls back to the Section 4.4 rule."""
    try:
        from paper_2606_30389_amd import runtime as R
    except ImportError as e:
        pytest.skip(f"libprr not built: {e}")
    rows = [
        {"context": 4096, "delta": 1.0, "select_us": 8.0, "spec_us": 4.0, "fused_prr_late_us": 16.0},
        {"context": 4096, "delta": 1.5, "select_us": 8.0, "spec_us": 5.0, "fused_prr_late_us": 15.0},
        {"context": 4096, "delta": 2.0, "select_us": 8.0, "spec_us": 9.0, "fused_prr_late_us": 14.0},
        {"context": 8192, "delta": 1.0, "select_us": 8.0, "spec_us": 4.0, "fused_prr_late_us": 16.0},
        {"context": 8192, "delta": 1.5, "select_us": 8.0, "spec_us": 5.0, "fused_prr_late_us": 17.0},
        {"context": 8192, "delta": 2.0, "select_us": 8.0, "spec_us": 6.0, "fused_prr_late_us": 18.0},
    ]
    assert R.pick_delta_step(rows, 4096) == (1.5, 15.0)  # delta 2 is faster but does not fit
    assert R.pick_delta_step(rows, 8192) == (1.0, 16.0)  # the rule would take 2
    assert R.pick_delta(rows, 8192) == 2.0
    d, us = R.pick_delta_step(rows, 6000)
    assert us is None and d == R.pick_delta(rows, 6000)
