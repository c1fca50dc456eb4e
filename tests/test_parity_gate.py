"""The parity gate used by the GPU tests rejects planted mistakes (planted in
oracle output on the CPU) and accepts only deviations it can attribute to a
ReLU decision within float32 rounding."""

import numpy as np
import pytest

import cases
from oracle import method as M


@pytest.fixture(scope="module")
def mlp_run():
    c = cases.case("mlp", 4, 2, 2, 2, B=8, IN=40, H=128, C=5, N=64, sigma=0.5, lr=0.1, seed=3)
    prob = cases.oracle_problem(c)
    mon = M.KinkMonitor(prob.H)
    st = M.run(prob, 1, monitor=mon)
    return prob, st, mon


def _perturb_unit(prob, W, h, rel):
    out = W.astype(np.float32).copy()
    blk = M.unpack(prob, out[0])
    blk["W1"][h, :] += rel * np.abs(M.unpack(prob, W[0])["W1"]).max()
    return out


def test_exact_copy_passes(mlp_run):
    prob, st, mon = mlp_run
    ok, det = cases.parity_report(prob, st.W.astype(np.float32), st.W, mon)
    assert ok and det["worst"][1] < 1e-6


def test_unexplained_unit_deviation_fails(mlp_run):
    prob, st, mon = mlp_run
    h = int(np.argmax(mon.min_margin))          # the unit farthest from any kink
    ok, det = cases.parity_report(prob, _perturb_unit(prob, st.W, h, 1e-3), st.W, mon)
    assert not ok


def test_kink_explained_unit_deviation_passes_only_when_small(mlp_run):
    prob, st, mon = mlp_run
    h = 7
    mon2 = M.KinkMonitor(prob.H)
    mon2.min_margin = mon.min_margin.copy()
    mon2.min_margin[h] = 1e-9                   # as if unit h had a near-zero pre-activation
    ok, det = cases.parity_report(prob, _perturb_unit(prob, st.W, h, 1e-3), st.W, mon2)
    assert ok and det["exempt_units"] == [h]
    ok, _ = cases.parity_report(prob, _perturb_unit(prob, st.W, h, 0.1), st.W, mon2)
    assert not ok                                # beyond the validity bound
    ok, _ = cases.parity_report(prob, _perturb_unit(prob, st.W, h, 1e-3), st.W, None)
    assert not ok                                # no kink evidence: strict gate


def test_too_many_exempt_units_fail(mlp_run):
    prob, st, mon = mlp_run
    mon2 = M.KinkMonitor(prob.H)
    mon2.min_margin = np.full(prob.H, 1e-9)
    W = st.W.astype(np.float32).copy()
    for h in range(10):
        W = _perturb_unit(prob, W.astype(np.float64), h, 1e-3)
    ok, det = cases.parity_report(prob, W, st.W, mon2)
    assert not ok


@pytest.mark.parametrize("block", ["b2", "W2"])
def test_other_blocks_stay_strict(mlp_run, block):
    prob, st, mon = mlp_run
    W = st.W.astype(np.float32).copy()
    blk = M.unpack(prob, W[1])
    blk[block].reshape(-1)[0] += 1e-3 * np.abs(blk[block]).max()
    ok, _ = cases.parity_report(prob, W, st.W, mon)
    assert not ok


def test_softmax_has_no_exception():
    c = cases.case("softmax", 2, 1, 1, 1, B=4, IN=10, C=3, N=20, lr=0.1)
    prob = cases.oracle_problem(c)
    st = M.run(prob, 1)
    W = st.W.astype(np.float32).copy()
    W[0, 3] += 1e-3 * np.abs(st.W).max()
    assert not cases.parity_report(prob, W, st.W, None)[0]
