"""The parity gate used by the GPU tests, checked both ways on the CPU.

It must reject planted mistakes (planted in oracle output) and accept a
deviation only when it is exactly the other correct branch of a ReLU decision
at a kink: the oracle re-run with that near-zero decision taken the other way
must then match every parameter to the strict tolerance."""

import numpy as np
import pytest

import cases
from oracle import method as M

CASE = cases.case("mlp", 4, 2, 2, 2, B=8, IN=40, H=128, C=5, N=64, sigma=0.5, lr=0.1, seed=3)


@pytest.fixture(scope="module")
def mlp_run():
    prob = cases.oracle_problem(CASE)
    mon = M.KinkMonitor(prob.H)
    st = M.run(prob, 1, monitor=mon)
    # a monitor with a wide threshold: decisions close to (not at) a kink,
    # whose flip changes the result far beyond rounding
    wide = M.KinkMonitor(prob.H, threshold=0.05)
    M.run(prob, 1, monitor=wide)
    return prob, st, mon, wide


def _rerun(prob):
    return lambda flips: M.run(prob, 1, flips=flips).W


def _perturb_unit(prob, W, h, rel):
    out = W.astype(np.float32).copy()
    blk = M.unpack(prob, out[0])
    blk["W1"][h, :] += rel * np.abs(M.unpack(prob, W[0])["W1"]).max()
    return out


def _monitor_with(prob, decisions):
    mon = M.KinkMonitor(prob.H)
    mon.decisions = list(decisions)
    return mon


def _flip_that_matters(prob, st, wide, k=0):
    """The k-th wide-threshold decision whose flip moves the result beyond the
    gate (so the plain gate rejects that run)."""
    found = []
    for d in sorted(wide.decisions, key=lambda d: d[4]):
        W = M.run(prob, 1, flips=frozenset([d[:4]])).W
        if not cases.parity_report(prob, W.astype(np.float32), st.W)[0]:
            found.append((d, W))
            if len(found) > k:
                return found[k]
    pytest.fail("no decision whose flip matters")


def test_exact_copy_passes(mlp_run):
    prob, st, mon, _ = mlp_run
    ok, det = cases.branch_parity(prob, st.W.astype(np.float32), st.W, mon, _rerun(prob))
    assert ok and det["worst"][1] < 1e-6 and "flipped" not in det


def test_unexplained_unit_deviation_fails(mlp_run):
    prob, st, mon, wide = mlp_run
    h = wide.decisions[0][3]                    # even a unit with candidate decisions
    got = _perturb_unit(prob, st.W, h, 1e-3)
    ok, det = cases.parity_report(prob, got, st.W)
    assert not ok and h in det["units"]
    ok, det = cases.branch_parity(prob, got, st.W, wide, _rerun(prob))
    assert not ok and det["candidates"]         # flips were tried, none explains it


def test_other_branch_of_a_flagged_decision_passes(mlp_run):
    prob, st, _, wide = mlp_run
    d, W = _flip_that_matters(prob, st, wide)
    got = W.astype(np.float32)
    assert not cases.parity_report(prob, got, st.W)[0]
    ok, det = cases.branch_parity(prob, got, st.W, _monitor_with(prob, [d]), _rerun(prob))
    assert ok and det["flipped"] == [d]
    # the same run is rejected when the decision was not flagged as near a kink
    ok, _ = cases.branch_parity(prob, got, st.W, _monitor_with(prob, []), _rerun(prob))
    assert not ok
    ok, _ = cases.branch_parity(prob, got, st.W, None, _rerun(prob))
    assert not ok


def test_two_flipped_decisions_are_found(mlp_run):
    prob, st, _, wide = mlp_run
    d1, _ = _flip_that_matters(prob, st, wide, 0)
    d2, _ = _flip_that_matters(prob, st, wide, 1)
    got = M.run(prob, 1, flips=frozenset([d1[:4], d2[:4]])).W.astype(np.float32)
    ok, det = cases.branch_parity(prob, got, st.W, _monitor_with(prob, [d1, d2]), _rerun(prob))
    assert ok and sorted(det["flipped"]) == sorted([d1, d2])


def test_flip_plus_a_mistake_fails(mlp_run):
    prob, st, _, wide = mlp_run
    d, W = _flip_that_matters(prob, st, wide)
    got = W.astype(np.float32).copy()
    blk = M.unpack(prob, got[2])
    blk["b2"][0] += 1e-3 * np.abs(blk["b2"]).max()
    ok, _ = cases.branch_parity(prob, got, st.W, _monitor_with(prob, [d]), _rerun(prob))
    assert not ok


@pytest.mark.parametrize("block", ["b2", "W2", "b1"])
def test_other_blocks_stay_strict(mlp_run, block):
    prob, st, mon, wide = mlp_run
    W = st.W.astype(np.float32).copy()
    blk = M.unpack(prob, W[1])
    blk[block].reshape(-1)[0] += 1e-3 * np.abs(blk[block]).max()
    ok, _ = cases.branch_parity(prob, W, st.W, wide, _rerun(prob))
    assert not ok


def test_softmax_gate_is_strict():
    c = cases.case("softmax", 2, 1, 1, 1, B=4, IN=10, C=3, N=20, lr=0.1)
    prob = cases.oracle_problem(c)
    st = M.run(prob, 1)
    W = st.W.astype(np.float32).copy()
    W[0, 3] += 1e-3 * np.abs(st.W).max()
    assert not cases.branch_parity(prob, W, st.W, None, _rerun(prob))[0]
    assert cases.branch_parity(prob, st.W.astype(np.float32), st.W, None, _rerun(prob))[0]
