"""hieravg_evaluate_noalloc (the evaluation entry point that allocates
nothing: its chunk buffers live in a file-scope device array) against
hieravg_evaluate, through the C ABI: two calls in a row on one handle, the
second over fewer rows, on the softmax model, the small-class MLP head, the
MLP with more than 32 classes and a 1024-wide hidden layer (a smaller chunk
than hieravg_evaluate takes, so several chunks and a ragged last one), and
the held-out split; a model too wide for the array is rejected."""

import ctypes

import numpy as np
import pytest

import cases
from oracle import method as M

pytestmark = pytest.mark.gpu

CASES = {
    "softmax": (cases.case("softmax", 3, 3, 3, 1, B=17, IN=33, C=17, N=5000, lr=0.2, seed=3), (4999, 1234)),
    "mlp_small_head": (cases.case("mlp", 4, 2, 2, 2, B=12, IN=150, H=70, C=6, N=3000, sigma=0.5, lr=0.05, seed=21),
                       (3000, 17)),
    "mlp_wide_hidden_large_c": (cases.case("mlp", 2, 2, 1, 1, B=8, IN=300, H=1024, C=40, N=3000, sigma=0.5,
                                           lr=0.05, seed=71), (2999, 1025)),
}


def _eval(L, fn, h, replica, split, n):
    loss, hits = ctypes.c_double(), ctypes.c_int64()
    rc = getattr(L, fn)(h, replica, split, n, ctypes.byref(loss), ctypes.byref(hits))
    assert rc == 0, (fn, rc, L.hieravg_last_error().decode())
    return loss.value, hits.value


@pytest.mark.parametrize("name", sorted(CASES))
def test_noalloc_evaluate_matches_evaluate(name, gpu_lib):
    L = gpu_lib
    c, (n1, n2) = CASES[name]
    prob = cases.oracle_problem(c)
    cfg = cases.native_config(c)
    h = L.hieravg_create_config(ctypes.byref(cfg))
    assert h, L.hieravg_last_error().decode()
    try:
        assert L.hieravg_round(h) == 0
        D = L.hieravg_dim(h)
        W = np.zeros((c["P"], D), dtype=np.float32)
        assert L.hieravg_params(h, W.ctypes.data, W.size) == 0
        # held-out rows exist only after hieravg_evaluate generated them
        loss, hits = ctypes.c_double(), ctypes.c_int64()
        assert L.hieravg_evaluate_noalloc(h, 0, 1, 10, ctypes.byref(loss), ctypes.byref(hits)) == -4
        for split in (0, 1):
            for replica, n in ((0, n1), (c["P"] - 1, n2)):  # two calls, the second over fewer rows
                print(f"[gpu case] noalloc {name} split {split} replica {replica} rows {n}", flush=True)
                want = _eval(L, "hieravg_evaluate", h, replica, split, n)
                got = _eval(L, "hieravg_evaluate_noalloc", h, replica, split, n)
                assert abs(got[0] - want[0]) <= 1e-4 * max(1.0, abs(want[0])), (got, want)
                if got[1] != want[1]:  # an argmax float32 may decide either way: a near-tie row
                    _, _, gaps = M.evaluate(prob, W[replica].astype(np.float64), np.arange(n), split)
                    assert abs(got[1] - want[1]) <= int(np.sum(gaps < 1e-5)), (got, want)
        assert L.hieravg_evaluate_noalloc(h, 0, 0, c["N"] + 1, ctypes.byref(loss), ctypes.byref(hits)) == -1
    finally:
        L.hieravg_destroy(h)


def test_noalloc_evaluate_rejects_a_model_beyond_the_scratch(gpu_lib):
    """2*hidden + classes beyond what one 16-row chunk of the array holds."""
    L = gpu_lib
    c = cases.case("mlp", 1, 1, 1, 1, B=1, IN=1, H=140000, C=2, N=4, lr=0.1, seed=72)
    cfg = cases.native_config(c)
    h = L.hieravg_create_config(ctypes.byref(cfg))
    assert h, L.hieravg_last_error().decode()
    try:
        loss, hits = ctypes.c_double(), ctypes.c_int64()
        assert L.hieravg_evaluate_noalloc(h, 0, 0, 4, ctypes.byref(loss), ctypes.byref(hits)) == -4
        assert "scratch" in L.hieravg_last_error().decode()
        # the allocating entry point still evaluates it
        assert L.hieravg_evaluate(h, 0, 0, 4, ctypes.byref(loss), ctypes.byref(hits)) == 0
        assert np.isfinite(loss.value) and 0 <= hits.value <= 4
    finally:
        L.hieravg_destroy(h)
