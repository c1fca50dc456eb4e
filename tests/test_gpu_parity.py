"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Gate (the normwise reading of "max relative error 1e-4" for float32): for
every replica and every parameter block, max|gpu - oracle| / max|oracle|
<= 1e-4 after the round(s).  Where several results are correct -- a ReLU
decision whose pre-activation was within float32 rounding of zero may come
out either way -- the oracle is re-run with such flagged decisions taken the
other way and the GPU must meet the same gate against one of those runs
(cases.branch_parity).  Minibatch indices must match bit for bit, and after
a round every replica row must be bit-identical (the global mean of
Algorithm 1 writes one value to all P learners; under delayed first-layer
updates, and in eager rounds of full-tile steps, W1's global mean is stored
once, so there the check covers b1, W2 and b2, and the next round's parity
is what shows that every learner read it).
"""

import numpy as np
import pytest

import cases
from oracle import method as M
from oracle import rng as R

pytestmark = pytest.mark.gpu

TOL = 1e-4


def _run_gpu(c, rounds=1, mode="auto"):
    from paper_1903_05133_amd import HierAvg
    print(f"[gpu case] {mode} {c}", flush=True)
    h = HierAvg(config=cases.native_config(c, mode))
    for _ in range(rounds):
        h.round()
    got = h.params()
    idx = h.last_indices() if c["kind"] != "averaging" else None
    steps = h.steps
    h.close()
    return got, idx, steps


def _oracle(c, rounds=1):
    """The oracle's run, its kink monitor and a re-run with flipped decisions."""
    prob = cases.oracle_problem(c)
    mon = M.KinkMonitor(prob.H) if prob.kind == M.MLP else None
    return M.run(prob, rounds, monitor=mon), mon, (lambda flips: M.run(prob, rounds, flips=flips).W)


def _identical_rows(prob, got, w1_too=True):
    """Every replica row equals row 0 (bit for bit), block by block."""
    for p in range(1, got.shape[0]):
        a, b = M.unpack(prob, got[p]), M.unpack(prob, got[0])
        for name in a:
            if name == "W1" and not w1_too:
                continue
            if not np.array_equal(a[name], b[name]):
                return False
    return True


def _check(c, got, idx, st, mon=None, rerun=None, mode="auto"):
    prob = cases.oracle_problem(c)
    if idx is not None:
        assert np.array_equal(idx.astype(np.int64), st.last_indices), "minibatch indices differ"
    assert np.all(np.isfinite(got))
    # W1 rows are compared only where W1 is stored per learner (EAGER rounds
    # that do not write the global mean of W1 once, to a common copy)
    w1_rows = mode == "eager" and not cases.eager_means_once(c)[0]
    assert _identical_rows(prob, got, w1_too=w1_rows), "replicas differ after the global mean"
    ok, det = cases.branch_parity(prob, got, st.W, mon, rerun)
    print(f"[gpu case] worst block error {det['worst']} flipped {det.get('flipped')} "
          f"candidates {len(det.get('candidates', []))}", flush=True)
    assert ok, det
    return det


SMALL = {
    # several N tiles, K splits and ragged tails in every dimension; B > 32
    "mlp_multi_tile": cases.case("mlp", 4, 2, 2, 2, B=40, IN=700, H=300, C=40, N=500, sigma=0.5, lr=0.05, seed=4),
    "mlp_ragged": cases.case("mlp", 6, 3, 2, 3, B=5, IN=100, H=70, C=3, N=37, sigma=0.5, lr=0.1, seed=1),
    "mlp_batch1_S1": cases.case("mlp", 2, 1, 1, 2, B=1, IN=64, H=64, C=16, N=10, lr=0.1, seed=2),
    "mlp_batch_150": cases.case("mlp", 2, 2, 1, 1, B=150, IN=200, H=130, C=7, N=300, lr=0.05, seed=6),
    # fused step kernel with the cluster mean of 8 learners, one 16-row batch tile
    "mlp_group_mean_S8": cases.case("mlp", 16, 8, 2, 2, B=12, IN=200, H=70, C=5, N=300, lr=0.1, seed=13),
    # block ends beyond the fused mean step (S * padded B over 256 rows): the
    # update with the cluster mean, then one forward GEMM per cluster; ragged
    # samples, rows and columns, and the more-than-32-class head (b1 stepped
    # in the update kernel)
    "mlp_update_mean_S8_B40": cases.case("mlp", 16, 8, 2, 2, B=40, IN=200, H=70, C=5, N=300, lr=0.1, seed=19),
    "mlp_update_mean_S16_c40": cases.case("mlp", 16, 16, 2, 2, B=20, IN=130, H=90, C=40, N=200, sigma=0.5,
                                          lr=0.05, seed=20),
    # fused step with the mean of 4 learners on the softmax model; ragged last column tile
    "softmax_group_mean_S4": cases.case("softmax", 8, 4, 1, 3, B=20, IN=130, C=12, N=90, lr=0.2, seed=14),
    # B = 32: the block update's stages are whole (step, learner) runs of
    # samples; ragged hidden and input widths, two learners per cluster
    "mlp_batch_32_ragged": cases.case("mlp", 6, 2, 3, 2, B=32, IN=200, H=70, C=5, N=300, lr=0.05, seed=15),
    # 17..32 classes (the delayed head's 32-class tiles) with 32- and 16-row
    # padded minibatches, both ragged
    "mlp_c24_batch_24": cases.case("mlp", 4, 2, 3, 2, B=24, IN=150, H=70, C=24, N=300, lr=0.05, seed=17),
    "mlp_c20_batch_10": cases.case("mlp", 4, 4, 4, 1, B=10, IN=90, H=100, C=20, N=200, lr=0.1, seed=18),
    "mlp_one_learner": cases.case("mlp", 1, 1, 3, 2, B=8, IN=96, H=33, C=5, N=64, lr=0.1, seed=7),
    "mlp_one_sample_dataset": cases.case("mlp", 4, 4, 2, 1, B=3, IN=50, H=20, C=2, N=1, lr=0.1, seed=8),
    "softmax_ragged": cases.case("softmax", 3, 3, 3, 1, B=17, IN=33, C=17, N=50, lr=0.2, seed=3),
    "softmax_single_class_dim": cases.case("softmax", 2, 1, 2, 2, B=4, IN=1, C=1, N=5, lr=0.1, seed=9),
    "averaging_ragged": cases.case("averaging", 4, 2, 2, 3, IN=1001, lr=0.1, momentum=0.9, seed=5),
    "averaging_S1": cases.case("averaging", 3, 1, 1, 2, IN=4099, lr=0.05, momentum=0.5, seed=10),
    "averaging_one_learner": cases.case("averaging", 1, 1, 2, 2, IN=67, lr=0.1, momentum=0.9, seed=11),
    "averaging_D1": cases.case("averaging", 2, 2, 1, 1, IN=1, lr=0.1, momentum=0.9, seed=12),
}


@pytest.mark.parametrize("name", sorted(SMALL))
def test_small_cases_match_oracle(name, gpu_lib):
    c = SMALL[name]
    got, idx, steps = _run_gpu(c, rounds=2, mode="eager")
    assert steps == 2 * c["K1"] * c["K2"]
    _check(c, got, idx, *_oracle(c, 2), mode="eager")


@pytest.mark.parametrize("name", ["mlp_update_mean_S8_B40", "mlp_update_mean_S16_c40"])
def test_update_mean_block_end_kernels(name, gpu_lib):
    """Eager block ends of S * B too large for the fused mean step take the
    update-with-mean kernel and the per-cluster forward GEMM."""
    from paper_1903_05133_amd import HierAvg
    c = SMALL[name]
    with HierAvg(config=cases.native_config(c, "eager")) as h:
        h.profile(True)
        h.round()
        stats = h.profile_read()
    assert "update1_gemm_group_mean" in stats and "fwd1_group_gemm" in stats, stats
    assert "step1_gemm_group_mean" not in stats and "group_mean" not in stats, stats


# Eager loss side at most 32 classes: the one-workgroup-per-16-samples head
# (16 or 32 class slots, hidden widths up to its LDS limit) and, past that
# limit, the two-kernel head over 32-unit slices.
EAGER_HEADS = {
    # 16 class slots, Hp = 1024, B = 20: two sample groups, the second ragged
    "fused16_h1000": (cases.case("mlp", 4, 2, 2, 2, B=20, IN=130, H=1000, C=7, N=300, sigma=0.5, lr=0.05, seed=61),
                      "head_fused"),
    # 32 class slots, Hp = 320, B = 40: three sample groups
    "fused32_h300": (cases.case("mlp", 4, 2, 2, 2, B=40, IN=100, H=300, C=20, N=300, sigma=0.5, lr=0.05, seed=62),
                     "head_fused"),
    # more than three K splits of the step's forward (the head's batched loads
    # for any split count): 32 class slots, 384 inputs in six splits; 16 class
    # slots, Hp = 1024, 320 inputs in five splits
    "fused32_h300_ks6": (cases.case("mlp", 4, 2, 2, 2, B=20, IN=384, H=300, C=20, N=300, sigma=0.5, lr=0.05,
                                    seed=64), "head_fused"),
    "fused16_h1000_ks5": (cases.case("mlp", 4, 2, 2, 2, B=20, IN=320, H=1000, C=7, N=300, sigma=0.5, lr=0.05,
                                     seed=65), "head_fused"),
    # 32 class slots with Hp = 640: past the fused head's LDS
    "slices_c20_h600": (cases.case("mlp", 4, 2, 2, 2, B=12, IN=100, H=600, C=20, N=300, sigma=0.5, lr=0.05,
                                   seed=63), "head_b"),
}


@pytest.mark.parametrize("name", sorted(EAGER_HEADS))
def test_eager_small_class_heads(name, gpu_lib):
    from paper_1903_05133_amd import HierAvg
    c, head = EAGER_HEADS[name]
    with HierAvg(config=cases.native_config(c, "eager")) as h:
        h.profile(True)
        h.round()
        stats = h.profile_read()
        h.profile(False)
        h.round()
        got = h.params()
        idx = h.last_indices()
    assert head in stats, stats
    assert ("head_a" in stats) == (head == "head_b") and ("head_fused" in stats) == (head == "head_fused"), stats
    _check(c, got, idx, *_oracle(c, 2), mode="eager")


# MLP cases within the delayed-update limits (at most 32 classes, B <= 32, K1 <= 8)
DELAYED = sorted(n for n, c in SMALL.items() if c["kind"] == "mlp" and c["C"] <= 32 and c["B"] <= 32)


@pytest.mark.parametrize("name", DELAYED)
def test_small_cases_delayed_updates_match_oracle(name, gpu_lib):
    c = SMALL[name]
    got, idx, steps = _run_gpu(c, rounds=2, mode="delayed")
    assert steps == 2 * c["K1"] * c["K2"]
    _check(c, got, idx, *_oracle(c, 2), mode="delayed")


LARGE_C_DELAYED = {
    # more than 32 classes: per step the pre-activation kernel with the Gram
    # correction, then the layer-2 GEMM head; ragged hidden width
    "mlp_c40_K1_3": cases.case("mlp", 4, 2, 3, 2, B=20, IN=130, H=70, C=40, N=300, sigma=0.5, lr=0.05, seed=41),
    "mlp_c100_K1_1": cases.case("mlp", 2, 2, 1, 3, B=7, IN=64, H=96, C=100, N=50, sigma=0.5, lr=0.1, seed=42),
    "mlp_c33_K1_8": cases.case("mlp", 4, 4, 8, 1, B=32, IN=96, H=64, C=33, N=200, sigma=0.5, lr=0.05, seed=43),
    # 1024 input features: the Gram blocks are summed over 8 feature splits
    # before the pre-activation kernel reads them; two blocks, so the block
    # update's cluster mean of b1, W2, b2 runs once before the global mean
    "mlp_c40_in1024_K1_4": cases.case("mlp", 4, 2, 4, 2, B=32, IN=1024, H=96, C=40, N=400, sigma=0.5, lr=0.05,
                                      seed=44),
}


@pytest.mark.parametrize("name", sorted(LARGE_C_DELAYED))
def test_large_class_delayed_updates_match_oracle(name, gpu_lib):
    from paper_1903_05133_amd import HierAvg
    c = LARGE_C_DELAYED[name]
    with HierAvg(config=cases.native_config(c, "delayed")) as h:
        h.profile(True)
        h.round()
        stats = h.profile_read()
        h.profile(False)
        h.round()
        got = h.params()
        idx = h.last_indices()
    assert "block_update_gemm" in stats and "z1_delayed" in stats and "head_step" not in stats
    # plain SGD, B <= 32: the hidden-error kernel also steps W2 and b2
    assert "bwd_hidden" in stats and "update2_gemm" not in stats
    if c["IN"] >= 1024:
        assert "gram_reduce" in stats
    _check(c, got, idx, *_oracle(c, 2), mode="delayed")


@pytest.mark.parametrize("K1,C,B", [(8, 7, 32), (6, 20, 32), (7, 12, 32), (5, 7, 20), (2, 5, 17)])
def test_delayed_updates_long_block(K1, C, B, gpu_lib):
    """Blocks of two to eight steps (K1 = 8 is the largest the delayed path
    takes) with 32-sample Gram blocks (full and ragged minibatches), 16- and
    32-class head tiles; S = 2, three blocks."""
    c = cases.case("mlp", 4, 2, K1, 3, B=B, IN=130, H=96, C=C, N=400, sigma=0.5, lr=0.05, seed=15)
    got, idx, _ = _run_gpu(c, rounds=1, mode="delayed")
    _check(c, got, idx, *_oracle(c, 1), mode="delayed")


def test_named_softmax_workload(gpu_lib):
    """Softmax regression 3072 -> 10, N = 2048, P=4 S=2 K1=2 K2=2 B=8, lr 0.05, seed 0."""
    c = cases.named("softmax_3072_10", 4, 2, 2, 2, 8, 0.05, seed=0)
    got, idx, _ = _run_gpu(c)
    _check(c, got, idx, *_oracle(c))


@pytest.mark.parametrize("mode", ["auto", "eager"])
def test_named_mlp_workload(mode, gpu_lib):
    """MLP 3072 -> 512 -> 10, N = 50000, P=16 S=4 K1=4 K2=4 B=32, lr 0.05 (the
    configuration the benchmark times; auto takes delayed updates), one full
    round."""
    c = cases.named("mlp_3072_512_10", 16, 4, 4, 4, 32, 0.05, seed=0)
    got, idx, _ = _run_gpu(c, mode=mode)
    _check(c, got, idx, *_oracle(c), mode=mode)


@pytest.mark.slow
def test_named_mlp_workload_64_learners(gpu_lib):
    """Same MLP at P=64 S=8 K1=8 K2=4 B=64, lr 0.1, one full round."""
    c = cases.named("mlp_3072_512_10", 64, 8, 8, 4, 64, 0.1, seed=0)
    got, idx, _ = _run_gpu(c)
    _check(c, got, idx, *_oracle(c))


def test_named_averaging_workload_sampled(gpu_lib):
    """Averaging-only workload at full size (P=32 replicas of 11.7M floats,
    S=4, K1=1, K2=4, momentum 0.9, lr 0.1), one round.  Coordinates never
    interact in this workload, so the oracle computes a sample of columns
    (random ones plus both ends) exactly."""
    c = cases.named("averaging_11_7M", 32, 4, 1, 4, 1, 0.1, seed=0)
    got, _, _ = _run_gpu(c)
    D = c["IN"]
    r = np.random.default_rng(0)
    cols = np.unique(np.concatenate([r.choice(D, 3000, replace=False), np.arange(64), np.arange(D - 64, D)]))
    st = M.run(cases.oracle_problem(c), 1, cols=cols)
    assert np.array_equal(got, np.repeat(got[:1], 32, axis=0))
    sub = got[:, cols].astype(np.float64)
    err = np.max(np.abs(sub - st.W)) / np.max(np.abs(st.W))
    print(f"[gpu case] averaging sampled error {err}", flush=True)
    assert err <= TOL


def test_averaging_stored_mean_and_rows_that_differ(gpu_lib):
    """Averaging kind: the global mean is stored once and the next round's
    first step reads it (profile: momentum_first_step); after set_params with
    rows that differ the first step reads every row (no first-step class),
    with equal rows it reads the stored value again.  Parameters and buffers
    against the oracle continuing from the same state, round by round."""
    from paper_1903_05133_amd import HierAvg
    c = cases.case("averaging", 8, 4, 1, 3, IN=1003, lr=0.1, momentum=0.9, seed=37)
    prob = cases.oracle_problem(c)
    st = M.create(prob)
    with HierAvg(config=cases.native_config(c)) as h:
        for r, edit in enumerate([None, "differ", "equal", None]):
            if edit is not None:
                w = h.params()
                if edit == "differ":
                    w[3] += np.float32(0.25)
                else:
                    w[:] = w[5]
                h.set_params(w)
                st.W = w.astype(np.float64)
            h.profile(True)
            h.round()
            stats = h.profile_read()
            h.profile(False)
            M.hieravg_round(prob, st)
            got, vgot = h.params(), h.momentum()
            first = "momentum_first_step" in stats
            assert first == (edit != "differ"), (r, edit, stats)
            assert stats["momentum_global_mean"][0] == 1 and h.finite()
            for arr, want in ((got, st.W), (vgot, st.V)):
                ok, det = cases.parity_report(prob, arr, want)
                print(f"[gpu case] averaging round {r} ({edit}) worst {det['worst']}", flush=True)
                assert ok, det


@pytest.mark.slow
def test_named_large_mlp_workload(gpu_lib):
    """MLP 150528 -> 1024 -> 1000, N = 100000, at its full dimensions on the
    path its configuration takes (AUTO: delayed first-layer updates, more
    than 32 classes): P=4, S=2, K1=4, K2=2, B=32, lr 0.02 -- Gram blocks over
    150528 features in 16 feature splits and their sum, the pre-activation
    kernel with the Gram correction at steps k > 0, two blocks (the block
    update's cluster mean of b1, W2, b2 runs between them) -- against the
    oracle: indices bit-exact, every block within the gate.  The full
    configuration (P=16, S=4, K1=4, K2=2, B=32) is then checked for what holds
    at any size (finite values, identical replicas after the global mean) and
    for what the oracle computes without the model: every learner's
    minibatch indices of the round, bit for bit."""
    import torch
    from paper_1903_05133_amd import HierAvg
    c = cases.named("mlp_150528_1024_1000", 4, 2, 4, 2, 32, 0.02, seed=0)
    print(f"[gpu case] {c}", flush=True)
    with HierAvg(config=cases.native_config(c)) as h:
        h.profile(True)
        h.round()
        stats = h.profile_read()
        h.profile(False)
        got = h.params()
        idx = h.last_indices()
    assert {"gram", "gram_reduce", "fwd1_block_gemm", "z1_delayed", "block_update_gemm"} <= set(stats)
    assert stats["block_update_gemm"][0] == 2 and stats["z1_delayed"][0] == 8
    assert stats["bwd_hidden"][0] == 8 and "update2_gemm" not in stats
    st, mon, rerun = _oracle(c)
    prob = cases.oracle_problem(c)
    assert np.array_equal(idx.astype(np.int64), st.last_indices), "minibatch indices differ"
    assert np.all(np.isfinite(got)) and _identical_rows(prob, got, w1_too=False)
    ok, det = cases.branch_parity(prob, got, st.W, mon, rerun, max_runs=2)
    print(f"[gpu case] worst block error {det['worst']} flipped {det.get('flipped')}", flush=True)
    assert ok, det
    del got, st
    full = cases.named("mlp_150528_1024_1000", 16, 4, 4, 2, 32, 0.02, seed=0)
    print(f"[gpu case] {full}", flush=True)
    with HierAvg(config=cases.native_config(full)) as h:
        h.round()
        w = h.params(device="cuda")
        assert bool(torch.isfinite(w).all())
        assert bool((w == w[:1]).all())
        del w
        torch.cuda.empty_cache()
        # the round's minibatches, bit for bit: learner j's draw at step t
        want = np.array([[R.draw_indices(full["seed"], j, t, full["B"], full["N"]) for j in range(full["P"])]
                         for t in range(full["K1"] * full["K2"])], dtype=np.int64)
        assert np.array_equal(h.last_indices().astype(np.int64), want.reshape(full["K2"], full["K1"], full["P"], -1))


def test_determinism_two_handles(gpu_lib):
    c = SMALL["mlp_multi_tile"]
    a, ia, _ = _run_gpu(c, rounds=2)
    b, ib, _ = _run_gpu(c, rounds=2)
    assert np.array_equal(a, b) and np.array_equal(ia, ib)


def test_params_to_device_and_set_params_round_trip(gpu_lib):
    import torch
    from paper_1903_05133_amd import HierAvg
    c = SMALL["mlp_ragged"]
    with HierAvg(config=cases.native_config(c)) as h:
        host = h.params()
        dev = h.params(device="cuda")
        assert np.array_equal(dev.cpu().numpy(), host)
        new = torch.randn_like(dev)
        h.set_params(new)
        assert np.array_equal(h.params(), new.cpu().numpy())
        h.set_params(host + 1.0)
        assert np.array_equal(h.params(), host + 1.0)
        with pytest.raises(Exception):
            h.params_into(dev.data_ptr(), dev.numel() - 1)


def test_resume_from_params_continues_the_trajectory(gpu_lib):
    """set_params followed by a round equals the oracle's round started from
    the same replicas (both draw minibatches from global step 0)."""
    from paper_1903_05133_amd import HierAvg
    c = SMALL["mlp_ragged"]
    prob = cases.oracle_problem(c)
    with HierAvg(config=cases.native_config(c)) as h:
        h.round()
        w1 = h.params()
    with HierAvg(config=cases.native_config(c)) as h2:
        h2.set_params(w1)
        h2.round()  # equal rows (a round-boundary state): delayed updates
        got = h2.params()
        h2.round()
        got2 = h2.params()
    st = M.create(prob)
    st.W = w1.astype(np.float64)
    M.hieravg_round(prob, st)
    ok, det = cases.parity_report(prob, got, st.W)
    assert ok, det
    M.hieravg_round(prob, st)
    ok, det = cases.parity_report(prob, got2, st.W)
    assert ok, det


@pytest.mark.parametrize("name", ["global_copy_B32", "cluster_copies_K1_1"])
def test_resume_after_common_copy_round(name, gpu_lib):
    """After an eager round that left the first layer in the common copy
    (the learner rows stale): params() expands it, and set_params of those
    values, in the same handle and in a fresh one, continues the oracle's
    trajectory (the next round reads the rows again, not the copy)."""
    from paper_1903_05133_amd import HierAvg
    c, _ = ONCE_CASES[name]
    prob = cases.oracle_problem(c)
    st = M.create(prob)
    M.hieravg_round(prob, st)
    with HierAvg(config=cases.native_config(c, "eager")) as h:
        h.round()
        w1 = h.params()
        ok, det = cases.parity_report(prob, w1, st.W)
        assert ok, det
        h.set_params(w1)
        assert h.finite()
        h.round()
        got_same = h.params()
    with HierAvg(config=cases.native_config(c, "eager")) as h2:
        h2.set_params(w1)
        h2.round()
        got_fresh = h2.params()
    # the same handle continues at global step T: the oracle's second round;
    # the fresh one draws from step 0: one oracle round started from w1
    M.hieravg_round(prob, st)
    ok, det = cases.parity_report(prob, got_same, st.W)
    assert ok, det
    st2 = M.create(prob)
    st2.W = w1.astype(np.float64)
    M.hieravg_round(prob, st2)
    ok, det = cases.parity_report(prob, got_fresh, st2.W)
    assert ok, det


def test_torch_stream_and_profile(gpu_lib):
    import torch
    from paper_1903_05133_amd import HierAvg
    c = SMALL["mlp_multi_tile"]
    ref, _, _ = _run_gpu(c)
    s = torch.cuda.Stream()
    with HierAvg(config=cases.native_config(c)) as h:
        h.set_stream(s)
        h.profile(True)
        h.round()
        stats = h.profile_read()
        h.set_stream(None)
        assert np.array_equal(h.params(), ref)
    # P=4 S=2 K1=2 K2=2, padded batch 48: the stand-alone forward at step 0,
    # the fused step (with the cluster mean at the end of block 0) at steps
    # 0-2, the last step's update with the global mean of W1, then that of
    # the other blocks.
    assert stats["fwd1_gemm"][0] == 1 and "update1_gemm" not in stats
    assert stats["step1_gemm"][0] == 2 and stats["step1_gemm_group_mean"][0] == 1
    assert stats["tail_group_mean"][0] == 1 and "group_mean" not in stats
    assert stats["update1_gemm_global_mean"][0] == 1 and stats["tail_global_mean"][0] == 1
    assert stats["draw_indices"][0] == 1 and "global_mean" not in stats
    assert all(ms >= 0.0 for _, ms in stats.values())


def test_delayed_head_wide_hidden_layer(gpu_lib):
    """18 learners x 16 hidden slices (H = 480, ragged last slice) = 288 head
    workgroups per launch, more than one per CU: one head launch per step and
    one for the block's last backward; parity with the oracle."""
    from paper_1903_05133_amd import HierAvg
    c = cases.case("mlp", 18, 3, 2, 2, B=12, IN=64, H=480, C=6, N=200, lr=0.05, seed=16)
    with HierAvg(config=cases.native_config(c, "delayed")) as h:
        h.profile(True)
        h.round()
        stats = h.profile_read()
        h.profile(False)
        got = h.params()
        idx = h.last_indices()
    assert stats["head_step"][0] == 4 and stats["head_step_end"][0] == 2
    _check(c, got, idx, *_oracle(c, 1))


def test_delayed_schedule_profile(gpu_lib):
    """Delayed updates, P=6 S=3 K1=2 K2=3: per block one forward of its steps
    and one update of the cluster copies, per step one fused head kernel
    (plus one for the backward of the block's last step); the
    Gram blocks once per round; eager round after set_params, delayed again
    after."""
    from paper_1903_05133_amd import HierAvg
    c = SMALL["mlp_ragged"]
    ref, _, _ = _run_gpu(c, mode="delayed")
    with HierAvg(config=cases.native_config(c, "delayed")) as h:
        h.profile(True)
        h.round()
        stats = h.profile_read()
        h.profile(False)
        assert np.array_equal(h.params(), ref)
        assert stats["fwd1_block_gemm"][0] == 3 and stats["head_step"][0] == 6 and stats["head_step_end"][0] == 3
        assert not {"head_a", "head_b"} & set(stats)
        assert stats["block_update_gemm"][0] == 3 and stats["gram"][0] == 1
        # the cluster means of b1, W2, b2 ride in the block updates, their
        # global mean in the launch that averages the cluster copies of W1
        assert not {"tail_group_mean", "tail_global_mean"} & set(stats)
        assert stats["w1_global_mean"][0] == 1
        assert not {"fwd1_gemm", "update1_gemm", "step1_gemm", "global_mean"} & set(stats)
        h.set_params(h.params())  # equal rows: still delayed
        h.profile(True)
        h.round()
        assert "fwd1_block_gemm" in h.profile_read() and "fwd1_gemm" not in h.profile_read()
        w = h.params()
        w[1, 0] += 1.0  # rows that differ: one eager round, then delayed again
        h.set_params(w)
        h.profile(False)
        h.profile(True)
        h.round()
        assert "fwd1_gemm" in h.profile_read()
        h.profile(False)
        h.profile(True)
        h.round()
        assert "fwd1_block_gemm" in h.profile_read() and "fwd1_gemm" not in h.profile_read()


def test_delayed_block_update_large_grid(gpu_lib):
    """Cluster updates with at least eight full 128 x 128 tiles per CU (8
    clusters x 4 x 64 tiles: the two-chain block-update tile) and the tail
    means of b1, W2, b2 in the same launch: P=16 S=2 K1=4 K2=2 B=32, a
    8192-512-10 MLP, two rounds against the oracle."""
    c = cases.case("mlp", 16, 2, 4, 2, B=32, IN=8192, H=512, C=10, N=300, sigma=0.5, lr=0.02, seed=44)
    got, idx, _ = _run_gpu(c, rounds=2, mode="delayed")
    _check(c, got, idx, *_oracle(c, 2), mode="delayed")


def test_delayed_block_forward_many_clusters(gpu_lib):
    """Block forwards of 8 clusters x 4 steps x 32 samples (1024 rows per
    cluster, 2048 inputs, 512 hidden units): with the split count that fills
    the GPU, 256 x 256 tiles would keep splits under 64 chunks, so the launch
    takes the 128 x 128 tile with one split over all 2048 inputs, the plan made
    for that tile.  P=64 S=8 K1=4 K2=1 B=32, one round against the oracle."""
    c = cases.case("mlp", 64, 8, 4, 1, B=32, IN=2048, H=512, C=10, N=2000, sigma=0.5, lr=0.05, seed=45)
    got, idx, _ = _run_gpu(c, rounds=1, mode="delayed")
    _check(c, got, idx, *_oracle(c, 1), mode="delayed")


@pytest.mark.parametrize("name", ["fused_wide", "fused_one_block", "separate_many_rows"])
def test_delayed_last_block_global_mean(name, gpu_lib):
    """The last block's update over all P learners from the mean of the
    cluster copies (the global mean of W1, b1, W2, b2 in the same launch)
    where W1 has at least 512 output tiles (8192 inputs x 512 units; also
    with one block per round, whose base is replica 0's W1, updated in
    place); with more rows than one update takes (K1*P*B = 8*72*32 > 16384)
    the last block updates the cluster copies and a separate launch averages
    them."""
    from paper_1903_05133_amd import HierAvg
    c = {"fused_wide": cases.case("mlp", 4, 2, 2, 3, B=16, IN=8192, H=512, C=6, N=200, sigma=0.5, lr=0.05, seed=19),
         "fused_one_block": cases.case("mlp", 4, 2, 3, 1, B=12, IN=8200, H=500, C=20, N=200, sigma=0.5, lr=0.05,
                                       seed=20),
         "separate_many_rows": cases.case("mlp", 72, 8, 8, 2, B=32, IN=64, H=64, C=5, N=500, sigma=0.5, lr=0.05,
                                          seed=21)}[name]
    with HierAvg(config=cases.native_config(c, "delayed")) as h:
        h.profile(True)
        h.round()
        stats = h.profile_read()
        h.profile(False)
        h.round()
        got = h.params()
        idx = h.last_indices()
    assert stats["block_update_gemm"][0] == c["K2"]
    assert ("w1_global_mean" in stats) == (name == "separate_many_rows")
    _check(c, got, idx, *_oracle(c, 2), mode="delayed")


def test_unfused_schedule_profile(gpu_lib):
    """S = 3 has no fused-mean kernel: block ends run the plain update, the
    whole-replica cluster mean and the stand-alone forward of the next step."""
    from paper_1903_05133_amd import HierAvg
    c = SMALL["mlp_ragged"]  # P=6 S=3 K1=2 K2=3
    with HierAvg(config=cases.native_config(c, "eager")) as h:
        h.profile(True)
        h.round()
        stats = h.profile_read()
    assert stats["group_mean"][0] == 2 and stats["fwd1_gemm"][0] == 3
    assert stats["update1_gemm"][0] == 3 and stats["step1_gemm"][0] == 3
    assert "step1_gemm_group_mean" not in stats


# ---------------------------------------------------------------- evaluation
EVAL_CASES = {
    "softmax_ragged": (SMALL["softmax_ragged"], "auto"),
    "mlp_ragged_delayed": (SMALL["mlp_ragged"], "delayed"),
    "mlp_multi_tile_large_C": (SMALL["mlp_multi_tile"], "eager"),
    "mlp_3072_512_10": (cases.named("mlp_3072_512_10", 16, 4, 4, 4, 32, 0.05, seed=0), "auto"),
    # full-tile eager steps: after the round every learner's first layer is the
    # once-written global mean, not a replica row
    "mlp_eager_common_w1": (cases.case("mlp", 8, 4, 2, 2, B=32, IN=192, H=128, C=6, N=400, sigma=0.5, lr=0.05,
                                       seed=71), "eager"),
}


@pytest.mark.parametrize("name", sorted(EVAL_CASES))
def test_evaluate_matches_oracle(name, gpu_lib):
    """Loss and accuracy of replicas after a round, on training and held-out
    rows, against the oracle evaluating the same parameters: loss within
    1e-4 relative; hit counts equal except rows whose two largest logits are
    within 1e-5 (relative) of each other, where float32 may decide either way."""
    from paper_1903_05133_amd import HierAvg
    c, mode = EVAL_CASES[name]
    prob = cases.oracle_problem(c)
    with HierAvg(config=cases.native_config(c, mode)) as h:
        h.round()
        W = h.params().astype(np.float64)
        # more rows than one 4096-row chunk on the held-out split of the small cases
        plan = [(0, 0, min(c["N"], 300)), (c["P"] - 1, 1, 300 if c["IN"] > 1000 else 5000)]
        for replica, split, n in plan:
            print(f"[gpu case] evaluate {name} replica {replica} split {split} rows {n}", flush=True)
            loss, correct = h.evaluate(replica, split, n)
            want, wc, gaps = M.evaluate(prob, W[replica], np.arange(n), split)
            assert abs(loss - want) <= 1e-4 * max(1.0, abs(want)), (loss, want)
            assert abs(correct - wc) <= int(np.sum(gaps < 1e-5)), (correct, wc)
        with pytest.raises(Exception):
            h.evaluate(c["P"], 0, 10)
        with pytest.raises(Exception):
            h.evaluate(0, 0, c["N"] + 1)


def test_convergence_runner(gpu_lib):
    """The multi-round runner: one JSON line per round plus a summary; the
    global model's training loss falls over the rounds."""
    import io
    import json
    from paper_1903_05133_amd import convergence
    buf = io.StringIO()
    # softmax model with noisy data (std 5) and lr 0.005: the loss falls from
    # about 1.6 to 0.3 over three rounds (oracle)
    summ = convergence.run("t", 0, 4, 2, 2, 2, 8, 0.005, 3, 256, noise=5.0, out=buf)
    lines = [json.loads(x) for x in buf.getvalue().splitlines()]
    per_round = [x for x in lines if "summary" not in x]
    assert [x["round"] for x in per_round] == [1, 2, 3] and lines[-1]["summary"]
    assert [x["steps"] for x in per_round] == [4, 8, 12]
    assert per_round[-1]["train_loss"] < per_round[0]["train_loss"]
    assert 0.0 <= summ["final_test_acc"] <= 1.0


def test_convergence_runner_momentum_schedule_and_resume(gpu_lib, tmp_path):
    """Runner with momentum, a step-size drop and checkpoints: a run resumed
    from the state after round 2 reports exactly the uninterrupted round 3."""
    import io
    import json
    from paper_1903_05133_amd import convergence
    kw = dict(noise=5.0, momentum=0.9, weight_decay=1e-3, lr_drops=[(3, 0.001)])
    full, part, rest = io.StringIO(), io.StringIO(), io.StringIO()
    convergence.run("a", 0, 4, 2, 2, 2, 8, 0.005, 3, 256, out=full, **kw)
    ck = str(tmp_path / "state.npz")
    convergence.run("b", 0, 4, 2, 2, 2, 8, 0.005, 2, 256, out=part, checkpoint=ck, **kw)
    convergence.run("c", 0, 4, 2, 2, 2, 8, 0.005, 3, 256, out=rest, resume=ck, **kw)
    a = [json.loads(x) for x in full.getvalue().splitlines() if "summary" not in x]
    c = [json.loads(x) for x in rest.getvalue().splitlines() if "summary" not in x]
    assert [x["lr"] for x in a] == [0.005, 0.005, 0.001]
    assert [x["round"] for x in c] == [3]
    for key in ("steps", "lr", "train_loss", "train_acc", "test_loss", "test_acc"):
        assert c[0][key] == a[2][key], key


def _schedule_run(c, schedule, mode="auto"):
    """Rounds with a per-round (lr, B) schedule through set_lr / set_batch,
    and the oracle's rounds with the same Problem changed per round."""
    import dataclasses
    from paper_1903_05133_amd import HierAvg
    prob = cases.oracle_problem(c)
    mon = M.KinkMonitor(prob.H) if prob.kind == M.MLP else None
    st = M.create(prob)
    data = M.Dataset(prob) if prob.kind != M.AVERAGING else None
    done = []  # the per-round problems so far

    def replay(flips):
        s2 = M.create(prob)
        for pr_ in done:
            M.hieravg_round(pr_, s2, data, None, flips)
        return s2.W

    print(f"[gpu case] schedule {mode} {schedule} {c}", flush=True)
    with HierAvg(config=cases.native_config(c, mode)) as h:
        for lr, B in schedule:
            h.set_lr(lr)
            if prob.kind != M.AVERAGING:
                h.set_batch(B)
            h.round()
            pr = dataclasses.replace(prob, lr=lr, B=B)
            M.hieravg_round(pr, st, data, mon)
            done.append(pr)
            got = h.params()
            if prob.kind != M.AVERAGING:
                assert np.array_equal(h.last_indices().astype(np.int64), st.last_indices)
            assert _identical_rows(prob, got, w1_too=mode == "eager" and not cases.eager_means_once(dict(c, B=B))[0])
            ok, det = cases.branch_parity(pr, got, st.W, mon, replay)
            print(f"[gpu case] lr={lr} B={B} worst {det['worst']} flipped {det.get('flipped')}", flush=True)
            assert ok, det
        assert h.steps == len(schedule) * prob.T


# Eager rounds of full-tile steps (B = 32 or 64) write the round-end global
# mean of the first layer once, to a common copy, and (S * B too large for the
# fused mean step) the block-end cluster means once, to cluster copies; the
# step after a mean reads its old first layer there.  Delayed rounds in
# between (AUTO, B <= 32 with K1 = 3, H = 128) start from that copy too.
ONCE_CASES = {
    "global_copy_schedule": (cases.case("mlp", 8, 4, 3, 2, B=64, IN=192, H=128, C=6, N=500, sigma=0.5, lr=0.05,
                                        seed=73), [(0.05, 64), (0.05, 64), (0.05, 32), (0.05, 64), (0.05, 64),
                                                   (0.05, 16)]),
    "cluster_copies_schedule": (cases.case("mlp", 16, 8, 3, 2, B=64, IN=192, H=128, C=6, N=600, sigma=0.5,
                                           lr=0.05, seed=74), [(0.05, 64), (0.05, 64), (0.05, 32), (0.05, 64)]),
    # every step ends a block: each update with the mean reads the copy the
    # previous one wrote (the first from the common copy)
    "cluster_copies_K1_1": (cases.case("mlp", 16, 8, 1, 3, B=64, IN=192, H=128, C=6, N=600, sigma=0.5, lr=0.05,
                                       seed=75), None),
    "global_copy_B32": (cases.case("mlp", 4, 2, 2, 3, B=32, IN=128, H=64, C=4, N=300, sigma=0.5, lr=0.05, seed=76),
                        None),
}


@pytest.mark.parametrize("name", sorted(ONCE_CASES))
def test_eager_means_written_once(name, gpu_lib):
    c, schedule = ONCE_CASES[name]
    if schedule is None:
        got, idx, steps = _run_gpu(c, rounds=2, mode="eager")
        _check(c, got, idx, *_oracle(c, 2), mode="eager")
    else:
        _schedule_run(c, schedule, "auto")


@pytest.mark.parametrize("mode", ["auto", "eager"])
def test_lr_schedule_matches_oracle(mode, gpu_lib):
    c = cases.case("mlp", 4, 2, 2, 2, B=12, IN=150, H=70, C=6, N=200, sigma=0.5, lr=0.1, seed=21)
    _schedule_run(c, [(0.1, 12), (0.05, 12), (0.02, 12)], mode)


def test_lr_schedule_softmax_and_momentum(gpu_lib):
    c = cases.case("softmax", 4, 2, 2, 1, B=10, IN=90, C=7, N=100, lr=0.2, seed=22)
    _schedule_run(c, [(0.2, 10), (0.07, 10)], "auto")
    c = cases.case("averaging", 4, 2, 2, 2, IN=777, lr=0.1, momentum=0.9, seed=23)
    _schedule_run(c, [(0.1, 1), (0.03, 1)], "auto")


def test_batch_schedule_switches_update_modes(gpu_lib):
    """B = 40 updates eagerly (beyond the delayed path's 32), B = 16 and 9
    take delayed updates; each switch back to eager first copies replica 0's
    common first layer to every learner.  Indices: the first B draws of a
    step do not depend on B."""
    c = cases.case("mlp", 4, 2, 2, 2, B=40, IN=150, H=70, C=6, N=300, sigma=0.5, lr=0.05, seed=24)
    _schedule_run(c, [(0.05, 40), (0.05, 16), (0.05, 40), (0.05, 9), (0.05, 16), (0.05, 33)], "auto")


K_GLOBAL_CASES = {
    "mlp_T5_K1_2": cases.case("mlp", 4, 2, 2, 1, B=8, IN=100, H=70, C=5, N=200, sigma=0.5, lr=0.1, seed=25,
                              k_global=5),
    "mlp_T7_K1_3_S4": cases.case("mlp", 8, 4, 3, 1, B=6, IN=64, H=40, C=3, N=90, sigma=0.5, lr=0.1, seed=26,
                                 k_global=7),
    "softmax_T3_K1_2": cases.case("softmax", 4, 4, 2, 1, B=5, IN=40, C=4, N=50, lr=0.2, seed=27, k_global=3),
    "averaging_T5_K1_2": cases.case("averaging", 4, 2, 2, 1, IN=999, lr=0.1, momentum=0.9, seed=28, k_global=5),
}


@pytest.mark.parametrize("name", sorted(K_GLOBAL_CASES))
def test_global_interval_not_multiple_of_k1(name, gpu_lib):
    """A round of k_global steps with a shorter last block (non-integer beta)."""
    c = K_GLOBAL_CASES[name]
    got, idx, steps = _run_gpu(c, rounds=2)
    assert steps == 2 * c["k_global"]
    if idx is not None:
        assert idx.shape == (c["k_global"], c["P"], c["B"])
    _check(c, got, idx, *_oracle(c, 2))


# ---------------------------------------------------- momentum and weight decay
MOMENTUM_CASES = {
    # small-class head and the update GEMM of the first layer
    "mlp_head_mom_wd": cases.case("mlp", 4, 2, 2, 2, B=12, IN=150, H=70, C=6, N=200, sigma=0.5, lr=0.05,
                                  momentum=0.9, weight_decay=0.01, seed=31),
    # 32 class slots of the small-class head, three sample groups
    "mlp_head32_mom_wd": cases.case("mlp", 4, 2, 2, 2, B=40, IN=100, H=300, C=20, N=300, sigma=0.5, lr=0.05,
                                    momentum=0.9, weight_decay=0.01, seed=64),
    # more than 32 classes: layer-2 forward GEMM and the update GEMM with bias
    "mlp_large_c_mom": cases.case("mlp", 4, 4, 2, 2, B=20, IN=130, H=80, C=40, N=300, sigma=0.5, lr=0.05,
                                  momentum=0.8, seed=32),
    "softmax_mom_wd": cases.case("softmax", 6, 3, 2, 2, B=9, IN=70, C=11, N=80, lr=0.1, momentum=0.9,
                                 weight_decay=0.02, seed=33),
    "mlp_avg_buffers": cases.case("mlp", 8, 4, 2, 2, B=8, IN=64, H=40, C=5, N=100, sigma=0.5, lr=0.05,
                                  momentum=0.9, weight_decay=0.005, avg_momentum=True, seed=34),
    "softmax_decay_only": cases.case("softmax", 4, 2, 3, 1, B=7, IN=50, C=4, N=60, lr=0.1, weight_decay=0.05,
                                     seed=35),
    "averaging_wd_avg_buffers": cases.case("averaging", 4, 2, 2, 2, IN=1001, lr=0.1, momentum=0.9,
                                           weight_decay=0.01, avg_momentum=True, seed=36),
}


# MLP cases the delayed schedule takes (plain buffers, B <= 32): heavy-ball blocks
HB_DELAYED = {
    "mlp_head_mom_wd": MOMENTUM_CASES["mlp_head_mom_wd"],
    "mlp_large_c_mom": MOMENTUM_CASES["mlp_large_c_mom"],
    # decay without momentum (no buffers): scalar block coefficients only
    "mlp_decay_only": cases.case("mlp", 4, 2, 3, 2, B=10, IN=90, H=70, C=5, N=100, sigma=0.5, lr=0.1,
                                 weight_decay=0.02, seed=37),
    # one block per round: the cluster updates and the separate mean of the copies
    "mlp_mom_one_block": cases.case("mlp", 6, 3, 3, 1, B=8, IN=64, H=40, C=4, N=80, sigma=0.5, lr=0.05,
                                    momentum=0.9, seed=38),
    # W1 with 512 output tiles: the last block's global update from the mean of the copies and buffers
    "mlp_wide_mom": cases.case("mlp", 4, 2, 2, 2, B=16, IN=8192, H=512, C=6, N=200, sigma=0.5, lr=0.02,
                               momentum=0.9, weight_decay=0.001, seed=39),
    # K1 = 5: four earlier steps' corrections per block, 20 to 32 classes
    "mlp_mom_long_block": cases.case("mlp", 4, 2, 5, 2, B=12, IN=100, H=96, C=20, N=150, sigma=0.5, lr=0.05,
                                     momentum=0.5, weight_decay=0.005, seed=40),
}


def _momentum_run(c, mode, rounds=2):
    from paper_1903_05133_amd import HierAvg
    print(f"[gpu case] momentum {mode} {c}", flush=True)
    with HierAvg(config=cases.native_config(c, mode)) as h:
        h.profile(True)
        for _ in range(rounds):
            h.round()
        stats = h.profile_read()
        got = h.params()
        vgot = h.momentum() if c["momentum"] > 0 or c["kind"] == "averaging" else None
        idx = h.last_indices() if c["kind"] != "averaging" else None
    return got, vgot, idx, stats


def _momentum_check(c, got, vgot, idx, mode, rounds=2):
    st, mon, rerun = _oracle(c, rounds)
    det = _check(c, got, idx, st, mon, rerun, mode=mode)
    if vgot is not None:
        prob = cases.oracle_problem(c)
        if det.get("flipped"):  # the buffers of the run whose branch the parameters matched
            st = M.run(prob, rounds, flips=frozenset(d[:4] for d in det["flipped"]))
        ok, det = cases.parity_report(prob, vgot, st.V)
        print(f"[gpu case] buffers: worst block error {det['worst']}", flush=True)
        assert ok, det
        if c["avg_momentum"]:
            assert np.array_equal(vgot, np.repeat(vgot[:1], vgot.shape[0], axis=0))


@pytest.mark.parametrize("name", sorted(MOMENTUM_CASES))
def test_momentum_and_weight_decay_match_oracle(name, gpu_lib):
    """Heavy-ball buffers and L2 decay in every update kernel, EAGER: parameters
    and buffers after two rounds against the oracle."""
    c = MOMENTUM_CASES[name]
    got, vgot, idx, stats = _momentum_run(c, "eager")
    assert "fwd1_block_gemm" not in stats and "step1_gemm" not in stats
    if c["avg_momentum"] and c["momentum"] > 0:
        assert "momentum_buffer_global_mean" in stats
    _momentum_check(c, got, vgot, idx, "eager")


@pytest.mark.parametrize("name", sorted(HB_DELAYED))
def test_momentum_and_weight_decay_delayed(name, gpu_lib):
    """Heavy-ball blocks: the first layer of every learner after k steps of
    heavy-ball SGD with decay is p_k W + q_k V + sum u G^T X (scalars from the
    recurrence), so the block forward, the Gram corrections and the block-end
    updates of the parameters and of every learner's buffer keep their GEMM
    form.  AUTO takes this schedule; parameters and buffers after two rounds
    against the oracle."""
    c = HB_DELAYED[name]
    got, vgot, idx, stats = _momentum_run(c, "auto")
    assert "fwd1_block_gemm" in stats and "scale_errors" in stats
    assert ("buffer_update_gemm" in stats) == (c["momentum"] > 0)
    assert ("fwd1_block_gemm_v" in stats) == (c["momentum"] > 0)
    _momentum_check(c, got, vgot, idx, "delayed")


@pytest.mark.parametrize("mode", ["delayed", "eager"])
def test_named_mlp_workload_momentum(mode, gpu_lib):
    """MLP 3072 -> 512 -> 10, P=16 S=4 K1=4 K2=4 B=32, lr 0.05 with momentum
    0.9 and weight decay 5e-4 (buffers per learner), one full round in both
    schedules: parameters and buffers against the oracle."""
    c = cases.named("mlp_3072_512_10", 16, 4, 4, 4, 32, 0.05, seed=0)
    c.update(momentum=0.9, weight_decay=5e-4)
    got, vgot, idx, stats = _momentum_run(c, mode, rounds=1)
    assert ("buffer_update_gemm" in stats) == (mode == "delayed")
    _momentum_check(c, got, vgot, idx, mode, rounds=1)


def test_momentum_checkpoint_resume(gpu_lib):
    """params + momentum buffers copied into a fresh handle continue the
    trajectory: the round after equals the oracle's second round."""
    from paper_1903_05133_amd import HierAvg
    c = MOMENTUM_CASES["mlp_head_mom_wd"]
    with HierAvg(config=cases.native_config(c)) as h:
        h.round()
        w, v = h.params(), h.momentum()
    with HierAvg(config=cases.native_config(c)) as h2:
        with pytest.raises(Exception):
            h2.set_momentum(v[:1])
        h2.set_params(w)
        h2.set_momentum(v)
        assert np.array_equal(h2.momentum(), v)
        # the oracle's second round draws from step T on; the fresh handle from step 0
        h2.round()
        got = h2.params()
    prob = cases.oracle_problem(c)
    st = M.create(prob)
    st.W, st.V = w.astype(np.float64), v.astype(np.float64)
    M.hieravg_round(prob, st)
    ok, det = cases.parity_report(prob, got, st.W)
    assert ok, det


def test_no_buffers_without_momentum(gpu_lib):
    from paper_1903_05133_amd import HierAvg
    with HierAvg(config=cases.native_config(MOMENTUM_CASES["softmax_decay_only"])) as h:
        with pytest.raises(Exception):
            h.momentum()


@pytest.mark.parametrize("name", ["delayed_mlp", "momentum_softmax", "eager_unequal_rows", "eager_common_copy"])
def test_checkpoint_resume_is_exact(name, gpu_lib, tmp_path):
    """save() after one round, load() into a fresh handle, one more round:
    bit for bit the second round of the uninterrupted run (same step counter,
    parameters, buffers and, for equal first-layer rows, the same schedule)."""
    from paper_1903_05133_amd import HierAvg
    c = {"delayed_mlp": SMALL["mlp_ragged"], "momentum_softmax": MOMENTUM_CASES["softmax_mom_wd"],
         "eager_unequal_rows": SMALL["mlp_ragged"], "eager_common_copy": ONCE_CASES["cluster_copies_schedule"][0]}[name]
    # eager_common_copy: eager rounds that leave the first layer in the common copy
    cfg = cases.native_config(c, "eager" if name == "eager_common_copy" else "auto")
    with HierAvg(config=cfg) as h:
        h.round()
        if name == "eager_unequal_rows":  # rows that differ: the resumed round must run eager
            w = h.params()
            w[1, 0] += 1.0
            h.set_params(w)
        h.save(str(tmp_path / "ck.npz"))
        h.round()
        ref, steps = h.params(), h.steps
        vref = h.momentum() if c["momentum"] > 0 else None
    with HierAvg(config=cfg) as h2:
        h2.load(str(tmp_path / "ck.npz"))
        h2.profile(True)
        h2.round()
        stats = h2.profile_read()
        assert h2.steps == steps
        assert np.array_equal(h2.params(), ref)
        if vref is not None:
            assert np.array_equal(h2.momentum(), vref)
    if name == "delayed_mlp":
        assert "fwd1_block_gemm" in stats
    if name == "eager_unequal_rows":
        assert "fwd1_block_gemm" not in stats


EDGE_CASES = {
    # many learners in one cluster (S = P = 512), one step per round
    "softmax_512_learners": cases.case("softmax", 512, 512, 1, 1, B=2, IN=8, C=3, N=16, lr=0.1, seed=51),
    # many learners in clusters of 2
    "mlp_256_learners_S2": cases.case("mlp", 256, 2, 2, 1, B=3, IN=10, H=5, C=2, N=40, lr=0.1, seed=52),
    # large minibatch (eager, several 16-row batch tiles and forward chunks)
    "mlp_batch_1000": cases.case("mlp", 2, 2, 1, 2, B=1000, IN=40, H=20, C=3, N=5000, sigma=0.5, lr=0.05, seed=53),
    # one input feature, one hidden unit, two classes
    "mlp_tiny_dims": cases.case("mlp", 4, 2, 2, 2, B=5, IN=1, H=1, C=2, N=9, lr=0.2, seed=54),
    # a long round: 100 steps, blocks of 7 (the last one of 2 steps)
    "softmax_100_steps": cases.case("softmax", 4, 2, 7, 1, B=4, IN=12, C=5, N=30, lr=0.05, seed=55, k_global=100),
    # averaging kind with 1024 replicas of a short vector
    "averaging_1024_rows": cases.case("averaging", 1024, 32, 1, 2, IN=300, lr=0.1, momentum=0.9, seed=56),
}


@pytest.mark.parametrize("name", sorted(EDGE_CASES))
def test_edge_shapes_match_oracle(name, gpu_lib):
    c = EDGE_CASES[name]
    got, idx, steps = _run_gpu(c, rounds=1)
    assert steps == (c["k_global"] or c["K1"] * c["K2"])
    _check(c, got, idx, *_oracle(c, 1))


@pytest.mark.parametrize("kind", ["softmax", "mlp_common_w1"])
def test_divergence_check(kind, gpu_lib):
    """hieravg_check_finite: finite replicas pass; a step size far too large
    for the data drives them to inf/NaN, which the check reports (MLP: with
    the first layer in the once-written common copy)."""
    from paper_1903_05133_amd import HierAvg
    if kind == "softmax":
        ok, mode = cases.case("softmax", 4, 2, 2, 1, B=8, IN=20, C=3, N=40, lr=0.1, seed=61), "auto"
    else:
        ok, mode = cases.case("mlp", 4, 2, 2, 2, B=32, IN=64, H=64, C=3, N=100, sigma=0.5, lr=0.1, seed=72), "eager"
    with HierAvg(config=cases.native_config(ok, mode)) as h:
        h.round()
        assert h.finite()
        h.set_lr(3.0e38)
        for _ in range(3):
            h.round()
        assert not h.finite()


def test_forced_allocation_failures_leave_no_broken_state(gpu_lib, monkeypatch):
    """Every device allocation of create made to fail in turn (debug hook):
    create returns NULL with a message naming the buffer, nothing leaks into
    the next handle, which computes the oracle's round."""
    import ctypes
    from paper_1903_05133_amd import HierAvg, native
    c = cases.case("mlp", 4, 2, 2, 2, B=8, IN=50, H=20, C=3, N=40, sigma=0.5, lr=0.1, seed=62)
    L = native.lib()
    failed = 0
    for n in range(1, 40):
        monkeypatch.setenv("HIERAVG_FAIL_ALLOC", str(n))
        cfg = cases.native_config(c)
        h = L.hieravg_create_config(ctypes.byref(cfg))
        if not h:
            assert "HIERAVG_FAIL_ALLOC" in L.hieravg_last_error().decode()
            failed += 1
        else:
            L.hieravg_destroy(h)
            break
    assert failed >= 5
    monkeypatch.delenv("HIERAVG_FAIL_ALLOC")
    got, idx, _ = _run_gpu(c)
    _check(c, got, idx, *_oracle(c))
