"""Pins of the oracle's Algorithm 1 (Sec. 3.1) against things other than itself.

* the special cases Sec. 3.1 names: K1 = K2 = 1 is synchronous parallel SGD
  (one minibatch-SGD step on the union of the P minibatches); S = 1 is K-AVG;
  K2 = K1 (one local block per round) is K-AVG;
* P = 1 is plain minibatch SGD;
* the references for those cases are written with torch.autograd and
  torch.optim.SGD on the CPU in float64 (a library routine, not the oracle's
  hand-written gradient);
* the worker-average dynamics stated in the proof of Thm 3.1;
* the pure-noise drift variance implied by the decomposition in Lemma 1;
* finite differences and a case worked by hand.
"""

import numpy as np
import pytest
import torch

from oracle import method as M
from oracle import rng

torch.set_default_dtype(torch.float64)


def small(kind, P, S, K1, K2, B=4, lr=0.1, seed=3, **kw):
    if kind == M.SOFTMAX:
        base = dict(IN=20, C=5, N=64, sigma=1.0)
    elif kind == M.MLP:
        base = dict(IN=20, H=12, C=5, N=64, sigma=0.5)
    else:
        base = dict(IN=1000, momentum=0.9)
    base.update(kw)
    return M.Problem(kind, P, S, K1, K2, B, lr=lr, seed=seed, **base)


# ------------------------------------------------------------- torch references
def torch_params(p, row):
    blk = M.unpack(p, np.array(row, dtype=np.float64))
    return {k: torch.tensor(v.copy(), requires_grad=True) for k, v in blk.items()}


def torch_loss(p, prm, X, y):
    X = torch.tensor(X)
    y = torch.tensor(y)
    if p.kind == M.SOFTMAX:
        z = X @ prm["W"].T + prm["b"]
    else:
        a = torch.relu(X @ prm["W1"].T + prm["b1"])
        z = a @ prm["W2"].T + prm["b2"]
    return torch.nn.functional.cross_entropy(z, y)


def flatten(p, prm):
    return np.concatenate([prm[name].detach().numpy().reshape(-1) for name, _ in M.segments(p)])


def torch_sgd_run(p, row, learner, t0, steps):
    """`steps` steps of torch.optim.SGD for one learner on its own draws."""
    prm = torch_params(p, row)
    opt = torch.optim.SGD(list(prm.values()), lr=p.lr64)
    for t in range(t0, t0 + steps):
        X, y = rng.data_rows(p.seed, rng.draw_indices(p.seed, learner, t, p.B, p.N), p.IN, p.C, p.sigma)
        opt.zero_grad()
        torch_loss(p, prm, X, y).backward()
        opt.step()
    return flatten(p, prm)


def kavg_reference(p, rounds_K, rounds):
    """K-AVG: every learner runs K SGD steps alone, then all average; repeated."""
    w = M.initial_replica(p)
    t = 0
    for _ in range(rounds):
        rows = [torch_sgd_run(p, w, j, t, rounds_K) for j in range(p.P)]
        w = np.mean(rows, axis=0)
        t += rounds_K
    return w


def relerr(a, b):
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


# ---------------------------------------------------------------------- pins
@pytest.mark.parametrize("kind", [M.SOFTMAX, M.MLP])
def test_finite_differences(kind):
    p = small(kind, 1, 1, 1, 1, B=3)
    r = np.random.default_rng(0)
    row = M.initial_replica(p) + 0.3 * r.standard_normal(p.D)
    X, y = rng.data_rows(p.seed, [1, 5, 9], p.IN, p.C, p.sigma)
    g = M.minibatch_gradient(p, row, X, y)
    eps = 1e-6
    for i in r.choice(p.D, size=40, replace=False):
        e = np.zeros(p.D)
        e[i] = eps
        fd = (M.loss(p, row + e, X, y) - M.loss(p, row - e, X, y)) / (2 * eps)
        assert abs(fd - g[i]) < 1e-7 * max(1.0, abs(fd)), (i, fd, g[i])


@pytest.mark.parametrize("kind", [M.SOFTMAX, M.MLP])
def test_gradient_matches_autograd(kind):
    p = small(kind, 1, 1, 1, 1, B=6)
    row = M.initial_replica(p) + 0.2 * np.random.default_rng(1).standard_normal(p.D)
    X, y = rng.data_rows(p.seed, np.arange(6) * 7, p.IN, p.C, p.sigma)
    prm = torch_params(p, row)
    torch_loss(p, prm, X, y).backward()
    want = np.concatenate([prm[n].grad.numpy().reshape(-1) for n, _ in M.segments(p)])
    assert relerr(M.minibatch_gradient(p, row, X, y), want) < 1e-12


def test_hand_worked_softmax_step():
    # IN=2, C=2, one sample x=(1,2), y=0, zero weights: logits 0, p=(1/2,1/2),
    # delta=(-1/2, 1/2); grad W = delta x^T, grad b = delta; lr 0.1.
    p = M.Problem(M.SOFTMAX, 1, 1, 1, 1, 1, IN=2, C=2, N=1, lr=0.1)
    g = M.minibatch_gradient(p, np.zeros(6), np.array([[1.0, 2.0]]), np.array([0]))
    assert np.allclose(g, [-0.5, -1.0, 0.5, 1.0, -0.5, 0.5], rtol=0, atol=1e-15)
    w = np.zeros(6) - p.lr64 * g
    lr = float(np.float32(0.1))
    assert np.allclose(w, lr * np.array([0.5, 1.0, -0.5, -1.0, 0.5, -0.5]), rtol=0, atol=1e-15)


@pytest.mark.parametrize("kind", [M.SOFTMAX, M.MLP])
@pytest.mark.parametrize("S", [1, 2, 4])
def test_k1_k2_one_is_synchronous_sgd(kind, S):
    """K1 = K2 = 1: one round is one SGD step with batch P*B on the union of
    the P minibatches (Sec. 3.1, synchronous parallel SGD)."""
    p = small(kind, 4, S, 1, 1)
    st = M.run(p, 1)
    w0 = M.initial_replica(p)
    idx = np.concatenate([rng.draw_indices(p.seed, j, 0, p.B, p.N) for j in range(p.P)])
    X, y = rng.data_rows(p.seed, idx, p.IN, p.C, p.sigma)
    prm = torch_params(p, w0)
    torch_loss(p, prm, X, y).backward()
    want = flatten(p, prm) - p.lr64 * np.concatenate([prm[n].grad.numpy().reshape(-1) for n, _ in M.segments(p)])
    for j in range(p.P):
        assert relerr(st.W[j], want) < 1e-12


@pytest.mark.parametrize("kind", [M.SOFTMAX, M.MLP])
def test_s_one_is_kavg(kind):
    """S = 1: a round is K-AVG with K = K1*K2 (Sec. 3.1)."""
    p = small(kind, 3, 1, 2, 3)
    st = M.run(p, 1)
    want = kavg_reference(p, p.K1 * p.K2, 1)
    assert relerr(st.W[0], want) < 1e-12


@pytest.mark.parametrize("S", [1, 2, 4])
def test_single_block_is_kavg(S):
    """K2 = 1 block per round (the paper's K2 = K1): K-AVG with K = K1, for
    any S, because the mean of equal-size group means is the global mean."""
    p = small(M.MLP, 4, S, 3, 1)
    st = M.run(p, 2)
    want = kavg_reference(p, 3, 2)
    assert relerr(st.W[1], want) < 1e-12


def test_s_equals_p_is_repeated_kavg():
    """S = P: every local mean is a global mean, so a round is K2 rounds of
    K-AVG with K = K1."""
    p = small(M.MLP, 3, 3, 2, 3)
    st = M.run(p, 1)
    want = kavg_reference(p, 2, 3)
    assert relerr(st.W[2], want) < 1e-12


@pytest.mark.parametrize("kind", [M.SOFTMAX, M.MLP])
def test_single_learner_is_minibatch_sgd(kind):
    p = small(kind, 1, 1, 3, 2)
    st = M.run(p, 2)
    want = torch_sgd_run(p, M.initial_replica(p), 0, 0, 12)
    assert relerr(st.W[0], want) < 1e-12


def test_named_softmax_workload_first_steps():
    """The 3072->10 workload shape, P = 1, against torch.optim.SGD."""
    p = M.preset(0, 1, 1, 2, 1, 0.05, 8, 0)
    st = M.run(p, 1)
    want = torch_sgd_run(p, M.initial_replica(p), 0, 0, 2)
    assert relerr(st.W[0], want) < 1e-12


def test_momentum_kavg_matches_torch_sgd_momentum():
    """Averaging-only workload with S = 1 (K-AVG): within a round each learner
    is torch.optim.SGD with momentum on its given gradients; the round ends
    with the mean of the parameters while every learner keeps its own buffer."""
    p = small(M.AVERAGING, 3, 1, 2, 2, lr=0.1, momentum=0.9)
    st = M.run(p, 2)
    w0 = M.initial_replica(p)
    first = [_torch_momentum_rows(p, w0, np.zeros(p.IN), j) for j in range(p.P)]
    mean1 = np.mean([w for w, _ in first], axis=0)
    second = [_torch_momentum_rows(p, mean1, v, j)[0] for j, (_, v) in enumerate(first)]
    assert relerr(st.W[0], np.mean(second, axis=0)) < 1e-12
    assert relerr(st.V[1], _torch_momentum_rows(p, mean1, first[1][1], 1)[1]) < 1e-12


def _torch_momentum_rows(p, w0, v0, j):
    w = torch.tensor(np.array(w0), requires_grad=True)
    opt = torch.optim.SGD([w], lr=p.lr64, momentum=p.mu64)
    if np.any(v0):
        opt.state[w]["momentum_buffer"] = torch.tensor(np.array(v0))
    for k in range(p.K1 * p.K2):
        w.grad = torch.tensor(rng.given_gradients(p.seed, k, j, p.IN, p.grad_std))
        opt.step()
    return w.detach().numpy(), opt.state[w]["momentum_buffer"].numpy().copy()


def test_means_make_replicas_identical_and_are_idempotent():
    p = small(M.MLP, 8, 4, 2, 2)
    st = M.create(p)
    data = M.Dataset(p)
    M.sgd_step_all(p, data, st)
    W = M.local_average(st.W, 4)
    for q in range(2):
        g = W[4 * q:4 * q + 4]
        assert np.array_equal(g, np.repeat(g[:1], 4, axis=0))
    assert np.array_equal(M.local_average(W, 4), W)
    G = M.global_average(st.W)
    assert np.array_equal(G, np.repeat(G[:1], 8, axis=0))
    assert not np.array_equal(G[0], W[0])


def test_worker_average_dynamics():
    """Proof of Thm 3.1: a step moves the worker average by
    -lr/(PB) * sum_j sum_s grad f(w^j; xi^j_s); a local mean leaves it fixed."""
    p = small(M.MLP, 4, 2, 1, 1)
    st = M.create(p)
    data = M.Dataset(p)
    M.sgd_step_all(p, data, st)
    st.W = st.W + 0.05 * np.random.default_rng(2).standard_normal(st.W.shape)  # distinct replicas
    before = st.W.mean(axis=0)
    total = np.zeros(p.D)
    for j in range(p.P):
        X, y = rng.data_rows(p.seed, rng.draw_indices(p.seed, j, st.t, p.B, p.N), p.IN, p.C, p.sigma)
        prm = torch_params(p, st.W[j])
        (torch_loss(p, prm, X, y) * p.B).backward()   # sum over s of grad f
        total += np.concatenate([prm[n].grad.numpy().reshape(-1) for n, _ in M.segments(p)])
    M.sgd_step_all(p, data, st)
    after = st.W.mean(axis=0)
    assert relerr(after - before, -p.lr64 / (p.P * p.B) * total) < 1e-10
    assert relerr(M.local_average(st.W, p.S).mean(axis=0), after) < 1e-14


def test_pure_noise_drift_variance():
    """Averaging-only, no momentum, i.i.d. given gradients of std sg: after
    eta completed blocks and t further steps every replica has drifted from
    the round's start by a mean-zero vector with per-coordinate variance
    lr^2 sg^2 (t + K1*eta/S) -- the two terms of the decomposition in Lemma 1
    (its own steps, and the S-fold averaged steps of earlier blocks).  After
    the global mean: lr^2 sg^2 K1 K2 / P."""
    P, S, K1, K2, D = 8, 4, 2, 3, 400000
    p = M.Problem(M.AVERAGING, P, S, K1, K2, IN=D, lr=0.1, momentum=0.0, grad_std=0.01, seed=5)
    st = M.create(p)
    w0 = st.W[0].copy()
    unit = p.lr64 ** 2 * float(np.float32(0.01)) ** 2
    tol = 0.03
    for eta in range(K2):
        for t in range(K1):
            v = np.mean((st.W - w0) ** 2)
            if eta or t:
                assert abs(v / (unit * (t + K1 * eta / S)) - 1) < tol, (eta, t)
            M.sgd_step_all(p, None, st)
        st.W = M.local_average(st.W, S)
    st.W = M.global_average(st.W)
    v = np.mean((st.W[0] - w0) ** 2)
    assert abs(v / (unit * K1 * K2 / P) - 1) < 2 * tol


@pytest.mark.parametrize("S", [2, 3])
def test_groups_are_contiguous_and_independent(S):
    """Before the global mean, the replicas of group q = {qS, ..., qS+S-1}
    follow K-AVG among those S learners alone (local averaging within a
    local cluster, Algorithm 1); no other learner influences them."""
    P, K1, K2 = 2 * S, 2, 3
    p = small(M.MLP, P, S, K1, K2)
    st = M.create(p)
    data = M.Dataset(p)
    for _ in range(K2):
        for _ in range(K1):
            M.sgd_step_all(p, data, st)
        st.W = M.local_average(st.W, S)
    for q in range(P // S):
        w = M.initial_replica(p)
        for b in range(K2):
            w = np.mean([torch_sgd_run(p, w, j, b * K1, K1) for j in range(q * S, q * S + S)], axis=0)
        for j in range(q * S, q * S + S):
            assert relerr(st.W[j], w) < 1e-12


def test_averaging_column_sampling_is_exact():
    """Restricting the averaging-only workload to a subset of coordinates
    gives exactly those coordinates of the full run."""
    p = small(M.AVERAGING, 4, 2, 2, 2, lr=0.1, momentum=0.9, IN=777)
    full = M.run(p, 2)
    cols = np.array([0, 5, 300, 776])
    part = M.run(p, 2, cols=cols)
    assert np.array_equal(part.W, full.W[:, cols])
    assert np.array_equal(part.V, full.V[:, cols])


# ---------------------------------------------------------------- evaluation
def test_evaluate_matches_torch_cross_entropy_and_argmax():
    """The evaluation loss is torch's softmax cross-entropy (float64, CPU) of
    the model's logits, and the count is torch's argmax accuracy."""
    import torch
    for kind in (M.MLP, M.SOFTMAX):
        p = M.Problem(kind, 2, 1, 1, 1, 4, IN=20, H=9, C=6, N=50, sigma=0.7, seed=21)
        st = M.create(p)
        row = st.W[0] + np.random.default_rng(0).normal(0, 0.3, p.D)  # off the initial point
        rows = np.arange(37)
        for split in (0, 1):
            loss, correct, gaps = M.evaluate(p, row, rows, split, chunk=10)
            X, y = rng.data_rows(p.seed, rows, p.IN, p.C, p.sigma, split)
            blk = M.unpack(p, row)
            Xt = torch.tensor(X)
            if kind == M.SOFTMAX:
                z = Xt @ torch.tensor(blk["W"]).T + torch.tensor(blk["b"])
            else:
                a = torch.relu(Xt @ torch.tensor(blk["W1"]).T + torch.tensor(blk["b1"]))
                z = a @ torch.tensor(blk["W2"]).T + torch.tensor(blk["b2"])
            want = torch.nn.functional.cross_entropy(z, torch.tensor(y)).item()
            assert abs(loss - want) <= 1e-12 * max(1.0, abs(want))
            assert correct == int((z.argmax(dim=1) == torch.tensor(y)).sum())
            assert gaps.shape == (37,) and np.all(gaps >= 0)


def test_held_out_rows_recipe():
    """Split 1 keeps the class means and takes its own label and noise
    streams; one element written out from the definition."""
    seed, IN, C, sigma = 4, 16, 3, 0.5
    X0, y0 = rng.data_rows(seed, np.arange(200), IN, C, sigma, 0)
    X1, y1 = rng.data_rows(seed, np.arange(200), IN, C, sigma, 1)
    assert not np.array_equal(y0, y1) and not np.array_equal(X0, X1)
    i, d = 17, 5
    key_n = rng.stream_key(seed, rng.TAG_TEST_NOISE)
    z = rng.normal_surrogate(key_n, np.array([i * IN + d], dtype=np.uint64))[0]
    mu = rng.class_means(seed, np.arange(C), IN)
    assert y1[i] == rng.h_scalar(rng.stream_key(seed, rng.TAG_TEST_LABEL), i) % C
    assert X1[i, d] == float(np.float32(mu[y1[i], d] + sigma * z))


# ------------------------------------------------ generalised global interval
@pytest.mark.parametrize("kind", [M.SOFTMAX, M.MLP])
def test_global_interval_in_steps_with_s_one_is_kavg(kind):
    """S = 1 with a global interval of T = 5 steps and K1 = 2 (a non-integer
    beta): local means are identities, so a round is K-AVG with K = 5
    (torch.optim.SGD per learner, then the mean)."""
    p = small(kind, 3, 1, 2, 1, k_global=5)
    st = M.run(p, 2)
    want = kavg_reference(p, 5, 2)
    for j in range(p.P):
        assert relerr(st.W[j], want) < 1e-12


def test_global_interval_in_steps_with_s_equal_p():
    """S = P, K1 = 2, T = 5: the local mean is the global mean, so a round is
    K-AVG rounds of 2, 2 and 1 steps (each ends with the mean of all P)."""
    p = small(M.MLP, 3, 3, 2, 1, k_global=5)
    st = M.run(p, 1)
    w = M.initial_replica(p)
    t = 0
    for K in (2, 2, 1):
        rows = [torch_sgd_run(p, w, j, t, K) for j in range(p.P)]
        w = np.mean(rows, axis=0)
        t += K
    for j in range(p.P):
        assert relerr(st.W[j], w) < 1e-12


def test_global_interval_equal_to_blocks_is_the_block_round():
    """T = K1 * K2 given as a step count reproduces the block round bit for bit."""
    a = M.run(small(M.MLP, 4, 2, 2, 3), 1)
    b = M.run(small(M.MLP, 4, 2, 2, 3, k_global=6), 1)
    assert np.array_equal(a.W, b.W) and np.array_equal(a.last_indices, b.last_indices)


# ------------------------------------------------ momentum and weight decay (MLP/softmax)
def torch_schedule_reference(p, rounds):
    """Algorithm 1's schedule with torch.optim.SGD (momentum, weight_decay,
    no dampening, no Nesterov) as every learner's step: one optimizer per
    learner for the whole run; after every K1 steps each group of S learners
    takes the mean of its parameters (and of its momentum buffers when
    avg_momentum), at the end of a round all P learners do."""
    w0 = M.initial_replica(p)
    prms = [torch_params(p, w0) for _ in range(p.P)]
    opts = [torch.optim.SGD(list(prm.values()), lr=p.lr64, momentum=p.mu64, weight_decay=p.wd64) for prm in prms]

    def average(groups):
        for grp in groups:
            for name in prms[0]:
                mean = torch.stack([prms[j][name].detach() for j in grp]).mean(dim=0)
                for j in grp:
                    prms[j][name].data.copy_(mean)
            if p.avg_momentum:
                for i, _ in enumerate(prms[0]):
                    bufs = [opts[j].state[list(prms[j].values())[i]]["momentum_buffer"] for j in grp]
                    mean = torch.stack(bufs).mean(dim=0)
                    for b in bufs:
                        b.copy_(mean)

    t = 0
    for _ in range(rounds):
        for tt in range(p.T):
            for j in range(p.P):
                X, y = rng.data_rows(p.seed, rng.draw_indices(p.seed, j, t, p.B, p.N), p.IN, p.C, p.sigma)
                opts[j].zero_grad()
                torch_loss(p, prms[j], X, y).backward()
                opts[j].step()
            t += 1
            if (tt + 1) % p.K1 == 0:
                average([range(q * p.S, q * p.S + p.S) for q in range(p.P // p.S)])
        average([range(p.P)])
    W = np.stack([flatten(p, prm) for prm in prms])
    V = np.stack([np.concatenate([opts[j].state[v]["momentum_buffer"].numpy().reshape(-1)
                                  for v in prms[j].values()]) for j in range(p.P)])
    return W, V


@pytest.mark.parametrize("kind", [M.SOFTMAX, M.MLP])
def test_single_learner_momentum_weight_decay_is_torch_sgd(kind):
    p = small(kind, 1, 1, 3, 2, momentum=0.9, weight_decay=0.01)
    st = M.run(p, 2)
    W, V = torch_schedule_reference(p, 2)
    assert relerr(st.W[0], W[0]) < 1e-12
    assert relerr(st.V[0], V[0]) < 1e-12


@pytest.mark.parametrize("avg", [False, True])
def test_hierarchical_momentum_buffers(avg):
    """P = 4 in groups of 2, K1 = 2, two blocks and two rounds: per-learner
    buffers carried across the means (or averaged with the parameters)."""
    p = small(M.MLP, 4, 2, 2, 2, momentum=0.8, weight_decay=0.005, avg_momentum=avg)
    st = M.run(p, 2)
    W, V = torch_schedule_reference(p, 2)
    assert relerr(st.W, W) < 1e-12
    assert relerr(st.V, V) < 1e-12
    # after the global mean: equal buffers exactly when they are averaged
    assert np.array_equal(st.V, np.repeat(st.V[:1], 4, axis=0)) == avg


def test_momentum_zero_is_plain_step():
    """mu = lambda = 0 reproduces the plain step bit for bit."""
    p = small(M.MLP, 4, 2, 2, 2)
    q = small(M.MLP, 4, 2, 2, 2, momentum=0.0, weight_decay=0.0, avg_momentum=True)
    assert np.array_equal(M.run(p, 2).W, M.run(q, 2).W)


def test_averaged_buffers_with_one_group_per_step_are_large_batch_momentum():
    """S = P, K1 = 1: every step ends with the mean of parameters and buffers,
    which is one learner with momentum on the mean gradient of the P*B
    samples of the step (the buffers being linear in the gradients)."""
    p = small(M.SOFTMAX, 3, 3, 1, 4, B=3, momentum=0.9, weight_decay=0.01, avg_momentum=True)
    st = M.run(p, 1)
    prm = torch_params(p, M.initial_replica(p))
    opt = torch.optim.SGD(list(prm.values()), lr=p.lr64, momentum=p.mu64, weight_decay=p.wd64)
    for t in range(4):
        Xs, ys = zip(*[rng.data_rows(p.seed, rng.draw_indices(p.seed, j, t, p.B, p.N), p.IN, p.C, p.sigma)
                       for j in range(p.P)])
        opt.zero_grad()
        torch_loss(p, prm, np.concatenate(Xs), np.concatenate(ys)).backward()
        opt.step()
    assert relerr(st.W[0], flatten(p, prm)) < 1e-12


# ------------------------------------------------------- ReLU decisions at a kink
def _kink_problem():
    return M.Problem(M.MLP, 1, 1, 1, 1, 2, IN=2, H=2, C=2, N=4)


def test_kink_monitor_margins_by_hand():
    """Two samples, two units.  z1 = X W1^T + b1 and the margins
    |z1| / (sum_k |x_k W1[h,k]| + |b1[h]|), written out:
      sample 0: unit 0  1*2 + 2*(-1) + 0   = 0     over 2 + 2 + 0      = 4     -> 0
                unit 1  1*.5 + 2*.25 - .5  = 0.5   over .5 + .5 + .5   = 1.5   -> 1/3
      sample 1: unit 0  3*2 + (-1)*(-1) + 0 = 7    over 6 + 1 + 0      = 7     -> 1
                unit 1  3*.5 - .25 - .5    = 0.75  over 1.5 + .25 + .5 = 2.25  -> 1/3"""
    X = np.array([[1.0, 2.0], [3.0, -1.0]])
    W1 = np.array([[2.0, -1.0], [0.5, 0.25]])
    b1 = np.array([0.0, -0.5])
    mon = M.KinkMonitor(2)
    mon.observe(X @ W1.T + b1, X, W1, b1, t=5, j=3)
    assert np.allclose(mon.min_margin, [0.0, 1.0 / 3.0], rtol=0, atol=1e-15)
    assert mon.decisions == [(5, 3, 0, 0, 0.0)]
    # a planted pre-activation just off zero: b1[0] = 2^-30 gives z1 = 2^-30
    # over 4 + 2^-30; b1[0] = 2^-12 gives a margin of about 2^-14, above the
    # default threshold 2^-16
    for b, flagged in ((2.0 ** -30, True), (2.0 ** -12, False)):
        mon = M.KinkMonitor(2)
        bb = np.array([b, -0.5])
        mon.observe(X @ W1.T + bb, X, W1, bb, t=0, j=0)
        want = b / (4.0 + b)
        assert abs(mon.min_margin[0] - want) <= 1e-15 * want
        assert [d[:4] for d in mon.decisions] == ([(0, 0, 0, 0)] if flagged else [])
    # the monitor sees every learner step of a run, labelled by step and learner
    p = M.Problem(M.MLP, 4, 2, 2, 1, 8, IN=20, H=12, C=5, N=64, sigma=0.5, lr=0.1, seed=3)
    mon = M.KinkMonitor(p.H, threshold=1.0)   # every decision
    M.run(p, 1, monitor=mon)
    assert len(mon.decisions) == p.T * p.P * p.B * p.H
    assert {(d[0], d[1]) for d in mon.decisions} == {(t, j) for t in range(p.T) for j in range(p.P)}


def test_flipped_decision_is_the_other_relu_derivative():
    """With z1[s, h] exactly 0 the activation is 0 on both branches, so taking
    the decision the other way only changes the derivative [z1 > 0] there:
    the gradient equals autograd's with d ReLU/dz = 1 at that one entry
    (relu(z) + (z - z.detach()) at (s, h): same value, derivative + 1)."""
    p = _kink_problem()
    row = np.zeros(M.param_count(p))
    blk = M.unpack(p, row)
    blk["W1"][:] = [[2.0, -1.0], [0.5, 0.25]]
    blk["b1"][:] = [0.0, -0.5]
    blk["W2"][:] = [[0.3, -0.7], [-0.2, 0.4]]
    blk["b2"][:] = [0.1, -0.1]
    X = np.array([[1.0, 2.0], [3.0, -1.0]])
    y = np.array([1, 0])
    plain = M.minibatch_gradient(p, row, X, y)
    flipped = M.minibatch_gradient(p, row, X, y, flips=[(0, 0)])

    def autograd(extra):
        prm = torch_params(p, row)
        z1 = torch.tensor(X) @ prm["W1"].T + prm["b1"]
        e = torch.zeros(2, 2)
        e[0, 0] = extra
        a1 = torch.relu(z1) + (z1 - z1.detach()) * e
        z2 = a1 @ prm["W2"].T + prm["b2"]
        torch.nn.functional.cross_entropy(z2, torch.tensor(y)).backward()
        return flatten_grad(p, prm)

    assert relerr(plain, autograd(0.0)) < 1e-14
    assert relerr(flipped, autograd(1.0)) < 1e-14
    d = M.unpack(p, flipped - plain)
    assert np.any(d["W1"][0] != 0) and np.all(d["W1"][1] == 0) and np.all(d["W2"] == 0)


def flatten_grad(p, prm):
    return np.concatenate([prm[name].grad.numpy().reshape(-1) for name, _ in M.segments(p)])


def test_flips_touch_only_their_learner_and_step():
    p = M.Problem(M.MLP, 2, 2, 2, 1, 4, IN=10, H=6, C=3, N=20, sigma=0.5, lr=0.1, seed=5)
    base = M.run(p, 1)
    same = M.run(p, 1, flips=frozenset([(7, 0, 0, 0)]))  # a step outside the round
    assert np.array_equal(base.W, same.W)
    moved = M.run(p, 1, flips=frozenset([(1, 1, 2, 3)]))
    assert not np.array_equal(base.W, moved.W)
