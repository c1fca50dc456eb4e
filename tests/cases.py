"""Workload descriptions shared by the GPU parity tests, smoke() and bench.py:
each case becomes a C-ABI config (for the HIP path) and an oracle Problem
(for the CPU oracle) built from the same numbers.  Holds none of the
method's arithmetic."""

import numpy as np

KINDS = {"softmax": 0, "mlp": 1, "averaging": 2}

# The named workloads (model ids of the C ABI) and their parameters.
NAMED = {
    "softmax_3072_10": dict(kind="softmax", IN=3072, C=10, N=2048, sigma=1.0),
    "mlp_3072_512_10": dict(kind="mlp", IN=3072, H=512, C=10, N=50000, sigma=0.5),
    "mlp_150528_1024_1000": dict(kind="mlp", IN=150528, H=1024, C=1000, N=100000, sigma=1.0),
    "averaging_11_7M": dict(kind="averaging", IN=11_700_000, momentum=0.9, init_std=0.01, grad_std=0.01),
}
MODEL_ID = {"softmax_3072_10": 0, "mlp_3072_512_10": 1, "mlp_150528_1024_1000": 2, "averaging_11_7M": 3}


def case(kind, P, S, K1, K2, B=1, IN=0, H=0, C=0, N=0, sigma=1.0, lr=0.05, momentum=0.0, init_std=0.01,
         grad_std=0.01, seed=0, k_global=0, weight_decay=0.0, avg_momentum=False):
    return dict(kind=kind, P=P, S=S, K1=K1, K2=K2, B=B, IN=IN, H=H, C=C, N=N, sigma=sigma, lr=lr,
                momentum=momentum, init_std=init_std, grad_std=grad_std, seed=seed, k_global=k_global,
                weight_decay=weight_decay, avg_momentum=avg_momentum)


def named(name, P, S, K1, K2, B, lr, seed=0):
    d = dict(NAMED[name])
    kind = d.pop("kind")
    return case(kind, P, S, K1, K2, B=B, lr=lr, seed=seed, **d)


UPDATE_MODES = {"auto": 0, "eager": 1, "delayed": 2}


def native_config(c, update_mode="auto"):
    from paper_1903_05133_amd import config
    return config(KINDS[c["kind"]], c["P"], c["S"], c["K1"], c["K2"], B=c["B"], in_dim=c["IN"], hidden=c["H"],
                  classes=c["C"], n_samples=c["N"], noise_std=c["sigma"], lr=c["lr"], momentum=c["momentum"],
                  init_std=c["init_std"], grad_std=c["grad_std"], seed=c["seed"],
                  update_mode=UPDATE_MODES[update_mode], k_global=c.get("k_global", 0),
                  weight_decay=c.get("weight_decay", 0.0), avg_momentum=c.get("avg_momentum", False))


def oracle_problem(c):
    from oracle import method as M
    return M.Problem(c["kind"], c["P"], c["S"], c["K1"], c["K2"], c["B"], IN=c["IN"], H=c["H"], C=c["C"],
                     N=c["N"], sigma=c["sigma"], lr=c["lr"], momentum=c["momentum"], init_std=c["init_std"],
                     grad_std=c["grad_std"], seed=c["seed"], k_global=c.get("k_global", 0),
                     weight_decay=c.get("weight_decay", 0.0), avg_momentum=c.get("avg_momentum", False))


def block_errors(prob, got, want):
    """Per replica and parameter block: max|got - want| / max|want| (the
    normwise reading of 'max relative error')."""
    from oracle import method as M
    out = {}
    for p in range(got.shape[0]):
        g = M.unpack(prob, np.asarray(got[p], dtype=np.float64))
        w = M.unpack(prob, np.asarray(want[p], dtype=np.float64))
        for name in g:
            denom = max(float(np.max(np.abs(w[name]))), 1e-30)
            out[(p, name)] = float(np.max(np.abs(g[name] - w[name]))) / denom
    return out


TOL = 1e-4            # float32 parity gate ("max relative error 1e-4")


def parity_report(prob, got, want):
    """Compare GPU replicas `got` [P, D] with oracle replicas `want`: every
    parameter block of every replica must agree to TOL (max|g - o| / max|o|
    over the block).  Returns (ok, details); details["units"] lists, for the
    MLP, the hidden units h whose parameters (row h of W1, b1[h], column h of
    W2) exceed TOL in some replica."""
    from oracle import method as M
    details = {"worst": (None, 0.0), "units": []}
    ok = True
    units = set()
    for p in range(got.shape[0]):
        g = M.unpack(prob, np.asarray(got[p], dtype=np.float64))
        w = M.unpack(prob, np.asarray(want[p], dtype=np.float64))
        err = {n: np.abs(g[n] - w[n]) / max(float(np.max(np.abs(w[n]))), 1e-30) for n in w}
        if prob.kind == M.MLP:
            unit_err = np.maximum.reduce([err["W1"].max(axis=1), err["b1"], err["W2"].max(axis=0)])
            units |= set(np.nonzero(unit_err > TOL)[0].tolist())
        for n, e in err.items():
            m = float(e.max()) if e.size else 0.0
            if m > details["worst"][1]:
                details["worst"] = ((p, n), m)
            if m > TOL:
                ok = False
                details.setdefault("fail", []).append((p, n, m))
    details["units"] = sorted(units)
    return ok, details


MAX_BRANCH_CANDIDATES = 6  # near-kink decisions on the failing units tried, smallest margins first
MAX_BRANCH_RUNS = 24       # oracle re-runs at most


def branch_parity(prob, got, want, monitor, rerun, max_runs=MAX_BRANCH_RUNS):
    """The parity gate where several results are correct.

    A ReLU decision [z1 > 0] whose pre-activation is within float32 rounding
    of zero (relative margin below the monitor's threshold, recorded by the
    oracle's KinkMonitor as (t, j, s, h)) may come out either way in any
    float32 evaluation; both are correct executions of Algorithm 1.  If `got`
    fails the TOL gate against the oracle run `want`, the flagged decisions on
    the failing hidden units are candidates: `rerun(flips)` re-runs the oracle
    with a set of them taken the other way, and `got` passes if it meets the
    same TOL gate, on every parameter, against one such run (subsets tried by
    size, then by margin).  Returns (ok, details); details["flipped"] names
    the decisions of the run that matched."""
    import itertools
    ok, det = parity_report(prob, got, want)
    if ok or monitor is None:
        return ok, det
    cands = sorted((d for d in monitor.decisions if d[3] in set(det["units"])), key=lambda d: d[4])
    cands = cands[:MAX_BRANCH_CANDIDATES]
    det["candidates"] = cands
    runs = 0
    for size in range(1, len(cands) + 1):
        for subset in itertools.combinations(cands, size):
            if runs >= max_runs:
                return False, det
            runs += 1
            ok2, det2 = parity_report(prob, got, rerun(frozenset(d[:4] for d in subset)))
            if ok2:
                det2["flipped"] = list(subset)
                det2["candidates"] = cands
                det2["unflipped_worst"] = det["worst"]
                return True, det2
    return False, det


def eager_means_once(c):
    """Whether an eager MLP round writes the first layer's global mean once
    (full-tile steps: B of 32 or 64, plain SGD, P a power of two up to 64)
    and its block-end cluster means once (S * B / 16 > 16: past the fused
    mean step), as the library plans it."""
    P, S, B = c["P"], c["S"], c["B"]
    pow2 = lambda n: 2 <= n <= 64 and n & (n - 1) == 0
    plain = c.get("momentum", 0.0) == 0.0 and c.get("weight_decay", 0.0) == 0.0
    upd_mean = S > 1 and pow2(S) and S * B // 16 > 16
    T = c.get("k_global", 0) or c["K1"] * c["K2"]  # steps per round
    once_global = (c["kind"] == "mlp" and plain and B in (32, 64) and pow2(P) and T >= 2
                   and (c["K1"] > 1 or S == 1 or upd_mean))
    return once_global, once_global and upd_mean
