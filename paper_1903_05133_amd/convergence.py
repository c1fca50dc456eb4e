"""Multi-round convergence runs of Hier-AVG on the synthetic workloads.

Each run trains one of the named models for a fixed budget of local SGD steps
per learner and, after every round, evaluates the global model (replica 0,
which every learner holds after the global mean) on training rows and on
held-out rows, printing one JSON line per round:

    {"run": ..., "round": r, "steps": t, "train_loss": ..., "train_acc": ...,
     "test_loss": ..., "test_acc": ..., "round_ms": ..., "eval_ms": ...}

(round_ms: host wall time of the round including its synchronisation;
eval_ms: both evaluations, the first held-out call including the generation
of the held-out rows).

and one summary line per run.  ``--sweep paper`` runs the interval and
cluster-size sweeps of the paper's experiments (Sec. 4) on the synthetic
data, with the paper's global interval K1*K2 written as ``k_global``:

  * k_global in {8, 16, 32} at P=32, K1=4, S=4;
  * K1 in {4, 8} and S in {2, 4} at P=16, k_global=32;
  * Hier-AVG against K-AVG (S=1) at the same P, K1 and k_global.

Optimizer and schedule options: ``--momentum``, ``--weight-decay``,
``--avg-momentum`` (heavy-ball buffers, L2 decay, buffers averaged with the
parameters), ``--lr-drop ROUND:LR`` (step schedule of Sec. 4, repeatable:
the step size from that round on), ``--k-global`` (round length in steps,
non-integer beta), ``--checkpoint PATH`` (state after every round, resumable
with ``--resume PATH``).

Everything runs through the C ABI on the GPU; the oracle is not used.

    python -m paper_1903_05133_amd.convergence --model 1 --P 16 --S 4 --K1 4 --K2 4 --rounds 16
    python -m paper_1903_05133_amd.convergence --momentum 0.9 --lr 0.02 --lr-drop 12:0.002 --rounds 16
    python -m paper_1903_05133_amd.convergence --sweep paper --steps 256
"""

import argparse
import json
import sys
import time

from . import native
from .hieravg import HierAvg, config

# kind, in_dim, hidden, classes, n_samples, noise std of the named models (include/hieravg.h)
MODELS = {
    0: (0, 3072, 0, 10, 2048, 1.0),
    1: (1, 3072, 512, 10, 50000, 0.5),
    2: (1, 150528, 1024, 1000, 100000, 1.0),
}


def run(name, model, P, S, K1, K2, B, lr, rounds, eval_rows, noise=None, seed=0, out=sys.stdout, momentum=0.0,
        weight_decay=0.0, avg_momentum=False, lr_drops=(), k_global=0, checkpoint=None, resume=None):
    kind, IN, H, C, N, sigma = MODELS[model]
    cfg = config(kind, P, S, K1, K2, B=B, in_dim=IN, hidden=H, classes=C, n_samples=N,
                 noise_std=sigma if noise is None else noise, lr=lr, seed=seed, momentum=momentum,
                 weight_decay=weight_decay, avg_momentum=avg_momentum, k_global=k_global)
    n_train = min(eval_rows, N)
    curve = []
    drops = dict(lr_drops)
    with HierAvg(config=cfg) as h:
        first = 1
        if resume:
            h.load(resume)
            first = h.steps // h.T + 1
        cur_lr = lr
        for r in range(1, first):
            cur_lr = drops.get(r, cur_lr)
        h.set_lr(cur_lr)
        for r in range(first, rounds + 1):
            if r in drops:
                cur_lr = drops[r]
                h.set_lr(cur_lr)
            t0 = time.perf_counter()
            h.round()
            h.sync()
            ms = (time.perf_counter() - t0) * 1e3
            t1 = time.perf_counter()
            tr_loss, tr_hit = h.evaluate(0, 0, n_train)
            te_loss, te_hit = h.evaluate(0, 1, eval_rows)
            ems = (time.perf_counter() - t1) * 1e3
            rec = {"run": name, "round": r, "steps": h.steps, "lr": cur_lr, "train_loss": float(f"{tr_loss:.7g}"),
                   "train_acc": round(tr_hit / n_train, 6), "test_loss": float(f"{te_loss:.7g}"),
                   "test_acc": round(te_hit / eval_rows, 6), "round_ms": round(ms, 3),
                   "eval_ms": round(ems, 3)}
            curve.append(rec)
            print(json.dumps(rec), file=out, flush=True)
            if checkpoint:
                h.save(checkpoint)
    last = curve[-1]
    summary = {"run": name, "summary": True, "model": model, "P": P, "S": S, "K1": K1, "K2": K2,
               "k_global": k_global or K1 * K2, "B": B, "lr": lr, "lr_drops": sorted(drops.items()),
               "momentum": momentum, "weight_decay": weight_decay, "avg_momentum": avg_momentum,
               "noise": sigma if noise is None else noise,
               "rounds": rounds, "steps": last["steps"], "final_test_loss": last["test_loss"],
               "final_test_acc": last["test_acc"],
               "best_test_loss": min(c["test_loss"] for c in curve)}
    print(json.dumps(summary), file=out, flush=True)
    return summary


def paper_sweep(steps, model, B, lr, eval_rows, noise, out=sys.stdout):
    """The interval / cluster-size sweeps at a fixed budget of `steps` local
    SGD steps per learner (rounded down to whole rounds)."""
    runs = []
    for kg in (8, 16, 32):
        runs.append((f"P32_S4_K1=4_kg={kg}", 32, 4, 4, kg // 4))
    for K1 in (4, 8):
        for S in (2, 4):
            runs.append((f"P16_S{S}_K1={K1}_kg=32", 16, S, K1, 32 // K1))
        runs.append((f"P16_KAVG_K1={K1}_kg=32", 16, 1, K1, 32 // K1))
    for kg in (8, 16, 32):
        runs.append((f"P32_KAVG_K1=4_kg={kg}", 32, 1, 4, kg // 4))
    results = []
    for name, P, S, K1, K2 in runs:
        rounds = max(1, steps // (K1 * K2))
        results.append(run(name, model, P, S, K1, K2, B, lr, rounds, eval_rows, noise, out=out))
    return results


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--model", type=int, default=1, choices=sorted(MODELS))
    ap.add_argument("--P", type=int, default=16)
    ap.add_argument("--S", type=int, default=4)
    ap.add_argument("--K1", type=int, default=4)
    ap.add_argument("--K2", type=int, default=4, help="local-averaging blocks per round (the paper's beta)")
    ap.add_argument("--B", type=int, default=32)
    ap.add_argument("--lr", type=float, default=0.05)
    ap.add_argument("--rounds", type=int, default=16)
    ap.add_argument("--eval-rows", type=int, default=4096)
    ap.add_argument("--noise", type=float, default=None, help="override the model's data noise std")
    ap.add_argument("--sweep", choices=["paper"], default=None)
    ap.add_argument("--steps", type=int, default=256, help="local SGD steps per learner of each sweep run")
    ap.add_argument("--momentum", type=float, default=0.0)
    ap.add_argument("--weight-decay", type=float, default=0.0)
    ap.add_argument("--avg-momentum", action="store_true")
    ap.add_argument("--lr-drop", action="append", default=[], metavar="ROUND:LR",
                    help="step size from round ROUND on (repeatable)")
    ap.add_argument("--k-global", type=int, default=0, help="SGD steps per round (0: K1*K2)")
    ap.add_argument("--checkpoint", default=None, help="write the state after every round (.npz)")
    ap.add_argument("--resume", default=None, help="continue from a --checkpoint file")
    a = ap.parse_args(argv)
    drops = [(int(d.split(":")[0]), float(d.split(":")[1])) for d in a.lr_drop]
    native.lib()
    if a.sweep == "paper":
        paper_sweep(a.steps, a.model, a.B, a.lr, a.eval_rows, a.noise)
    else:
        run("single", a.model, a.P, a.S, a.K1, a.K2, a.B, a.lr, a.rounds, a.eval_rows, a.noise,
            momentum=a.momentum, weight_decay=a.weight_decay, avg_momentum=a.avg_momentum, lr_drops=drops,
            k_global=a.k_global, checkpoint=a.checkpoint, resume=a.resume)


if __name__ == "__main__":
    main()
