"""Benchmark of the Hier-AVG hot path on one MI355X.

One bench "step" is one Hier-AVG round (Algorithm 1, Sec. 3.1: K2 blocks of
K1 local SGD steps of all P learners, the cluster means and the global mean)
of the headline workload: the 3-layer MLP 150528 -> 1024 ReLU -> 1000 with
softmax cross-entropy (155.2M parameters per replica), P=16, S=4, K1=4,
K2=2, B=32, lr=0.02, on synthetic ImageNet-shaped data (N=100000 rows of
224*224*3 features: class-mean pattern ~N(0,1) + N(0,1) noise, 1000
classes).  This is the largest single-GPU workload.  `value` is
learner-SGD-steps per second (P*K1*K2 per round) with the dataset (60.2 GB)
and the replicas (9.9 GB) resident in HBM.

Also reported, on the same JSON line:
  roofline      the dominant kernel of the headline round (largest launches x
                duration): algorithmic flops (or bytes) per launch over its
                mean duration, timed with HIP events on the handle's stream
                around a graph of back-to-back launches of it; `traffic` is the
                HBM bytes per launch from rocprofv3 FETCH_SIZE / WRITE_SIZE
                counters (profiles/traffic.json) while the kernel's source is
                unchanged since they were taken
  configs       the other workloads, each timed the same way: softmax
                3072 -> 10 (P=4, launch-bound: us per round, launches per
                step), MLP 3072-512-10 at P=16 and at P=64 (B=64, MFMA-bound),
                and the averaging-only workload (P=32 replicas of 11.7M floats,
                heavy-ball momentum, cluster mean every step, global mean
                every 4): HBM GB/s of the averaging kernels as a fraction of
                8 TB/s
  cpu_baseline  the CPU oracle (float64 numpy) on a sample of the headline
                workload: one SGD step of all 16 learners, on this host's
                cores, and one learner's step on one thread
"""

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)
sys.path.insert(0, os.path.join(ROOT, "tests"))

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
FP32_MFMA_PEAK_TFLOPS = 157.3  # MI355X dense fp32 matrix
F = 4                          # bytes per float

HEADLINE = "mlp_150528_1024_1000"
# name -> (named workload, P, S, K1, K2, B, lr, rounds timed)
WORKLOADS = {
    "softmax_3072_10": ("softmax_3072_10", 4, 2, 2, 2, 8, 0.05, 400),
    "mlp_3072_512_10": ("mlp_3072_512_10", 16, 4, 4, 4, 32, 0.05, 200),
    "mlp_3072_512_10_p64": ("mlp_3072_512_10", 64, 8, 8, 4, 64, 0.1, 20),
    "averaging_11_7M": ("averaging_11_7M", 32, 4, 1, 4, 1, 0.1, 20),
    HEADLINE: ("mlp_150528_1024_1000", 16, 4, 4, 2, 32, 0.02, None),
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# ---------------------------------------------------------------- algorithmic work
def step_work(c):
    """Algorithmic flops and bytes of one learner's SGD step: the forward and
    weight-gradient products (no input gradient), every parameter read and
    written once, the sampled rows and labels read once."""
    B, IN, H, C = c["B"], c["IN"], c["H"], c["C"]
    if c["kind"] == "softmax":
        D = C * IN + C
        return 4 * B * IN * C, 8 * D + 4 * B * IN + 4 * B
    D = H * IN + H + C * H + C
    return 4 * B * IN * H + 6 * B * H * C, 8 * D + 4 * B * IN + 4 * B


def mlp_kernel_work(P, S, K1, K2, B, IN, H, C, once=(False, False)):
    """Algorithmic (bytes, flops) per launch of each kernel class of an MLP
    round: every operand a launch needs read once and every result written
    once, at its logical (unpadded) size.  Split-K partial sums are an
    implementation choice and are not counted.  The delayed-update block
    kernels differ between the first block (every cluster reads replica 0's
    W1) and the others (each cluster reads its own copy); their bytes are the
    mean over the K2 blocks of a round."""
    G = P // S
    pairs = K1 * (K1 - 1) // 2
    tail = H + C * H + C  # b1, W2, b2: their cluster (global) mean rides in the block update
    bases = (1 + (K2 - 1) * G) / K2          # W1 bases read per block, mean over the blocks
    k_avg = (K1 - 1) / 2.0                   # earlier steps corrected per step, mean over a block
    # block update, per block b: its bases read (replica 0's W1 for b = 0, the
    # G cluster copies after), its result written (G copies; the last block:
    # the global mean, once), the block's errors and minibatch rows read, and
    # the cluster (last block: global) mean of b1, W2, b2 read and written
    upd = 0.0
    for b in range(K2):
        last = b == K2 - 1
        upd += (1 if b == 0 else G) * H * IN + (1 if last else G) * H * IN + K1 * P * B * (H + IN)
        upd += 2 * P * tail if (P > 1 if last else S > 1) else 0
    upd /= K2
    return {
        # forward of a block's K1 steps from the block-start bases: the bases,
        # the K1*P minibatches, the K1*P pre-activation blocks
        "fwd1_block_gemm": (F * (bases * H * IN + K1 * P * B * IN + K1 * P * B * H), K1 * P * 2 * B * H * IN),
        "block_update_gemm": (F * upd, K1 * P * 2 * B * H * IN),
        # Gram blocks of the round: every minibatch row read once, blocks written
        "gram": (F * (K2 * K1 * P * B * IN + K2 * P * pairs * B * B), K2 * P * pairs * 2 * B * B * IN),
        "w1_global_mean": (F * ((G + 1) * H * IN + 2 * P * tail), G * H * IN + P * tail),
        # pre-activations of one step with the Gram correction of the earlier
        # steps (more than 32 classes)
        "z1_delayed": (F * P * (B * H + H + k_avg * (B * H + B * B) + B * H), P * 2 * B * B * H * k_avg),
        # (a round's first forward from the once-written global mean: W1 read once)
        "fwd1_gemm": (F * ((1 if once[0] else P) * H * IN + P * B * IN + P * B * H), P * 2 * B * H * IN),
        "reduce1": (P * F * (H + B * H), P * B * H),
        "fwd2_gemm": (P * F * (C * H + B * H + B * C), P * 2 * B * C * H),
        "softmax_grad": (P * F * (C + 2 * B * C) + P * B * 8, P * B * C * 4),
        "bwd_hidden": (P * F * (B * C + C * H + 2 * B * H), P * 2 * B * C * H),
        "update2_gemm": (P * F * (2 * C * H + B * C + B * H + 2 * C), P * 2 * B * C * H),
        "update1_gemm": (P * F * (2 * H * IN + B * H + B * IN + 2 * H), P * 2 * B * H * IN),
        # update of W1 at step t and forward of step t+1: W1 read and written
        # once, G1 and the two minibatches read, the next pre-activations
        # written once; the cluster-mean variant moves the same bytes
        "step1_gemm": (P * F * (2 * H * IN + 2 * B * H + 2 * B * IN), P * 4 * B * H * IN),
        "step1_gemm_group_mean": (P * F * (2 * H * IN + 2 * B * H + 2 * B * IN), P * 4 * B * H * IN),
        # update of every learner's W1 with the cluster (or global) mean: W1
        # read once per learner, the mean written to every row or once per
        # cluster (once), G1 and the minibatch read
        "update1_gemm_group_mean": (F * (P * H * IN + (G if once[1] else P) * H * IN + P * B * H + P * B * IN),
                                    P * 2 * B * H * IN),
        "update1_gemm_global_mean": (F * (P * H * IN + (1 if once[0] else P) * H * IN + P * B * H + P * B * IN),
                                     P * 2 * B * H * IN),
        # next step's forward from each cluster's common W1: one copy per
        # cluster, the minibatches, the pre-activations
        "fwd1_group_gemm": (F * (G * H * IN + P * B * IN + P * B * H), P * 2 * B * H * IN),
    }


def kernel_work(c, classes=None):
    """Algorithmic (bytes, flops) per launch of each kernel class; `classes`
    (the classes a round launched) tells whether the hidden-error kernel also
    took the second layer's step (no update2_gemm in the round)."""
    P, S, K1, K2 = c["P"], c["S"], c["K1"], c["K2"]
    if c["kind"] == "averaging":
        D = c["IN"]
        return {
            # read w, v, g and write w, v of every learner
            "momentum": (20 * P * D, 0), "momentum_group_mean": (20 * P * D, 0),
            # every learner's w read from the stored global mean once; v, g read and v, w written per learner
            "momentum_first_step": (16 * P * D + 4 * D, 0),
            # w, v, g read and v written per learner; the common mean written once
            "momentum_global_mean": (16 * P * D + 4 * D, 0),
        }
    if c["kind"] == "softmax":
        B, IN, C = c["B"], c["IN"], c["C"]
        D = C * IN + C
        return {"fwd1_gemm": (P * F * (C * IN + B * IN + B * C), P * 2 * B * C * IN),
                "update1_gemm": (P * F * (2 * D + B * C + B * IN), P * 2 * B * C * IN),
                "step1_gemm": (P * F * (2 * D + 2 * B * C + 2 * B * IN), P * 4 * B * C * IN),
                "step1_gemm_group_mean": (P * F * (2 * D + 2 * B * C + 2 * B * IN), P * 4 * B * C * IN),
                "global_mean": (2 * F * P * D, P * D)}
    import cases
    w = mlp_kernel_work(P, S, K1, K2, c["B"], c["IN"], c["H"], c["C"], cases.eager_means_once(c))
    if classes is not None and "bwd_hidden" in classes and "update2_gemm" not in classes:
        # hidden error and the W2 step in one pass: G2, W2, Z1 read, G1 and W2 written
        B, H, C = c["B"], c["H"], c["C"]
        w["bwd_hidden"] = (P * F * (B * C + 2 * C * H + 2 * B * H + C), P * 4 * B * C * H)
    D = c["H"] * c["IN"] + c["H"] + c["C"] * c["H"] + c["C"]
    tail = D - c["H"] * c["IN"]
    w["group_mean"] = (2 * F * P * D, P * D)
    w["global_mean"] = (2 * F * P * D, P * D)
    w["tail_group_mean"] = (2 * F * P * tail, P * tail)
    w["tail_global_mean"] = (2 * F * P * tail, P * tail)
    return w


def source_record(path, workload, kernel_class):
    """The committed counter record of `kernel_class` in `workload`
    (profiles/<path>), or None when the kernel's source has changed since the
    counters were taken."""
    try:
        rec = json.load(open(os.path.join(ROOT, "profiles", path)))["workloads"][workload]["kernels"][kernel_class]
        cur = hashlib.sha256(open(os.path.join(ROOT, rec["source"]), "rb").read()).hexdigest()
    except (OSError, KeyError, ValueError):
        return None
    return rec if cur == rec["source_sha256"] else None


# ---------------------------------------------------------------- one workload
def run_workload(name, rounds, warmup, reps=None):
    """Create the workload's handle, run `warmup` rounds, time `rounds` rounds
    with HIP events on the handle's stream, then profile one more pass
    (launch counts per kernel class) and time every kernel class over a graph
    of back-to-back launches of it."""
    import torch
    import cases
    from paper_1903_05133_amd import HierAvg

    wl, P, S, K1, K2, B, lr, _ = WORKLOADS[name]
    c = cases.named(wl, P, S, K1, K2, B, lr, seed=0)
    h = HierAvg(config=cases.native_config(c))
    stream = torch.cuda.Stream()
    h.set_stream(stream)
    for _ in range(warmup):
        h.round()
    h.sync()
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record(stream)
    t0 = time.perf_counter()
    for _ in range(rounds):
        h.round()
    end.record(stream)
    h.sync()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = start.elapsed_time(end)
    log(f"[bench] {name}: {rounds} rounds in {ms:.3f} ms (host wall {wall * 1e3:.3f} ms)")
    # One more pass with HIP events around every launch: launch counts and
    # time shares per kernel class.
    h.profile(True)
    h.round()
    stats = h.profile_read()
    h.profile(False)
    h.sync()
    # Per-launch durations: each kernel class over a graph of back-to-back
    # launches between two HIP events on the handle's stream (spreads the
    # events' own cost).  This changes the replicas, so it comes last.
    if reps is None:
        reps = 200 if ms / rounds < 5.0 else 20
    dur_ms = {k: h.time_kernel(k, reps) for k in stats if k != "draw_indices"}
    h.close()
    torch.cuda.empty_cache()
    return c, ms / rounds, stats, dur_ms


def summarize(name, c, ms_round, stats, dur_ms):
    """Per-config record: round time, learner-steps/s, launches, the
    method's algorithmic flops and bytes per round as fractions of the peaks,
    and every kernel class with its measured duration and roofline."""
    P, K1, K2 = c["P"], c["K1"], c["K2"]
    work = kernel_work(c, stats)
    kernels = {}
    total = sum(t for _, t in stats.values())
    for k, (n, tot) in stats.items():
        avg = dur_ms.get(k, tot / n)
        b, fl = work.get(k, (0, 0))
        kernels[k] = {"launches": n, "avg_us": round(avg * 1e3, 3), "share": round(tot / total, 4),
                      "GBps": round(b / (avg * 1e-3) / 1e9, 1) if b else None,
                      "TFLOPs": round(fl / (avg * 1e-3) / 1e12, 2) if fl else None,
                      "mfma_frac": round(fl / (avg * 1e-3) / 1e12 / FP32_MFMA_PEAK_TFLOPS, 4) if fl else None,
                      "hbm_frac": round(b / (avg * 1e-3) / 1e9 / HBM_PEAK_GBS, 4) if b else None}
    launches = sum(n for n, _ in stats.values())
    out = {"workload": name, "P": P, "S": c["S"], "K1": K1, "K2": K2, "ms_per_round": round(ms_round, 5),
           "us_per_round": round(ms_round * 1e3, 2), "launches_per_round": launches,
           "launches_per_step": round(launches / (K1 * K2), 2), "kernels": kernels}
    if c["kind"] == "averaging":
        round_bytes = sum(n * work.get(k, (0, 0))[0] for k, (n, _) in stats.items())
        out.update({"D": c["IN"], "momentum": c["momentum"], "lr": c["lr"], "alg_bytes_per_round": round_bytes,
                    "round_GBps": round(round_bytes / (ms_round * 1e-3) / 1e9, 1)})
        out["round_frac"] = round(out["round_GBps"] / HBM_PEAK_GBS, 4)
        return out
    fl, by = step_work(c)
    steps = P * K1 * K2
    out.update({"B": c["B"], "lr": c["lr"], "N": c["N"], "learner_steps_per_round": steps,
                "learner_steps_per_s": round(steps / (ms_round * 1e-3), 1),
                "schedule": "delayed" if "fwd1_block_gemm" in stats else "eager",
                "round_mfma_frac": round(steps * fl / (ms_round * 1e-3) / 1e12 / FP32_MFMA_PEAK_TFLOPS, 4),
                "round_alg_bytes_frac": round(steps * by / (ms_round * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)})
    return out


def roofline(c, stats, dur_ms):
    """The dominant kernel (largest launches x duration among the kernels
    with a stated algorithmic work) against the peak of the resource whose
    ideal time for that work is longer."""
    work = kernel_work(c, stats)
    dom = max((k for k in dur_ms if work.get(k, (0, 0))[1] or work.get(k, (0, 0))[0]),
              key=lambda k: dur_ms[k] * stats[k][0])
    avg_s = dur_ms[dom] * 1e-3
    b, fl = work[dom]
    if fl / (FP32_MFMA_PEAK_TFLOPS * 1e12) > b / (HBM_PEAK_GBS * 1e9):
        roof = {"kernel": dom, "bound": "mfma", "achieved": round(fl / avg_s / 1e12, 2),
                "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(fl / avg_s / 1e12 / FP32_MFMA_PEAK_TFLOPS, 4)}
    else:
        roof = {"kernel": dom, "bound": "hbm", "achieved": round(b / avg_s / 1e9, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(b / avg_s / 1e9 / HBM_PEAK_GBS, 4)}
    tr = source_record("traffic.json", HEADLINE, dom)
    mu = source_record("mfma.json", HEADLINE, dom)
    roof.update({"traffic": None if tr is None else round(tr["bytes"]),
                 "alg_bytes_per_launch": round(b), "alg_flops_per_launch": fl, "avg_us": round(avg_s * 1e6, 3),
                 "hbm_frac": round(b / avg_s / 1e9 / HBM_PEAK_GBS, 4),
                 "mfma_frac": round(fl / avg_s / 1e12 / FP32_MFMA_PEAK_TFLOPS, 4) if fl else None,
                 "mfma_util_counter": None if mu is None else round(mu["mfma_util"], 4)})
    return roof


# ---------------------------------------------------------------- CPU oracle
def cpu_baseline():
    """The oracle (float64 numpy, as it stands) on a sample of the headline
    workload: the first SGD step of all 16 learners (16 learner-steps; the
    state and data generator set up untimed), with numpy's BLAS on every core
    of this process's affinity set, then one learner's next step with BLAS
    limited to one thread."""
    import cases
    from oracle import method as M
    from threadpoolctl import threadpool_info, threadpool_limits
    cores = len(os.sched_getaffinity(0))
    blas = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    wl, P, S, K1, K2, B, lr, _ = WORKLOADS[HEADLINE]
    c = cases.named(wl, P, S, K1, K2, B, lr, seed=0)
    prob = cases.oracle_problem(c)
    st = M.create(prob)
    data = M.Dataset(prob)
    t0 = time.perf_counter()
    M.sgd_step_all(prob, data, st)
    dt = time.perf_counter() - t0
    with threadpool_limits(1):
        t1 = time.perf_counter()
        M.learner_step(prob, data, st, 0)
        dt1 = time.perf_counter() - t1
    return {"value": round(P / dt, 3), "unit": "learner-steps/s", "cores": cores, "kind": "oracle",
            "sample": f"first SGD step of all {P} learners of {HEADLINE} (P=16 S=4 K1=4 K2=2 B=32): {P} "
                      f"learner-steps in {dt:.2f} s, float64 numpy, BLAS threads {blas}; the cluster and global "
                      f"means are not in the sample",
            "blas_threads": blas,
            "value_1thread": round(1.0 / dt1, 4),
            "sample_1thread": f"learner 0's second SGD step, BLAS limited to 1 thread: {dt1:.2f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50, help="timed rounds of the headline workload (50: about 1 s)")
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--only", default=None, help="time only these workloads, comma-separated (profiling runs)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first copy a 1 GiB tensor 3 times (a plain copy kernel of known bytes for counter runs)")
    ap.add_argument("--quick", action="store_true",
                    help="counter runs: every workload times --steps rounds and 3 launches per kernel class")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the Hier-AVG learners are rows of one replica array on a single "
              "MI355X; the library has no multi-GPU path", file=sys.stderr)
        sys.exit(2)
    import torch
    assert torch.cuda.is_available(), "bench.py needs the GPU"
    torch.cuda.set_device(0)
    if args.copy_calibration:
        src = torch.ones(1 << 28, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        torch.cuda.empty_cache()

    configs = {}
    head = None
    for name, spec in WORKLOADS.items():
        if args.only and name not in args.only.split(","):
            continue
        reps = 3 if args.quick else None
        if name == HEADLINE:
            c, ms, stats, dur = run_workload(name, args.steps, args.warmup, reps)
            head = (c, ms, stats, dur)
        else:
            c, ms, stats, dur = run_workload(name, args.steps if args.quick else spec[7], args.warmup if args.quick else 5,
                                             reps)
            configs[name] = summarize(name, c, ms, stats, dur)
        log(f"[bench] {name} done: {ms:.4f} ms/round")
    cpu = None if (args.no_cpu_baseline or args.only) else cpu_baseline()
    if cpu:
        log(f"[bench] cpu baseline done: {cpu['value']} learner-steps/s on {cpu['cores']} cores")
    if head is None:
        print(json.dumps({"configs": configs}), flush=True)
        return
    c, ms, stats, dur = head
    summ = summarize(HEADLINE, c, ms, stats, dur)
    line = {
        "metric": "learner-SGD-steps/sec and averaging HBM GB/s (frac of peak), 1 MI355X",
        "value": summ["learner_steps_per_s"],
        "unit": "learner-steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": HEADLINE, "P": c["P"], "S": c["S"], "K1": c["K1"], "K2": c["K2"], "B": c["B"],
                   "lr": c["lr"], "N": c["N"], "seed": c["seed"], "learner_steps_per_round": summ["learner_steps_per_round"],
                   "schedule": summ["schedule"]},
        "roofline": roofline(c, stats, dur),
        "cpu_baseline": cpu,
        "round_mfma_frac": summ["round_mfma_frac"],
        "round_alg_bytes_frac": summ["round_alg_bytes_frac"],
        "launches_per_round": summ["launches_per_round"],
        "kernels": summ["kernels"],
        "configs": configs,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
