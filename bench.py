"""Benchmark of the Hier-AVG hot path on one MI355X.

One bench "step" is one Hier-AVG round (K2 blocks of K1 local SGD steps of
all P learners, the cluster means and the global mean) of the MLP
3072 -> 512 -> 10 workload with P=16, S=4, K1=4, K2=4, B=32, lr=0.05 on
synthetic data (N=50000 rows: class-mean pattern + N(0, 0.5) noise).
`value` is learner-SGD-steps per second (P*K1*K2 per round) with the dataset
and replicas resident in HBM.

Also reported, on the same JSON line:
  roofline      the dominant kernel of the round (largest launches x duration):
                algorithmic bytes (or flops) per launch over its mean duration,
                timed with HIP events on the handle's stream around 200
                back-to-back launches of it after the timed rounds
  averaging     the averaging-only workload (P=32 replicas of 11.7M floats,
                S=4, K1=1, K2=4, heavy-ball momentum 0.9, lr 0.1): HBM GB/s of
                the fused update + cluster mean and update + global mean
                kernels as a fraction of the 8 TB/s peak
  cpu_baseline  the CPU oracle (float64 numpy) on one round of the same
                workload, on this host's cores
"""

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)
sys.path.insert(0, os.path.join(ROOT, "tests"))

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
FP32_MFMA_PEAK_TFLOPS = 157.3  # MI355X dense fp32 matrix


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# ---------------------------------------------------------------- algorithmic work
def mlp_kernel_work(P, S, K1, K2, B, IN, H, C):
    """Algorithmic bytes and flops per launch of each kernel class of one MLP
    step (all P learners): every operand the step needs read once and every
    result written once, at its logical (unpadded) size.  Split-K partial
    sums are an implementation choice and are not counted.  The delayed-update
    kernels are counted for the launch that is timed (step 0 of block 0,
    where every learner reads replica 0's W1)."""
    f = 4
    G = P // S
    pairs = K1 * (K1 - 1) // 2
    tail = H + C * H + C  # b1, W2, b2: their cluster (global) mean rides in the block update (W1 mean)
    return {
        # forward of block 0's K1 steps from the common W1: W1 once, the
        # K1*P minibatches, the K1*P pre-activation blocks
        "fwd1_block_gemm": (f * (H * IN + K1 * P * B * IN + K1 * P * B * H), K1 * P * 2 * B * H * IN),
        # block end: the base read once, G cluster copies written, the block's
        # hidden errors and minibatch rows read
        "block_update_gemm": (f * (H * IN + G * H * IN + K1 * P * B * (H + IN) + 2 * P * tail),
                              K1 * P * 2 * B * H * IN),
        # Gram blocks of the round: every minibatch row read once, blocks written
        "gram": (f * (K2 * K1 * P * B * IN + K2 * P * pairs * B * B), K2 * P * pairs * 2 * B * B * IN),
        "w1_global_mean": (f * ((G + 1) * H * IN + 2 * P * tail), G * H * IN + P * tail),
        "fwd1_gemm": (P * f * (H * IN + B * IN + B * H), P * 2 * B * H * IN),
        "reduce1": (P * f * (H + B * H), P * B * H),
        "fwd2_gemm": (P * f * (C * H + B * H + B * C), P * 2 * B * C * H),
        "softmax_grad": (P * f * (C + 2 * B * C) + P * B * 8, P * B * C * 4),
        "bwd_hidden": (P * f * (B * C + C * H + 2 * B * H), P * 2 * B * C * H),
        "update2_gemm": (P * f * (2 * C * H + B * C + B * H + 2 * C), P * 2 * B * C * H),
        "update1_gemm": (P * f * (2 * H * IN + B * H + B * IN + 2 * H), P * 2 * B * H * IN),
        # update of W1 at step t and forward of step t+1: W1 read and written
        # once, G1 and the two minibatches read, the next pre-activations
        # written once; the group-mean variant moves the same bytes
        "step1_gemm": (P * f * (2 * H * IN + 2 * B * H + 2 * B * IN), P * 4 * B * H * IN),
        "step1_gemm_group_mean": (P * f * (2 * H * IN + 2 * B * H + 2 * B * IN), P * 4 * B * H * IN),
    }


def mean_bytes(P, D):
    return 2 * 4 * P * D


def counter_mfma_util(kernel_class):
    """MfmaUtil (fraction) of `kernel_class` from the committed counter summary
    (profiles/mfma.json), or None when the kernel's source has changed since."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "mfma.json")
    try:
        rec = json.load(open(path))["kernels"][kernel_class]
        cur = hashlib.sha256(open(os.path.join(ROOT, rec["source"]), "rb").read()).hexdigest()
    except (OSError, KeyError, ValueError):
        return None
    return rec["mfma_util"] if cur == rec["source_sha256"] else None


def counter_traffic(kernel_class):
    """HBM bytes per launch of `kernel_class` from the committed counter
    summary (profiles/traffic.json: FETCH_SIZE and WRITE_SIZE passes scaled by
    a calibration stream), or None when the kernel's source has changed since
    the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        rec = json.load(open(path))["kernels"][kernel_class]
        cur = hashlib.sha256(open(os.path.join(ROOT, rec["source"]), "rb").read()).hexdigest()
    except (OSError, KeyError, ValueError):
        return None
    return rec["bytes"] if cur == rec["source_sha256"] else None


# ---------------------------------------------------------------- main workload
def bench_mlp(args):
    import torch
    import cases
    from paper_1903_05133_amd import HierAvg

    c = cases.named("mlp_3072_512_10", 16, 4, 4, 4, 32, 0.05, seed=0)
    P, K1, K2, B = c["P"], c["K1"], c["K2"], c["B"]
    IN, H, C = c["IN"], c["H"], c["C"]
    h = HierAvg(config=cases.native_config(c))
    stream = torch.cuda.Stream()
    h.set_stream(stream)
    for _ in range(args.warmup):
        h.round()
    h.sync()
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record(stream)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        h.round()
    end.record(stream)
    h.sync()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = start.elapsed_time(end)
    log(f"[bench] mlp: {args.steps} rounds in {ms:.3f} ms (host wall {wall * 1e3:.3f} ms)")

    # Second timed pass with HIP events around every launch.
    h.profile(True)
    start.record(stream)
    for _ in range(args.steps):
        h.round()
    end.record(stream)
    stats = h.profile_read()
    h.profile(False)
    torch.cuda.synchronize()
    ms_prof = start.elapsed_time(end)
    # Per-launch durations: every kernel class of the round timed over 200
    # back-to-back launches between two HIP events on the handle's stream (the
    # event pair adds a few microseconds to a single launch; here it is spread
    # over 200).  This changes the replicas, so it comes last.
    dur_ms = {name: h.time_kernel(name, 200) for name in stats if name != "draw_indices"}
    h.close()

    work = mlp_kernel_work(P, c["S"], K1, K2, B, IN, H, C)
    D = H * IN + H + C * H + C
    work["group_mean"] = (mean_bytes(P, D), P * D)
    work["global_mean"] = (mean_bytes(P, D), P * D)
    work["tail_group_mean"] = (mean_bytes(P, D - H * IN), P * (D - H * IN))
    work["tail_global_mean"] = (mean_bytes(P, D - H * IN), P * (D - H * IN))
    kernels = {}
    for name, (n, tot) in stats.items():
        avg = dur_ms.get(name, tot / n)
        b, fl = work.get(name, (0, 0))
        kernels[name] = {"launches": n, "avg_us": round(avg * 1e3, 3), "share": None, "GBps": round(b / (avg * 1e-3) / 1e9, 1) if b else None,
                         "TFLOPs": round(fl / (avg * 1e-3) / 1e12, 2) if fl else None}
    total = sum(t for _, t in stats.values())
    for name, (n, tot) in stats.items():
        kernels[name]["share"] = round(tot / total, 4)
    # the dominant kernel among those with a stated algorithmic work
    dom = max((k for k in dur_ms if k in work), key=lambda k: dur_ms[k] * stats[k][0])
    avg_s = dur_ms[dom] * 1e-3
    b, fl = work[dom]
    traffic = counter_traffic(dom)
    # The bound is the resource whose ideal time for the kernel's algorithmic
    # work is longer: HBM bytes at 8 TB/s or fp32 MFMA flops at 157.3 TFLOP/s.
    mfma_bound = fl / (FP32_MFMA_PEAK_TFLOPS * 1e12) > b / (HBM_PEAK_GBS * 1e9)
    if mfma_bound:
        roof = {"kernel": dom, "bound": "mfma", "achieved": round(fl / avg_s / 1e12, 2),
                "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(fl / avg_s / 1e12 / FP32_MFMA_PEAK_TFLOPS, 4)}
    else:
        roof = {"kernel": dom, "bound": "hbm", "achieved": round(b / avg_s / 1e9, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(b / avg_s / 1e9 / HBM_PEAK_GBS, 4)}
    roof.update({"traffic": None if traffic is None else round(traffic),
                 "alg_bytes_per_launch": b, "alg_flops_per_launch": fl, "avg_us": round(avg_s * 1e6, 3),
                 "hbm_frac": round(b / avg_s / 1e9 / HBM_PEAK_GBS, 4),
                 "mfma_frac": round(fl / avg_s / 1e12 / FP32_MFMA_PEAK_TFLOPS, 4) if fl else None})
    mu = counter_mfma_util(dom)
    roof["mfma_util_counter"] = None if mu is None else round(mu, 4)
    steps_per_round = P * K1 * K2
    return {
        "value": steps_per_round * args.steps / (ms * 1e-3),
        "ms_per_step": ms / args.steps,
        "profiled_ms_per_step": ms_prof / args.steps,
        "config": {"workload": "mlp_3072_512_10", "P": P, "S": c["S"], "K1": K1, "K2": K2, "B": B, "lr": c["lr"],
                   "N": c["N"], "seed": c["seed"], "learner_steps_per_round": steps_per_round},
        "roofline": roof,
        "kernels": kernels,
    }


# ---------------------------------------------------------------- averaging-only
def bench_averaging(args):
    import torch
    import cases
    from paper_1903_05133_amd import HierAvg

    c = cases.named("averaging_11_7M", 32, 4, 1, 4, 1, 0.1, seed=0)
    P, D = c["P"], c["IN"]
    h = HierAvg(config=cases.native_config(c))
    stream = torch.cuda.Stream()
    h.set_stream(stream)
    for _ in range(2):
        h.round()
    h.sync()
    rounds = args.avg_rounds
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for _ in range(rounds):
        h.round()
    end.record(stream)
    h.sync()
    ms = start.elapsed_time(end)
    h.profile(True)
    for _ in range(rounds):
        h.round()
    stats = h.profile_read()
    h.profile(False)
    dur_ms = {name: h.time_kernel(name, 20) for name in stats}
    h.close()
    per_launch = 20 * P * D  # read w, v, g; write w, v
    out = {"config": {"workload": "averaging_11_7M", "P": P, "S": c["S"], "K1": c["K1"], "K2": c["K2"], "D": D,
                      "momentum": c["momentum"], "lr": c["lr"]},
           "ms_per_round": ms / rounds, "alg_bytes_per_launch": per_launch, "kernels": {}}
    for name, (n, tot) in stats.items():
        avg_s = dur_ms[name] * 1e-3
        gbs = per_launch / avg_s / 1e9
        out["kernels"][name] = {"launches": n, "avg_us": round(avg_s * 1e6, 2), "GBps": round(gbs, 1),
                                "frac": round(gbs / HBM_PEAK_GBS, 4)}
    round_bytes = per_launch * c["K1"] * c["K2"]
    out["round_GBps"] = round(round_bytes / (ms / rounds * 1e-3) / 1e9, 1)
    out["round_frac"] = round(out["round_GBps"] / HBM_PEAK_GBS, 4)
    return out


# ---------------------------------------------------------------- CPU oracle
def cpu_baseline():
    import cases
    from oracle import method as M
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = 1
    c = cases.named("mlp_3072_512_10", 16, 4, 4, 4, 32, 0.05, seed=0)
    prob = cases.oracle_problem(c)
    # whole rounds of the timed workload until about 10 s of CPU work (at most 8)
    st = M.create(prob)
    data = M.Dataset(prob)
    rounds = 0
    t0 = time.perf_counter()
    while rounds < 8 and (rounds == 0 or time.perf_counter() - t0 < 10.0):
        M.hieravg_round(prob, st, data)
        rounds += 1
    dt = time.perf_counter() - t0
    steps = rounds * c["P"] * c["K1"] * c["K2"]
    return {"value": round(steps / dt, 2), "unit": "learner-steps/s", "cores": threads, "kind": "oracle",
            "sample": f"{rounds} round{'s' if rounds > 1 else ''} of mlp_3072_512_10 (P=16 S=4 K1=4 K2=4 B=32): {steps} learner-steps "
                      f"in {dt:.2f} s, float64 numpy"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--avg-rounds", type=int, default=20)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-averaging", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the Hier-AVG learners are rows of one replica array on a single "
              "MI355X; multi-GPU sharding is not part of this build", file=sys.stderr)
        sys.exit(2)
    import torch
    assert torch.cuda.is_available(), "bench.py needs the GPU"
    torch.cuda.set_device(0)

    res = bench_mlp(args)
    log(f"[bench] mlp done: {res['value']:.0f} learner-steps/s, {res['ms_per_step']:.4f} ms/round")
    avg = None if args.no_averaging else bench_averaging(args)
    if avg:
        log(f"[bench] averaging done: {avg['round_GBps']} GB/s per round")
    cpu = None if args.no_cpu_baseline else cpu_baseline()
    if cpu:
        log(f"[bench] cpu baseline done: {cpu['value']} learner-steps/s on {cpu['cores']} threads")
    line = {
        "metric": "learner-SGD-steps/sec and averaging HBM GB/s (frac of peak), 1 MI355X",
        "value": round(res["value"], 1),
        "unit": "learner-steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(res["ms_per_step"], 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": res["config"],
        "roofline": res["roofline"],
        "cpu_baseline": cpu,
        "averaging": avg,
        "profiled_ms_per_step": round(res["profiled_ms_per_step"], 5),
        "kernels": res["kernels"],
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
