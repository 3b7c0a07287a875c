"""Benchmark: training frames/s of one learner step on one MI355X.

A step is the whole learner step of H-ADPSGD for one mini-batch: BLSTM
forward, softmax cross-entropy forward/backward, BPTT, and the fused ADPSGD
update (which also refreshes the bf16 operand copy), all through the C ABI.
Inputs are seeded synthetic tensors with the paper's shapes, resident in HBM
before timing starts.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload full_b128]

Prints one JSON line.  Only one GPU is supported: the learner step is one
GPU's share of the paper's system."""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "training frames/sec per GPU (BLSTM fwd+bwd+update); MFMA util %, HBM GB/s %"
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3      # MI355X dense fp32 MFMA
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E


def kernel_work(name, c, n_params, fused_gx=False):
    """Algorithmic work of all launches of kernel `name` in one step:
    (bound, amount, unit, launches).  FLOPs count 2 per multiply-add of the
    products the step needs; bytes count each tensor read or written once.
    fused_gx: the persistent forward computes the input projection itself
    (no gemm_gx launch), so its work includes that product."""
    L, D, H, P, K, T, B = (c[k] for k in "LDHPKTB")
    M = T * B
    es = 2 if c["precision"] == "bf16" else 4
    Dl = [D] + [2 * H] * (L - 1)
    if name == "gemm_gx":
        return "mfma", sum(2 * 2 * M * 4 * H * d for d in Dl), "flop", L
    if name in ("lstm_rec_fwd", "lstm_rec_bwd", "lstm_rec_fwd_persist", "lstm_rec_bwd_persist"):
        # the recurrent products h_prev W_hh^T (forward) or da W_hh (BPTT);
        # the first step of each direction has no previous state
        rec = L * (T - 1) * 2 * 2 * B * 4 * H * H
        if fused_gx and name == "lstm_rec_fwd_persist":
            rec += sum(2 * 2 * M * 4 * H * d for d in Dl)
        return "mfma", rec, "flop", None
    if name == "gemm_bwd_group":
        # per layer above layer 0, right after its BPTT: dX (the weight
        # gradients of every layer follow the last BPTT, in gemm_dw_group)
        return "mfma", (L - 1) * 2 * M * 2 * H * 8 * H, "flop", L - 1
    if name == "gemm_dw_group":
        # dW_ih and dW_hh of every layer, up to 12 products per launch
        return "mfma", (sum(2 * 2 * 4 * H * d * M for d in Dl) + L * 2 * 2 * 4 * H * H * (T - 1) * B), "flop", \
            -(-2 * L // 12)
    if name == "gemm_dwih":
        return "mfma", sum(2 * 2 * 4 * H * d * M for d in Dl), "flop", L
    if name == "gemm_dwhh":
        return "mfma", L * 2 * 2 * 4 * H * H * (T - 1) * B, "flop", L
    if name == "gemm_dx":
        return "mfma", (L - 1) * 2 * M * 2 * H * 8 * H, "flop", L - 1
    if name == "gemm_z":
        return "mfma", 2 * M * P * 2 * H, "flop", 1
    if name in ("gemm_logits", "gemm_logits_ds", "gemm_dws", "gemm_dz"):
        return "mfma", 2 * M * K * P, "flop", 1
    if name in ("logits_blk", "logits_ds_blk"):
        # the logits products as class-block kernels (W_s block in registers)
        return "mfma", 2 * M * K * P, "flop", 1
    if name == "gemm_dws_dz":
        # dW_s and dz in one launch
        return "mfma", 2 * 2 * M * K * P, "flop", 1
    if name in ("gemm_dwl", "gemm_dy"):
        return "mfma", 2 * M * P * 2 * H, "flop", 1
    if name == "gemm_dwl_dy":
        return "mfma", 2 * 2 * M * P * 2 * H, "flop", 1
    if name == "softmax_ce_rows":
        Kp = (K + 7) // 8 * 8
        return "hbm", 2 * M * Kp * es + 8 * M, "byte", 1
    if name == "adpsgd_update":
        return "hbm", n_params * (4 * 4 + (2 if es == 2 else 0)), "byte", 1
    return None


def recorded_traffic(kernel, workload):
    """HBM bytes per launch of `kernel`, from the rocprofv3 FETCH_SIZE /
    WRITE_SIZE counters recorded in profiles/traffic.json (each divided by
    what the same counter reads for a plain device copy of known size).
    None when no record matches this kernel and workload, or when the
    kernel's source file has changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        rec = json.load(fh)
    for r in rec.get("kernels", []):
        if r["kernel"] != kernel or r["workload"] != workload:
            continue
        src = os.path.join(ROOT, r["source"])
        if not os.path.exists(src):
            return None
        with open(src, "rb") as fh:
            if hashlib.sha256(fh.read()).hexdigest() != r["source_sha256"]:
                return None
        return int((r["fetch_kib_per_dispatch"] / rec["copy_factor_fetch"]
                    + r["write_kib_per_dispatch"] / rec["copy_factor_write"]) * 1024)
    return None


def calibrate_copy(mib):
    """A plain device-to-device copy of `mib` MiB (one torch copy kernel),
    run three times: the reference for scaling the HBM byte counters."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"calibrate_copy_bytes": n * 4, "launches": 3}), flush=True)


def peak_for(bound, precision):
    if bound == "hbm":
        return PEAK_HBM_GBS, "GB/s"
    return (PEAK_BF16_TFLOPS if precision == "bf16" else PEAK_FP32_TFLOPS), "TFLOP/s"


def cpu_baseline(cfg, budget_s=12.0, one_thread_s=6.0):
    """The float64 oracle on the host cores, on a bounded slice of the same
    workload: the full layer dimensions with B=16 sequences, whole steps
    (gradient + update) repeated until the time budget is spent; then the
    same on one BLAS thread.  Frames/s of the slice (the oracle's cost is
    linear in B, so the slice's rate is the workload's)."""
    import numpy as np
    from oracle import blstm_ref as ref
    from paper_1907_05701_amd import inputs
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threadpool_limits = None
        threads = os.cpu_count()
    Bs = min(16, cfg["B"])
    dims = ref.Dims(L=cfg["L"], D=cfg["D"], H=cfg["H"], P=cfg["P"], K=cfg["K"], T=cfg["T"], B=Bs)
    n = ref.param_count(dims)
    theta = inputs.params(n)
    peer = inputs.peer(theta)
    x = inputs.features(dims.T, Bs, dims.D)
    lab = inputs.labels(dims.T, Bs, dims.K, dist=cfg["label_dist"])

    def rate(budget):
        steps, t0 = 0, time.perf_counter()
        while True:
            g = ref.learner_gradient(theta, dims, x, lab)
            ref.adpsgd_update(theta, peer, g["grad"], cfg["lr"])
            steps += 1
            el = time.perf_counter() - t0
            if el >= budget or steps >= 50:
                return steps, el

    steps, el = rate(budget_s)
    out = {"value": round(steps * dims.T * Bs / el, 2), "unit": "frames/s", "cores": int(threads),
           "kind": "oracle", "nproc": os.cpu_count(), "omp_num_threads": os.environ.get("OMP_NUM_THREADS"),
           "sample": f"{steps} float64 oracle step(s) (gradient + update) at the workload's layer "
                     f"dimensions with B={Bs} of {cfg['B']} sequences, {el:.1f} s on {threads} BLAS threads"}
    if threadpool_limits is not None:
        with threadpool_limits(limits=1):
            s1, e1 = rate(one_thread_s)
        out["one_thread_value"] = round(s1 * dims.T * Bs / e1, 2)
        out["one_thread_sample"] = f"{s1} step(s), {e1:.1f} s on 1 BLAS thread"
    return out


CLASSES = {
    "gate_projection": ("gemm_gx",),
    "backward_products": ("gemm_bwd_group", "gemm_dw_group", "gemm_dwih", "gemm_dwhh", "gemm_dx"),
    "head_products": ("gemm_z", "gemm_logits", "gemm_logits_ds", "logits_blk", "logits_ds_blk", "gemm_dws", "gemm_dz",
                      "gemm_dws_dz", "gemm_dwl", "gemm_dy", "gemm_dwl_dy"),
    "recurrence_fwd": ("lstm_rec_fwd_persist", "lstm_rec_fwd"),
    "recurrence_bwd": ("lstm_rec_bwd_persist", "lstm_rec_bwd"),
}


def class_rates(st, cfg, lr, steps):
    """Per-class MFMA rates of `steps` eager learner steps: each class's
    algorithmic FLOPs over its kernels' summed event time, against the bf16
    peak; and the recurrences' time per time step."""
    from paper_1907_05701_amd import binding as bd
    import torch
    bd.blstm_timing_begin("")
    for _ in range(steps):
        st.step(lr)
    per = bd.blstm_timing_end(cap=128)
    torch.cuda.synchronize()
    ms = {k: v[1] / steps for k, v in per.items()}
    fused = "gemm_gx" not in ms and "lstm_rec_fwd_persist" in ms
    mfma = {}
    for cls, names in CLASSES.items():
        t = sum(ms.get(k, 0.0) for k in names)
        flop = 0
        for k in names:
            if k not in ms:
                continue
            w = kernel_work(k, cfg, st.n, fused_gx=fused)
            if w is not None and k not in ("gemm_logits_ds", "logits_ds_blk"):   # the logits count once (recomputed for ds)
                flop += w[1]
        if t > 0:
            tf = flop / (t * 1e-3) / 1e12
            mfma[cls] = {"ms_per_step": round(t, 4), "gflop_per_step": round(flop / 1e9, 2),
                         "tflops": round(tf, 1), "frac_of_peak": round(tf / PEAK_BF16_TFLOPS, 4)}
    L, T = cfg["L"], cfg["T"]
    rec = {}
    for key, cls in (("fwd", "recurrence_fwd"), ("bwd", "recurrence_bwd")):
        if cls in mfma:
            rec[key] = round(mfma[cls]["ms_per_step"] * 1e3 / (L * T), 3)
    # the forward launches' time includes the input projection when fused,
    # the BPTT launches' the sum of the layer above's dX partials when those
    # reductions (one per layer above layer 0) are not launched
    rec["fwd_includes_input_projection"] = fused
    n_red = per.get("splitk_reduce_group", (0, 0.0))[0] / steps
    rec["bwd_includes_dx_partial_sums"] = "lstm_rec_bwd_persist" in ms and n_red < L - 1
    return {"mfma": mfma, "recurrence_step_us": rec,
            "kernel_ms": {k: round(v, 4) for k, v in sorted(ms.items(), key=lambda kv: -kv[1])}}


def update_rate(cfg, n, iters):
    """The fused update alone at the paper's parameter count with 8 resident
    replica gradients (the update-only workload), timed with HIP events on
    the launching stream: HBM GB/s of its algorithmic bytes."""
    import torch
    from paper_1907_05701_amd import binding as bd
    from paper_1907_05701_amd import inputs
    R = 8
    dev = torch.device("cuda:0")
    theta0 = inputs.params(n)
    th = torch.from_numpy(theta0).to(dev)
    pe = torch.from_numpy(inputs.peer(theta0)).to(dev)
    gs = [torch.from_numpy(g).to(dev) for g in inputs.replica_grads(n, R)]
    s = torch.cuda.current_stream()
    for _ in range(3):
        bd.adpsgd_step(th, pe, gs, 1.0 / R, cfg["lr"], 0, None)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(s)
    for _ in range(iters):
        bd.adpsgd_step(th, pe, gs, 1.0 / R, cfg["lr"], 0, None)
    e1.record(s)
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / iters
    nbytes = update_bytes(n, R, False, False)
    gbs = nbytes / us / 1e3
    del gs, th, pe
    torch.cuda.empty_cache()
    return {"n": n, "R": R, "bytes_per_param": nbytes // n, "us": round(us, 2), "GB/s": round(gbs, 1),
            "frac_of_peak": round(gbs / PEAK_HBM_GBS, 4)}


def update_bytes(n, R, write_peer, shadow):
    """Algorithmic HBM bytes of one fused update: R replica gradients, theta
    and theta_peer read once, theta written (and theta_peer, the bf16 copy)."""
    return n * (4 * R + 4 + 4 + 4 + (4 if write_peer else 0) + (2 if shadow else 0))


def cpu_update_baseline(n, R, lr, budget_s=12.0):
    """The float32-order oracle update on the host on a bounded slice of the
    parameter vector, in GB/s of the same algorithmic bytes."""
    import numpy as np
    from oracle import blstm_ref as ref
    from paper_1907_05701_amd import inputs
    ns = min(n, 1 << 22)
    theta = inputs.params(ns)
    peer = inputs.peer(theta)
    grads = inputs.replica_grads(ns, R)
    reps, t0 = 0, time.perf_counter()
    while True:
        ref.adpsgd_update_fp32(theta, peer, grads, 1.0 / R, lr)
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s or reps >= 200:
            break
    return {"value": round(update_bytes(ns, R, False, False) * reps / el / 1e9, 3), "unit": "GB/s", "cores": 1,
            "kind": "oracle",
            "sample": f"{reps} float32-order oracle update(s) of the first {ns} of {n} parameters "
                      f"with R={R}, {el:.1f} s (numpy, one thread)"}


def bench_update(args, cfg):
    """The update-only workload: R resident replica gradients of the full
    model's flat parameter vector, fused sum + SGD + pairwise averaging.
    Timed with HIP events on the launching stream; value in HBM GB/s of the
    algorithmic bytes, for the plain update and its variants (peer write,
    bf16 operand copy)."""
    import torch
    from paper_1907_05701_amd import binding as bd
    from paper_1907_05701_amd import inputs
    R, lr = cfg["R"], cfg["lr"]
    n = bd.blstm_param_count(bd.make_dims(*(cfg[k] for k in "LDHPKTB"), "fp32"))
    dev = torch.device("cuda:0")
    theta0 = inputs.params(n)
    th = torch.from_numpy(theta0).to(dev)
    pe = torch.from_numpy(inputs.peer(theta0)).to(dev)
    gs = [torch.from_numpy(g).to(dev) for g in inputs.replica_grads(n, R)]
    lp = torch.empty(n, dtype=torch.bfloat16, device=dev)
    s = torch.cuda.current_stream()
    variants = {"plain": (0, None), "write_peer": (bd.ADPSGD_WRITE_PEER, None), "bf16_copy": (0, lp),
                "write_peer_bf16_copy": (bd.ADPSGD_WRITE_PEER, lp)}
    res = {}
    for name, (flags, shadow) in variants.items():
        for _ in range(args.warmup):
            bd.adpsgd_step(th, pe, gs, 1.0 / R, lr, flags, shadow)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(s)
        for _ in range(args.steps):
            bd.adpsgd_step(th, pe, gs, 1.0 / R, lr, flags, shadow)
        e1.record(s)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / args.steps
        nbytes = update_bytes(n, R, flags & bd.ADPSGD_WRITE_PEER, shadow is not None)
        res[name] = {"bytes_per_param": nbytes // n, "us": round(us, 2), "GB/s": round(nbytes / us / 1e3, 1)}
    base = res["plain"]
    out = {"metric": "fused replica-sum + SGD + averaging update, HBM GB/s", "value": base["GB/s"],
           "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "ms_per_step": round(base["us"] / 1e3, 4), "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "fp32", "data": "synthetic",
           "config": {"workload": args.workload, "n": n, "R": R, "lr": lr},
           "roofline": {"bound": "hbm", "achieved": base["GB/s"], "peak": PEAK_HBM_GBS, "unit": "GB/s",
                        "frac": round(base["GB/s"] / PEAK_HBM_GBS, 5),
                        "traffic": recorded_traffic("adpsgd_update", args.workload), "kernel": "adpsgd_update",
                        "avg_launch_us": base["us"], "algorithmic_per_launch": update_bytes(n, R, False, False),
                        "algorithmic_unit": "byte"},
           "variants": res}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_update_baseline(n, R, lr)
    print(json.dumps(out), flush=True)


def bench_ring(args, cfg):
    """S super-learners of N replicas in the ring of eq. 7 on one GPU: a
    round is S*N learner gradients and S updates (each learner's update
    overlapped with the next learner's gradients).  value = all learners'
    frames per second."""
    import torch
    from paper_1907_05701_amd import inputs
    from paper_1907_05701_amd.ring import LearnerRing
    shape = {k: cfg[k] for k in "LDHPKTB"}
    S, N, lr = cfg["S"], cfg["N"], cfg["lr"]
    ring = LearnerRing(shape, S, N, precision=cfg["precision"])
    n = ring.steps[0][0].n
    thetas = [inputs.params(n, seed=s) for s in range(S)]
    batches = [[(inputs.features(cfg["T"], cfg["B"], cfg["D"], seed=100 + 10 * s + r),
                 inputs.labels(cfg["T"], cfg["B"], cfg["K"], seed=200 + 10 * s + r, dist=cfg["label_dist"]))
                for r in range(N)] for s in range(S)]
    ring.load(thetas, batches)
    for _ in range(args.warmup):
        ring.round(lr)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        ring.round(lr)
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    ring.check_recurrence()
    value = ring.frames_per_round * args.steps / el
    out = {"metric": "ring of learners (eq. 7): training frames/s of all learners on one GPU",
           "value": round(value, 1), "unit": "frames/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "ms_per_step": round(el * 1e3 / args.steps, 4), "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": cfg["precision"], "data": "synthetic",
           "config": {"workload": args.workload, **shape, "super_learners": S, "replicas": N,
                      "frames_per_round": ring.frames_per_round, "mode": "eager"}}
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="full_b128")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-update-measure", action="store_true",
                    help="skip the fused-update (8 replicas) measurement of the main workload")
    ap.add_argument("--breakdown", action="store_true", help="per-kernel times to stderr")
    ap.add_argument("--mode", choices=("graph", "eager"), default="graph",
                    help="replay the timed steps as one HIP graph, or launch them one by one")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (counter calibration)")
    args = ap.parse_args()
    if args.calibrate_copy:
        calibrate_copy(args.calibrate_copy)
        return
    if args.gpus != 1:
        print(f"bench.py measures one learner on one GPU; --gpus {args.gpus} is not supported "
              "(the multi-GPU exchange of the paper is not part of this library)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_1907_05701_amd import binding as bd
    from paper_1907_05701_amd import inputs
    from paper_1907_05701_amd.step import LearnerStep

    cfg = dict(inputs.CONFIGS[args.workload])
    if "R" in cfg:
        bench_update(args, cfg)
        return
    if "S" in cfg:
        bench_ring(args, cfg)
        return
    shape = {k: cfg[k] for k in "LDHPKTB"}
    st = LearnerStep(**shape, precision=cfg["precision"])
    theta = inputs.params(st.n)
    st.load(theta, inputs.features(cfg["T"], cfg["B"], cfg["D"]),
            inputs.labels(cfg["T"], cfg["B"], cfg["K"], dist=cfg["label_dist"]), inputs.peer(theta))
    lr = cfg["lr"]
    frames = cfg["T"] * cfg["B"]

    for _ in range(args.warmup):
        st.step(lr)
    torch.cuda.synchronize()
    # find the dominant kernel on one extra untimed step, run the way the
    # timed steps run (in graph mode: captured, with its event records, and
    # replayed)
    bd.blstm_timing_begin("")
    st.step(lr)
    per = bd.blstm_timing_end()
    torch.cuda.synchronize()
    ranked = sorted(per.items(), key=lambda kv: -kv[1][1])
    if args.breakdown:
        tot = sum(v[1] for v in per.values())
        for name, (cnt, ms) in ranked:
            print(f"  {name:22s} {cnt:5d} launches {ms * 1e3:10.1f} us {100 * ms / tot:5.1f}%",
                  file=sys.stderr)
    fused_gx = "gemm_gx" not in per and "lstm_rec_fwd_persist" in per
    dominant = next(n for n, _ in ranked if kernel_work(n, cfg, st.n, fused_gx) is not None)

    # timed region: K steps, the dominant kernel bracketed by HIP events on
    # the stream it runs on.  In graph mode the K steps (with their event
    # records) are captured once and replayed as one graph.
    if args.mode == "graph":
        warm = st.capture(lr, steps=1)
        for _ in range(max(args.warmup, 1)):
            warm.replay()
        torch.cuda.synchronize()
        graph = st.capture(lr, steps=args.steps)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        graph.replay()
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
    else:
        torch.cuda.synchronize()
        bd.blstm_timing_begin(dominant)
        t0 = time.perf_counter()
        for _ in range(args.steps):
            st.step(lr)
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
    if args.mode == "graph":
        # event records inside a graph carry no timestamps: time the dominant
        # kernel on eager steps right after the timed replay
        bd.blstm_timing_begin(dominant)
        for _ in range(args.steps):
            st.step(lr)
        torch.cuda.synchronize()
    dom = bd.blstm_timing_end()[dominant]
    st.check_recurrence()   # raises if a persistent launch's exchange wait gave up
    loss = float(st.loss.cpu()[0])

    # per-class achieved rates over a few eager steps with every kernel timed
    # by HIP events on its stream (each run of per-step launches is one pair)
    classes = class_rates(st, cfg, lr, steps=min(args.steps, 5))
    update = update_rate(cfg, st.n, iters=20) if not args.no_update_measure else None

    ms_per_step = elapsed * 1e3 / args.steps
    value = frames * args.steps / elapsed
    bound, amount, unit, _ = kernel_work(dominant, cfg, st.n, fused_gx)
    n_launch, total_ms = dom
    per_launch = amount * args.steps / n_launch
    avg_s = total_ms / n_launch / 1e3
    achieved = per_launch / avg_s / (1e9 if bound == "hbm" else 1e12)
    peak, punit = peak_for(bound, cfg["precision"])
    roofline = {"bound": bound, "achieved": round(achieved, 3), "peak": peak, "unit": punit,
                "frac": round(achieved / peak, 5), "traffic": recorded_traffic(dominant, args.workload),
                "kernel": dominant,
                "avg_launch_us": round(avg_s * 1e6, 3),
                "algorithmic_per_launch": per_launch, "algorithmic_unit": unit}
    out = {"metric": METRIC, "value": round(value, 1), "unit": "frames/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
           "dtype": cfg["precision"], "data": "synthetic",
           "config": {"workload": args.workload, **shape, "frames_per_step": frames, "mode": args.mode,
                      "params": st.n, "label_dist": cfg["label_dist"]},
           "loss_last_step": loss, "roofline": roofline, "mfma_by_class": classes["mfma"],
           "recurrence_step_us": classes["recurrence_step_us"], "kernel_ms_per_step": classes["kernel_ms"]}
    if update is not None:
        out["update_r8"] = update
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
