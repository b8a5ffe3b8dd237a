#!/usr/bin/env python3
"""Benchmark of the exit-head training step (EE-Tuning) on one MI355X.

A step is one ee_multi_exit_step over one synthetic batch: for every exit,
forward (norm, optional SwiGLU MLP, vocabulary projection, cross-entropy),
backward into the exit's own parameters, weighted loss.  Inputs are resident
in HBM before the timed region starts.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

Prints one JSON line on stdout; progress goes to stderr.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "exit-head fwd+bwd tokens/sec at h=4096,V=32000; % bf16 MFMA peak"
PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}   # MI355X dense MFMA
PEAK_HBM_GBS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
# launch name -> label of the counter-measured traffic of the same kernel
TRAFFIC_LABEL = {"exit norm": "norm (one pass)", "mlp pre-norm": "norm (one pass)",
                 "exit norm rms": "norm statistics", "mlp pre-norm rms": "norm statistics",
                 "exit norm apply": "norm apply", "mlp pre-norm apply": "norm apply"}


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_flops(w, name):
    """Algorithmic flops of one launch of each GEMM of the step (2 per MAC)."""
    N, h, V, I = w.n_tokens, w.hidden, w.vocab, w.intermediate
    table = {
        "logits + softmax partials": 2 * N * h * V,
        "output-matrix gradient": 2 * N * h * V,
        "gate and up projections + swiglu": 2 * 2 * N * h * I,
        "down projection + residual": 2 * N * h * I,
        "dZ": 2 * N * h * V,
        "dA + swiglu backward, down gradient": 2 * 2 * N * h * I,
        "gate and up gradients": 2 * 2 * N * h * I,
    }
    return table.get(name)


def step_flops(w):
    """Algorithmic flops per step: 4hV per token per Norm/Embedding exit and
    14hI + 6hV per token per MLP exit (the gain gradients come from the
    weight-gradient GEMMs, so no dU product is needed)."""
    N, h, V, I = w.n_tokens, w.hidden, w.vocab, w.intermediate
    per = 14 * h * I + 6 * h * V if w.kind == 2 else 4 * h * V
    return per * N * w.n_exits


def side_pass_bytes(w, name):
    """Algorithmic HBM bytes of one launch of the step's HBM-bound passes:
    what each pass must read and write at least (the norm in one pass: read
    the rows, write their scales, Z and the token-contiguous copy of x_hat, or
    U and the token-contiguous copy of U_hat; norm statistics: read the rows;
    norm apply: read the rows and the scales, write as the one pass does;
    cross-entropy reduce: read the softmax partials; G's row sums (a bias
    in the unshifted form): read P' and the coefficients, write the
    per-chunk sums;
    seed: read P and write G in place; operand scale: read and write the
    token-contiguous x_hat, read the per-token coefficients)."""
    N, h, V, I = w.n_tokens, w.hidden, w.vocab, w.intermediate
    es = 2 if w.dtype == "bf16" else 4
    ldn = (N + 63) // 64 * 64
    slices = (V + 63) // 64
    table = {
        "exit norm": N * h * es + N * 4 + N * h * es + h * ldn * es,
        "mlp pre-norm": N * h * es + N * 4 + N * h * es + h * ldn * es,
        "exit norm rms": N * h * (4 if w.kind == 2 else es) + N * 4,
        "mlp pre-norm rms": N * h * es + N * 4,
        "exit norm apply": N * h * (4 if w.kind == 2 else es) + N * 4 + N * h * es + h * ldn * es,
        "mlp pre-norm apply": N * h * es + N * 4 + N * h * es + h * ldn * es,
        "cross-entropy reduce": 2 * slices * ldn * 4 + 3 * N * 4,
        "logit seed": 2 * V * ldn * es + slices * ldn * 4,
        "operand scale (or seed, if out of range) and loss": 2 * h * ldn * es + 2 * N * 4,
        "logit-gradient row sums (unshifted form)": V * ldn * es + ldn * 4 + ((ldn + 2047) // 2048) * V * 4,
        "exit norm backward": 2 * N * h * 4 + N * h * es,
    }
    return table.get(name)


def profile_figure(workload, kernel):
    """Mean duration (ms) of a kernel in the committed rocprofv3 kernel-trace
    summary of this workload, if it was taken on the current sources."""
    from paper_2402_00518_amd.traffic import source_digest
    try:
        data = json.load(open(os.path.join(ROOT, "profiles", "kernel_times.json")))
    except (OSError, ValueError):
        return None
    rec = data.get(workload, {}).get(kernel)
    if not rec or rec.get("source_digest") != source_digest():
        return None
    return rec


def measured_traffic(workload, kernel):
    """HBM bytes per launch (read + write, copy-calibrated) from committed
    rocprofv3 counter runs, if they were taken on the current kernel sources;
    else None."""
    from paper_2402_00518_amd.traffic import source_digest
    try:
        data = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    rec = data.get(workload, {}).get(kernel)
    if not rec or rec.get("source_digest") != source_digest():
        return None
    return rec.get("bytes_per_launch")


def adam_leg(sess, steps, warmup):
    """The Adam update of every exit parameter (fp32 master, bf16 parameter)
    after the step: HBM-bound, 30 algorithmic bytes per parameter (read g, m,
    v, master; write m, v, master and the bf16 copy; 28 for fp32 without a
    master)."""
    import torch
    sess.init_optimizer(master=True)
    for t in range(1, warmup + 1):
        sess.update(t, 1e-4)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for t in range(warmup + 1, warmup + steps + 1):
        sess.update(t, 1e-4)
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / steps
    n_params, n_bytes = 0, 0
    for params in sess.params:
        for p in params.values():
            n_params += p.numel()
            n_bytes += p.numel() * (30 if p.dtype == torch.bfloat16 else 28)
    gbps = n_bytes / (ms / 1e3) / 1e9
    return {"ms": ms, "params": n_params, "bytes_per_launch": n_bytes, "achieved_GBps": gbps,
            "peak_GBps": PEAK_HBM_GBS, "frac": gbps / PEAK_HBM_GBS, "bound": "hbm"}


def decode_leg(sess, rows_list=(1, 8, 32), iters=50):
    """The confidence-based exit decision of exit 0 at decode (forward only,
    a few rows): HBM-bound, algorithmic bytes = every exit weight read once
    plus the rows' hidden states.  Reports the whole call and, from the
    library's kernel timer, the output-matrix kernel alone."""
    import torch
    from paper_2402_00518_amd import binding as B
    e = sess.c_exits[0]
    es = 2 if sess.dtype == B.EE_BF16 else 4
    w_bytes = sum(p.numel() * p.element_size() for p in sess.params[0].values())
    w_out_bytes = sess.params[0]["w_out"].numel() * es
    out = {}
    for rows in rows_list:
        x = sess.x[0][:rows]
        ws_bytes = B.ee_decode_workspace_bytes(e, rows)
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
        tok = torch.empty(rows, dtype=torch.int32, device="cuda")
        conf = torch.empty(rows, dtype=torch.float32, device="cuda")
        flag = torch.empty(rows, dtype=torch.int32, device="cuda")
        stream = torch.cuda.current_stream().cuda_stream
        call = lambda: B.ee_exit_decide(e, x, rows, 0.9, tok, conf, flag, ws, ws_bytes, stream)
        for _ in range(5):
            call()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(iters):
            call()
        b.record()
        torch.cuda.synchronize()
        us = a.elapsed_time(b) / iters * 1e3
        B.ee_profile_start()
        for _ in range(iters):
            call()
        kt = B.ee_profile_stop()
        n, t = kt["decode logits partials"]
        k_us = t / n * 1e3
        total = w_bytes + rows * sess.hidden * es
        out[str(rows)] = {"us": us, "achieved_GBps": total / (us / 1e6) / 1e9,
                          "logits_kernel_us": k_us,
                          "logits_kernel_GBps": w_out_bytes / (k_us / 1e6) / 1e9,
                          "frac": (w_out_bytes / (k_us / 1e6) / 1e9) / PEAK_HBM_GBS}
    return {"bound": "hbm", "peak_GBps": PEAK_HBM_GBS, "threshold": 0.9, "rows": out}


def copy_calibration(mib, copies=3):
    """Plain device-to-device copies of a known size; a counter run over the
    bench reads them to calibrate FETCH_SIZE and WRITE_SIZE."""
    import torch
    src = torch.ones(mib << 18, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(copies):
        dst.copy_(src)
    torch.cuda.synchronize()
    log(f"copy calibration: {copies} copies of {mib} MiB")


def cpu_model():
    """The host CPU's model name, from /proc/cpuinfo."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(batch, sample_tokens, min_seconds=10.0):
    """The fp64 oracle on the host cores this process may run on, BLAS
    threads set to that count."""
    import numpy as np
    import oracle as O
    import workloads as W
    cores = len(os.sched_getaffinity(0))
    try:
        from threadpoolctl import threadpool_limits
        limiter = threadpool_limits(limits=cores, user_api="blas")
    except Exception:
        limiter = None
    w = batch.workload
    n = w.n_tokens if sample_tokens <= 0 else min(sample_tokens, w.n_tokens)
    exits = O.exits_from_batch(batch)
    xs = [W.decode(x[:n]) for x in batch.hidden]
    y = batch.targets[:n]
    # Repeat the step until at least min_seconds of CPU work have been timed.
    reps, dt = 0, 0.0
    while reps == 0 or (dt < min_seconds and reps < 16):
        t0 = time.perf_counter()
        O.multi_exit_step(exits, xs, y, list(w.exit_weights))
        dt += time.perf_counter() - t0
        reps += 1
    threads = cores
    try:
        from threadpoolctl import threadpool_info
        threads = max((p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"),
                      default=cores)
    except Exception:
        pass
    if limiter is not None:
        limiter.restore_original_limits()
    return {"value": reps * n / dt, "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
            "cpu_model": cpu_model(), "blas_threads": int(threads),
            "sample": f"first {n} of {w.n_tokens} tokens, all {w.n_exits} exit(s), full h={w.hidden} "
                      f"V={w.vocab}; fp64 numpy forward+backward, {reps} step(s) in {dt:.1f} s",
            "seconds": dt}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="llama7b_norm")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-sample-tokens", type=int, default=0,
                    help="tokens of the batch the oracle runs on (0: all)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-kernel-pass", action="store_true")
    ap.add_argument("--no-update-leg", action="store_true",
                    help="skip timing the Adam update and the decode-time exit decision")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="after the step, copy a buffer of this size 3 times (counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py: the exit-head step runs on one GPU only; --gpus {args.gpus} is not supported",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import workloads as W
    from paper_2402_00518_amd import binding as B
    from paper_2402_00518_amd.session import Session

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    B.lib()
    w = W.WORKLOADS[args.workload]
    log(f"workload {w.name}: N={w.n_tokens} h={w.hidden} V={w.vocab} I={w.intermediate} "
        f"exits={w.n_exits} {w.dtype}")
    t0 = time.time()
    batch = W.make_batch(w, args.seed)
    sess = Session.from_batch(batch)
    torch.cuda.synchronize()
    log(f"inputs generated and resident in HBM ({time.time() - t0:.1f} s)")

    for _ in range(args.warmup):
        sess.step()
    torch.cuda.synchronize()
    sess.check_device_error()
    log(f"warmup {args.warmup} steps done, loss {sess.loss_total.item():.5f}")

    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(args.steps):
        sess.step()
    stop.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / args.steps
    loss = sess.loss_total.item()
    log(f"timed {args.steps} steps: {ms:.4f} ms/step, loss {loss:.5f}")

    flops = step_flops(w)
    peak = PEAK_TFLOPS[w.dtype]
    tokens_per_s = w.n_tokens / (ms / 1e3)
    out = {
        "metric": METRIC,
        "value": tokens_per_s,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "kind": ["embedding", "norm", "mlp"][w.kind],
                   "n_tokens": w.n_tokens, "hidden": w.hidden, "vocab": w.vocab,
                   "intermediate": w.intermediate, "exits": w.n_exits,
                   "exit_weights": list(w.exit_weights)},
        "mfma_peak_frac": flops / (ms / 1e3) / (peak * 1e12),
        "step_tflops": flops / (ms / 1e3) / 1e12,
        "loss": loss,
    }

    if not args.no_kernel_pass:
        B.ee_profile_start()
        for _ in range(args.steps):
            sess.step()
        kt = B.ee_profile_stop()
        kernels = {k: {"launches": n, "avg_ms": t / n} for k, (n, t) in kt.items()}
        out["kernels"] = kernels
        dom = max(kernels, key=lambda k: kernels[k]["avg_ms"] * kernels[k]["launches"])
        f = kernel_flops(w, dom)
        avg_s = kernels[dom]["avg_ms"] / 1e3
        if f is not None:
            ach = f / avg_s / 1e12
            out["roofline"] = {"bound": "mfma", "kernel": dom, "achieved": ach, "peak": peak,
                               "unit": "TFLOP/s", "frac": ach / peak,
                               "traffic": measured_traffic(w.name, dom),
                               "flops_per_launch": f, "avg_ms": kernels[dom]["avg_ms"]}
            prof = profile_figure(w.name, dom)
            if prof is not None:
                # the same kernel in the committed rocprofv3 summary (another run)
                pa = f / (prof["avg_us"] / 1e6) / 1e12
                out["roofline"].update({"profile_avg_ms": prof["avg_us"] / 1e3, "profile_achieved": pa,
                                        "profile_frac": pa / peak, "profile_file": prof["file"]})
        log(f"dominant kernel {dom}: {kernels[dom]['avg_ms']:.4f} ms")
        side = {}
        for k, rec in kernels.items():
            nb = side_pass_bytes(w, k)
            if nb is None:
                continue
            gbps = nb / (rec["avg_ms"] / 1e3) / 1e9
            side[k] = {"avg_ms": rec["avg_ms"], "algorithmic_bytes": nb, "achieved_GBps": gbps,
                       "peak_GBps": PEAK_HBM_GBS, "frac": gbps / PEAK_HBM_GBS, "bound": "hbm",
                       "traffic": measured_traffic(w.name, TRAFFIC_LABEL.get(k, k))}
        out["hbm_passes"] = side

    if not args.no_update_leg:
        out["adam_update"] = adam_leg(sess, args.steps, args.warmup)
        a = out["adam_update"]
        log(f"adam update: {a['ms']:.4f} ms, {a['achieved_GBps']:.0f} GB/s ({100 * a['frac']:.1f}% of HBM peak)")

    if not args.no_update_leg:
        out["exit_decision"] = decode_leg(sess)
        for r, d in out["exit_decision"]["rows"].items():
            log(f"exit decision rows={r}: {d['us']:.1f} us per call, output-matrix kernel {d['logits_kernel_us']:.1f} us "
                f"({d['logits_kernel_GBps']:.0f} GB/s, {100 * d['frac']:.1f}% of HBM peak)")

    if args.copy_calibration_mib > 0:
        copy_calibration(args.copy_calibration_mib)

    if not args.no_cpu_baseline:
        log("cpu baseline: oracle on the batch ...")
        out["cpu_baseline"] = cpu_baseline(batch, args.cpu_sample_tokens)
        log(f"cpu baseline {out['cpu_baseline']['value']:.1f} tokens/s")

    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
