"""Benchmark: tokens/s of batched linear-chain CRF inference on one MI355X.

One step is one pass of the whole hot path over one batch: ts_chain_marginals (log Z and
edge marginals: tree up-sweep, root, outside sweep, per-edge marginals) and
ts_chain_viterbi (max-plus tree, backpointers, backtrace).  Both calls only read the
potentials, so the step is one call of ts_chain_marginals_viterbi, which on the
single-launch path runs both passes in one launch, side by side (--graph replays a captured
HIP graph of that call instead).  Inputs, outputs and workspaces are resident in HBM before
the timed region.  Prints one JSON line.

Default workload: the paper-shaped batch (B=32, N=25, C=20, N(0,1) potentials, lengths
uniform in [13, 25]).  --workload selects another of the five seeded workloads.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK = 8.0e12          # bytes/s
MFMA_F32_PEAK = 157.3e12   # flop/s, dense fp32 matrix
# fp64 vector: 78.6 TFLOP/s counts an FMA as two flops, i.e. 256 CUs x 4 SIMDs x 16 lanes x
# 2.4 GHz = 39.3e12 lane-instructions/s; a max-plus pair is two of them (add, max)
VALU_F64_OPS_PEAK = 39.3e12

PAPER_CONTEXT_TOKENS_PER_S = 390e3   # Table 1, K80, batch 32, N=25, C=20 (context only)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="paper",
                    choices=["tiny", "paper", "mid", "hmm", "long"])
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="bound on the oracle's CPU-baseline run (0 disables it)")
    ap.add_argument("--graph", action="store_true",
                    help="replay one captured HIP graph per step instead of calling the library")
    ap.add_argument("--sweep", choices=["depth", "labels"], default=None,
                    help="instead of the step: log Z by the scan against the left-to-right "
                         "kernel over sequence lengths (depth: B=16, C=20) or label counts "
                         "(labels: B=16, N=20); one JSON line per point")
    ap.add_argument("--ops", action="store_true",
                    help="instead of the step: time each entry point separately on the "
                         "workload (log Z by the scan and left to right, marginals, entropy, "
                         "log-density, sampling); one JSON line per entry point")
    ap.add_argument("--semi", choices=["semi", "semi_long"], default=None,
                    help="instead of the step: the semi-Markov CRF on a seeded workload "
                         "(semi: B=32 N=25 K=5 C=20, the paper's Table 1 shape; semi_long: "
                         "B=8 N=1024 K=8 C=32); one JSON line")
    ap.add_argument("--samples", type=int, default=64,
                    help="samples per sequence for the sampling entry point under --ops")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="only run a plain device copy of this size (traffic-counter scale)")
    return ap.parse_args()


def algorithmic(pot, lens):
    """Algorithmic HBM bytes and semiring work of one call of each entry point."""
    B, E, C, _ = pot.shape
    Eb = (lens.astype("int64") - 1)
    valid = int(Eb.sum())
    products = int((Eb - 1).clip(min=0).sum())          # tree products, C^3 pairs each
    marg_bytes = 4 * C * C * valid + 4 * C * C * B * E + 4 * B      # read valid, write all
    vit_bytes = 4 * C * C * valid + 4 * B * (E + 1) + 4 * B          # read valid, path+score
    step_bytes = marg_bytes + vit_bytes - 4 * C * C * valid         # one read of the input
    pairs = products * C ** 3
    return dict(marg_bytes=marg_bytes, vit_bytes=vit_bytes, step_bytes=step_bytes, pairs=pairs,
                marg_flops=2 * pairs, vit_ops=2 * pairs, valid_edges=valid)


def measured_traffic(kernel, workload):
    """HBM bytes per launch of `kernel` on `workload` from a committed rocprofv3 summary
    (FETCH_SIZE + WRITE_SIZE, copy-calibrated) in profiles/, or None when there is none or
    the kernel's source has changed since the counters were taken."""
    import glob
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.md"))):
        kv = {}
        for line in open(path):
            if " = " in line:
                k, v = line.strip().split(" = ", 1)
                kv[k] = v
        if kv.get("kernel") != kernel or kv.get("workload") != workload:
            continue
        src = os.path.join(ROOT, kv.get("source", ""))
        if not os.path.isfile(src):
            return None
        if code_hash(src) != kv.get("source_sha256"):
            return None
        return int(kv["traffic_bytes_per_launch"])
    return None


def code_hash(path):
    """sha256 of a source file's code: comments, blank lines and indentation removed, so
    that only a change to the code itself invalidates a stored measurement."""
    import hashlib
    import re
    lines = []
    for line in open(path):
        line = re.sub(r"//.*", "", line).strip()
        if line:
            lines.append(line)
    return hashlib.sha256("\n".join(lines).encode()).hexdigest()


def cpu_baseline(pot, lens, seconds):
    import oracle
    reps, t0 = 0, time.perf_counter()
    while True:
        oracle.marginals(pot, lens)
        oracle.viterbi(pot, lens)
        reps += 1
        el = time.perf_counter() - t0
        if el >= seconds:
            break
    B, E = pot.shape[0], pot.shape[1]
    return {"value": B * (E + 1) * reps / el, "unit": "tokens/s",
            "cores": min(oracle.max_threads(), B), "kind": "oracle",
            "sample": f"the full batch, oracle marginals + Viterbi repeated {reps}x "
                      f"({el:.1f} s, float64, OpenMP over sequences)"}


def calibrate_copy(mib):
    import torch
    n = mib * (1 << 20) // 4
    src = torch.randn(n, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n * 4, "copy_bytes_written": n * 4}))


def sweep(kind, reps=20):
    """Time ts_chain_logpartition (the scan) against ts_chain_logpartition_sequential (the
    left-to-right forward algorithm) on seeded N(0,1) potentials with full lengths: the
    depth-versus-work trade-off of the parallel scan (the paper's Fig. 4a and 4c shapes)."""
    import numpy as np
    import torch

    from paper_2002_00876_amd import binding

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    points = ([(16, n, 20) for n in (26, 51, 101, 201, 301, 401, 501)] if kind == "depth"
              else [(16, 20, c) for c in (10, 20, 40, 60, 80, 100)])
    for B, N, C in points:
        rng = np.random.default_rng(1000 + N + C)
        pot = torch.from_numpy(rng.standard_normal((B, N - 1, C, C)).astype(np.float32)).to(dev)
        ws = binding._workspace(binding.OP_LOGPARTITION, B, N, C, dev)[0]
        out = torch.empty(B, dtype=torch.float32, device=dev)

        def timed(fn):
            fn()
            torch.cuda.synchronize()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(reps):
                fn()
            e1.record(stream)
            torch.cuda.synchronize()
            return e0.elapsed_time(e1) / reps

        ms_scan = timed(lambda: binding.logpartition(pot, out=out, ws=ws))
        ms_seq = timed(lambda: binding.logpartition_sequential(pot, out=out))
        fused = binding.workspace_bytes(binding.OP_LOGPARTITION, B, N, C) == 0
        print(json.dumps({"sweep": kind, "B": B, "N": N, "C": C,
                          "scan_ms": round(ms_scan, 5), "sequential_ms": round(ms_seq, 5),
                          "scan_path": "single launch" if fused else "multi-launch tree",
                          "scan_tokens_per_s": round(B * N / (ms_scan * 1e-3), 1),
                          "sequential_tokens_per_s": round(B * N / (ms_seq * 1e-3), 1),
                          "scan_speedup": round(ms_seq / ms_scan, 3)}), flush=True)


def ops(w, samples, reps=50):
    """Time each entry point separately on one workload: the hot path's calls and the
    quantities read off their outputs (entropy, log-density of the Viterbi labels, samples).
    ms is the mean of back-to-back calls by HIP events on the library's stream; extra_ms is
    the time over the call the entry point builds on."""
    import numpy as np
    import torch

    from paper_2002_00876_amd import binding, workloads

    pot_h, lens_h = workloads.generate(w)
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    pot = torch.from_numpy(pot_h).to(dev)
    lens = torch.from_numpy(lens_h).to(dev)
    B, E, C, _ = pot.shape
    N = E + 1
    path, _ = binding.viterbi(pot, lens)
    labels = torch.where(path >= 0, path, torch.zeros_like(path)).contiguous()
    u = torch.from_numpy(np.random.default_rng(7).random((samples, B, N), dtype=np.float32))
    u = u.to(dev)
    wss = {op: binding._workspace(op, B, N, C, dev)[0] for op in range(7)}
    logz = torch.empty(B, dtype=torch.float32, device=dev)
    marg = torch.empty_like(pot)
    h = torch.empty(B, dtype=torch.float32, device=dev)
    lp = torch.empty(B, dtype=torch.float32, device=dev)
    paths = torch.empty((samples, B, N), dtype=torch.int32, device=dev)
    calls = {
        "logpartition": (lambda: binding.logpartition(pot, lens, out=logz,
                                                      ws=wss[binding.OP_LOGPARTITION]), None),
        "logpartition_sequential": (lambda: binding.logpartition_sequential(pot, lens, out=logz),
                                    None),
        "marginals": (lambda: binding.marginals(pot, lens, out=(logz, marg),
                                                ws=wss[binding.OP_MARGINALS]), None),
        "entropy": (lambda: binding.entropy(pot, lens, out=h, ws=wss[binding.OP_ENTROPY]),
                    "marginals"),
        "log_density": (lambda: binding.log_density(pot, labels, lens, out=lp,
                                                    ws=wss[binding.OP_LOG_DENSITY]),
                        "logpartition"),
        "sample": (lambda: binding.sample(pot, u, lens, out=paths, ws=wss[binding.OP_SAMPLE]),
                   "marginals"),
    }
    ms = {}
    for name, (fn, base) in calls.items():
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        ms[name] = e0.elapsed_time(e1) / reps
        tokens = B * N * (samples if name == "sample" else 1)
        line = {"op": name, "workload": f"{w.name}: B={B} N={N} C={C}", "ms": round(ms[name], 5),
                "tokens_per_s": round(tokens / (ms[name] * 1e-3), 1)}
        if name == "sample":
            line["samples_per_sequence"] = samples
        if base is not None:
            line["extra_ms"] = round(ms[name] - ms[base], 5)
        print(json.dumps(line), flush=True)


def semi(name, steps, warmup):
    """Semi-Markov CRF: log Z + segment marginals and the best segmentation per step (the
    chain scan over K*C expanded states), HIP-event timed like the chain step."""
    import torch

    from paper_2002_00876_amd import binding, workloads

    sp_h, lens_h = workloads.generate_semi(name)
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    sp = torch.from_numpy(sp_h).to(dev)
    lens = torch.from_numpy(lens_h).to(dev)
    B, E, K, C, _ = sp.shape
    N = E + 1
    logz = torch.empty(B, dtype=torch.float32, device=dev)
    marg = torch.empty_like(sp)
    path = torch.empty((B, N), dtype=torch.int32, device=dev)
    seglen = torch.empty((B, N - 1), dtype=torch.int32, device=dev)
    score = torch.empty(B, dtype=torch.float32, device=dev)
    ws_m = binding._semi_workspace(binding.OP_MARGINALS, B, N, K, C, dev)[0]
    ws_v = binding._semi_workspace(binding.OP_VITERBI, B, N, K, C, dev)[0]

    def marg_call():
        binding.semi_marginals(sp, lens, out=(logz, marg), ws=ws_m)

    def vit_call():
        binding.semi_viterbi(sp, lens, out=(path, seglen, score), ws=ws_v)

    def step():
        marg_call()
        vit_call()

    def timed(fn, n):
        for _ in range(max(warmup, 1)):
            fn()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(n):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    ms_step = timed(step, steps)
    ms_marg = timed(marg_call, steps)
    ms_vit = timed(vit_call, steps)
    fused = binding.workspace_bytes(binding.OP_MARGINALS, B, N, K * C) == 0
    print(json.dumps({
        "metric": "semi-Markov tokens/sec (log Z + segment marginals + best segmentation)",
        "value": round(B * N / (ms_step * 1e-3), 1), "unit": "tokens/s",
        "ms_per_step": round(ms_step, 5), "steps": steps, "warmup": warmup,
        "config": {"workload": f"{name}: B={B} N={N} K={K} C={C}", "expanded_labels": K * C,
                   "chain_path": "fused single launch" if fused else "multi-launch tree"},
        "breakdown": {"marginals_ms": round(ms_marg, 5), "viterbi_ms": round(ms_vit, 5)},
        "paper_context": {"tokens_per_s": 87e3,
                          "note": "Table 1 semi-Markov, K80, B=32 N=25 C=20 K=5; log Z only"},
    }), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2002_00876_amd import binding, workloads

    if args.calibrate_copy_mib:
        calibrate_copy(args.calibrate_copy_mib)
        return
    if args.sweep:
        binding.lib()
        sweep(args.sweep)
        return
    binding.lib()   # fail loudly if the HIP library is missing
    if args.semi:
        semi(args.semi, args.steps, args.warmup)
        return
    w = workloads.WORKLOADS[args.workload]
    if args.ops:
        ops(w, args.samples)
        return
    pot_h, lens_h = workloads.generate(w)
    dev = torch.device("cuda:0")
    pot = torch.from_numpy(pot_h).to(dev)
    lens = torch.from_numpy(lens_h).to(dev)
    B, E, C, _ = pot.shape
    N = E + 1
    logz = torch.empty(B, dtype=torch.float32, device=dev)
    marg = torch.empty_like(pot)
    path = torch.empty((B, N), dtype=torch.int32, device=dev)
    score = torch.empty(B, dtype=torch.float32, device=dev)
    ws_m = binding._workspace(binding.OP_MARGINALS, B, N, C, dev)[0]
    ws_v = binding._workspace(binding.OP_VITERBI, B, N, C, dev)[0]
    ws_mv = binding._workspace(binding.OP_MARGINALS_VITERBI, B, N, C, dev)[0]
    stream = torch.cuda.current_stream(dev)

    def marg_call():
        binding.marginals(pot, lens, out=(logz, marg), ws=ws_m)

    def vit_call():
        binding.viterbi(pot, lens, out=(path, score), ws=ws_v)

    def step():
        # the whole path in one call: one launch on the single-launch path, where the
        # marginals and the Viterbi workgroups run side by side
        binding.marginals_viterbi(pot, lens, out=(logz, marg, path, score), ws=ws_mv)

    # warm up first: the first call of each entry point sets the kernels' LDS limits
    for _ in range(max(args.warmup, 1)):
        step()
    marg_call()
    vit_call()
    torch.cuda.synchronize()

    run = step
    if args.graph:
        graph = torch.cuda.CUDAGraph()
        cap = torch.cuda.Stream(device=dev)
        cap.wait_stream(stream)
        with torch.cuda.stream(cap):
            with torch.cuda.graph(graph, stream=cap):
                step()
        stream.wait_stream(cap)
        torch.cuda.synchronize()
        run = graph.replay
        for _ in range(max(args.warmup, 1)):
            run()
        torch.cuda.synchronize()

    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record(stream)
    for _ in range(args.steps):
        run()
    t_end.record(stream)
    torch.cuda.synchronize()
    total_ms = t_start.elapsed_time(t_end)
    ms_step = total_ms / args.steps

    # per-call durations: each entry point issued n times back to back on the stream its
    # kernels run on, bracketed by two HIP events; on the single-launch path one call is one
    # kernel, so this is that kernel's average duration (launch gaps included)
    def per_call(fn, n):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(n):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    n_calls = max(10, min(args.steps, 200))
    ms_marg = per_call(marg_call, n_calls)
    ms_vit = per_call(vit_call, n_calls)

    alg = algorithmic(pot_h, lens_h)
    tokens = B * N
    value = tokens / (ms_step * 1e-3)

    # the roofline of the step's dominant kernel.  On the single-launch path the step is one
    # kernel (k_small_both), timed back to back; on the multi-launch tree the whole call is
    # timed and the bound is the sum of its kernels' bounds.
    fused = binding.workspace_bytes(binding.OP_MARGINALS_VITERBI, B, N, C) == 0
    ms_call = per_call(step, n_calls)
    dom = "k_small_both" if fused else "ts_chain_marginals_viterbi (multi-launch)"
    t_mem = alg["step_bytes"] / HBM_PEAK
    t_mfma = alg["marg_flops"] / MFMA_F32_PEAK
    t_f64 = alg["vit_ops"] / VALU_F64_OPS_PEAK
    sec = ms_call * 1e-3
    # the binding resource is the one with the longest time at its peak: on the single-launch
    # path the log-semiring and the max-plus workgroups run side by side on different CUs
    if t_mem >= max(t_mfma, t_f64):
        achieved = alg["step_bytes"] / sec / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK / 1e9,
                "unit": "GB/s", "frac": round(achieved / (HBM_PEAK / 1e9), 5)}
    elif t_mfma >= t_f64:
        achieved = alg["marg_flops"] / sec / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 3), "peak": MFMA_F32_PEAK / 1e12,
                "unit": "TFLOP/s", "frac": round(achieved / (MFMA_F32_PEAK / 1e12), 5)}
    else:
        achieved = alg["vit_ops"] / sec / 1e12
        roof = {"bound": "alu", "achieved": round(achieved, 3), "peak": VALU_F64_OPS_PEAK / 1e12,
                "unit": "TFLOP/s", "frac": round(achieved / (VALU_F64_OPS_PEAK / 1e12), 5)}
    roof["traffic"] = measured_traffic(dom, w.name) if fused else None
    roof["kernel"] = dom
    roof["kernel_ms"] = round(ms_call, 5)
    roof["algorithmic_bytes"] = alg["step_bytes"]
    roof["roofline_ms"] = round(max(t_mem, t_mfma, t_f64) * 1e3, 6)

    out = {
        "metric": "tokens/sec for linear-chain logZ+marginals (B,N,C); % of HBM/compute roofline",
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{w.name}: B={B} N={N} C={C}", "B": B, "N": N, "C": C,
                   "lengths": "uniform" if w.len_range else "fixed",
                   "step": "ts_chain_marginals_viterbi (log Z, marginals, Viterbi path and score)"
                           + (", replayed as a HIP graph" if args.graph else ""),
                   "path": "fused single launch per call" if fused else "multi-launch tree"},
        "breakdown": {"marginals_ms": round(ms_marg, 5), "viterbi_ms": round(ms_vit, 5),
                      "separate_calls_ms": round(ms_marg + ms_vit, 5),
                      "marginals_tokens_per_s": round(tokens / (ms_marg * 1e-3), 1),
                      "valid_tokens_per_s": round(float(lens_h.sum()) / (ms_step * 1e-3), 1)},
        "dtype_note": "log semiring in fp32 (fp32 MFMA, float64 row/column offsets); "
                      "Viterbi max-plus in float64",
        "paper_context": {"tokens_per_s": PAPER_CONTEXT_TOKENS_PER_S,
                          "note": "Table 1, K80, B=32 N=25 C=20; not the same metric"},
        "roofline": roof,
    }
    if args.cpu_seconds > 0:
        out["cpu_baseline"] = cpu_baseline(pot_h, lens_h, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
