"""Benchmark: tokens/s of batched linear-chain CRF inference on one MI355X.

One timed step is one call of ts_chain_marginals over one batch: log Z and the edge
marginals (tree up-sweep, root, outside sweep, per-edge marginals), the quantity the
metric names.  The Viterbi call (max-plus tree, backpointers, backtrace) and the combined
call ts_chain_marginals_viterbi (the whole hot path: both trees, the Viterbi one on a side
stream) are timed too and reported in `breakdown`.  --step selects another call as the
timed step; --graph replays a captured HIP graph of it.  Inputs, outputs and workspaces are
resident in HBM before the timed region.  Prints one JSON line.

Default workload: the HMM-style batch (B=16, N=1024, C=256; potentials log_softmax_j(T) +
emissions, full lengths), the largest of the five seeded workloads.  --workload selects
another (paper: B=32 N=25 C=20, the paper's Table 1 linear-chain shape).
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
MFMA_BF16_PEAK = 2.5e15    # flop/s, dense bf16 matrix
# The tree's 128-wide full tiles (C a multiple of 128) multiply float32 operands as three bf16
# parts each, six bf16 products per float32 product: their float32-equivalent peak
MFMA_BF16X6_PEAK = MFMA_BF16_PEAK / 6
# fp64 vector: 78.6 TFLOP/s counts an FMA as two flops, i.e. 256 CUs x 4 SIMDs x 16 lanes x
# 2.4 GHz = 39.3e12 lane-instructions/s; a max-plus pair is two of them (add, max)
VALU_F64_OPS_PEAK = 39.3e12

PAPER_CONTEXT_TOKENS_PER_S = 390e3   # Table 1, K80, batch 32, N=25, C=20 (context only)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="hmm",
                    choices=["tiny", "paper", "mid", "hmm", "long"])
    ap.add_argument("--step", default="marginals", choices=["marginals", "viterbi", "both"],
                    help="the call one timed step makes (default: ts_chain_marginals, the "
                         "metric's log Z + marginals)")
    ap.add_argument("--only", action="store_true",
                    help="time the step only and print a short line (for profiler runs: no "
                         "other calls, no CPU baseline)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="bound on the oracle's CPU-baseline run (0 disables it)")
    ap.add_argument("--graph", action="store_true",
                    help="replay one captured HIP graph per step instead of calling the library")
    ap.add_argument("--sweep", choices=["depth", "labels", "large"], default=None,
                    help="instead of the step: log Z by the scan against the left-to-right "
                         "kernel over sequence lengths (depth: B=16, C=20), label counts "
                         "(labels: B=16, N=20) or long sequences of many labels (large: B=4, "
                         "C=128 and 256, N=512..8192); one JSON line per point")
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


def node_scan_level(E, D):
    """The level at which log Z's up-sweep stops for the recursion over that level's nodes
    (at most 128 labels on the tree), 0 for the tree to the root; the same cost model as the
    workspace plan (node_scan_level in paper_2002_00876_amd/csrc/api.cpp)."""
    level_us, step_us, scan_us, root_us = 12.0, 1.0, 5.0, 10.0
    best, level = D * level_us + root_us, 0
    for l in range(1, D):
        t = l * level_us + ((E + (1 << l) - 1) >> l) * step_us + scan_us
        if t < best:
            best, level = t, l
    return level


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
    depth-versus-work trade-off of the parallel scan (the paper's Fig. 4a and 4c shapes, and
    long sequences of 128 and 256 labels, where the tree does C times the serial work)."""
    import numpy as np
    import torch

    from paper_2002_00876_amd import binding

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    if kind == "depth":
        points = [(16, n, 20) for n in (26, 51, 101, 201, 301, 401, 501)]
    elif kind == "labels":
        points = [(16, 20, c) for c in (10, 20, 40, 60, 80, 100)]
    else:
        points = ([(4, n, c) for c in (128, 256) for n in (512, 1024, 2048, 4096, 8192)]
                  + [(16, 1024, 256)])
        reps = 3
    for B, N, C in points:
        if kind == "large":
            # drawn on the device (gigabytes of potentials; no oracle takes part)
            g = torch.Generator(device=dev)
            g.manual_seed(1000 + N + C)
            pot = torch.randn((B, N - 1, C, C), generator=g, device=dev, dtype=torch.float32)
        else:
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
        D = max(0, (N - 2).bit_length())                     # levels above the N - 1 leaves
        lscan = node_scan_level(N - 1, D) if 64 < C <= 128 and D >= 2 else 0
        path = ("single launch" if fused else "chunks" if C <= 64 else
                f"tree to level {lscan}, recursion over its nodes" if lscan else "multi-launch tree")
        tree_flop = 2 * B * max(N - 2, 0) * C ** 3           # tree products: 2 C^3 flop each
        serial_flop = 2 * B * (N - 1) * C ** 2              # left to right: 2 C^2 per step
        print(json.dumps({"sweep": kind, "B": B, "N": N, "C": C,
                          "tree_flop": tree_flop, "serial_flop": serial_flop,
                          "scan_ms": round(ms_scan, 5), "sequential_ms": round(ms_seq, 5),
                          "scan_path": path,
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


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline_streamed(pot, lens, seconds):
    """The oracle's log Z + marginals (float64 forward-backward of every sequence, then
    the marginals of every edge, formed range by range into one reusable buffer so the
    float64 tensor is never held whole), repeated until `seconds` have passed."""
    import numpy as np

    import oracle
    B, E, C, _ = pot.shape
    chunk = max(1, (1 << 22) // (C * C))
    buf = np.empty((chunk, C, C), np.float64)
    reps, t0 = 0, time.perf_counter()
    while True:
        msg = oracle.Messages(pot, lens)
        for b in range(B):
            Eb = int(lens[b]) - 1
            for e0 in range(0, Eb, chunk):
                msg.edge_marginals(b, e0, min(Eb, e0 + chunk), out=buf[:min(Eb, e0 + chunk) - e0])
        reps += 1
        el = time.perf_counter() - t0
        if el >= seconds:
            break
    return {"value": B * (E + 1) * reps / el, "unit": "tokens/s",
            "cores": oracle.max_threads(), "kind": "oracle",
            "cpu_model": cpu_model(),
            "sample": f"the full batch: oracle log Z + marginals (float64 forward-backward, "
                      f"OpenMP over sequences; marginals of every valid edge, OpenMP over "
                      f"edges), {reps} pass(es) in {el:.1f} s"}


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

    def both_call():
        # the whole hot path in one call: on the single-launch path one launch, where the
        # marginals and the Viterbi workgroups run side by side; on the multi-launch tree
        # the Viterbi sequence runs on a side stream beside the marginals sequence
        binding.marginals_viterbi(pot, lens, out=(logz, marg, path, score), ws=ws_mv)

    step = {"marginals": marg_call, "viterbi": vit_call, "both": both_call}[args.step]
    # warm up first: the first call of each entry point sets the kernels' LDS limits
    for _ in range(max(args.warmup, 1)):
        step()
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
    if args.only:
        print(json.dumps({"step": args.step, "workload": w.name, "steps": args.steps,
                          "ms_per_step": round(ms_step, 5)}), flush=True)
        return

    # per-call durations: each entry point issued n times back to back on the stream its
    # kernels run on, bracketed by two HIP events
    def per_call(fn, n):
        for _ in range(2):
            fn()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(n):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    n_calls = max(5, min(args.steps, 200))
    ms_marg = ms_step if args.step == "marginals" and not args.graph else per_call(marg_call, n_calls)
    ms_vit = per_call(vit_call, n_calls)
    ms_both = per_call(both_call, n_calls)

    alg = algorithmic(pot_h, lens_h)
    tokens = B * N
    value = tokens / (ms_step * 1e-3)

    # Roofline of the timed call.  On the single-launch path the marginals call is one
    # kernel (k_small_log); on the multi-launch tree it is a sequence of kernels whose bound
    # is the call's algorithmic work: read the valid edges and write all marginals (HBM),
    # and 2 C^3 flop per tree product on the matrix cores (MFMA: fp32, or for C a multiple
    # of 128 the six-product bf16 split at 2.5 PFLOP/s / 6).  The binding resource is the
    # one with the longer time at its peak.
    fused = binding.workspace_bytes(binding.OP_MARGINALS, B, N, C) == 0
    bf16x6 = not fused and C > 64 and C % 128 == 0
    cmp_peak = MFMA_BF16X6_PEAK if bf16x6 else MFMA_F32_PEAK

    def roofline(kind, sec):
        if kind == "marginals":
            t_mem, t_cmp = alg["marg_bytes"] / HBM_PEAK, alg["marg_flops"] / cmp_peak
            if t_mem >= t_cmp:
                a = alg["marg_bytes"] / sec / 1e9
                r = {"bound": "hbm", "achieved": round(a, 2), "peak": HBM_PEAK / 1e9,
                     "unit": "GB/s", "frac": float(f"{a / (HBM_PEAK / 1e9):.4g}")}
            else:
                a = alg["marg_flops"] / sec / 1e12
                r = {"bound": "mfma", "achieved": round(a, 3), "peak": round(cmp_peak / 1e12, 2),
                     "unit": "TFLOP/s", "frac": float(f"{a / (cmp_peak / 1e12):.4g}"),
                     "peak_note": ("bf16 dense 2500 TFLOP/s / 6: six bf16 products per float32 "
                                   "product (three-part split of each operand)" if bf16x6 else
                                   "fp32 dense MFMA")}
            r["algorithmic_bytes"] = alg["marg_bytes"]
            r["algorithmic_flops"] = alg["marg_flops"]
        else:
            t_mem, t_cmp = alg["vit_bytes"] / HBM_PEAK, alg["vit_ops"] / VALU_F64_OPS_PEAK
            if t_mem >= t_cmp:
                a = alg["vit_bytes"] / sec / 1e9
                r = {"bound": "hbm", "achieved": round(a, 2), "peak": HBM_PEAK / 1e9,
                     "unit": "GB/s", "frac": float(f"{a / (HBM_PEAK / 1e9):.4g}")}
            else:
                a = alg["vit_ops"] / sec / 1e12
                r = {"bound": "alu", "achieved": round(a, 3), "peak": VALU_F64_OPS_PEAK / 1e12,
                     "unit": "T fp64 add/max per s", "frac": float(f"{a / (VALU_F64_OPS_PEAK / 1e12):.4g}")}
            r["algorithmic_bytes"] = alg["vit_bytes"]
            r["algorithmic_fp64_ops"] = alg["vit_ops"]
        r["roofline_ms"] = round(max(t_mem, t_cmp) * 1e3, 6)
        return r

    roof = roofline("marginals", ms_marg * 1e-3)
    dom = "k_small_log" if fused else "ts_chain_marginals"
    roof["traffic"] = measured_traffic(dom, w.name)
    if fused:
        roof["kernel"] = dom
    elif C <= 64:
        roof["kernel"] = ("ts_chain_marginals (the call's kernel sequence: k_chunk_up, "
                          "k_chunk_scan, k_chunk_form)")
    else:
        roof["kernel"] = ("ts_chain_marginals (the call's kernel sequence: k_leaf_max, "
                          "k_up_log per level, k_root_log, k_down_log per level, k_form_*)")
    roof["kernel_ms"] = round(ms_marg, 5)
    roof_v = roofline("viterbi", ms_vit * 1e-3)

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
                   "step": {"marginals": "ts_chain_marginals (log Z and edge marginals)",
                            "viterbi": "ts_chain_viterbi (path and score)",
                            "both": "ts_chain_marginals_viterbi (log Z, marginals, Viterbi)"}[
                                args.step] + (", replayed as a HIP graph" if args.graph else ""),
                   "path": ("fused single launch per call" if fused else
                            "chunks: three launches per call" if C <= 64 else
                            "multi-launch tree")},
        "breakdown": {"marginals_ms": round(ms_marg, 5), "viterbi_ms": round(ms_vit, 5),
                      "marginals_viterbi_ms": round(ms_both, 5),
                      "marginals_tokens_per_s": round(tokens / (ms_marg * 1e-3), 1),
                      "viterbi_tokens_per_s": round(tokens / (ms_vit * 1e-3), 1),
                      "whole_path_tokens_per_s": round(tokens / (ms_both * 1e-3), 1),
                      "valid_tokens_per_s": round(float(lens_h.sum()) / (ms_step * 1e-3), 1),
                      "viterbi_roofline": roof_v},
        "dtype_note": "log semiring in fp32 precision (products on the bf16 matrix cores from "
                      "three-part bf16 splits of the fp32 operands for 128-wide tiles, fp32 MFMA "
                      "elsewhere; float64 row/column offsets); Viterbi max-plus in float64",
        "paper_context": {"tokens_per_s": PAPER_CONTEXT_TOKENS_PER_S,
                          "note": "Table 1, K80, B=32 N=25 C=20; not the same metric"},
        "roofline": roof,
    }
    if args.cpu_seconds > 0:
        out["cpu_baseline"] = cpu_baseline_streamed(pot_h, lens_h, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
