#!/usr/bin/env python3
"""Benchmark of the BSR product Y = X W^T + b on one MI355X.

Default workload: a BERT-base attention layer -- four 768x768 projections (Q, K, V, O), each
pruned to 32x1 blocks at 10% block density, applied to one batch of 1 x 128 tokens.  One step
computes the four products, issued as one bsr_spmm_batched call (one kernel launch; workloads
with more products use one call per 8).  Inputs are seeded synthetic tensors
(paper_2106_08846_amd/workloads.py), pruned on the GPU by bsr_prune_from_dense, and resident in
device memory when timing starts.

The step is timed as --steps direct issues of its prepared calls (arguments marshalled once,
one foreign call per launch); --graph times HIP graph replays of the same calls instead, and
both figures are reported.
Prints one JSON line: effective GFLOP/s (2 * nnz * tokens per call, summed over the step), the
roofline position of the product kernel (average launch duration from HIP events recorded on
the launch stream), the same-shape dense fp32/bf16 GEMM, and the CPU oracle on this host.
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import platform
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
FP32_PEAK_TFLOPS = 157.3       # MI355X fp32 matrix (dense)
BF16_PEAK_TFLOPS = 2516.6      # MI355X bf16 matrix (dense)
METRIC = "BSR SpMM effective GFLOP/s (2*nnz*tokens)"
KERNEL_SOURCES = "paper_2106_08846_amd/csrc"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_spmm.md")


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="bert_base_attn",
                    help="bert_base_attn | single_768 | sweep:RxC | "
                         "fused_qkv:RxC:density[:bf16] | bert_large:RxC | "
                         "ffn:RxC[:density[:tokens]][:bf16] | "
                         "attn_block[:RxC[:density[:batch[:seq]]]]; RxC@R2xC2 prunes with "
                         "R x C blocks and multiplies the matrix re-blocked to R2 x C2")
    ap.add_argument("--slices", type=int, default=0,
                    help="block-row slices per token tile (0: the library's choice)")
    ap.add_argument("--graph", action="store_true",
                    help="time the step as HIP graph replays instead of direct calls")
    ap.add_argument("--no-graph", action="store_true",
                    help="skip the graph-replay figure (e.g. under counter collection)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="approximate CPU time spent timing the oracle baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB --steps times (the reference "
                         "kernel for scaling HBM byte counters) and exit")
    return ap.parse_args()


def build_workload(spec: str):
    from paper_2106_08846_amd import workloads as G
    parts = spec.split(":")
    kind = parts[0]
    if kind == "bert_base_attn":
        return G.bert_base_attention()
    if kind == "single_768":
        return G.single_768()
    # A block field "RxC@R2xC2" prunes with R x C blocks and runs the product on the same
    # matrix re-blocked to R2 x C2 (bsr_reblock).
    block = parts[1].split("@") if len(parts) > 1 else ["32x1"]
    R, C = (int(v) for v in block[0].split("x"))
    fine = tuple(int(v) for v in block[1].split("x")) if len(block) > 1 else None
    bf16 = parts[-1] == "bf16"
    if bf16 and kind in ("sweep", "bert_large"):
        raise SystemExit(f"{spec}: the {kind} workload is fp32 only")
    if kind == "sweep":
        wl = G.block_sweep(R, C)
    elif kind == "fused_qkv":
        wl = G.fused_qkv(R, C, float(parts[2]), bf16=bf16)
    elif kind == "bert_large":
        wl = G.bert_large_zipf(R, C)
    elif kind == "ffn":
        density = float(parts[2]) if len(parts) > 2 and parts[2] != "bf16" else 0.1
        tokens = int(parts[3]) if len(parts) > 3 and parts[3] != "bf16" else 128
        wl = G.bert_base_ffn(R, C, density, tokens=tokens, bf16=bf16)
    else:
        raise SystemExit(f"unknown workload {spec}")
    if fine is not None:
        wl.notes["reblock"] = fine
        wl.name += f"_as_{fine[0]}x{fine[1]}"
    return wl


def kernel_source_hash() -> str:
    """sha256 over libbsr's kernel and launch sources (counters go stale when it changes)."""
    h = hashlib.sha256()
    for path in sorted(glob.glob(os.path.join(ROOT, KERNEL_SOURCES, "*"))):
        if os.path.isfile(path) and path.endswith((".hip", ".h", ".cpp")):
            h.update(os.path.basename(path).encode())
            with open(path, "rb") as f:
                h.update(f.read())
    return h.hexdigest()


def measured_traffic(workload: str) -> dict | None:
    """HBM bytes per launch from the committed counter summary, if it is for this source."""
    try:
        with open(TRAFFIC_FILE) as f:
            text = f.read()
    except OSError:
        return None
    m = re.search(r"```json\n(.*?)\n```", text, re.S)
    if not m:
        return None
    table = json.loads(m.group(1))
    if table.get("kernel_source_sha256") != kernel_source_hash():
        return None
    return table.get("workloads", {}).get(workload)


def calibrate_copy(args) -> int:
    import torch
    n = args.calibrate_copy * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(args.steps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"calibrate_copy_bytes_read": 4 * n, "calibrate_copy_bytes_written": 4 * n,
                      "launches": args.steps}), flush=True)
    return 0


def main() -> int:
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the library has no "
              "multi-GPU path, so run it with --gpus 1.", file=sys.stderr, flush=True)
        return 2

    import torch
    from paper_2106_08846_amd import bsr as B

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    if args.calibrate_copy:
        return calibrate_copy(args)
    if args.workload.startswith("attn_block"):
        return bench_attention_block(args)
    dev = torch.device("cuda:0")
    wl = build_workload(args.workload)
    bf16 = wl.bf16
    print(f"# workload {wl.name}: {len(wl.projections)} projections", file=sys.stderr,
          flush=True)

    # Inputs to the device; prune every weight on the GPU.
    X32 = [torch.from_numpy(x).to(dev) for x in wl.X]
    Xs = [B.bsr_cast_f32_bf16(x) for x in X32] if bf16 else X32
    calls = []
    for p in wl.projections:
        N, K = p.W.shape
        k = p.k if p.k is not None else B.bsr_prune_count(N, K, p.R, p.C, p.density)
        Wd = torch.from_numpy(p.W).to(dev)
        M = B.bsr_prune_from_dense(Wd, p.R, p.C, k=k)
        if bf16:
            M = M.to_bf16()
        if "reblock" in wl.notes:
            M = B.bsr_reblock(M, *wl.notes["reblock"])
        bias = torch.from_numpy(p.bias).to(dev)
        T = wl.X[p.x_index].shape[0]
        Y = torch.empty((T, N), dtype=torch.float32, device=dev)
        calls.append(dict(X=Xs[p.x_index], M=M, bias=bias, Y=Y, Wd=Wd, T=T, N=N, K=K, R=M.R,
                          C=M.C, k=M.nnzb))
    # The step's products go to bsr_spmm_batched in groups of up to 8 (one kernel launch each:
    # Q, K, V and O of a layer share one launch).
    groups = [calls[i:i + 8] for i in range(0, len(calls), 8)]
    runs = [B.SpmmBatchCall([(c["X"], c["M"], c["bias"], c["Y"]) for c in grp],
                            slices=args.slices or None) for grp in groups]
    torch.cuda.synchronize()

    def step():
        for run in runs:
            run()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def time_steps(fn, n):
        torch.cuda.synchronize()
        start.record()
        for _ in range(n):
            fn()
        end.record()
        torch.cuda.synchronize()
        return start.elapsed_time(end) / n

    eager_ms = time_steps(step, args.steps)
    graph_ms = None
    if args.graph or not args.no_graph:
        g = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            step()
        for _ in range(args.warmup):
            g.replay()
        graph_ms = time_steps(g.replay, args.steps)
    ms_per_step = graph_ms if args.graph else eager_ms

    flops_step = sum(2.0 * c["k"] * c["R"] * c["C"] * c["T"] for c in calls)
    value = flops_step / (ms_per_step * 1e-3) / 1e9

    # Roofline of the product kernel: average device duration of one launch.  Each launch gets a
    # pair of HIP events that the library records at the kernel's own start and end on the
    # launch stream (hipExtLaunchKernel), so host gaps and dispatch overhead are excluded.
    sx = 2 if bf16 else 4
    n_ev = max(1, min(args.steps, 400 // len(runs) + 1))
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(len(runs) * n_ev)]
    for a, b in ev:
        a.record()
        b.record()
    torch.cuda.synchronize()
    i = 0
    for _ in range(n_ev):
        for run in runs:
            run.timed(*ev[i])
            i += 1
    torch.cuda.synchronize()
    launch_ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))

    def launch_bytes(c):
        nb_rows = c["N"] // c["R"]
        return (c["T"] * c["K"] * sx + c["k"] * c["R"] * c["C"] * sx + 4 * c["k"]
                + 4 * (nb_rows + 1) + 4 * c["N"] + 4 * c["T"] * c["N"])

    bytes_launch = sum(launch_bytes(c) for c in calls) / len(runs)
    flops_launch = flops_step / len(runs)
    peak_flops = (BF16_PEAK_TFLOPS if bf16 else FP32_PEAK_TFLOPS) * 1e12
    ai = flops_launch / bytes_launch
    gbs = bytes_launch / (launch_ms * 1e-3) / 1e9
    tfs = flops_launch / (launch_ms * 1e-3) / 1e12
    if ai > peak_flops / (HBM_PEAK_GBS * 1e9):
        roof = {"bound": "mfma", "achieved": tfs, "peak": peak_flops / 1e12,
                "unit": "TFLOP/s", "frac": tfs / (peak_flops / 1e12)}
    else:
        roof = {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": gbs / HBM_PEAK_GBS}
    tr = measured_traffic(wl.name)
    roof.update({"traffic": tr["bytes_per_launch"] if tr else None,
                 "kernel": " + ".join(dict.fromkeys(tiled_kernel_name(c) for c in calls)),
                 "launch_us": launch_ms * 1e3,
                 "algorithmic_bytes_per_launch": bytes_launch,
                 "flops_per_launch": flops_launch, "arithmetic_intensity": ai,
                 "achieved_gbs": gbs, "achieved_tflops": tfs})

    out = {
        "metric": METRIC, "value": value, "unit": "GFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if bf16 else "f32", "data": "synthetic",
        "config": {"workload": wl.name, "products_per_step": len(calls),
                   "launches_per_step": len(runs),
                   "tokens": calls[0]["T"], "N": calls[0]["N"], "K": calls[0]["K"],
                   "block": f"{calls[0]['R']}x{calls[0]['C']}",
                   "density": wl.projections[0].density,
                   "nnz_per_call": [c["k"] * c["R"] * c["C"] for c in calls][:8],
                   "timing": "hip_graph_replay" if args.graph else "direct_calls",
                   "slices": args.slices or "auto"},
        "eager_ms_per_step": eager_ms,
        "graph_ms_per_step": graph_ms,
        "roofline": roof,
    }

    if not args.no_dense:
        Wds = [c["Wd"].to(torch.bfloat16) if bf16 else c["Wd"] for c in calls]
        Xd = [c["X"] for c in calls]

        def dense_step():
            for c, W, X in zip(calls, Wds, Xd):
                if bf16:
                    c["Y"].copy_(torch.matmul(X, W.t()).float() + c["bias"])
                else:
                    torch.addmm(c["bias"], X, W.t(), out=c["Y"])

        for _ in range(args.warmup):
            dense_step()
        out["dense_gemm_ms_per_step"] = time_steps(dense_step, args.steps)

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, calls, args.cpu_seconds)

    print(json.dumps(out), flush=True)
    return 0


def bench_attention_block(args) -> int:
    """The BERT-base attention block on pruned weights: Q/K/V BSR products (one launch),
    scaled dot-product attention (bsr_attention), the O BSR product; beside it the same block
    with dense hipBLASLt GEMMs on the unpruned weights and the same attention kernel.

    --workload attn_block[:RxC[:density[:batch[:seq]]]], default 32x1, 0.1, 1 x 128 tokens."""
    import torch
    from paper_2106_08846_amd import bsr as B
    from paper_2106_08846_amd import workloads as G

    parts = args.workload.split(":")
    R, C = (int(v) for v in parts[1].split("x")) if len(parts) > 1 else (32, 1)
    density = float(parts[2]) if len(parts) > 2 else 0.1
    batch = int(parts[3]) if len(parts) > 3 else 1
    seq = int(parts[4]) if len(parts) > 4 else 128
    heads = 12
    dev = torch.device("cuda:0")
    wl = G.bert_base_attention(R, C, density, tokens=batch * seq)
    X = torch.from_numpy(wl.X[0]).to(dev)
    mats, biases, dense = [], [], []
    for p in wl.projections:
        Wd = torch.from_numpy(p.W).to(dev)
        mats.append(B.bsr_prune_from_dense(Wd, R, C, k=B.bsr_prune_count(768, 768, R, C, density)))
        biases.append(torch.from_numpy(p.bias).to(dev))
        dense.append(Wd)
    call = B.AttentionBlockCall(X, mats[0], biases[0], mats[1], biases[1], mats[2], biases[2],
                                mats[3], biases[3], batch, seq, heads)
    T = batch * seq
    Wqkv = torch.cat(dense[:3], 0).contiguous()
    bqkv = torch.cat(biases[:3], 0).contiguous()
    qkv = torch.empty((T, 3 * 768), device=dev)
    ctx = torch.empty((T, 768), device=dev)
    Yd = torch.empty((T, 768), device=dev)

    def dense_block():
        torch.addmm(bqkv, X, Wqkv.t(), out=qkv)
        B.bsr_attention(qkv[:, :768], qkv[:, 768:1536], qkv[:, 1536:], batch, seq, heads, O=ctx)
        torch.addmm(biases[3], ctx, dense[3].t(), out=Yd)

    # Time per block: `n` blocks issued back to back (prepared calls, one foreign call per
    # kernel), between two events on the current stream; the launch gaps are included.
    def timed(fn, n):
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(n):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / n * 1e3

    sparse_us = timed(call, args.steps)
    dense_us = timed(dense_block, args.steps)
    qkv_us = timed(call.qkv, args.steps)
    attn_us = timed(call.attention, args.steps)
    out_us = timed(call.out, args.steps)
    flops = sum(2.0 * m.nnzb * m.R * m.C * T for m in mats) + 4.0 * batch * heads * seq * seq * 64
    out = {
        "metric": "BERT attention block latency (BSR Q/K/V/O products + attention)",
        "value": sparse_us, "unit": "us", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": sparse_us / 1e3, "higher_is_better": False,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"attn_block_bert_base_{R}x{C}_d{int(round(density * 100))}"
                               f"_b{batch}_s{seq}", "tokens": T, "heads": heads,
                   "block": f"{R}x{C}", "density": density},
        "dense_block_us": dense_us, "sparse_over_dense": sparse_us / dense_us,
        "breakdown_us": {"qkv_products": qkv_us, "attention": attn_us, "o_product": out_us},
        "effective_gflops": flops / (sparse_us * 1e-6) / 1e9,
    }
    print(json.dumps(out), flush=True)
    return 0


TILED_SHAPES = ((32, 1), (16, 1), (32, 32), (16, 16))
VALU_SHAPES = ((1, 1), (1, 2), (1, 4), (1, 8), (1, 16), (1, 32), (2, 1), (4, 1), (8, 1), (2, 2),
               (4, 4), (8, 8))


def tiled_kernel_name(c) -> str:
    """The kernel libbsr's automatic choice launches for this product: the matrix-core tiled
    kernel, else the vector-ALU tile kernel, each in its column-chunked form when the 32-token
    X tile does not fit in LDS, else the generic kernel.  (An estimate for the label: the
    library's plan decides, and the kernel trace shows what ran.)"""
    bf = c["M"].dtype == 1
    shape = (c["R"], c["C"])
    flag = "true" if bf else "false"
    xb = 2 if bf and shape != (16, 1) else 4
    fits = 32 * (c["K"] + 8) * xb + 4 * c["N"] + 4 * (c["N"] // c["R"] + 8) <= 160 * 1024
    if shape in TILED_SHAPES:
        # 16x16 rows with at least 8 stored blocks on average run four-block units.
        w = 4 if shape == (16, 16) and c["k"] >= 8 * (c["N"] // 16) else 1
        if fits:
            return f"spmm_tiled_kernel<{c['R']}, {c['C']}, 16, {flag}, {w}> via bsr_spmm_batched"
        return f"spmm_kchunk_kernel<{c['R']}, {c['C']}, {flag}, {w}> via bsr_spmm_batched"
    if shape in VALU_SHAPES and not (bf and shape == (1, 1)):
        kern = "spmm_vtile_kernel" if fits else "spmm_vtile_chunk_kernel"
        return f"{kern}<{c['R']}, {c['C']}, {flag}> via bsr_spmm_batched"
    return "spmm_generic_kernel via bsr_spmm_batched"


def cpu_baseline(wl, calls, seconds: float) -> dict:
    """The C oracle (fp64 naive BSR loop, OpenMP over tokens) on this host's cores.

    The sample is the whole step, repeated until about `seconds` of wall time have passed; the
    rate is in GFLOP/s of the same metric (2 * nnz * tokens per call).
    """
    import torch
    from oracle import bsr_oracle as O
    from oracle import cpu_oracle
    cores = len(os.sched_getaffinity(0))
    cpu_oracle.set_num_threads(cores)
    host = []
    for c, p in zip(calls, wl.projections):
        ip = c["M"].indptr.cpu().numpy()
        ix = c["M"].indices.cpu().numpy()[:c["k"]]
        d = c["M"].data[:c["k"]]
        if d.dtype != torch.float32:
            dt = O.bf16_to_f32(d.contiguous().view(torch.int16).cpu().numpy().view(np.uint16))
        else:
            dt = d.cpu().numpy()
        X = wl.X[p.x_index]
        if wl.bf16:
            X = O.bf16_roundtrip(X)
        host.append((X, ip, ix, dt.reshape(c["k"], c["R"], c["C"]), c["N"], p.bias, c))
    # Run whole steps until the time budget is spent (at least one step).
    step_tokens = sum(h[0].shape[0] for h in host)
    flops = 0.0
    reps = 0
    t0 = time.perf_counter()
    while True:
        for X, ip, ix, dt, N, b, c in host:
            cpu_oracle.spmm(X, ip, ix, dt, N, b)
            flops += 2.0 * c["k"] * c["R"] * c["C"] * X.shape[0]
        reps += 1
        if time.perf_counter() - t0 >= seconds:
            break
    sample = (f"{reps} x the full step ({len(host)} calls, {step_tokens} token-rows in all)")
    el = time.perf_counter() - t0
    return {"value": flops / el / 1e9, "unit": "GFLOP/s", "cores": cpu_oracle.num_threads(),
            "kind": "oracle", "sample": sample, "seconds": el,
            "cpu": cpu_model()}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.machine()


if __name__ == "__main__":
    sys.exit(main())
