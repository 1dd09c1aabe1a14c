#!/usr/bin/env python3
"""Benchmark of the BSR product Y = X W^T + b on one MI355X.

Default workload (the headline): BERT-large attention -- 24 layers x four 1024x1024 projections
(Q, K, V, O), each pruned to linear 32x1 blocks at 10% block density with Zipf(1.2)-skewed
block-rows, applied to 16 x 384 = 6144 tokens per layer.  One step computes all 96 products,
issued as 12 bsr_spmm_batched calls of 8 products (one kernel launch each).  A step walks about
3.4 GB of inputs and outputs, more than the 256 MB last-level cache holds, so every step runs
cold.  Inputs are seeded synthetic tensors (paper_2106_08846_amd/workloads.py), pruned on the GPU
by bsr_prune_from_dense, and resident in device memory when timing starts.

Timing: --warmup untimed steps, then exactly --steps steps between two synchronisations, with an
event between consecutive steps, so that the JSON line carries the mean step time (the value)
and the median, p10 and p90 of the per-step times (at least 50 samples; more steps are sampled
after the timed region when --steps is smaller).  The roofline position divides the
algorithmic bytes or flops of one launch by the timed region's time per launch (the step time
over the launches of a step, launch gaps included, so an upper bound of the kernel's own time);
the durations that HIP events recorded at each product kernel's own start and end
(hipExtLaunchKernel) are reported beside it.

Beside the headline, unless --no-rows, the same line carries the block-shape rows of the other
configurations, each timed per launch with those kernel events and reported as median, p10, p90:
  * the BERT-large 32x32 stack (fp32 matrix cores), cold by construction like the headline;
  * the fused QKV weight 2304x768 at 4096 tokens, 32x1 and 16x16 blocks at 5-40% density, fp32
    and bf16, cold: 8 rotating copies of (X, BSR, bias, Y), 400 MB or more in all;
  * the 768x768 block-shape sweep at 128 tokens (nine shapes, the GPU analog of the paper's
    Table 1) and the BERT-base Q/K/V/O step, with the same-shape dense GEMM beside each.
The CPU oracle (plain C, fp64) is timed on this host's cores on a bounded sample of the headline
workload, and one-threaded on the 128-token workloads.
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

ARITH_SPLIT = 2      # bsr_arith: fp32 data split into three bf16 pieces
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
FP32_PEAK_TFLOPS = 157.3       # MI355X fp32 matrix (dense)
BF16_PEAK_TFLOPS = 2516.6      # MI355X bf16 matrix (dense)
METRIC = "BSR SpMM effective GFLOP/s (2*nnz*tokens)"
KERNEL_SOURCES = "paper_2106_08846_amd/csrc"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_spmm.md")
MIN_SAMPLES = 50
ROTATE_SETS = 8


def parse(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="bert_large:32x1",
                    help="bert_large:RxC | fused_qkv:RxC:density[:bf16] | sweep:RxC | "
                         "bert_base_attn | single_768 | ffn:RxC[:density[:tokens]][:bf16] | "
                         "attn_block[:RxC[:density[:batch[:seq]]]]; RxC@R2xC2 prunes with "
                         "R x C blocks and multiplies the matrix re-blocked to R2 x C2")
    ap.add_argument("--slices", type=int, default=0,
                    help="block-row slices per token tile (0: the library's choice)")
    ap.add_argument("--rotate", type=int, default=0,
                    help="copies of every input and output to rotate through (0: 1 for "
                         "workloads that exceed the last-level cache by themselves, else 8)")
    ap.add_argument("--no-plan", action="store_true",
                    help="run the products without per-matrix plans")
    ap.add_argument("--arith", choices=("native", "split"), default="native",
                    help="arithmetic of the per-matrix plans: native (fp32 data on fp32 matrix "
                         "cores) or split (fp32 data as three bf16 pieces on bf16 matrix cores)")
    ap.add_argument("--graph", action="store_true",
                    help="time the step as HIP graph replays instead of direct calls")
    ap.add_argument("--no-rows", action="store_true",
                    help="headline only: skip the block-shape rows of the other workloads")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="approximate CPU time spent timing the oracle on the headline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB --steps times (the reference "
                         "kernel for scaling HBM byte counters) and exit")
    ap.add_argument("--roof-probe", action="store_true",
                    help="only time plain device stores, copies and reads (torch kernels) of "
                         "the product outputs' sizes and of 256 MiB, as the HBM rates a simple "
                         "kernel reaches here, and exit")
    ap.add_argument("--trace-summary", metavar="CSV",
                    help="only summarise a rocprofv3 kernel trace (kernel_trace.csv) per kernel "
                         "and launch grid, and exit (no GPU needed)")
    return ap.parse_args(argv)


def trace_summary(path: str) -> int:
    """Per (kernel, grid, workgroup, LDS) group of a rocprofv3 kernel trace: dispatches and the
    mean, median, p10 and p90 duration in microseconds, largest total time first.  Separates
    the launches of one kernel that differ in grid, such as the headline products (8 per
    launch: grid y = 8) and single-product rows (grid y = 1)."""
    import csv
    groups = {}
    with open(path, newline="") as f:
        for r in csv.DictReader(f):
            key = (r["Kernel_Name"], r["Grid_Size_X"], r["Grid_Size_Y"], r["Workgroup_Size_X"],
                   r["LDS_Block_Size"])
            us = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1000.0
            groups.setdefault(key, []).append(us)
    print("| dispatches | mean us | median us | p10 us | p90 us | grid | workgroup | LDS | kernel |")
    print("|---|---|---|---|---|---|---|---|---|")
    for key, v in sorted(groups.items(), key=lambda kv: -sum(kv[1])):
        q = pct(v)
        print(f"| {q['n']} | {q['mean']:.2f} | {q['median']:.2f} | {q['p10']:.2f} | "
              f"{q['p90']:.2f} | {key[1]} x {key[2]} | {key[3]} | {key[4]} | {key[0]} |")
    return 0


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
        from paper_2106_08846_amd import bsr as B
        wl = G.bert_large_zipf(R, C, B.bsr_prune_count(1024, 1024, R, C, 0.1))
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


def pct(samples) -> dict:
    """Median, p10, p90 and mean of a list of times."""
    a = np.asarray(samples, dtype=np.float64)
    return {"median": float(np.median(a)), "p10": float(np.percentile(a, 10)),
            "p90": float(np.percentile(a, 90)), "mean": float(a.mean()), "n": int(a.size)}


def roof_probe(args) -> int:
    """HBM rates of plain torch kernels: a store (fill) of the fused-QKV output (4096 x 2304
    fp32, 37.7 MB) and of the BERT-large output of one launch (8 x 6144 x 1024 fp32), and a
    store, a copy and a read (sum) of 256 MiB; median of 20 event-timed runs after 3 warm-up
    runs each.  The floor a product kernel's own stores and reads can reach on this GPU."""
    import torch
    dev = "cuda:0"
    res = {}

    def time_us(fn, reps=20):
        for _ in range(3):
            fn()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(reps)]
        for a, b in ev:
            a.record()
            fn()
            b.record()
        torch.cuda.synchronize()
        return pct([a.elapsed_time(b) * 1e3 for a, b in ev])

    for name, n in (("store_fused_qkv_output", 4096 * 2304),
                    ("store_bert_large_launch_output", 8 * 6144 * 1024),
                    ("store_256MiB", (256 << 20) // 4)):
        t = torch.empty(n, dtype=torch.float32, device=dev)
        q = time_us(lambda: t.fill_(1.0))
        res[name] = {"bytes": 4 * n, "us_median": q["median"], "us_p10": q["p10"],
                     "us_p90": q["p90"], "tbs": 4 * n / q["median"] / 1e6}
        del t
    n = (256 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    q = time_us(lambda: dst.copy_(src))
    res["copy_256MiB"] = {"bytes": 8 * n, "us_median": q["median"], "tbs": 8 * n / q["median"] / 1e6}
    acc = torch.empty((), dtype=torch.float32, device=dev)
    q = time_us(lambda: torch.sum(src, dim=0, out=acc))
    res["read_256MiB"] = {"bytes": 4 * n, "us_median": q["median"], "tbs": 4 * n / q["median"] / 1e6}
    print(json.dumps({"roof_probe": res, "peak_tbs": HBM_PEAK_GBS / 1e3}), flush=True)
    return 0


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


# ------------------------------------------------------------------------------- device setup


class Prepared:
    """A workload on the device: every projection pruned on the GPU, its product prepared as
    bsr_spmm_batched calls of up to 8 products, `sets` copies of every tensor to rotate through
    (copy s of a launch only touches set s)."""

    def __init__(self, wl, sets: int, slices: int = 0, plans: bool = True, arith: int = 0):
        import torch
        from paper_2106_08846_amd import bsr as B
        dev = torch.device("cuda:0")
        self.wl = wl
        self.bf16 = wl.bf16
        X32 = [torch.from_numpy(x).to(dev) for x in wl.X]
        Xs = [B.bsr_cast_f32_bf16(x) for x in X32] if wl.bf16 else X32
        del X32
        self.calls = []          # one dict per projection (set 0)
        self.dense = []          # dense weights (for the GEMM comparison)
        mats = []
        for p in wl.projections:
            N, K = p.W.shape
            k = p.k if p.k is not None else B.bsr_prune_count(N, K, p.R, p.C, p.density)
            Wd = torch.from_numpy(p.W).to(dev)
            M = B.bsr_prune_from_dense(Wd, p.R, p.C, k=k)
            if wl.bf16:
                M = M.to_bf16()
            if "reblock" in wl.notes:
                M = B.bsr_reblock(M, *wl.notes["reblock"])
            self.dense.append(Wd.to(torch.bfloat16) if wl.bf16 else Wd)
            mats.append((M, torch.from_numpy(p.bias).to(dev)))
            T = wl.X[p.x_index].shape[0]
            self.calls.append(dict(T=T, N=N, K=K, R=M.R, C=M.C, k=M.nnzb, x_index=p.x_index))
        self.sets, self.products = [], []
        for s in range(sets):
            xs = Xs if s == 0 else [x.clone() for x in Xs]
            prods = []
            for c, (M, b) in zip(self.calls, mats):
                if s > 0:
                    M = B.BSRMatrix(M.n_rows, M.n_cols, M.R, M.C, M.indptr.clone(),
                                    M.indices.clone(), M.data.clone(), M.nnzb)
                    b = b.clone()
                Y = torch.empty((c["T"], c["N"]), dtype=torch.float32, device=dev)
                prods.append((xs[c["x_index"]], M, b, Y))
            # Per-matrix plans (prepared once, like the pruning) where the block shape has one.
            pls = [self._plan(B, p[1], arith) if plans else None for p in prods]
            self.planned = any(pl is not None for pl in pls)
            self.plan_arith = next((pl.arith for pl in pls if pl is not None), 0)
            groups = [range(i, min(i + 8, len(prods))) for i in range(0, len(prods), 8)]
            self.sets.append([B.SpmmBatchCall([prods[i] for i in g], slices=slices or None,
                                              plans=[pls[i] for i in g]) for g in groups])
            self.products.append(prods)
        self.Xs = Xs
        torch.cuda.synchronize()

    @staticmethod
    def _plan(B, M, arith: int = 0):
        try:
            return B.bsr_plan_prepare(M, arith=arith)
        except B.BSRError as e:
            if e.status == 9 and arith != 0:   # no split plan for this dtype: the native one
                return Prepared._plan(B, M, 0)
            if e.status == 9:      # no plan for this block shape
                return None
            raise

    @property
    def launches_per_step(self) -> int:
        return len(self.sets[0])

    def flops_step(self) -> float:
        return sum(2.0 * c["k"] * c["R"] * c["C"] * c["T"] for c in self.calls)

    def bytes_step(self) -> float:
        """Algorithmic bytes: X read once per product, the BSR arrays, the bias, Y written."""
        sx = 2 if self.bf16 else 4
        tot = 0.0
        for c in self.calls:
            tot += (c["T"] * c["K"] * sx + c["k"] * c["R"] * c["C"] * sx + 4 * c["k"]
                    + 4 * (c["N"] // c["R"] + 1) + 4 * c["N"] + 4 * c["T"] * c["N"])
        return tot

    def step(self, s: int = 0):
        for run in self.sets[s]:
            run()

    def launch_times_us(self, rounds: int) -> list:
        """Kernel-event durations of every launch, visiting the sets round robin."""
        import torch
        ev = []
        for r in range(rounds):
            for run in self.sets[r % len(self.sets)]:
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record()
                b.record()
                ev.append((run, a, b))
        torch.cuda.synchronize()
        for run, a, b in ev:
            run.timed(a, b)
        torch.cuda.synchronize()
        return [a.elapsed_time(b) * 1e3 for _, a, b in ev]


def step_times_ms(fn, n: int, rotate: int = 1):
    """Run fn(i % rotate) n times with an event between consecutive calls; returns (total ms
    between the first and last event, per-call ms)."""
    import torch
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
    torch.cuda.synchronize()
    ev[0].record()
    for i in range(n):
        fn(i % rotate)
        ev[i + 1].record()
    torch.cuda.synchronize()
    per = [ev[i].elapsed_time(ev[i + 1]) for i in range(n)]
    return ev[0].elapsed_time(ev[n]), per


def roofline(prep, launch_us_mean: float) -> dict:
    """Roofline position of one launch taking launch_us_mean microseconds."""
    flops = prep.flops_step() / prep.launches_per_step
    nbytes = prep.bytes_step() / prep.launches_per_step
    # The matrix-core roof of the instructions the products run on: bf16 for bf16 data and
    # for fp32 data split into bf16 pieces, fp32 otherwise.
    on_bf16 = prep.bf16 or getattr(prep, "plan_arith", 0) == ARITH_SPLIT
    peak = (BF16_PEAK_TFLOPS if on_bf16 else FP32_PEAK_TFLOPS) * 1e12
    ai = flops / nbytes
    gbs = nbytes / (launch_us_mean * 1e-6) / 1e9
    tfs = flops / (launch_us_mean * 1e-6) / 1e12
    if ai > peak / (HBM_PEAK_GBS * 1e9):
        r = {"bound": "mfma", "achieved": tfs, "peak": peak / 1e12, "unit": "TFLOP/s",
             "frac": tfs / (peak / 1e12)}
    else:
        r = {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
             "frac": gbs / HBM_PEAK_GBS}
    r.update({"launch_us": launch_us_mean, "algorithmic_bytes_per_launch": nbytes,
              "flops_per_launch": flops, "arithmetic_intensity": ai, "achieved_gbs": gbs,
              "achieved_tflops": tfs})
    return r


def dense_times_us(prep, rounds: int) -> dict:
    """Same-shape dense GEMM per launch group: torch.addmm (fp32) or matmul (bf16) on the
    unpruned weights, timed per group of the step's products with events, sets rotated."""
    import torch
    outs = [[torch.empty((c["T"], c["N"]), dtype=torch.float32, device="cuda:0")
             for c in prep.calls] for _ in range(len(prep.sets))]
    biases = [[p[2] for p in prods] for prods in prep.products]
    xs_sets = [[p[0] for p in prods] for prods in prep.products]
    Ws = prep.dense

    def group(s, lo, hi):
        for i in range(lo, hi):
            X, W, b, Y = xs_sets[s][i], Ws[i], biases[s][i], outs[s][i]
            if prep.bf16:
                Y.copy_(torch.matmul(X, W.t()).float() + b)
            else:
                torch.addmm(b, X, W.t(), out=Y)

    n = len(prep.calls)
    bounds = [(i, min(i + 8, n)) for i in range(0, n, 8)]
    for s in range(len(prep.sets)):          # warm-up
        for lo, hi in bounds:
            group(s, lo, hi)
    times = []
    for r in range(rounds):
        s = r % len(prep.sets)
        for lo, hi in bounds:
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            group(s, lo, hi)
            b.record()
            times.append((a, b))
    torch.cuda.synchronize()
    return pct([a.elapsed_time(b) * 1e3 for a, b in times])


# ------------------------------------------------------------------------------------- rows


def row(spec: str, rotate: int, rounds: int, dense: bool, label: str | None = None,
        plans: bool = True, arith: int = 0) -> dict:
    """One block-shape row: per-launch kernel-event times (median, p10, p90), effective rates,
    roof fraction, the same launches timed back to back (mean per launch, launch gaps
    included), and the dense GEMM beside it."""
    import torch
    print(f"# row {spec}", file=sys.stderr, flush=True)
    wl = build_workload(spec)
    prep = Prepared(wl, rotate, plans=plans, arith=arith)
    for s in range(rotate):
        prep.step(s)
    torch.cuda.synchronize()
    lt = pct(prep.launch_times_us(rounds))
    r = roofline(prep, lt["mean"])
    loop_ms, _ = step_times_ms(prep.step, rounds, rotate)   # the same launches back to back
    c0 = prep.calls[0]
    out = {"workload": wl.name, "spec": spec, "block": f"{c0['R']}x{c0['C']}",
           "dtype": "bf16" if wl.bf16 else "f32", "tokens": c0["T"], "plans": prep.planned,
           "plan_arithmetic": ({1: "native", 2: "bf16x3 split"}[prep.plan_arith]
                               if prep.planned else None),
           "products_per_launch": len(prep.calls) // prep.launches_per_step,
           "launches": lt["n"],
           "protocol": (f"cold: {rotate} rotating copies of every input and output"
                        if rotate > 1 else
                        ("cold by construction: the stack exceeds the last-level cache"
                         if spec.startswith("bert_large") else "warm, launches back to back")),
           "launch_us": {k: lt[k] for k in ("median", "p10", "p90", "mean")},
           "loop_us_per_launch": loop_ms * 1e3 / (rounds * prep.launches_per_step),
           "effective_tflops": r["achieved_tflops"], "effective_tbs": r["achieved_gbs"] / 1e3,
           "roof": {k: r[k] for k in ("bound", "frac", "arithmetic_intensity")},
           "frac_of_hbm": r["achieved_gbs"] / HBM_PEAK_GBS,
           "frac_of_matrix_peak": r["achieved_tflops"] / ((BF16_PEAK_TFLOPS if wl.bf16 else
                                                           FP32_PEAK_TFLOPS))}
    if label:
        out["label"] = label
    if dense:
        d = dense_times_us(prep, rounds)
        out["dense_us"] = {k: d[k] for k in ("median", "p10", "p90")}
        out["sparse_over_dense"] = lt["median"] / d["median"]
    del prep
    torch.cuda.empty_cache()
    return out


def rows(args) -> dict:
    """The other configurations' block-shape rows (see the module docstring)."""
    res = {}
    dense = not args.no_dense
    pl = not args.no_plan
    other = "bert_large:32x32" if args.workload != "bert_large:32x32" else "bert_large:32x1"
    res["bert_large_zipf"] = [row(other, 1, 5, dense, plans=pl)]
    if pl:
        # The headline stack with split-arithmetic plans (fp32 data as bf16 pieces on the bf16
        # matrix cores), and the fused QKV 32x1 rows the same way.
        res["bert_large_zipf"].append(row("bert_large:32x1", 1, 5, dense, plans=pl,
                                          arith=ARITH_SPLIT))
    qkv = []
    for shape in ("32x1", "16x16"):
        for dt in ("", ":bf16"):
            for d in ("0.05", "0.1", "0.2", "0.4"):
                qkv.append(row(f"fused_qkv:{shape}:{d}{dt}", ROTATE_SETS, 8 * ROTATE_SETS,
                               dense, plans=pl))
    if pl:
        for d in ("0.05", "0.1", "0.2", "0.4"):
            qkv.append(row(f"fused_qkv:32x1:{d}", ROTATE_SETS, 8 * ROTATE_SETS, dense, plans=pl,
                           arith=ARITH_SPLIT))
    res["fused_qkv"] = qkv
    res["sweep_T128"] = [row(f"sweep:{s}", 1, 100, dense, plans=pl) for s in
                         ("1x1", "8x1", "16x1", "32x1", "1x32", "4x4", "8x8", "16x16", "32x32")]
    res["bert_base_attn_T128"] = [row("bert_base_attn", 1, 100, dense, plans=pl)]
    res["iht_bert_base"] = [iht_row(32, 1, 0.1), iht_row(1, 32, 0.1)]
    return res


def iht_row(R: int, C: int, density: float, iters: int = 20) -> dict:
    """The iterative projection for Eq. 2 on one BERT-base projection (768 x 768, the Q weight
    of the BERT-base workload) with the reconstruction loss of 4096 synthetic calibration
    tokens: GPU time per iteration (product, dense expansion, update, prune), the loss before
    and after, and the fp64 oracle's time per iteration on this host."""
    import torch
    from paper_2106_08846_amd import bsr as B
    from paper_2106_08846_amd import workloads as G
    print(f"# row iht {R}x{C}", file=sys.stderr, flush=True)
    w = G.bert_base_attention()
    W0 = w.projections[0].W
    N, K = W0.shape
    X = G.fused_qkv(R, C, density, tokens=4096).X[0]         # 4096 x 768 activations
    # H = X^T X by the library's own product (X^T as the input, X^T with all its blocks as the
    # matrix); the 1/T of the loss is left in the step size (only eta H enters the iteration).
    XT = torch.from_numpy(np.ascontiguousarray(X.T)).to("cuda:0")
    full = B.bsr_prune_from_dense(XT, 32, 1, k=(XT.shape[0] // 32) * XT.shape[1])
    H = B.bsr_spmm(XT, full)
    del full
    eta = float(1.0 / torch.linalg.eigvalsh(H.double())[-1])   # the step bound 1/lambda_max
    k = B.bsr_prune_count(N, K, R, C, density)
    W0d = torch.from_numpy(W0).to("cuda:0")
    B.bsr_iht(W0d, H, R, C, k, eta, 2)                       # warm-up
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    M = B.bsr_iht(W0d, H, R, C, k, eta, iters)
    b.record()
    torch.cuda.synchronize()
    total_us = a.elapsed_time(b) * 1e3
    a.record()
    B.bsr_iht(W0d, H, R, C, k, eta, 0)
    b.record()
    torch.cuda.synchronize()
    setup_us = a.elapsed_time(b) * 1e3
    Hd, W064 = H.double(), W0d.double()

    def loss(Wt):
        E = Wt.double() - W064
        return float(0.5 * torch.sum((E @ Hd) * E))
    f0 = loss(B.bsr_to_dense(B.bsr_prune_from_dense(W0d, R, C, k=k)))
    f1 = loss(B.bsr_to_dense(M))
    from oracle import iht_oracle as I
    Hh, W0h = H.double().cpu().numpy(), W0.astype(np.float64)
    t0 = time.perf_counter()
    I.iht(W0h, Hh, R, C, k, eta, 2)
    cpu_ms = (time.perf_counter() - t0) * 1e3 / 3          # three projections, two gradients
    return {"workload": f"iht_bert_base_768_{R}x{C}_d{int(density * 100)}", "block": f"{R}x{C}",
            "iterations": iters, "k": k, "eta": eta, "hessian": "X^T X of 4096 tokens",
            "us_per_iteration": (total_us - setup_us) / iters, "setup_us": setup_us,
            "loss_one_shot": f0, "loss_after": f1,
            "cpu_oracle_ms_per_iteration": cpu_ms, "cpu_oracle_threads": "numpy (BLAS) default"}


# --------------------------------------------------------------------------- CPU baselines


def cpu_baseline(wl, seconds: float) -> dict:
    """The C oracle (fp64 naive BSR loop, OpenMP over tokens) on this host's cores, on a bounded
    sample of the workload: its first product, pruned by the numpy oracle, over all its tokens;
    three samples of about seconds / 3 each, median rate.  Plus one-thread runs of the
    128-token workloads (whole steps), median of three samples each."""
    from oracle import bsr_oracle as O
    from oracle import cpu_oracle
    cores = len(os.sched_getaffinity(0))

    def host_product(wl, p):
        ip, ix, dt = O.prune(p.W, p.R, p.C, k=p.k if p.k is not None else
                             O.prune_count(p.W.shape[0], p.W.shape[1], p.R, p.C, p.density))
        X = wl.X[p.x_index]
        if wl.bf16:
            X = O.bf16_roundtrip(X)
            dt = O.bf16_roundtrip(dt)
        return X, ip, ix, dt, p.W.shape[0], p.bias, 2.0 * len(ix) * p.R * p.C * X.shape[0]

    def rate(prods, budget):
        """Median over three samples of the rate of repeated whole passes over `prods`."""
        rates = []
        for _ in range(3):
            flops, t0 = 0.0, time.perf_counter()
            while True:
                for X, ip, ix, dt, N, b, f in prods:
                    cpu_oracle.spmm(X, ip, ix, dt, N, b)
                    flops += f
                if time.perf_counter() - t0 >= budget:
                    break
            rates.append(flops / (time.perf_counter() - t0) / 1e9)
        return float(np.median(rates)), rates

    cpu_oracle.set_num_threads(cores)
    p0 = wl.projections[0]
    head = [host_product(wl, p0)]
    value, samples = rate(head, seconds / 3)
    out = {"value": value, "unit": "GFLOP/s", "cores": cpu_oracle.num_threads(),
           "kind": "oracle",
           "sample": (f"product {p0.name} of {wl.name} ({p0.W.shape[0]}x{p0.W.shape[1]}, "
                      f"{p0.R}x{p0.C} blocks, {wl.X[p0.x_index].shape[0]} tokens), repeated "
                      f"for about {seconds / 3:.1f} s per sample; median of 3 samples"),
           "samples_gflops": samples, "cpu": cpu_model()}
    cpu_oracle.set_num_threads(1)
    single = {}
    for spec in ("single_768", "bert_base_attn", "sweep"):
        if spec == "sweep":
            from paper_2106_08846_amd import workloads as G
            prods = []
            for R, C in G.SHAPES_SWEEP:
                w = G.block_sweep(R, C)
                prods.append(host_product(w, w.projections[0]))
        else:
            w = build_workload(spec)
            prods = [host_product(w, p) for p in w.projections]
        single[spec] = rate(prods, 0.3)[0]
    cpu_oracle.set_num_threads(cores)
    out["single_thread_gflops"] = single
    return out


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.machine()


# ------------------------------------------------------------------------------------- main


TILED_SHAPES = ((32, 1), (16, 1), (32, 32), (16, 16))
VALU_SHAPES = ((1, 1), (1, 2), (1, 4), (1, 8), (1, 16), (1, 32), (2, 1), (4, 1), (8, 1), (2, 2),
               (4, 4), (8, 8))


def kernel_name(c, bf16: bool, planned: bool = False, persistent: bool = False,
                plan_arith: int = 1, paired: bool = False) -> str:
    """The kernel libbsr's automatic choice launches for this product: the flat-stream kernel
    for 32x1 and 16x1 (its planned form with a plan), the matrix-core tiled kernel for square
    blocks, else the vector-ALU tile kernel, each in its column-chunked form when the 32-token
    X tile does not fit in LDS, else the generic kernel.  (A label: the library's plan decides,
    and the kernel trace shows what ran.)"""
    shape = (c["R"], c["C"])
    flag = "true" if bf16 else "false"
    xb = 2 if bf16 and shape != (16, 1) else 4
    fits = 32 * (c["K"] + 8) * xb + 4 * c["N"] + 4 * (c["N"] // c["R"] + 8) <= 160 * 1024
    if shape in ((32, 1), (16, 1)) and fits:
        pl = (2 if plan_arith == 2 else 1) if planned and shape == (32, 1) else 0
        kern = "spmm_flat_persistent_kernel" if persistent else "spmm_flat_kernel"
        # bf16 32x1 with long rows and many tokens takes 64-token tiles when they fit in LDS.
        nb = c["N"] // 32
        t64 = (bf16 and shape == (32, 1) and c["k"] >= 128 * nb and -(-c["T"] // 64) >= 32
               and ((2 * (c["K"] + 1) * 72 + 255) // 256 * 256 + 16 * 2048 + 4 * c["N"]
                    + 4 * (2 * nb + 10)) <= 160 * 1024)
        pair = ", true" if paired and persistent and pl else ""
        return f"{kern}<{c['R']}, {flag}, {pl}, {64 if t64 else 32}{pair}>"
    if shape in TILED_SHAPES:
        w = 4 if shape == (16, 16) and c["k"] >= 8 * (c["N"] // 16) else 1
        if fits:
            return f"spmm_tiled_kernel<{c['R']}, {c['C']}, 16, {flag}, {w}>"
        return f"spmm_kchunk_kernel<{c['R']}, {c['C']}, {flag}, {w}>"
    if shape in VALU_SHAPES and not (bf16 and shape == (1, 1)):
        kern = "spmm_vtile_kernel" if fits else "spmm_vtile_chunk_kernel"
        return f"{kern}<{c['R']}, {c['C']}, {flag}>"
    return "spmm_generic_kernel"


def main(argv=None) -> int:
    args = parse(argv)
    if args.trace_summary:
        return trace_summary(args.trace_summary)
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the library has no "
              "multi-GPU path, so run it with --gpus 1.", file=sys.stderr, flush=True)
        return 2

    import torch

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    if args.calibrate_copy:
        return calibrate_copy(args)
    if args.roof_probe:
        return roof_probe(args)
    if args.workload.startswith("attn_block"):
        return bench_attention_block(args)
    wl = build_workload(args.workload)
    rotate = args.rotate or (1 if args.workload.startswith("bert_large") else ROTATE_SETS)
    print(f"# workload {wl.name}: {len(wl.projections)} projections, {rotate} set(s)",
          file=sys.stderr, flush=True)
    arith = ARITH_SPLIT if args.arith == "split" else 0
    prep = Prepared(wl, rotate, args.slices, plans=not args.no_plan, arith=arith)
    for i in range(args.warmup):
        prep.step(i % rotate)
    torch.cuda.synchronize()

    fn = prep.step
    if args.graph:
        graphs = []
        side = torch.cuda.Stream()
        for s in range(rotate):
            g = torch.cuda.CUDAGraph()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):
                prep.step(s)
            torch.cuda.current_stream().wait_stream(side)
            torch.cuda.synchronize()
            with torch.cuda.graph(g):
                prep.step(s)
            graphs.append(g)
        for i in range(args.warmup):
            graphs[i % rotate].replay()
        fn = lambda s: graphs[s].replay()   # noqa: E731

    # The timed region: exactly --steps steps.
    total_ms, per_step = step_times_ms(fn, args.steps, rotate)
    ms_per_step = total_ms / args.steps
    samples = list(per_step)
    if len(samples) < MIN_SAMPLES:     # more samples for the percentiles, outside the region
        samples += step_times_ms(fn, MIN_SAMPLES - len(samples), rotate)[1]
    st = pct(samples)
    print(f"# timed {args.steps} steps: {ms_per_step:.4f} ms per step", file=sys.stderr,
          flush=True)

    # A launch with more (token tile, slice) items than the GPU's 256 CUs runs the persistent
    # form of the flat kernel (at least one item per product and tile; the library's automatic
    # slice count is 1 when tiles alone fill the GPU).
    per_launch = len(prep.calls) // prep.launches_per_step
    persistent = per_launch * -(-prep.calls[0]["T"] // 32) > 256
    # Planned products 2i and 2i + 1 of a launch that share X run paired in the persistent
    # kernel (one item per X tile for both).
    paired = (persistent and prep.planned and per_launch % 2 == 0 and
              all(prep.calls[i]["x_index"] == prep.calls[i + 1]["x_index"]
                  for i in range(0, len(prep.calls) - 1, 2)))
    # Roofline of the product kernel: the timed region's time per launch.  The kernel-event
    # durations of every launch over a few more steps (at least 60 launches) go beside it.
    rounds = max(rotate, -(-60 // prep.launches_per_step))
    lt = pct(prep.launch_times_us(rounds))
    roof = roofline(prep, ms_per_step * 1e3 / prep.launches_per_step)
    tr = measured_traffic(wl.name)
    roof.update({"traffic": tr["bytes_per_launch"] if tr else None,
                 "launch_us_source": "timed region / launches per step",
                 "kernel": " + ".join(dict.fromkeys(kernel_name(c, wl.bf16, prep.planned,
                                                                persistent, prep.plan_arith,
                                                                paired)
                                                    for c in prep.calls)),
                 "kernel_event_us": {k: lt[k] for k in ("mean", "median", "p10", "p90", "n")}})

    value = prep.flops_step() / (ms_per_step * 1e-3) / 1e9
    c0 = prep.calls[0]
    out = {
        "metric": METRIC, "value": value, "unit": "GFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if wl.bf16 else "f32", "data": "synthetic",
        "config": {"workload": wl.name, "products_per_step": len(prep.calls),
                   "launches_per_step": prep.launches_per_step,
                   "tokens": c0["T"], "N": c0["N"], "K": c0["K"],
                   "block": f"{c0['R']}x{c0['C']}",
                   "density": wl.projections[0].density,
                   "nnz_per_call": [c["k"] * c["R"] * c["C"] for c in prep.calls][:8],
                   "timing": "hip_graph_replay" if args.graph else "direct_calls",
                   "rotating_sets": rotate, "slices": args.slices or "auto",
                   "plans": prep.planned,
                   "plan_arithmetic": ({1: "native", 2: "bf16x3 split"}[prep.plan_arith]
                                       if prep.planned else None)},
        "step_ms": {k: st[k] for k in ("median", "p10", "p90", "n")},
        "roofline": roof,
    }
    if not args.no_dense:
        d = dense_times_us(prep, rounds)
        out["dense_gemm_ms_per_step"] = d["median"] * prep.launches_per_step / 1e3
        out["dense_gemm_us_per_launch"] = {k: d[k] for k in ("median", "p10", "p90")}
    del prep
    torch.cuda.empty_cache()

    if not args.no_rows:
        print("# rows", file=sys.stderr, flush=True)
        out["rows"] = rows(args)
    if not args.no_cpu_baseline:
        print("# cpu baseline", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)

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


if __name__ == "__main__":
    sys.exit(main())
