"""Benchmark: top-k attention at L = 32768, k = 64 (1 x 16 heads, d = 64, bf16,
chunk 1024, planted top set) on one MI355X.

One step = one ``topk_attn`` call (score tiles, select, fallback, softmax and
gather) over the whole workload, with inputs already resident in HBM. Prints ONE
JSON line with queries/s, score TFLOP/s, the roofline of the dominant kernel
(the fused MFMA score+filter scan; its duration from HIP events recorded by the
library on the launch stream over the timed region), and the fp64 CPU oracle
timed on a bounded sample of the same workload (``cpu_baseline``).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "top-k attn queries/s + score TFLOP/s (% bf16 MFMA peak) at L=32k,k=64"
PEAK_BF16_TFLOPS = 2516.6          # MI355X dense bf16 MFMA, published
PEAK_HBM_GBS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "fused_scan_c3_traffic.json")
CSRC = os.path.join(ROOT, "paper_2106_06899_amd", "csrc")
SCAN_BEGIN = "// ------------------------------------------------------------------ fused path: scan"
SCAN_END = "// ------------------------------------------------------------------ fused path: select"


def scan_source_digest() -> str:
    """Digest of the scan kernel's own source (its section of topk_kernels.hip: the
    argument block, launch shape and kernel), with line comments and blank lines left
    out: counter readings stay valid while its code is unchanged."""
    with open(os.path.join(CSRC, "topk_kernels.hip")) as f:
        text = f.read()
    a, b = text.index(SCAN_BEGIN), text.index(SCAN_END)
    code = []
    for line in text[a:b].splitlines():
        line = line.split("//", 1)[0].rstrip()
        if line:
            code.append(line)
    return hashlib.sha256("\n".join(code).encode()).hexdigest()[:16]


def traffic_for_current_kernel(workload: str, path: int):
    """HBM bytes per scan launch from committed rocprofv3 counter runs, or None when
    they are missing, were taken on another workload or a different kernel source,
    or the call does not run the fused scan."""
    if path != 1:
        return None
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_sha") != scan_source_digest() or t.get("workload") != workload:
        return None
    return t.get("bytes_per_launch")


def _is_scan_ablation(name: str) -> bool:
    """The score-only ablation of the scan (fifth template argument true), which the
    benchmark also runs: its dispatches are not the scan's."""
    if "k_fused_scan<" not in name:
        return False
    args = [a.strip() for a in name.split("k_fused_scan<", 1)[1].split(">", 1)[0].split(",")]
    return len(args) > 4 and args[4] == "true"


def _pmc_average(path: str, kernel_substr: str) -> float:
    """Average counter value per dispatch (KiB) of the kernels whose name holds
    kernel_substr (the scan's score-only ablation excluded)."""
    import csv
    vals = [float(r["Counter_Value"]) for r in csv.DictReader(open(path))
            if kernel_substr in r["Kernel_Name"] and not _is_scan_ablation(r["Kernel_Name"])]
    if not vals:
        raise SystemExit(f"no dispatch of {kernel_substr} in {path}")
    return sum(vals) / len(vals)


def write_traffic(scan_fetch: str, scan_write: str, copy_fetch: str, copy_write: str, copy_bytes: int,
                  command: str) -> dict:
    """HBM bytes per scan launch from rocprofv3 FETCH_SIZE / WRITE_SIZE runs, each
    scaled by what the same counter reads for a plain device copy of copy_bytes."""
    f_copy = _pmc_average(copy_fetch, "copyBuffer")
    w_copy = _pmc_average(copy_write, "copyBuffer")
    kib = copy_bytes / 1024.0
    ff, fw = kib / f_copy, kib / w_copy
    fetch = _pmc_average(scan_fetch, "k_fused_scan") * ff * 1024.0
    write = _pmc_average(scan_write, "k_fused_scan") * fw * 1024.0
    rec = {"kernel_source_sha": scan_source_digest(), "workload": "c3", "bytes_per_launch": fetch + write,
           "fetch_bytes_per_launch": fetch, "write_bytes_per_launch": write,
           "fetch_factor": ff, "write_factor": fw, "copy_bytes": copy_bytes, "command": command}
    os.makedirs(os.path.dirname(TRAFFIC_FILE), exist_ok=True)
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(rec, f, indent=1)
        f.write("\n")
    return rec


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, x, budget_s: float):
    """Time the fp64 oracle (as it stands) on whole query chunks of the workload, one
    chunk per task on a thread pool of as many threads as this process may run on
    (``os.sched_getaffinity``, at most 16), each task with one BLAS thread, until
    about ``budget_s`` seconds have passed; report queries/s."""
    from concurrent.futures import FIRST_COMPLETED, ThreadPoolExecutor, wait
    from oracle import topk_oracle as o
    from threadpoolctl import threadpool_limits
    cores = min(len(os.sched_getaffinity(0)), 16)
    if w.kind == "attn":
        Q, K, V = (x[n].values for n in ("Q", "K", "V"))
        chunks = [(b, h, c0) for b in range(w.B) for h in range(w.H) for c0 in range(0, w.Lq, w.chunk)]

        def one(t):
            b, h, c0 = t
            i = np.arange(c0, min(c0 + w.chunk, w.Lq))
            o.topk_rows(Q[b, h, i], K[b, h], V[b, h], w.k, o.valid_lengths(i, w.Lk, w.causal), "softmax", w.scale)
            return i.size
    else:  # feed-forward: tokens against the rows of W1 (keys) and W2 (values), ReLU weights
        X, W1, W2 = (x[n].values for n in ("X", "W1", "W2"))
        chunks = list(range(0, w.N, w.chunk))

        def one(c0):
            i = np.arange(c0, min(c0 + w.chunk, w.N))
            o.topk_rows(X[i], W1, W2, w.k, np.full(i.size, w.d_ff), "relu")
            return i.size

    done = 0
    with threadpool_limits(1), ThreadPoolExecutor(cores) as ex:
        t0 = time.perf_counter()
        it = iter(chunks)
        running = {ex.submit(one, t) for t in [next(it) for _ in range(min(cores, len(chunks)))]}
        submitted = len(running)
        while running:
            fin, running = wait(running, return_when=FIRST_COMPLETED)
            done += sum(f.result() for f in fin)
            if time.perf_counter() - t0 < budget_s:
                for _ in fin:
                    if submitted < len(chunks):
                        running.add(ex.submit(one, next(it)))
                        submitted += 1
        el = time.perf_counter() - t0
    return {"value": done / el, "unit": "queries/s", "cores": cores, "kind": "oracle",
            "cpu": _cpu_model(),
            "sample": f"{done} queries = {done // w.chunk} chunks of {w.chunk} rows of the same workload "
                      f"(fp64 NumPy, {cores} threads with one BLAS thread each, {el:.1f} s)"}


def bench_backward(args, w, x, dev_tensor):
    """Time the backward pass of one workload: the forward runs once in debug mode to
    produce its cache (selected keys, their raw scores); each timed step is one
    backward call. Roofline: the bytes the call must move at least once (Q, d_out, K,
    V and the cache read, the three gradients written) against the HBM peak; beside it
    the gathered rows (4 rows of d elements per selected (query, key) pair: V and K per
    query, d_out and Q per key), which L2 and MALL mostly serve."""
    import torch
    import paper_2106_06899_amd as tk
    from paper_2106_06899_amd import workloads as wl
    elem = 2 if w.dtype == wl.BF16 else 4
    if w.kind == "attn":
        q, k, v = (dev_tensor(x[n]) for n in ("Q", "K", "V"))
        _, idx, dots = tk.attn(q, k, v, w.k, w.chunk, w.causal, w.scale, debug=True)
        g = torch.randn(q.shape, generator=torch.Generator().manual_seed(5), dtype=torch.float32).to(q.dtype).to(q.device)
        step = lambda: tk.attn_backward(q, k, v, idx, dots, g, w.scale)  # noqa: E731
        rows, keys, d = w.B * w.H * w.Lq, w.B * w.H * w.Lk, w.d
    else:
        a, b1, b2 = (dev_tensor(x[n]) for n in ("X", "W1", "W2"))
        _, idx, dots = tk.ffn(a, b1, b2, w.k, w.chunk, debug=True)
        g = torch.randn(a.shape, generator=torch.Generator().manual_seed(5), dtype=torch.float32).to(a.dtype).to(a.device)
        step = lambda: tk.ffn_backward(a, b1, b2, idx, dots, g)  # noqa: E731
        rows, keys, d = w.N, w.d_ff, w.d_model
    pairs = int((idx >= 0).sum().item())
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    tk.profile_begin()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    stages = tk.profile_end()
    ms_step = 1e3 * elapsed / args.steps
    bwd_ms = stages["backward"][0] / max(stages["backward"][1], 1)
    # HBM roofline on the bytes the call must move at least once: Q and d_out (rows),
    # K and V (keys) read, the cache (index, score) read, d_Q, d_K, d_V written. The
    # per-pair row gathers (V[j], K[j] per row; d_out[i], Q[i] per key) are far larger
    # but mostly hit L2/MALL, so they are reported beside it, not against HBM.
    io_bytes = (2 * rows + 2 * keys) * d * elem + pairs * 8 + (rows + 2 * keys) * d * elem
    gathered = pairs * 4 * d * elem
    achieved = io_bytes / (bwd_ms / 1e3) / 1e9
    rec = {
        "metric": "top-k attention backward (input checkpointing) queries/s",
        "value": rows / (ms_step / 1e3), "unit": "queries/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16" if w.dtype == wl.BF16 else "f32", "data": "synthetic",
        "config": {"workload": f"{w.name}: {w.note}", "selected_pairs": pairs},
        "roofline": {"kernel": "backward call (list build, row and key gathers)", "bound": "hbm", "achieved": achieved,
                     "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": achieved / PEAK_HBM_GBS, "traffic": None,
                     "algorithmic_bytes_per_launch": io_bytes, "avg_launch_ms": bwd_ms},
        "gathered_rows": {"bytes_per_launch": gathered, "GB_per_s": gathered / (bwd_ms / 1e3) / 1e9,
                          "served_from": "L2 / MALL mostly (each selected pair gathers four rows)"},
    }
    print(json.dumps(rec), flush=True)


def _timed(step, steps, warmup):
    """Average ms of `steps` calls of step() after `warmup` untimed ones (synchronised)."""
    import torch
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    return 1e3 * (time.perf_counter() - t0) / steps


def bench_layer(args):
    """The multi-head attention layer at BERT-base shape (d_model 768, 12 heads of 64),
    causal, k = 128, chunk 1024 (the paper's single-layer benchmark setting), one JSON
    line per sequence length: forward and forward + backward time per step, tokens/s,
    the peak of PyTorch's allocator, and the library's per-stage times."""
    import torch
    import paper_2106_06899_amd as tk
    from paper_2106_06899_amd import layers
    dev = torch.device("cuda:0")
    for L in (int(t) for t in args.lengths.split(",")):
        torch.manual_seed(11)
        layer = layers.TopkMultiheadAttention(768, 12, 128, 1024, causal=True, device=dev, dtype=torch.bfloat16)
        x = torch.randn(1, L, 768, device=dev, dtype=torch.bfloat16).requires_grad_()
        g = torch.randn(1, L, 768, device=dev, dtype=torch.bfloat16)

        def fwd():
            with torch.no_grad():
                layer(x)

        def train():
            layer(x).backward(g)

        torch.cuda.synchronize()
        torch.cuda.reset_peak_memory_stats(dev)
        ms_fwd = _timed(fwd, args.steps, args.warmup)
        peak_fwd = torch.cuda.max_memory_allocated(dev)
        torch.cuda.reset_peak_memory_stats(dev)
        tk.profile_begin()
        ms_train = _timed(train, args.steps, args.warmup)
        st = tk.profile_end()
        peak_train = torch.cuda.max_memory_allocated(dev)
        n = args.steps + args.warmup
        stages = {k_: round(v[0] / n, 4) for k_, v in st.items() if v[1]}
        print(json.dumps({
            "metric": "top-k multi-head attention layer tokens/s, forward + backward (BERT-base, causal, k=128, C=1024)",
            "value": L / (ms_train / 1e3), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": ms_train, "ms_forward": ms_fwd, "higher_is_better": True,
            "dtype": "bf16", "data": "synthetic (N(0,1) tokens, default-initialised projections)",
            "config": {"workload": f"attention layer d_model 768, 12 heads x 64, causal, k 128, chunk 1024, L {L}",
                       "batch": 1, "seq_len": L},
            "peak_gib_forward": peak_fwd / 2**30, "peak_gib_train": peak_train / 2**30,
            "library_stage_ms_per_step": stages}), flush=True)
        del layer, x, g


def bench_paper_ff(args):
    """The feed-forward layer at the paper's benchmark shape: 2^18 tokens (batch 512 x
    length 512), d_model 768, k = 512, query chunk 2^14, one JSON line per d_ff."""
    import torch
    import paper_2106_06899_amd as tk
    from paper_2106_06899_amd import layers
    dev = torch.device("cuda:0")
    N, dm, k, C = 1 << 18, 768, 512, 1 << 14
    gen = torch.Generator(device=dev).manual_seed(12)
    x = torch.randn(N, dm, device=dev, dtype=torch.bfloat16, generator=gen).requires_grad_()
    g = torch.randn(N, dm, device=dev, dtype=torch.bfloat16, generator=gen)
    fits = []
    for dff in (int(t) for t in args.d_ff.split(",")):
        w1 = (0.02 * torch.randn(dff, dm, device=dev, generator=gen)).to(torch.bfloat16).requires_grad_()
        w2 = (0.02 * torch.randn(dff, dm, device=dev, generator=gen)).to(torch.bfloat16).requires_grad_()

        def fwd():
            with torch.no_grad():
                tk.ffn(x, w1, w2, k, C)

        def train():
            layers.topk_feed_forward(x, w1, w2, k, C).backward(g)

        torch.cuda.synchronize()
        torch.cuda.reset_peak_memory_stats(dev)
        tk.profile_begin()
        ms_fwd = _timed(fwd, args.steps, args.warmup)
        st_f = tk.profile_end()
        peak_fwd = torch.cuda.max_memory_allocated(dev)
        torch.cuda.reset_peak_memory_stats(dev)
        tk.profile_begin()
        ms_train = _timed(train, args.steps, args.warmup)
        st = tk.profile_end()
        peak_train = torch.cuda.max_memory_allocated(dev)
        n = args.steps + args.warmup
        score_ms = st_f["score"][0] / n
        print(json.dumps({
            "metric": "top-k feed-forward layer tokens/s, forward + backward (2^18 tokens, d_model 768, k=512, C=2^14)",
            "value": N / (ms_train / 1e3), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": ms_train, "ms_forward": ms_fwd, "higher_is_better": True,
            "dtype": "bf16", "data": "synthetic (X ~ N(0,1), W1, W2 ~ N(0, 0.02^2))",
            "config": {"workload": f"feed-forward layer N 2^18, d_model 768, d_ff {dff}, k 512, chunk 2^14",
                       "d_ff": dff},
            "score_tflops": 2.0 * N * dff * dm / (score_ms / 1e3) / 1e12,
            "forward_workspace_gib": tk.ffn_workspace_bytes(N, dm, dff, k, C) / 2**30,
            "peak_gib_forward": peak_fwd / 2**30, "peak_gib_train": peak_train / 2**30,
            "library_stage_ms_per_step": {k_: round(v[0] / n, 4) for k_, v in st.items() if v[1]}}), flush=True)
        fits.append((dff, peak_train / 2**30))
        del w1, w2
        x.grad = None
    if len(fits) >= 2:
        # least-squares line through (d_ff, peak GiB of a training step); the largest
        # d_ff whose fitted peak stays within 30 GiB (the paper's Fig. 3b extrapolation)
        xs = np.array([f[0] for f in fits], dtype=np.float64)
        ys = np.array([f[1] for f in fits], dtype=np.float64)
        slope, icpt = np.polyfit(xs, ys, 1)
        print(json.dumps({
            "metric": "largest d_ff whose forward + backward peak memory fits 30 GiB (linear fit)",
            "value": float((30.0 - icpt) / slope) if slope > 0 else None, "unit": "hidden units",
            "n_gpus": 1, "higher_is_better": True, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": "feed-forward layer N 2^18, d_model 768, k 512, chunk 2^14",
                       "fit_points": [[int(a), round(b, 4)] for a, b in fits]},
            "gib_per_hidden_unit": slope, "intercept_gib": icpt}), flush=True)


def bench_chunk_sweep(args):
    """Forward pass of one BERT-base multi-head self-attention layer (d_model 768, 12
    heads of 64, bidirectional) at L = 65536 for each query chunk size, with top-k
    attention (k = 128) and with query chunking alone (the top-k disabled: every key,
    the paper's comparison baseline): time, the peak of PyTorch's allocator (inputs,
    projections, outputs and the library's workspace, which is a PyTorch tensor) and
    the workspace the library asks for (none for the baseline's streaming softmax)."""
    import torch
    import paper_2106_06899_amd as tk
    from paper_2106_06899_amd import layers
    dev = torch.device("cuda:0")
    L = args.sweep_length
    torch.manual_seed(13)
    x = torch.randn(1, L, 768, device=dev, dtype=torch.bfloat16)
    runs = [(int(t), b, 128) for t in args.chunks.split(",") for b in (0, 1)] + \
           [(int(t), 0, None) for t in args.chunks.split(",")]
    for C, budget, kk in runs:
        torch.manual_seed(14)
        layer = layers.TopkMultiheadAttention(768, 12, kk, C, causal=False, device=dev, dtype=torch.bfloat16)

        def fwd():
            with torch.no_grad():
                layer(x)

        tk.set_memory_budget(budget)  # 0: default budget; 1: one chunk in flight (sequential chunks)
        torch.cuda.synchronize()
        torch.cuda.reset_peak_memory_stats(dev)
        tk.profile_begin()
        ms = _timed(fwd, args.steps, args.warmup)
        st = tk.profile_end()
        ws = tk.attn_workspace_bytes(1, 12, L, L, 64, kk, C, False) if kk else 0
        tk.set_memory_budget(0)
        n = args.steps + args.warmup
        print(json.dumps({
            "metric": "multi-head attention layer forward ms vs query chunk size (BERT-base, L 65536)",
            "value": ms, "unit": "ms", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
            "ms_per_step": ms, "higher_is_better": False, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": f"attention layer d_model 768, 12 heads x 64, bidirectional, L {L}, chunk {C}, "
                                   + (f"top-{kk}" if kk else "query chunking without top-k (every key)"),
                       "chunk": C, "seq_len": L, "k": kk,
                       "chunks_in_flight": "one (sequential)" if budget else "default budget",
                       "path": tk.attn_path(1, 12, L, L, 64, kk, C, False, tk.TOPK_BF16) if kk else "dense"},
            "peak_gib": torch.cuda.max_memory_allocated(dev) / 2**30,
            "workspace_gib": ws / 2**30,
            "library_stage_ms_per_step": {k_: round(v[0] / n, 4) for k_, v in st.items() if v[1]}}), flush=True)
        del layer


def bench_memory_sweep(args):
    """Memory and time of the c3 workload (16 heads, d 64, k 64, chunk 1024, planted
    top set) at several sequence lengths L = Lq = Lk: the peak of PyTorch's allocator
    during a call (the inputs, the output and the library's workspace, which the
    binding allocates as a PyTorch tensor) minus the inputs and the output, the
    workspace the library asks for, and the time per call. One JSON line per length,
    then one with the growth per doubling of L (the method's memory is linear in L)."""
    import torch
    import paper_2106_06899_amd as tk
    from paper_2106_06899_amd import workloads as wl
    dev = torch.device("cuda:0")
    lengths = [int(t) for t in args.mem_lengths.split(",")]
    extra = {}
    for L in lengths:
        w = wl.WORKLOADS["c3"].scaled(Lq=L, Lk=L)
        print(f"[bench] memory sweep L={L}: generating", file=sys.stderr, flush=True)
        x = wl.make_inputs(w)
        q, k, v = (torch.from_numpy(np.ascontiguousarray(x[n].bits)).view(torch.bfloat16).to(dev)
                   for n in ("Q", "K", "V"))
        del x
        io_bytes = 4 * q.numel() * q.element_size()  # Q, K, V and the output

        def step():
            tk.attn(q, k, v, w.k, w.chunk, w.causal, w.scale)

        torch.cuda.synchronize()
        torch.cuda.reset_peak_memory_stats(dev)
        ms = _timed(step, args.steps, args.warmup)
        peak = torch.cuda.max_memory_allocated(dev)
        ws = tk.attn_workspace_bytes(w.B, w.H, L, L, w.d, w.k, w.chunk, w.causal)
        extra[L] = peak - io_bytes
        print(json.dumps({
            "metric": "top-k attention peak memory above inputs and output vs sequence length",
            "value": extra[L] / 2**30, "unit": "GiB", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
            "ms_per_step": ms, "queries_per_s": w.queries / (ms / 1e3), "higher_is_better": False,
            "dtype": "bf16", "data": "synthetic",
            "config": {"workload": f"c3 shape at L {L}: 1x16 heads, d 64, k 64, chunk 1024, planted top set",
                       "seq_len": L, "path": tk.attn_path(w.B, w.H, L, L, w.d, w.k, w.chunk, w.causal)},
            "peak_gib": peak / 2**30, "inputs_and_output_gib": io_bytes / 2**30,
            "workspace_gib": ws / 2**30}), flush=True)
        del q, k, v
    growth = {f"{a}->{b}": extra[b] / extra[a] for a, b in zip(lengths, lengths[1:]) if b == 2 * a}
    print(json.dumps({"metric": "growth of peak memory above inputs and output per doubling of L",
                      "value": max(growth.values()) if growth else None, "unit": "ratio",
                      "higher_is_better": False, "per_doubling": growth}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="c3")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="only run a plain device-to-device copy of BYTES bytes 5 times (counter calibration)")
    ap.add_argument("--write-traffic", nargs=4, metavar=("SCAN_FETCH", "SCAN_WRITE", "COPY_FETCH", "COPY_WRITE"),
                    help="write the scan's HBM bytes per launch from four rocprofv3 counter_collection.csv files")
    ap.add_argument("--copy-bytes", type=int, default=1 << 30)
    ap.add_argument("--traffic-command", default="")
    ap.add_argument("--memory-sweep", action="store_true",
                    help="peak memory and time of the c3 workload at several sequence lengths")
    ap.add_argument("--mem-lengths", default="4096,8192,16384,32768,65536", help="lengths for --memory-sweep")
    ap.add_argument("--layer", action="store_true",
                    help="time the multi-head attention layer (BERT-base shape, causal, k 128, chunk 1024)")
    ap.add_argument("--lengths", default="4096,16384,65536", help="sequence lengths for --layer")
    ap.add_argument("--chunk-sweep", action="store_true",
                    help="forward of one BERT-base attention layer at L 65536, k 128, for each query chunk size")
    ap.add_argument("--chunks", default="64,128,256,512,1024,2048,4096", help="chunk sizes for --chunk-sweep")
    ap.add_argument("--sweep-length", type=int, default=65536)
    ap.add_argument("--paper-ff", action="store_true",
                    help="time the feed-forward layer at the paper's shape (2^18 tokens, d_model 768, k 512)")
    ap.add_argument("--d-ff", default="2048,4096,8192,16384,32768,65536", help="d_ff values for --paper-ff")
    ap.add_argument("--backward", action="store_true",
                    help="time the backward pass (input checkpointing) instead of the forward")
    args = ap.parse_args()
    if args.write_traffic:
        print(json.dumps(write_traffic(*args.write_traffic, args.copy_bytes, args.traffic_command)))
        return
    if args.copy_probe:
        import torch
        src = torch.ones(args.copy_probe // 4, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": src.numel() * 4, "launches": 5}))
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for {args.gpus}); there is no multi-GPU path.",
              file=sys.stderr)
        sys.exit(2)

    if args.memory_sweep:
        bench_memory_sweep(args)
        return
    if args.layer:
        bench_layer(args)
        return
    if args.paper_ff:
        bench_paper_ff(args)
        return
    if args.chunk_sweep:
        bench_chunk_sweep(args)
        return

    import torch
    import paper_2106_06899_amd as tk
    from paper_2106_06899_amd import workloads as wl

    w = wl.WORKLOADS[args.workload]
    print(f"[bench] generating {w.name}: {w.note}", file=sys.stderr, flush=True)
    x = wl.make_inputs(w)
    dev = torch.device("cuda:0")

    def dev_tensor(t):
        return torch.from_numpy(np.ascontiguousarray(t.bits)).view(torch.bfloat16).to(dev) \
            if t.dtype == wl.BF16 else torch.from_numpy(t.values).to(dev)

    if w.kind == "attn":
        q, k, v = (dev_tensor(x[n]) for n in ("Q", "K", "V"))
        step = lambda: tk.attn(q, k, v, w.k, w.chunk, w.causal, w.scale)  # noqa: E731
        flops = 2.0 * w.d * (w.B * w.H) * (w.Lq * (w.Lq + 1) / 2 if w.causal else w.Lq * w.Lk)
        path = tk.attn_path(w.B, w.H, w.Lq, w.Lk, w.d, w.k, w.chunk, w.causal,
                            tk.TOPK_BF16 if w.dtype == wl.BF16 else tk.TOPK_F32)
    else:
        a, b, c = (dev_tensor(x[n]) for n in ("X", "W1", "W2"))
        step = lambda: tk.ffn(a, b, c, w.k, w.chunk)  # noqa: E731
        flops = 2.0 * w.d_model * w.N * w.d_ff
        path = tk.ffn_path(w.N, w.d_model, w.d_ff, w.k, w.chunk)
    queries = w.queries
    if args.backward:
        bench_backward(args, w, x, dev_tensor)
        return

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    print(f"[bench] warmup done ({args.warmup} steps)", file=sys.stderr, flush=True)

    tk.profile_begin()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    stages = tk.profile_end()
    ms_step = 1e3 * elapsed / args.steps
    print(f"[bench] timed {args.steps} steps: {ms_step:.3f} ms/step", file=sys.stderr, flush=True)

    scan_ms, scan_n = stages["score"]
    scan_avg_s = scan_ms / max(scan_n, 1) / 1e3
    launches_per_step = scan_n / args.steps
    flops_per_launch = flops / max(launches_per_step, 1)
    achieved = flops_per_launch / scan_avg_s / 1e12
    score_tflops_call = flops / (ms_step / 1e3) / 1e12
    traffic = traffic_for_current_kernel(w.name, path)

    # score + select: the fused path's candidate select finishes what the scan's filter
    # started, so the pair is reported as one figure beside the scan alone
    sel_ms = stages["select"][0] / args.steps
    score_step_ms = scan_ms / args.steps
    score_select = {"ms_per_step": score_step_ms + sel_ms,
                    "tflops": flops / ((score_step_ms + sel_ms) / 1e3) / 1e12}
    score_select["frac"] = score_select["tflops"] / PEAK_BF16_TFLOPS
    core = None
    if path == 1 and w.kind == "attn" and w.d == 64 and 32 < w.k <= 64 and not w.causal:
        # the scan's score-core ablation at the same launch shape (no filter): its ceiling
        for abl in (False, True):
            tk.scan_ablation(q, k, w.k, w.chunk, score_only=abl)  # warm-up
        torch.cuda.synchronize()
        res = {}
        for abl in (False, True):
            tk.profile_begin()
            for _ in range(5):
                tk.scan_ablation(q, k, w.k, w.chunk, score_only=abl)
            torch.cuda.synchronize()
            st_ = tk.profile_end()["score"]
            res[abl] = st_[0] / max(st_[1], 1)
        core = {"kernel": "k_fused_scan score-only ablation (MFMA, K tiles, block maxima; no filter)",
                "avg_launch_ms": res[True], "tflops": flops_per_launch / (res[True] / 1e3) / 1e12,
                "full_scan_same_run_ms": res[False]}
        core["frac"] = core["tflops"] / PEAK_BF16_TFLOPS
    mt, mhz = tk.probe_mfma()
    mfma = {"sustained_tflops": mt, "frac_of_datasheet": mt / PEAK_BF16_TFLOPS, "shader_clock_mhz": mhz,
            "note": "register-only v_mfma_f32_32x32x16_bf16 stream, two waves per SIMD on every CU"}

    cpu = None
    if not args.no_cpu:
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        cpu = cpu_baseline(w, x, args.cpu_seconds)

    rec = {
        "metric": METRIC,
        "value": queries / (ms_step / 1e3),
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == wl.BF16 else "f32",
        "data": "synthetic",
        "config": {"workload": f"{w.name}: {w.note}", "B": w.B, "H": w.H, "Lq": w.Lq, "Lk": w.Lk, "d": w.d,
                   "k": w.k, "chunk": w.chunk, "causal": w.causal, "scale": w.scale,
                   "path": {1: "fused", 2: "chunk-tile", 3: "chunk-tile rows below 1024 R, fused above", 4: "filtered chunk-tile"}.get(path, path)} if w.kind == "attn" else
                  {"workload": f"{w.name}: {w.note}", "N": w.N, "d_model": w.d_model, "d_ff": w.d_ff, "k": w.k,
                   "chunk": w.chunk, "path": {1: "fused", 2: "chunk-tile", 3: "chunk-tile rows below 1024 R, fused above", 4: "filtered chunk-tile"}.get(path, path)},
        "score_tflops_whole_call": score_tflops_call,
        "score_frac_of_bf16_peak_whole_call": score_tflops_call / PEAK_BF16_TFLOPS,
        "stage_ms_per_step": {s: stages[s][0] / args.steps for s in stages},
        "score_select": score_select,
        "score_core_ceiling": core,
        "mfma_probe": mfma,
        "roofline": {
            "kernel": {1: f"k_fused_scan (d={w.d})",
                       2: "score stage: k_tile_scores_mfma" if w.dtype == wl.BF16 and w.d % 32 == 0 else
                          "score stage: k_tile_scores (fp32)",
                       3: "score stage: k_tile_scores_mfma (rows below 1024 R) + k_fused_scan",
                       4: "score stage: k_tile_scores_mfma sample + k_filter_threshold + "
                          + ("thresholded k_fused_scan (direct appends)"
                             if (w.d if w.kind == "attn" else w.d_model) == 128 and w.dtype == wl.BF16
                             else "filtered k_tile_scores_mfma")}.get(path, str(path)),
            "bound": "mfma",
            "achieved": achieved,
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": achieved / PEAK_BF16_TFLOPS,
            "traffic": traffic,
            "algorithmic_flops_per_launch": flops_per_launch,
            "avg_launch_ms": scan_avg_s * 1e3,
        },
        "cpu_baseline": cpu,
    }
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
