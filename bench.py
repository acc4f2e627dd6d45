#!/usr/bin/env python3
"""Benchmark of the AQLM token-generation product on one MI355X.

Default workload (one "step"): the linear layers of one Llama-2-70B decode
step at batch 1 on one GPU - 80 blocks x {q, o: 8192x8192; k, v: 1024x8192;
gate, up: 28672x8192; down: 8192x28672} = 560 AQLM 2x8 (g = 8)
matrix-vector products (17.16 GB), each layer with its own random codes,
codebooks, scales and input vector, all resident in HBM, launched back to
back on one stream as one HIP graph (320 launches: grouped q/k/v, o, grouped
gate/up, down per block).  ``value`` is the step's algorithmic HBM bytes
(codes + codebooks + scales + x + y of every layer) divided by the measured
step time; tokens/s-equivalent is 1 / step time (linear layers only:
attention, norms, embeddings and the LM head are not part of the step).

Also reported on the same JSON line:
  roofline      the dominant kernel against 8 TB/s: algorithmic bytes per
                launch over its average launch duration, measured live with
                HIP events around the timed graph replays (gaps included);
                beside it, the committed rocprofv3 kernel trace of this
                command for the same kernel source (profiles/
                kernel_durations.txt): its per-kernel average and the share
                of its step the kernels filled.
                ``traffic`` is the HBM bytes per launch from the committed
                counter summary (null once the source has changed);
  cpu_baseline  the CPU oracle (dequantize + fp64 product) timed on the host
                cores on a sample of the step's layers, scaled to the step,
                with the CPU model and a one-thread time;
  secondary     the same step as one persistent launch (aqlm_gemv_step), the
                Llama-2-7B steps in 2x8 and 1x16, single layers rotated
                over >= 1 GiB of replicas (so HBM, not the 256 MB MALL, is
                measured), the small-batch / prefill products,
                dequantization, the gradients through Eq. 2 and the Phase-1
                beam search.

The timed region is bracketed by two short spin kernels outside its events,
so that ``--summarize-trace`` can pick its dispatches out of a rocprofv3
kernel trace.  Only one GPU is supported: --gpus N with N > 1 exits with a
message.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0      # MI355X HBM3E, vendor peak
MFMA_F16_PEAK_TFS = 2500.0  # MI355X dense fp16 matrix peak

WORKLOADS = {
    # name: (model shapes key, M, B)
    "llama2-7b-2x8": ("7b", 2, 8),
    "llama2-7b-1x16": ("7b", 1, 16),
    "llama2-70b-2x8": ("70b", 2, 8),
}


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse_args():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--spread-steps", type=int, default=20,
                    help="event-timed replays of the per-step spread pass after the timed region (counter runs "
                         "use few: every dispatch is serialised under counter collection)")
    ap.add_argument("--workload", default="llama2-70b-2x8", choices=sorted(WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-secondary", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="CPU-baseline time budget (all threads)")
    ap.add_argument("--batch-case", metavar="M,B,n[,1]", action="append",
                    help="only time the 11008x4096 product of this format and token count "
                         "(repeatable) and print its row; a fourth field 1 times the workspace "
                         "product (aqlm_gemm) instead")
    ap.add_argument("--summarize-trace", metavar="KERNEL_TRACE_CSV",
                    help="print per-kernel durations of the dispatches inside the timed region of a "
                         "rocprofv3 kernel trace (--kernel-trace) of a bench.py run, and exit")
    ap.add_argument("--compare-paths", action="store_true",
                    help="only time the batch-1 2x8 launches of the Llama-2-70B step (and a 65536x8192 layer) "
                         "through both kernel families (codeword gathers, partial-product tables) and exit")
    ap.add_argument("--backward", action="store_true",
                    help="only time the gradients through Eq. 2 (aqlm_backward) and exit")
    ap.add_argument("--persistent", action="store_true",
                    help="only the workload's step as one persistent launch (aqlm_gemv_step) beside its graph")
    ap.add_argument("--tiled", action="store_true",
                    help="the decode step over tiled 8-bit codes (aqlm_gemv_grouped_tiled), beside the row-major graph")
    ap.add_argument("--sorted", action="store_true",
                    help="only the workload's step (a 1x16 one) over chunk-sorted codes beside its graph")
    ap.add_argument("--single-layers", action="store_true",
                    help="only the single-layer matrix-vector rows (incl. bit-packed codes)")
    ap.add_argument("--beam-search", action="store_true",
                    help="only time the Phase-1 beam search (aqlm_beam_search) and exit")
    ap.add_argument("--once", action="store_true",
                    help="with --compare-paths: launch each family once per case, untimed (for counter runs)")
    ap.add_argument("--floors", action="store_true",
                    help="only run the microbenchmarks of the GPU's limits (launch, dependent load, HBM read "
                         "stream, matrix-core issue rate, LDS and L2 gathers) and exit")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 256 MiB device copy a few times (the reference kernel for "
                         "scaling HBM byte counters) and exit")
    return ap.parse_args()


class DeviceLayer:
    def __init__(self, seed, d_out, d_in, M, B, n=1, x=None, packed=False, g=8):
        from paper_2401_06118_amd import format as fmt
        from paper_2401_06118_amd import synth
        self.shape = fmt.AqlmShape(d_out, d_in, M, B, g)
        make = synth.device_packed_layer if packed else synth.device_layer
        self.codes, self.codebooks, self.scales, xg = make(seed, d_out, d_in, M, B, g=g, n=n)
        self.x = xg if x is None else x
        import torch
        self.y = torch.empty((n, d_out), dtype=torch.float16, device="cuda")
        self.n = n

    def problem(self):
        return (self.codes, self.codebooks, self.scales, self.x[0], self.y[0])

    def gemv(self, aq):
        aq.gemv(self.codes, self.codebooks, self.scales, self.x[0], out=self.y[0])

    def gemm(self, aq):
        aq.gemm_small_batch(self.codes, self.codebooks, self.scales, self.x, out=self.y)

    def gemm_ws(self, aq, ws):
        aq.gemm(self.codes, self.codebooks, self.scales, self.x, workspace=ws, out=self.y)


def decode_step_layers(model: str, M: int, B: int, seed0: int):
    """Per block, in order: q, k, v, o, gate, up, down.  q/k/v read one shared
    input vector and gate/up another, as in the model."""
    import torch

    from paper_2401_06118_amd import format as fmt
    n_blocks, projs = fmt.LLAMA2_BLOCKS[model]
    gen = torch.Generator(device="cuda")
    gen.manual_seed(seed0 + 7)
    layers = []
    for b in range(n_blocks):
        x_attn = torch.randn((1, projs[0][1]), device="cuda", generator=gen).half()
        x_mlp = torch.randn((1, projs[4][1]), device="cuda", generator=gen).half()
        shared = {0: x_attn, 1: x_attn, 2: x_attn, 4: x_mlp, 5: x_mlp}
        for p, (d_out, d_in) in enumerate(projs):
            layers.append(DeviceLayer(seed0 + 16 * b + p, d_out, d_in, M, B, x=shared.get(p)))
    return layers


def launches_by_dependency(layers, aq):
    """One launch per dependency level of a block: grouped (q, k, v), o,
    grouped (gate, up), down."""
    out = []
    for b in range(0, len(layers), 7):
        q, k, v, o, gate, up, down = layers[b:b + 7]
        out.append(lambda q=q, k=k, v=v: aq.gemv_grouped([q.problem(), k.problem(), v.problem()]))
        out.append(lambda o=o: o.gemv(aq))
        out.append(lambda gate=gate, up=up: aq.gemv_grouped([gate.problem(), up.problem()]))
        out.append(lambda down=down: down.gemv(aq))
    return out


def launches_tiled(layers, tiled, aq):
    """launches_by_dependency over tiled codes (aqlm_gemv_grouped_tiled),
    writing the same outputs."""
    out = []
    for b in range(0, len(layers), 7):
        grp = lambda idx: (lambda: aq.gemv_tiled_grouped([(tiled[i], layers[i].x[0], layers[i].y[0]) for i in idx]))
        out += [grp([b, b + 1, b + 2]), grp([b + 3]), grp([b + 4, b + 5]), grp([b + 6])]
    return out


def graph_of(launches):
    """Capture the launch list into one HIP graph (torch.cuda.CUDAGraph)."""
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for fn in launches:  # warm-up outside capture (sets kernel attributes once)
            fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for fn in launches:
            fn()
    torch.cuda.synchronize()
    return g


MARKER_CYCLES = 20000  # spin kernel that brackets a timed region (about 10 us)


def time_steps(fn, steps, warmup, markers=False):
    """ms per call of fn over `steps` calls bracketed by a HIP event pair on
    the current stream, after `warmup` untimed calls.  markers: a short spin
    kernel goes out before the start event and after the end event (outside
    the timed region) so a kernel trace shows where the region starts and
    ends."""
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    if markers:
        torch.cuda._sleep(MARKER_CYCLES)
    start.record()
    for _ in range(steps):
        fn()
    end.record()
    if markers:
        torch.cuda._sleep(MARKER_CYCLES)
    torch.cuda.synchronize()
    return start.elapsed_time(end) / steps  # ms


def step_spread(fn, steps):
    """Per-step durations from an event pair around each step, in a pass of
    its own after the timed region (the events between steps would perturb
    it): p10, median and p90 in ms."""
    import torch
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    torch.cuda.synchronize()
    for a, b in ev:
        a.record()
        fn()
        b.record()
    torch.cuda.synchronize()
    ts = sorted(a.elapsed_time(b) for a, b in ev)
    q = lambda f: ts[min(len(ts) - 1, int(f * len(ts)))]
    return {"p10": q(0.1), "median": q(0.5), "p90": q(0.9), "steps": steps}


def per_launch_ms(launches, reps):
    """Average time of each launch between a HIP event pair recorded around it
    on the launching (torch current) stream, over `reps` passes.  Each pass
    starts behind a spin kernel long enough for the host to queue every event
    and launch first, so the pairs time the GPU, not the host's enqueue rate.
    An event pair also counts the dispatch of the launch and the events
    themselves, so this is an upper bound of the kernel's duration."""
    import torch
    ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in launches]
          for _ in range(reps)]
    torch.cuda.synchronize()
    for r in range(reps):
        torch.cuda._sleep(int(2.4e9 * (0.005 + 60e-6 * len(launches))))
        for (a, b), fn in zip(ev[r], launches):
            a.record()
            fn()
            b.record()
        torch.cuda.synchronize()
    return [sum(ev[r][i][0].elapsed_time(ev[r][i][1]) for r in range(reps)) / reps for i in range(len(launches))]


def source_digest(*names):
    """Digest of kernel sources with comments and whitespace removed, so that
    it changes with the code and not with its comments."""
    import re
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2401_06118_amd", "csrc", n), encoding="utf-8") as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        text = re.sub(r"//[^\n]*", "", text)
        h.update("".join(text.split()).encode())
    return h.hexdigest()[:16]


def _profile_lookup(fname: str, key: str, digest: str):
    """Fields after (key, digest) on the matching line of profiles/<fname>."""
    path = os.path.join(ROOT, "profiles", fname)
    if not os.path.exists(path):
        return None
    for line in open(path):
        parts = line.split()
        if len(parts) >= 3 and parts[0] == key and parts[1] == digest:
            return parts[2:]
    return None


def measured_traffic(kernel_key: str, digest: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or
    None if there is none for this kernel source."""
    f = _profile_lookup("traffic.txt", kernel_key, digest)
    return float(f[0]) if f else None


def traced_duration(kernel_key: str, digest: str):
    """(average kernel duration in us, dispatches per step, the traced run's
    event-timed ms per step) over the timed graph replays, from the committed
    rocprofv3 kernel-trace summary of this workload, or None if there is none
    for this kernel source."""
    f = _profile_lookup("kernel_durations.txt", kernel_key, digest)
    return (float(f[0]), float(f[1]), float(f[2])) if f else None


def summarize_trace(csv_path: str):
    """Per-kernel durations of the dispatches between the first two marker
    spin kernels (the timed region of the headline step) of a rocprofv3
    kernel_trace.csv."""
    import csv
    rows = []
    with open(csv_path, newline="") as f:
        for r in csv.DictReader(f):
            rows.append((int(r["Start_Timestamp"]), int(r["End_Timestamp"]), r["Kernel_Name"]))
    rows.sort()
    marks = [i for i, r in enumerate(rows) if "spin_kernel" in r[2]]
    if len(marks) < 2:
        raise SystemExit("no pair of marker kernels in the trace")
    inside = rows[marks[0] + 1:marks[1]]
    by = {}
    for t0, t1, name in inside:
        by.setdefault(name, []).append((t1 - t0) / 1000.0)
    window_us = (rows[marks[1]][0] - rows[marks[0]][1]) / 1000.0
    out = {"window_us": window_us, "dispatches": len(inside), "kernels": {}}
    for name, d in sorted(by.items(), key=lambda kv: -sum(kv[1])):
        d.sort()
        out["kernels"][name] = {"calls": len(d), "total_us": sum(d), "avg_us": sum(d) / len(d),
                                "median_us": d[len(d) // 2], "min_us": d[0], "max_us": d[-1]}
    return out


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(layers, budget_s):
    """Oracle (dequantize + fp64 product) on the host cores, one layer of each
    distinct shape, repeated until the budget is spent; scaled to the step.
    The two parts are timed separately.  Then one pass over the same layers
    with one thread."""
    import numpy as np

    import oracle
    shapes = {}
    for L in layers:
        shapes.setdefault((L.shape.d_out, L.shape.d_in), []).append(L)
    per_shape = {}
    host = {}
    for key, ls in shapes.items():
        L = ls[0]
        codes = L.codes.cpu().numpy()
        if L.shape.B > 8:
            codes = codes.view(np.uint16)
        host[key] = (codes, L.codebooks.cpu().numpy(), L.scales.cpu().numpy(), L.x.cpu().numpy())
        per_shape[key] = ([], [])
    threads = oracle.num_threads()
    t_end = time.perf_counter() + budget_s
    rounds = 0
    while True:
        for key, (codes, cb, sc, x) in host.items():
            t0 = time.perf_counter()
            w = oracle.dequantize(codes, cb, sc)
            t1 = time.perf_counter()
            oracle.matmul_f16(w, x)
            t2 = time.perf_counter()
            per_shape[key][0].append(t1 - t0)
            per_shape[key][1].append(t2 - t1)
        rounds += 1
        if time.perf_counter() > t_end or rounds >= 500:
            break
    deq_s = sum(len(shapes[k]) * float(np.median(v[0])) for k, v in per_shape.items())
    mm_s = sum(len(shapes[k]) * float(np.median(v[1])) for k, v in per_shape.items())
    step_s = deq_s + mm_s
    # one thread, one pass
    one_s = 0.0
    try:
        oracle.set_threads(1)
        one_threads = oracle.num_threads()
        for key, (codes, cb, sc, x) in host.items():
            t0 = time.perf_counter()
            oracle.matmul_f16(oracle.dequantize(codes, cb, sc), x)
            one_s += len(shapes[key]) * (time.perf_counter() - t0)
    finally:
        oracle.set_threads(threads)
    step_bytes = sum(L.shape.gemv_bytes(1) for L in layers)
    return {
        "value": step_bytes / step_s / 1e9,
        "unit": "GB/s",
        "cores": threads,
        "kind": "oracle",
        "sample": (f"one layer of each of the {len(shapes)} distinct shapes, dequantize + fp64 product, "
                   f"median of {rounds} runs each, step time = sum over shapes of count x median "
                   f"({step_s:.3f} s per step, {1.0 / step_s:.4f} tok/s-eq)"),
        "cpu_model": cpu_model(),
        "host_cpus": os.cpu_count(),
        "split_s_per_step": {"dequantize": deq_s, "fp64_product": mm_s},
        "one_thread": {"value": step_bytes / one_s / 1e9, "unit": "GB/s", "threads": one_threads,
                       "s_per_step": one_s,
                       "sample": "one run of each distinct shape on one thread, scaled by its count in the step"},
    }


def single_layer_rows(aq, torch):
    """Single layers rotated over >= 1 GiB of replicas so each call reads HBM."""
    rows = []
    for name, (d_out, d_in, M, B) in {
        "4096x4096 2x8": (4096, 4096, 2, 8),
        "4096x4096 1x16": (4096, 4096, 1, 16),
        "11008x4096 1x16": (11008, 4096, 1, 16),
        "4096x11008 1x16": (4096, 11008, 1, 16),
        "4096x4096 1x15": (4096, 4096, 1, 15),
        "11008x4096 1x15": (11008, 4096, 1, 15),
        "11008x4096 2x12": (11008, 4096, 2, 12),
        "11008x4096 2x16": (11008, 4096, 2, 16),
        "28672x8192 2x8": (28672, 8192, 2, 8),
        "11008x4096 2x15": (11008, 4096, 2, 15),
        # bit-packed codes (B bits per code, rows padded to 32-bit words)
        "11008x4096 2x12 packed": (11008, 4096, 2, 12),
        "11008x4096 2x15 packed": (11008, 4096, 2, 15),
        "11008x4096 1x15 packed": (11008, 4096, 1, 15),
        "4096x4096 2x12 packed": (4096, 4096, 2, 12),
        # chunk-sorted codes (aqlm_gemv_sorted)
        "4096x4096 1x16 sorted": (4096, 4096, 1, 16),
        "11008x4096 1x16 sorted": (11008, 4096, 1, 16),
        "4096x11008 1x16 sorted": (4096, 11008, 1, 16),
        "28672x8192 1x16 sorted": (28672, 8192, 1, 16),
        "8192x28672 1x16 sorted": (8192, 28672, 1, 16),
        "11008x4096 2x16 sorted": (11008, 4096, 2, 16),
        "11008x4096 1x15 sorted": (11008, 4096, 1, 15),
        # larger groups (about two bits per weight, like 2x8)
        "4096x4096 4x8 gs16": (4096, 4096, 4, 8),
        "4096x4096 8x8 gs32": (4096, 4096, 8, 8),
        "4096x4096 15x8 gs64": (4096, 4096, 15, 8),
    }.items():
        from paper_2401_06118_amd import format as fmt
        packed = name.endswith("packed")
        g = int(name.split(" gs")[1]) if " gs" in name else 8
        shp = fmt.AqlmShape(d_out, d_in, M, B, g)
        code_bytes = shp.packed_codes_bytes() if packed else shp.codes_bytes()
        reps = max(2, min(256, (1 << 30) // code_bytes + 1))
        sorted_ = name.endswith("sorted")
        if sorted_:
            # one layer sorted on the host, its sorted arrays copied per replica
            import copy
            src = DeviceLayer(900000, d_out, d_in, M, B)
            base = aq.SortedCodes(src.codes, src.codebooks, src.scales)
            sbytes = base.entries.numel() * 4
            reps = max(2, min(256, (1 << 30) // sbytes + 1))
            layers = []
            for i in range(reps):
                c = copy.copy(base)
                c.entries, c.index = base.entries.clone(), base.index.clone()
                c.codebooks = src.codebooks.clone()
                layers.append(c)
            ws = base.workspace
            x0, y0 = src.x[0], src.y[0]
            calls = [lambda c=c: c.gemv(x0, out=y0) for c in layers]
            for c in layers:
                c.workspace = ws
        else:
            layers = [DeviceLayer(900000 + i, d_out, d_in, M, B, packed=packed, g=g) for i in range(reps)]
            calls = [lambda L=L: L.gemv(aq) for L in layers]
        g = graph_of(calls)
        ms = time_steps(g.replay, steps=3, warmup=1) / reps
        pair = per_launch_ms(calls[: min(reps, 64)], reps=2)
        pair_ms = sum(pair) / len(pair)
        del g
        b = shp.packed_gemv_bytes(1) if packed else shp.gemv_bytes(1)
        pb = shp.paper_gemv_bytes(1)  # codes at B bits each
        row = {"layer": name, "bytes": b, "paper_bytes": pb, "GBs_paper_bytes": pb / (ms * 1e6),
               "us_per_call": ms * 1e3, "frac_per_call": b / (ms * 1e6) / HBM_PEAK_GBS,
               "GBs_per_call": b / (ms * 1e6), "event_pair_us": pair_ms * 1e3,
               "GBs_event_pair": b / (pair_ms * 1e6), "replicas": reps}
        if sorted_:
            # bytes the sorted product streams (entries: 4 per code plus pads)
            row["sorted_entry_bytes"] = sbytes
            row["GBs_sorted_entries"] = sbytes / (ms * 1e6)
        rows.append(row)
        del layers
        torch.cuda.empty_cache()
    return rows


def batch_rows(aq, torch, cases=None):
    """11008x4096 1x16, 4x8, 2x12 and 2x16 with n activation rows (the small-batch
    and prefill path), plus dequantization of the same layers.  ``cases``, a
    list of (M, B, n), restricts the run to those products (no
    dequantization)."""
    rows = []
    for M, B in ((1, 16), (4, 8), (2, 12), (2, 16)):
        ns = (1, 4, 16, 256, 2048) if cases is None else sorted({c[2] for c in cases if c[:2] == (M, B)})
        for n in ns:
            from paper_2401_06118_amd import format as fmt
            shp = fmt.AqlmShape(11008, 4096, M, B)
            name = f"11008x4096 {M}x{B}"
            if cases is None or (M, B, n) in cases:
                reps = 1 if n >= 256 else max(2, (1 << 30) // shp.codes_bytes() + 1)
                layers = [DeviceLayer(800000 + 7 * i + n, 11008, 4096, M, B, n=n) for i in range(reps)]
                g = graph_of([lambda L=L: L.gemm(aq) for L in layers])
                ms = time_steps(g.replay, steps=max(3, 8 // reps), warmup=1) / reps
                del g
                b = shp.gemv_bytes(n)
                rows.append({"layer": name, "n": n, "us": ms * 1e3,
                             "GBs": b / (ms * 1e6), "TFLOPs": shp.flops(n) / (ms * 1e9),
                             "mfma_frac": shp.flops(n) / (ms * 1e9) / MFMA_F16_PEAK_TFS})
                if B == 8 and n <= 16:
                    # the same products over tiled codes (aqlm_gemm_small_batch_tiled)
                    ref = [L.y.clone() for L in layers]
                    tl = [aq.TiledCodes(L.codes, L.codebooks, L.scales) for L in layers]
                    g = graph_of([lambda L=L, t=t: t.gemm_small_batch(L.x, out=L.y) for L, t in zip(layers, tl)])
                    ms = time_steps(g.replay, steps=max(3, 8 // reps), warmup=1) / reps
                    del g
                    same = all(torch.equal(r.view(torch.int16), L.y.view(torch.int16)) for r, L in zip(ref, layers))
                    rows.append({"layer": name, "n": n, "op": "tiled codes", "us": ms * 1e3,
                                 "GBs": b / (ms * 1e6), "bit_identical_to_row_major": same})
                    del ref, tl
                del layers
                torch.cuda.empty_cache()
            # the workspace path (aqlm_gemm: dequantize once, dense fp16 product)
            if n >= 256 and (cases is None or (M, B, n, 1) in cases):
                L = DeviceLayer(800000 + n, 11008, 4096, M, B, n=n)
                need = aq.gemm_workspace_bytes(L.codes, L.codebooks, L.scales, n)
                ws = torch.empty((need,), dtype=torch.uint8, device="cuda")
                g = graph_of([lambda: L.gemm_ws(aq, ws)])
                ms = time_steps(g.replay, steps=8, warmup=1)
                del g
                rows.append({"layer": name, "n": n, "op": "gemm with workspace", "us": ms * 1e3,
                             "TFLOPs": shp.flops(n) / (ms * 1e9),
                             "mfma_frac": shp.flops(n) / (ms * 1e9) / MFMA_F16_PEAK_TFS})
                del L, ws
                torch.cuda.empty_cache()
        if cases is not None:
            continue
        L = DeviceLayer(700000 + M, 11008, 4096, M, B)
        w = torch.empty((11008, 4096), dtype=torch.float16, device="cuda")
        ms = time_steps(lambda: aq.dequantize(L.codes, L.codebooks, L.scales, out=w), steps=10, warmup=3)
        rows.append({"layer": f"11008x4096 M={M} B={B}", "op": "dequantize", "us": ms * 1e3,
                     "GBs": L.shape.dequant_bytes() / (ms * 1e6)})
        del w, L
        torch.cuda.empty_cache()
    return rows


def backward_rows(aq, torch):
    """Gradients through Eq. 2 (aqlm_backward) for 2x8 and 4x8 layers of
    Llama-2-7B shapes: the weight-gradient contraction (2 n d_out d_in flops)
    on the matrix cores plus the scatter into the codebook and scale
    gradients."""
    from paper_2401_06118_amd import format as fmt
    rows = []
    for d_out, d_in, M, n in ((11008, 4096, 2, 256), (11008, 4096, 2, 2048), (4096, 11008, 4, 2048)):
        L = DeviceLayer(500000 + n + M, d_out, d_in, M, 8, n=n)
        dy = torch.randn((n, d_out), device="cuda").half()
        dcb = torch.zeros(tuple(L.codebooks.shape), dtype=torch.float32, device="cuda")
        ds = torch.zeros((d_out,), dtype=torch.float32, device="cuda")
        ms = time_steps(lambda: aq.backward(L.codes, L.codebooks, L.scales, L.x, dy, dcodebooks=dcb, dscales=ds),
                        steps=5, warmup=1)
        fl = fmt.AqlmShape(d_out, d_in, M, 8).flops(n)
        rows.append({"layer": f"{d_out}x{d_in} {M}x8", "n": n, "us": ms * 1e3, "TFLOPs": fl / (ms * 1e9),
                     "mfma_frac": fl / (ms * 1e9) / MFMA_F16_PEAK_TFS})
        del L, dy, dcb, ds
        torch.cuda.empty_cache()
    return rows


def beam_rows(aq, torch):
    """Phase-1 beam search (aqlm_beam_search): one sweep over every code
    position of 2x8 layers, H = X X^T from 512 random calibration vectors."""
    rows = []
    for d_out, d_in, M, beam in ((4096, 1024, 2, 4), (4096, 2048, 2, 8)):
        gen = torch.Generator(device="cuda")
        gen.manual_seed(400000 + d_in + beam)
        x = torch.randn((d_in, 512), device="cuda", generator=gen)
        h = (x @ x.T).contiguous()
        w = (torch.randn((d_out, d_in), device="cuda", generator=gen) * 0.05).contiguous()
        L = DeviceLayer(400000 + d_in, d_out, d_in, M, 8)
        codes0 = L.codes.clone()
        ms = []
        for _ in range(2):
            L.codes.copy_(codes0)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            loss = aq.beam_search(w, h, L.codes, L.codebooks, L.scales, beam=beam, sweeps=1)
            torch.cuda.synchronize()
            ms.append((time.perf_counter() - t0) * 1e3)
        steps = d_in // 8 * M
        rows.append({"layer": f"{d_out}x{d_in} {M}x8", "beam": beam, "sweeps": 1, "ms": min(ms),
                     "rows_per_s": d_out / (min(ms) / 1e3),
                     "candidates_per_s": d_out * steps * beam * 256 / (min(ms) / 1e3),
                     "mean_loss": float(loss.mean())})
        del L, x, h, w
        torch.cuda.empty_cache()
    return rows


def kernel_name(M: int, B: int) -> str:
    """Device kernel that serves a batch-1 product of this format."""
    if B == 8 and M in (1, 2, 4):
        return "aqlm::k_gemv_ks"
    if B == 16 and M == 1:
        return "aqlm::k_gemv_mfma"
    return "aqlm::k_gemv"


PATH_CASES = {
    # name: shapes of one grouped launch (2x8)
    "70b gate/up": [(28672, 8192)] * 2,
    "70b down": [(8192, 28672)],
    "70b q/k/v": [(8192, 8192), (1024, 8192), (1024, 8192)],
    "70b o": [(8192, 8192)],
    "7b gate/up": [(11008, 4096)] * 2,
    "65536x8192": [(65536, 8192)],
}


def compare_paths(aq, torch, once=False):
    """Both kernel families on the same launches, and the gather kernel over
    tiled codes: each case's grouped launch rotated over >= 1 GiB of
    independent layers (so HBM is read), timed per launch from a graph of the
    rotation; plus the relative L2 difference of the two families' results
    and whether the tiled product equals the row-major one bit for bit."""
    from paper_2401_06118_amd import format as fmt
    rows = []
    for name, shapes in PATH_CASES.items():
        b = sum(fmt.AqlmShape(o, k, 2, 8).gemv_bytes(1) for o, k in shapes)
        reps = 1 if once else max(2, (1 << 30) // b + 1)
        sets = []
        for r in range(reps):
            ls = [DeviceLayer(600000 + 31 * r + i, o, k, 2, 8) for i, (o, k) in enumerate(shapes)]
            for L in ls[1:]:
                if L.x.shape == ls[0].x.shape:
                    L.x = ls[0].x
            sets.append(ls)
        res = {"launch": name, "shapes": shapes, "bytes": b, "replicas": reps}
        outs = {}
        for path in ("gather", "table"):
            calls = [lambda ls=ls, path=path: aq.gemv_grouped([L.problem() for L in ls], path=path) for ls in sets]
            if once:
                calls[0]()
                torch.cuda.synchronize()
            else:
                g = graph_of(calls)
                us = time_steps(g.replay, steps=5, warmup=1) / reps * 1e3
                del g
                res[f"{path}_us"] = us
                res[f"{path}_GBs"] = b / (us * 1e3)
            outs[path] = [L.y.double().clone() for L in sets[0]]
        res["rel_l2_diff"] = max(float((a - c).norm() / c.norm()) for a, c in zip(outs["table"], outs["gather"]))
        # the gather kernel over tiled codes (same arithmetic: bit-identical)
        tsets = [[aq.TiledCodes(L.codes, L.codebooks, L.scales) for L in ls] for ls in sets]
        calls = [lambda ls=ls, ts=ts: aq.gemv_tiled_grouped([(t, L.x[0], L.y[0]) for t, L in zip(ts, ls)])
                 for ls, ts in zip(sets, tsets)]
        if once:
            calls[0]()
            torch.cuda.synchronize()
        else:
            g = graph_of(calls)
            us = time_steps(g.replay, steps=5, warmup=1) / reps * 1e3
            del g
            res["tiled_us"] = us
            res["tiled_GBs"] = b / (us * 1e3)
        res["tiled_bit_identical"] = all(torch.equal(L.y.double(), r) for L, r in zip(sets[0], outs["gather"]))
        del tsets
        rows.append(res)
        log(f"{name}: " + ", ".join(f"{k} {v:.2f}" for k, v in res.items() if k.endswith("_us")))
        del sets
        torch.cuda.empty_cache()
    return rows


COPY_BYTES = 256 << 20


def copy_calibration():
    """A plain device-to-device copy of known size: it reads and writes
    COPY_BYTES once per launch, so HBM byte counters taken on it give the
    scale between counter readings and bytes moved."""
    import torch
    src = torch.empty(COPY_BYTES, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": COPY_BYTES, "launches": 5}), flush=True)


CLOCK_GHZ = 2.4  # MI355X peak engine clock


def floors(torch):
    """Microbenchmarks of the limits the kernels are measured against
    (paper_2401_06118_amd/floors/floors.hip, a library of its own), each a
    HIP graph of back-to-back launches timed with an event pair; per-clock
    figures assume the 2.4 GHz peak clock."""
    import ctypes
    lib = ctypes.CDLL(os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2401_06118_amd",
                                   "libaqlm_floors.so"))
    vp, ci, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
    lib.floor_empty.argtypes = [ci, vp]
    lib.floor_dep_load.argtypes = [vp, vp, ci, vp]
    lib.floor_read.argtypes = [vp, sz, vp, ci, vp]
    lib.floor_mfma.argtypes = [vp, ci, ci, vp]
    lib.floor_lds_gather.argtypes = [vp, ci, ci, ci, vp]
    lib.floor_l2_gather.argtypes = [vp, ctypes.c_uint32, vp, ci, ci, vp]
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    stream = lambda: torch.cuda.current_stream().cuda_stream  # noqa: E731

    def ok(st):
        if st != 0:
            raise RuntimeError(f"floor launch failed: hipError {st}")

    def graph_launch_ms(call, reps, steps=5):
        g = graph_of([call] * reps)
        ms = time_steps(g.replay, steps=steps, warmup=2) / reps
        del g
        return ms

    rows = []
    ms = graph_launch_ms(lambda: ok(lib.floor_empty(cus, stream())), 200)
    rows.append({"floor": "empty launch", "workgroups": cus, "threads": 1024, "us": ms * 1e3})
    src = torch.ones(cus * 64, dtype=torch.int32, device="cuda")
    dst = torch.empty(cus * 1024, dtype=torch.int32, device="cuda")
    ms = graph_launch_ms(lambda: ok(lib.floor_dep_load(src.data_ptr(), dst.data_ptr(), cus, stream())), 200)
    rows.append({"floor": "one dependent load (line in L2), barrier, store", "workgroups": cus, "threads": 1024,
                 "us": ms * 1e3})
    del src, dst
    buf = torch.ones(1 << 30, dtype=torch.uint8, device="cuda")
    out = torch.empty(cus * 16 * 256, dtype=torch.int32, device="cuda")
    ms = graph_launch_ms(lambda: ok(lib.floor_read(buf.data_ptr(), (1 << 30) // 16, out.data_ptr(), cus * 16,
                                                 stream())), 10)
    rows.append({"floor": "HBM read stream, 1 GiB", "GBs": (1 << 30) / (ms * 1e6)})
    del buf, out
    iters = 2000
    out = torch.empty(cus * 4 * 256, dtype=torch.float32, device="cuda")
    ms = graph_launch_ms(lambda: ok(lib.floor_mfma(out.data_ptr(), cus * 4, iters, stream())), 3)
    mfmas = cus * 4 * 4 * iters * 8
    rows.append({"floor": "v_mfma_f32_16x16x32_f16, 4 waves per SIMD, 8 chains each",
                 "clocks_per_mfma_per_simd": ms * 1e-3 * CLOCK_GHZ * 1e9 * cus * 4 / mfmas,
                 "TFLOPs": mfmas * 16 * 16 * 32 * 2 / (ms * 1e9)})
    del out
    out = torch.empty(cus * 1024, dtype=torch.int32, device="cuda")
    for copies in (1, 8, 16):
        iters = 500
        ms = graph_launch_ms(lambda: ok(lib.floor_lds_gather(out.data_ptr(), cus, iters, copies, stream())), 3)
        nbytes = cus * 1024 * iters * 8 * 16
        rows.append({"floor": f"LDS 16-byte gathers, {copies} table copies", "bytes_per_clock_per_cu":
                     nbytes / (ms * 1e-3 * CLOCK_GHZ * 1e9 * cus)})
    tab = torch.ones(1 << 20, dtype=torch.uint8, device="cuda")
    iters = 50
    ms = graph_launch_ms(lambda: ok(lib.floor_l2_gather(tab.data_ptr(), (1 << 20) // 16, out.data_ptr(), cus, iters,
                                                      stream())), 3)
    rows.append({"floor": "16-byte gathers from a 1 MiB table in L2", "gathers_per_clock_per_cu":
                 cus * 1024 * iters * 8 / (ms * 1e-3 * CLOCK_GHZ * 1e9 * cus)})
    return rows


def decode_step(model, M, B, seed0, aq, steps, warmup, markers=False, spread_steps=20, tiled=False):
    """Build a decode step, capture it as one graph and time its replays.
    tiled: the codes are also stored tiled (aqlm_tile_codes, before anything
    is timed) and the step runs over those."""
    layers = decode_step_layers(model, M, B, seed0)
    step_bytes = sum(L.shape.gemv_bytes(1) for L in layers)
    log(f"{model} {M}x{B}: {len(layers)} layers built")
    if tiled:
        tl = [aq.TiledCodes(L.codes, L.codebooks, L.scales) for L in layers]
        launches = launches_tiled(layers, tl, aq)
    else:
        launches = launches_by_dependency(layers, aq)
    graph = graph_of(launches)
    log(f"{model} {M}x{B}: graph captured")
    ms = time_steps(graph.replay, steps, warmup, markers=markers)
    spread = step_spread(graph.replay, max(1, spread_steps))
    return layers, launches, graph, ms, spread, step_bytes


def persistent_step_row(layers, graph, aq, torch, steps, step_bytes, graph_ms):
    """The same decode step as one persistent launch (aqlm_gemv_step): the
    block's four dependency levels, one level barrier each, timed like the
    graph; its outputs are compared bit for bit with the graph's."""
    levels = []
    for b in range(0, len(layers), 7):
        q, k, v, o, gate, up, down = layers[b:b + 7]
        levels += [[q.problem(), k.problem(), v.problem()], [o.problem()], [gate.problem(), up.problem()],
                   [down.problem()]]
    step = aq.DecodeStep(levels)
    step.run()
    step.status()
    ys = [L.y.clone() for L in layers]
    graph.replay()
    torch.cuda.synchronize()
    same = all(torch.equal(a.view(torch.int16), L.y.view(torch.int16)) for a, L in zip(ys, layers))
    del ys
    ms = time_steps(step.run, steps, 2)
    step.status()
    return {"ms_per_step": ms, "GBs": step_bytes / (ms * 1e6), "frac": step_bytes / (ms * 1e6) / HBM_PEAK_GBS,
            "levels": len(levels), "launches": 1, "vs_graph": graph_ms / ms, "bit_identical_to_graph": same}


def sorted_step_row(layers, aq, torch, steps, step_bytes, graph_ms, markers=False):
    """The 1x16 decode step over chunk-sorted codes (aqlm_gemv_sorted):
    grouped q/k/v, o, grouped gate/up, down, as one graph; outputs compared
    with the row-major graph's (relative L2)."""
    import time
    t0 = time.time()
    srt = [aq.SortedCodes(L.codes, L.codebooks, L.scales) for L in layers]
    sort_s = time.time() - t0
    entry_bytes = sum(s.entries.numel() * 4 + s.index.numel() * 4 for s in srt)
    rows = max(sum(L.shape.d_out for L in layers[b:b + 3]) for b in range(0, len(layers), 7))
    rows = max(rows, max(sum(L.shape.d_out for L in layers[b + 4:b + 6]) for b in range(0, len(layers), 7)))
    ws = torch.zeros((aq._lib.load().aqlm_gemv_sorted_workspace_bytes(rows, 1, 16),), dtype=torch.uint8,
                     device="cuda")
    ref = [L.y.clone() for L in layers]
    launches = []
    for b in range(0, len(layers), 7):
        q, k, v, o, gate, up, down = [(srt[b + i], layers[b + i]) for i in range(7)]
        grp = lambda items: (lambda: aq.gemv_sorted_grouped([(s, L.x[0], L.y[0]) for s, L in items], workspace=ws))
        launches += [grp([q, k, v]), grp([o]), grp([gate, up]), grp([down])]
    g = graph_of(launches)
    g.replay()
    torch.cuda.synchronize()
    err = max(float(torch.linalg.norm((L.y.float() - r.float())) / max(float(torch.linalg.norm(r.float())), 1e-30))
              for L, r in zip(layers, ref))
    ms = time_steps(g.replay, steps, 2, markers=markers)
    del g, srt, ref
    return {"ms_per_step": ms, "GBs": step_bytes / (ms * 1e6), "frac": step_bytes / (ms * 1e6) / HBM_PEAK_GBS,
            "tok_s_eq": 1000.0 / ms, "launches": len(launches), "vs_row_major_graph": graph_ms / ms,
            "sorted_bytes_per_step": entry_bytes, "GBs_sorted_bytes": entry_bytes / (ms * 1e6),
            "host_sort_s": sort_s, "max_rel_l2_vs_row_major": err}


def row_major_step_row(layers, graph, aq, torch, steps, step_bytes, graph_ms):
    """The decode step over the row-major codes (aqlm_gemv_grouped /
    aqlm_gemv), timed like the tiled graph `graph`; outputs compared bit for
    bit with that graph's."""
    graph.replay()
    torch.cuda.synchronize()
    ref = [L.y.clone() for L in layers]
    g = graph_of(launches_by_dependency(layers, aq))
    g.replay()
    torch.cuda.synchronize()
    same = all(torch.equal(a.view(torch.int16), L.y.view(torch.int16)) for a, L in zip(ref, layers))
    del ref
    ms = time_steps(g.replay, steps, 2)
    del g
    return {"ms_per_step": ms, "GBs": step_bytes / (ms * 1e6), "frac": step_bytes / (ms * 1e6) / HBM_PEAK_GBS,
            "tiled_speedup": ms / graph_ms, "bit_identical_to_tiled": same}


def tiled_step_row(layers, aq, torch, steps, step_bytes, graph_ms, markers=False):
    """The decode step over tiled codes (aqlm_tile_codes once per layer, then
    aqlm_gemv_grouped_tiled): grouped q/k/v, o, grouped gate/up, down, as one
    graph; outputs compared bit for bit with the row-major graph's (which
    the caller has just replayed)."""
    import time
    t0 = time.time()
    tl = [aq.TiledCodes(L.codes, L.codebooks, L.scales) for L in layers]
    torch.cuda.synchronize()
    tile_s = time.time() - t0
    ys = [torch.empty_like(L.y[0]) for L in layers]
    launches = []
    for b in range(0, len(layers), 7):
        grp = lambda idx: (lambda: aq.gemv_tiled_grouped([(tl[i], layers[i].x[0], ys[i]) for i in idx]))
        launches += [grp([b, b + 1, b + 2]), grp([b + 3]), grp([b + 4, b + 5]), grp([b + 6])]
    g = graph_of(launches)
    g.replay()
    torch.cuda.synchronize()
    same = all(torch.equal(y.view(torch.int16), L.y[0].view(torch.int16)) for y, L in zip(ys, layers))
    ms = time_steps(g.replay, steps, 2, markers=markers)
    del g, tl, ys
    return {"ms_per_step": ms, "GBs": step_bytes / (ms * 1e6), "frac": step_bytes / (ms * 1e6) / HBM_PEAK_GBS,
            "tok_s_eq": 1000.0 / ms, "launches": len(launches), "vs_row_major_graph": graph_ms / ms,
            "bit_identical_to_row_major": same, "tile_s": tile_s}


def step_seed(M: int) -> int:
    return 1000 * (1 if M == 2 else 2)


def main():
    args = parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU only; --gpus {args.gpus} is not supported "
              "(no multi-GPU path exists).", file=sys.stderr)
        sys.exit(2)
    if args.summarize_trace:
        print(json.dumps(summarize_trace(args.summarize_trace)), flush=True)
        return
    if args.copy_calibration:
        copy_calibration()
        return
    import torch
    if args.floors:
        print(json.dumps({"floors": floors(torch)}), flush=True)
        return
    import paper_2401_06118_amd as aq
    from paper_2401_06118_amd import _lib

    _lib.load()  # fail loudly if the HIP library is missing
    if args.backward:
        print(json.dumps({"backward": backward_rows(aq, torch)}), flush=True)
        return
    if args.beam_search:
        print(json.dumps({"beam_search": beam_rows(aq, torch)}), flush=True)
        return
    if args.single_layers:
        print(json.dumps({"single_layers": single_layer_rows(aq, torch)}), flush=True)
        return
    if args.compare_paths:
        print(json.dumps({"paths": compare_paths(aq, torch, once=args.once)}), flush=True)
        return
    if args.batch_case:
        cases = [tuple(int(v) for v in c.split(",")) for c in args.batch_case]
        print(json.dumps({"batch": batch_rows(aq, torch, cases)}), flush=True)
        return

    model, M, B = WORKLOADS[args.workload]
    if args.persistent:
        layers, launches, graph, ms, spread, step_bytes = decode_step(model, M, B, step_seed(M), aq, args.steps,
                                                                      args.warmup)
        row = persistent_step_row(layers, graph, aq, torch, args.steps, step_bytes, ms)
        print(json.dumps({"workload": args.workload, "graph_ms_per_step": ms, "persistent_step": row}), flush=True)
        return
    if args.tiled:
        if B != 8:
            sys.exit("bench.py: --tiled needs a workload with 8-bit codes")
        layers, launches, graph, ms, spread, step_bytes = decode_step(model, M, B, step_seed(M), aq, args.steps,
                                                                      args.warmup)
        graph.replay()
        torch.cuda.synchronize()
        row = tiled_step_row(layers, aq, torch, args.steps, step_bytes, ms, markers=True)
        print(json.dumps({"workload": args.workload, "graph_ms_per_step": ms, "tiled_codes": row}), flush=True)
        return
    if args.sorted:
        if B < 15:
            sys.exit("bench.py: --sorted needs a workload with 15- or 16-bit codes (llama2-7b-1x16)")
        layers, launches, graph, ms, spread, step_bytes = decode_step(model, M, B, step_seed(M), aq, args.steps,
                                                                      args.warmup)
        row = sorted_step_row(layers, aq, torch, args.steps, step_bytes, ms, markers=True)
        print(json.dumps({"workload": args.workload, "graph_ms_per_step": ms, "sorted_codes": row}), flush=True)
        return
    tiled = B == 8  # (8-bit codes: the step reads tiled codes)
    layers, launches, graph, ms, spread, step_bytes = decode_step(
        model, M, B, step_seed(M), aq, args.steps, args.warmup, markers=True, spread_steps=args.spread_steps,
        tiled=tiled)
    log(f"{args.workload}: {len(layers)} layers in {len(launches)} launches, {step_bytes / 1e9:.3f} GB per step; "
        f"step {ms:.4f} ms (graph replay)")

    # Dominant kernel: every launch of the step is the matrix-vector kernel
    # (grouped or single).  Its average launch duration is measured live: HIP
    # events on the launch stream around the timed graph replays, divided by
    # the launches (gaps between kernels included).  The committed kernel
    # trace of this command (same kernel source) is reported beside it: its
    # per-kernel average, and what share of its own run's step the kernels
    # filled, which bounds how much of the live figure is gaps.  Boxes differ
    # by several per cent, so the two agree only when taken on the same box.
    bytes_per_launch = step_bytes / len(launches)
    avg_us = ms * 1e3 / len(launches)
    digest = source_digest("gemv_mfma.hip", "stream_common.h", "common.h", "launch.h")
    kname = kernel_name(M, B)
    key = f"{kname}:{args.workload}"
    traced = traced_duration(key, digest)
    trace = None
    if traced is not None:
        trace = {"avg_launch_us": traced[0], "dispatches_per_step": traced[1],
                 "kernel_ms_per_step": traced[0] * traced[1] / 1e3, "traced_run_ms_per_step": traced[2],
                 "kernel_share_of_step": traced[0] * traced[1] / 1e3 / traced[2],
                 "frac": bytes_per_launch / (traced[0] * 1e3) / HBM_PEAK_GBS,
                 "source": "rocprofv3 kernel trace of this command over the timed graph replays "
                           "(profiles/kernel_durations.txt)"}
    achieved = bytes_per_launch / (avg_us * 1e3)
    traffic = measured_traffic(key, digest)

    result = {
        "metric": "achieved HBM GB/s & roofline % for AQLM GEMV (batch 1); decode tokens/s-equivalent",
        "value": step_bytes / (ms * 1e6),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16 (fp32 accumulate)",
        "data": "synthetic: uniform codes, N(0,0.02) fp16 codebooks, U[0.5,1.5] fp16 scales, N(0,1) fp16 x",
        "config": {
            "workload": f"Llama-2-{model.upper()} decode step on one GPU, linear layers only, AQLM {M}x{B} "
                        f"g8, batch 1: {len(layers)} GEMVs in {len(launches)} launches (per block: grouped "
                        f"q/k/v, o, grouped gate/up, down), replayed as one HIP graph"
                        + (", codes stored tiled (1 KiB tiles of 16 rows x 64 code bytes, written before "
                           "timing)" if tiled else ""),
            "code_layout": "tiled" if tiled else "row-major",
            "layers": len(layers),
            "launches": len(launches),
            "bytes_per_step": step_bytes,
            "parallelism": "single GPU",
        },
        "ms_per_step_spread": spread,
        "tokens_per_s_equivalent": 1000.0 / ms,
        "roofline_frac_step": step_bytes / (ms * 1e6) / HBM_PEAK_GBS,
        "roofline": {
            "bound": "hbm",
            "kernel": kname,
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS,
            "traffic": traffic,
            "bytes_per_launch": bytes_per_launch,
            "avg_launch_us": avg_us,
            "duration_source": "HIP events around the timed graph replays on the launch stream / launches",
            "trace": trace,
            "source_digest": digest,
        },
    }
    persistent = row_major = None
    if not args.no_secondary:
        persistent = persistent_step_row(layers, graph, aq, torch, max(5, args.steps // 2), step_bytes, ms)
        log(f"{args.workload} as one persistent launch: {persistent['ms_per_step']:.4f} ms per step")
        if tiled:
            row_major = row_major_step_row(layers, graph, aq, torch, max(5, args.steps // 2), step_bytes, ms)
            log(f"{args.workload} over row-major codes: {row_major['ms_per_step']:.4f} ms per step")
    del layers, launches, graph
    torch.cuda.empty_cache()

    if not args.no_secondary:
        sec = {"persistent_step": persistent, "row_major_codes": row_major}
        for other in ("llama2-7b-2x8", "llama2-7b-1x16"):
            if other == args.workload:
                continue
            om, oM, oB = WORKLOADS[other]
            ol, olaunch, og, oms, osp, ob = decode_step(om, oM, oB, step_seed(oM) + 4000, aq,
                                                        max(5, args.steps // 2), 2)
            pair = per_launch_ms(olaunch, reps=2)
            row = {"ms_per_step": oms, "GBs": ob / (oms * 1e6), "frac": ob / (oms * 1e6) / HBM_PEAK_GBS,
                   "tok_s_eq": 1000.0 / oms, "spread": osp, "event_pair_sum_ms": sum(pair),
                   "GBs_event_pair": ob / (sum(pair) * 1e6)}
            if oM == 2:
                row["persistent_step"] = persistent_step_row(ol, og, aq, torch, max(5, args.steps // 2), ob, oms)
                og.replay()
                torch.cuda.synchronize()
                row["tiled_codes"] = tiled_step_row(ol, aq, torch, max(5, args.steps // 2), ob, oms)
                # the same step without grouping (224 single launches), and
                # without the block's dependencies (8 independent GEMVs per launch)
                g1 = graph_of([lambda L=L: L.gemv(aq) for L in ol])
                ms1 = time_steps(g1.replay, args.steps, 2)
                fused = [lambda c=ol[i:i + 8]: aq.gemv_grouped([L.problem() for L in c]) for i in range(0, len(ol), 8)]
                g8 = graph_of(fused)
                ms8 = time_steps(g8.replay, args.steps, 2)
                row["ungrouped_224_launches"] = {"ms_per_step": ms1, "GBs": ob / (ms1 * 1e6)}
                row["independent_8_per_launch"] = {"launches": len(fused), "ms_per_step": ms8,
                                                   "GBs": ob / (ms8 * 1e6)}
                del g1, g8
            if oM == 1:
                row["sorted_codes"] = sorted_step_row(ol, aq, torch, max(5, args.steps // 2), ob, oms)
                log(f"{other} over sorted codes: {row['sorted_codes']['ms_per_step']:.4f} ms per step")
            sec[other] = row
            del ol, olaunch, og
            torch.cuda.empty_cache()
            log(f"{other}: {oms:.4f} ms per step")
        sec["single_layers"] = single_layer_rows(aq, torch)
        log("single layers done")
        sec["batch"] = batch_rows(aq, torch)
        log("batch / dequantize done")
        sec["backward"] = backward_rows(aq, torch)
        log("backward done")
        sec["beam_search"] = beam_rows(aq, torch)
        log("beam search done")
        sec["floors"] = floors(torch)
        log("floors done")
        result["secondary"] = sec
    if not args.no_cpu_baseline:
        layers = decode_step_layers(model, M, B, step_seed(M))
        log("cpu baseline (oracle) ...")
        result["cpu_baseline"] = cpu_baseline(layers, args.cpu_seconds)
        del layers
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
