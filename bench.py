"""Benchmark of the CompressKV prefill-end KV eviction path on one MI355X.

One step = the whole path (score, select, gather) over every layer of the
workload, with all inputs already resident in HBM. By default one
ckv_compress_stack call runs all layers on one stream: the two K passes of
every layer, then the pooling, selection and gather of all layers in two or
three launches; a second leg ("side_stream_variant") times the same call with
a side stream on which every other layer's K passes run. --schedule layers issues one
ckv_compress_layer per layer instead; --pipeline runs ckv_score (both K passes
and the pooling) of layer l+1 on one stream while ckv_select and ckv_gather of
layer l run on another. Prints one JSON line.

  python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]

The metric is prompt tokens compressed per second per layer:
  value = sum_prompts(L) * n_layers / step_time.
The roofline object covers the dominant kernel, timed with HIP events recorded
around each of its launches inside the timed region (on the launch stream).
"""
from __future__ import annotations

import argparse
import ctypes
import gc
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0   # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    # a few warm-up steps: the first ones after the layers are drawn run slower
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--workload", default="llama8b-128k-stack")
    p.add_argument("--layers", type=int, default=0, help="limit the layer count (0 = all)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-profile-variant", action="store_true",
                   help="skip the timing of the layer-error profile (decode attention over the "
                        "full and the compact cache, W_O projection)")
    p.add_argument("--no-decode-variant", action="store_true",
                   help="skip the timing of one decoding step over the full and the compact caches")
    p.add_argument("--no-lse-variant", action="store_true",
                   help="skip the second measurement, with the window rows' log-sum-exp supplied "
                        "by the caller (one pass over K)")
    p.add_argument("--cpu-threads", type=int, default=0,
                   help="oracle threads for cpu_baseline (0 = the usable CPUs, at most 16)")
    p.add_argument("--cpu-seconds", type=float, default=15.0,
                   help="wall time the cpu_baseline sample aims for")
    p.add_argument("--no-side-variant", action="store_true",
                   help="skip the leg that times the stack with a side stream")
    p.add_argument("--no-stream-ceiling", action="store_true",
                   help="skip the streaming-read ceiling probe (bench_stream.so)")
    p.add_argument("--stream-ceiling-only", action="store_true",
                   help="run only the streaming-read ceiling probe and print its JSON")
    p.add_argument("--configs", default="llama8b-32k-layer,llama8b-32k-stack,qwen7b-ragged-batch",
                   help="other workloads measured after the headline one, comma-separated "
                        "('' for none); each gets its own step time and roofline")
    p.add_argument("--time-every", type=int, default=32, metavar="N",
                   help="K-pass launches of every N-th layer carry start/end events (the layer "
                        "offset rotates with the step, so every layer is sampled); each timed "
                        "launch delays its neighbours' dispatch by 5-9 microseconds, so the "
                        "default samples one layer per step of 32 layers")
    p.add_argument("--stack-slots", type=int, default=0,
                   help="--schedule stack: layer slots of workspace (0 = one per layer); the "
                        "selection stages run in launches covering that many layers")
    p.add_argument("--stack-side", type=int, default=0,
                   help="--schedule stack: 1 gives ckv_compress_stack a side stream, on which "
                        "every other layer's K passes run (two launches in flight, so each "
                        "launch's own duration includes the other's share of HBM); 0 (default) "
                        "runs them all on one stream, and a second leg times the side-stream "
                        "schedule")
    p.add_argument("--schedule", choices=("stack", "layers"), default="stack",
                   help="stack: one ckv_compress_stack call over all layers (default); "
                        "layers: one ckv_compress_layer per layer (see --streams)")
    p.add_argument("--streams", type=int, default=1,
                   help="--schedule layers: layers are issued round-robin on this many streams "
                        "(one workspace each); launches then overlap and per-launch times include it")
    p.add_argument("--scope", choices=("group", "shared"), default="group",
                   help="group: the workload's per-group head mask (default); shared: the "
                        "paper's layer-shared selection with 4 retrieval heads per layer")
    p.add_argument("--pipeline", action="store_true",
                   help="two-stream pipeline (ckv_score of layer l+1 beside ckv_select and "
                        "ckv_gather of layer l) instead of one ckv_compress_layer per layer")
    p.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                   help="first run an elementwise kernel that reads and writes MIB MiB (the "
                        "reference for scaling FETCH_SIZE / WRITE_SIZE counters)")
    p.add_argument("--summarize-trace", metavar="DIR",
                   help="print a markdown summary of a rocprofv3 --kernel-trace --stats "
                        "output directory and exit (no GPU needed)")
    p.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                   help="print the calibrated per-launch HBM traffic from two rocprofv3 --pmc "
                        "runs (FETCH_SIZE, WRITE_SIZE) and exit (no GPU needed)")
    p.add_argument("--summarize-counters", nargs="+", metavar="DIR",
                   help="print per-kernel SQ counters (mean per dispatch) and the MFMA busy "
                        "fraction from rocprofv3 --pmc output directories and exit (no GPU "
                        "needed)")
    p.add_argument("--copy-mib", type=int, default=1024,
                   help="size the calibration copy used, for --summarize-pmc")
    return p.parse_args()


class Hip:
    """Raw HIP events through the runtime library (torch events only see torch's stream)."""

    def __init__(self):
        self.lib = ctypes.CDLL("libamdhip64.so")
        self.lib.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.lib.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.free = []  # events handed back by destroy(), reused by event()

    def event(self):
        if self.free:
            return self.free.pop()
        e = ctypes.c_void_p()
        rc = self.lib.hipEventCreate(ctypes.byref(e))
        if rc != 0:
            raise RuntimeError("hipEventCreate failed: %d" % rc)
        return e.value

    def elapsed_ms(self, a, b) -> float:
        out = ctypes.c_float()
        rc = self.lib.hipEventElapsedTime(ctypes.byref(out), a, b)
        if rc != 0:
            raise RuntimeError("hipEventElapsedTime failed: %d" % rc)
        return out.value

    def destroy(self, e):
        # kept for reuse: creating and destroying hundreds of events per
        # measurement left later measurements' launches slow to submit
        self.free.append(e)


KERNEL_SOURCES = ("paper_2508_02401_amd/csrc/ckv_score.hip", "paper_2508_02401_amd/csrc/ckv_select.hip",
                  "paper_2508_02401_amd/csrc/ckv_device.h", "paper_2508_02401_amd/csrc/ckv_internal.h",
                  "paper_2508_02401_amd/build.py")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic_llama8b-128k-stack.md")


def kernel_source_hash() -> str:
    import hashlib
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def committed_traffic(kernel: str):
    """Counter-measured HBM bytes per launch of `kernel` from the committed
    summary, or None when there is none or the kernel sources changed since."""
    try:
        with open(TRAFFIC_FILE) as f:
            text = f.read()
    except OSError:
        return None
    start = text.find("```json")
    if start < 0:
        return None
    end = text.find("```", start + 7)
    try:
        data = json.loads(text[start + 7:end])
    except ValueError:
        return None
    if data.get("source_sha256") != kernel_source_hash():
        return None
    entry = data.get("kernels", {}).get(kernel)
    return None if entry is None else float(entry["traffic_bytes_per_launch"])


def _kernel_short(name: str) -> str:
    import re
    m = re.search(r"ckv::\(anonymous namespace\)::(\w+)", name)
    if m:
        return m.group(1)
    if "neg_kernel" in name:
        return "calibration_copy(neg)"
    if "stream_copy_kernel" in name:
        return "stream_copy_kernel"
    m = re.search(r"stream_read_kernel<(\d+)>", name)
    if m:
        return "stream_read_kernel<%s> (%s)" % (m.group(1), STREAM_KINDS[int(m.group(1))])
    return name[:60]


def summarize_trace(d: str) -> None:
    import csv
    import glob
    stats = glob.glob(os.path.join(d, "**", "*kernel_stats.csv"), recursive=True)
    if not stats:
        raise SystemExit("no kernel_stats.csv under " + d)
    rows = list(csv.DictReader(open(stats[0])))
    # this library's kernels (the torch kernels are the input draws, outside
    # the timed region)
    rows = [r for r in rows if "ckv::" in r["Name"] or "stream_" in r["Name"]]
    print("| kernel | calls | total ms | avg us | min us | max us | % of all GPU time |")
    print("|---|---|---|---|---|---|---|")
    for r in rows:
        print("| %s | %s | %.3f | %.2f | %.2f | %.2f | %.2f |" % (
            _kernel_short(r["Name"]), r["Calls"], float(r["TotalDurationNs"]) / 1e6,
            float(r["AverageNs"]) / 1e3, float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3,
            float(r["Percentage"])))


def _pmc_means(d: str, counter: str):
    import csv
    import glob
    import collections
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit("no counter_collection.csv under " + d)
    vals = collections.defaultdict(list)
    for r in csv.DictReader(open(files[0])):
        if r["Counter_Name"] == counter:
            vals[_kernel_short(r["Kernel_Name"])].append(float(r["Counter_Value"]))
    return {k: (sum(v) / len(v), len(v)) for k, v in vals.items()}


def summarize_pmc(fetch_dir: str, write_dir: str, copy_mib: int) -> None:
    fetch = _pmc_means(fetch_dir, "FETCH_SIZE")
    write = _pmc_means(write_dir, "WRITE_SIZE")
    copy_bytes = copy_mib * 1024 * 1024
    cal = "calibration_copy(neg)"
    if cal not in fetch or cal not in write:
        raise SystemExit("the calibration copy kernel is missing from the counter runs")
    # counters are in KiB per dispatch; scale so that the copy reads and
    # writes exactly copy_bytes
    f_scale = copy_bytes / (fetch[cal][0] * 1024.0)
    w_scale = copy_bytes / (write[cal][0] * 1024.0)
    print("calibration: elementwise copy of %d MiB read %.1f KiB and wrote %.1f KiB per dispatch"
          % (copy_mib, fetch[cal][0], write[cal][0]))
    print("scale factors: FETCH_SIZE x %.4f, WRITE_SIZE x %.4f" % (f_scale, w_scale))
    print()
    print("| kernel | dispatches | FETCH_SIZE KiB | WRITE_SIZE KiB | calibrated HBM MB per launch |")
    print("|---|---|---|---|---|")
    out = {}
    for k in sorted(fetch):
        if k == cal or k not in write or not k.endswith("_kernel"):
            continue  # only this library's kernels
        t = fetch[k][0] * 1024.0 * f_scale + write[k][0] * 1024.0 * w_scale
        out[k] = {"fetch_kib": fetch[k][0], "write_kib": write[k][0],
                  "traffic_bytes_per_launch": t}
        print("| %s | %d | %.1f | %.1f | %.2f |" % (k, fetch[k][1], fetch[k][0], write[k][0], t / 1e6))
    print()
    print("```json")
    print(json.dumps({"source_sha256": kernel_source_hash(), "fetch_scale": f_scale,
                      "write_scale": w_scale, "kernels": out}, indent=1))
    print("```")


# MI355X: 256 CUs of 4 SIMDs each, in 8 XCDs of 4 shader engines (SQ cycle
# counters are summed over the shader engines, busy-cycle counters over SIMDs)
N_SIMD = 1024
N_SE = 32


def summarize_counters(dirs) -> None:
    """Per-kernel SQ counters (mean per dispatch) from rocprofv3 --pmc runs,
    with the MFMA pipe's busy fraction: busy SIMD-cycles over SIMDs x the
    dispatch's cycles (SQ_CYCLES / shader engines)."""
    import csv
    import glob
    import collections
    vals = collections.defaultdict(lambda: collections.defaultdict(list))
    for d in dirs:
        files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
        if not files:
            raise SystemExit("no counter_collection.csv under " + d)
        for r in csv.DictReader(open(files[0])):
            k = _kernel_short(r["Kernel_Name"])
            if k.endswith("_kernel"):
                vals[k][r["Counter_Name"]].append(float(r["Counter_Value"]))
    names = sorted({c for v in vals.values() for c in v})
    ks = sorted(vals)
    mean = {k: {c: sum(v) / len(v) for c, v in vals[k].items()} for k in ks}
    print("| counter (mean per dispatch) | " + " | ".join(ks) + " |")
    print("|---|" + "---|" * len(ks))
    for c in names:
        print("| %s | " % c + " | ".join("%.4g" % mean[k][c] if c in mean[k] else "—"
                                       for k in ks) + " |")
    busy, per = [], []
    for k in ks:
        m = mean[k]
        b = m.get("SQ_VALU_MFMA_BUSY_CYCLES")
        busy.append("%.1f%%" % (100.0 * b / (N_SIMD * m["SQ_CYCLES"] / N_SE))
                    if b is not None and m.get("SQ_CYCLES") else "—")
        per.append("%.1f" % (b / m["SQ_INSTS_MFMA"]) if b is not None and m.get("SQ_INSTS_MFMA")
                   else "—")
    print("| MFMA pipe busy (of SIMD-cycles) | " + " | ".join(busy) + " |")
    print("| busy cycles per MFMA | " + " | ".join(per) + " |")


STREAM_SRC = os.path.join(ROOT, "bench_stream.hip")
STREAM_LIB = os.path.join(ROOT, "bench_stream.so")
STREAM_KINDS = {0: "global_load_dwordx4", 1: "global_load_dwordx4 nontemporal",
                2: "global_load_lds_dwordx4 (the K passes' route)"}


def build_stream_probe() -> str:
    """Compile bench_stream.hip (the streaming-read ceiling probe) in-tree."""
    import subprocess
    from paper_2508_02401_amd import build as B
    tmp = STREAM_LIB + ".tmp%d" % os.getpid()
    subprocess.run([B.HIPCC, "-x", "hip"] + B.COMMON + ["-shared", STREAM_SRC, "-o", tmp],
                   check=True)
    os.replace(tmp, STREAM_LIB)
    return STREAM_LIB


def stream_ceiling(dev, reps: int = 4, gib: int = 2, hot_mib: int = 128):
    """Streaming-read rate of the GPU with each read route of bench_stream.so:
    a cold sweep of a `gib` GiB buffer (8x the Infinity Cache, so nearly every
    byte comes from HBM) at several grid sizes, and a hot re-read of `hot_mib`
    MiB that the previous sweep left in the Infinity Cache. Times from events
    around each launch on torch's current stream (the probe launches there)."""
    import torch

    if not os.path.exists(STREAM_LIB):
        raise RuntimeError("bench_stream.so is not built; run __graft_entry__.build()")
    lib = ctypes.CDLL(STREAM_LIB)
    lib.bench_stream_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p,
                                      ctypes.c_int, ctypes.c_int, ctypes.c_void_p]
    lib.bench_stream_read.restype = ctypes.c_int
    lib.bench_stream_copy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                      ctypes.c_int, ctypes.c_void_p]
    lib.bench_stream_copy.restype = ctypes.c_int
    n = gib << 30
    buf = torch.full((n // 2,), 1.0, dtype=torch.bfloat16, device=dev)
    sink = torch.zeros(256, dtype=torch.int32, device=dev)
    st = torch.cuda.current_stream()

    def launch(nbytes, grid, kind):
        rc = lib.bench_stream_read(buf.data_ptr(), nbytes, sink.data_ptr(), grid, kind,
                                   st.cuda_stream)
        if rc != 0:
            raise RuntimeError("bench_stream_read failed: hipError %d" % rc)

    def timed(nbytes, grid, kind, warm):
        ts = []
        for _ in range(reps):
            if warm:
                launch(nbytes, grid, kind)  # leaves the bytes in the Infinity Cache
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(st)
            launch(nbytes, grid, kind)
            b.record(st)
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b))
        ts.sort()
        return ts[len(ts) // 2]  # median

    out = {"cold_bytes": n, "hot_bytes": hot_mib << 20, "routes": {}}
    best = 0.0
    for kind, name in STREAM_KINDS.items():
        cold = {}
        for grid in (1024, 2048, 4096, 8192):
            ms = timed(n, grid, kind, False)
            cold[grid] = n / (ms / 1e3) / 1e9
        g_best = max(cold, key=cold.get)
        hot_ms = timed(hot_mib << 20, g_best, kind, True)
        out["routes"][name] = {"cold_gbs_by_grid": cold, "cold_gbs": cold[g_best],
                               "best_grid": g_best,
                               "hot_gbs": (hot_mib << 20) / (hot_ms / 1e3) / 1e9}
        best = max(best, cold[g_best])
    out["ceiling_gbs"] = best
    out["ceiling_frac_of_peak"] = best / HBM_PEAK_GBS
    # an even read/write mix: the first half of the buffer copied to the second
    half = n // 2
    copy = {}
    for grid in (1024, 2048, 4096, 8192):
        ts = []
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(st)
            rc = lib.bench_stream_copy(buf.data_ptr(), buf.data_ptr() + half, half, grid,
                                       st.cuda_stream)
            if rc != 0:
                raise RuntimeError("bench_stream_copy failed: hipError %d" % rc)
            b.record(st)
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b))
        ts.sort()
        copy[grid] = 2 * half / (ts[len(ts) // 2] / 1e3) / 1e9  # bytes read + written
    g_best = max(copy, key=copy.get)
    out["copy"] = {"what": "stream_copy_kernel: %d MiB copied, bytes read + written per second"
                           % (half >> 20), "gbs_by_grid": copy, "gbs": copy[g_best],
                   "frac_of_peak": copy[g_best] / HBM_PEAK_GBS}
    del buf
    torch.cuda.empty_cache()
    return out


def calibration_copy(mib: int) -> None:
    import torch
    n = mib * 1024 * 1024 // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(3):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    print("bench: calibration copy of %d MiB done" % mib, file=sys.stderr, flush=True)
    del src, dst
    torch.cuda.empty_cache()


def build_layers(args, wl, dev, n_layers, shared):
    """Draw the workload's layers on the device, with Algorithm 1 budgets (or
    the workload's fixed budget) and output buffers. Returns (desc, layers,
    budgets[prompt][layer], element size); layers[l] = (mask, seqs)."""
    import numpy as np
    import torch

    import paper_2508_02401_amd as ckv
    from paper_2508_02401_amd import synth

    desc = ckv.layer_desc(wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.window, wl.dtype, 0.0,
                          wl.pool, wl.pool_kernel,
                          ckv.CKV_KEEP_WINDOW | (ckv.CKV_SHARE_LAYER if shared else 0))
    elt = torch.tensor([], dtype=wl.dtype).element_size()
    errs = synth.layer_errors(wl)
    budgets = []  # [prompt][layer]
    for L in wl.seq_lens:
        if wl.budget is not None:
            budgets.append([wl.budget] * wl.n_layers)
        else:
            total, m, M = synth.budget_params(wl, L)
            b, st = ckv.ckv_allocate_budgets(errs, total, m, M)
            if st != ckv.CKV_OK:
                raise RuntimeError("Algorithm 1 could not meet the total")
            budgets.append([int(x) for x in b])
    print("bench: drawing %d layers of %s" % (n_layers, wl.name), file=sys.stderr, flush=True)
    layers = []
    for l in range(n_layers):
        inp = synth.layer_inputs(wl, l, dev)
        seqs = [ckv.alloc_outputs(desc, ckv.Seq(inp.q_win[s], inp.k[s], inp.v[s], budgets[s][l]),
                                  with_scores=False)
                for s in range(len(wl.seq_lens))]
        layers.append((synth.shared_head_mask(wl, l) if shared else inp.mask, seqs))
    return desc, layers, budgets, elt


def measure(args, wl, desc, layers, budgets, elt, dev, hip, schedule, shared=False,
            copies=None, timed=("rowstats", "score")):
    """Time args.steps steps of one schedule over the drawn layers and compute
    the metric, the path's HBM rate and the dominant K pass's roofline.

    schedule: "stack" (one ckv_compress_stack call per step, optionally with a
    side stream), "layers" (ckv_compress_layer per layer over args.streams
    streams), "pipeline" (ckv_score on one stream, ckv_select + ckv_gather on a
    second, one layer apart) or "rotate" (one ckv_compress_layer per step on the
    next of `copies`, distinct copies of a single layer's inputs, so every step
    reads its K and V from HBM rather than from the 256 MB Infinity Cache).
    Returns (result dict, stage means)."""
    import numpy as np
    import torch

    import paper_2508_02401_amd as ckv

    main = torch.cuda.current_stream()
    n_layers = len(layers)
    side = None
    n_streams = 1
    if schedule == "stack":
        stack_slots = args.stack_slots if args.stack_slots > 0 else n_layers
        if args.stack_side:
            side = torch.cuda.Stream()
            n_streams = 2
        ws_bytes = max(ckv.ckv_workspace_bytes(desc, seqs) for _, seqs in layers)
        ws_stack = torch.empty(stack_slots * ws_bytes, dtype=torch.uint8, device=dev)
        stack_masks = np.stack([m for m, _ in layers])
        stack_seqs = [sq for _, sq in layers]
        sched_text = ("ckv_compress_stack: the two K passes layer by layer%s, then pooling + "
                      "selection + gather as two launches (three when a unit keeps over 512 rows) "
                      "per batch of %d layers"
                      % (", consecutive layers alternating between two streams"
                         if args.stack_side else "", stack_slots))

        def step(events=None):
            if events is not None:
                ns_ = ckv.CKV_NUM_STAGES
                ckv.ckv_set_stack_stage_events(
                    [[None] * ns_ if x is None else x[0] for x in events],
                    [[None] * ns_ if x is None else x[1] for x in events])
            ckv.ckv_compress_stack(desc, stack_masks, stack_seqs, ws_stack, main, side)
            if events is not None:
                ckv.ckv_set_stack_stage_events(None, None)
    elif schedule == "pipeline":
        n_streams = 2
        side = torch.cuda.Stream()
        ws_bytes = max(ckv.ckv_workspace_bytes(desc, seqs) for _, seqs in layers)
        wss = [torch.empty(ws_bytes, dtype=torch.uint8, device=dev) for _ in range(2)]
        score_bufs = [[torch.empty((wl.num_kv_heads, L - wl.window), dtype=torch.float32,
                                   device=dev) for L in wl.seq_lens] for _ in range(2)]
        for li, (mask, seqs) in enumerate(layers):
            for si, sq in enumerate(seqs):
                sq.scores = score_bufs[li % 2][si]
        scored = [torch.cuda.Event(enable_timing=False) for _ in range(2)]
        selected = [torch.cuda.Event(enable_timing=False) for _ in range(2)]
        sched_text = ("pipeline: K passes + pooling on stream A, selection + gather on stream B, "
                      "one layer apart")

        def step(events=None):
            side.wait_stream(main)
            for li, (mask, seqs) in enumerate(layers):
                slot = li % 2
                if events is not None:
                    ckv.ckv_set_stage_events(*(events[li] if events[li] is not None
                                               else (None, None)))
                if li >= 2:
                    main.wait_event(selected[slot])  # layer li-2 is done with this slot
                ckv.ckv_score(desc, mask, seqs, wss[slot], main)
                scored[slot].record(main)
                side.wait_event(scored[slot])
                ckv.ckv_select(desc, seqs, wss[slot], side)
                ckv.ckv_gather(desc, seqs, side)
                selected[slot].record(side)
            if events is not None:
                ckv.ckv_set_stage_events(None, None)
            main.wait_stream(side)
    elif schedule == "rotate":
        assert n_layers == 1 and copies
        mask = layers[0][0]
        ws = torch.empty(max(ckv.ckv_workspace_bytes(desc, c) for c in copies), dtype=torch.uint8,
                         device=dev)
        turn = [0]
        sched_text = ("ckv_compress_layer, one layer per step, rotating over %d distinct copies "
                      "of its inputs (%.2f GB) so that K and V come from HBM"
                      % (len(copies), sum(int(sq.k.numel() + sq.v.numel()) * elt
                                          for c in copies for sq in c) / 1e9))

        def step(events=None):
            c = copies[turn[0] % len(copies)]
            turn[0] += 1
            if events is not None and events[0] is not None:
                ckv.ckv_set_stage_events(events[0][0], events[0][1])
            ckv.ckv_compress_layer(desc, mask, c, ws, main)
            if events is not None and events[0] is not None:
                ckv.ckv_set_stage_events(None, None)
    else:
        n_streams = max(1, args.streams)
        streams = [main] + [torch.cuda.Stream() for _ in range(n_streams - 1)]
        ws_bytes = max(ckv.ckv_workspace_bytes(desc, seqs) for _, seqs in layers)
        wss = [torch.empty(ws_bytes, dtype=torch.uint8, device=dev) for _ in range(n_streams)]
        sched_text = "ckv_compress_layer per layer, round-robin over streams"

        def step(events=None):
            for st in streams[1:]:
                st.wait_stream(main)
            for li, (mask, seqs) in enumerate(layers):
                si = li % n_streams
                if events is not None:
                    ckv.ckv_set_stage_events(*(events[li] if events[li] is not None
                                               else (None, None)))
                ckv.ckv_compress_layer(desc, mask, seqs, wss[si], streams[si])
            if events is not None:
                ckv.ckv_set_stage_events(None, None)
            for st in streams[1:]:
                main.wait_stream(st)
    torch.cuda.synchronize()

    # Warm up, then time args.steps steps. Only the stages in `timed` (the K
    # passes) carry kernel start/end events, and only on every N-th layer of a
    # step (the offset rotates with the step): each timed launch delays the
    # dispatch of its neighbours by a few microseconds, so the other stages and
    # layers are left untimed (their times are in the rocprofv3 kernel trace).
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ns = ckv.CKV_NUM_STAGES
    idx = {n: ckv.STAGE_NAMES.index(n) for n in timed}
    i_pool, i_sel, i_gat = (ckv.STAGE_NAMES.index(n) for n in ("pool", "select", "gather"))
    # the stack's selection launches carry the events of the batch's first
    # layer: with one batch, layer 0's pool begin and gather end bracket them
    sel_timed = schedule == "stack" and args.stack_slots <= 0
    # The stack launches each K pass for up to CKV_STACK_LAYERS_PER_LAUNCH
    # consecutive layers of a batch at once, with the first layer's events:
    # chunk[l] lists the layers of the launch that starts at layer l.
    chunk = {}
    if schedule == "stack":
        per = ckv.stack_layers_per_launch(wl.seq_lens)
        batch = args.stack_slots if args.stack_slots > 0 else n_layers
        for b0 in range(0, n_layers, batch):
            for c in range(b0, min(b0 + batch, n_layers), per):
                chunk[c] = list(range(c, min(c + per, b0 + batch, n_layers)))
    else:
        chunk = {l: [l] for l in range(n_layers)}
    starts = sorted(chunk)
    every = max(1, min(len(starts), round(args.time_every / max(len(v) for v in chunk.values()))))
    ev = []  # ev[step][layer] = (begin, end) arrays, or None for an untimed layer
    kp_timed = []  # kp_timed[step][layer]: the K passes carry events
    for k in range(args.steps):
        per_layer, flags = [], []
        for li in range(n_layers):
            kp = li in chunk and (starts.index(li) + k) % every == 0
            sel = sel_timed and li == 0 and k % 4 == 0  # selection events: every 4th step
            flags.append(kp)
            if not kp and not sel:
                per_layer.append(None)
                continue
            b, e = [None] * ns, [None] * ns
            if kp:
                for n in timed:
                    b[idx[n]], e[idx[n]] = hip.event(), hip.event()
            if sel:
                b[i_pool], e[i_pool] = hip.event(), hip.event()
                b[i_sel], e[i_gat] = hip.event(), hip.event()
            per_layer.append((b, e))
        ev.append(per_layer)
        kp_timed.append(flags)
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    # no garbage collection while steps are enqueued: a collection over the
    # objects of earlier measurements stalls submission for milliseconds
    gc.collect()
    gc.disable()
    wall0 = time.perf_counter()
    t_start.record(main)
    for k in range(args.steps):
        step(ev[k])
    t_end.record(main)
    host_s = time.perf_counter() - wall0  # enqueueing alone
    torch.cuda.synchronize()
    wall_s = time.perf_counter() - wall0
    gc.enable()
    ms_per_step = t_start.elapsed_time(t_end) / args.steps
    stage_ms = {n: [] for n in timed}
    sel_ms = []
    sampled = []
    for k in range(args.steps):
        for li in range(n_layers):
            if ev[k][li] is None:
                continue
            b, e = ev[k][li]
            if kp_timed[k][li]:
                sampled.append(li)
                for n in timed:
                    stage_ms[n].append(hip.elapsed_ms(b[idx[n]], e[idx[n]]))
            if b[i_pool] is not None:
                sel_ms.append(hip.elapsed_ms(b[i_pool], e[i_gat]))
            for x in b + e:
                if x is not None:
                    hip.destroy(x)
    stage_avg = {n: float(np.mean(v)) for n, v in stage_ms.items()}

    tokens_per_layer = sum(wl.seq_lens)
    value = tokens_per_layer * n_layers / (ms_per_step / 1e3)
    n_kv, d, w = wl.num_kv_heads, wl.head_dim, wl.window
    G = wl.num_q_heads // n_kv

    def groups_read(mask):
        # KV heads whose keys are streamed: those with a chosen query head
        return len(set((np.nonzero(mask)[0] // G).tolist()))

    # algorithmic bytes of the whole path per layer: K once, the chosen Q rows,
    # the retained K/V rows read and written, the indices
    n_sg = 1 if shared else n_kv  # index rows written per prompt
    path_bytes = 0
    for li, (mask, seqs) in enumerate(layers):
        n_chosen = int(np.count_nonzero(mask))
        for s, L in enumerate(wl.seq_lens):
            n_ret = min(int(seqs[s].budget), L)
            path_bytes += groups_read(mask) * L * d * elt + n_chosen * w * d * elt \
                + 4 * n_kv * n_ret * d * elt + 4 * n_sg * n_ret
    path_gbs = path_bytes / (ms_per_step / 1e3) / 1e9

    # dominant kernel: the timed K pass with the longest mean launch
    dom = max(timed, key=lambda n: stage_avg[n])
    dom_bytes, flops = [], []
    for l0 in sampled:
        b = f = 0
        for li in chunk[l0]:  # the layers of the timed launch
            mask = layers[li][0]
            n_chosen = int(np.count_nonzero(mask))
            for L in wl.seq_lens:
                n_rd = groups_read(mask)
                if dom == "rowstats":
                    # every key of the prompt and the chosen Q rows
                    b += n_rd * L * d * elt + n_chosen * w * d * elt
                else:
                    # prefix keys, chosen Q rows, and the window sum of every
                    # chosen head written per prefix token
                    b += n_rd * (L - w) * d * elt + n_chosen * w * d * elt + n_chosen * (L - w) * 4
                f += 2 * n_chosen * w * (L if dom == "rowstats" else (L - w)) * d
        dom_bytes.append(b)
        flops.append(f)
    dom_gbs = float(np.mean(dom_bytes)) / (stage_avg[dom] / 1e3) / 1e9
    dom_tflops = float(np.mean(flops)) / (stage_avg[dom] / 1e3) / 1e12
    # The K-pass phase of the step as a whole: with a side stream two K-pass
    # launches are in flight at once (one per stream), so a launch's own
    # duration overstates its share of the step. Phase = step time minus the
    # selection launches (timed on layer 0's events); bytes = the algorithmic
    # bytes of every layer's timed passes.
    kpass_phase = None
    if sel_ms:
        ph_bytes = 0
        for mask, seqs in layers:
            n_chosen = int(np.count_nonzero(mask))
            for L in wl.seq_lens:
                n_rd = groups_read(mask)
                if "rowstats" in timed:
                    ph_bytes += n_rd * L * d * elt + n_chosen * w * d * elt
                ph_bytes += n_rd * (L - w) * d * elt + n_chosen * w * d * elt + n_chosen * (L - w) * 4
        ph_ms = ms_per_step - float(np.mean(sel_ms))
        kpass_phase = {"what": "the K passes of all %d layers (%s), %s: their algorithmic bytes "
                               "over the step time minus the selection launches"
                               % (n_layers, " + ".join(timed),
                                  "two launches in flight, one per stream" if side is not None
                                  else "one stream"),
                       "ms": ph_ms, "selection_ms": float(np.mean(sel_ms)),
                       "bytes": ph_bytes, "gbs": ph_bytes / (ph_ms / 1e3) / 1e9,
                       "frac": ph_bytes / (ph_ms / 1e3) / 1e9 / HBM_PEAK_GBS}
    res = {
        "ms_per_step": ms_per_step,
        "value": value,
        "config": {"workload": wl.name, "layers": n_layers, "q_heads": wl.num_q_heads,
                   "kv_heads": n_kv, "head_dim": d, "seq_lens": list(wl.seq_lens),
                   "window": w, "pool": "max" if wl.pool == 1 else "avg",
                   "pool_kernel": wl.pool_kernel, "heads_per_group": list(wl.n_sel_choices),
                   "budget_avg": float(np.mean([sq.budget for _, seqs in layers for sq in seqs])),
                   "parallelism": "single GPU",
                   "head_scope": "layer-shared, 4 heads per layer" if shared else "per KV group",
                   "streams": n_streams, "schedule": sched_text},
        "path_hbm_gbs": path_gbs,
        "path_hbm_frac": path_gbs / HBM_PEAK_GBS,
        "path_bytes_per_step": path_bytes,
        "stage_ms_avg": stage_avg,
        "kpass_phase": kpass_phase,
        "roofline": {"kernel": dom + ("_layers_kernel" if max(len(v) for v in chunk.values()) > 1
                                      else "_kernel"),
                     "bound": "hbm", "achieved": dom_gbs,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": dom_gbs / HBM_PEAK_GBS,
                     "traffic": None, "avg_launch_ms": stage_avg[dom],
                     "algorithmic_bytes_per_launch": float(np.mean(dom_bytes)),
                     "timed_launches": len(sampled),
                     "layers_per_launch": max(len(v) for v in chunk.values()),
                     "launches_in_flight": 2 if side is not None else 1,
                     "mfma_tflops": dom_tflops, "mfma_frac_bf16": dom_tflops / BF16_PEAK_TFLOPS},
        "wall_s_timed": wall_s,
        "host_enqueue_ms_per_step": host_s * 1e3 / args.steps,
    }
    return res


def side_stream_leg(args, wl, desc, layers, budgets, elt, dev, hip, shared=False):
    """The same stack step with a side stream for every other layer's K passes:
    its step time and the K-pass phase's aggregate rate (per-launch durations
    overlap there, so no per-launch roofline)."""
    import copy

    a2 = copy.copy(args)
    a2.stack_side = 1
    r = measure(a2, wl, desc, layers, budgets, elt, dev, hip, "stack", shared)
    return {"what": "ckv_compress_stack with a side stream: consecutive layers' K passes "
                    "alternate between two streams, two launches in flight",
            "ms_per_step": r["ms_per_step"], "value": r["value"],
            "path_hbm_frac": r["path_hbm_frac"], "kpass_phase": r["kpass_phase"]}


def rotate_copies(desc, layers, dev, min_bytes: int = 512 << 20, min_copies: int = 8):
    """Distinct copies of a single layer's inputs (with their own outputs), at
    least min_copies of them and at least min_bytes of K and V in total."""
    import paper_2508_02401_amd as ckv

    seqs = layers[0][1]
    per = sum(int(sq.k.numel() + sq.v.numel()) * sq.k.element_size() for sq in seqs)
    n = max(min_copies, -(-min_bytes // per))
    copies = [seqs]
    for _ in range(n - 1):
        c = []
        for sq in seqs:
            x = ckv.Seq(sq.q_win.clone(), sq.k.clone(), sq.v.clone(), sq.budget)
            c.append(ckv.alloc_outputs(desc, x, with_scores=False))
        copies.append(c)
    return copies


def main():
    args = parse()
    if args.summarize_trace:
        summarize_trace(args.summarize_trace)
        return
    if args.summarize_pmc:
        summarize_pmc(args.summarize_pmc[0], args.summarize_pmc[1], args.copy_mib)
        return
    if args.summarize_counters:
        summarize_counters(args.summarize_counters)
        return
    if args.gpus != 1:
        print("bench.py runs on one GPU only: the eviction path has no multi-GPU mode (every KV "
              "head, layer and prompt is independent, so a multi-GPU run would shard by KV head "
              "or layer with no communication).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2508_02401_amd as ckv
    from paper_2508_02401_amd import synth

    ckv.load()
    dev = torch.device("cuda:0")
    if args.stream_ceiling_only:
        print(json.dumps({"stream_ceiling": stream_ceiling(dev)}), flush=True)
        return
    if args.calibrate_copy > 0:
        calibration_copy(args.calibrate_copy)
    wl = synth.WORKLOADS[args.workload]
    n_layers = wl.n_layers if args.layers <= 0 else min(args.layers, wl.n_layers)
    shared = args.scope == "shared"
    hip = Hip()
    desc, layers, budgets, elt = build_layers(args, wl, dev, n_layers, shared)
    schedule = "pipeline" if args.pipeline else args.schedule
    copies = None
    if n_layers == 1 and schedule == "stack":
        # a single layer fits in the Infinity Cache: rotate distinct copies
        schedule = "rotate"
        copies = rotate_copies(desc, layers, dev)
    res = measure(args, wl, desc, layers, budgets, elt, dev, hip, schedule, shared, copies)
    del copies
    ms_per_step = res["ms_per_step"]
    path_bytes = res["path_bytes_per_step"]
    n_kv, d, w = wl.num_kv_heads, wl.head_dim, wl.window
    G = wl.num_q_heads // n_kv
    tokens_per_layer = sum(wl.seq_lens)
    dom = res["roofline"]["kernel"]
    traffic = committed_traffic(dom) if wl.name == "llama8b-128k-stack" else None
    roof = dict(res["roofline"])
    roof["traffic"] = traffic
    roof["traffic_gbs"] = None if traffic is None else traffic / (roof["avg_launch_ms"] / 1e3) / 1e9
    result = {
        "metric": "prompt tokens compressed/sec per layer (L=32K/128K) + achieved HBM GB/s",
        "value": res["value"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": {torch.bfloat16: "bf16", torch.float16: "f16", torch.float32: "f32"}[wl.dtype],
        "data": "synthetic (seeded N(0,1) Q/K/V with planted sink and span keys; no real "
                "activations or datasets)",
        "config": res["config"],
        "path_hbm_gbs": res["path_hbm_gbs"],
        "path_hbm_frac": res["path_hbm_frac"],
        "stage_ms_avg": res["stage_ms_avg"],
        "kpass_phase": res["kpass_phase"],
        "roofline": roof,
        "wall_s_timed": res["wall_s_timed"],
        "host_enqueue_ms_per_step": res["host_enqueue_ms_per_step"],
    }

    def leg(key, fn, into=result):
        # a leg that fails records its error; the headline line still prints
        try:
            into[key] = fn()
        except Exception as exc:  # noqa: BLE001
            print("bench: leg %s failed: %r" % (key, exc), file=sys.stderr, flush=True)
            into[key] = {"error": repr(exc)}

    if schedule == "stack" and not args.stack_side and not args.no_side_variant:
        leg("side_stream_variant",
            lambda: side_stream_leg(args, wl, desc, layers, budgets, elt, dev, hip, shared))

    def lse_leg():
        # The same step with the window rows' log-sum-exp supplied by the
        # caller (a causal prefill attention kernel keeps it per query row):
        # the row-statistics pass is skipped and K is read once. The values
        # are computed here beforehand (fp32 logits of the chosen heads, a
        # causal mask and a log-sum-exp), outside the timed region.
        scale = 1.0 / float(np.sqrt(d))
        for mask, seqs in layers:
            for sq in seqs:
                L = sq.k.shape[1]
                lse = torch.full((wl.num_q_heads, w), float("nan"), dtype=torch.float32, device=dev)
                causal = (torch.arange(L, device=dev)[None, :]
                          > (L - w + torch.arange(w, device=dev))[:, None])
                for g in range(n_kv):
                    heads = [int(h) for h in np.nonzero(mask)[0] if int(h) // G == g]
                    if not heads:
                        continue
                    kt = sq.k[g].float().t().contiguous()  # [d, L]
                    for h in heads:
                        logits = (sq.q_win[h].float() @ kt) * scale
                        lse[h] = torch.logsumexp(logits.masked_fill(causal, float("-inf")), dim=1)
                    del kt
                sq.lse = lse
        torch.cuda.synchronize()
        try:
            r_lse = measure(args, wl, desc, layers, budgets, elt, dev, hip,
                            "stack" if schedule == "rotate" else schedule, shared, timed=("score",))
        finally:
            for mask, seqs in layers:
                for sq in seqs:
                    sq.lse = None
        ms_lse = r_lse["ms_per_step"]
        return {
            "what": "same step with the window rows' log-sum-exp supplied by the caller's prefill "
                    "attention: no row-statistics pass, K read once",
            "ms_per_step": ms_lse, "value": tokens_per_layer * n_layers / (ms_lse / 1e3),
            "path_hbm_gbs": path_bytes / (ms_lse / 1e3) / 1e9,
            "path_hbm_frac": path_bytes / (ms_lse / 1e3) / 1e9 / HBM_PEAK_GBS,
            "score_kernel_avg_us": r_lse["stage_ms_avg"]["score"] * 1e3,
            "kpass_phase": r_lse["kpass_phase"]}

    if not args.no_lse_variant:
        leg("caller_lse_variant", lse_leg)

    if not args.no_profile_variant:
        leg("error_profile", lambda: error_profile(args, wl, layers, dev, hip))
    if not args.no_decode_variant:
        leg("decode_step", lambda: decode_step(wl, layers, dev))
        # last: it overwrites the compact caches the legs above read
        leg("streaming_preset", lambda: streaming_preset(wl, layers, dev))

    if not args.no_cpu_baseline:
        leg("cpu_baseline", lambda: cpu_baseline(wl, layers, args.cpu_threads, args.cpu_seconds))
    del layers
    torch.cuda.empty_cache()

    # the other workloads of the metric, each with its own step and roofline
    others = {}
    def other_config(name):
        owl = synth.WORKLOADS[name]
        od, ol, ob, oe = build_layers(args, owl, dev, owl.n_layers, False)
        if owl.n_layers == 1:
            oc = rotate_copies(od, ol, dev)
            r = measure(args, owl, od, ol, ob, oe, dev, hip, "rotate", False, oc)
            del oc
        else:
            r = measure(args, owl, od, ol, ob, oe, dev, hip, "stack", False)
            if not args.stack_side and not args.no_side_variant:
                r["side_stream_variant"] = side_stream_leg(args, owl, od, ol, ob, oe, dev, hip)
        r.pop("path_bytes_per_step", None)
        del ol
        torch.cuda.empty_cache()
        return r

    for name in [x for x in args.configs.split(",") if x and x != wl.name]:
        leg(name, lambda: other_config(name), others)
    if others:
        result["other_configs"] = others
    if not args.no_stream_ceiling:
        leg("stream_ceiling", lambda: stream_ceiling(dev))
    print(json.dumps(result), flush=True)


def error_profile(args, wl, layers, dev, hip, T: int = 16, n_layers: int = 8, reps: int = 3):
    """Time ckv_layer_error (Eq. 6-8) on the first layers of the workload: T
    synthetic decode queries per layer, attention over the full prompt cache and
    over the compact cache the timed step just wrote, a random W_O of the model's
    shape (D = H * d). Bytes: K and V of the full cache read once, the compact
    cache, and W_O."""
    import numpy as np
    import torch

    import paper_2508_02401_amd as ckv

    n_layers = min(n_layers, len(layers))
    H, n_kv, d = wl.num_q_heads, wl.num_kv_heads, wl.head_dim
    D = H * d
    desc = ckv.attn_desc(H, n_kv, d, wl.dtype)
    gen = torch.Generator(device=dev).manual_seed(7)
    q_dec = torch.randn((T, H, d), generator=gen, device=dev).to(wl.dtype)
    w_o = (torch.randn((D, H * d), generator=gen, device=dev) / float(np.sqrt(H * d))).to(wl.dtype)
    jobs = []
    for mask, seqs in layers[:n_layers]:
        sq = seqs[0]
        full, comp = ckv.kv_cache(sq.k, sq.v), ckv.kv_cache(sq.k_out, sq.v_out)
        jobs.append((full, comp, sq.k.shape[1], sq.k_out.shape[1]))
    ws = torch.empty(max(ckv.ckv_layer_error_workspace_bytes(desc, T, n, nc, D) for _, _, n, nc in jobs),
                     dtype=torch.uint8, device=dev)
    ratio = torch.empty((n_layers, T), dtype=torch.float32, device=dev)
    e = torch.empty(n_layers, dtype=torch.float32, device=dev)

    def run():
        for i, (full, comp, _, _) in enumerate(jobs):
            ckv.ckv_layer_error(desc, q_dec, full, comp, w_o, 1e-6, ratio[i], e[i:i + 1], ws)

    run()
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(reps):
        run()
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / (reps * n_layers)
    elt = torch.tensor([], dtype=wl.dtype).element_size()
    n, nc = jobs[0][2], jobs[0][3]
    bytes_layer = 2 * n_kv * (n + nc) * d * elt + D * H * d * elt
    return {"what": "ckv_layer_error per layer: decode attention of %d synthetic queries over the "
                    "full %d-token cache and the compact cache, W_O [%d x %d] projection, ratios "
                    "(Eq. 6-8); %d layers x %d reps" % (T, n, D, H * d, n_layers, reps),
            "ms_per_layer": ms, "hbm_gbs": bytes_layer / (ms / 1e3) / 1e9,
            "hbm_frac": bytes_layer / (ms / 1e3) / 1e9 / HBM_PEAK_GBS,
            "e_first_layers": [float(x) for x in e.cpu()]}


def decode_step(wl, layers, dev, reps: int = 3):
    """One decoding step (one query token) over every layer's cache, as one
    ragged batch per cache kind (ckv_decode_attention_batch): the full prompt
    caches, then the compact caches the timed step wrote (Eq. 3-4). Bytes: K
    and V of every cache read once."""
    import numpy as np
    import torch

    import paper_2508_02401_amd as ckv

    H, n_kv, d = wl.num_q_heads, wl.num_kv_heads, wl.head_dim
    desc = ckv.attn_desc(H, n_kv, d, wl.dtype)
    gen = torch.Generator(device=dev).manual_seed(11)
    elt = torch.tensor([], dtype=wl.dtype).element_size()
    res = {}
    for kind in ("full", "compact"):
        seqs, outs, nbytes, lens = [], [], 0, []
        for mask, layer_seqs in layers:
            for sq in layer_seqs:
                k, v = (sq.k, sq.v) if kind == "full" else (sq.k_out, sq.v_out)
                q = torch.randn((1, H, d), generator=gen, device=dev).to(wl.dtype)
                o = torch.empty((1, H, d), dtype=torch.float32, device=dev)
                seqs.append(ckv.decode_seq(q, ckv.kv_cache(k, v), o))
                outs.append((q, o))
                nbytes += 2 * n_kv * k.shape[1] * d * elt
                lens.append(int(k.shape[1]))
        ws = torch.empty(ckv.ckv_decode_batch_workspace_bytes(desc, seqs), dtype=torch.uint8,
                         device=dev)
        ckv.ckv_decode_attention_batch(desc, seqs, ws)
        torch.cuda.synchronize()
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0.record()
        for _ in range(reps):
            ckv.ckv_decode_attention_batch(desc, seqs, ws)
        t1.record()
        torch.cuda.synchronize()
        ms = t0.elapsed_time(t1) / reps
        res[kind] = {"ms": ms, "cached_tokens_per_head": [min(lens), int(np.mean(lens)), max(lens)],
                     "hbm_gbs": nbytes / (ms / 1e3) / 1e9}
        del ws, outs
    return {"what": "one decoding step (1 query token per layer, all %d layers as one ragged "
                    "batch) over the full prompt caches and over the compact caches" % len(layers),
            "full_ms": res["full"]["ms"], "compact_ms": res["compact"]["ms"],
            "speedup": res["full"]["ms"] / res["compact"]["ms"],
            "full_hbm_gbs": res["full"]["hbm_gbs"],
            "compact_tokens_min_mean_max": res["compact"]["cached_tokens_per_head"]}


def streaming_preset(wl, layers, dev, reps: int = 3):
    """The StreamingLLM-style preset (ckv_streaming_select, 4 sink tokens) on
    every layer with the layer's budget: index rows and K/V gather, no
    scoring. Bytes: the kept K and V rows read and written, and the indices."""
    import torch

    import paper_2508_02401_amd as ckv

    desc = ckv.layer_desc(wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.window, wl.dtype, 0.0,
                          wl.pool, wl.pool_kernel)
    elt = torch.tensor([], dtype=wl.dtype).element_size()

    def run():
        for mask, seqs in layers:
            ckv.ckv_streaming_select(desc, seqs, 4)

    run()
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(reps):
        run()
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / (reps * len(layers))
    kept = sum(int(sq.k_out.shape[1]) for _, seqs in layers for sq in seqs) / len(layers)
    nbytes = wl.num_kv_heads * kept * (4 * wl.head_dim * elt + 4)
    return {"what": "ckv_streaming_select per layer (first 4 + most recent tokens, the layer's "
                    "budget), one launch per layer", "ms_per_layer": ms,
            "hbm_gbs": nbytes / (ms / 1e3) / 1e9}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(wl, layers, threads: int, min_seconds: float = 15.0):
    """The fp64 oracle on a bounded sample of the timed workload: the same
    inputs (converted to fp64 on the device and copied to the host, untimed)
    and the same per-layer Algorithm 1 budgets. Independent (layer, prompt, KV
    head) calls of the oracle's single-threaded group selection run
    concurrently on `threads` host threads (ctypes releases the GIL), a batch
    of whole layers at a time, until about min_seconds of wall time are spent.
    The value is prompt tokens per second per layer, like the GPU's."""
    import concurrent.futures as cf

    import numpy as np
    import torch

    import oracle

    n_avail = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    # at most 16 threads: the CPU share of one GPU on a shared host
    n_threads = threads if threads > 0 else max(1, min(n_avail or 1, 16))
    n_kv, G = wl.num_kv_heads, wl.num_q_heads // wl.num_kv_heads
    scale = 1.0 / float(np.sqrt(wl.head_dim))
    pool = oracle.POOL_MAX if wl.pool == 1 else oracle.POOL_AVG
    tasks_per_layer = n_kv * len(wl.seq_lens)
    per_batch = max(1, -(-n_threads // tasks_per_layer))  # layers per batch: every thread busy

    def run(q_sel, k, budget):
        oracle.select_group(q_sel, k, wl.window, scale, pool, wl.pool_kernel, budget)

    spent, layers_done, n_calls = 0.0, 0, 0
    with cf.ThreadPoolExecutor(max_workers=n_threads) as ex:
        li = 0
        while li < len(layers) and spent < min_seconds:
            batch = layers[li:li + per_batch]
            jobs = []
            for mask, seqs in batch:
                for sq in seqs:
                    for g in range(n_kv):
                        heads = [g * G + t for t in range(G) if mask[g * G + t]]
                        if not heads:
                            continue
                        q_sel = sq.q_win[heads].double().cpu().numpy()
                        k = sq.k[g].double().cpu().numpy()
                        jobs.append((q_sel, k, int(sq.budget)))
            t0 = time.perf_counter()
            for f in [ex.submit(run, *j) for j in jobs]:
                f.result()
            spent += time.perf_counter() - t0
            n_calls += len(jobs)
            layers_done += len(batch)
            li += per_batch
            del jobs
    tokens = sum(wl.seq_lens) * layers_done
    return {"value": tokens / spent, "unit": "tokens/s", "cores": n_threads,
            "threads": n_threads, "host_cpus": os.cpu_count(), "cpus_available": n_avail,
            "cpu_model": cpu_model(), "kind": "oracle",
            "sample": "layers 0-%d of %s (the timed inputs and their Algorithm 1 budgets): %d "
                      "single-threaded fp64 oracle calls, one per (layer, prompt, KV head), "
                      "%d at a time; %.1f s of wall time" % (layers_done - 1, wl.name, n_calls,
                                                             n_threads, spent)}


if __name__ == "__main__":
    main()
