#!/usr/bin/env python3
"""Benchmark of the few-bit activation hot path on one MI355X.

One step = one forward (y = f(x), classify, pack b-bit codes) plus one
backward (unpack, grad_in = grad_out * v[idx]) over the whole tensor: every
row of the hot path.  Default workload: GELU, 3 bits, bf16 x of shape
[16, 2048, 8192] (268,435,456 elements) drawn as 0.99 N(0,1) + 0.01 N(0,10^2),
grad_out ~ N(0,1), inputs resident in HBM before timing starts.

Prints ONE JSON line.  `value` is the whole-step throughput in GB/s of
algorithmic bytes: forward reads x (s bytes) and writes y (s) and codes
(b/8); backward reads grad_out (s) and codes (b/8) and writes grad_in (s).

  python bench.py [--steps K] [--warmup W] [--workload NAME] [--bits B]
  python bench.py --all-configs                (one JSON line per workload and bit width)
  python bench.py --sweep [--sweep-n N]        (every activation x type x bits)
  python bench.py --summarize-trace DIR [--summarize-counters FETCH_DIR WRITE_DIR]
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "fwd+bwd GB/s & % HBM peak (elements/s), GELU 3-bit bf16 [16,2048,8192]"
HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E, published


def algorithmic_bytes(n: int, dtype: str, bits: int) -> float:
    s = 4 if dtype == "f32" else 2
    return n * (2 * s + bits / 8.0)


def _code_tokens(src: str) -> str:
    """C/C++ source without comments and with whitespace runs collapsed:
    an edit of comments or layout does not change the kernels."""
    out, i, n = [], 0, len(src)
    while i < n:
        c = src[i]
        if src.startswith("//", i):
            j = src.find("\n", i)
            i = n if j < 0 else j
        elif src.startswith("/*", i):
            j = src.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        elif c in "\"'":
            j = i + 1
            while j < n and src[j] != c:
                j += 2 if src[j] == "\\" else 1
            out.append(src[i:j + 1])
            i = j + 1
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def kernel_source_hash() -> str:
    """Hash of the kernel source's code (comments and layout ignored)."""
    h = hashlib.sha256()
    for f in ("paper_2202_00441_amd/csrc/fewbit.hip",):
        with open(os.path.join(ROOT, f), encoding="utf-8") as fh:
            h.update(_code_tokens(fh.read()).encode())
    return h.hexdigest()[:16]


def kernel_name(kind: str, dtype: str, bits: int, act: str, n: int, table_min: int) -> str:
    """Name of the library kernel a pass runs, as the rocprofv3 summaries
    print it."""
    if kind == "bwd":
        return f"bwd32_kernel<f32,{bits}>" if dtype == "f32" else f"bwd_kernel<{dtype},{bits}>"
    if dtype == "f32":
        return f"fwd32_kernel<f32,{bits},{act}>"
    k = "fwd16_kernel" if n >= table_min else "fwd16v_kernel"
    return f"{k}<{dtype},{bits},{act}>"


def measured_traffic(workload: str, bits: int, kernel: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if
    it was taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as fh:
            d = json.load(fh)
    except (OSError, ValueError):
        return None
    if d.get("kernel_source_hash") != kernel_source_hash():
        return None
    rec = d.get("launches", {}).get(f"{workload}/b{bits}/{kernel}")
    return rec.get("hbm_bytes") if rec else None


# ---------------------------------------------------------------- rocprofv3 summaries
DT_NAMES = {0: "f32", 1: "f16", 2: "bf16"}
ACT_NAMES = {0: "gelu", 1: "silu", 2: "sigmoid", 3: "tanh", 4: "relu", 5: "selu", 6: "softplus"}


def _kernel_key(name: str):
    """'fwd16_kernel<bf16,3,gelu>' style key of a library kernel named in a
    rocprofv3 csv, 'ceiling_fwd<64>' style for the streaming reference
    kernels, or the plain name for any other kernel."""
    import re
    m = re.search(r"stream_kernel<([0-9]), ?([0-9]), ?([0-9]+), ?(true|false)>", name)
    if m:
        kind = {"0": "copy", "1": "fwd", "2": "bwd"}[m.group(1)]
        return f"ceiling_{kind}<{m.group(3)}{',paired' if m.group(4) == 'true' else ''}>"
    m = re.search(r"persist_kernel<([0-9]), ?([0-9])>", name)
    if m:
        return f"ceiling_{ {'0': 'copy', '1': 'fwd', '2': 'bwd'}[m.group(1)]}<persistent>"
    m = re.search(r"(fwd16v_kernel|fwd16_kernel|fwd32_kernel|bwd32_kernel|bwd_kernel)<([0-9, ]+)>", name)
    if not m:
        base = name.replace("(anonymous namespace)::", "").replace("void ", "")
        return base.split("(")[0].strip() or name
    args = [int(a) for a in m.group(2).split(",")]
    if m.group(1) in ("fwd16_kernel", "fwd16v_kernel"):
        return f"{m.group(1)}<{DT_NAMES[args[0]]},{args[1]},{ACT_NAMES[args[2]]}>"
    if m.group(1) == "fwd32_kernel":
        return f"fwd32_kernel<f32,{args[0]},{ACT_NAMES[args[1]]}>"
    if m.group(1) == "bwd32_kernel":
        return f"bwd32_kernel<f32,{args[0]}>"
    return f"bwd_kernel<{DT_NAMES[args[0]]},{args[1]}>"


def _csv(path):
    import csv
    with open(path, newline="") as fh:
        return list(csv.DictReader(fh))


def _one(directory, suffix):
    import glob
    hits = sorted(glob.glob(os.path.join(directory, "**", "*" + suffix), recursive=True))
    if not hits:
        raise SystemExit(f"no *{suffix} under {directory}")
    return hits[0]


def summarize_rocprof(trace_dir, fetch_dir, write_dir, workload, bits, out_traffic):
    """Print the per-kernel summary of a `rocprofv3 --kernel-trace --stats`
    run and, given the two counter runs (FETCH_SIZE, WRITE_SIZE), the HBM
    bytes per launch of the library kernels, calibrated against the
    benchmark's streaming copy kernel of the same runs (which reads and
    writes `copy_bytes` each); optionally store those bytes in
    profiles/traffic.json."""
    import workloads as WL
    w = WL.WORKLOADS[workload]
    s = 4 if w.dtype == "f32" else 2
    alg = algorithmic_bytes(w.n, w.dtype, bits)
    tiles = w.n // 512
    # the streaming reference kernels move whole tiles only
    ceil_bytes = {"copy": tiles * 1024 * s, "fwd": algorithmic_bytes(tiles * 512, w.dtype, bits),
                  "bwd": algorithmic_bytes(tiles * 512, w.dtype, bits)}
    copy_bytes = tiles * 512 * s            # the copy kernel's bytes each way
    lines = []
    if trace_dir:
        lines.append("kernel                              calls   avg_us     min_us     max_us   "
                     "alg_GB/s  frac_8TB/s")
        for r in _csv(_one(trace_dir, "kernel_stats.csv")):
            key = _kernel_key(r["Name"])
            avg = float(r["AverageNs"]) / 1e3
            if key.startswith(("fwd", "bwd")):
                b = alg
            elif key.startswith("ceiling_"):
                b = ceil_bytes[key.split("_")[1].split("<")[0]]
            else:
                b = None            # not a streaming kernel of this workload
            rate = (f"{b / (avg * 1e-6) / 1e9:10.1f} {b / (avg * 1e-6) / 1e9 / HBM_PEAK_GBPS:10.4f}"
                    if b else f"{'-':>10s} {'-':>10s}")
            lines.append(f"{key:34s} {int(r['Calls']):6d} {avg:9.2f} {float(r['MinNs']) / 1e3:10.2f} "
                         f"{float(r['MaxNs']) / 1e3:10.2f} {rate}")
    traffic = {}
    if fetch_dir and write_dir:
        per = {}
        for counter, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
            for r in _csv(_one(d, "counter_collection.csv")):
                if r["Counter_Name"] != counter:
                    continue
                key = _kernel_key(r["Kernel_Name"])
                per.setdefault(key, {}).setdefault(counter, []).append(
                    float(r["Counter_Value"]) * 1024.0)
        copy = [k for k in per if k.startswith("ceiling_copy")]
        if not copy:
            raise SystemExit("no streaming copy kernel in the counter runs to calibrate against")
        cp = per[copy[0]]
        f_fetch = copy_bytes / (sum(cp["FETCH_SIZE"]) / len(cp["FETCH_SIZE"]))
        f_write = copy_bytes / (sum(cp["WRITE_SIZE"]) / len(cp["WRITE_SIZE"]))
        lines.append("")
        lines.append(f"calibration on {copy[0]} ({copy_bytes} B read + {copy_bytes} B written "
                     f"per launch): FETCH_SIZE x {f_fetch:.4f}, WRITE_SIZE x {f_write:.4f}")
        lines.append("kernel                              launches  fetch_B        write_B        "
                     "hbm_B          alg_B          hbm/alg")
        for key, c in sorted(per.items()):
            if not key.startswith(("fwd", "bwd")) or "FETCH_SIZE" not in c or "WRITE_SIZE" not in c:
                continue
            fb = f_fetch * sum(c["FETCH_SIZE"]) / len(c["FETCH_SIZE"])
            wb = f_write * sum(c["WRITE_SIZE"]) / len(c["WRITE_SIZE"])
            lines.append(f"{key:34s} {len(c['FETCH_SIZE']):8d}  {fb:14.0f} {wb:14.0f} "
                         f"{fb + wb:14.0f} {alg:14.0f} {(fb + wb) / alg:8.4f}")
            kind = "fwd" if key.startswith("fwd") else "bwd"
            traffic[f"{workload}/b{bits}/{kind}"] = {
                "kernel": key, "fetch_bytes": round(fb), "write_bytes": round(wb),
                "hbm_bytes": round(fb + wb), "algorithmic_bytes": alg,
                "calibration": {"kernel": copy[0], "bytes_each_way": copy_bytes,
                                "fetch_factor": f_fetch, "write_factor": f_write}}
        if out_traffic:
            # keep the other workloads' entries taken on the same kernel source
            path = os.path.join(ROOT, "profiles", "traffic.json")
            launches = {}
            try:
                with open(path) as fh:
                    old = json.load(fh)
                if old.get("kernel_source_hash") == kernel_source_hash():
                    launches = old.get("launches", {})
            except (OSError, ValueError):
                pass
            launches.update(traffic)
            rec = {"kernel_source_hash": kernel_source_hash(),
                   "launches": dict(sorted(launches.items()))}
            with open(os.path.join(ROOT, "profiles", "traffic.json"), "w") as fh:
                json.dump(rec, fh, indent=1)
                fh.write("\n")
    print("\n".join(lines))


SQ_DERIVED_NOTE = ("per element = x 64 lanes / elements; LDS conflict cycles per LDS "
                   "instruction; waiting share = SQ_WAIT_ANY / SQ_WAVE_CYCLES; VALU busy = "
                   "SQ_ACTIVE_INST_VALU / SQ_BUSY_CU_CYCLES")


def summarize_sq(dirs, workload):
    """Average per dispatch of the SQ counters of one or more `rocprofv3
    --pmc` runs, per kernel, and a few ratios for the library kernels."""
    import workloads as WL
    w = WL.WORKLOADS[workload]
    per = {}
    order = []
    for d in dirs:
        for r in _csv(_one(d, "counter_collection.csv")):
            key = _kernel_key(r["Kernel_Name"])
            name = r["Counter_Name"]
            if name not in order:
                order.append(name)
            per.setdefault(key, {}).setdefault(name, {}).setdefault(r["Dispatch_Id"], 0.0)
            per[key][name][r["Dispatch_Id"]] += float(r["Counter_Value"])
    # the library kernels, and the plain streaming copy for reference
    keys = sorted((k for k in per if k.startswith(("fwd", "bwd")) or k == "ceiling_copy<64>"),
                  key=lambda k: (not k.startswith(("fwd", "bwd")), k))
    avg = {k: {c: sum(v.values()) / len(v) for c, v in per[k].items()} for k in keys}
    lines = ["counter                  " + "".join(f"{k[:30]:>32s}" for k in keys)]
    for c in order:
        lines.append(f"{c:24s} " + "".join(
            f"{avg[k][c]:32.4g}" if c in avg[k] else f"{'-':>32s}" for k in keys))
    lines.append("")
    lines.append(f"# derived ({SQ_DERIVED_NOTE}; {w.n:,} elements):")
    for k in keys:
        if not k.startswith(("fwd", "bwd")):
            continue
        a = avg[k]
        parts = []
        if "SQ_INSTS_VALU" in a:
            parts.append(f"VALU instructions per element {a['SQ_INSTS_VALU'] * 64 / w.n:.2f}")
        if "SQ_INSTS_LDS" in a:
            parts.append(f"LDS instructions per element {a['SQ_INSTS_LDS'] * 64 / w.n:.2f}")
        if "SQ_LDS_BANK_CONFLICT" in a and a.get("SQ_INSTS_LDS"):
            parts.append(f"LDS conflict cycles per LDS instruction "
                         f"{a['SQ_LDS_BANK_CONFLICT'] / a['SQ_INSTS_LDS']:.2f}")
        if "SQ_WAIT_ANY" in a and a.get("SQ_WAVE_CYCLES"):
            parts.append(f"waiting share {a['SQ_WAIT_ANY'] / a['SQ_WAVE_CYCLES']:.2f}")
        if "SQ_ACTIVE_INST_VALU" in a and a.get("SQ_BUSY_CU_CYCLES"):
            parts.append(f"VALU busy {a['SQ_ACTIVE_INST_VALU'] / a['SQ_BUSY_CU_CYCLES']:.2f}")
        lines.append(f"#   {k}: " + ", ".join(parts))
    print("\n".join(lines))


def cpu_baseline(w, bits, x_np, g_np, seconds=10.0, chunk=1 << 22):
    """The oracle on the host: its threaded mode on the host's cores (at
    most 16, the CPU share of one GPU) over the whole input, or until
    `seconds` of wall time, then its single-threaded mode for `seconds`.
    It uses the oracle's own fitted table (tests/golden/tables.json)."""
    import numpy as np
    import oracle as O
    act = {"gelu": O.GELU, "silu": O.SILU, "sigmoid": O.SIGMOID, "tanh": O.TANH}[w.act]
    odt = {"f32": O.F32, "f16": O.F16, "bf16": O.BF16}[w.dtype]
    with open(os.path.join(ROOT, "tests", "golden", "tables.json")) as fh:
        spec = json.load(fh)[f"{w.name}/b{bits}"]
    s = np.float32([float.fromhex(h) for h in spec["s"]])
    v = np.float32([float.fromhex(h) for h in spec["v"]])

    def run(threads, budget):
        done, t_total, pos = 0, 0.0, 0
        while t_total < budget and pos < x_np.size:
            xs = x_np[pos:pos + chunk * threads]
            gs = g_np[pos:pos + chunk * threads]
            t0 = time.perf_counter()
            _, codes = O.fwd(act, odt, bits, s, xs, threads=threads)
            O.bwd(odt, bits, v, gs, codes, threads=threads)
            t_total += time.perf_counter() - t0
            done += xs.size
            pos += xs.size
        return done, t_total

    per_elem = algorithmic_bytes(1, w.dtype, bits) * 2        # fwd + bwd bytes per element
    host = host_cpu()
    # one GPU's share of the host: the GPU machines give each GPU 16 CPUs, so the
    # threaded oracle uses at most 16 threads whatever the host has
    threads = max(1, min(16, host["cpus"]))
    n_mt, t_mt = run(threads, seconds)
    n_st, t_st = run(1, seconds)
    return {
        "value": round(n_mt / t_mt * per_elem / 1e9, 4),
        "unit": "GB/s",
        "cores": threads,
        "kind": "oracle",
        "host_cpus": host["cpus"],
        "cpu_model": host["model"],
        "threads_why": "at most 16 threads: one GPU's CPU share on this machine",
        "elements_per_s": round(n_mt / t_mt, 1),
        "single_thread": {"value": round(n_st / t_st * per_elem / 1e9, 4), "unit": "GB/s",
                          "elements_per_s": round(n_st / t_st, 1)},
        "sample": f"first {n_mt} elements of the same workload, forward + backward, scalar C "
                  f"oracle in double, {threads} threads, {t_mt:.1f} s; single thread: first "
                  f"{n_st} elements, {t_st:.1f} s",
    }


def host_cpu() -> dict:
    """Logical CPUs of this host and their model name (/proc/cpuinfo)."""
    model = None
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"cpus": os.cpu_count() or 1, "model": model}


def sweep(n: int, steps: int, warmup: int) -> None:
    """Forward and backward of every activation x storage type x bit width on
    n seeded synthetic elements (x ~ N(0, 3^2), grad_out ~ N(0, 1)), tables
    fitted under N(0, 3^2) on [-30, 30]; HIP events on the launch stream,
    inputs resident in HBM.  One JSON line per combination."""
    import numpy as np
    import torch
    import paper_2202_00441_amd as P
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    gen = torch.Generator(device=dev).manual_seed(5)
    x32 = torch.randn(n, device=dev, generator=gen) * 3.0
    g32 = torch.randn(n, device=dev, generator=gen)
    stream = torch.cuda.current_stream()
    for dtype, tdt in (("f32", torch.float32), ("f16", torch.float16), ("bf16", torch.bfloat16)):
        x, g = x32.to(tdt), g32.to(tdt)
        y, gin = torch.empty_like(x), torch.empty_like(g)
        for act in ("gelu", "silu", "sigmoid", "tanh", "relu", "selu", "softplus"):
            for bits in (1, 2, 3, 4):
                table = P.fit_table(act, bits, P.Weight(P.W_NORMAL, -30.0, 30.0, 0.0, 3.0), 2000)
                codes = torch.empty(P.packed_words(n, bits), dtype=torch.int32, device=dev)
                for _ in range(warmup):
                    P.fwd(table, x, y=y, codes=codes)
                    P.bwd(table, g, codes, grad_in=gin)
                ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
                torch.cuda.synchronize()
                for k in range(steps):
                    ev[k][0].record(stream)
                    P.fwd(table, x, y=y, codes=codes)
                    ev[k][1].record(stream)
                    P.bwd(table, g, codes, grad_in=gin)
                    ev[k][2].record(stream)
                torch.cuda.synchronize()
                fwd_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
                bwd_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in ev]))
                b = algorithmic_bytes(n, dtype, bits)
                print(json.dumps({
                    "act": act, "dtype": dtype, "bits": bits, "n": n,
                    "fwd_kernel": kernel_name("fwd", dtype, bits, act, n,
                                              0 if dtype == "f32" else P.fwd16_table_min(act, bits, dtype)),
                    "fwd_ms": round(fwd_ms, 5), "fwd_frac_peak": round(b / (fwd_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                    "bwd_ms": round(bwd_ms, 5), "bwd_frac_peak": round(b / (bwd_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                }), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="gelu_bf16_lm_ffn_16x2048x8192")
    ap.add_argument("--bits", type=int, default=3)
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--fwd-kernel", choices=("auto", "table", "element"), default="auto",
                    help="fp16 / bf16 forward kernel: the library's choice by size (auto), or "
                         "forced with the table's kernel-choice flags (diagnostics)")
    ap.add_argument("--memory", action="store_true",
                    help="report activation memory held for backward, vanilla vs few-bit, on a "
                         "GPT-2-small-shaped stack of feed-forward blocks, instead of timing")
    ap.add_argument("--sweep", action="store_true",
                    help="time forward and backward for every activation, storage type and bit "
                         "width on --sweep-n elements (one JSON line each) instead of the headline")
    ap.add_argument("--sweep-n", type=int, default=1 << 26)
    ap.add_argument("--all-configs", action="store_true",
                    help="every workload and bit width: back-to-back and cold kernel times, "
                         "same-run ceilings and fit time, one JSON line each")
    ap.add_argument("--summarize-trace", metavar="DIR",
                    help="summarise a rocprofv3 --kernel-trace --stats output directory")
    ap.add_argument("--summarize-counters", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="calibrated HBM bytes from FETCH_SIZE and WRITE_SIZE runs")
    ap.add_argument("--summarize-sq", nargs="+", metavar="PMC_DIR",
                    help="print per-kernel averages of the SQ counters of rocprofv3 --pmc runs")
    ap.add_argument("--write-traffic", action="store_true",
                    help="with --summarize-counters: store profiles/traffic.json")
    args = ap.parse_args()

    if args.summarize_sq:
        summarize_sq(args.summarize_sq, args.workload)
        return
    if args.summarize_trace or args.summarize_counters:
        fd, wd = args.summarize_counters or (None, None)
        summarize_rocprof(args.summarize_trace, fd, wd, args.workload, args.bits,
                          args.write_traffic)
        return

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: this path runs on one GPU; figures for more than one GPU are not "
              "measured here (the method is pointwise and shards without communication).",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import workloads as WL
    import paper_2202_00441_amd as P

    if args.memory:
        from paper_2202_00441_amd.memory import compare
        torch.cuda.set_device(0)
        rows = []
        for dtype in (torch.bfloat16, torch.float32):
            for bits in (1, 2, 3, 4):
                rows.append(compare(d=768, d_ff=3072, layers=12, tokens=8 * 256, bits=bits,
                                    dtype=dtype))
        print(json.dumps({
            "metric": "activation memory held for backward, vanilla vs few-bit GELU",
            "config": {"workload": "12 feed-forward blocks x -> x + W2 GELU(W1 x), d 768, "
                                   "d_ff 3072 (GPT-2 small), 8 x 256 tokens, random weights"},
            "rows": rows,
        }), flush=True)
        return

    if args.sweep:
        sweep(args.sweep_n, args.steps, args.warmup)
        return

    if args.all_configs:
        all_configs(args)
        return

    w = WL.WORKLOADS[args.workload]
    bits = args.bits
    assert bits in w.bits, f"{w.name} runs bits {w.bits}"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    t0 = time.time()
    x_np, g_np = WL.inputs(w)
    print(f"[bench] generated {w.name} n={w.n} in {time.time() - t0:.1f}s", file=sys.stderr,
          flush=True)
    x, g = _upload(x_np, w.dtype, dev), _upload(g_np, w.dtype, dev)
    y = torch.empty_like(x)
    gin = torch.empty_like(g)
    n = w.n
    codes = torch.empty(P.packed_words(n, bits), dtype=torch.int32, device=dev)

    table, fit_ms = fit_timed(P, w, bits)
    table = table.with_flags(table.flags | fwd_kernel_flag(P, args.fwd_kernel))

    def step():
        P.fwd(table, x, y=y, codes=codes)
        P.bwd(table, g, codes, grad_in=gin)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # per-kernel events on the stream the kernels are launched on
    stream = torch.cuda.current_stream()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for k in range(args.steps):
        ev[k][0].record(stream)
        P.fwd(table, x, y=y, codes=codes)
        ev[k][1].record(stream)
        P.bwd(table, g, codes, grad_in=gin)
        ev[k][2].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    print(f"[bench] {args.steps} timed steps done", file=sys.stderr, flush=True)

    fwd_ms = [ev[k][0].elapsed_time(ev[k][1]) for k in range(args.steps)]
    bwd_ms = [ev[k][1].elapsed_time(ev[k][2]) for k in range(args.steps)]
    fwd_avg = sum(fwd_ms) / len(fwd_ms)
    bwd_avg = sum(bwd_ms) / len(bwd_ms)
    bytes_pass = algorithmic_bytes(n, w.dtype, bits)
    ms_per_step = wall * 1e3 / args.steps
    gbps = 2 * bytes_pass / (ms_per_step * 1e-3) / 1e9

    # what this device streams for the same byte mixes, same run
    ceil = ceilings(x, y, g, gin, codes, n, bits)
    # the same kernels cold (1 GiB copied through the caches before each)
    cold = cold_times(P, table, x, y, g, gin, codes, reps=10)
    print("[bench] ceilings and cold runs done", file=sys.stderr, flush=True)

    dom = "fwd" if fwd_avg >= bwd_avg else "bwd"
    dom_ms = fwd_avg if dom == "fwd" else bwd_avg
    achieved = bytes_pass / (dom_ms * 1e-3) / 1e9
    traffic = measured_traffic(w.name, bits, dom)

    out = {
        "metric": METRIC,
        "value": round(gbps, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        # arithmetic of the path: f, the compares and the gradient products in
        # fp32 (the 16-bit forward looks up outputs evaluated in fp32);
        # tensors are stored in the workload's type
        "dtype": "f32",
        "storage_dtype": w.dtype,
        "data": "synthetic (seeded numpy draws, see workloads.py)",
        "config": config_of(w, bits),
        "pct_hbm_peak": round(100 * gbps / HBM_PEAK_GBPS, 2),
        "elements_per_s": round(2 * n / (ms_per_step * 1e-3), 1),
        "fwd": kernel_record(fwd_ms, bytes_pass, n, ceil["fwd"]),
        "bwd": kernel_record(bwd_ms, bytes_pass, n, ceil["bwd"]),
        "cold": {k: stats_record(v, bytes_pass) for k, v in cold.items()} | {
            "what": "each kernel alone after 1 GiB copied through the caches (10 runs, outside "
                    "the timed steps)"},
        "ceiling": ceil,
        "fit_ms": fit_ms,
        "roofline": {
            "kernel": kernel_name(dom, w.dtype, bits, w.act, n, forced_min(P, w, bits, args.fwd_kernel)),
            "bound": "hbm",
            "achieved": round(achieved, 2),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBPS, 4),
            "traffic": traffic,
            "bytes_per_launch": bytes_pass,
            "avg_launch_ms": round(dom_ms, 5),
            "ceiling_GB/s": ceil[dom]["GB/s"],
            "frac_of_ceiling": round(achieved / ceil[dom]["GB/s"], 4),
        },
        "cpu_baseline": None,
        # context only, not a target: the memory the method saves, as the
        # paper's memory table (Sec. 4) reports it for whole models (share of
        # activation memory, per bit width; hardware not stated).  bench.py
        # --memory measures the same mechanism on a synthetic GPT-2-small
        # feed-forward stack.
        "paper_context": {
            "what": "memory saving of few-bit activations, paper's memory table (Sec. 4), hardware not stated",
            "saving_by_bits": {"GPT-2 (seq 256)": [0.42, 0.41, 0.39, 0.38],
                               "RoBERTa-base (seq 256)": [0.16, 0.15, 0.15, 0.14],
                               "ResNet-101 (256x256)": [0.30, 0.29, 0.28, 0.27]},
            "bits": [1, 2, 3, 4],
        },
    }
    fwd_kernel = kernel_name("fwd", w.dtype, bits, w.act, n, forced_min(P, w, bits, args.fwd_kernel))
    out["fwd"]["kernel"] = fwd_kernel
    out["bwd"]["kernel"] = kernel_name("bwd", w.dtype, bits, w.act, n, 0)
    if args.fwd_kernel != "auto":
        out["fwd_kernel_forced"] = args.fwd_kernel
    if fwd_kernel.startswith("fwd16_kernel"):
        # the table forward runs one persistent workgroup per CU: its rate
        # against what that launch shape streams for the same bytes
        out["fwd"]["frac_of_persistent_shape"] = round(
            bytes_pass / (fwd_avg * 1e-3) / 1e9 / ceil["fwd_persistent_shape"]["GB/s"], 4)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, bits, x_np, g_np, args.cpu_seconds)
    print(json.dumps(out), flush=True)


# ---------------------------------------------------------------- timing helpers
def _upload(a, dtype: str, dev):
    import numpy as np
    import torch
    view = np.int32 if dtype == "f32" else np.int16
    tdt = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[dtype]
    return torch.from_numpy(a.view(view)).to(dev).view(tdt)


def table_min(P, w, bits: int) -> int:
    """Size from which the workload's fp16 / bf16 forward runs the table
    kernel (0 for fp32, which has none)."""
    return 0 if w.dtype == "f32" else P.fwd16_table_min(w.act, bits, w.dtype)


def fwd_kernel_flag(P, choice: str) -> int:
    """Kernel-choice flag for a forced fp16 / bf16 forward kernel (0: the
    library's choice by size)."""
    return {"auto": 0, "table": P.FLAG_TABLE_FWD, "element": P.FLAG_ELEMENT_FWD}[choice]


def forced_min(P, w, bits: int, choice: str) -> int:
    """table_min as the forced choice makes it: 0 (always the table kernel)
    or never."""
    if choice == "table":
        return 0
    if choice == "element":
        return 2 ** 63 - 1
    return table_min(P, w, bits)


def config_of(w, bits: int) -> dict:
    return {
        "workload": f"{w.name}: {w.act.upper()} {bits}-bit {w.dtype} {list(w.shape)}",
        "act": w.act, "bits": bits, "shape": list(w.shape), "n": w.n,
        "x": {"normal": f"N(0,{w.x_scale}^2)",
              "mixture": f"0.99 N(0,{w.x_scale}^2) + 0.01 N(0,{10 * w.x_scale}^2)",
              "uniform": f"U(-{w.x_scale},{w.x_scale})"}[w.x_dist],
        "grad_out": f"N(0,{w.g_sigma}^2)",
        "table": f"fewbit_fit_table {w.fit}",
    }


def fit_timed(P, w, bits: int, reps: int = 3):
    """The workload's table from the host fit (Sec. 3, done once per
    activation), and the fit's wall time in ms over `reps` fits."""
    ts, table = [], None
    for _ in range(reps):
        t0 = time.perf_counter()
        table = P.fit_table(w.act, bits, P.Weight.from_spec(w.fit), w.fit["n_grid"])
        ts.append((time.perf_counter() - t0) * 1e3)
    return table, {"min": round(min(ts), 3), "mean": round(sum(ts) / len(ts), 3),
                   "n_grid": w.fit["n_grid"], "reps": reps}


def stats_record(ms, bytes_pass: float) -> dict:
    import statistics
    med = statistics.median(ms)
    return {"ms": round(sum(ms) / len(ms), 5), "median_ms": round(med, 5),
            "min_ms": round(min(ms), 5),
            "frac_peak": round(bytes_pass / (sum(ms) / len(ms) * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
            "frac_peak_median": round(bytes_pass / (med * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4)}


def kernel_record(ms, bytes_pass: float, n: int, ceil) -> dict:
    avg = sum(ms) / len(ms)
    rec = {"GB/s": round(bytes_pass / (avg * 1e-3) / 1e9, 2),
           "elements_per_s": round(n / (avg * 1e-3), 1)} | stats_record(ms, bytes_pass)
    if ceil:
        rec["frac_of_ceiling"] = round(bytes_pass / (avg * 1e-3) / 1e9 / ceil["GB/s"], 4)
    return rec


def _events(stream, fn, reps: int):
    """Per-launch ms of `reps` back-to-back launches of fn on `stream`."""
    import torch
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(reps)]
    for e0, e1 in ev:
        e0.record(stream)
        fn()
        e1.record(stream)
    torch.cuda.synchronize()
    return [e0.elapsed_time(e1) for e0, e1 in ev]


def ceilings(x, y, g, gin, codes, n: int, bits: int, reps: int = 20) -> dict:
    """Rate of the streaming reference kernels (ceiling/ceiling.hip) on the
    workload's own buffers: a copy of x, the forward's byte mix (read x,
    write y and the codes) and the backward's (read grad_out and the codes,
    write grad_in), each over the whole 512-element tiles, in its fastest
    launch shape (one wave per tile: 64 or 256 threads per workgroup in tile
    order, or 64 threads with tiles 2p and 2p+1 on one XCD) by the median of
    `reps` back-to-back launches."""
    import torch
    import ceiling as CL
    stream = torch.cuda.current_stream()
    tiles = n // 512
    out = {}
    for kind, src, dst in (("copy", x, y), ("fwd", x, y), ("bwd", g, gin)):
        b = tiles * CL.tile_bytes(kind, src.element_size(), bits)
        best = None
        for shape in CL.SHAPES:
            def fn(kind=kind, shape=shape, src=src, dst=dst):
                CL.stream(kind, shape, src, dst, None if kind == "copy" else codes, tiles, bits)
            for _ in range(3):
                fn()
            rec = stats_record(_events(stream, fn, reps), b)
            rec = {"GB/s": round(b / (rec["median_ms"] * 1e-3) / 1e9, 2),
                   "shape": {64: "64 threads", 256: "256 threads", 65: "64 threads, paired"}[shape],
                   "bytes": b} | rec
            if best is None or rec["median_ms"] < best["median_ms"]:
                best = rec
        out[kind] = best
    # the forward mix in the 16-bit table forward's own launch shape (one
    # persistent workgroup per CU): what that shape streams, not a ceiling
    b = tiles * CL.tile_bytes("fwd", x.element_size(), bits)

    def fn():
        CL.stream("fwd", CL.PERSISTENT, x, y, codes, tiles, bits)
    for _ in range(3):
        fn()
    rec = stats_record(_events(stream, fn, reps), b)
    out["fwd_persistent_shape"] = {"GB/s": round(b / (rec["median_ms"] * 1e-3) / 1e9, 2),
                                   "shape": "persistent, one 512-thread workgroup per CU",
                                   "bytes": b} | rec
    out["what"] = ("streaming reference kernels moving the same bytes (16-byte non-temporal "
                   "buffer accesses, one wave per 512-element tile); GB/s by the median launch; "
                   "fwd_persistent_shape: the forward mix in the table forward's launch shape")
    return out


def cold_times(P, table, x, y, g, gin, codes, reps: int = 10) -> dict:
    """Each pass alone after 1 GiB has been copied through the caches, so
    nothing of the previous pass is left in the 256 MB memory-side cache."""
    import torch
    dev = x.device
    stream = torch.cuda.current_stream()
    fl_src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
    fl_dst = torch.empty_like(fl_src)
    cold = {"fwd": [], "bwd": []}
    for _ in range(reps):
        for which in ("fwd", "bwd"):
            fl_dst.copy_(fl_src)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            if which == "fwd":
                P.fwd(table, x, y=y, codes=codes)
            else:
                P.bwd(table, g, codes, grad_in=gin)
            e1.record(stream)
            torch.cuda.synchronize()
            cold[which].append(e0.elapsed_time(e1))
    del fl_src, fl_dst
    return cold


def all_configs(args) -> None:
    """Every workload and bit width: back-to-back and cold per-kernel times,
    the same-run ceilings for its byte mixes and the fit time; one JSON line
    each.  The small workloads fit in the memory-side cache, so their cold
    figures are the ones that count."""
    import torch
    import workloads as WL
    import paper_2202_00441_amd as P
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    for name, w in WL.WORKLOADS.items():
        x_np, g_np = WL.inputs(w)
        x, g = _upload(x_np, w.dtype, dev), _upload(g_np, w.dtype, dev)
        del x_np, g_np
        y, gin = torch.empty_like(x), torch.empty_like(g)
        for bits in w.bits:
            codes = torch.empty(P.packed_words(w.n, bits), dtype=torch.int32, device=dev)
            table, fit_ms = fit_timed(P, w, bits)
            table = table.with_flags(fwd_kernel_flag(P, args.fwd_kernel))
            for _ in range(args.warmup):
                P.fwd(table, x, y=y, codes=codes)
                P.bwd(table, g, codes, grad_in=gin)
            fwd = _events(stream, lambda: P.fwd(table, x, y=y, codes=codes), args.steps)
            bwd = _events(stream, lambda: P.bwd(table, g, codes, grad_in=gin), args.steps)
            b = algorithmic_bytes(w.n, w.dtype, bits)
            ceil = ceilings(x, y, g, gin, codes, w.n, bits)
            cold = cold_times(P, table, x, y, g, gin, codes, reps=10)
            tm = forced_min(P, w, bits, args.fwd_kernel)
            fk = kernel_name("fwd", w.dtype, bits, w.act, w.n, tm)
            fwd_rec = kernel_record(fwd, b, w.n, ceil["fwd"])
            if fk.startswith("fwd16_kernel"):
                fwd_rec["frac_of_persistent_shape"] = round(
                    b / (sum(fwd) / len(fwd) * 1e-3) / 1e9 / ceil["fwd_persistent_shape"]["GB/s"], 4)
            print(json.dumps({
                "config": config_of(w, bits), "storage_dtype": w.dtype,
                "bytes_per_pass": b,
                "fwd_kernel": fk,
                "bwd_kernel": kernel_name("bwd", w.dtype, bits, w.act, w.n, tm),
                "fwd": fwd_rec,
                "bwd": kernel_record(bwd, b, w.n, ceil["bwd"]),
                "cold": {"fwd": kernel_record(cold["fwd"], b, w.n, None),
                         "bwd": kernel_record(cold["bwd"], b, w.n, None),
                         "step_frac_peak": round(2 * b / ((sum(cold["fwd"]) + sum(cold["bwd"]))
                                                          / len(cold["fwd"]) * 1e-3) / 1e9
                                                 / HBM_PEAK_GBPS, 4)},
                "ceiling": ceil, "fit_ms": fit_ms,
            }), flush=True)
            del codes
        del x, g, y, gin
        torch.cuda.empty_cache()


if __name__ == "__main__":
    main()
