"""Throughput of one pipeline stage's work per mini-batch on one MI355X.

Workload (default): partition 1 of the 4-way split of a 5-level U-Net
(base 64 -> 1024 channels), input 32x64x192x192 bf16 ~ N(0,1), m = 8
micro-batches, checkpoint = always.  A step is the whole stage: the m
forwards F_{i,1} (keeping only their inputs), then for i = m..1 the
recompute F'_{i,1}, the backward B_{i,1} (data gradient of the stage input
included) and the accumulation of g_i.  Upstream gradients of the stage's
output and of its three exported skips are seeded inputs, resident in HBM
with everything else before timing starts.

Prints one JSON line.  `--gpus N` with N > 1 is not supported: this build
runs on a single GPU.
"""
import argparse
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, HERE)

BF16_PEAK = 2.5e15      # MI355X dense bf16 MFMA, FLOP/s
HBM_PEAK = 8.0e12       # MI355X HBM3E, B/s


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# ---------------------------------------------------------------- profiles
# rocprofv3 summaries live in profiles/ as text.  The HBM traffic of the
# dominant kernel comes from two counter runs (FETCH_SIZE, WRITE_SIZE, KiB
# per dispatch), each scaled by what the same counter reads for a device
# copy of known size.  A summary records a hash of the kernel sources; the
# bench reports its traffic only while the sources are unchanged.
PROFILES = os.path.join(HERE, "profiles")
KERNEL_SOURCES = ["paper_2004_09910_amd/csrc/conv_mfma.hip",
                  "paper_2004_09910_amd/csrc/conv_rowtile.hip",
                  "paper_2004_09910_amd/csrc/conv_rows32.hip",
                  "paper_2004_09910_amd/csrc/wgrad_rows.hip",
                  "paper_2004_09910_amd/csrc/elementwise.hip",
                  "paper_2004_09910_amd/csrc/mfma_util.h",
                  "paper_2004_09910_amd/csrc/common.h"]
PROFILE_COMMANDS = {
    "trace": "rocprofv3 --kernel-trace --stats --output-format csv -d rocprof_out/prof_kt -o kt "
             "-- python3 bench.py --steps 10 --warmup 2 --no-cpu-baseline",
    "fetch": "rocprofv3 --pmc FETCH_SIZE --output-format csv -d rocprof_out/prof_fetch -o f "
             "-- python3 bench.py --eager --steps 1 --warmup 1 --no-cpu-baseline",
    "write": "rocprofv3 --pmc WRITE_SIZE --output-format csv -d rocprof_out/prof_write -o w "
             "-- python3 bench.py --eager --steps 1 --warmup 1 --no-cpu-baseline",
    "copy_fetch": "rocprofv3 --pmc FETCH_SIZE --output-format csv -d rocprof_out/prof_cfetch -o cf "
                  "-- python3 bench.py --copy-calibration",
    "copy_write": "rocprofv3 --pmc WRITE_SIZE --output-format csv -d rocprof_out/prof_cwrite -o cw "
                  "-- python3 bench.py --copy-calibration",
    "mfma": "rocprofv3 --pmc SQ_VALU_MFMA_BUSY_CYCLES SQ_BUSY_CU_CYCLES GRBM_GUI_ACTIVE "
            "--output-format csv -d rocprof_out/prof_mfma -o m "
            "-- python3 bench.py --eager --steps 1 --warmup 1 --no-cpu-baseline",
    "lds": "rocprofv3 --pmc SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_LDS_BANK_CONFLICT SQ_WAIT_INST_LDS "
           "SQ_INSTS_LDS SQ_WAVE_CYCLES --output-format csv -d rocprof_out/prof_lds -o l "
           "-- python3 bench.py --eager --steps 1 --warmup 1 --no-cpu-baseline",
}
N_SIMD = 1024           # MI355X: 256 CUs x 4 SIMDs
CLOCK_GHZ = 2.4         # MI355X peak engine clock


KERNEL_FILES = [("conv3x3_rows32", "conv_rows32.hip"), ("conv_wgrad_rows", "wgrad_rows.hip"),
                ("conv3x3_rowtile", "conv_rowtile.hip"), ("conv_", "conv_mfma.hip"),
                ("splitk_reduce", "conv_mfma.hip"), ("", "elementwise.hip")]


def kernel_source_hash(kernel=None):
    """Hash of the sources a kernel is built from (its own .hip file and the
    shared headers; all kernel sources when no kernel is named)."""
    import hashlib
    h = hashlib.sha256()
    files = KERNEL_SOURCES
    if kernel is not None:
        own = next(f for prefix, f in KERNEL_FILES if kernel.startswith(prefix))
        files = ["paper_2004_09910_amd/csrc/" + own, "paper_2004_09910_amd/csrc/mfma_util.h",
                 "paper_2004_09910_amd/csrc/common.h"]
    for rel in files:
        with open(os.path.join(HERE, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def short_kernel_name(full):
    """'void ns::(anonymous namespace)::k<2, 4>(int, ...)' -> 'k<2,4>'."""
    n = full.replace("(anonymous namespace)::", "")
    if n.startswith("void "):
        n = n[5:]
    depth, cut = 0, len(n)
    for i, ch in enumerate(n):
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0:
            cut = i
            break
    n = n[:cut]
    head, sep, tail = n.partition("<")
    head = head.split("::")[-1]
    n = (head + sep + tail).replace(" ", "")
    # the wave-layout template argument is named the way the launchers name
    # their profiling scopes: ",8w" / ",12w" for the eight- and twelve-wave
    # layouts, else nothing
    args = tail.rstrip(">").replace(" ", "").split(",") if sep else []
    if head == "conv3x3_rows32" and len(args) == 6:
        n = (f"{head}<{','.join(args[:4])}{',8w' if args[4] == '1' else ''}"
             f"{',rk' if args[5] != '0' else ''}>")
    elif head == "conv_wgrad_rows" and len(args) == 4:
        n = f"{head}<{','.join(args[:3])}{ {'2': ',8w', '3': ',12w'}.get(args[3], '')}>"
    return n


def _counter_means(path):
    import csv
    import glob
    sums, counts = {}, {}
    for f in glob.glob(os.path.join(path, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            k = short_kernel_name(r["Kernel_Name"])
            sums[k] = sums.get(k, 0.0) + float(r["Counter_Value"])
            counts[k] = counts.get(k, 0) + 1
    return {k: sums[k] / counts[k] for k in sums}, counts


def summarize_profiles(out_dir, workload):
    """Writes profiles/kernel_trace_<workload>.md and
    profiles/traffic_<kernel>_<workload>.md from the rocprofv3 runs listed in
    PROFILE_COMMANDS (their output under out_dir)."""
    import csv
    import glob
    import json as _json
    os.makedirs(PROFILES, exist_ok=True)
    stats_csv = glob.glob(os.path.join(out_dir, "prof_kt", "**", "*kernel_stats.csv"), recursive=True)[0]
    rows = list(csv.DictReader(open(stats_csv)))
    # per-dispatch durations: the last 10 of the 23 steps the trace command
    # runs (2 warmup, 1 replay after capture, 10 timed replays, 10 eager
    # one-stream steps) are the pass bench.py times each launch in
    trace_csv = glob.glob(os.path.join(out_dir, "prof_kt", "**", "*kernel_trace.csv"), recursive=True)[0]
    per = {}
    for r in csv.DictReader(open(trace_csv)):
        per.setdefault(short_kernel_name(r["Kernel_Name"]), []).append(
            (int(r["Start_Timestamp"]), int(r["End_Timestamp"]) - int(r["Start_Timestamp"])))
    eager = {}
    for k, v in per.items():
        v.sort()
        tail = v[len(v) - round(len(v) * 10 / 23):]
        eager[k] = sum(d for _, d in tail) / len(tail) / 1e3 if tail else float("nan")
    lines = [f"# Kernel trace: {workload}", "",
             "Command (from the repository root on the GPU host):", "",
             "    " + PROFILE_COMMANDS["trace"], "",
             "rocprofv3 `--stats` summary (all dispatches of the run: warmup, HIP-graph replays with "
             "concurrency lanes, and the eager one-stream pass that bench.py times each launch in). "
             "The last column averages only that eager pass (the last 10 of the run's 23 steps, "
             "from the per-dispatch trace).", "",
             "| kernel | calls | avg us | total ms | % | eager-pass avg us |",
             "|---|---:|---:|---:|---:|---:|"]
    for r in rows:
        nm = short_kernel_name(r['Name'])
        lines.append(f"| `{nm}` | {r['Calls']} | "
                     f"{float(r['AverageNs']) / 1e3:.2f} | {float(r['TotalDurationNs']) / 1e6:.3f} | "
                     f"{float(r['Percentage']):.2f} | {eager.get(nm, float('nan')):.2f} |")
    with open(os.path.join(PROFILES, f"kernel_trace_{workload}.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    if os.path.isdir(os.path.join(out_dir, "prof_mfma")) and os.path.isdir(os.path.join(out_dir, "prof_lds")):
        summarize_counters(out_dir, workload, eager)
    if not os.path.isdir(os.path.join(out_dir, "prof_fetch")):
        return
    top = short_kernel_name(rows[0]["Name"])
    fetch, nf = _counter_means(os.path.join(out_dir, "prof_fetch"))
    write, nw = _counter_means(os.path.join(out_dir, "prof_write"))
    cf, _ = _counter_means(os.path.join(out_dir, "prof_cfetch"))
    cw, _ = _counter_means(os.path.join(out_dir, "prof_cwrite"))
    copy_k = [k for k in cf if "copyBuffer" in k or "copy" in k.lower()]
    gib_kib = float(1 << 20)                       # 1 GiB copied, in KiB
    f_fetch = gib_kib / cf[copy_k[0]]
    f_write = gib_kib / cw[copy_k[0]]
    fb = fetch[top] * 1024 * f_fetch
    wb = write[top] * 1024 * f_write
    group = 1
    for line in open(os.path.join(out_dir, "prof_fetch.log")):
        if line.startswith("{"):
            group = int(_json.loads(line)["config"].get("group", 1))
    info = {"kernel": top, "workload": workload, "group": group, "fetch_bytes": fb, "write_bytes": wb,
            "bytes_per_launch": fb + wb, "dispatches": nf.get(top, 0),
            "fetch_scale": f_fetch, "write_scale": f_write, "source_hash": kernel_source_hash(top)}
    tl = [f"# HBM traffic of `{top}`: {workload}", "",
          "Commands (from the repository root on the GPU host):", ""]
    for k in ("fetch", "write", "copy_fetch", "copy_write"):
        tl.append("    " + PROFILE_COMMANDS[k])
    tl += ["",
           f"- FETCH_SIZE, mean per dispatch: {fetch[top]:.1f} KiB over {nf.get(top, 0)} dispatches; "
           f"a 1 GiB device copy reads {cf[copy_k[0]]:.1f} KiB, so the scale is {f_fetch:.4f}.",
           f"- WRITE_SIZE, mean per dispatch: {write[top]:.1f} KiB over {nw.get(top, 0)} dispatches; "
           f"the copy writes {cw[copy_k[0]]:.1f} KiB, scale {f_write:.4f}.",
           f"- Launches: {group} micro-batch{'es' if group > 1 else ''} per launch.",
           f"- HBM bytes per launch: {fb / 1e6:.2f} MB read + {wb / 1e6:.2f} MB written = "
           f"{(fb + wb) / 1e6:.2f} MB.", "",
           "Other kernels of the same runs (mean KiB per dispatch, unscaled):", "",
           "| kernel | FETCH_SIZE | WRITE_SIZE |", "|---|---:|---:|"]
    for k in sorted(fetch, key=lambda k: -fetch[k] * nf[k])[:12]:
        tl.append(f"| `{k}` | {fetch[k]:.1f} | {write.get(k, float('nan')):.1f} |")
    tl += ["", "traffic_json: " + _json.dumps(info)]
    safe = top.replace("<", "_").replace(">", "").replace(",", "_")
    with open(os.path.join(PROFILES, f"traffic_{safe}_{workload}.md"), "w") as f:
        f.write("\n".join(tl) + "\n")
    print(_json.dumps(info))


def _counters_by_kernel(path):
    """{kernel: {counter: [value per dispatch]}} from a rocprofv3 --pmc run
    (each value summed over the counter's dimensions), plus the dispatches'
    durations in ns under '_ns'."""
    import csv
    import glob
    out = {}
    for f in glob.glob(os.path.join(path, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            k = short_kernel_name(r["Kernel_Name"])
            d = out.setdefault(k, {})
            d.setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
            if r["Counter_Name"] == "SQ_VALU_MFMA_BUSY_CYCLES":
                d.setdefault("_ns", []).append(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
    return out


def summarize_counters(out_dir, workload, eager_us=None):
    """Writes profiles/counters_<workload>.md from the two counter runs
    (PROFILE_COMMANDS 'mfma' and 'lds') over one eager step.

    Per kernel, means per dispatch of:
      MFMA GFLOP    512 x SQ_INSTS_VALU_MFMA_MOPS_BF16 (the counter is the
                    multiply and add operations divided by 512);
      FLOP / busy   MFMA FLOP per SQ_VALU_MFMA_BUSY_CYCLES summed over SIMDs
                    (1024 is the full dense bf16 rate of one SIMD);
      MFMA busy     SQ_VALU_MFMA_BUSY_CYCLES / (1024 SIMDs x duration x
                    2.4 GHz), with the duration of the counter run's own
                    dispatches and with the eager-pass duration of the kernel
                    trace;
      LDS           bank-conflict cycles per LDS instruction, and the share of
                    wave time spent waiting to issue an LDS instruction
                    (SQ_WAIT_INST_LDS / SQ_WAVE_CYCLES, both in quad-cycles)."""
    import math
    a = _counters_by_kernel(os.path.join(out_dir, "prof_mfma"))
    b = _counters_by_kernel(os.path.join(out_dir, "prof_lds"))

    def mean(d, k, c):
        v = d.get(k, {}).get(c)
        return sum(v) / len(v) if v else float("nan")
    rows = []
    for k in a:
        busy = mean(a, k, "SQ_VALU_MFMA_BUSY_CYCLES")
        us_c = mean(a, k, "_ns") / 1e3
        flop = 512.0 * mean(b, k, "SQ_INSTS_VALU_MFMA_MOPS_BF16")
        lds = mean(b, k, "SQ_INSTS_LDS")
        conf = mean(b, k, "SQ_LDS_BANK_CONFLICT")
        wait = mean(b, k, "SQ_WAIT_INST_LDS")
        wave = mean(b, k, "SQ_WAVE_CYCLES")
        us = (eager_us or {}).get(k, float("nan"))
        rows.append({"kernel": k, "dispatches": len(a[k].get("_ns", [])), "us_c": us_c, "us": us,
                     "busy_c": busy / (N_SIMD * us_c * CLOCK_GHZ * 1e3),
                     "busy_e": busy / (N_SIMD * us * CLOCK_GHZ * 1e3),
                     "flop": flop,
                     "conf_per_lds": conf / lds if lds > 0 else float("nan"),
                     "lds_wait": wait / wave if wave > 0 else float("nan"),
                     "flop_per_busy": flop / busy if busy > 0 else float("nan")})
    rows.sort(key=lambda r: -(r["us_c"] * r["dispatches"]))
    import json as _json
    group = 1
    log = os.path.join(out_dir, "mfma.log")
    if os.path.exists(log):
        for line in open(log):
            if line.startswith("{"):
                group = int(_json.loads(line)["config"].get("group", 1))
    per_launch = f"{group} micro-batch{'es' if group > 1 else ''} per launch"
    lines = [f"# MFMA and LDS counters: {workload}", "",
             "Commands (from the repository root on the GPU host; one counter group per run):", "",
             "    " + PROFILE_COMMANDS["mfma"], "    " + PROFILE_COMMANDS["lds"], "",
             f"Means per dispatch over one eager step ({per_launch}). "
             "`MFMA GFLOP` = 512 x SQ_INSTS_VALU_MFMA_MOPS_BF16. `FLOP/busy cycle` = those FLOPs "
             "per SQ_VALU_MFMA_BUSY_CYCLES (summed over SIMDs): 1024 means every busy MFMA cycle "
             "of a SIMD does the full dense bf16 work (32x32x16: 32768 FLOP in 32 cycles). "
             "`MFMA busy` = SQ_VALU_MFMA_BUSY_CYCLES / (1024 SIMDs x duration x 2.4 GHz), with "
             "the duration of the counter run's own dispatches (`busy, counter run`) and with "
             f"the eager-pass duration of the kernel trace (`kernel_trace_{workload}.md`; "
             "`busy, eager`). `LDS wait` = SQ_WAIT_INST_LDS / SQ_WAVE_CYCLES, the share of wave "
             "time spent waiting to issue an LDS instruction. (GRBM_GUI_ACTIVE and "
             "SQ_BUSY_CU_CYCLES were collected too but carry a per-dispatch overhead of "
             "10-30 thousand cycles, so they are not used as denominators.)", "",
             "| kernel | dispatches | MFMA GFLOP | FLOP/busy cycle | us, counter run | "
             "MFMA busy, counter run | eager us | MFMA busy, eager | "
             "LDS conflict cycles/instr | LDS wait |",
             "|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|"]

    def f(v, fmt):
        return "-" if not (isinstance(v, float) and math.isfinite(v)) else format(v, fmt)
    for r in rows:
        if not (r["flop"] > 0 or r["us_c"] > 5):
            continue
        lines.append(f"| `{r['kernel']}` | {r['dispatches']} | {f(r['flop'] / 1e9, '.2f')} | "
                     f"{f(r['flop_per_busy'], '.0f')} | {f(r['us_c'], '.2f')} | "
                     f"{f(100 * r['busy_c'], '.1f')}% | {f(r['us'], '.2f')} | "
                     f"{f(100 * r['busy_e'], '.1f')}% | {f(r['conf_per_lds'], '.3f')} | "
                     f"{f(100 * r['lds_wait'], '.1f')}% |")
    with open(os.path.join(PROFILES, f"counters_{workload}.md"), "w") as fh:
        fh.write("\n".join(lines) + "\n")
    return rows


def recorded_traffic(kernel, workload, group):
    """HBM bytes per launch of `kernel` from a profiles/ summary taken with
    the current kernel sources and the same micro-batches per launch, else
    None."""
    import glob
    import json as _json
    try:
        cur = kernel_source_hash(kernel)
    except (OSError, StopIteration):
        return None
    for path in glob.glob(os.path.join(PROFILES, "traffic_*.md")):
        for line in open(path):
            if line.startswith("traffic_json: "):
                info = _json.loads(line[len("traffic_json: "):])
                if info.get("kernel") == kernel and info.get("workload") == workload and \
                        info.get("source_hash") == cur and info.get("group", 1) == group:
                    return info["bytes_per_launch"]
    return None


def roofline_of(dom, per_step_div):
    """Roofline entry of the dominant kernel from its profiled launches:
    algorithmic FLOPs (or bytes) per launch over the mean launch time.  A
    contraction is priced against the bf16 MFMA peak unless its arithmetic
    intensity is below half the ridge point (2.5 PFLOP/s / 8 TB/s), where it
    is plainly HBM-bound and priced against HBM; both fractions are listed."""
    sec = dom["ms"] * 1e-3
    tflops = dom["flops"] / sec / 1e12
    gbps = dom["bytes"] / sec / 1e9
    ridge = BF16_PEAK / HBM_PEAK
    if dom["flops"] > 0 and dom["flops"] / dom["bytes"] >= 0.5 * ridge:
        roof = {"bound": "mfma", "achieved": tflops, "peak": BF16_PEAK / 1e12, "unit": "TFLOP/s",
                "frac": tflops / (BF16_PEAK / 1e12), "traffic": None}
    else:
        roof = {"bound": "hbm", "achieved": gbps, "peak": HBM_PEAK / 1e9, "unit": "GB/s",
                "frac": gbps / (HBM_PEAK / 1e9), "traffic": None}
    roof["mfma_frac"] = tflops / (BF16_PEAK / 1e12)
    roof["hbm_frac"] = gbps / (HBM_PEAK / 1e9)
    roof["algorithmic_bytes_per_launch"] = dom["bytes"] / dom["launches"]
    roof["algorithmic_flops_per_launch"] = dom["flops"] / dom["launches"]
    roof["kernel"] = dom["name"]
    roof["launches_per_step"] = dom["launches"] / per_step_div
    roof["avg_launch_us"] = 1e3 * dom["ms"] / dom["launches"]
    return roof


def network_bench(args, wl, mode):
    """A whole network trained by tgp_pipeline_step (MSE loss, Algorithm 1
    clock order over all partitions), one step captured as a HIP graph and
    replayed; per-kernel durations from an eager one-lane pass afterwards;
    per-partition times from the per-layer measurement (tgp_layer_times)."""
    import torch
    import paper_2004_09910_amd as tgp
    from paper_2004_09910_amd.harness import Session, nchw_to_device_nhwc
    from workloads import specs, synth
    from workloads.specs import BF16
    net, B, m = wl.net, wl.batch, wl.m
    lanes = (args.lanes or 2) if m > 1 else 1
    log("setting up", wl.name)
    sess = Session(net, BF16, n=wl.n)
    sess.plan(B, m, mode, lanes)
    _, xraw = synth.input_x(net, B, BF16)
    oh, ow = net.out_hw()
    _, traw = synth.target_like((B, net.out_channels(), oh, ow), BF16)
    x = nchw_to_device_nhwc(xraw, BF16)
    t = nchw_to_device_nhwc(traw, BF16)
    del xraw, traw
    loss = torch.zeros(1, dtype=torch.float32, device="cuda")
    y = torch.empty((B, oh, ow, net.out_channels()), dtype=x.dtype, device="cuda")
    cur = lambda: torch.cuda.current_stream().cuda_stream
    log("warmup", args.warmup)
    for _ in range(max(args.warmup, 1)):
        sess.pipeline_step(x, t, loss, y, stream=cur())
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        sess.pipeline_step(x, t, loss, y, stream=cur())
    graph.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        graph.replay()
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / args.steps
    del graph
    log(f"timed {args.steps} steps (graph): {ms_step:.2f} ms/step")
    # per-kernel durations: one eager step with a single lane
    sess.plan(B, m, mode, 1)
    tgp.profile_enable(True)
    tgp.profile_read()
    sess.pipeline_step(x, t, loss, y, stream=cur())
    torch.cuda.synchronize()
    stats = tgp.profile_read()
    tgp.profile_enable(False)
    stats.sort(key=lambda r: -r["ms"])
    for r in stats[:12]:
        log(f"  {r['name']:32s} n={r['launches']:6d} {r['ms']:9.3f} ms "
            f"{(r['flops'] / (r['ms'] * 1e-3) / 1e12) if r['ms'] > 0 else 0:8.1f} TF/s")
    roof = roofline_of(stats[0], 1)
    roof["traffic"] = recorded_traffic(stats[0]["name"], wl.name, False)
    roof["timed"] = "one eager step with one lane, each launch timed"
    fwd = net.flops_per_sample()
    r_fac = {specs.CKPT_ALWAYS: 1.0, specs.CKPT_EXCEPT_LAST: (m - 1) / m,
             specs.CKPT_NEVER: 0.0}[mode]
    # forward, recompute and weight gradient of every layer; no data
    # gradient for the first layer (the network input needs none)
    step_flops = B * (sum(fwd) * (2.0 + r_fac) + sum(fwd[1:]))
    planned = memory_account(net, B, m, mode)
    b = B // m
    log("per-layer times")
    us = sess.layer_times(b, mode, iters=2)
    parts = []
    for lo, hi in sess.bounds:
        parts.append(m * sum(us[lo:hi]) / 1e3)
    sess.close()
    out = {
        "metric": "pipeline step samples/sec at 1 MI355X (whole network, all partitions in "
                  "clock order); MFMA util % of bf16 peak",
        "value": B * 1e3 / ms_step, "unit": "samples/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": wl.name, "network": net.name, "partitions": wl.n,
                   "balance": list(sess.balance), "global_batch": B, "micro_batches": m,
                   "checkpoint": args.mode,
                   "input": f"{B}x{net.in_channels}x{net.height}x{net.width}",
                   "launch": "hip_graph", "lanes": lanes},
        "mfma_util_pct": 100.0 * step_flops / (ms_step * 1e-3) / BF16_PEAK,
        "step_tflop": step_flops / 1e12,
        "planned_memory_gb": planned[3] / 1e9 if planned else None,
        "partition_ms_per_step": [round(p, 2) for p in parts],
        "partition_note": "m x the per-layer times of one micro-batch (F, F' and B plus the "
                          "accumulation, eager launches), summed per partition",
        "roofline": roof,
        "cpu_baseline": None,
        "cpu_baseline_note": "not run: one single-sample float64 oracle pass of this network "
                             "takes minutes on the host",
    }
    print(json.dumps(out), flush=True)


def cpu_baseline(wl, lo, hi, samples, dtype):
    """The oracle (float64 CPU, bf16 storage points) on a bounded sample of the
    same workload: `samples` single-sample forward + backward passes of the
    stage at full per-sample shape."""
    import numpy as np
    try:
        from threadpoolctl import threadpool_info
        cores = max([d.get("num_threads", 1) for d in threadpool_info()] + [1])
    except Exception:
        cores = os.cpu_count()
    host = host_cpu_info()
    import oracle
    from oracle import network
    from workloads import synth
    net = wl.net
    P = oracle.net_params(net, dtype)
    ex = network.exported_stashes(net, lo, hi)
    shapes = net.shapes()
    out_shapes = [(net.layers[hi - 1].cout,) + tuple(shapes[hi - 1])]
    for sid in ex:
        k = [q for q, L in enumerate(net.layers) if L.stash_id == sid][0]
        out_shapes.append((net.layers[k].cout,) + tuple(shapes[k]))
    xs = synth.quantize(synth.normal(101, (samples, net.in_channels, net.height, net.width)), dtype)[0]
    Gs = [synth.quantize(synth.normal(102 + k, (samples,) + s), dtype)[0] for k, s in enumerate(out_shapes)]
    t0 = time.perf_counter()
    for s in range(samples):
        network.run(net, P, xs[s:s + 1], lo=lo, hi=hi, out_grads=[g[s:s + 1] for g in Gs],
                    storage="bf16")
    dt = time.perf_counter() - t0
    return {"value": samples / dt, "unit": "samples/s", "cores": cores, "kind": "oracle",
            "sample": f"{samples} single-sample forward+backward passes of the stage at full "
                      f"per-sample shape (no recompute, float64 with bf16 storage rounding), "
                      f"{dt:.1f} s",
            "cores_note": "threads of the BLAS pool the oracle's float64 contractions ran on",
            **host}


def host_cpu_info():
    """Logical CPUs of the host, those this process may run on, and the CPU
    model from /proc/cpuinfo."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        usable = None
    return {"host_logical_cpus": os.cpu_count(), "usable_cpus": usable, "cpu_model": model}


def memory_account(net, B, m, mode):
    """Bytes one training step of `net` needs on the device, all of it caller
    memory (the library allocates nothing): bf16 weights, fp32 biases, fp32
    gradient accumulators, the tgp_plan workspace, and the bf16 input, target
    and output plus the loss.  Returns (parameters, parameter bytes,
    workspace bytes, total bytes), or None if the plan is refused."""
    import paper_2004_09910_amd as tgp
    from paper_2004_09910_amd.harness import layer_tuple
    from workloads.specs import BF16
    h = tgp.net_create([layer_tuple(L) for L in net.layers], net.in_channels, net.height,
                       net.width, BF16)
    try:
        tgp.set_partition(h, 1)
        ws = tgp.plan(h, B, m, mode)
    except tgp.TgpError:
        return None
    finally:
        tgp.net_destroy(h)
    w = sum(L.cout * L.taps * L.cin for L in net.layers)
    nb = sum(L.cout for L in net.layers if L.bias)
    pbytes = 2 * w + 4 * nb + 4 * (w + nb)
    oh, ow = net.out_hw()
    io = 2 * B * (net.in_channels * net.height * net.width + 2 * net.out_channels() * oh * ow) + 4
    return w + nb, pbytes, ws, pbytes + ws + io


MEM_SHAPE = dict(B=32, hw=192, in_ch=3, levels=6)   # the paper's U-Net memory benchmark


def largest_unet(budget, m, mode, channels):
    """(blocks per level, first-level channels, memory_account) of the
    six-level U-Net of MEM_SHAPE with the most parameters whose planned
    memory fits `budget` bytes, over the channel counts given and any
    number of blocks."""
    from workloads import specs
    B, hw, in_ch, levels = (MEM_SHAPE[k] for k in ("B", "hw", "in_ch", "levels"))
    best = None
    for C in channels:
        def fits(blocks):
            net = specs.unet(levels, C, in_ch, hw, f"unet6-B{blocks}-C{C}", blocks=blocks)
            a = memory_account(net, B, m, mode)
            return a if a is not None and a[3] <= budget else None
        if not fits(1):
            continue
        lo, hi = 1, 2
        while fits(hi) and hi < 512:
            lo, hi = hi, hi * 2
        while hi - lo > 1:          # largest blocks count that fits
            mid = (lo + hi) // 2
            if fits(mid):
                lo = mid
            else:
                hi = mid
        a = fits(lo)
        if best is None or a[0] > best[2][0]:
            best = (lo, C, a)
    return best


def memory_report():
    """U-Net memory benchmark analog (Sec. 4.2.2 and its table): the largest
    U-Net (B conv blocks per level, C channels at the first level; six levels,
    so five down-samplings; 3x192x192 input, 1x192x192 output, batch 32) whose
    planned memory fits one MI355X, without checkpointing or micro-batches and
    with checkpointing at m = 8 and m = 32."""
    from workloads import specs
    from workloads.specs import CKPT_ALWAYS, CKPT_NEVER
    HBM = 288e9
    B, hw, in_ch, levels = 32, 192, 3, 6
    settings = [("no checkpointing, m = 1", 1, CKPT_NEVER),
                ("checkpointing (always), m = 8", 8, CKPT_ALWAYS),
                ("checkpointing (always), m = 32", 32, CKPT_ALWAYS)]
    channels = [32, 48, 64, 72, 96, 128, 160, 192, 224, 256, 320, 384]
    rows = []
    for label, m, mode in settings:
        blocks, C, (params, pbytes, ws, total) = largest_unet(HBM, m, mode, channels)
        log(f"{label}: (B, C) = ({blocks}, {C}), {params / 1e9:.2f}B parameters, {total / 1e9:.1f} GB")
        rows.append({"setting": label, "m": m, "blocks": blocks, "channels": C, "params": params,
                     "param_gb": pbytes / 1e9, "workspace_gb": ws / 1e9, "total_gb": total / 1e9})
    lines = ["# U-Net memory benchmark analog: largest model on one MI355X", "",
             "Command (from the repository root; the search runs on the host planner, the check "
             "below on the GPU):", "", "    python3 bench.py --memory", "",
             f"Six-level U-Net (five down-samplings), B conv blocks per level, C channels at the "
             f"first level, input 3x192x192, output 1x192x192, batch {B}, bf16.  Memory is what "
             "the caller allocates: bf16 weights, fp32 biases and accumulators (6 bytes per "
             "weight), the `tgp_plan` workspace and the input, target and output.  Budget "
             f"{HBM / 1e9:.0f} GB.  Among C in {channels} and any B, the configuration with the "
             "most parameters that fits:", "",
             "| setting | (B, C) | parameters | parameter memory | workspace | total |",
             "|---|---|---:|---:|---:|---:|"]
    for r in rows:
        lines.append(f"| {r['setting']} | ({r['blocks']}, {r['channels']}) | {r['params'] / 1e9:.2f}B | "
                     f"{r['param_gb']:.1f} GB | {r['workspace_gb']:.1f} GB | {r['total_gb']:.1f} GB |")
    scale = memory_at_scale()
    if scale:
        lines += ["", f"The planner's choice under a {scale[0]['budget_gb']:.0f} GB budget, trained "
                  "for one `tgp_pipeline_step` on the GPU (weights drawn on the device; the "
                  "3-channel first layer runs the direct kernels); allocated is torch's peak over "
                  "creation, planning and the step, including the caller's tensors:", "",
                  "| setting | (B, C) | parameters | planned | allocated peak | workspace | step |",
                  "|---|---|---:|---:|---:|---:|---:|"]
        for c in scale:
            lines.append(f"| {c['setting']} | ({c['blocks']}, {c['channels']}) | "
                         f"{c['params'] / 1e9:.2f}B | {c['planned_gb']:.3f} GB | "
                         f"{c['allocated_gb']:.3f} GB | {c['workspace_gb']:.3f} GB | "
                         f"{c['step_s']:.2f} s |")
    check = memory_check()
    if check:
        lines += ["", "Planned against allocated memory on the GPU for the 5-level, 64-channel network "
                  "(64x192x192 input, batch 32), one `tgp_pipeline_step` each; allocated is "
                  "torch's peak over the step, including the caller's tensors:", "",
                  "| setting | planned | allocated peak | workspace |", "|---|---:|---:|---:|"]
        for c in check:
            lines.append(f"| {c['setting']} | {c['planned_gb']:.3f} GB | {c['allocated_gb']:.3f} GB | "
                         f"{c['workspace_gb']:.3f} GB |")
    os.makedirs(PROFILES, exist_ok=True)
    with open(os.path.join(PROFILES, "memory_unet.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print(json.dumps({"largest": rows, "check": check, "at_scale": scale}), flush=True)


def memory_at_scale(budget=64e9):
    """On a GPU: the largest U-Net of MEM_SHAPE that the planner fits in
    `budget` bytes without checkpointing (m = 1) and with checkpointing at
    m = 8, each created, planned and trained for one pipeline step; planned
    bytes against torch's allocated peak."""
    import torch
    if not torch.cuda.is_available():
        return None
    from paper_2004_09910_amd.harness import Session
    from workloads import specs
    from workloads.specs import BF16, CKPT_ALWAYS, CKPT_NEVER
    B, hw, in_ch, levels = (MEM_SHAPE[k] for k in ("B", "hw", "in_ch", "levels"))
    out = []
    for label, m, mode in [("no checkpointing, m = 1", 1, CKPT_NEVER),
                           ("checkpointing (always), m = 8", 8, CKPT_ALWAYS)]:
        blocks, C, acct = largest_unet(budget, m, mode, [64, 96, 128, 160, 192, 224, 256])
        net = specs.unet(levels, C, in_ch, hw, f"unet6-B{blocks}-C{C}", blocks=blocks)
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        torch.cuda.reset_peak_memory_stats()
        base = torch.cuda.memory_allocated()
        log(f"memory at scale: {label}: (B, C) = ({blocks}, {C}), {acct[0] / 1e9:.2f}B parameters")
        sess = Session(net, BF16, n=1, init="device")
        ws = sess.plan(B, m, mode)
        x = torch.randn((B, hw, hw, in_ch), device="cuda").to(torch.bfloat16)
        oh, ow = net.out_hw()
        t = torch.randn((B, oh, ow, net.out_channels()), device="cuda").to(torch.bfloat16)
        loss = torch.zeros(1, dtype=torch.float32, device="cuda")
        y = torch.empty_like(t)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        sess.pipeline_step(x, t, loss, y)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        peak = torch.cuda.max_memory_allocated() - base
        log(f"  planned {acct[3] / 1e9:.3f} GB, allocated peak {peak / 1e9:.3f} GB, step {dt:.2f} s, "
            f"loss {float(loss.item()):.4g}")
        out.append({"setting": label, "budget_gb": budget / 1e9, "blocks": blocks, "channels": C,
                    "params": acct[0], "planned_gb": acct[3] / 1e9, "allocated_gb": peak / 1e9,
                    "workspace_gb": ws / 1e9, "step_s": dt, "loss": float(loss.item())})
        sess.close()
        del sess, x, t, y, loss
        torch.cuda.empty_cache()
    return out


def memory_check():
    """On a GPU: plan, allocate and run one pipeline step of the 5-level,
    64-channel U-Net at batch 32 without and with checkpointing; the planned
    bytes against torch's allocated peak."""
    import torch
    if not torch.cuda.is_available():
        return None
    from paper_2004_09910_amd.harness import Session, nchw_to_device_nhwc
    from workloads import specs, synth
    from workloads.specs import BF16, CKPT_ALWAYS, CKPT_NEVER
    wl = specs.unet_network()
    net = wl.net
    out = []
    for label, m, mode in [("no checkpointing, m = 1", 1, CKPT_NEVER),
                           ("checkpointing (always), m = 8", 8, CKPT_ALWAYS)]:
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        torch.cuda.reset_peak_memory_stats()
        base = torch.cuda.memory_allocated()
        sess = Session(net, BF16, n=1)
        ws = sess.plan(wl.batch, m, mode)
        _, xraw = synth.input_x(net, wl.batch, BF16)
        h, w = net.out_hw()
        _, traw = synth.target_like((wl.batch, net.out_channels(), h, w), BF16)
        x = nchw_to_device_nhwc(xraw, BF16)
        t = nchw_to_device_nhwc(traw, BF16)
        loss = torch.zeros(1, dtype=torch.float32, device="cuda")
        y = torch.empty((wl.batch, h, w, net.out_channels()), dtype=x.dtype, device="cuda")
        log(f"memory check: {label}")
        sess.pipeline_step(x, t, loss, y)
        torch.cuda.synchronize()
        peak = torch.cuda.max_memory_allocated() - base
        planned = memory_account(net, wl.batch, m, mode)[3]
        out.append({"setting": label, "planned_gb": planned / 1e9, "allocated_gb": peak / 1e9,
                    "workspace_gb": ws / 1e9})
        sess.close()
        del sess, x, t, y, loss
    return out


def sweep_report(steps, warmup):
    """The whole 5-level U-Net (4 partitions, batch 32) trained by
    tgp_pipeline_step, one step captured as a HIP graph (two lanes when
    m > 1), for m in 1, 4, 16, 32 under each checkpoint mode: samples/s,
    the recompute overhead against never, the planned memory and whether
    every gradient is bit-identical to the never run at the same m (the
    checkpoint modes change only when values are computed, Sec. 2.1)."""
    import numpy as np
    import torch
    from paper_2004_09910_amd.harness import Session, nchw_to_device_nhwc
    from workloads import specs, synth
    from workloads.specs import BF16, CKPT_NAMES

    wl = specs.unet_network()
    net, B = wl.net, wl.batch
    _, xraw = synth.input_x(net, B, BF16)
    oh, ow = net.out_hw()
    _, traw = synth.target_like((B, net.out_channels(), oh, ow), BF16)
    x = nchw_to_device_nhwc(xraw, BF16)
    t = nchw_to_device_nhwc(traw, BF16)
    loss = torch.zeros(1, dtype=torch.float32, device="cuda")
    y = torch.empty((B, oh, ow, net.out_channels()), dtype=x.dtype, device="cuda")
    rows = []
    for m in (1, 4, 16, 32):
        grads = {}
        for mode_name in ("never", "except_last", "always"):
            mode = CKPT_NAMES[mode_name]
            lanes = 2 if m > 1 else 1
            log(f"sweep: m={m} {mode_name}")
            sess = Session(net, BF16, n=wl.n)
            sess.plan(B, m, mode, lanes)
            for _ in range(warmup):
                sess.pipeline_step(x, t, loss, y, stream=torch.cuda.current_stream().cuda_stream)
            torch.cuda.synchronize()
            grads[mode_name] = sess.grads64()
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                sess.pipeline_step(x, t, loss, y, stream=torch.cuda.current_stream().cuda_stream)
            graph.replay()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(steps):
                graph.replay()
            torch.cuda.synchronize()
            ms = (time.perf_counter() - t0) * 1e3 / steps
            total = memory_account(net, B, m, mode)[3]
            rows.append({"m": m, "mode": mode_name, "ms_per_step": ms, "samples_per_s": B * 1e3 / ms,
                         "memory_gb": total / 1e9, "loss": float(loss.item())})
            del graph
            sess.close()
        for mode_name in ("except_last", "always"):
            same = all(np.array_equal(grads[mode_name][k][0], grads["never"][k][0]) and
                       (grads["never"][k][1] is None or
                        np.array_equal(grads[mode_name][k][1], grads["never"][k][1]))
                       for k in grads["never"])
            for r in rows:
                if r["m"] == m and r["mode"] == mode_name:
                    r["bit_identical_to_never"] = same
    for r in rows:
        base = next(q for q in rows if q["m"] == r["m"] and q["mode"] == "never")
        r["recompute_overhead"] = r["ms_per_step"] / base["ms_per_step"] - 1.0
    lines = [f"# Checkpoint / micro-batch sweep: {wl.name}", "",
             "Command (from the repository root on the GPU host):", "",
             f"    python3 bench.py --sweep --steps {steps} --warmup {warmup}", "",
             f"The 5-level, 64-channel U-Net in {wl.n} partitions (FLOP balance), batch {B}, "
             "trained by `tgp_pipeline_step` (MSE loss), one step captured as a HIP graph "
             "and replayed; two concurrency lanes when m > 1.  Memory is the planned total "
             "(parameters, accumulators, workspace, input, target, output).  The overhead is the "
             "step time against never at the same m; the paper's bound for recomputing every "
             "forward is one extra forward, a third of forward plus backward.", "",
             "| m | mode | ms/step | samples/s | overhead vs never | memory | gradients = never |",
             "|---:|---|---:|---:|---:|---:|---|"]
    for r in rows:
        ident = "" if r["mode"] == "never" else ("bit-identical" if r["bit_identical_to_never"] else "DIFFER")
        lines.append(f"| {r['m']} | {r['mode']} | {r['ms_per_step']:.2f} | {r['samples_per_s']:.0f} | "
                     f"{100 * r['recompute_overhead']:+.1f}% | {r['memory_gb']:.2f} GB | {ident} |")
    os.makedirs(PROFILES, exist_ok=True)
    with open(os.path.join(PROFILES, f"sweep_{wl.name}.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print(json.dumps({"network": wl.name, "rows": rows}), flush=True)


def balance_report(mode_name, iters=5):
    """Per-layer times (tgp_layer_times: F, F' and B plus the accumulation of
    one micro-batch, eager launches) of the whole 5-level U-Net at the bench's
    micro-batch of 4, and the 4-way partitions the min-max rule picks on them
    and on forward FLOPs."""
    import math
    import paper_2004_09910_amd as tgp
    from paper_2004_09910_amd.harness import Session
    from workloads import specs
    from workloads.specs import BF16, CKPT_NAMES

    wl = specs.unet_network()
    net = wl.net
    b = wl.batch // wl.m
    log("setting up", wl.name)
    sess = Session(net, BF16, n=wl.n)
    flop_bal = list(sess.balance)
    us = sess.layer_times(b, CKPT_NAMES[mode_name], iters=iters)
    ns = [int(math.floor(float(u) * 1000.0 + 0.5)) for u in us]
    time_bal = tgp.balance_minmax(ns, wl.n)
    flops = [tgp.layer_flops(sess.h, k) for k in range(len(net.layers))]
    sess.close()

    def parts(bal):
        out, lo = [], 0
        for c in bal:
            out.append(sum(us[lo:lo + c]))
            lo += c
        return out

    ft, tt = parts(flop_bal), parts(time_bal)
    lines = [f"# Per-layer times and time-based balance: {wl.name}", "",
             "Command (from the repository root on the GPU host):", "",
             f"    python3 bench.py --balance-by-time --mode {mode_name}", "",
             f"Micro-batch of {b} samples at {net.height}x{net.width}, checkpoint mode {mode_name}; "
             f"each time is the mean of {iters} eager runs of F (and F' when checkpointed), B and "
             "the accumulation of a one-layer partition (`tgp_layer_times`), launch gaps included.",
             "", "| layer | GFLOP/sample (fwd) | us | us per GFLOP |", "|---|---:|---:|---:|"]
    for L, f, u in zip(net.layers, flops, us):
        lines.append(f"| {L.name} | {f / 1e9:.3f} | {u:.1f} | {u / (f / 1e9 * b):.2f} |")
    lines += ["", "| partition rule | balance | per-partition us | slowest us |", "|---|---|---|---:|",
              f"| forward FLOPs | {flop_bal} | {[round(v, 1) for v in ft]} | {max(ft):.1f} |",
              f"| measured time | {time_bal} | {[round(v, 1) for v in tt]} | {max(tt):.1f} |"]
    os.makedirs(PROFILES, exist_ok=True)
    with open(os.path.join(PROFILES, f"layer_times_{wl.name}.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print(json.dumps({"network": wl.name, "micro_batch": b, "mode": mode_name,
                      "layer_us": [round(u, 2) for u in us], "flop_balance": flop_bal,
                      "time_balance": time_bal, "flop_balance_slowest_us": round(max(ft), 2),
                      "time_balance_slowest_us": round(max(tt), 2)}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--cpu-samples", type=int, default=None,
                    help="single-sample oracle passes for cpu_baseline (default: about 20 s "
                         "of CPU work for the workload)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--workload", default="unet5-stage1of4",
                    choices=["unet5-stage1of4", "amoeba18-c256-stage", "unet6-c128-network"],
                    help="unet5-stage1of4 is the headline; the depthwise/pointwise cell stage "
                         "and the 6-level U-Net network print a line of their own")
    ap.add_argument("--mode", default=None, choices=["always", "except_last", "never"],
                    help="checkpoint mode (default: the workload's own)")
    ap.add_argument("--lanes", type=int, default=None,
                    help="concurrency lanes: micro-batch i runs on stream (i - 1) %% lanes "
                         "(default: the group size, at least 2)")
    ap.add_argument("--group", type=int, default=16, choices=[1, 2, 4, 8, 16],
                    help="micro-batches per stage call and kernel launch (halved until it "
                         "divides the lanes and m)")
    ap.add_argument("--one-stream", dest="one_stream", action="store_true", default=None,
                    help="issue the whole step on one stream, accumulations included (the "
                         "default with several micro-batches per launch)")
    ap.add_argument("--lane-streams", dest="one_stream", action="store_false",
                    help="issue micro-batches on lane streams and the accumulations on one more "
                         "stream (the default with one micro-batch per launch)")
    ap.add_argument("--eager", action="store_true", help="time eager launches instead of a HIP graph")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run three device-to-device copies of 1 GiB (the reference "
                         "kernel that scales the HBM byte counters)")
    ap.add_argument("--summarize-profiles", metavar="DIR",
                    help="write the profiles/ summaries from rocprofv3 output under DIR")
    ap.add_argument("--memory", action="store_true",
                    help="only run the U-Net memory benchmark analog: the largest (blocks, "
                         "channels) U-Net whose planned memory fits one MI355X, with and "
                         "without checkpointing, and (on a GPU) the planned against the "
                         "allocated memory of the 5-level network; writes "
                         "profiles/memory_unet.md")
    ap.add_argument("--sweep", action="store_true",
                    help="only run the checkpoint / micro-batch sweep of the whole 5-level "
                         "U-Net pipeline (m in 1, 4, 16, 32 under each checkpoint mode): "
                         "samples/s, recompute overhead, planned memory and bit-identity of "
                         "gradients across modes; writes profiles/sweep_unet5-network.md")
    ap.add_argument("--balance-by-time", action="store_true",
                    help="only measure per-layer times of the whole 5-level U-Net at the "
                         "bench's micro-batch, compare the time-based and FLOP-based 4-way "
                         "partitions and write profiles/layer_times_<network>.md")
    args = ap.parse_args()
    if args.summarize_profiles:
        from workloads import specs
        summarize_profiles(args.summarize_profiles, specs.unet_stage().name)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}); this build has no "
              f"multi-GPU path", file=sys.stderr)
        sys.exit(2)

    import torch
    if args.copy_calibration:
        src = torch.ones(1 << 29, dtype=torch.bfloat16, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": src.numel() * 2, "copy_bytes_written": dst.numel() * 2,
                          "launches": 3}), flush=True)
        return
    if args.balance_by_time:
        balance_report(args.mode or "always")
        return
    if args.memory:
        memory_report()
        return
    if args.sweep:
        sweep_report(args.steps, args.warmup)
        return
    import paper_2004_09910_amd as tgp
    from paper_2004_09910_amd.harness import Session, nchw_to_device_nhwc
    from workloads import specs, synth
    from workloads.specs import BF16, CKPT_NAMES

    wl = specs.ALL[args.workload]
    if args.mode is None:
        args.mode = {v: k for k, v in CKPT_NAMES.items()}[wl.mode]
    mode = CKPT_NAMES[args.mode]
    if wl.kind != "stage":
        network_bench(args, wl, mode)
        return
    net = wl.net
    log("setting up", wl.name)
    sess = Session(net, BF16, n=wl.n, bind_layers=None)
    lo, hi = sess.bounds[0]
    while args.group > 1 and wl.m % args.group:
        args.group //= 2
    if args.lanes is None:
        args.lanes = max(2, args.group)
    while args.group > 1 and min(args.lanes, wl.m) % args.group:
        args.group //= 2
    sess.plan(wl.batch, wl.m, mode, args.lanes)
    sess.group = args.group
    if args.one_stream is None:
        # measured: with two micro-batches per launch the accumulations on a
        # stream of their own slow the persistent convolutions they overlap
        # more than they gain; with one per launch, two lane streams win
        args.one_stream = args.group > 1
    B, m = wl.batch, wl.m
    _, xraw = synth.input_x(net, B, BF16)
    x = nchw_to_device_nhwc(xraw, BF16)
    C, H, W = sess.part_out_shape(1)
    y = torch.empty((B, H, W, C), dtype=torch.bfloat16, device="cuda")
    _, g0 = synth.target_like((B, C, H, W), BF16, 0)
    dy = nchw_to_device_nhwc(g0, BF16)
    dx = torch.empty_like(x)
    b = B // m
    for k, sid in enumerate(sess.exported_stashes(1)):
        _, gk = synth.target_like((B,) + sess.stash_shape(sid), BF16, 1 + k)
        gd = nchw_to_device_nhwc(gk, BF16)
        for i in range(1, m + 1):
            sess.stash_view(i, sid, True).copy_(gd[(i - 1) * b:i * b])
    del xraw
    stream = torch.cuda.current_stream().cuda_stream
    torch.cuda.synchronize()

    log("warmup", args.warmup)
    for _ in range(args.warmup):
        sess.stage_step(1, x, y, dy, dx, stream, serial=args.one_stream)
    torch.cuda.synchronize()

    # One step captured as a HIP graph: the ~600 launches of a step replay
    # without host launch overhead.  Events recorded under capture cannot be
    # read back, so per-kernel durations come from an eager pass of the same
    # step right after the timed replays.
    graph = None
    if not args.eager:
        try:
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                sess.stage_step(1, x, y, dy, dx, torch.cuda.current_stream().cuda_stream,
                                serial=args.one_stream)
            graph.replay()
            torch.cuda.synchronize()
        except Exception as exc:
            log(f"graph capture failed, timing eager launches: {exc}")
            graph = None
    profiled_graph = False

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    if graph is not None:
        for s_ in range(args.steps):
            graph.replay()
    else:
        tgp.profile_enable(True)
        tgp.profile_read()
        for s_ in range(args.steps):
            sess.stage_step(1, x, y, dy, dx, stream, serial=args.one_stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    if graph is not None and profiled_graph:
        stats = tgp.profile_read()            # per-kernel events of the last replay
        per_step_div = 1
    elif graph is not None:
        # kernel durations from an eager pass of the same step on one stream,
        # so that each launch is timed alone
        tgp.profile_enable(True)
        tgp.profile_read()
        for s_ in range(args.steps):
            sess.stage_step(1, x, y, dy, dx, stream, serial=True)
        torch.cuda.synchronize()
        stats = tgp.profile_read()
        per_step_div = args.steps
    else:
        stats = tgp.profile_read()
        per_step_div = args.steps
    tgp.profile_enable(False)
    elapsed = t1 - t0
    ms_step = 1e3 * elapsed / args.steps
    log(f"timed {args.steps} steps ({'graph' if graph is not None else 'eager'}): {ms_step:.3f} ms/step")

    fwd_flops = sum(net.flops_per_sample()[lo:hi]) * B
    recompute = {specs.CKPT_ALWAYS: 1.0, specs.CKPT_EXCEPT_LAST: (m - 1) / m,
                 specs.CKPT_NEVER: 0.0}[mode]
    step_flops = fwd_flops * (3.0 + recompute)    # forward, recompute, dgrad, wgrad
    samples_s = B * args.steps / elapsed

    stats.sort(key=lambda r: -r["ms"])
    for r in stats:
        log(f"  {r['name']:32s} n={r['launches'] / per_step_div:7.1f}/step {r['ms'] / per_step_div:8.3f} ms/step "
            f"{(r['flops'] / (r['ms'] * 1e-3) / 1e12) if r['ms'] > 0 else 0:8.1f} TF/s "
            f"{(r['bytes'] / (r['ms'] * 1e-3) / 1e9) if r['ms'] > 0 else 0:8.1f} GB/s")
    dom = stats[0]
    roof = roofline_of(dom, per_step_div)
    roof["traffic"] = recorded_traffic(dom["name"], wl.name, args.group)
    roof["timed"] = "eager pass of the step on one stream, each launch timed alone" \
        if graph is not None else "the timed eager steps"
    if args.group > 1:
        roof["timed"] += f"; {args.group} micro-batches per launch"
    kernel_ms = sum(r["ms"] for r in stats) / per_step_div

    out = {
        "metric": "stage fwd+recompute+bwd samples/sec at 1 MI355X; MFMA util % of bf16 peak",
        "value": samples_s, "unit": "samples/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": wl.name, "network": net.name, "partition": f"{wl.stage_j} of {wl.n}",
                   "layers": hi - lo, "global_batch": B, "micro_batches": m,
                   "checkpoint": args.mode, "input": f"{B}x{net.in_channels}x{net.height}x{net.width}",
                   "dx_in": True, "launch": "hip_graph" if graph is not None else "eager",
                   "lanes": args.lanes, "group": args.group, "one_stream": args.one_stream},
        "mfma_util_pct": 100.0 * step_flops / (ms_step * 1e-3) / BF16_PEAK,
        "step_tflop": step_flops / 1e12,
        "kernel_busy_ms_per_step": kernel_ms,
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        log("cpu baseline")
        samples = args.cpu_samples or {"unet5-stage1of4": 40}.get(wl.name, 12)
        out["cpu_baseline"] = cpu_baseline(wl, lo, hi, samples, BF16)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
