"""Throughput of RegVGGT's per-frame hot path on one MI355X.

Workload: the 24-layer ViT-L-shaped stream (16 heads x 64, 1041 tokens per frame =
28x37 patches + 5 special tokens, budget 10 tokens per head per frame, 2x2 query
sampling) of 1000 frames, whose memory grows from empty to 9,990 rows per (layer, head)
(Sec. 3.3 Eq. 6: 10 rows per frame).  One step = one frame: for each of the 24 layers,
attention of the frame over that layer's memory with per-query LSE (rv_attend_frame),
then one deferred launch that computes every layer's LSE-saliency, selects each head's
top 10 and appends them (rv_admit_layers).

--steps 1000 times the whole stream in order from an empty memory.  --steps K < 1000
times a stratified sample of it: frame t_i = floor((i + 1/2) 1000 / K) for i < K, each
attended and admitted at the memory length it has in the stream (t_i x 10 rows), so the
mean context of the timed frames equals the stream's (about 6,036).  Each layer's memory
is filled once with generator rows to the longest of those lengths, and the frames run
back to back, longest memory first, each preceded by a host-side length change
(rv_mem_truncate, no device work).

Every timed frame's Q/K/V (distinct per layer and frame, seeded) is generated on the GPU
and resident in HBM before timing starts (153 MB per frame).  The timed region covers the
steps only, between device synchronisations.  HIP events on the compute stream bracket
each frame's attention launches and its admission launch; they give the attention
kernel's average duration, from which the roofline fraction is computed.  The oracle is
timed on the host on a bounded sample (one layer of each of 24 stratified frames at its
stream memory length) and extrapolated to frames/s.

Prints one JSON line on stdout; progress goes to stderr.
"""
import argparse
import glob
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6   # MI355X dense bf16 MFMA: 256 CU x 2.4 GHz x 4096 flop/clk
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
PROFILES = os.path.join(ROOT, "profiles")
CSRC = os.path.join(ROOT, "paper_2609_23286_amd", "csrc")
# Kernel -> the sources whose text decides its memory traffic; counters recorded for
# other sources are stale and are not reported.
_HOST = ("rv_internal.h", "rv_plan.h", "rv_plan.cpp", "rv_host.cpp")
KERNEL_SOURCES = {"attn_fwd_kernel": ("attend.hip",) + _HOST,
                  "attn_merge_kernel": ("attend.hip",) + _HOST,
                  "sal_kernel": ("admit.hip",) + _HOST,
                  "select_kernel": ("admit.hip",) + _HOST}
ADMISSION_KERNELS = ("sal_kernel", "select_kernel")  # one launch each per frame
COPY_CALIBRATION_BYTES = 256 << 20   # read and written once by the calibration copy
WARMUP_MIN_S = 0.1                   # least wall time of warm-up frames (when --warmup > 0)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def attention_flops(N, H, d, ctx):
    """Algorithmic flops of one attention launch: 2*d (Q.K) + 2*d (P.V) per
    (head, query, context key) pair."""
    return 4.0 * d * H * N * ctx


def admit_bytes(N, H, d, n_q, k):
    """Algorithmic HBM bytes of the saliency + top-k + append phase for one layer."""
    return (n_q * H * d * 2          # sampled query rows
            + N * H * d * 2          # the frame's keys
            + n_q * H * 4            # LSE of the sampled queries
            + N * H * 4 * 2          # saliency written, then read by the selection
            + 2 * k * H * d * 2 * 2  # K and V rows read and appended
            + k * H * 8)             # provenance


def _code_only(text):
    """Source text without comments and whitespace (so that editing a comment does not
    mark recorded counters stale)."""
    import re
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    return re.sub(r"\s+", "", text)


def kernel_source_hash(kernel):
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        with open(os.path.join(CSRC, f), encoding="utf-8") as fh:
            h.update(_code_only(fh.read()).encode())
    return h.hexdigest()[:16]


def traffic_path(kernel, workload):
    return os.path.join(PROFILES, f"{kernel}__{workload}__hbm_traffic.md")


def recorded_counters(kernel, workload):
    """(HBM bytes per launch, dispatches counted) from the committed counter summary, or
    None when there is none or the kernel's sources changed since it was taken."""
    try:
        text = open(traffic_path(kernel, workload)).read()
    except OSError:
        return None
    kv = {}
    for line in text.splitlines():
        if line.startswith("- ") and ": " in line:
            k, v = line[2:].split(": ", 1)
            kv[k.strip("` ")] = v.strip("` ")
    if kv.get("source_hash") != kernel_source_hash(kernel):
        return None
    try:
        return float(kv["hbm_bytes_per_launch"]), int(kv["dispatches"].split()[0])
    except (KeyError, ValueError, IndexError):
        return None


def recorded_traffic(kernel, workload):
    rec = recorded_counters(kernel, workload)
    return None if rec is None else rec[0]


def attention_traffic(workload):
    """HBM bytes of one layer's attention step: the forward launch plus, averaged over
    the stream, the merge launch that split plans add."""
    fwd, merge = recorded_counters("attn_fwd_kernel", workload), recorded_counters("attn_merge_kernel", workload)
    if fwd is None or merge is None:
        return None
    return fwd[0] + merge[0] * merge[1] / fwd[1]


def admission_traffic(workload):
    """HBM bytes of one frame's admission (one saliency and one selection launch)."""
    parts = [recorded_traffic(k, workload) for k in ADMISSION_KERNELS]
    return None if any(p is None for p in parts) else sum(parts)


def bench_args():
    """This command's benchmark arguments, without the summary options."""
    n_args = {"--pmc-summary": 2, "--trace-summary": 2, "--mfma-summary": 4}
    out, skip = [], 0
    for a in sys.argv[1:]:
        if skip:
            skip -= 1
            continue
        if a in n_args:
            skip = n_args[a]
            continue
        out.append(a)
    return " ".join(out)


def timed_start(dispatches, steps, layers):
    """Start timestamp of the timed frames in a profiled benchmark run, from its dispatches
    [(kernel name, start timestamp)]: the first of the last steps x layers attention
    launches (a frame-staging launch before it in the frame counts too).  Earlier
    dispatches are the input generation and the warm-up frames.  None (keep everything)
    when steps or layers is not given or the run has fewer launches."""
    if not steps or not layers:
        return None
    attn = sorted(t for n, t in dispatches if "attn_fwd_kernel" in n)
    if len(attn) < steps * layers:
        return None
    t0 = attn[-steps * layers]
    stage = sorted(t for n, t in dispatches if "stage_layers_kernel" in n)
    if len(stage) >= steps:
        t0 = min(t0, stage[-steps])
    return t0


def counter_rows(d):
    """Rows of every *counter_collection.csv under d."""
    import csv
    rows = []
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        rows.extend(csv.DictReader(open(f)))
    return rows


def timed_counter_rows(rows, steps, layers):
    """The counter rows of the timed frames' dispatches (all rows when that is unknown)."""
    first = {}
    for r in rows:
        first.setdefault(r["Dispatch_Id"], (r["Kernel_Name"], int(r["Start_Timestamp"])))
    t0 = timed_start(list(first.values()), steps, layers)
    return rows if t0 is None else [r for r in rows if int(r["Start_Timestamp"]) >= t0]


def summarize_pmc(fetch_dir, write_dir, workload, steps=None, layers=None):
    """Reduce two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE; counter CSVs) of this
    benchmark started with --copy-calibration into per-launch HBM traffic of the timed
    frames' dispatches (timed_start; all dispatches when steps or layers is None).  The
    calibration copy reads and writes COPY_CALIBRATION_BYTES once; the counters'
    readings for it give the factors that turn KiB per dispatch into bytes."""

    def per_kernel(rows, counter):
        out = {}
        for r in rows:
            if r["Counter_Name"] == counter:
                out.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
        return out

    f_rows, w_rows = counter_rows(fetch_dir), counter_rows(write_dir)
    fetch_all, write_all = per_kernel(f_rows, "FETCH_SIZE"), per_kernel(w_rows, "WRITE_SIZE")
    fetch = per_kernel(timed_counter_rows(f_rows, steps, layers), "FETCH_SIZE")
    write = per_kernel(timed_counter_rows(w_rows, steps, layers), "WRITE_SIZE")

    def find(d, key):
        hits = [v for k, v in d.items() if key in k]
        if not hits:
            raise SystemExit(f"no dispatch of {key} in the counter CSVs")
        return hits[0]

    copy_key = "neg_kernel"
    cf = max(find(fetch_all, copy_key))
    cw = max(find(write_all, copy_key))
    f_scale = COPY_CALIBRATION_BYTES / (cf * 1024.0)
    w_scale = COPY_CALIBRATION_BYTES / (cw * 1024.0)
    for kernel in KERNEL_SOURCES:
        fv, wv = find(fetch, kernel), find(write, kernel)
        f_kib, w_kib = sum(fv) / len(fv), sum(wv) / len(wv)
        total = f_kib * 1024.0 * f_scale + w_kib * 1024.0 * w_scale
        lines = [
            f"# {kernel}: HBM traffic per launch, {workload}",
            "",
            "Two counter passes over the whole benchmark (one per counter), each with the",
            "calibration copy of 256 MiB run first:",
            "",
            "```",
            "cd /tmp && export TMPDIR=/tmp",
            "timeout -s KILL 600 rocprofv3 --pmc FETCH_SIZE --output-format csv -d <out>/fetch -o fetch -- \\",
            f"    python /root/repo/bench.py {bench_args()} --no-cpu-baseline --copy-calibration",
            "timeout -s KILL 600 rocprofv3 --pmc WRITE_SIZE --output-format csv -d <out>/write -o write -- \\",
            f"    python /root/repo/bench.py {bench_args()} --no-cpu-baseline --copy-calibration",
            f"python /root/repo/bench.py {bench_args()} --pmc-summary <out>/fetch <out>/write",
            "```",
            "",
            f"- dispatches: {len(fv)} (FETCH_SIZE pass), {len(wv)} (WRITE_SIZE pass)"
            + (", those of the timed frames" if steps and layers else ""),
            f"- fetch_kib_per_dispatch_mean: {f_kib:.1f}",
            f"- write_kib_per_dispatch_mean: {w_kib:.1f}",
            f"- copy_fetch_kib: {cf:.1f} (for {COPY_CALIBRATION_BYTES} bytes read)",
            f"- copy_write_kib: {cw:.1f} (for {COPY_CALIBRATION_BYTES} bytes written)",
            f"- fetch_scale: {f_scale:.4f}",
            f"- write_scale: {w_scale:.4f}",
            f"- hbm_bytes_per_launch: {total:.0f}",
            f"- source_hash: {kernel_source_hash(kernel)}",
            "",
            "The source hash covers the code (comments and whitespace removed) of "
            + ", ".join(KERNEL_SOURCES[kernel]) + "; the benchmark",
            "reports this traffic only while that code is unchanged.",
        ]
        path = traffic_path(kernel, workload)
        with open(path, "w") as fh:
            fh.write("\n".join(lines) + "\n")
        print(f"{kernel}: {f_kib:.1f} KiB fetched, {w_kib:.1f} KiB written per dispatch -> "
              f"{total / 1e6:.2f} MB per launch ({path})")


MFMA_PASSES = (("SQ_VALU_MFMA_BUSY_CYCLES", "SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_VALU_MFMA_COEXEC_CYCLES",
                "SQ_INSTS_MFMA", "GRBM_GUI_ACTIVE"),
               ("SQ_ACTIVE_INST_VALU", "SQ_INSTS_VALU", "SQ_INSTS_VALU_TRANS_F32", "SQ_BUSY_CYCLES",
                "GRBM_GUI_ACTIVE"),
               ("SQ_WAVE_CYCLES", "SQ_WAIT_ANY", "SQ_WAIT_INST_ANY", "SQ_ACTIVE_INST_ANY", "SQ_LDS_IDX_ACTIVE",
                "SQ_LDS_BANK_CONFLICT", "GRBM_GUI_ACTIVE"))
MI355X_XCDS, MI355X_SIMDS = 8, 1024    # 8 XCDs x 32 CUs x 4 SIMDs


def mfma_path(workload):
    return os.path.join(PROFILES, f"attn_fwd_kernel__{workload}__mfma.md")


def summarize_mfma(dir_a, dir_b, dir_c, bench_json, workload):
    """Reduce three rocprofv3 --pmc runs of this benchmark (the counters of MFMA_PASSES) into
    per-dispatch matrix-core, vector-ALU and wave-state activity of each kernel over the
    timed frames' dispatches, and tie the attention kernel's to the benchmark line of the
    same command (bench_json)."""
    bench = json.loads(open(bench_json).read().strip().splitlines()[-1])

    def per_kernel(d):
        out = {}
        for r in timed_counter_rows(counter_rows(d), bench["steps"], bench["config"].get("layers")):
            name = r["Kernel_Name"].replace("rv::(anonymous namespace)::", "").split("(")[0]
            out.setdefault(name, {}).setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
            if r["Counter_Name"] == "GRBM_GUI_ACTIVE":
                out[name].setdefault("duration_ns", []).append(
                    float(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])))
        return out

    a, b, w = per_kernel(dir_a), per_kernel(dir_b), per_kernel(dir_c)
    mean = lambda v: sum(v) / len(v)
    lines = [f"# Matrix-core and vector-ALU activity per dispatch, {workload}", "",
             "Three counter passes over the benchmark command (one run each, the program after `--`):", "",
             "```", "cd /tmp && export TMPDIR=/tmp"]
    for i, cs in enumerate(MFMA_PASSES):
        lines.append(f"timeout -s KILL 600 rocprofv3 --pmc {' '.join(cs)} --output-format csv -d <out>/m{i} "
                     f"-o m{i} -- python /root/repo/bench.py {bench_args()} --no-cpu-baseline")
    lines += [f"python /root/repo/bench.py {bench_args()} --mfma-summary <out>/m0 <out>/m1 <out>/m2 "
              "<kernel-trace run's json>",
              "```",
              "", "Counters are summed over the chip (GRBM_GUI_ACTIVE over its 8 XCDs).  Per dispatch:",
              "`busy` = SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / 8 x 1024 SIMDs), the fraction of SIMD",
              "cycles the matrix core is busy (rocprofv3's MfmaUtil); `busy@2.4` = the same busy cycles over",
              "1024 SIMDs x the dispatch's duration (its timestamps) x 2.4 GHz, i.e. executed MFMA work as a",
              "fraction of the dense peak (dispatches run one at a time under counter collection, so the",
              "durations are a little longer than in the kernel trace); `coexec` = SQ_VALU_MFMA_COEXEC_CYCLES /",
              "SQ_VALU_MFMA_BUSY_CYCLES, the share of those cycles in which a vector instruction was also",
              "issued; `valu` = 4 x SQ_ACTIVE_INST_VALU / (GRBM_GUI_ACTIVE / 8 x 1024), vector-ALU cycles per",
              "SIMD cycle (quad-cycle units); `bf16 flops` = 512 x SQ_INSTS_VALU_MFMA_MOPS_BF16.  Wave states",
              "(shares of SQ_WAVE_CYCLES, the cycles waves are resident): `issuing` = SQ_ACTIVE_INST_ANY,",
              "`waiting` = SQ_WAIT_ANY (on a counter -- memory, LDS -- or a barrier), `ready` = SQ_WAIT_INST_ANY",
              "(an instruction ready but not issued); `lds conflict` = SQ_LDS_BANK_CONFLICT / SQ_LDS_IDX_ACTIVE.",
              "",
              "| Kernel | dispatches | duration us | GUI cycles / XCD | busy | busy@2.4 | coexec | valu | MFMA instrs | "
              "bf16 flops | VALU instrs | exp/log (f32 trans) instrs | issuing | waiting | ready | lds conflict |",
              "|---|---|---|---|---|---|---|---|---|---|---|---|---|---|---|---|"]
    rows = {}
    for name in sorted(set(a) | set(b)):
        if name not in KERNEL_SOURCES:
            continue
        ca, cb, cw = a.get(name, {}), b.get(name, {}), w.get(name, {})
        try:
            gui = mean(ca["GRBM_GUI_ACTIVE"]) / MI355X_XCDS
            busy = mean(ca["SQ_VALU_MFMA_BUSY_CYCLES"])
            dur = mean(ca["duration_ns"])
            r = {"n": len(ca["GRBM_GUI_ACTIVE"]), "gui": gui, "busy": busy / (gui * MI355X_SIMDS),
                 "dur": dur, "busy24": busy / (MI355X_SIMDS * dur * 2.4),
                 "coexec": mean(ca["SQ_VALU_MFMA_COEXEC_CYCLES"]) / max(busy, 1.0),
                 "mfma": mean(ca["SQ_INSTS_MFMA"]), "flops": 512.0 * mean(ca["SQ_INSTS_VALU_MFMA_MOPS_BF16"]),
                 "valu": 4.0 * mean(cb["SQ_ACTIVE_INST_VALU"]) / (mean(cb["GRBM_GUI_ACTIVE"]) / MI355X_XCDS
                                                                 * MI355X_SIMDS),
                 "vinst": mean(cb["SQ_INSTS_VALU"]), "trans": mean(cb["SQ_INSTS_VALU_TRANS_F32"])}
            wc = max(mean(cw["SQ_WAVE_CYCLES"]), 1.0)
            r.update({"issuing": mean(cw["SQ_ACTIVE_INST_ANY"]) / wc, "waiting": mean(cw["SQ_WAIT_ANY"]) / wc,
                      "ready": mean(cw["SQ_WAIT_INST_ANY"]) / wc,
                      "ldsconf": mean(cw["SQ_LDS_BANK_CONFLICT"]) / max(mean(cw["SQ_LDS_IDX_ACTIVE"]), 1.0)})
        except KeyError as e:
            raise SystemExit(f"{name}: counter {e} missing from the CSVs")
        rows[name] = r
        lines.append(f"| `{name}` | {r['n']} | {r['dur'] / 1e3:.1f} | {r['gui']:.0f} | {100 * r['busy']:.1f} % | "
                     f"{100 * r['busy24']:.1f} % | {100 * r['coexec']:.1f} % | "
                     f"{100 * r['valu']:.1f} % | {r['mfma']:.0f} | {r['flops']:.3e} | {r['vinst']:.0f} | "
                     f"{r['trans']:.0f} | {100 * r['issuing']:.0f} % | {100 * r['waiting']:.0f} % | "
                     f"{100 * r['ready']:.0f} % | {100 * r['ldsconf']:.0f} % |")
    f = rows.get("attn_fwd_kernel")
    if f:
        alg = bench["roofline"]["algorithmic_flops_per_launch"]
        lines += ["", "The attention forward kernel against the benchmark line of the same command (its kernel-trace",
                  "run, whose line is not distorted by counter collection):", "",
                  f"- algorithmic flops per launch (4 x 64 per query-key pair): {alg:.4e}; bf16 MFMA flops "
                  f"executed per dispatch: {f['flops']:.4e} (x{f['flops'] / alg:.3f}: query tiles padded to 128 "
                  "rows and key tiles to 64)",
                  f"- executed MFMA work {100 * f['busy24']:.1f} % of the dense peak over the dispatch's own "
                  f"duration; matrix core busy {100 * f['busy']:.1f} % of SIMD cycles; a vector instruction issued in "
                  f"{100 * f['coexec']:.1f} % of those; vector ALU active {100 * f['valu']:.1f} % of SIMD cycles",
                  f"- waves issue in {100 * f['issuing']:.0f} % of their resident cycles, wait on a counter or barrier "
                  f"in {100 * f['waiting']:.0f} % and hold a ready instruction that is not issued in "
                  f"{100 * f['ready']:.0f} %",
                  f"- benchmark line: {bench['roofline']['achieved']:.1f} TFLOP/s = "
                  f"{100 * bench['roofline']['frac']:.1f} % of {bench['roofline']['peak']} TFLOP/s for the "
                  f"attention step (forward + merge launches, {bench['roofline']['avg_launch_us']:.1f} us per "
                  "layer by HIP events)",
                  f"- source_hash: {kernel_source_hash('attn_fwd_kernel')}"]
    path = mfma_path(workload)
    with open(path, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print(f"wrote {path}")


def summarize_trace(trace_dir, bench_json, workload):
    """Write profiles/kernel_trace__<workload>.md from a rocprofv3 --kernel-trace --stats
    run of this benchmark (its *_kernel_trace.csv, the timed frames' dispatches: see
    timed_start) and the JSON line that run printed."""
    import csv
    traces = glob.glob(os.path.join(trace_dir, "**", "*kernel_trace.csv"), recursive=True)
    if not traces:
        raise SystemExit(f"no kernel_trace.csv under {trace_dir}")
    bench = json.loads(open(bench_json).read().strip().splitlines()[-1])

    def short(name):
        name = name.replace("rv::(anonymous namespace)::", "").replace("(anonymous namespace)::", "")
        return name.split("(")[0]

    disp = [(r["Kernel_Name"], int(r["Start_Timestamp"]), int(r["End_Timestamp"]))
            for r in csv.DictReader(open(traces[0]))]
    t0 = timed_start([(n, t) for n, t, _ in disp], bench["steps"], bench["config"].get("layers"))
    durs = {}
    for n, t, e in disp:
        if t0 is None or t >= t0:
            durs.setdefault(short(n), []).append(e - t)
    grand = sum(sum(v) for v in durs.values()) or 1
    rows = sorted(({"Name": k, "Calls": len(v), "TotalDurationNs": sum(v), "AverageNs": sum(v) / len(v),
                    "Percentage": 100.0 * sum(v) / grand, "MinNs": min(v), "MaxNs": max(v)}
                   for k, v in durs.items()), key=lambda r: -r["TotalDurationNs"])
    avg = {r["Name"]: r["AverageNs"] / 1e3 for r in rows}
    total = {r["Name"]: r["TotalDurationNs"] / 1e3 for r in rows}
    calls = {r["Name"]: r["Calls"] for r in rows}
    # One attention step = attn_fwd_kernel, plus attn_merge_kernel for a split plan.
    attn_step = ((total.get("attn_fwd_kernel", 0.0) + total.get("attn_merge_kernel", 0.0))
                 / max(calls.get("attn_fwd_kernel", 1), 1))
    lines = [f"# Kernel time summary: {workload} benchmark", "",
             "Command (on the MI355X, from the repository root):", "", "```",
             "cd /tmp && export TMPDIR=/tmp",
             "rocprofv3 --kernel-trace --stats --output-format csv -d <out>/trace -o bench -- \\",
             f"    python /root/repo/bench.py {bench_args()} --no-cpu-baseline > <out>/trace.json",
             f"python /root/repo/bench.py {bench_args()} --trace-summary <out>/trace <out>/trace.json", "```", "",
             "Kernel statistics of the timed frames' dispatches (durations in ns, from the trace:",
             "everything from the first of the timed frames' attention launches on; the input",
             "generation and the warm-up frames before it are left out):", "",
             "| Kernel | Calls | Total ns | Average ns | % | Min ns | Max ns |", "|---|---|---|---|---|---|---|"]
    for r in rows:
        lines.append(f"| `{r['Name']}` | {r['Calls']} | {int(r['TotalDurationNs'])} | "
                     f"{r['AverageNs']:.0f} | {r['Percentage']:.2f} | {r['MinNs']} | {r['MaxNs']} |")
    adm = sum(avg.get(k, 0.0) for k in ADMISSION_KERNELS)
    lines += ["", "The same run's benchmark line (HIP events on the compute stream):", "",
              f"- frames/s: {bench['value']:.1f}",
              f"- attention: {bench['roofline']['avg_launch_us']:.1f} us per layer step (events around "
              f"the forward launch and, for split plans, the merge launch) vs {attn_step:.1f} us "
              f"(rocprofv3: attn_fwd_kernel + attn_merge_kernel time per attn_fwd_kernel call; "
              f"attn_fwd_kernel alone averages {avg.get('attn_fwd_kernel', 0.0):.1f} us)",
              f"- admission: {bench['phases']['admission_ms'] / bench['steps'] * 1e3:.1f} us per frame (events; "
              f"the pair also spans the launch gaps) vs {adm:.1f} us (rocprofv3 averages of "
              + " + ".join(ADMISSION_KERNELS) + ")",
              f"- attention roofline: {bench['roofline']['achieved']:.1f} TFLOP/s = "
              f"{100 * bench['roofline']['frac']:.1f} % of {bench['roofline']['peak']}"]
    path = os.path.join(PROFILES, f"kernel_trace__{workload}.md")
    with open(path, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print(f"wrote {path}")


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(cfg, samples, budget, qs, mem_len, mean_ctx):
    """Time the oracle as it stands on a bounded sample of the timed workload: for each
    (layer, frame) in `samples`, one layer of that frame (all heads, all queries,
    LSE-saliency, top-k, append) at the memory length that frame has in the stream.
    Frames per second = 1 / (mean time per layer-frame x layers x (stream mean context /
    sample mean context))."""
    import oracle
    from paper_2609_23286_amd import synth
    N, H = cfg.n_tokens, cfg.n_heads
    qidx = oracle.qsub_index(*qs)
    rows = max(mem_len(l, t) for l, t in samples) + budget
    memK, memV = synth.memory_prefill(cfg, 0, rows)   # memory rows; contents do not affect time
    omem = oracle.Memory(H, cfg.head_dim, rows)
    omem.K[:], omem.V[:] = memK, memV
    dt, ctx = 0.0, 0
    for l, t in samples:
        Q, K, V = synth.frame_qkv(cfg, l, t)
        omem.len = mem_len(l, t)
        ctx += omem.len + N
        t0 = time.perf_counter()
        oracle.step(omem, Q, K, V, qidx, budget)
        dt += time.perf_counter() - t0
    per_layer = dt / len(samples)
    per_frame = per_layer * cfg.n_layers * (mean_ctx / (ctx / len(samples)))
    return {"value": 1.0 / per_frame, "unit": "frames/s", "cores": oracle.num_threads(),
            "cpu_model": cpu_model(), "kind": "oracle",
            "sample": (f"{len(samples)} layer-frames of the timed frames (one layer each: {H} heads, all {N} "
                       f"queries, saliency, top-{budget}, append) at their stream memory lengths, mean "
                       f"context {ctx / len(samples):.0f}, {dt:.1f} s in all; scaled x{cfg.n_layers} layers "
                       f"and to the timed frames' mean context {mean_ctx:.0f}")}


def unit_rates():
    """Matrix-core and vector-ALU (exponential) rates and their overlap on this GPU: one
    workgroup of eight waves per CU runs the probe of rvs_unit_rates; prints one JSON line
    (--unit-rates-summary turns it into profiles/unit_rates__mi355x.md)."""
    import ctypes
    import torch
    from paper_2609_23286_amd import rv
    torch.cuda.set_device(0)
    n_cus = torch.cuda.get_device_properties(0).multi_processor_count
    iters = 4000
    s = rv._load_synth()
    s.rvs_unit_rates.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.POINTER(ctypes.c_float)]
    s.rvs_unit_rates.restype = ctypes.c_int
    ns = (ctypes.c_float * 11)()
    if s.rvs_unit_rates(n_cus, iters, ns):
        raise SystemExit("rvs_unit_rates failed")
    keys = ("mfma_wave", "valu_wave", "mfma_wave_and_valu_wave", "one_wave_both", "two_mfma_waves",
            "two_mfma_waves_zero_operands", "two_valu_waves", "fma_wave", "two_fma_waves", "exp_wave",
            "two_exp_waves")
    print(json.dumps({"ns_per_iter": dict(zip(keys, (float(x) for x in ns))), "cus": n_cus, "iterations": iters}),
          flush=True)


def unit_rates_summary(json_path):
    r = json.loads(open(json_path).read().strip().splitlines()[-1])
    t = r["ns_per_iter"]
    t_m, t_v, t_mv, t_b, t_mm, t_mz, t_vv = (t[k] for k in (
        "mfma_wave", "valu_wave", "mfma_wave_and_valu_wave", "one_wave_both", "two_mfma_waves",
        "two_mfma_waves_zero_operands", "two_valu_waves"))
    t_f, t_ff, t_e, t_ee = (t[k] for k in ("fma_wave", "two_fma_waves", "exp_wave", "two_exp_waves"))
    hidden = (t_m + t_v - t_mv) / t_m
    clk_mfma = 32 / (t_mm / 8)        # GHz if an MFMA takes its 32 cycles
    clk = 2.4                          # the vector-ALU modes' clock under counters (2.37-2.40 GHz)
    fma_1, fma_2 = t_f * clk / 32, t_ff * clk / 64      # SIMD cycles per FMA: one wave, two waves
    exp_1, exp_2 = t_e * clk / 32, t_ee * clk / 64
    # the chained VALU body (16 exponentials, 32 FMA/add) at the single-unit costs of two waves
    body_pred = 16 * exp_2 + 32 * fma_2
    lines = ["# Unit rates on one MI355X: matrix core, vector-ALU exponentials, and their overlap", "",
             "Command (on the MI355X, from the repository root):", "", "```",
             "python bench.py --unit-rates > unit_rates.json",
             "python bench.py --unit-rates-summary unit_rates.json", "```", "",
             f"One workgroup of eight waves per CU ({r['cus']} CUs; wave w runs on SIMD w % 4), "
             f"{r['iterations']} iterations of:",
             "MFMA body = 4 independent `v_mfma_f32_32x32x16_bf16`; VALU body = 8 independent chains of",
             "2 x (FMA, `v_exp_f32`, add) = 16 exponentials + 32 FMA/add; FMA body = 32 independent FMAs;",
             "exp body = 32 independent `v_exp_f32`.  Time per iteration:", "",
             "| Waves per SIMD | ns per iteration |", "|---|---|",
             f"| one MFMA wave | {t_m:.1f} |", f"| two MFMA waves | {t_mm:.1f} (two bodies) |",
             f"| two MFMA waves, all-zero operands | {t_mz:.1f} (two bodies) |",
             f"| one VALU wave | {t_v:.1f} |", f"| two VALU waves | {t_vv:.1f} (two bodies) |",
             f"| one MFMA wave + one VALU wave | {t_mv:.1f} |",
             f"| one wave running both bodies | {t_b:.1f} |",
             f"| one FMA wave | {t_f:.1f} |", f"| two FMA waves | {t_ff:.1f} (two bodies) |",
             f"| one exp wave | {t_e:.1f} |", f"| two exp waves | {t_ee:.1f} (two bodies) |", "",
             f"- two MFMA waves per SIMD: {t_mm / 8:.1f} ns per 32x32x16 bf16 MFMA; at its 32 cycles the SIMD "
             f"runs at {clk_mfma:.2f} GHz ({100 * clk_mfma / 2.4:.0f} % of the 2.4 GHz of the dense peak); "
             f"{t_mz / 8:.1f} ns with all-zero operands ({32 / (t_mz / 8):.2f} GHz at the same cycle count)",
             f"- independent FMAs (cycles at {clk} GHz, about the clock of the vector-ALU modes under "
             f"counters): {fma_1:.1f} SIMD cycles each from one wave (one wave's issue limit), {fma_2:.1f} from two",
             f"- independent exponentials: {exp_1:.1f} SIMD cycles each from one wave, {exp_2:.1f} from two: with "
             f"two waves issuing, `v_exp_f32` holds the vector ALU {exp_2 / fma_2:.1f}x as long as an FMA",
             f"- two VALU waves per SIMD: {t_vv:.1f} ns for two bodies = {t_vv * clk / 2:.0f} cycles per body "
             f"against {body_pred:.0f} at the single-unit costs above (the chains' dependencies cost the rest)",
             f"- one VALU wave alone: {t_v:.1f} ns per body, {t_v / (t_vv / 2):.2f}x the two-wave time per body: one "
             "wave's issue limit and its exponential-to-add dependencies leave the vector ALU idle part of the time",
             f"- one MFMA wave alone: {t_m / 4:.1f} ns per MFMA (one wave's loop leaves issue gaps that a second "
             "wave fills)",
             f"- share of the MFMA time hidden under VALU work on the same SIMD (one wave of each): "
             f"{100 * hidden:.0f} %"]
    path = os.path.join(PROFILES, "unit_rates__mi355x.md")
    with open(path, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print(f"wrote {path}")


UNIT_RATE_COUNTERS = ("SQ_ACTIVE_INST_VALU", "SQ_INSTS_VALU", "SQ_INSTS_VALU_TRANS_F32", "SQ_VALU_MFMA_BUSY_CYCLES",
                      "GRBM_GUI_ACTIVE")
UNIT_RATE_MODES = ("one MFMA wave", "one VALU wave", "one MFMA wave + one VALU wave", "one wave running both bodies",
                   "two MFMA waves", "two MFMA waves, all-zero operands", "two VALU waves", "one FMA wave",
                   "two FMA waves", "one exp wave", "two exp waves")


def unit_rates_counters(counter_dir, iters=4000):
    """Write profiles/unit_rates__mi355x__counters.md from a rocprofv3 --pmc run (the
    counters of UNIT_RATE_COUNTERS) of `bench.py --unit-rates`: per probe mode, the clock
    the chip ran at and how busy the vector ALU and the matrix core were."""
    import csv
    import re
    acc = {}
    for f in glob.glob(os.path.join(counter_dir, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            m = re.search(r"(?:unit|issue)_rate_kernel<(\d+)>", r["Kernel_Name"])
            if not m:
                continue
            d = acc.setdefault((int(m.group(1)), r["Dispatch_Id"]), {})
            d[r["Counter_Name"]] = float(r["Counter_Value"])
            d["ns"] = float(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
    if not acc:
        raise SystemExit(f"no unit_rate_kernel dispatches under {counter_dir}")
    lines = ["# Unit-rate probe under counters: clock, vector-ALU and matrix-core activity per mode", "",
             "Command (on the MI355X, from the repository root; the program after `--`):", "", "```",
             "cd /tmp && export TMPDIR=/tmp",
             f"timeout -s KILL 120 rocprofv3 --pmc {' '.join(UNIT_RATE_COUNTERS)} --output-format csv "
             "-d <out>/ur -o ur -- python /root/repo/bench.py --unit-rates",
             "python /root/repo/bench.py --unit-rates-counters <out>/ur", "```", "",
             "Each mode launches twice with the same iteration count (a warm-up, then the timed launch); the",
             "rows average both.  `clock` = GRBM_GUI_ACTIVE / 8 XCDs / the dispatch's duration; `valu busy` =",
             "4 x SQ_ACTIVE_INST_VALU / (GUI cycles per XCD x 1024 SIMDs), counted over all SIMDs whether or",
             "not the mode gives them VALU work; `mfma busy` = SQ_VALU_MFMA_BUSY_CYCLES over the same SIMD",
             f"cycles; instructions are per VALU-issuing wave and iteration ({iters} iterations).", "",
             "| Mode | ns per iteration | clock GHz | valu busy | mfma busy | VALU instrs / wave / iter | "
             "of them exp |", "|---|---|---|---|---|---|---|"]
    valu_waves = {0: 4, 1: 4, 2: 8, 3: 4, 4: 8, 5: 8, 6: 8, 7: 4, 8: 8, 9: 4, 10: 8}  # waves issuing VALU (MFMA counts)
    for mode in sorted({k[0] for k in acc}):
        ds = [d for (m, _), d in acc.items() if m == mode]
        mean = lambda key: sum(d[key] for d in ds) / len(ds)
        ns = mean("ns")
        gui = mean("GRBM_GUI_ACTIVE") / MI355X_XCDS
        simd = gui * MI355X_SIMDS
        n_waves = 256 * valu_waves[mode]
        lines.append(f"| {UNIT_RATE_MODES[mode] if mode < len(UNIT_RATE_MODES) else mode} | "
                     f"{ns / iters:.1f} | {gui / ns:.2f} | {100 * 4 * mean('SQ_ACTIVE_INST_VALU') / simd:.1f} % | "
                     f"{100 * mean('SQ_VALU_MFMA_BUSY_CYCLES') / simd:.1f} % | "
                     f"{mean('SQ_INSTS_VALU') / n_waves / iters:.1f} | "
                     f"{mean('SQ_INSTS_VALU_TRANS_F32') / n_waves / iters:.1f} |")
    path = os.path.join(PROFILES, "unit_rates__mi355x__counters.md")
    with open(path, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print(f"wrote {path}")


def library_context(config_name):
    """The attention layer step beside the vendor stack on the same inputs: rv_attend_frame
    (outputs and LSE) against torch's fused scaled_dot_product_attention (flash, then
    memory-efficient backend; never the unfused path) over the same [memory ; frame] keys,
    at several memory lengths, plus a dense bf16 GEMM for the sustained matrix rate.  Prints
    one JSON line (--library-context-summary writes the profile)."""
    import torch
    import torch.nn.functional as F
    from torch.nn.attention import SDPBackend, sdpa_kernel
    from paper_2609_23286_amd import rv, synth
    cfg = synth.CONFIGS[config_name]
    N, H, d = cfg.n_tokens, cfg.n_heads, cfg.head_dim
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    rv.init()
    reps = 50
    m_list = [0, 2000, 5000, 9990]
    buf = torch.empty((1, 3, N, H, d), dtype=torch.int16, device=dev)
    rv.gpu_frame_qkv(cfg, 1, buf, 0, 1)
    Qf, Kf, Vf = buf[0, 0], buf[0, 1], buf[0, 2]
    mk = torch.empty((H, max(m_list), d), dtype=torch.int16, device=dev)
    mv = torch.empty_like(mk)
    rv.gpu_normal(cfg.seed, synth.PREFILL_FRAME, 0, synth.TAG_MEMK, mk, cfg.sigma)
    rv.gpu_normal(cfg.seed, synth.PREFILL_FRAME, 0, synth.TAG_MEMV, mv, cfg.sigma)
    rv.reserve_workspace(N, H, max(m_list), 1)
    out = torch.empty_like(Qf)
    lse = torch.empty((H, N), dtype=torch.float32, device=dev)
    q_b = Qf.view(torch.bfloat16).permute(1, 0, 2).unsqueeze(0).contiguous()

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        e1.synchronize()
        return e0.elapsed_time(e1) * 1e3 / reps

    rows = []
    for M in m_list:
        mkM = mk[:, :M].contiguous()
        mvM = mv[:, :M].contiguous()
        ctx = M + N
        flops = attention_flops(N, H, d, ctx)
        row = {"mem_len": M, "context": ctx, "flops": flops}
        rv.attend_frame(Qf, Kf, Vf, None, out, lse, memK=mkM, memV=mvM, mem_len=M, head_stride=M)
        # raw C call with pre-marshalled arguments, so that the host stays ahead of the GPU
        import ctypes
        lib, vp = rv.lib(), ctypes.c_void_p
        c_args = (vp(Qf.data_ptr()), vp(Kf.data_ptr()), vp(Vf.data_ptr()), N, vp(mkM.data_ptr() if M else 0),
                  vp(mvM.data_ptr() if M else 0), M, M, H, d, None, vp(out.data_ptr()), vp(lse.data_ptr()), None,
                  vp(torch.cuda.current_stream().cuda_stream))
        if lib.rv_attend_frame(*c_args):
            raise rv.RVError(1, lib.rv_last_error().decode())
        row["rv_us"] = timed(lambda: lib.rv_attend_frame(*c_args))
        k_b = torch.cat([mkM, Kf.permute(1, 0, 2)], dim=1).view(torch.bfloat16).unsqueeze(0).contiguous()
        v_b = torch.cat([mvM, Vf.permute(1, 0, 2)], dim=1).view(torch.bfloat16).unsqueeze(0).contiguous()
        ours = (out.view(torch.bfloat16).float().permute(1, 0, 2))
        for name, backend in (("flash", SDPBackend.FLASH_ATTENTION), ("efficient", SDPBackend.EFFICIENT_ATTENTION)):
            try:
                with sdpa_kernel([backend]):
                    o = F.scaled_dot_product_attention(q_b, k_b, v_b)
                    torch.cuda.synchronize()
                    row[f"{name}_us"] = timed(lambda: F.scaled_dot_product_attention(q_b, k_b, v_b))
                row[f"{name}_max_abs_diff"] = float((o[0].float() - ours).abs().max())
            except RuntimeError as exc:
                row[f"{name}_us"] = None
                row[f"{name}_error"] = str(exc).splitlines()[0][:160]
        rows.append(row)
        log(json.dumps(row))
        del k_b, v_b, mkM, mvM
    n = 8192
    a = torch.randn((n, n), dtype=torch.bfloat16, device=dev)
    b = torch.randn((n, n), dtype=torch.bfloat16, device=dev)
    c = torch.empty((n, n), dtype=torch.bfloat16, device=dev)
    gemm_us = timed(lambda: torch.matmul(a, b, out=c))
    gemm = {"m": n, "n": n, "k": n, "us": gemm_us, "tflops": 2 * n ** 3 / gemm_us / 1e6}
    print(json.dumps({"config": config_name, "tokens": N, "heads": H, "head_dim": d, "reps": reps,
                      "rows": rows, "gemm_bf16": gemm, "torch": torch.__version__,
                      "hip": getattr(torch.version, "hip", None)}), flush=True)


def library_context_summary(json_path):
    r = json.loads(open(json_path).read().strip().splitlines()[-1])
    N, H, d = r["tokens"], r["heads"], r["head_dim"]
    lines = [f"# Attention layer step ({N} queries x {H} heads x {d}, memory + frame keys) beside torch's fused "
             "attention on one MI355X", "",
             "Command (on the MI355X, from the repository root):", "", "```",
             f"python bench.py --config {r['config']} --library-context > library_context.json",
             "python bench.py --library-context-summary library_context.json", "```", "",
             f"Same inputs for both (frame 1 of the {r['config']} stream, layer 0; memory rows from the prefill "
             f"generator), mean of {r['reps']} back-to-back calls after one untimed call, HIP events on one "
             f"stream.  `rv_attend_frame` also writes the per-query LSE; torch's call returns the output only "
             f"(torch {r['torch']}, HIP {r['hip']}).  TFLOP/s counts 4 N H d (M + N) per call; the peak is "
             f"{PEAK_BF16_TFLOPS} TFLOP/s.", "",
             "| memory rows M | rv_attend_frame us | TFLOP/s (% peak) | torch flash us | torch mem-efficient us "
             "| rv speed-up vs best torch | max abs diff of outputs |",
             "|---|---|---|---|---|---|---|"]
    for row in r["rows"]:
        tf = row["flops"] / row["rv_us"] / 1e6
        cand = [row.get("flash_us"), row.get("efficient_us")]
        cand = [c for c in cand if c]
        best = min(cand) if cand else None
        fmt = lambda v: f"{v:.1f}" if v else "n/a"
        diffs = [row.get(k) for k in ("flash_max_abs_diff", "efficient_max_abs_diff") if row.get(k) is not None]
        lines.append(f"| {row['mem_len']} | {row['rv_us']:.1f} | {tf:.0f} ({100 * tf / PEAK_BF16_TFLOPS:.1f} %) | "
                     f"{fmt(row.get('flash_us'))} | {fmt(row.get('efficient_us'))} | "
                     f"{(best / row['rv_us']) if best else float('nan'):.2f}x | "
                     f"{max(diffs) if diffs else float('nan'):.3g} |")
    errs = sorted({row[k] for row in r["rows"] for k in ("flash_error", "efficient_error") if row.get(k)})
    for e in errs:
        lines.append(f"\nA torch backend was unavailable: {e}")
    g = r["gemm_bf16"]
    lines += ["", f"Dense bf16 GEMM through torch.matmul ({g['m']} x {g['n']} x {g['k']}): {g['us']:.0f} us = "
              f"{g['tflops']:.0f} TFLOP/s = {100 * g['tflops'] / PEAK_BF16_TFLOPS:.1f} % of the dense peak "
              "(the library's sustained matrix rate on this GPU)."]
    path = os.path.join(PROFILES, f"attention_vs_torch_sdpa__{r['config']}_layer_step.md")
    with open(path, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print(f"wrote {path}")


def stratified(n_stream, n):
    """n frames of an n_stream-frame stream, one from the middle of each of n equal
    stretches: t_i = floor((i + 1/2) n_stream / n)."""
    return [int((i + 0.5) * n_stream / n) for i in range(n)]


def workload_key(cfg, n_stream, steps, variant):
    """Name under which counter profiles of this run are filed (None for variants)."""
    if variant:
        return None
    return cfg.name if steps >= n_stream else f"{cfg.name}__{steps}of{n_stream}"


def main():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=1000,
                   help="frames timed; fewer than the stream's frames times a stratified sample of them "
                        "(frame t_i = floor((i + 1/2) T / steps), each at the memory length it has in the stream)")
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--config", default="vitl_stack_1000")
    p.add_argument("--stream-frames", type=int, default=None,
                   help="length T of the stream the frames are drawn from (default: the configuration's)")
    p.add_argument("--policy", choices=("all", "paper"), default="all",
                   help="all: every layer regulated, no anchor (the configuration's setting); paper: "
                        "layers 11-17 regulated, first frame kept whole in every layer (Sec. 4.1)")
    p.add_argument("--stride", type=int, default=None, help="query window s (default: the config's, 2)")
    p.add_argument("--gamma", type=float, default=None, help="retention rate: budget = floor(gamma N)")
    p.add_argument("--shared", action="store_true",
                   help="head-averaged selection (one top-k per layer) instead of head-specific")
    p.add_argument("--staged", action="store_true",
                   help="stage each frame's K/V in the memory arenas (rv_mem_stage_frames, timed as its "
                        "own phase), attend over the contiguous arena (rv_attend_staged) and admit by "
                        "in-place compaction (rv_admit_staged_layers)")
    p.add_argument("--fused", action="store_true",
                   help="saliency in the attention epilogue (rv_attend_frame_fused, per 128-query block) "
                        "and admission from those rows (rv_admit_layers_tiled)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-samples", type=int, default=24, help="layer-frames the oracle is timed on")
    p.add_argument("--copy-calibration", action="store_true",
                   help="run a 256 MiB device copy before the stream (HBM counter calibration)")
    p.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                   help="summarise two rocprofv3 --pmc runs of this command into profiles/ and exit")
    p.add_argument("--mfma-summary", nargs=4, metavar=("PASS0_DIR", "PASS1_DIR", "PASS2_DIR", "BENCH_JSON"),
                   help="summarise the three rocprofv3 --pmc passes of MFMA_PASSES over this command into "
                        "profiles/ and exit")
    p.add_argument("--unit-rates", action="store_true",
                   help="measure the matrix-core and exponential rates and their overlap (one JSON line) and exit")
    p.add_argument("--unit-rates-summary", metavar="JSON", help="write profiles/unit_rates__mi355x.md and exit")
    p.add_argument("--unit-rates-counters", metavar="DIR",
                   help="write profiles/unit_rates__mi355x__counters.md from a rocprofv3 --pmc run of --unit-rates "
                        "and exit")
    p.add_argument("--library-context", action="store_true",
                   help="time the attention layer step beside torch's fused attention on the same inputs "
                        "(one JSON line) and exit")
    p.add_argument("--library-context-summary", metavar="JSON",
                   help="write profiles/attention_vs_torch_sdpa__<config>_layer_step.md and exit")
    p.add_argument("--trace-summary", nargs=2, metavar=("TRACE_DIR", "BENCH_JSON"),
                   help="summarise a rocprofv3 --kernel-trace --stats run of this command into profiles/ "
                        "and exit")
    args = p.parse_args()
    if args.unit_rates:
        unit_rates()
        return
    if args.unit_rates_summary:
        unit_rates_summary(args.unit_rates_summary)
        return
    if args.unit_rates_counters:
        unit_rates_counters(args.unit_rates_counters)
        return
    if args.library_context:
        library_context(args.config)
        return
    if args.library_context_summary:
        library_context_summary(args.library_context_summary)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: this path has no multi-GPU mode "
              f"(--gpus {args.gpus} requested)", file=sys.stderr)
        sys.exit(2)

    from paper_2609_23286_amd import synth
    cfg = synth.CONFIGS[args.config]
    L, H, N, d, k = cfg.n_layers, cfg.n_heads, cfg.n_tokens, cfg.head_dim, cfg.budget
    if args.gamma is not None:
        k = int(args.gamma * N)
    stride = args.stride or cfg.stride
    n_stream = args.stream_frames or cfg.n_frames
    K_steps, W = args.steps, args.warmup
    if not 1 <= K_steps <= n_stream:
        raise SystemExit(f"--steps must be in [1, {n_stream}] (the stream's length)")
    full = K_steps == n_stream
    variant = []
    if args.policy == "paper":
        variant.append("paper layer policy: layers 11-17 regulated, first frame kept whole in every layer")
    if stride != cfg.stride:
        variant.append(f"{stride}x{stride} query windows")
    if args.gamma is not None:
        variant.append(f"gamma {args.gamma}")
    if args.shared:
        variant.append("head-averaged selection")
    if args.staged:
        variant.append("frames staged in the arenas by a copy kernel (timed as staging_ms, inside the "
                       "wall clock), attention over the contiguous arena, admission by in-place compaction")
    if args.fused:
        variant.append("saliency in the attention epilogue (per 128-query block), admission from those rows")
    wkey = workload_key(cfg, n_stream, K_steps, variant)
    if args.trace_summary:
        summarize_trace(*args.trace_summary, wkey or cfg.name)
        return
    if args.pmc_summary:
        summarize_pmc(*args.pmc_summary, wkey or cfg.name, steps=K_steps, layers=cfg.n_layers)
        return
    if args.mfma_summary:
        summarize_mfma(*args.mfma_summary, wkey or cfg.name)
        return

    import torch
    from paper_2609_23286_amd import rv

    qs = (cfg.grid_h, cfg.grid_w, cfg.n_special, stride)
    n_q = len(range(0, cfg.grid_h, stride)) * len(range(0, cfg.grid_w, stride))
    anchor = args.policy == "paper"
    regulated = [l for l in range(L) if args.policy == "all" or 10 <= l <= 16]
    admit_fn = "rv_admit_layers_shared" if args.shared else "rv_admit_layers"
    if args.staged and args.shared:
        raise SystemExit("--staged supports head-specific selection only")
    if args.fused and (args.staged or args.shared or args.policy == "paper"):
        raise SystemExit("--fused runs the configuration's own policy with head-specific selection only")

    def mem_len(l, t):
        """Rows of layer l's memory when frame t of the stream is attended."""
        n = cfg.prefill
        if anchor and t > 0:
            n += N
        if l in regulated:
            n += max(0, t - (1 if anchor else 0)) * k
        return n

    # Frames: the whole stream in order from its initial memory, or a stratified sample
    # of it taken longest memory first, each layer's memory cut back (rv_mem_truncate,
    # host-side only) to the length the frame has in the stream, so the timed frames run
    # back to back.  The W warm-up frames repeat the first timed frame (below).
    if full:
        timed = list(range(n_stream))
    else:
        timed = sorted(stratified(n_stream, K_steps), reverse=True)
    frame_ids = sorted(set(timed))

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    rv.init()

    frame_bytes = L * 3 * N * H * d * 2
    free, total = torch.cuda.mem_get_info()
    log(f"{cfg.name}: L={L} H={H} N={N} k={k}; {'whole' if full else 'stratified'} "
        f"{K_steps} of {n_stream} frames; inputs {len(frame_ids) * frame_bytes / 1e9:.1f} GB, "
        f"device free {free / 1e9:.1f} of {total / 1e9:.1f} GB")
    if len(frame_ids) * frame_bytes > free - 16e9:
        raise SystemExit("not enough device memory to keep every timed frame's inputs resident "
                         "(time fewer --steps: they are a stratified sample of the stream)")

    if args.copy_calibration:
        x = torch.ones(COPY_CALIBRATION_BYTES // 4, dtype=torch.float32, device=dev)
        y = torch.empty_like(x)
        torch.neg(x, out=y)
        torch.cuda.synchronize()
        del x, y

    # ---- inputs: every frame resident in HBM --------------------------------------
    t0 = time.perf_counter()
    frames = {}
    for t in frame_ids:
        buf = torch.empty((L, 3, N, H, d), dtype=torch.int16, device=dev)
        rv.gpu_frame_qkv(cfg, t, buf)
        frames[t] = buf
    torch.cuda.synchronize()
    log(f"generated {len(frame_ids)} frames in {time.perf_counter() - t0:.1f} s")

    rows_max = [max(mem_len(l, t) for t in frame_ids) for l in range(L)]
    cap = max(rows_max) + (N if anchor else k) + 64 + (N if args.staged else 0)
    mems = [rv.Memory(H, reserve_tokens=cap, max_tokens=cap) for _ in range(L)]

    def fill_memories(rows_of):
        """Each layer's memory gets rows_of(l) rows: near-Gaussian N(0, sigma^2) rows drawn
        like the configuration's prefill (tags 4/5), standing in for prefilled and admitted
        tokens (attention and admission time do not depend on the values)."""
        for l, m in enumerate(mems):
            m.reset()
            n = rows_of(l)
            if n:
                pk = torch.empty((H, n, d), dtype=torch.int16, device=dev)
                pv = torch.empty_like(pk)
                rv.gpu_normal(cfg.seed, synth.PREFILL_FRAME, l, synth.TAG_MEMK, pk, cfg.sigma)
                rv.gpu_normal(cfg.seed, synth.PREFILL_FRAME, l, synth.TAG_MEMV, pv, cfg.sigma)
                m.write(pk, pv)
                del pk, pv
        torch.cuda.synchronize()

    rv.reserve_workspace(N, H, max(rows_max), L)
    out = torch.empty((L, N, H, d), dtype=torch.int16, device=dev)
    lse = torch.empty((L, H, N), dtype=torch.float32, device=dev)
    sal = torch.empty((L, H, N), dtype=torch.float32, device=dev)
    n_qb = -(-N // 128)
    tiles = torch.empty((L, H, n_qb, N), dtype=torch.float32, device=dev) if args.fused else None

    # Raw C calls with pre-marshalled arguments keep the host ahead of the GPU.
    import ctypes
    lib = rv.lib()
    vp = ctypes.c_void_p
    s_h = vp(stream.cuda_stream)
    q = rv.rv_qsub(*qs)
    qref = ctypes.byref(q)
    arr = vp * L
    out_p = [vp(out[l].data_ptr()) for l in range(L)]
    lse_p = [vp(lse[l].data_ptr()) for l in range(L)]
    sal_arr = arr(*[sal[l].data_ptr() for l in range(L)])
    lse_arr = arr(*[lse[l].data_ptr() for l in range(L)])
    mem_arr = arr(*[m.handle.value for m in mems])
    views = [m.view() for m in mems]  # capacity is reserved: arenas never move
    frame_ptrs = {}
    for t in frame_ids:
        fb = frames[t]
        qp = [fb[l, 0].data_ptr() for l in range(L)]
        kp = [fb[l, 1].data_ptr() for l in range(L)]
        vpp = [fb[l, 2].data_ptr() for l in range(L)]
        frame_ptrs[t] = (qp, kp, vpp, arr(*qp), arr(*kp), arr(*vpp))

    tiles_p = [vp(tiles[l].data_ptr()) for l in range(L)] if args.fused else None
    qsub_c = rv.rv_qsub(*qs)
    reg_arr = lambda ptrs: (vp * len(regulated))(*[ptrs[l] for l in regulated])
    reg_sal = reg_arr([sal[l].data_ptr() for l in range(L)])
    reg_lse = reg_arr([lse[l].data_ptr() for l in range(L)])
    reg_mem = reg_arr([m.handle.value for m in mems])
    reg_frames = {t: (reg_arr(f[0]), reg_arr(f[1]), reg_arr(f[2])) for t, f in frame_ptrs.items()}
    reg_tiles = reg_arr([tiles[l].data_ptr() for l in range(L)]) if args.fused else None
    admit = getattr(lib, admit_fn)

    def run_frame(t, ev=None):
        qp, kp, vpp, qa, ka, va = frame_ptrs[t]
        if not full:
            for l in range(L):
                st = lib.rv_mem_truncate(mems[l].handle, mem_len(l, t))
                if st:
                    raise rv.RVError(st, lib.rv_last_error().decode())
        # Timing events, two per frame (three with staging): the frame's start, which also
        # ends the previous frame's admission (every event costs the GPU a few
        # microseconds, so adjacent boundaries share one), and the end of its attention.
        if ev is not None:
            ev[0].record(stream)
        if args.staged:  # the producer's part: the frame's K/V into each arena's tail
            st = lib.rv_mem_stage_frames(L, mem_arr, ka, va, N, s_h)
            if st:
                raise rv.RVError(st, lib.rv_last_error().decode())
            if ev is not None:
                ev[1].record(stream)
        for l in range(L):
            if args.staged:
                st = lib.rv_attend_staged(vp(qp[l]), N, mems[l].handle, None, out_p[l], lse_p[l], None, s_h)
            elif args.fused and l in regulated:
                mk, mv, hs = views[l]
                st = lib.rv_attend_frame_fused(vp(qp[l]), vp(kp[l]), vp(vpp[l]), N, vp(mk), vp(mv),
                                               lib.rv_mem_len(mems[l].handle), hs, H, d, ctypes.byref(qsub_c),
                                               out_p[l], lse_p[l], tiles_p[l], s_h)
            else:
                mk, mv, hs = views[l]
                st = lib.rv_attend_frame(vp(qp[l]), vp(kp[l]), vp(vpp[l]), N, vp(mk), vp(mv),
                                         lib.rv_mem_len(mems[l].handle), hs, H, d, None, out_p[l], lse_p[l],
                                         None, s_h)
            if st:
                raise rv.RVError(st, lib.rv_last_error().decode())
        if ev is not None:
            ev[2].record(stream)
        if anchor and t == 0:  # the global anchor: the first frame whole, in every layer (Eq. 4)
            if args.staged:
                st = lib.rv_admit_staged_layers(L, qa, lse_arr, N, qref, N, mem_arr, t, sal_arr, None, s_h)
            else:
                st = admit(L, qa, ka, va, lse_arr, N, qref, N, mem_arr, t, sal_arr, None, s_h)
        elif regulated and k > 0:
            rq, rk, rvv = reg_frames[t]
            if args.staged:
                st = lib.rv_admit_staged_layers(len(regulated), rq, reg_lse, N, qref, k, reg_mem, t, reg_sal,
                                                None, s_h)
            elif args.fused:
                st = lib.rv_admit_layers_tiled(len(regulated), reg_tiles, N, k, rk, rvv, reg_mem, t, reg_sal, None,
                                               s_h)
            else:
                st = admit(len(regulated), rq, rk, rvv, reg_lse, N, qref, k, reg_mem, t, reg_sal, None, s_h)
        else:
            st = 0
        if st:
            raise rv.RVError(st, lib.rv_last_error().decode())

    # ---- warm-up, then the timed frames --------------------------------------------
    # Warm-up: runs of the first timed frame on the memories it starts from, each
    # followed by cutting every memory back to that start (host-side), so that the timed
    # frames follow warm-up work on the same data: W of them, and (W > 0) as many more as
    # fill WARMUP_MIN_S of wall time.  The device reaches its sustained speed only after
    # some tens of milliseconds under load: after 5 warm-up frames (≈ 6 ms) a 20-frame
    # sample ran 3 % slower than the same frames inside the whole stream, after 50 or
    # more as fast.  (Warming up on other frames and then refilling the memories, as
    # before, also left the device idle just before timing.)
    initial = (lambda l: mem_len(l, 0)) if full else (lambda l: rows_max[l])
    fill_memories(initial)
    start_len = [m.len for m in mems]
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in timed]
    end_event = torch.cuda.Event(enable_timing=True)
    warm_runs, t_warm = 0, time.perf_counter()
    while warm_runs < W or (W > 0 and time.perf_counter() - t_warm < WARMUP_MIN_S):
        run_frame(timed[0])
        for l, m in enumerate(mems):
            m.truncate(start_len[l])
        warm_runs += 1
        if warm_runs % 10 == 0:  # (so that the wall clock follows the device)
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i, t in enumerate(timed):
        run_frame(t, events[i])
        if (i + 1) % 250 == 0:
            log(f"enqueued {i + 1} frames")
    end_event.record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    rv.device_status()
    if full:
        assert all(m.len == mem_len(l, n_stream) for l, m in enumerate(mems))

    # frame i: attention from its start (after the staging copies, when staged) to its
    # attention end; admission from there to the next frame's start (the last: end_event)
    attn_start = (lambda i: events[i][1]) if args.staged else (lambda i: events[i][0])
    frame_end = lambda i: events[i + 1][0] if i + 1 < len(timed) else end_event
    attn_ms_i = lambda i: attn_start(i).elapsed_time(events[i][2])
    admit_ms_i = lambda i: events[i][2].elapsed_time(frame_end(i))
    for i in sorted({0, len(timed) // 2, len(timed) - 1}):
        t = timed[i]
        log(f"frame {t}: attention {attn_ms_i(i) * 1e3 / L:.1f} us/launch "
            f"(context {mem_len(regulated[0] if regulated else 0, t) + N}), "
            f"admission {admit_ms_i(i) * 1e3:.1f} us")
    attn_ms = sum(attn_ms_i(i) for i in range(len(timed)))
    admit_ms = sum(admit_ms_i(i) for i in range(len(timed)))
    stage_ms = sum(events[i][0].elapsed_time(events[i][1]) for i in range(len(timed))) if args.staged else None
    n_timed = len(timed)
    flops = sum(attention_flops(N, H, d, mem_len(l, t) + N) for t in timed for l in range(L))
    n_attn = n_timed * L
    attn_avg_s = attn_ms / 1e3 / n_attn
    achieved_tf = flops / n_attn / attn_avg_s / 1e12
    bytes_admit = sum(admit_bytes(N, H, d, n_q, N) * L if (anchor and t == 0)
                      else admit_bytes(N, H, d, n_q, k) * len(regulated) for t in timed)
    admit_gbs = bytes_admit / (admit_ms / 1e3) / 1e9
    log(f"timed {n_timed} frames in {elapsed:.3f} s: attention {attn_ms:.1f} ms "
        f"({attn_avg_s * 1e6:.1f} us/launch, {achieved_tf:.1f} TFLOP/s), admission {admit_ms:.1f} ms "
        f"({admit_ms / n_timed * 1e3:.1f} us/frame, {admit_gbs:.0f} GB/s)")

    mean_ctx = sum(mem_len(l, t) + N for t in timed for l in range(L)) / n_attn
    if full:
        sampling = f"the whole {n_stream}-frame stream in order from "
        sampling += f"{cfg.prefill} prefilled memory rows" if cfg.prefill else "empty memory"
    else:
        sampling = (f"{n_timed} of its {n_stream} frames, stratified (frame t_i = floor((i + 1/2) {n_stream} / "
                    f"{n_timed})), each at the memory length it has in the stream ({cfg.prefill} prefilled + "
                    f"{k} per frame), timed back to back longest first")
    workload = (f"{cfg.name}: {n_stream}-frame stream, {L} layers x {H} heads x {d}, {N} tokens/frame "
                f"({cfg.grid_h}x{cfg.grid_w} patches + {cfg.n_special} special), budget {k}/head/frame, "
                f"{stride}x{stride} query sampling; {sampling}; mean context {mean_ctx:.0f}"
                + "".join("; " + v for v in variant))
    result = {
        "metric": f"frames/sec (attend+saliency+admit, {L} layers) at {n_stream}-frame stream; % MFMA/HBM peak",
        "value": n_timed / elapsed,
        "unit": "frames/s",
        "n_gpus": 1,
        "steps": n_timed,
        "warmup": W, "warmup_frames_run": warm_runs,
        "ms_per_step": elapsed / n_timed * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded Philox streams of ViT-L token shape, 1% planted salient keys)",
        "config": {"workload": workload, "layers": L, "heads": H, "head_dim": d, "tokens_per_frame": N,
                   "budget": k, "stream_frames": n_stream, "timed_frames": timed if not full else "all",
                   "mean_context": mean_ctx, "sampled_queries": n_q, "query_window": stride,
                   "regulated_layers": len(regulated), "anchor": anchor,
                   "selection": "head-averaged" if args.shared else "head-specific",
                   "staged_frames": bool(args.staged), "prefill_rows": cfg.prefill},
        "roofline": {"kernel": "attn_fwd_kernel (+ attn_merge_kernel on split plans)", "bound": "mfma",
                     "achieved": achieved_tf,
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": achieved_tf / PEAK_BF16_TFLOPS,
                     "traffic": attention_traffic(wkey) if wkey else None,
                     "avg_launch_us": attn_avg_s * 1e6,
                     "algorithmic_flops_per_launch": flops / n_attn},
        "phases": {"attention_ms": attn_ms, "admission_ms": admit_ms, "staging_ms": stage_ms,
                   "admission_roofline": {"kernel": "sal_kernel + select_kernel", "bound": "hbm",
                                          "achieved": admit_gbs,
                                          "peak": PEAK_HBM_GBS, "unit": "GB/s",
                                          "frac": admit_gbs / PEAK_HBM_GBS,
                                          "traffic": admission_traffic(wkey) if wkey else None,
                                          "algorithmic_bytes_per_launch": bytes_admit / n_timed}},
    }
    for m in mems:
        m.close()
    del frames
    if not args.no_cpu_baseline:
        log("timing the oracle on a host sample ...")
        ns = max(1, args.cpu_samples)
        samples = [(i % L, t) for i, t in enumerate(stratified(n_stream, ns))]
        samples = [(regulated[i % len(regulated)] if regulated else l, t) for i, (l, t) in enumerate(samples)]
        result["cpu_baseline"] = cpu_baseline(cfg, samples, k, qs, mem_len, mean_ctx)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
