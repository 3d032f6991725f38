"""Summary of the rocprofv3 runs behind bench.py's roofline figures.

Three runs of ``bench.py`` on the GPU (see ``commands``): a kernel trace with
statistics, then one counter pass with FETCH_SIZE and one with WRITE_SIZE
(each counter in KiB per dispatch).  The counter passes start with
``--copy-mib 1024``: one elementwise kernel that reads 1 GiB and writes 1 GiB,
whose counter values scale every other dispatch to bytes.  This module turns
the CSV output of those runs into ``profiles/expert_gemm_<workload>_traffic.md``,
including the machine-readable record that ``bench.py`` reads back while the
kernel sources still hash to the recorded value.

    python -m paper_2604_15821_amd.counters <workload> <directory with the run outputs>
    python -m paper_2604_15821_amd.counters --trace <workload> <steps> <directory>
    python -m paper_2604_15821_amd.counters --mfma <workload> <directory>

The second form summarises a kernel-trace run alone into profiles/kernels_<workload>.md,
the third a counter pass of executed matrix work into profiles/mfma_<workload>.md.
"""
from __future__ import annotations

import collections
import csv
import json
import os
import re
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def commands(workload: str, out: str = "$OUT") -> list[str]:
    """The three rocprofv3 command lines (run from /tmp with TMPDIR=/tmp, repo at $R, outputs under $OUT)."""
    bench = "python3 $R/bench.py"
    return [
        f"rocprofv3 --kernel-trace --stats --output-format csv -d {out}/tr_k_{workload} -o run -- "
        f"{bench} --workload {workload} --steps 10 --warmup 2 --no-cpu-baseline",
        f"rocprofv3 --pmc FETCH_SIZE --output-format csv -d {out}/tr_f_{workload} -o run -- "
        f"{bench} --workload {workload} --steps 2 --warmup 0 --no-cpu-baseline --copy-mib 1024",
        f"rocprofv3 --pmc WRITE_SIZE --output-format csv -d {out}/tr_w_{workload} -o run -- "
        f"{bench} --workload {workload} --steps 2 --warmup 0 --no-cpu-baseline --copy-mib 1024",
    ]


def family(kernel_name: str) -> str:
    """Kernel family of a dispatch, as bench.py's profiler groups launches."""
    n = kernel_name
    if "gemm_rows_kernel" in n:
        return "dense_gemm" if "EpiDense" in n else "expert_gemm"
    if "wgrad_skinny" in n:
        return "dense_gemm"
    if "gemm_wgrad_kernel" in n or "wgrad_reduce" in n:
        return "wgrad"
    if re.search(r"(dispatch_x|edge_p[234]|tri_(dispatch|p[234]|combine|gather|combine_p3))_kernel", n):
        return "edge"
    if re.search(r"(combine_fwd|gather_atom|scatter_rev|combine_p3)_kernel", n):
        return "atom"
    if re.search(r"attn_(fwd|bwd|tan|rev)(_mfma|_tiled)?_kernel", n):
        return "attention"
    if "elementwise_kernel" in n or "vectorized" in n:
        return "copy"
    return "other"


# Sources that define the expert GEMM kernels, their operand loaders and epilogues,
# and their launch configuration: a counter record of that family is valid only for these.
EXPERT_GEMM_SOURCES = ("common.h", "gemm.h", "internal.h")
CSRC = os.path.join(ROOT, "paper_2604_15821_amd", "csrc")
PROFILES = os.path.join(ROOT, "profiles")


def kernel_sources_sha256() -> str:
    """Hash of the expert GEMM kernels' sources: measured counters are valid only for these."""
    import hashlib
    h = hashlib.sha256()
    for name in EXPERT_GEMM_SOURCES:
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()


def measured_traffic(workload: str, family: str = "expert_gemm"):
    """HBM bytes per launch of a kernel family from the committed rocprofv3 counter summary
    (FETCH_SIZE and WRITE_SIZE, each scaled by a plain copy kernel of known size), or None
    when no summary matches this workload or the kernel sources changed since it was taken."""
    path = os.path.join(PROFILES, f"{family}_{workload}_traffic.md")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        for line in f:
            if line.startswith("traffic-json:"):
                rec = json.loads(line.split(":", 1)[1])
                if rec.get("sources_sha256") != kernel_sources_sha256():
                    return None
                return rec["fetch_bytes_per_launch"] + rec["write_bytes_per_launch"]
    return None


def _counter(path: str, name: str):
    per, names = collections.defaultdict(float), {}
    with open(path) as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] != name:
                continue
            k = int(r["Dispatch_Id"])
            per[k] += float(r["Counter_Value"])
            names[k] = r["Kernel_Name"]
    return per, names


def summarize(workload: str, runs: str) -> str:
    """Markdown summary of the three runs found under `runs`."""
    fetch, fnames = _counter(f"{runs}/tr_f_{workload}/run_counter_collection.csv", "FETCH_SIZE")
    write, wnames = _counter(f"{runs}/tr_w_{workload}/run_counter_collection.csv", "WRITE_SIZE")
    copy_f = [fetch[k] for k in fetch if family(fnames[k]) == "copy" and fetch[k] > 5e5]
    copy_w = [write[k] for k in write if family(wnames[k]) == "copy" and write[k] > 5e5]
    kf, kw = 1048576.0 / copy_f[0], 1048576.0 / copy_w[0]
    agg = collections.defaultdict(lambda: [0, 0.0, 0.0])
    for k in fetch:
        a = agg[family(fnames[k])]
        a[0] += 1
        a[1] += fetch[k] * 1024 * kf
    for k in write:
        agg[family(wnames[k])][2] += write[k] * 1024 * kw
    dur = collections.defaultdict(list)
    with open(f"{runs}/tr_k_{workload}/run_kernel_trace.csv") as f:
        for r in csv.DictReader(f):
            dur[family(r["Kernel_Name"])].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    with open(f"{runs}/tr_k_{workload}/run_kernel_stats.csv") as f:
        stats = list(csv.DictReader(f))
    bench_line = None
    log = f"{runs}/tr_k_{workload}.log"
    if os.path.exists(log):
        lines = [x for x in open(log) if x.startswith("{")]
        bench_line = json.loads(lines[-1]) if lines else None
    ex = agg["expert_gemm"]
    rec = {"workload": workload, "family": "expert_gemm", "sources_sha256": kernel_sources_sha256(),
           "launches_counted": ex[0], "fetch_bytes_per_launch": ex[1] / ex[0], "write_bytes_per_launch": ex[2] / ex[0],
           "fetch_scale": kf, "write_scale": kw}
    L = [f"# Kernel time and HBM traffic, training step, workload `{workload}`", "",
         "Commands (run from /tmp on an MI355X with `TMPDIR=/tmp`, repo at `$R`, outputs under `$OUT`), three separate runs:", "",
         "```", *commands(workload), "```", "",
         f"Summarised by `python -m paper_2604_15821_amd.counters {workload} $OUT`.", "",
         "FETCH_SIZE and WRITE_SIZE are KiB per dispatch. Each is scaled by what the same counter reads for the",
         "calibration kernel of the `--copy-mib 1024` runs: one elementwise kernel that reads 1 GiB and writes 1 GiB.",
         f"The scale factors are fetch x{kf:.3f} and write x{kw:.3f}. Traffic is averaged over every dispatch of",
         "the counter runs (their breakdown and timed steps).", "",
         "| family | launches | avg us (kernel trace) | HBM read MB/launch | HBM write MB/launch |",
         "|---|---:|---:|---:|---:|"]
    for fam in ["expert_gemm", "wgrad", "dense_gemm", "edge", "atom", "other"]:
        if agg[fam][0]:
            d, a = dur.get(fam, [0.0]), agg[fam]
            L.append(f"| {fam} | {a[0]} | {sum(d) / max(len(d), 1):.1f} | {a[1] / a[0] / 1e6:.1f} | "
                     f"{a[2] / a[0] / 1e6:.1f} |")
    L += ["", "The kernel-trace run uses bench.py's default two streams: in the double and final backward the "
          "expert weight gradients (wgrad) run beside the edge, atom and small dense kernels, whose averages "
          "above are therefore longer than alone; the expert products never overlap another product.",
          "", "Kernel statistics of the kernel-trace run (rocprofv3 --stats, all dispatches including warm-up):", "",
          "| kernel | calls | avg us | total ms | % |", "|---|---:|---:|---:|---:|"]
    for r in stats[:30]:
        n = re.sub(r"\(.*", "", r["Name"].replace("janus::", ""))
        L.append(f"| `{n}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                 f"{float(r['TotalDurationNs']) / 1e6:.2f} | {float(r['Percentage']):.2f} |")
    if bench_line:
        roof = {k: v for k, v in bench_line["roofline"].items() if k != "traffic"}
        L += ["", "bench.py line of the kernel-trace run (its own HIP-event timing on the library's stream):", "",
              "```", json.dumps({k: bench_line[k] for k in ("value", "unit", "ms_per_step")}), json.dumps(roof), "```",
              "", f"expert_gemm average launch: bench HIP events in the timed region {roof['avg_launch_ms'] * 1e3:.1f} us; "
              f"kernel trace {sum(dur['expert_gemm']) / len(dur['expert_gemm']):.1f} us (all dispatches of the run)."]
    algorithmic = algorithmic_bytes(bench_line)
    if algorithmic:
        ar, aw = algorithmic
        L += ["", "Algorithmic bytes per expert-GEMM launch (average over the 8 products of a block):",
              f"read {ar / 1e6:.0f} MB, write {aw / 1e6:.0f} MB; measured read / algorithmic = "
              f"{rec['fetch_bytes_per_launch'] / ar:.2f}, write = {rec['write_bytes_per_launch'] / aw:.2f}."]
    L += ["", "Machine-readable record read by bench.py (valid while the sources of the expert GEMM kernels, "
          "`csrc/common.h`, `csrc/gemm.h` and `csrc/internal.h`, hash to `sources_sha256`):", "",
          "traffic-json: " + json.dumps(rec)]
    return "\n".join(L) + "\n"


def algorithmic_bytes(bench_line: dict):
    """Average algorithmic HBM bytes (read, write) per expert-GEMM launch of a block of the
    edge MoE, from the workload of a bench.py line: the 8 products G1-G6, G9, G10 over
    M = k Ne slot rows with [M, h] and [M, d] fp32 tensors (operands, stored
    pre-activations and adjoints read once, outputs written once; M per launch, that is
    per workspace chunk).  None with triplets (their products join the family)."""
    if not bench_line or bench_line.get("triplets", 0):
        return None
    c = bench_line["config"]
    # slot rows of one launch: a batch split over workspace chunks runs every product once
    # per chunk, so M comes from the roofline's per-launch work (2 M d h) when it is there
    roof = bench_line.get("roofline") or {}
    if roof.get("kernel") == "expert_gemm" and roof.get("flops_per_launch"):
        M = roof["flops_per_launch"] / (2.0 * c["d"] * c["d_hidden"])
    else:
        M = c["top_k"] * c["edges"]
    H, D = 4.0 * M * c["d_hidden"], 4.0 * M * c["d"]
    reads = D + H + (D + H) + H + (D + 2 * H) + H + (D + 2 * H) + H      # G1 G2 G3 G4 G5 G6 G9 G10
    writes = H + D + 2 * H + D + 2 * H + D + H + D
    return reads / 8, writes / 8


def trace_command(workload: str, steps: int, out: str = "$OUT") -> str:
    """The rocprofv3 kernel-trace command of one workload (run from /tmp with TMPDIR=/tmp);
    a name ending in _serial is that workload run on one stream (bench.py --serial)."""
    wl, serial = (workload[:-7], " --serial") if workload.endswith("_serial") else (workload, "")
    return (f"rocprofv3 --kernel-trace --stats --output-format csv -d {out}/trace_{workload} -o run -- "
            f"python3 $R/bench.py --workload {wl} --steps {steps} --warmup 1 --breakdown-steps 1 "
            f"--no-cpu-baseline{serial}")


def trace_summary(workload: str, runs: str, steps: int) -> str:
    """Markdown summary of one kernel-trace run: per-family and per-kernel time."""
    with open(f"{runs}/trace_{workload}/run_kernel_stats.csv") as f:
        stats = list(csv.DictReader(f))
    fam = collections.defaultdict(lambda: [0, 0.0])
    for r in stats:
        a = fam[family(r["Name"])]
        a[0] += int(r["Calls"])
        a[1] += float(r["TotalDurationNs"]) / 1e6
    bench_line = None
    log = f"{runs}/trace_{workload}.log"
    if os.path.exists(log):
        lines = [x for x in open(log) if x.startswith("{")]
        bench_line = json.loads(lines[-1]) if lines else None
    L = [f"# Kernel time, training step, workload `{workload}`", "",
         "Command (run from /tmp on an MI355X with `TMPDIR=/tmp`, repo at `$R`, outputs under `$OUT`):", "",
         "```", trace_command(workload, steps), "```", "",
         f"Summarised by `python -m paper_2604_15821_amd.counters --trace {workload} {steps} $OUT`.",
         f"All dispatches of the run ({steps} timed + 1 warm-up + 1 breakdown step). Families follow the",
         "kernel names: products that use the expert GEMM kernels (the attention q|k|v and Wo products",
         "too) count as expert_gemm here; bench.py's own profiler files those under dense_gemm.",
         ("One stream: every kernel ran alone." if workload.endswith("_serial") else
          "Two streams (bench.py's default): in the double and final backward the expert weight gradients "
          "run beside the edge, atom and small dense kernels, whose durations here are therefore longer "
          "than alone; the expert products never overlap another product."), "",
         "| family | dispatches | total ms | % |", "|---|---:|---:|---:|"]
    tot = sum(v[1] for v in fam.values()) or 1.0
    for k, v in sorted(fam.items(), key=lambda kv: -kv[1][1]):
        L.append(f"| {k} | {v[0]} | {v[1]:.2f} | {100 * v[1] / tot:.1f} |")
    L += ["", "| kernel | calls | avg us | total ms | % |", "|---|---:|---:|---:|---:|"]
    for r in stats[:25]:
        n = re.sub(r"\(.*", "", r["Name"].replace("janus::", ""))
        L.append(f"| `{n}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                 f"{float(r['TotalDurationNs']) / 1e6:.2f} | {float(r['Percentage']):.2f} |")
    if bench_line:
        L += ["", "bench.py line of the same run (its own HIP-event timing):", "", "```",
              json.dumps({k: bench_line[k] for k in ("value", "unit", "ms_per_step")}), "```"]
    return "\n".join(L) + "\n"


# Executed fp32 matrix work and matrix-pipe busy cycles per dispatch.  rocprofv3's own
# derived metrics define MfmaFlopsF32 = 512 SQ_INSTS_VALU_MFMA_MOPS_F32 and MfmaUtil =
# sum(SQ_VALU_MFMA_BUSY_CYCLES) / (max over XCDs of GRBM_GUI_ACTIVE x 1024 SIMDs); the CSV
# gives GRBM_GUI_ACTIVE summed over the 8 XCDs, whose max is taken as that sum / 8.
MFMA_COUNTERS = ("SQ_INSTS_VALU_MFMA_MOPS_F32", "SQ_VALU_MFMA_BUSY_CYCLES", "GRBM_GUI_ACTIVE")
N_XCD, N_SIMD = 8, 1024
MFMA_RUN_STEPS = 2   # the counter pass below runs one breakdown step and one timed step


def mfma_command(workload: str, out: str = "$OUT") -> str:
    """The rocprofv3 counter pass of one workload (run from /tmp with TMPDIR=/tmp)."""
    return (f"rocprofv3 --pmc {' '.join(MFMA_COUNTERS)} --output-format csv -d {out}/tr_m_{workload} -o run -- "
            f"python3 $R/bench.py --workload {workload} --steps 1 --warmup 0 --breakdown-steps 1 --no-cpu-baseline")


# bench.py's family names for the counter families whose work is all on the matrix cores
# (bench.py's dense family also counts the skinny bias-weight gradients, which run on the
# vector ALU, so its executed matrix work is not comparable)
_BENCH_FAMILY = {"expert_gemm": "expert_gemm", "wgrad": "expert_wgrad"}


def mfma_summary(workload: str, runs: str) -> str:
    """Markdown summary of one counter pass: executed fp32 MFMA work against the algorithmic
    work bench.py counts, matrix-pipe busy fraction and clock, per kernel and per family."""
    per = collections.defaultdict(lambda: collections.defaultdict(float))
    names, dur = {}, {}
    with open(f"{runs}/tr_m_{workload}/run_counter_collection.csv") as f:
        for r in csv.DictReader(f):
            k = int(r["Dispatch_Id"])
            per[k][r["Counter_Name"]] += float(r["Counter_Value"])
            names[k] = r["Kernel_Name"]
            dur[k] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9
    bench_line = None
    log = f"{runs}/tr_m_{workload}.log"
    if os.path.exists(log):
        lines = [x for x in open(log) if x.startswith("{")]
        bench_line = json.loads(lines[-1]) if lines else None
    kern = collections.defaultdict(lambda: [0, 0.0, 0.0, 0.0, 0.0])   # dispatches, s, flops, busy, gui/8
    fam = collections.defaultdict(lambda: [0, 0.0])                   # dispatches, executed flops
    for k, c in per.items():
        n = re.sub(r"\(.*", "", names[k].replace("janus::", ""))
        flops = 512.0 * c["SQ_INSTS_VALU_MFMA_MOPS_F32"]
        a = kern[n]
        a[0] += 1
        a[1] += dur[k]
        a[2] += flops
        a[3] += c["SQ_VALU_MFMA_BUSY_CYCLES"]
        a[4] += c["GRBM_GUI_ACTIVE"] / N_XCD
        f = fam[family(names[k])]
        f[0] += 1
        f[1] += flops
    L = [f"# Executed fp32 matrix work, training step, workload `{workload}`", "",
         "Command (run from /tmp on an MI355X with `TMPDIR=/tmp`, repo at `$R`, outputs under `$OUT`):", "",
         "```", mfma_command(workload), "```", "",
         f"Summarised by `python -m paper_2604_15821_amd.counters --mfma {workload} $OUT`. Executed work is "
         "512 x SQ_INSTS_VALU_MFMA_MOPS_F32 (rocprofv3's MfmaFlopsF32); the matrix-pipe busy fraction is "
         "SQ_VALU_MFMA_BUSY_CYCLES over (GRBM_GUI_ACTIVE / 8) x 1024 SIMDs (its MfmaUtil; the CSV sums "
         "GRBM_GUI_ACTIVE over the 8 XCDs); the clock is GRBM_GUI_ACTIVE / 8 over the dispatch's duration. "
         "Dispatches run one at a time under the counter pass, so durations are those of each kernel alone.", ""]
    if bench_line:
        L += ["Per family, per training step (the algorithmic work is what bench.py counts for the same run: "
              "2 x rows x K x N per product, no padding):", "",
              "| family | dispatches per step | executed TFLOP per step | algorithmic TFLOP per step | executed / algorithmic |",
              "|---|---:|---:|---:|---:|"]
        fams = _BENCH_FAMILY
        if bench_line["config"].get("attention_heads"):
            # the q|k|v and Wo products run on the expert kernels but count as dense in bench.py
            fams = {"attention": "attention"}
        for cf, bf in fams.items():
            kb = bench_line.get("kernels", {}).get(bf)
            if not kb or not fam[cf][0]:
                continue
            steps = MFMA_RUN_STEPS
            alg = kb.get("flops_per_step", kb["tflops"] * kb["ms_per_step"] * 1e9) * 1e-12
            ex = fam[cf][1] / steps / 1e12
            L.append(f"| {cf} | {fam[cf][0] / steps:.0f} | {ex:.3f} | {alg:.3f} | {ex / alg:.4f} |")
        L.append("")
    L += ["| kernel | dispatches | avg us | executed GFLOP per dispatch | TFLOP/s | MFMA busy | clock GHz |",
          "|---|---:|---:|---:|---:|---:|---:|"]
    for n, a in sorted(kern.items(), key=lambda kv: -kv[1][1]):
        if a[2] <= 0:
            continue
        L.append(f"| `{n}` | {a[0]} | {a[1] / a[0] * 1e6:.1f} | {a[2] / a[0] / 1e9:.2f} | {a[2] / a[1] / 1e12:.1f} | "
                 f"{a[3] / (a[4] * N_SIMD):.3f} | {a[4] / a[1] / 1e9:.2f} |")
    return "\n".join(L) + "\n"


if __name__ == "__main__":
    if len(sys.argv) > 1 and sys.argv[1] == "--mfma":
        wl, runs = sys.argv[2], sys.argv[3]
        out = os.path.join(ROOT, "profiles", f"mfma_{wl}.md")
        with open(out, "w") as f:
            f.write(mfma_summary(wl, runs))
        print(out)
        sys.exit(0)
    if len(sys.argv) > 1 and sys.argv[1] == "--trace":
        wl, steps = sys.argv[2], int(sys.argv[3])
        runs = sys.argv[4]
        out = os.path.join(ROOT, "profiles", f"kernels_{wl}.md")
        with open(out, "w") as f:
            f.write(trace_summary(wl, runs, steps))
        print(out)
        sys.exit(0)
    wl = sys.argv[1]
    runs = sys.argv[2]
    text = summarize(wl, runs)
    out = os.path.join(ROOT, "profiles", f"expert_gemm_{wl}_traffic.md")
    with open(out, "w") as f:
        f.write(text)
    print(out)
