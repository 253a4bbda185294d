#!/usr/bin/env python3
"""Benchmark of the subgraph GCN training step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload yelp10k]

A step is one gcn_train_step: forward through every layer (pair sums of the
redundancy-reduced graph, aggregation, both weight transforms with fused
ReLU / concatenation), classifier, loss, backward (masked input gradients,
the transposed aggregation, weight gradients) and the gradient-descent
update of every weight, on one seeded synthetic subgraph already resident in
device memory. Default workload: the largest single-subgraph one, a
10,000-vertex Chung-Lu subgraph (power-law exponent 2.5, mean degree 20),
3 layers, f_in 300, 512 per branch, 100-way sigmoid BCE (the Yelp-like
widths of Table 2), fp32, aggregation on the graph reduced by 5 rounds of
Algorithms 1-3 (threshold 2, at most n/2 pair sums).

Prints ONE JSON line: steps/s (value), the dominant kernel's roofline
position measured with HIP events on the launch stream, the aggregation's
position against HBM (compulsory bytes, and the counter-measured bytes when
recorded for the current sources) and against a read-only streaming probe,
and the CPU oracle's throughput on a bounded sample of the same workload.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "subgraph GCN fwd+bwd steps/s; SpMM GB/s and GEMM TFLOPS as % of MI355X peak"
PEAK_FP32_MFMA_TFLOPS = 157.3    # MI355X dense fp32 matrix
PEAK_BF16_MFMA_TFLOPS = 2500.0   # MI355X dense bf16 matrix
PEAK_HBM_GBS = 8000.0            # MI355X HBM3E


def parse():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="yelp10k")
    ap.add_argument("--profile-steps", type=int, default=10)
    ap.add_argument("--theta", type=int, default=None,
                    help="reduction threshold (pairs held by more lists than this are summed "
                         "ahead); default: the workload's")
    ap.add_argument("--seg-len", type=int, default=0,
                    help="list segment length of the device work list (0: library default)")
    ap.add_argument("--precision", choices=("fp32", "bf16"), default="fp32",
                    help="dense products in fp32 or with bf16 operands (fp32 accumulation)")
    ap.add_argument("--graph", action="store_true",
                    help="replay the step from a captured HIP graph")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="CPU oracle sample budget (seconds of work)")
    ap.add_argument("--workers", type=int, default=0,
                    help="host preparation threads of the stream workload (0: min(16, cores))")
    ap.add_argument("--stream-len", type=int, default=64)
    ap.add_argument("--device-workers", type=int, default=6,
                    help="stream workload: workers of the pipeline that reduces on the GPU")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="also run one plain device copy of this size (HBM counter "
                         "calibration under rocprofv3 --pmc)")
    ap.add_argument("--order", choices=("paper", "narrow"), default="paper",
                    help="paper: aggregate H then transform (Eq. 1); narrow: transform "
                         "first where the input is wider than h")
    ap.add_argument("--no-narrow", action="store_true",
                    help="skip the extra timing of the narrow-side order")
    ap.add_argument("--no-adam", action="store_true",
                    help="skip the extra timing of the step with the Adam update")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the extra figures (bf16 step of the workload; ppi8k fp32 "
                         "step, reduced and direct)")
    ap.add_argument("--no-direct", action="store_true",
                    help="skip the direct-aggregation comparison run (counter runs)")
    ap.add_argument("--infer", action="store_true",
                    help="time gcn_infer (forward pass into logits) on a whole synthetic "
                         "graph instead of the training step")
    ap.add_argument("--infer-n", type=int, default=60000,
                    help="with --infer: vertices of the whole graph")
    ap.add_argument("--trace-summary", metavar="KERNEL_STATS_CSV",
                    help="no GPU: turn a rocprofv3 --kernel-trace --stats kernel_stats.csv "
                         "of this script into the per-class table under profiles/")
    ap.add_argument("--traced-args", default="--no-cpu-baseline --no-direct --no-narrow --no-adam --no-extra",
                    help="with --trace-summary: the arguments the traced run was given")
    ap.add_argument("--bench-line", help="with --trace-summary: the JSON line the traced run "
                                         "printed (event timings shown beside the trace)")
    ap.add_argument("--l2-summary", metavar="COUNTER_CSV",
                    help="no GPU: turn a rocprofv3 TCC_HIT_sum / TCC_MISS_sum counter file of "
                         "this script into the L2 hit-rate table under profiles/")
    ap.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="no GPU: turn two rocprofv3 --pmc counter files (FETCH_SIZE, "
                         "WRITE_SIZE) of a --calib-copy-mib run into the per-launch "
                         "HBM traffic table under profiles/")
    ap.add_argument("--mfma-summary", metavar="COUNTER_CSV",
                    help="no GPU: turn one rocprofv3 --pmc pass (MfmaUtil and MFMA, LDS "
                         "and wait counters) into the per-class table under profiles/")
    return ap.parse_args()


# ---------------------------------------------------------------- HBM traffic
#
# Per-launch HBM bytes come from two rocprofv3 --pmc runs of this script
# (FETCH_SIZE, then WRITE_SIZE, KiB per dispatch), each scaled by what the
# same counter reads for one plain device copy of known size in the same run.
# The table lives in profiles/<workload>_hbm_traffic.md together with a hash
# of the sources each kernel class is built and launched from; when the
# sources change the stored figure no longer describes the kernel and the
# roofline reports traffic as null.

CSRC = os.path.join(ROOT, "paper_2001_02498_amd", "csrc")
_CLASS_SOURCES = {
    "gemm": ["gemm.hip", "kernels.h", "api.hip"],
    "agg": ["agg.hip", "kernels.h", "api.hip", "host_graph.cpp"],
    "loss": ["loss.hip", "kernels.h", "api.hip"],
    "sgd": ["gemm.hip", "kernels.h", "api.hip"],
    "gather": ["gather.hip"],
}
_SAMPLED_NAMES = ("yelpfull",)
_ROLE_CLASS = ["gemm_fwd", "gemm_cls", "gemm_dx", "gemm_cls_dx", "gemm_dw", "gemm_cls_dw",
               "gemm_fwd_in", "gemm_dw_in"]


def _family(cls):
    if cls.startswith("gemm") or cls == "splitk_finish":
        return "gemm"
    if cls in ("pair_sums", "list_sums"):
        return "agg"
    if cls.startswith("loss"):
        return "loss"
    if cls == "gather_rows":
        return "gather"
    return "sgd"


def source_hash(cls):
    import hashlib
    h = hashlib.sha256()
    for f in _CLASS_SOURCES[_family(cls)] + ["../synth.py"]:
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def kernel_class(name):
    """Timing class of a demangled kernel name (the classes gcn_profile_read
    reports), or None for kernels that are not the library's."""
    import re
    for key, suffix in (("gemm_kernel<", ""), ("gemm_bf16_kernel<", "_bf16"),
                        ("gemm_h16_kernel<", "_bf16"), ("gemm_h16s_kernel<", "_bf16")):
        if key in name:
            m = re.search(r"\(gcn::GemmRole\)(\d+)", name)
            return _ROLE_CLASS[int(m.group(1))] + suffix if m else None
    for key, cls in (("pair_sums_kernel<", "pair_sums"), ("list_sums_kernel<", "list_sums"),
                     ("sgd_reduce_kernel", "sgd_reduce"),
                     ("splitk_finish_kernel", "splitk_finish"), ("loss_kernel<", "loss_rows"),
                     ("mean_kernel", "loss_mean"), ("to_bf16_kernel", "to_bf16"),
                     ("gather_rows_kernel<", "gather_rows")):
        if key in name:
            return cls
    return None


def _counter_rows(path):
    import csv
    with open(path) as fh:
        return [(r["Kernel_Name"], float(r["Counter_Value"])) for r in csv.DictReader(fh)]


def pmc_summary(fetch_csv, write_csv, workload, cmd_args):
    """Writes profiles/<workload>_hbm_traffic.md from two counter files."""
    import collections
    per = {}
    scale = {}
    for counter, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        rows = _counter_rows(path)
        copy = [v for k, v in rows if "copyBuffer" in k]
        if len(copy) != 1:
            sys.exit(f"bench.py: expected one calibration copy in {path}, found {len(copy)}")
        if cmd_args["calib_copy_mib"] <= 0:
            sys.exit("bench.py: --pmc-summary needs the run's --calib-copy-mib")
        scale[counter] = cmd_args["calib_copy_mib"] * 1024.0 / copy[0]   # true per counted
        acc = collections.defaultdict(list)
        for k, v in rows:
            c = kernel_class(k)
            if c:
                acc[c].append(v)
        per[counter] = acc
    classes = sorted(per["FETCH_SIZE"], key=lambda c: -sum(per["FETCH_SIZE"][c]))
    table = {}
    for c in classes:
        f = per["FETCH_SIZE"][c]
        w = per["WRITE_SIZE"].get(c, [])
        if not w or len(w) != len(f):
            continue
        fk, wk = sum(f) / len(f), sum(w) / len(w)
        table[c] = dict(dispatches=len(f), fetch_kib=round(fk, 1), write_kib=round(wk, 1),
                        bytes_per_launch=round(1024.0 * (fk * scale["FETCH_SIZE"]
                                                         + wk * scale["WRITE_SIZE"])),
                        source_hash=source_hash(c))
    bargs = (f"--workload {workload} --steps {cmd_args['steps']} --warmup {cmd_args['warmup']} "
             f"--profile-steps {cmd_args['profile_steps']} --no-cpu-baseline --no-direct "
             f"--no-narrow --no-adam --no-extra "
             f"--calib-copy-mib {cmd_args['calib_copy_mib']}")
    lines = [
        f"# HBM traffic per launch, {workload} training step",
        "",
        "Counters from two rocprofv3 passes over the same bench run (run from /tmp with",
        "TMPDIR=/tmp; `$R` is the repository root):",
        "",
        "```",
        f"rocprofv3 --pmc FETCH_SIZE --output-format csv -d OUT -o fetch -- python3 $R/bench.py {bargs}",
        f"rocprofv3 --pmc WRITE_SIZE --output-format csv -d OUT -o write -- python3 $R/bench.py {bargs}",
        f"python3 bench.py {bargs} --pmc-summary OUT/fetch_counter_collection.csv "
        "OUT/write_counter_collection.csv",
        "```",
        "",
        f"Calibration: one plain device copy of {cmd_args['calib_copy_mib']} MiB in the same "
        f"run; its true bytes over the counted ones give the factors FETCH_SIZE "
        f"x{scale['FETCH_SIZE']:.4f} and WRITE_SIZE x{scale['WRITE_SIZE']:.4f}, which multiply "
        "every kernel's counters below.",
        "",
        "| kernel class | dispatches | FETCH_SIZE KiB/disp | WRITE_SIZE KiB/disp | HBM bytes/launch (scaled) |",
        "|---|---:|---:|---:|---:|",
    ]
    for c, t in table.items():
        lines.append(f"| {c} | {t['dispatches']} | {t['fetch_kib']} | {t['write_kib']} | "
                     f"{t['bytes_per_launch']:,} |")
    lines += ["", "```json",
              json.dumps(dict(workload=workload, scale=scale, classes=table), indent=1),
              "```", ""]
    out = os.path.join(ROOT, "profiles", f"{workload}_hbm_traffic.md")
    with open(out, "w") as fh:
        fh.write("\n".join(lines))
    print(out)


def l2_summary(counter_csv, workload, cmd_args):
    """Writes profiles/<workload>_l2_hit_rate.md: per kernel class, the L2
    (TCC) hits and misses per launch from one rocprofv3 pass; misses go on
    to the Infinity Cache or HBM."""
    import collections
    import csv
    acc = collections.defaultdict(lambda: collections.defaultdict(list))
    with open(counter_csv) as fh:
        for r in csv.DictReader(fh):
            c = kernel_class(r["Kernel_Name"])
            if c:
                acc[c][r["Counter_Name"]].append(float(r["Counter_Value"]))
    bargs = (f"--workload {workload} --steps {cmd_args['steps']} --warmup {cmd_args['warmup']} "
             f"--profile-steps {cmd_args['profile_steps']} --no-cpu-baseline --no-direct "
             f"--no-narrow --no-adam --no-extra")
    lines = [f"# L2 hit rate per kernel class, {workload} training step", "",
             "One rocprofv3 counter pass over a bench run (run from /tmp with TMPDIR=/tmp; "
             "`$R` is the repository root):", "", "```",
             f"rocprofv3 --pmc TCC_HIT_sum TCC_MISS_sum --output-format csv -d OUT -o l2 -- "
             f"python3 $R/bench.py {bargs}",
             f"python3 bench.py {bargs} --l2-summary OUT/l2_counter_collection.csv", "```", "",
             "Hits and misses are L2 (TCC) requests summed over the eight XCDs; a miss is "
             "served by the Infinity Cache or HBM.", "",
             "| kernel class | dispatches | L2 hits / launch | L2 misses / launch | hit rate |",
             "|---|---:|---:|---:|---:|"]
    rows = []
    for c, d in acc.items():
        h, m = d.get("TCC_HIT_sum", []), d.get("TCC_MISS_sum", [])
        if not h or len(h) != len(m):
            continue
        hk, mk = sum(h) / len(h), sum(m) / len(m)
        rows.append((c, len(h), hk, mk, hk / max(hk + mk, 1.0)))
    for c, n, hk, mk, rate in sorted(rows, key=lambda r: -(r[2] + r[3])):
        lines.append(f"| {c} | {n} | {hk:,.0f} | {mk:,.0f} | {rate:.3f} |")
    lines.append("")
    out = os.path.join(ROOT, "profiles", f"{workload}_l2_hit_rate.md")
    with open(out, "w") as fh:
        fh.write("\n".join(lines))
    print(out)


MFMA_COUNTERS = ("MfmaUtil SQ_INSTS_VALU_MFMA_MOPS_F32 SQ_INSTS_VALU_MFMA_MOPS_BF16 "
                 "LdsBankConflict SQ_WAIT_INST_ANY SQ_BUSY_CU_CYCLES")


def mfma_summary(counter_csv, workload, cmd_args):
    """Writes profiles/<workload>[_bf16]_mfma_util.md: per kernel class and
    launch, the matrix-core utilisation (MfmaUtil: MFMA busy cycles over
    active cycles of all 1,024 SIMDs, in %), the MFMA operations the
    counters saw (x512 flops) against the algorithmic flops, LDS bank
    conflicts and issue waits, from one rocprofv3 pass."""
    import collections
    import csv
    acc = collections.defaultdict(lambda: collections.defaultdict(list))
    with open(counter_csv) as fh:
        for r in csv.DictReader(fh):
            c = kernel_class(r["Kernel_Name"])
            if c:
                acc[c][r["Counter_Name"]].append(float(r["Counter_Value"]))
    bf16 = cmd_args.get("precision") == "bf16"
    bargs = (f"--workload {workload} --steps {cmd_args['steps']} --warmup {cmd_args['warmup']} "
             f"--profile-steps {cmd_args['profile_steps']} --no-cpu-baseline --no-direct "
             f"--no-narrow --no-adam --no-extra" + (" --precision bf16" if bf16 else ""))
    tag = f"{workload}_bf16" if bf16 else workload
    lines = [f"# Matrix-core utilisation per kernel class, {tag} training step", "",
             "One rocprofv3 counter pass over a bench run (run from /tmp with TMPDIR=/tmp; "
             "`$R` is the repository root):", "", "```",
             f"rocprofv3 --pmc {MFMA_COUNTERS} --output-format csv -d OUT -o mfma -- "
             f"python3 $R/bench.py {bargs}",
             f"python3 bench.py {bargs} --mfma-summary OUT/mfma_counter_collection.csv", "```",
             "",
             "MfmaUtil is rocprofv3's derived metric: SQ_VALU_MFMA_BUSY_CYCLES summed over the "
             "SIMDs over GRBM_GUI_ACTIVE times the 1,024 SIMDs, in %, averaged over the "
             "class's dispatches. MFMA GFLOP = (MOPS_F32 + MOPS_BF16) x 512 per launch. "
             "LdsBankConflict: % of active cycles the LDS stalled on bank conflicts. "
             "SQ_WAIT_INST_ANY and SQ_BUSY_CU_CYCLES are per launch, summed over the "
             "GPU.", "",
             "| kernel class | dispatches | MfmaUtil % | MFMA GFLOP / launch | LdsBankConflict % "
             "| SQ_WAIT_INST_ANY / launch | SQ_BUSY_CU_CYCLES / launch |",
             "|---|---:|---:|---:|---:|---:|---:|"]

    def mean(d, k):
        v = d.get(k, [])
        return sum(v) / len(v) if v else float("nan")
    rows = []
    for c, d in acc.items():
        n = max(len(v) for v in d.values())
        mops = mean(d, "SQ_INSTS_VALU_MFMA_MOPS_F32") + mean(d, "SQ_INSTS_VALU_MFMA_MOPS_BF16")
        rows.append((c, n, mean(d, "MfmaUtil"), mops * 512 / 1e9, mean(d, "LdsBankConflict"),
                     mean(d, "SQ_WAIT_INST_ANY"), mean(d, "SQ_BUSY_CU_CYCLES")))
    for c, n, u, gf, lds, wait, busy in sorted(rows, key=lambda r: -r[3]):
        lines.append(f"| {c} | {n} | {u:.1f} | {gf:.3f} | {lds:.2f} | {wait:,.0f} | "
                     f"{busy:,.0f} |")
    lines.append("")
    out = os.path.join(ROOT, "profiles", f"{tag}_mfma_util.md")
    with open(out, "w") as fh:
        fh.write("\n".join(lines))
    print(out)


def trace_summary(stats_csv, workload, cmd_args, bench_line=None):
    """Writes profiles/<workload>_train_step_kernel_stats.md from a rocprofv3
    kernel_stats.csv: per kernel and per timing class, calls and mean
    duration."""
    import collections
    import csv
    with open(stats_csv) as fh:
        rows = list(csv.DictReader(fh))
    by_cls = collections.defaultdict(lambda: [0, 0.0])
    lines_k = []
    for r in rows:
        c = kernel_class(r["Name"])
        calls, tot = int(r["Calls"]), float(r["TotalDurationNs"])
        if c:
            by_cls[c][0] += calls
            by_cls[c][1] += tot
        name = r["Name"].replace("gcn::(anonymous namespace)::", "")
        name = name.split("(", 1)[0] if name.startswith("void ") else name[:90]
        lines_k.append(f"| {c or '-'} | `{name[:110]}` | {calls} | "
                       f"{float(r['AverageNs']) / 1e3:.2f} | {tot / 1e6:.3f} |")
    bargs = f"--workload {workload} {cmd_args}"
    bf16 = "--precision bf16" in cmd_args
    infer = "--infer" in cmd_args
    what = "inference" if infer else "training step"
    tag = (f"{workload}_bf16" if bf16 else workload) + ("_infer" if infer else "_train_step")
    out = [f"# Kernel durations, {workload} {'bf16 ' if bf16 else ''}{what} "
           "(rocprofv3 kernel trace)", "",
           "```", "cd /tmp && export TMPDIR=/tmp",
           f"rocprofv3 --kernel-trace --stats --output-format csv -d OUT -o run -- "
           f"python3 $R/bench.py {bargs}",
           f"python3 bench.py --workload {workload} --traced-args='{cmd_args}' "
           "--trace-summary OUT/run_kernel_stats.csv --bench-line OUT/line.json", "```",
           "", ("The run covers the device-only pass over the sampled minibatches (gathers "
                "and steps), then the host-pipelined, device-reduction-pipelined and mixed "
                "passes; the device reduction's own kernels are listed per kernel below, "
                "outside the timing classes." if workload in _SAMPLED_NAMES else
                "The run covers the device-only pass over the 64 subgraphs, then the "
                "host-pipelined, device-reduction-pipelined and mixed passes; the device "
                "reduction's own kernels are listed per kernel below, outside the timing "
                "classes." if workload == "stream8k" else
                "The run covers the warm-up, timed and profiled inference calls on the "
                "reduced graph." if infer and "--no-direct" in cmd_args else
                "The run covers the warm-up, timed and profiled steps of the reduced-graph "
                "step alone." if all(f in cmd_args for f in ("--no-direct", "--no-narrow", "--no-adam", "--no-extra")) else
                "The run also covers the comparison runs bench.py times beside the step "
                "(their kernels are counted in the same classes)."), "",
           "## Per timing class (the classes bench.py times with HIP events)", "",
           "| class | calls | mean us | total ms |", "|---|---:|---:|---:|"]
    for c, (n, tot) in sorted(by_cls.items(), key=lambda kv: -kv[1][1]):
        out.append(f"| {c} | {n} | {tot / n / 1e3:.2f} | {tot / 1e6:.3f} |")
    if bench_line:
        out += ["", "Event timing in the same process (bench.py `kernels`, mean us per launch):", "",
                "| class | mean us (events) |", "|---|---:|"]
        for c, k in bench_line["kernels"].items():
            out.append(f"| {c} | {k['avg_us']} |")
    out += ["", "## Per kernel", "", "| class | kernel | calls | mean us | total ms |",
            "|---|---|---:|---:|---:|"] + lines_k + [""]
    path = os.path.join(ROOT, "profiles", f"{tag}_kernel_stats.md")
    with open(path, "w") as fh:
        fh.write("\n".join(out))
    print(path)


def stored_traffic(workload, cls):
    """Scaled HBM bytes per launch of `cls` from the committed counter table,
    or None when there is none or the kernel's sources have changed since."""
    path = os.path.join(ROOT, "profiles", f"{workload}_hbm_traffic.md")
    if not os.path.exists(path):
        return None
    txt = open(path).read()
    try:
        blob = json.loads(txt.split("```json", 1)[1].split("```", 1)[0])
        t = blob["classes"][cls]
    except (IndexError, KeyError, ValueError):
        return None
    return t["bytes_per_launch"] if t["source_hash"] == source_hash(cls) else None


class Setup:
    """Inputs of one workload on the device, ready for timed steps."""

    def __init__(self, wl, reduce, inp, seg_len=0, precision=0, order=0, optim=None):
        import torch
        from paper_2001_02498_amd import gcn
        self.gcn, self.wl = gcn, wl
        t0 = time.perf_counter()
        g = gcn.subgraph_build(wl.n, inp.src, inp.dst)
        t1 = time.perf_counter()
        red = gcn.redundancy_reduce(g, theta=wl.theta, max_rounds=wl.rounds if reduce else 0,
                                    max_aux=wl.max_aux)
        t2 = time.perf_counter()
        self.host_ms = dict(subgraph_build=1e3 * (t1 - t0), reduction=1e3 * (t2 - t1))
        self.info = red.info()
        self.dg = gcn.DeviceGraph(red, seg_len=seg_len)

        def mat(x, ld=None):
            import numpy as np
            x = np.asarray(x, dtype=np.float32)
            ld = ld or (x.shape[1] + 3) // 4 * 4
            buf = torch.zeros((x.shape[0], ld), dtype=torch.float32)
            buf[:, :x.shape[1]] = torch.from_numpy(x)
            return buf.cuda()[:, :x.shape[1]]

        self.X = mat(inp.X)
        self.Ws = [mat(w, wl.h) for w in inp.W_self]
        self.Wn = [mat(w, wl.h) for w in inp.W_neigh]
        self.Wc = torch.from_numpy(inp.W_cls.copy()).cuda()
        self.labels = torch.from_numpy(inp.labels).cuda()
        self.P = gcn.make_params(self.Ws, self.Wn, self.Wc)
        self.desc = gcn.model_desc(wl.L, wl.f_in, wl.h, wl.C, wl.loss, self.X.stride(0),
                                   precision=precision, order=order)
        self.ws = gcn.alloc_ws(gcn.workspace_bytes(self.dg, self.desc))
        self.loss = torch.zeros(1, device="cuda")
        # optimiser states (zero, shaped like the weights) when not plain descent
        self.opt, self.S = None, [None, None]
        if optim is not None:
            self.opt = gcn.optim(optim, wl.lr)
            self.states = []
            for _ in range(2 if optim == gcn.OPT_ADAM else 1):
                t = ([torch.zeros_like(w) for w in self.Ws], [torch.zeros_like(w) for w in self.Wn],
                     torch.zeros_like(self.Wc))
                self.states.append(t)
                self.S[len(self.states) - 1] = gcn.make_params(*t)
        torch.cuda.synchronize()

    def step(self):
        if self.opt is not None:
            self.gcn.train_step_optim(self.dg, self.desc, self.P, self.X, self.labels, self.opt,
                                      self.loss, self.ws, state1=self.S[0], state2=self.S[1])
            return
        self.gcn.train_step(self.dg, self.desc, self.P, self.X, self.labels, self.wl.lr,
                            self.loss, self.ws)

    def capture(self):
        """Record one step into a HIP graph (stream capture on a side stream)."""
        import torch
        self.step()                       # warm: first launches load code objects
        torch.cuda.synchronize()
        self.graph = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream()
        with torch.cuda.stream(s):
            self.graph.capture_begin()
            self.step()
            self.graph.capture_end()
        torch.cuda.synchronize()

    def timed(self, steps, warmup, graph=False):
        import torch
        run = self.step
        if graph:
            self.capture()
            run = self.graph.replay
        for _ in range(warmup):
            run()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            run()
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / steps

    def profile(self, steps):
        import torch
        gcn = self.gcn
        gcn.profile_enable(4096)
        for _ in range(steps):
            self.step()
        torch.cuda.synchronize()
        prof = gcn.profile_read(reset=True)
        gcn.profile_disable()
        return prof


def kernel_table(prof, steps):
    out = {}
    for name, e in prof.items():
        n = e["launches"]
        avg_s = e["total_ms"] / n * 1e-3
        out[name] = dict(
            launches_per_step=n / steps,
            avg_us=round(avg_s * 1e6, 2),
            ms_per_step=round(e["total_ms"] / steps, 4),
            tflops=round(e["flops"] / n / avg_s / 1e12, 2) if e["flops"] else 0.0,
            gbs=round(e["bytes"] / n / avg_s / 1e9, 1) if e["bytes"] else 0.0,
            flops_per_launch=e["flops"] / n, bytes_per_launch=e["bytes"] / n)
    return out


def roofline(name, k, workload):
    """Roofline position of one kernel class: algorithmic flops (GEMM) or
    bytes (everything else) per launch over the mean event-timed launch.
    `traffic` is the counter-measured HBM bytes per launch (None when not
    measured for the current sources); `algorithmic_bytes` sits beside it
    for comparison."""
    traffic = stored_traffic(workload, name)
    extra = dict(traffic=traffic, traffic_unit="bytes/launch",
                 algorithmic_bytes=round(k["bytes_per_launch"]))
    if name.startswith("gemm"):
        # a GEMM is bound by whichever of its flops (at the matrix peak of its
        # operand type) and its compulsory bytes (at HBM peak) takes longer
        peak = PEAK_BF16_MFMA_TFLOPS if name.endswith("_bf16") else PEAK_FP32_MFMA_TFLOPS
        t_flops = k["flops_per_launch"] / (peak * 1e12)
        t_bytes = k["bytes_per_launch"] / (PEAK_HBM_GBS * 1e9)
        if t_flops >= t_bytes:
            achieved = k["flops_per_launch"] / (k["avg_us"] * 1e-6) / 1e12
            return dict(kernel=name, bound="mfma", achieved=round(achieved, 2), peak=peak,
                        unit="TFLOP/s", frac=round(achieved / peak, 4), **extra)
    achieved = k["bytes_per_launch"] / (k["avg_us"] * 1e-6) / 1e9
    return dict(kernel=name, bound="hbm", achieved=round(achieved, 1), peak=PEAK_HBM_GBS,
                unit="GB/s", frac=round(achieved / PEAK_HBM_GBS, 4), **extra)


def achievable_bandwidth(mib=1024, reps=10):
    """Device-copy bandwidth (read + write bytes per second) of a buffer far
    larger than the caches, timed with events."""
    import torch
    a = torch.ones((mib << 20) // 4, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    b.copy_(a)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    gbs = 2.0 * a.numel() * 4 * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del a, b
    return round(gbs, 1)


def read_bandwidth(mib=2048, reps=10):
    """HBM bandwidth of a read-only kernel (gcn_read_probe: every word of a
    buffer 8x the Infinity Cache read once), timed with events on the stream
    it is launched on: the denominator for kernels that mostly read."""
    import torch
    from paper_2001_02498_amd import gcn
    a = torch.ones((mib << 20) // 4, dtype=torch.float32, device="cuda")
    sink = torch.empty(gcn.READ_PROBE_SINK, dtype=torch.float32, device="cuda")
    gcn.read_probe(a, sink)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        gcn.read_probe(a, sink)
    e1.record()
    torch.cuda.synchronize()
    assert float(sink.sum().item()) == float(a.numel()), "read probe summed wrongly"
    gbs = a.numel() * 4.0 * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del a, sink
    return round(gbs, 1)


def aggregation_compulsory(wl, info):
    """Compulsory bytes of one step's list-sum launches: every extended row
    (n + naux of them) read once, every output row written once, the lists
    and row pointers read once -- the floor under the algorithmic count,
    which charges every neighbour-row gather."""
    n, naux, nnz = wl.n, info["naux"], int(info["nnz"])
    widths = [wl.f_in] + [2 * wl.h] * (wl.L - 1) + [wl.h] * (wl.L - 1)
    per = [4.0 * F * (n + naux) + 4.0 * F * n + 4.0 * (n + 1 + nnz) for F in widths]
    return sum(per) / len(per)


def aggregation_roofline(wl, info, ktab, read_gbs):
    """The list sums against HBM. achieved = compulsory bytes per launch
    (every extended row read once, every output written once, the lists
    read once) over the mean event-timed launch; frac against the 8 TB/s
    peak, frac_of_achievable against the read-only probe measured in the
    same process. The algorithmic count, which charges every neighbour-row
    gather (most served by L2 and the Infinity Cache), is reported beside it
    as gather_GBs, and the counter-measured bytes (traffic) when recorded
    for the current sources."""
    k = ktab["list_sums"]
    t = k["avg_us"] * 1e-6
    comp = aggregation_compulsory(wl, info)
    achieved = comp / t / 1e9
    traffic = stored_traffic(wl.name, "list_sums")
    out = dict(kernel="list_sums", bound="hbm", achieved=round(achieved, 1),
               peak=PEAK_HBM_GBS, unit="GB/s", frac=round(achieved / PEAK_HBM_GBS, 4),
               bytes="compulsory", compulsory_bytes=round(comp),
               achievable_read_GBs=read_gbs,
               frac_of_achievable=None if not read_gbs else round(achieved / read_gbs, 4),
               traffic=traffic, traffic_unit="bytes/launch",
               traffic_GBs=None if traffic is None else round(traffic / t / 1e9, 1),
               gather_bytes=round(k["bytes_per_launch"]),
               gather_GBs=round(k["bytes_per_launch"] / t / 1e9, 1),
               avg_us=k["avg_us"])
    return out


def cpu_baseline(wl, inp, budget_s):
    import threadpoolctl
    from oracle import gcn as og
    from oracle import graph as gr
    rp, cl = gr.subgraph_build(wl.n, inp.src, inp.dst)
    params = dict(W_self=inp.W_self, W_neigh=inp.W_neigh, b=[None] * wl.L, W_cls=inp.W_cls,
                  b_cls=None)
    og.train_step(rp, cl, inp.X, params, inp.labels, wl.loss, wl.lr)   # warm caches
    reps, t0 = 0, time.perf_counter()
    while True:
        og.train_step(rp, cl, inp.X, params, inp.labels, wl.loss, wl.lr)
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s or reps >= 100:
            break
    threads = max((p.get("num_threads", 1) for p in threadpoolctl.threadpool_info()
                   if p.get("user_api") == "blas"), default=1)
    return dict(value=round(reps / el, 4), unit="steps/s", cores=int(threads), kind="oracle",
                sample=f"{reps} float64 oracle steps (forward, loss, backward, update; "
                       f"aggregation as D^-1 A H) of {wl.name} in {el:.1f} s; "
                       f"BLAS threads {threads}, os.cpu_count {os.cpu_count()}")


def _mat(x, ld=None):
    import numpy as np
    import torch
    x = np.asarray(x, dtype=np.float32)
    ld = ld or (x.shape[1] + 3) // 4 * 4
    buf = torch.zeros((x.shape[0], ld), dtype=torch.float32)
    buf[:, :x.shape[1]] = torch.from_numpy(x)
    return buf.cuda()[:, :x.shape[1]]


class _Desc:
    """Holds a device-graph descriptor the way DeviceGraph does."""

    def __init__(self, desc):
        self.desc = desc


def run_stream(args):
    """The epoch-shaped stream: 64 independently seeded subgraphs, one model.

    Phase A prepares every subgraph on the host, uploads all of them and
    times the device steps alone. Phase B runs the Section 4.4 schedule:
    host workers prepare subgraph i+1.. while the device trains on i; each
    image is copied on a copy stream into one of two device slots, and the
    compute stream waits on the copy's event."""
    import collections
    import concurrent.futures as cf

    import torch

    from paper_2001_02498_amd import gcn, synth

    K = args.stream_len
    wls = [synth.stream_workload(i) for i in range(K)]
    wl = wls[0]
    with cf.ThreadPoolExecutor(8) as ex:
        inps = list(ex.map(synth.make_inputs, wls))
    print(f"[bench] stream of {K} subgraphs: inputs ready", file=sys.stderr, flush=True)
    Xs = [_mat(inp.X) for inp in inps]
    Ys = [torch.from_numpy(inp.labels).cuda() for inp in inps]
    Ws = [_mat(w, wl.h) for w in inps[0].W_self]
    Wn = [_mat(w, wl.h) for w in inps[0].W_neigh]
    Wc = torch.from_numpy(inps[0].W_cls.copy()).cuda()
    P = gcn.make_params(Ws, Wn, Wc)
    desc = gcn.model_desc(wl.L, wl.f_in, wl.h, wl.C, wl.loss, Xs[0].stride(0))
    loss = torch.zeros(1, device="cuda")

    # Phase A: host preparation one subgraph at a time, then device steps alone
    prep_ms, dgs = [], []
    for inp in inps:
        t0 = time.perf_counter()
        red = gcn.redundancy_reduce(gcn.subgraph_build(wl.n, inp.src, inp.dst), theta=wl.theta,
                                    max_rounds=wl.rounds, max_aux=wl.max_aux, num_threads=1)
        prep_ms.append(1e3 * (time.perf_counter() - t0))
        dgs.append(gcn.DeviceGraph(red, seg_len=args.seg_len))
    ws_bytes = max(gcn.workspace_bytes(d, desc) for d in dgs)
    ws = gcn.alloc_ws(ws_bytes)
    img_bytes = max(d.nbytes for d in dgs)

    def step(dg, i):
        gcn.train_step(dg, desc, P, Xs[i], Ys[i], wl.lr, loss, ws)

    for i in range(min(args.warmup, K)):
        step(dgs[i], i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(K):
        step(dgs[i], i)
    torch.cuda.synchronize()
    gpu_ms = 1e3 * (time.perf_counter() - t0) / K
    gcn.profile_enable(8192)
    for i in range(min(args.profile_steps, K)):
        step(dgs[i], i)
    torch.cuda.synchronize()
    prof = gcn.profile_read(reset=True)
    gcn.profile_disable()
    print(f"[bench] device only: {gpu_ms:.3f} ms/step", file=sys.stderr, flush=True)

    # Phase B: the overlapped schedule (GPU-reducing workers get a device
    # workspace share each, sized up front for the largest subgraph)
    dev_share = gcn.device_reduce_bytes(
        [gcn.subgraph_build(wl.n, inp.src, inp.dst) for inp in inps], 1, theta=wl.theta,
        max_rounds=wl.rounds, max_aux=wl.max_aux)
    slots = [gcn.alloc_ws(img_bytes) for _ in range(2)]
    copy = torch.cuda.Stream()
    comp = torch.cuda.current_stream()

    def overlapped(workers, device_reduce, device_workers=None):
        slot_free = [None, None]
        held = collections.deque()
        infos = []
        nw = workers + (device_workers or 0)
        ndev = device_workers or (workers if device_reduce else 0)
        dws = gcn.alloc_ws(ndev * dev_share) if ndev else None
        pipe = gcn.Pipeline(theta=wl.theta, max_rounds=wl.rounds, max_aux=wl.max_aux,
                            seg_len=args.seg_len, workers=workers, depth=2 * nw + 2,
                            pinned=True, num_threads=1, device_reduce=device_reduce,
                            device_workers=device_workers, device_ws=dws)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for inp in inps:
            pipe.submit(wl.n, inp.src, inp.dst)
        for i in range(K):
            jid, ptr, nb, info = pipe.next()
            infos.append(info)
            slot = i % 2
            with torch.cuda.stream(copy):
                if slot_free[slot] is not None:
                    copy.wait_event(slot_free[slot])
                d = gcn.upload_image(ptr, nb, slots[slot], stream=copy)
                copied = torch.cuda.Event()
                copied.record(copy)
            comp.wait_event(copied)
            step(_Desc(d), i)
            done = torch.cuda.Event()
            done.record(comp)
            slot_free[slot] = done
            held.append((jid, copied))
            while len(held) > 1:
                j, e = held.popleft()
                e.synchronize()
                pipe.release(j)
        torch.cuda.synchronize()
        ms = 1e3 * (time.perf_counter() - t0) / K
        for j, _ in held:
            pipe.release(j)
        pipe.close()
        return ms, infos

    workers = args.workers or min(16, os.cpu_count() or 1)
    pipe_ms, infos = overlapped(workers, False)
    print(f"[bench] pipelined with {workers} workers: {pipe_ms:.3f} ms/step",
          file=sys.stderr, flush=True)
    dworkers = args.device_workers
    dev_ms, dinfos = overlapped(dworkers, True)
    print(f"[bench] pipelined with {dworkers} workers reducing on the GPU: {dev_ms:.3f} ms/step",
          file=sys.stderr, flush=True)
    hmix = max(1, workers - dworkers)
    mix_ms, minfos = overlapped(hmix, False, dworkers)
    print(f"[bench] pipelined with {hmix} host and {dworkers} GPU-reducing workers: "
          f"{mix_ms:.3f} ms/step", file=sys.stderr, flush=True)
    ktab = kernel_table(prof, min(args.profile_steps, K))
    dominant = max(ktab, key=lambda k: ktab[k]["ms_per_step"])
    roof = roofline(dominant, ktab[dominant], "stream8k")
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(wl, inps[0], args.cpu_seconds)
    reduce_ms = [inf.reduce_ms for inf in infos]
    return {
        "metric": METRIC,
        "value": round(1e3 / pipe_ms, 3),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(pipe_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": (f"stream8k: {K} independently seeded {wl.n}-vertex Chung-Lu subgraphs "
                         f"(exponent {wl.gamma}, mean degree {wl.dbar}), {wl.L}-layer GCN, f_in "
                         f"{wl.f_in}, {wl.h} per branch, {wl.C}-class softmax CE, reduced graph "
                         f"({wl.rounds} rounds, threshold {wl.theta}, budget {wl.budget} n); host "
                         f"preparation of later subgraphs overlapped with device training"),
            "n": wl.n, "host_workers": workers, "parallelism": "single GPU",
        },
        "roofline": {k: v for k, v in roof.items() if k != "kernel"} | {"kernel": dominant},
        "cpu_baseline": cpu,
        "device_only_ms_per_step": round(gpu_ms, 4),
        "host_prepare_ms_per_subgraph": {
            "one_thread_mean": round(sum(prep_ms) / K, 2),
            "in_pipeline_reduce_mean": round(sum(reduce_ms) / K, 2)},
        "device_reduction_pipeline": {
            "ms_per_step": round(dev_ms, 4), "steps_per_s": round(1e3 / dev_ms, 3),
            "workers": dworkers,
            "reduce_ms_mean": round(sum(i.reduce_ms for i in dinfos) / K, 3),
            "note": "the same schedule with each worker running Algorithms 1-3 on the GPU "
                    "(gcn_redundancy_reduce_device, identical result) on a stream of its own"},
        "mixed_reduction_pipeline": {
            "ms_per_step": round(mix_ms, 4), "steps_per_s": round(1e3 / mix_ms, 3),
            "host_workers": hmix, "device_workers": dworkers,
            "note": "host and GPU-reducing workers taking jobs from one queue "
                    "(gcn_pipeline_create_mixed)"},
        "kernels": {k: {kk: vv for kk, vv in v.items()
                        if kk not in ("flops_per_launch", "bytes_per_launch")}
                    for k, v in ktab.items()},
    }


def cpu_baseline_sampled(wl, fi, budget_s):
    """The oracle per sampled minibatch: its walk and induced subgraph on the
    full graph (plain loops), then its training step; the full graph's CSR is
    built once beforehand, as the library builds it once."""
    import threadpoolctl
    from oracle import gcn as og
    from oracle import graph as gr
    from oracle import sample as osample
    rp, cl = gr.subgraph_build(wl.n_full, fi.src, fi.dst)
    params = dict(W_self=fi.W_self, W_neigh=fi.W_neigh, b=[None] * wl.L, W_cls=fi.W_cls,
                  b_cls=None)
    reps, t0 = 0, time.perf_counter()
    while True:
        V = osample.frontier_sample(rp, cl, wl.m, wl.budget, wl.sample_seed(reps),
                                    wl.max_steps)
        srp, scl = osample.induce(rp, cl, V)
        og.train_step(srp, scl, fi.X[V], params, fi.labels[V], wl.loss, wl.lr)
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s or reps >= 100:
            break
    threads = max((p.get("num_threads", 1) for p in threadpoolctl.threadpool_info()
                   if p.get("user_api") == "blas"), default=1)
    return dict(value=round(reps / el, 4), unit="steps/s", cores=int(threads), kind="oracle",
                sample=f"{reps} sampled minibatches of {wl.name} (oracle walk and induced "
                       f"subgraph, then a float64 oracle step) in {el:.1f} s; BLAS threads "
                       f"{threads} (the walk and induction are single-threaded), "
                       f"os.cpu_count {os.cpu_count()}")


def run_sampled(args):
    """Minibatches sampled from one full graph (Section 3.1), trained in turn.

    The full graph's CSR lives on the host, its features and labels in device
    memory. A minibatch = frontier sampling + induced subgraph + reduction +
    packing (host workers, gcn_pipeline_submit_sample), one upload of the
    image with the sampled ids, gathers of the minibatch's feature and label
    rows on the device, and the training step. Phase A prepares every
    minibatch first and times the device work alone (gathers + step); phase B
    overlaps host preparation with device training (Section 4.4), with the
    reduction on the host workers, then on the GPU."""
    import collections

    import numpy as np
    import torch

    from paper_2001_02498_amd import gcn, synth

    wl = synth.SAMPLED[args.workload]
    K = args.stream_len
    t0 = time.perf_counter()
    fi = synth.make_full_inputs(wl)
    full = gcn.subgraph_build(wl.n_full, fi.src, fi.dst)
    X_full = _mat(fi.X)
    Y_full = torch.from_numpy(fi.labels).cuda()
    frp, _ = full.csr()
    fdeg = np.diff(frp)
    print(f"[bench] full graph {wl.n_full} vertices, {full.nnz} list entries: inputs ready in "
          f"{time.perf_counter() - t0:.1f} s", file=sys.stderr, flush=True)
    Ws = [_mat(w, wl.h) for w in fi.W_self]
    Wn = [_mat(w, wl.h) for w in fi.W_neigh]
    Wc = torch.from_numpy(fi.W_cls.copy()).cuda()
    P = gcn.make_params(Ws, Wn, Wc)
    desc = gcn.model_desc(wl.L, wl.f_in, wl.h, wl.C, wl.loss, X_full.stride(0))
    loss = torch.zeros(1, device="cuda")
    Xb = torch.empty((wl.budget, X_full.stride(0)), dtype=torch.float32, device="cuda")
    Yb = torch.empty(wl.budget, dtype=torch.int32, device="cuda")
    seeds = [wl.sample_seed(i) for i in range(K)]
    workers = args.workers or min(16, os.cpu_count() or 1)

    dev_share = []   # the GPU-reducing workers' workspace share, once known

    def new_pipe(nw, device_reduce, device_workers=None):
        tot = nw + (device_workers or 0)
        ndev = device_workers or (nw if device_reduce else 0)
        if ndev and not dev_share:
            # sized up front from the minibatches' own walks, taken on the host
            gs = [gcn.subgraph_induce(full, gcn.sample_frontier(full, wl.m, wl.budget, sd,
                                                                 wl.max_steps)[0])
                  for sd in seeds]
            dev_share.append(gcn.device_reduce_bytes(gs, 1, theta=wl.theta,
                                                     max_rounds=wl.rounds, max_aux=wl.max_aux))
        dws = gcn.alloc_ws(ndev * dev_share[0]) if ndev else None
        return gcn.Pipeline(theta=wl.theta, max_rounds=wl.rounds, max_aux=wl.max_aux,
                            seg_len=args.seg_len, workers=nw, depth=2 * tot + 2, pinned=True,
                            num_threads=1, device_reduce=device_reduce,
                            device_workers=device_workers, device_ws=dws)

    # Phase A: every minibatch prepared and resident, then device work alone
    pipe = new_pipe(workers, False)
    images, infos = [], []
    for sd in seeds:
        pipe.submit_sample(full, wl.m, wl.budget, sd, wl.max_steps)
    for i in range(K):
        jid, ptr, nb, info = pipe.next()
        buf = gcn.alloc_ws(nb)
        d = gcn.upload_image(ptr, nb, buf)
        torch.cuda.synchronize()
        pipe.release(jid)
        images.append((buf, d, nb))
        infos.append(info)
    pipe.close()
    dgs = [_Desc(d) for _, d, _ in images]
    ws = gcn.alloc_ws(max(gcn.workspace_bytes(d, desc) for d in dgs))
    img_bytes = max(nb for _, _, nb in images)

    def step(i, dg, buf, info):
        n = info.n
        vidx = buf[info.vertices_offset:info.vertices_offset + 4 * n].view(torch.int32)
        X = Xb[:n, :wl.f_in]
        gcn.gather_rows(X_full, vidx, X)
        gcn.gather_rows(Y_full, vidx, Yb[:n])
        gcn.train_step(dg, desc, P, X, Yb[:n], wl.lr, loss, ws)

    for i in range(min(args.warmup, K)):
        step(i, dgs[i], images[i][0], infos[i])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(K):
        step(i, dgs[i], images[i][0], infos[i])
    torch.cuda.synchronize()
    gpu_ms = 1e3 * (time.perf_counter() - t0) / K
    gcn.profile_enable(8192)
    for i in range(min(args.profile_steps, K)):
        step(i, dgs[i], images[i][0], infos[i])
    torch.cuda.synchronize()
    prof = gcn.profile_read(reset=True)
    gcn.profile_disable()
    print(f"[bench] device only: {gpu_ms:.3f} ms/step", file=sys.stderr, flush=True)

    # Phase B: the overlapped schedule
    slots = [gcn.alloc_ws(img_bytes) for _ in range(2)]
    copy = torch.cuda.Stream()
    comp = torch.cuda.current_stream()

    def overlapped(nw, device_reduce, device_workers=None):
        slot_free = [None, None]
        held = collections.deque()
        got = []
        p = new_pipe(nw, device_reduce, device_workers)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for sd in seeds:
            p.submit_sample(full, wl.m, wl.budget, sd, wl.max_steps)
        for i in range(K):
            jid, ptr, nb, info = p.next()
            got.append(info)
            slot = i % 2
            with torch.cuda.stream(copy):
                if slot_free[slot] is not None:
                    copy.wait_event(slot_free[slot])
                d = gcn.upload_image(ptr, nb, slots[slot], stream=copy)
                copied = torch.cuda.Event()
                copied.record(copy)
            comp.wait_event(copied)
            step(i, _Desc(d), slots[slot], info)
            done = torch.cuda.Event()
            done.record(comp)
            slot_free[slot] = done
            held.append((jid, copied))
            while len(held) > 1:
                j, e = held.popleft()
                e.synchronize()
                p.release(j)
        torch.cuda.synchronize()
        ms = 1e3 * (time.perf_counter() - t0) / K
        for j, _ in held:
            p.release(j)
        p.close()
        return ms, got

    pipe_ms, pinfos = overlapped(workers, False)
    print(f"[bench] pipelined with {workers} workers: {pipe_ms:.3f} ms/step", file=sys.stderr,
          flush=True)
    dworkers = args.device_workers
    dev_ms, dinfos = overlapped(dworkers, True)
    print(f"[bench] pipelined with {dworkers} workers reducing on the GPU: {dev_ms:.3f} ms/step",
          file=sys.stderr, flush=True)
    hmix = max(1, workers - dworkers)
    mix_ms, _ = overlapped(hmix, False, dworkers)
    print(f"[bench] pipelined with {hmix} host and {dworkers} GPU-reducing workers: "
          f"{mix_ms:.3f} ms/step", file=sys.stderr, flush=True)
    ktab = kernel_table(prof, min(args.profile_steps, K))
    dominant = max(ktab, key=lambda k: ktab[k]["ms_per_step"])
    roof = roofline(dominant, ktab[dominant], wl.name)
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline_sampled(wl, fi, args.cpu_seconds)

    def mean(xs):
        return round(float(np.mean(xs)), 3)
    return {
        "metric": METRIC,
        "value": round(1e3 / pipe_ms, 3),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(pipe_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": (f"{wl.name}: {K} minibatches of {wl.budget} vertices sampled by "
                         f"frontier sampling ({wl.m} walkers) from a {wl.n_full}-vertex "
                         f"Chung-Lu graph (exponent {wl.gamma}, mean degree {wl.dbar:.2f}); "
                         f"{wl.L}-layer GCN, f_in {wl.f_in}, {wl.h} per branch, {wl.C}-class "
                         f"softmax CE, reduced graph ({wl.rounds} rounds, threshold "
                         f"{wl.theta}, budget {wl.aux_budget} n); host preparation of later "
                         f"minibatches overlapped with device training"),
            "n_full": wl.n_full, "full_nnz": int(full.nnz), "full_max_degree": int(fdeg.max()),
            "host_workers": workers, "parallelism": "single GPU",
        },
        "roofline": {k: v for k, v in roof.items() if k != "kernel"} | {"kernel": dominant},
        "cpu_baseline": cpu,
        "device_only_ms_per_step": round(gpu_ms, 4),
        "minibatch": {"n_mean": mean([i.n for i in infos]),
                      "nnz_mean": mean([i.nnz_direct for i in infos]),
                      "nnz_reduced_mean": mean([i.nnz for i in infos]),
                      "naux_mean": mean([i.naux for i in infos]),
                      "walk_steps_mean": mean([i.steps for i in infos])},
        "host_ms_per_minibatch": {"sample": mean([i.sample_ms for i in pinfos]),
                                  "induce": mean([i.build_ms for i in pinfos]),
                                  "reduce": mean([i.reduce_ms for i in pinfos]),
                                  "pack": mean([i.pack_ms for i in pinfos])},
        "device_reduction_pipeline": {
            "ms_per_step": round(dev_ms, 4), "steps_per_s": round(1e3 / dev_ms, 3),
            "workers": dworkers, "reduce_ms_mean": mean([i.reduce_ms for i in dinfos])},
        "mixed_reduction_pipeline": {
            "ms_per_step": round(mix_ms, 4), "steps_per_s": round(1e3 / mix_ms, 3),
            "host_workers": hmix, "device_workers": dworkers},
        "kernels": {k: {kk: vv for kk, vv in v.items()
                        if kk not in ("flops_per_launch", "bytes_per_launch")}
                    for k, v in ktab.items()},
    }


class InferSetup(Setup):
    """A whole graph and the model on the device, ready for timed inference."""

    def __init__(self, *a, **kw):
        super().__init__(*a, **kw)
        import torch
        wl = self.wl
        self.Z = torch.empty((wl.n, (wl.C + 3) // 4 * 4), device="cuda")[:, :wl.C]

    def step(self):
        self.gcn.infer(self.dg, self.desc, self.P, self.X, self.Z, self.ws)


def infer_workload(n):
    """The ppi8k model (2 layers, f_in 50, 512 per branch, 121 classes) on a
    whole n-vertex graph of the same structure (Chung-Lu, exponent 2.5, mean
    degree 15): the stand-in for inference on an un-sampled graph."""
    from paper_2001_02498_amd import synth
    import dataclasses
    ppi = synth.WORKLOADS["ppi8k"]
    wl = synth.small_workload(n, ppi.dbar, ppi.L, ppi.f_in, ppi.h, ppi.C, ppi.loss, (7, n),
                              gamma=ppi.gamma, theta=ppi.theta, rounds=ppi.rounds,
                              label_p=ppi.label_p, budget=ppi.budget)
    return dataclasses.replace(wl, name=f"full{n // 1000}k")


def cpu_forward_baseline(wl, inp, budget_s):
    """The oracle's forward pass (aggregation as D^-1 A H) on the same graph."""
    import threadpoolctl
    from oracle import gcn as og
    from oracle import graph as gr
    rp, cl = gr.subgraph_build(wl.n, inp.src, inp.dst)
    params = dict(W_self=inp.W_self, W_neigh=inp.W_neigh, b=[None] * wl.L, W_cls=inp.W_cls,
                  b_cls=None)
    reps, t0 = 0, time.perf_counter()
    while True:
        og.forward(rp, cl, inp.X, params)
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s or reps >= 20:
            break
    threads = max((p.get("num_threads", 1) for p in threadpoolctl.threadpool_info()
                   if p.get("user_api") == "blas"), default=1)
    return dict(value=round(reps * wl.n / el, 1), unit="vertices/s", cores=int(threads),
                kind="oracle",
                sample=f"{reps} float64 oracle forward passes of {wl.name} in {el:.1f} s; "
                       f"BLAS threads {threads}, os.cpu_count {os.cpu_count()}")


def run_infer(args):
    import dataclasses

    from paper_2001_02498_amd import gcn, synth
    wl = infer_workload(args.infer_n)
    inp = synth.make_inputs(wl)
    print(f"[bench] whole graph {wl.name}: inputs ready", file=sys.stderr, flush=True)
    prec = gcn.PREC_BF16 if args.precision == "bf16" else gcn.PREC_FP32
    order = gcn.ORDER_NARROW if args.order == "narrow" else gcn.ORDER_PAPER
    red = InferSetup(wl, True, inp, args.seg_len, prec, order)
    ms = 1e3 * red.timed(args.steps, args.warmup)
    print(f"[bench] timed {args.steps} inference calls: {ms:.3f} ms/call", file=sys.stderr,
          flush=True)
    direct = None
    if not args.no_direct:
        d = InferSetup(dataclasses.replace(wl, reduce=False), False, inp, args.seg_len, prec,
                       order)
        direct = 1e3 * d.timed(args.steps, args.warmup)
        print(f"[bench] direct aggregation: {direct:.3f} ms/call", file=sys.stderr, flush=True)
        del d
    extra = {}
    if not args.no_extra:
        if prec == gcn.PREC_FP32:
            d = Setup(wl, wl.reduce, inp, args.seg_len, gcn.PREC_BF16, order)
            extra["bf16_ms_per_step"] = round(1e3 * d.timed(args.steps, args.warmup,
                                                            args.graph), 4)
            del d
        if wl.name != "ppi8k":
            pw = synth.WORKLOADS["ppi8k"]
            pin = synth.make_inputs(pw)
            for key, reduce in (("ppi8k_fp32_ms_per_step", True),
                                ("ppi8k_fp32_direct_ms_per_step", False)):
                d = Setup(dataclasses.replace(pw, reduce=reduce), reduce, pin, args.seg_len,
                          gcn.PREC_FP32, order)
                extra[key] = round(1e3 * d.timed(args.steps, args.warmup, args.graph), 4)
                del d
        print(f"[bench] extra figures: {extra}", file=sys.stderr, flush=True)
    prof = red.profile(args.profile_steps)
    ktab = kernel_table(prof, args.profile_steps)
    dominant = max(ktab, key=lambda k: ktab[k]["ms_per_step"])
    roof = roofline(dominant, ktab[dominant], wl.name)
    cpu = None if args.no_cpu_baseline else cpu_forward_baseline(wl, inp, args.cpu_seconds)
    i = red.info
    return {
        "metric": "whole-graph GCN inference (forward pass into logits) vertices/s",
        "value": round(wl.n / (ms * 1e-3), 1),
        "unit": "vertices/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_call": round(ms, 4),
        "higher_is_better": True,
        "dtype": "f32" if args.precision == "fp32" else "bf16 (dense products; fp32 accumulate)",
        "order": args.order,
        "data": "synthetic",
        "config": {
            "workload": (f"{wl.name}: the ppi8k model ({wl.L} layers, f_in {wl.f_in}, {wl.h} "
                         f"per branch, {wl.C} classes) on a whole {wl.n}-vertex Chung-Lu graph "
                         f"(exponent {wl.gamma}, mean degree {wl.dbar}), reduced on the host "
                         f"({wl.rounds} rounds, threshold {wl.theta})"),
            "n": wl.n, "nnz": int(red.dg.desc.nnz), "naux": i["naux"],
        },
        "roofline": {k: v for k, v in roof.items() if k != "kernel"} | {"kernel": dominant},
        "cpu_baseline": cpu,
        "direct_aggregation_ms_per_call": None if direct is None else round(direct, 4),
        "host_preprocess_ms": {k: round(v, 2) for k, v in red.host_ms.items()},
        "kernels": {k: {kk: vv for kk, vv in v.items()
                        if kk not in ("flops_per_launch", "bytes_per_launch")}
                    for k, v in ktab.items()},
    }


def main():
    args = parse()
    if args.trace_summary:
        line = None
        if args.bench_line:
            with open(args.bench_line) as fh:
                line = json.loads(fh.read().strip().splitlines()[-1])
        trace_summary(args.trace_summary, args.workload, args.traced_args, line)
        return
    if args.l2_summary:
        l2_summary(args.l2_summary, args.workload, vars(args))
        return
    if args.mfma_summary:
        mfma_summary(args.mfma_summary, args.workload, vars(args))
        return
    if args.pmc_summary:
        # the counted run's arguments are given again on this command line
        pmc_summary(*args.pmc_summary, args.workload, vars(args))
        return
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU only (asked for --gpus {args.gpus}); "
              "the path shards by subgraph across GPUs but no multi-GPU run exists",
              file=sys.stderr)
        sys.exit(2)
    import dataclasses

    import torch

    from paper_2001_02498_amd import synth

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    if args.infer:
        print(json.dumps(run_infer(args)), flush=True)
        return
    if args.workload == "stream8k":
        print(json.dumps(run_stream(args)), flush=True)
        return
    if args.workload in synth.SAMPLED:
        print(json.dumps(run_sampled(args)), flush=True)
        return
    wl = synth.WORKLOADS[args.workload]
    if args.theta is not None:
        wl = dataclasses.replace(wl, theta=args.theta)
    inp = synth.make_inputs(wl)
    print(f"[bench] workload {wl.name}: inputs ready", file=sys.stderr, flush=True)

    from paper_2001_02498_amd import gcn
    prec = gcn.PREC_BF16 if args.precision == "bf16" else gcn.PREC_FP32
    order = gcn.ORDER_NARROW if args.order == "narrow" else gcn.ORDER_PAPER
    red = Setup(wl, wl.reduce, inp, args.seg_len, prec, order)
    ms = 1e3 * red.timed(args.steps, args.warmup, args.graph)
    print(f"[bench] timed {args.steps} steps: {ms:.3f} ms/step", file=sys.stderr, flush=True)
    direct = None
    if wl.reduce and not args.no_direct:
        d = Setup(dataclasses.replace(wl, reduce=False), False, inp, args.seg_len, prec)
        direct = 1e3 * d.timed(args.steps, args.warmup, args.graph)
        print(f"[bench] direct aggregation: {direct:.3f} ms/step", file=sys.stderr, flush=True)
        del d
    narrow = None
    if order == gcn.ORDER_PAPER and not args.no_narrow:
        d = Setup(wl, wl.reduce, inp, args.seg_len, prec, gcn.ORDER_NARROW)
        narrow = 1e3 * d.timed(args.steps, args.warmup, args.graph)
        print(f"[bench] narrow-side order: {narrow:.3f} ms/step", file=sys.stderr, flush=True)
        del d
    adam = None
    if not args.no_adam:
        d = Setup(wl, wl.reduce, inp, args.seg_len, prec, order, optim=gcn.OPT_ADAM)
        adam = 1e3 * d.timed(args.steps, args.warmup, args.graph)
        print(f"[bench] Adam update: {adam:.3f} ms/step", file=sys.stderr, flush=True)
        del d
    extra = {}
    if not args.no_extra:
        if prec == gcn.PREC_FP32:
            d = Setup(wl, wl.reduce, inp, args.seg_len, gcn.PREC_BF16, order)
            extra["bf16_ms_per_step"] = round(1e3 * d.timed(args.steps, args.warmup,
                                                            args.graph), 4)
            del d
        if wl.name != "ppi8k":
            pw = synth.WORKLOADS["ppi8k"]
            pin = synth.make_inputs(pw)
            for key, reduce in (("ppi8k_fp32_ms_per_step", True),
                                ("ppi8k_fp32_direct_ms_per_step", False)):
                d = Setup(dataclasses.replace(pw, reduce=reduce), reduce, pin, args.seg_len,
                          gcn.PREC_FP32, order)
                extra[key] = round(1e3 * d.timed(args.steps, args.warmup, args.graph), 4)
                del d
        print(f"[bench] extra figures: {extra}", file=sys.stderr, flush=True)
    prof = red.profile(args.profile_steps)
    ktab = kernel_table(prof, args.profile_steps)
    dominant = max(ktab, key=lambda k: ktab[k]["ms_per_step"])
    roof = roofline(dominant, ktab[dominant], wl.name)
    # (the bandwidth probes are skipped in counter runs, whose only plain
    # copy is the calibration one)
    rd_bw = None if args.calib_copy_mib else read_bandwidth()
    agg = aggregation_roofline(wl, red.info, ktab, rd_bw) if "list_sums" in ktab else None
    print(f"[bench] profiled {args.profile_steps} steps; dominant {dominant}",
          file=sys.stderr, flush=True)

    if args.calib_copy_mib:
        nbytes = args.calib_copy_mib << 20
        a = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda").fill_(1.0)
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(wl, inp, args.cpu_seconds)
        print(f"[bench] cpu baseline: {cpu['value']} steps/s", file=sys.stderr, flush=True)

    i = red.info
    line = {
        "metric": METRIC,
        "value": round(1e3 / ms, 3),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if args.precision == "fp32" else "bf16 (dense products; fp32 accumulate)",
        "launch": "hip-graph replay" if args.graph else "eager stream launches",
        "order": args.order,
        "data": "synthetic",
        "config": {
            "workload": (f"{wl.name}: {wl.L}-layer GCN step on a {wl.n}-vertex Chung-Lu "
                         f"subgraph (exponent {wl.gamma}, mean degree {wl.dbar}), f_in "
                         f"{wl.f_in}, {wl.h} per branch, {wl.C} classes "
                         f"({'sigmoid BCE' if wl.loss else 'softmax CE'}), "
                         + (f"aggregation on the reduced graph ({wl.rounds} rounds, "
                            f"threshold {wl.theta})" if wl.reduce else "direct aggregation")),
            "n": wl.n, "nnz": int(red.dg.desc.nnz), "naux": i["naux"],
            "nnz_direct": int(i["stats"][0][2] + i["stats"][0][1]) if i["stats"] else
            int(red.dg.desc.nnz),
            "parallelism": "single GPU",
        },
        "roofline": {k: v for k, v in roof.items() if k != "kernel"} | {"kernel": dominant},
        "cpu_baseline": cpu,
        "direct_aggregation_ms_per_step": None if direct is None else round(direct, 4),
        "narrow_order_ms_per_step": None if narrow is None else round(narrow, 4),
        "adam_ms_per_step": None if adam is None else round(adam, 4),
        "host_preprocess_ms": {k: round(v, 2) for k, v in red.host_ms.items()},
        "aggregation_roofline": agg,
        "extra": extra,
        "kernels": {k: {kk: vv for kk, vv in v.items()
                        if kk not in ("flops_per_launch", "bytes_per_launch")}
                    for k, v in ktab.items()},
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
