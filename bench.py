"""Benchmark of the MI355X branch-verification step.

One step = sb_verify_forward (target forward over a B x k branch tree on a
shared prefix KV cache, LM head, softmax statistics) + sb_accept_resample
(the lossless accept/select/resample walk), on one GPU, inputs resident in
HBM.  Default workload: Llama-2-7B-shaped bf16 decoder (32 layers, hidden
4096, 32 heads x 128, FFN 11008, vocabulary 32000), prefix P = 2048,
B = 4 branches x k = 8 drafts (33 rows).

    python bench.py [--gpus 1] [--steps K] [--warmup W]

Prints one JSON line: verified tokens/s (B*k scored drafts per step), the
dominant kernel's HBM roofline fraction measured with HIP events inside
the timed steps, and the CPU oracle's throughput on a bounded sample of the
same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0   # MI355X HBM3E, vendor figure
MFMA_PEAK_TFS = 2500.0  # MI355X dense bf16 matrix-core peak, vendor figure
DOMINANT = "gate_up"    # kernel class holding the most bytes per step


COPY_BYTES = 1 << 29     # plain device copy used to scale the HBM byte counters
PMC_STEPS = 3            # timed steps of a counter run (--steps 3)
CPU_REPEATS = 2          # whole CPU oracle steps timed (about 15 s on 16 cores)
WORKLOAD = "llama7b_b4k8_p2048"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", f"traffic_gate_up_{WORKLOAD}.md")
# sources the dominant GEMM kernel is built from (its byte counters are
# stale once any of them changes)
GEMM_SOURCES = ("paper_2506_01979_amd/csrc/k_gemm.hip", "paper_2506_01979_amd/csrc/k_gemm_swiglu.hip",
                "paper_2506_01979_amd/csrc/sb_gemm_kernel.h", "paper_2506_01979_amd/csrc/sb_device.h",
                "paper_2506_01979_amd/csrc/sb_internal_fwd.h")
# kernels of one verify step, in launch order: embed, the layers, final
# norm, LM head, stats.  A layer is norm, QKV, attention, [attention merge],
# O, [post-attention norm, unless O applies it], gate/up, down.


def kernel_class(name: str, prev: str) -> str:
    """Class of a verify-step kernel from its name (prev: the class of the
    kernel before it, which tells the O projection from the down one)."""
    if "k_embed_meta" in name:
        return "embed"
    if "k_rmsnorm_pack" in name:
        return "norm"
    if "k_attn_merge" in name:
        return "attn_merge"
    if "k_attn" in name:
        return "attn"
    if "k_softmax_stats" in name:
        return "stats"
    if "k_walk" in name:
        return "accept_walk"
    if "k_rollback" in name:
        return "rollback"
    m = re.search(r"k_gemm(?:_wide)?<(\d+)", name)
    if m:
        epi = int(m.group(1))
        if epi in (1, 4):  # residual projections
            return "down" if prev == "gate_up" else "o"
        return {0: "qkv", 2: "gate_up", 3: "lm_head"}.get(epi, "gemm")
    return "other"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def gemm_source_sha() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in GEMM_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def _counter_rows(d):
    import csv
    import glob
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise FileNotFoundError(f"no counter_collection.csv under {d}")
    per = {}
    for f in files:
        for r in csv.DictReader(open(f)):
            key = int(r["Dispatch_Id"])
            e = per.setdefault(key, {"name": r["Kernel_Name"], "values": {}})
            e["values"][r["Counter_Name"]] = e["values"].get(r["Counter_Name"], 0.0) + \
                float(r["Counter_Value"])
    return [per[k] for k in sorted(per)]


def _step_dispatches(rows, last):
    """(class, record) of every dispatch of the last `last` complete verify
    steps (k_embed_meta .. k_softmax_stats; the timed ones, since earlier
    steps generate the drafts on partial trees)."""
    steps = []
    i = 0
    while i < len(rows):
        if "k_embed_meta" not in rows[i]["name"]:
            i += 1
            continue
        j = i + 1
        while j < len(rows) and "k_softmax_stats" not in rows[j]["name"] and \
                "k_embed_meta" not in rows[j]["name"]:
            j += 1
        if j < len(rows) and "k_softmax_stats" in rows[j]["name"]:
            prev, step = "", []
            for r in rows[i:j + 1]:
                prev = kernel_class(r["name"], prev)
                step.append((prev, r))
            steps.append(step)
        i = j
    return [x for st in steps[-last:] for x in st]


def _gate_up_dispatches(rows, n_layers, last):
    """Dispatch records of the gate/up GEMM in the last `last` complete verify
    steps."""
    out = [r for c, r in _step_dispatches(rows, last) if c == "gate_up"]
    if len(out) != last * n_layers:
        raise RuntimeError(f"expected {last * n_layers} gate/up launches, found {len(out)}")
    return out


def pmc_summary(fetch_dir: str, write_dir: str) -> str:
    """Markdown summary of two rocprofv3 --pmc runs of
    `bench.py --copy-calibration` (FETCH_SIZE, then WRITE_SIZE): HBM bytes
    per gate/up launch, each counter scaled by what it reads for the final
    device copy of COPY_BYTES bytes."""
    from paper_2506_01979_amd import synth
    shape = synth.WORKLOADS[WORKLOAD].shape
    res = {}
    for counter, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        rows = _counter_rows(d)
        gu = _gate_up_dispatches(rows, shape.n_layers, PMC_STEPS)
        copy = rows[-1]
        kib = sum(g["values"][counter] for g in gu) / len(gu)
        copy_kib = copy["values"][counter]
        res[counter] = {"kib_per_launch": kib, "launches": len(gu), "copy_kernel": copy["name"],
                        "copy_kib": copy_kib, "scale": COPY_BYTES / (copy_kib * 1024.0),
                        "kernel": gu[0]["name"]}
    f, w = res["FETCH_SIZE"], res["WRITE_SIZE"]
    fetch_b = f["kib_per_launch"] * 1024.0 * f["scale"]
    write_b = w["kib_per_launch"] * 1024.0 * w["scale"]
    nb = algorithmic_bytes(shape, synth.WORKLOADS[WORKLOAD].kv_len, synth.WORKLOADS[WORKLOAD].n_rows)
    rec = {"workload": WORKLOAD, "kernel": f["kernel"], "launches": f["launches"],
           "fetch_kib_per_launch": round(f["kib_per_launch"], 1),
           "write_kib_per_launch": round(w["kib_per_launch"], 1),
           "copy_bytes": COPY_BYTES, "copy_kernel": f["copy_kernel"],
           "copy_fetch_kib": round(f["copy_kib"], 1), "copy_write_kib": round(w["copy_kib"], 1),
           "fetch_scale": round(f["scale"], 4), "write_scale": round(w["scale"], 4),
           "traffic_bytes": int(fetch_b + write_b),
           "algorithmic_bytes": nb["gate_up_launch"],
           "gemm_source_sha256": gemm_source_sha()}
    cmd = ("cd /tmp && export TMPDIR=/tmp && "
           "rocprofv3 --pmc FETCH_SIZE --output-format csv -d <repo>/out/pmc_fetch -o run -- "
           "python3 <repo>/bench.py --steps 3 --warmup 1 --no-cpu-baseline --no-alpha-sweep "
           "--no-hrad --no-draft --no-graph --copy-calibration; the same with --pmc WRITE_SIZE into "
           "out/pmc_write; then "
           "python3 bench.py --pmc-summary out/pmc_fetch out/pmc_write")
    return "\n".join([
        f"# HBM traffic of the gate/up GEMM launch, {WORKLOAD}",
        "",
        f"Command: `{cmd}`",
        "",
        f"- kernel: `{f['kernel']}`, {f['launches']} launches (every layer of the last {PMC_STEPS} "
        f"timed steps)",
        f"- FETCH_SIZE {f['kib_per_launch']:.1f} KiB/launch, scale {f['scale']:.4f} "
        f"(copy of {COPY_BYTES} B reads {f['copy_kib']:.1f} KiB, `{f['copy_kernel']}`)",
        f"- WRITE_SIZE {w['kib_per_launch']:.1f} KiB/launch, scale {w['scale']:.4f} "
        f"(same copy writes {w['copy_kib']:.1f} KiB)",
        f"- traffic {(fetch_b + write_b) / 1e6:.2f} MB/launch vs algorithmic "
        f"{nb['gate_up_launch'] / 1e6:.2f} MB/launch",
        "",
        json.dumps(rec),
        ""])


def measured_traffic(workload: str):
    """HBM bytes per dominant launch from the committed counter summary, or
    None when there is none, it measured another workload, or the kernel
    sources changed since."""
    try:
        with open(TRAFFIC_FILE) as fh:
            line = [l for l in fh if l.startswith("{")][-1]
        rec = json.loads(line)
    except (OSError, IndexError, ValueError):
        return None
    if rec.get("gemm_source_sha256") != gemm_source_sha() or rec.get("workload") != workload:
        return None
    return rec["traffic_bytes"]


def trace_summary(trace_dir: str, workload: str = WORKLOAD) -> str:
    """Markdown per-kernel summary of a rocprofv3 --kernel-trace --stats run
    of bench.py: the whole-run stats table, then the kernels of the last 5
    complete verify steps in launch order."""
    import csv
    import glob
    stats = glob.glob(os.path.join(trace_dir, "**", "*kernel_stats.csv"), recursive=True)[0]
    trace = glob.glob(os.path.join(trace_dir, "**", "*kernel_trace.csv"), recursive=True)[0]
    rows = sorted(csv.DictReader(open(trace)), key=lambda r: int(r["Start_Timestamp"]))
    # a step: k_embed_meta .. k_softmax_stats, then the accept walk and the
    # rollback when they follow
    steps = []
    for i, r in enumerate(rows):
        if "k_embed_meta" not in r["Kernel_Name"]:
            continue
        j = i + 1
        while j < len(rows) and "k_softmax_stats" not in rows[j]["Kernel_Name"] and \
                "k_embed_meta" not in rows[j]["Kernel_Name"]:
            j += 1
        if j >= len(rows) or "k_softmax_stats" not in rows[j]["Kernel_Name"]:
            continue
        for tail in ("k_walk", "k_rollback"):
            if j + 1 < len(rows) and tail in rows[j + 1]["Kernel_Name"]:
                j += 1
        steps.append((i, j + 1))
    steps = steps[-5:]
    agg, span = {}, []
    for i, e in steps:
        span.append((int(rows[e - 1]["End_Timestamp"]) - int(rows[i]["Start_Timestamp"])) / 1e3)
        prev = ""
        for j in range(i, e):
            r = rows[j]
            d = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
            prev = kernel_class(r["Kernel_Name"], prev)
            a = agg.setdefault(prev, {"name": set(), "us": []})
            a["name"].add(r["Kernel_Name"].replace("sb::(anonymous namespace)::", ""))
            a["us"].append(d)
    wl = "" if workload == WORKLOAD else f" --workload {workload}"
    out = [f"# Kernel trace of the verify step, {workload}", "",
           "Command: `cd /tmp && export TMPDIR=/tmp && rocprofv3 --kernel-trace --stats "
           "--output-format csv -d <repo>/out/prof_step -o run -- python3 <repo>/bench.py "
           f"--steps 10 --warmup 3 --no-cpu-baseline --no-alpha-sweep --no-hrad --no-draft --no-graph{wl}`, "
           f"then `python3 bench.py --trace-summary out/prof_step{wl}`", "",
           f"Last {len(steps)} complete steps (embed .. stats, then the accept walk and the rollback "
           f"when traced): span "
           + ", ".join(f"{x:.1f}" for x in span) + " us", "",
           "| class | kernel | launches/step | avg us | min us | us/step |",
           "|---|---|---|---|---|---|"]
    tot = 0.0
    for c, a in sorted(agg.items(), key=lambda kv: -sum(kv[1]["us"])):
        per = sum(a["us"]) / len(steps)
        tot += per
        out.append(f"| {c} | `{', '.join(sorted(a['name']))}` | {len(a['us']) // len(steps)} | "
                   f"{sum(a['us']) / len(a['us']):.2f} | {min(a['us']):.2f} | {per:.1f} |")
    out += [f"| total | | | | | {tot:.1f} |", "", "Whole-run `--stats` (all launches, incl. "
            "draft generation and warmup):", "", "| kernel | calls | avg us | min us | max us | % |",
            "|---|---|---|---|---|---|"]
    for r in list(csv.DictReader(open(stats)))[:16]:
        out.append(f"| `{r['Name'].replace('sb::(anonymous namespace)::', '')[:70]}` | {r['Calls']} | "
                   f"{float(r['AverageNs']) / 1e3:.2f} | {float(r['MinNs']) / 1e3:.2f} | "
                   f"{float(r['MaxNs']) / 1e3:.2f} | {float(r['Percentage']):.2f} |")
    return "\n".join(out) + "\n"


def draft_trace_summary(trace_dir: str) -> str:
    """Markdown summary of the draft side in a rocprofv3 --kernel-trace
    --stats run of bench.py: the draft-side kernels' whole-run stats, then one
    drafting round broken down by kernel (the windows between consecutive
    branch-point launches of the timed rounds, each holding one round's
    continuation steps and the next round's root step)."""
    import collections
    import csv
    import glob
    import re
    stats = glob.glob(os.path.join(trace_dir, "**", "*kernel_stats.csv"), recursive=True)[0]
    trace = glob.glob(os.path.join(trace_dir, "**", "*kernel_trace.csv"), recursive=True)[0]
    rows = sorted(csv.DictReader(open(trace)), key=lambda r: int(r["Start_Timestamp"]))
    short = lambda n: (re.search(r"(k_[A-Za-z0-9_]+)", n) or re.search(r"(\S+)", n)).group(1)
    sel = [i for i, r in enumerate(rows) if "k_branch_select" in r["Kernel_Name"]]
    # the timed rounds: the 3rd .. 22nd branch-point launches (two warmup rounds first)
    wins = [(sel[j], sel[j + 1]) for j in range(2, min(21, len(sel) - 1))]
    agg = collections.defaultdict(list)
    spans, busy = [], []
    for a, b in wins:
        per = collections.Counter()
        for r in rows[a:b]:
            per[short(r["Kernel_Name"])] += (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        for k, v in per.items():
            agg[k].append(v)
        spans.append((int(rows[b]["Start_Timestamp"]) - int(rows[a]["Start_Timestamp"])) / 1e3)
        busy.append(sum(per.values()))
    counts = collections.Counter(short(r["Kernel_Name"]) for r in rows[wins[0][0]:wins[0][1]])
    out = ["# Kernel trace of the draft side: 68M draft round (k_max 4, depth 8, prefix 2048), "
           "branch-point candidates and draft sampler", "",
           "Command: `cd /tmp && export TMPDIR=/tmp && rocprofv3 --kernel-trace --stats "
           "--output-format csv -d <repo>/out/prof_draft -o run -- python3 <repo>/bench.py "
           "--steps 10 --warmup 3 --no-cpu-baseline --no-alpha-sweep --no-hrad --no-graph`, then "
           "`python3 bench.py --draft-trace-summary out/prof_draft`", "",
           f"One round ({len(wins)} rounds): kernel time {sum(busy) / len(busy):.1f} us, "
           f"span under the tracer {sum(spans) / len(spans):.1f} us", "",
           "| kernel | launches/round | us/round | avg us |", "|---|---|---|---|"]
    for k, v in sorted(agg.items(), key=lambda kv: -sum(kv[1])):
        per = sum(v) / len(wins)
        out.append(f"| `{k}` | {counts[k]} | {per:.1f} | {per / max(1, counts[k]):.2f} |")
    out += ["", "Whole-run `--stats` of the draft-side kernels (rounds, the candidate and sampler "
            "timing loops, the overlap runs):", "",
            "| kernel | calls | avg us | min us | max us |", "|---|---|---|---|---|"]
    for r in csv.DictReader(open(stats)):
        if re.search(r"k_branch_|k_draft_", r["Name"]):
            out.append(f"| `{short(r['Name'])}` | {r['Calls']} | "
                       f"{float(r['AverageNs']) / 1e3:.2f} | {float(r['MinNs']) / 1e3:.2f} | "
                       f"{float(r['MaxNs']) / 1e3:.2f} |")
    return "\n".join(out) + "\n"


def algorithmic_bytes(shape, P_kv: int, n: int) -> dict:
    """Bytes the verify step must move at least once (bf16 weights read once,
    prefix KV read once, tree KV written, fp32 logits written and read)."""
    H, F, V, L = shape.hidden, shape.ffn, shape.vocab, shape.n_layers
    qd, kvd = shape.q_dim, shape.kv_dim
    per_layer_w = (H * (qd + 2 * kvd) + qd * H + 3 * H * F) * 2 + 2 * H * 4
    weights = L * per_layer_w + V * H * 2 + H * 4 + n * H * 2
    prefix_kv = L * 2 * P_kv * kvd * 2
    tree_kv = L * 2 * n * kvd * 2
    logits = n * V * 4 * 2
    gate_up = 2 * F * H * 2 + n * H * 2 + n * F * 2
    return {"step": weights + prefix_kv + tree_kv + logits, "weights": weights,
            "prefix_kv": prefix_kv, "gate_up_launch": gate_up}


def class_bytes(shape, P_kv: int, n: int, split_down: int = 4) -> dict:
    """Algorithmic bytes of one launch per kernel class (the weight or KV
    stream it must read once, plus its activation inputs and outputs)."""
    H, F, V = shape.hidden, shape.ffn, shape.vocab
    qd, kvd = shape.q_dim, shape.kv_dim
    return {
        "qkv": H * (qd + 2 * kvd) * 2 + n * H * 2 + n * (qd + 2 * kvd) * 2,
        "o": qd * H * 2 + n * qd * 2 + n * H * 4 * 2 + n * H * 2,
        "gate_up": 2 * F * H * 2 + n * H * 2 + n * F * 2,
        "down": F * H * 2 + n * F * 2 + split_down * n * H * 4,
        "lm_head": V * H * 2 + n * H * 2 + n * V * 4,
        "attn": 2 * (P_kv + n) * kvd * 2 + n * qd * 2,
    }


def counter_summary(fetch_dir: str, write_dir: str, mfma_dir: str, workload: str = WORKLOAD) -> str:
    """Markdown summary of three rocprofv3 --pmc runs of `bench.py
    --copy-calibration` (FETCH_SIZE; WRITE_SIZE; SQ_VALU_MFMA_BUSY_CYCLES,
    SQ_INSTS_VALU_MFMA_MOPS_BF16, GRBM_GUI_ACTIVE with --kernel-trace): per
    kernel class of the last timed steps, HBM bytes per launch (each counter
    scaled by what it reads for the final device copy of COPY_BYTES bytes)
    against the class's algorithmic bytes, and the matrix cores' busy share
    and bf16 FLOPs."""
    import csv
    import glob
    from paper_2506_01979_amd import synth
    w = synth.WORKLOADS[workload]
    shape = w.shape
    per = {}
    scales = {}
    for counter, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        rows = _counter_rows(d)
        copy = rows[-1]
        if "copy" not in copy["name"].lower():
            raise RuntimeError(f"last dispatch of {d} is not the calibration copy: {copy['name']}")
        scales[counter] = (COPY_BYTES / (copy["values"][counter] * 1024.0), copy["name"],
                           copy["values"][counter])
        for c, r in _step_dispatches(rows, PMC_STEPS):
            per.setdefault(c, {}).setdefault(counter, []).append(r["values"][counter])
    rows = _counter_rows(mfma_dir)
    names = {}
    for c, r in _step_dispatches(rows, PMC_STEPS):
        e = per.setdefault(c, {})
        for k in ("SQ_VALU_MFMA_BUSY_CYCLES", "SQ_INSTS_VALU_MFMA_MOPS_BF16", "GRBM_GUI_ACTIVE"):
            e.setdefault(k, []).append(r["values"].get(k, 0.0))
        names[c] = r["name"].replace("sb::(anonymous namespace)::", "")
    # kernel durations of the counter run (--kernel-trace in the same pass)
    dur = {}
    trace = glob.glob(os.path.join(mfma_dir, "**", "*kernel_trace.csv"), recursive=True)
    if trace:
        tr = sorted(csv.DictReader(open(trace[0])), key=lambda r: int(r["Start_Timestamp"]))
        recs = [{"name": r["Kernel_Name"], "d": (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3}
                for r in tr]
        for c, r in _step_dispatches(recs, PMC_STEPS):
            dur.setdefault(c, []).append(r["d"])
    simds = 4 * 256
    cb = class_bytes(shape, w.kv_len, w.n_rows)
    mean = lambda xs: sum(xs) / len(xs) if xs else float("nan")
    out = [f"# Hardware counters per kernel class of the verify step, {workload}", "",
           "Commands (each its own run): `cd /tmp && export TMPDIR=/tmp && rocprofv3 --pmc FETCH_SIZE "
           "--output-format csv -d <repo>/out/pmc_fetch -o run -- python3 <repo>/bench.py --steps 3 "
           "--warmup 1 --no-cpu-baseline --no-alpha-sweep --no-hrad --no-draft --no-graph "
           "--copy-calibration`; the same with `--pmc WRITE_SIZE` into out/pmc_write; the same with "
           "`--kernel-trace --pmc SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_VALU_MFMA_MOPS_BF16 GRBM_GUI_ACTIVE` "
           "into out/pmc_mfma; then `python3 bench.py --counter-summary out/pmc_fetch out/pmc_write "
           "out/pmc_mfma`.", "",
           f"HBM bytes: FETCH_SIZE and WRITE_SIZE (KiB per dispatch) times the factor that makes a "
           f"plain device copy of {COPY_BYTES} bytes read and write that many "
           f"(FETCH x {scales['FETCH_SIZE'][0]:.4f}, WRITE x {scales['WRITE_SIZE'][0]:.4f}; "
           f"copy kernel `{scales['FETCH_SIZE'][1]}`).  Matrix-core work: bf16 MFMA FLOPs = "
           "SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512 per launch (padded token rows included; the "
           "attention's P.V product counts twice, hi and lo parts), over the launch's duration in "
           f"the same run: the MFMA utilisation is that rate against the dense bf16 peak "
           f"({MFMA_PEAK_TFS:.0f} TFLOP/s).  Busy share: SQ_VALU_MFMA_BUSY_CYCLES / "
           f"(GRBM_GUI_ACTIVE / 8 XCDs x {simds} SIMDs) (the counter file sums GRBM_GUI_ACTIVE over "
           "the 8 XCDs).  The counter run serialises kernels, so its durations, and the rates, "
           "are a little below the untraced run's.", "",
           "| class | launches/step | HBM read MB | HBM write MB | algorithmic MB | traffic / algorithmic "
           "| bf16 MFMA GFLOP per launch | TFLOP/s | MFMA utilisation % | MFMA busy % |",
           "|---|---|---|---|---|---|---|---|---|---|"]
    recs = {}
    order = ["qkv", "attn", "attn_merge", "o", "norm", "gate_up", "down", "lm_head", "stats", "embed"]
    for c in order:
        e = per.get(c)
        if not e or "FETCH_SIZE" not in e:
            continue
        n_l = len(e["FETCH_SIZE"]) / PMC_STEPS
        rd = mean(e["FETCH_SIZE"]) * 1024 * scales["FETCH_SIZE"][0]
        wr = mean(e["WRITE_SIZE"]) * 1024 * scales["WRITE_SIZE"][0]
        busy = mean([b / (g / 8 * simds) * 100 if g else 0.0 for b, g in
                     zip(e.get("SQ_VALU_MFMA_BUSY_CYCLES", []), e.get("GRBM_GUI_ACTIVE", []))])
        flops = mean(e.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", [])) * 512
        d = mean(dur.get(c, []))
        tfs = flops / (d * 1e-6) / 1e12 if d == d and d > 0 else float("nan")
        alg = cb.get(c)
        ratio = (rd + wr) / alg if alg else None
        out.append(f"| {c} | {n_l:.0f} | {rd / 1e6:.2f} | {wr / 1e6:.2f} | "
                   f"{alg / 1e6:.2f} | {ratio:.3f} | " if alg else
                   f"| {c} | {n_l:.0f} | {rd / 1e6:.2f} | {wr / 1e6:.2f} | — | — | ")
        util = tfs / MFMA_PEAK_TFS * 100 if tfs == tfs else float("nan")
        out[-1] += f"{flops / 1e9:.2f} | {tfs:.1f} | {util:.2f} | {busy:.2f} |"
        recs[c] = {"read_bytes": int(rd), "write_bytes": int(wr), "algorithmic_bytes": alg,
                   "bf16_flops": int(flops), "tflops": round(tfs, 2) if tfs == tfs else None,
                   "mfma_util_pct": round(util, 3) if util == util else None,
                   "mfma_busy_pct": round(busy, 3),
                   "duration_us_counter_run": round(d, 2) if d == d else None}
    out += ["", "Kernels: " + "; ".join(f"{c} `{names[c]}`" for c in order if c in names), "",
            json.dumps({"workload": workload, "classes": recs, "gemm_source_sha256": gemm_source_sha()}), ""]
    return "\n".join(out)


def partial_tree(parents, depth: int):
    """Rows of the tree with depth < `depth`, in ascending row order, with
    parents re-indexed; returns (rows, parents)."""
    from paper_2506_01979_amd import synth

    dep = synth.tree_depths(np.asarray(parents))
    rows = [i for i in range(len(parents)) if dep[i] < depth]
    pos = {r: i for i, r in enumerate(rows)}
    return rows, [-1] + [pos[int(parents[r])] for r in rows[1:]]


def make_drafts(api, synth, m, k_, v_, kv_len, root_tok, parents, alpha, q_temp, seed):
    """Drafts generated depth by depth over the tree `parents`: q = alpha *
    p_target + (1 - alpha) * softmax(N(0,1)/q_temp) of the parent's target
    row; the children of one row are i.i.d. draws from one q."""
    import torch

    V = m.shape.vocab
    n = len(parents)
    dep = synth.tree_depths(np.asarray(parents))
    first = {}
    for i in range(1, n):
        first.setdefault(int(parents[i]), i)
    g = np.random.default_rng(seed)
    qrand = synth.softmax_rows(synth.random_logits(n, V, 1.0 / q_temp, seed=seed + 7))
    tokens = np.zeros(n, dtype=np.int32)
    tokens[0] = root_tok
    q = np.zeros((n, V), dtype=np.float32)
    for depth in range(1, int(dep.max()) + 1):
        rows, par = partial_tree(parents, depth)
        nr = len(rows)
        logits = torch.empty((nr, V), dtype=torch.float32, device="cuda")
        stats = api.new_stats(nr)
        m.sb_verify_forward(k_, v_, kv_len, torch.from_numpy(tokens[rows]).cuda(), par, 1.0,
                            logits, stats, m.workspace(nr, kv_len))
        lg = logits.cpu().numpy().astype(np.float64)
        lg -= lg.max(axis=1, keepdims=True)
        p = np.exp(lg)
        p /= p.sum(axis=1, keepdims=True)
        for row in range(1, n):
            if dep[row] != depth:
                continue
            parent = int(parents[row])
            pr = p[rows.index(parent)]
            qr = qrand[first[parent]]   # siblings share one q
            qq = alpha * pr + (1 - alpha) * qr.astype(np.float64)
            qq /= qq.sum()
            q[row] = qq.astype(np.float32)
            tokens[row] = g.choice(V, p=qq)
    return tokens, q


class _PerLayer:
    """Read-only sequence whose items are built when indexed (the oracle walks
    the layers in order, so one layer's float32 copy is alive at a time)."""

    def __init__(self, n, make):
        self.n, self.make = n, make

    def __len__(self):
        return self.n

    def __getitem__(self, i):
        if not 0 <= i < self.n:
            raise IndexError(i)
        return self.make(i)


def cpu_baseline(shape, host_bits, kv_host, kv_len, inp, n_layers_sample: int) -> dict:
    """The oracle as it stands, on the host cores: its bf16-emulation forward
    of the same model on the same inputs (embedding, n_layers_sample decoder
    layers, final norm, LM head) and its accept walk.  With every layer
    sampled (the default) this is one whole verify step; with fewer, the
    per-layer time is extrapolated to the full depth."""
    from oracle import decoder, sampling
    from paper_2506_01979_amd import synth

    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        cores = len(os.sched_getaffinity(0))

    def layer(l):
        lw = {n: synth.bits_to_f32(host_bits[(n, l)]) for n in synth.LAYER_MATS}
        lw["attn_norm"] = synth.norm_gain(shape)
        lw["mlp_norm"] = synth.norm_gain(shape)
        return lw

    def weights(nl):
        return {"embed": synth.bits_to_f32(host_bits[("embed", None)]),
                "lm_head": synth.bits_to_f32(host_bits[("lm_head", None)]),
                "final_norm": synth.norm_gain(shape), "layers": _PerLayer(nl, layer)}

    Kp = _PerLayer(n_layers_sample, lambda l: synth.bits_to_f32(kv_host[l][0]))
    Vp = _PerLayer(n_layers_sample, lambda l: synth.bits_to_f32(kv_host[l][1]))
    full = n_layers_sample >= shape.n_layers
    reps = CPU_REPEATS if full else 1
    times = {}
    for nl in ((n_layers_sample,) if full else (0, n_layers_sample)):
        sh = shape.with_layers(nl)   # 0 layers: embedding, final norm, LM head only
        W = weights(nl)
        fwd = walk = 0.0
        for _ in range(reps):
            t0 = time.perf_counter()
            lg, _, _ = decoder.tree_forward(sh, W, Kp, Vp, kv_len, inp["tokens"], inp["parents"],
                                            "bf16")
            t1 = time.perf_counter()
            sampling.accept_resample(inp["tokens"], inp["parents"], lg.astype(np.float32), 1.0,
                                     inp["q"], inp["u"])
            t2 = time.perf_counter()
            fwd += (t1 - t0) / reps
            walk += (t2 - t1) / reps
        times[nl] = (fwd, walk)
        del W
    n_draft = len(inp["parents"]) - 1
    if full:
        fwd, walk = times[n_layers_sample]
        step_s = fwd + walk
        sample = (f"{reps} whole verify steps on the host, averaged: the oracle's bf16-emulation "
                  f"forward of all {shape.n_layers} layers (+ embedding, final norm, LM head) "
                  f"{fwd:.2f}s and its accept walk {walk:.3f}s per step, same weights, prefix KV, "
                  f"tree, q and u as the GPU step")
    else:
        head, walk = times[0]
        per_layer = max(0.0, times[n_layers_sample][0] - head) / n_layers_sample
        step_s = head + walk + per_layer * shape.n_layers
        sample = (f"oracle bf16-emulation forward of layers 0..{n_layers_sample - 1} of "
                  f"{shape.n_layers} (+ embedding, final norm, LM head) and the accept walk "
                  f"on the same inputs; step time = head {head:.2f}s + walk {walk:.3f}s + "
                  f"{shape.n_layers} x per-layer {per_layer:.2f}s")
    return {"value": n_draft / step_s, "unit": "verified tokens/s", "cores": int(cores),
            "kind": "oracle", "sample": sample, "step_s": step_s}


SWEEP_PREFIXES = (512, 4096, 8192)
SWEEP_TREES = [(b, k) for b in (1, 2, 4, 8) for k in (4, 8, 16)]


def run_sweep(args, api, synth, m, shape, dev) -> None:
    """One model, every (prefix, B, k) of the sweep: the prefix KV (seeded
    N(0,1) bf16) filled once for the longest prefix and read in part for the
    shorter ones; per configuration drafts mixed at --alpha, warmup, then
    --steps timed verify steps (forward + accept walk + rollback).  Prints
    one JSON line per configuration, then a markdown table."""
    import torch
    p_max = max(SWEEP_PREFIXES)
    n_max = 1 + max(b * k for b, k in SWEEP_TREES)
    k_, v_ = m.new_kv(p_max + n_max + 16)
    t0 = time.time()
    for l in range(shape.n_layers):
        kb = synth.synthetic_kv(shape, l, p_max - 1, p_max - 1, 0, as_bits=True)
        vb = synth.synthetic_kv(shape, l, p_max - 1, p_max - 1, 1, as_bits=True)
        k_[l, :, :p_max - 1] = torch.from_numpy(kb.view(np.int16)).view(torch.bfloat16).to(dev)
        v_[l, :, :, :p_max - 1] = torch.from_numpy(vb.view(np.int16)).view(torch.bfloat16).to(dev).transpose(1, 2)
    log(f"prefix KV ready ({p_max - 1} slots) in {time.time() - t0:.1f}s")
    stream = torch.cuda.current_stream()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    rows = []
    for P in SWEEP_PREFIXES:
        kv_len = P - 1
        root = int(synth.prefix_tokens(shape.vocab, P)[-1])
        for B, kd in SWEEP_TREES:
            parents = synth.branch_parents(B, kd)
            n = len(parents)
            tokens, q = make_drafts(api, synth, m, k_, v_, kv_len, root, parents, args.alpha,
                                    0.7, 11)
            d_tok = torch.from_numpy(tokens).to(dev)
            d_q = torch.from_numpy(q).to(dev)
            d_u = torch.from_numpy(synth.uniforms(n, 1)).to(dev)
            logits = torch.empty((n, shape.vocab), dtype=torch.float32, device=dev)
            stats = api.new_stats(n, dev)
            ws = m.workspace(n, kv_len)
            sws = torch.empty(api.sb_sample_workspace_bytes(shape.vocab), dtype=torch.uint8,
                              device=dev)
            res = api.new_result(dev)
            new_len = torch.zeros(1, dtype=torch.int32, device=dev)

            def step():
                m.sb_verify_forward(k_, v_, kv_len, d_tok, parents, 1.0, logits, stats, ws, stream)
                api.sb_accept_resample(d_tok, parents, logits, stats, 1.0, d_q, d_u, res, sws,
                                       stream)
                m.sb_kv_rollback(k_, v_, kv_len, res, new_len, stream)
            for _ in range(args.warmup):
                step()
            torch.cuda.synchronize()
            ev0.record(stream)
            for _ in range(args.steps):
                step()
            ev1.record(stream)
            torch.cuda.synchronize()
            ms = ev0.elapsed_time(ev1) / args.steps
            nb = algorithmic_bytes(shape, kv_len, n)["step"]
            r = api.decode_result(res)
            rec = {"workload": f"{shape.name} B={B} k={kd} prefix {P}", "prefix": P,
                   "branches": B, "depth": kd, "rows": n, "ms_per_step": round(ms, 4),
                   "verified_tokens_per_s": round((n - 1) / (ms * 1e-3), 1),
                   "step_bytes": nb, "step_hbm_frac": round(nb / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                   "accepted": r["n_accepted"], "alpha": args.alpha}
            rows.append(rec)
            print(json.dumps(rec), flush=True)
            del ws, logits
    out = [f"| prefix | B | k | rows | ms/step | verified tok/s | GB/step | step HBM fraction |",
           "|---|---|---|---|---|---|---|---|"]
    for r in rows:
        out.append(f"| {r['prefix']} | {r['branches']} | {r['depth']} | {r['rows']} | "
                   f"{r['ms_per_step']:.3f} | {r['verified_tokens_per_s']:.0f} | "
                   f"{r['step_bytes'] / 1e9:.2f} | {r['step_hbm_frac']:.3f} |")
    print("\n".join(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=WORKLOAD)
    ap.add_argument("--alpha", type=float, default=0.6)
    ap.add_argument("--tree", choices=("branch", "fork"), default="branch",
                    help="branch: the workload's B x k branches off the root; fork: a chain "
                         "of --trunk drafts, then B branches of --fork-depth drafts")
    ap.add_argument("--trunk", type=int, default=4)
    ap.add_argument("--fork-depth", type=int, default=7)
    ap.add_argument("--cpu-layers", type=int, default=0,
                    help="decoder layers the CPU oracle runs (0: all of them)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-alpha-sweep", action="store_true")
    ap.add_argument("--no-graph", action="store_true",
                    help="skip the HIP-graph replay measurement")
    ap.add_argument("--no-hrad", action="store_true",
                    help="skip the H-RAD measurement (feature tap + predictor)")
    ap.add_argument("--no-draft", action="store_true",
                    help="skip the draft-side measurement (68M draft round, candidates, sampler)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="end with a device copy of known size (for rocprofv3 --pmc runs)")
    ap.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="summarise two rocprofv3 --pmc runs of this script and exit")
    ap.add_argument("--counter-summary", nargs=3, metavar=("FETCH_DIR", "WRITE_DIR", "MFMA_DIR"),
                    help="per-class summary of three rocprofv3 --pmc runs of this script and exit")
    ap.add_argument("--draft-trace-summary", metavar="TRACE_DIR",
                    help="print the draft-side summary of a rocprofv3 kernel trace and exit")
    ap.add_argument("--trace-summary", metavar="TRACE_DIR",
                    help="summarise a rocprofv3 --kernel-trace --stats run of this script and exit")
    ap.add_argument("--sweep", action="store_true",
                    help="time the workload's shape over prefixes 512 / 4096 / 8192 and "
                         "B in {1, 2, 4, 8} x k in {4, 8, 16} (one JSON line per configuration, "
                         "then a markdown table) and exit")
    args = ap.parse_args()
    if args.pmc_summary:
        print(pmc_summary(*args.pmc_summary))
        return
    if args.counter_summary:
        print(counter_summary(*args.counter_summary, args.workload))
        return
    if args.trace_summary:
        print(trace_summary(args.trace_summary, args.workload))
        return
    if args.draft_trace_summary:
        print(draft_trace_summary(args.draft_trace_summary), end="")
        return

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print(json.dumps({"error": "this build runs on one GPU; --gpus must be 1"}), flush=True)
        sys.exit(2)

    import torch

    from paper_2506_01979_amd import api, synth

    w = synth.WORKLOADS[args.workload]
    shape = w.shape
    if args.cpu_layers <= 0 or args.cpu_layers > shape.n_layers:
        args.cpu_layers = shape.n_layers
    B, kd, P = w.branches, w.depth, w.prefix
    if args.tree == "fork":
        parents = synth.fork_parents(args.trunk, B, args.fork_depth)
        tree_desc = f"chain of {args.trunk} + fork of B={B} x {args.fork_depth} drafts"
    else:
        parents = synth.branch_parents(B, kd)
        tree_desc = f"B={B} branches x k={kd} drafts"
    kv_len, n = w.kv_len, len(parents)
    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")

    t0 = time.time()
    host_bits = {}

    def tensor_fn(name, layer=None):
        if name.endswith("norm"):
            return synth.norm_gain(shape)
        bits = synth.weight(shape, name, layer, 0, as_bits=True)
        if not args.no_cpu_baseline and (layer is None or layer < args.cpu_layers):
            host_bits[(name, layer)] = bits
        return bits

    m = api.Model(shape, tensor_fn, device=dev)
    log(f"weights generated, uploaded and packed in {time.time() - t0:.1f}s")
    if args.sweep:
        run_sweep(args, api, synth, m, shape, dev)
        return

    def fill_prefix(shp, kb_, vb_, keep=None):
        for l in range(shp.n_layers):
            kb = synth.synthetic_kv(shp, l, kv_len, kv_len, 0, as_bits=True)
            vb = synth.synthetic_kv(shp, l, kv_len, kv_len, 1, as_bits=True)
            kb_[l, :, :kv_len] = torch.from_numpy(kb.view(np.int16)).view(torch.bfloat16).to(dev)
            vb_[l, :, :, :kv_len] = torch.from_numpy(vb.view(np.int16)).view(torch.bfloat16).to(dev).transpose(1, 2)
            if keep is not None and l < args.cpu_layers:
                keep[l] = (kb, vb)

    cap = kv_len + n + 16
    k_, v_ = m.new_kv(cap)
    kv_host = {}
    fill_prefix(shape, k_, v_, kv_host)
    log(f"prefix KV ready ({kv_len} slots) at {time.time() - t0:.1f}s")

    root = int(synth.prefix_tokens(shape.vocab, P)[-1])
    tokens, q = make_drafts(api, synth, m, k_, v_, kv_len, root, parents, args.alpha, w.q_temp, 11)
    u = synth.uniforms(n, 1)
    inp = {"tokens": tokens, "parents": parents, "q": q, "u": u}

    d_tok = torch.from_numpy(tokens).to(dev)
    d_q = torch.from_numpy(q).to(dev)
    d_u = torch.from_numpy(u).to(dev)
    logits = torch.empty((n, shape.vocab), dtype=torch.float32, device=dev)
    stats = api.new_stats(n, dev)
    ws = m.workspace(n, kv_len)
    sws = torch.empty(api.sb_sample_workspace_bytes(shape.vocab), dtype=torch.uint8, device=dev)
    res = api.new_result(dev)
    stream = torch.cuda.current_stream()

    new_len = torch.zeros(1, dtype=torch.int32, device=dev)

    def step(st=None):
        # a0-a8: tree metadata ... LM head + stats, the accept walk, and the
        # rollback that compacts the kept path behind the prefix (it moves
        # tree slots only, which the next step's forward rewrites)
        st = st or stream
        m.sb_verify_forward(k_, v_, kv_len, d_tok, parents, 1.0, logits, stats, ws, st)
        api.sb_accept_resample(d_tok, parents, logits, stats, 1.0, d_q, d_u, res, sws, st)
        m.sb_kv_rollback(k_, v_, kv_len, res, new_len, st)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # the timed steps: K steps between two events, nothing else enqueued
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    ms_per_step = ev0.elapsed_time(ev1) / args.steps

    # per-step times (an event pair around each step: their median) and the
    # step without the rollback (forward + accept walk, the verify-and-accept
    # time), each over K more steps
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    torch.cuda.synchronize()
    for e0, e1 in evs:
        e0.record(stream)
        step()
        e1.record(stream)
    torch.cuda.synchronize()
    ms_median = float(np.median([e0.elapsed_time(e1) for e0, e1 in evs]))

    def step_no_rollback():
        m.sb_verify_forward(k_, v_, kv_len, d_tok, parents, 1.0, logits, stats, ws, stream)
        api.sb_accept_resample(d_tok, parents, logits, stats, 1.0, d_q, d_u, res, sws, stream)
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(args.steps):
        step_no_rollback()
    ev1.record(stream)
    torch.cuda.synchronize()
    ms_no_rollback = ev0.elapsed_time(ev1) / args.steps

    # the same K steps again with HIP events around every launch of the
    # dominant kernel (its average duration for the roofline); the events
    # cost time of their own, so this loop is not the step time
    m.sb_timer_start(DOMINANT, args.steps * shape.n_layers)
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    evented_ms = ev0.elapsed_time(ev1) / args.steps
    k_ms, k_launches = m.sb_timer_stop()

    r = api.decode_result(res)
    if int(new_len.item()) != kv_len + 1 + r["n_accepted"]:
        raise RuntimeError("rollback length does not match the accepted path")

    # The same step captured once in a HIP graph and replayed (kernel
    # arguments, including kv_len and the tree, are fixed in the graph).
    graph_ms = None
    if not args.no_graph:
        gs = torch.cuda.Stream()
        gs.wait_stream(stream)
        with torch.cuda.stream(gs):
            step(gs)            # warm outside the capture
        gs.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=gs):
            step(gs)
        graph.replay()
        torch.cuda.synchronize()
        ev0.record(stream)
        for _ in range(args.steps):
            graph.replay()
        ev1.record(stream)
        torch.cuda.synchronize()
        graph_ms = ev0.elapsed_time(ev1) / args.steps
        rg = api.decode_result(res)
        if rg != r:
            raise RuntimeError("graph replay changed the step's result")

    # H-RAD (Section "H-RAD"): the step again with the last 4 layers' hidden
    # states tapped, and the predictor on the walk's result (random MLP
    # weights: the trained ones are not available).  Not part of `value`.
    hrad_out = None
    if not args.no_hrad:
        HK = 4
        taps = torch.empty((HK, n, shape.hidden), dtype=torch.float32, device=dev)
        m.sb_model_set_tap(taps, HK, n)
        torch.cuda.synchronize()
        ev0.record(stream)
        for _ in range(args.steps):
            step()
        ev1.record(stream)
        torch.cuda.synchronize()
        tap_ms = ev0.elapsed_time(ev1) / args.steps
        m.sb_model_set_tap(None)
        gw = np.random.default_rng(5)
        din = (HK + 1) * shape.hidden
        hw = {"w1": gw.standard_normal((256, din)) / np.sqrt(din), "b1": gw.standard_normal(256) * 0.1,
              "w2": gw.standard_normal((64, 256)) / 16.0, "b2": gw.standard_normal(64) * 0.1,
              "w3": gw.standard_normal((3, 64)) / 8.0, "b3": gw.standard_normal(3) * 0.1}
        hw = {key: torch.from_numpy(val.astype(np.float32)).to(dev) for key, val in hw.items()}
        hws = torch.empty(api.lib.sb_hrad_workspace_bytes(), dtype=torch.uint8, device=dev)
        lg3 = torch.empty(3, dtype=torch.float32, device=dev)
        cls = torch.empty(1, dtype=torch.int32, device=dev)
        for _ in range(3):
            m.sb_hrad_predict(taps, HK, n, res, hw, lg3, cls, hws, stream)
        reps = 100
        torch.cuda.synchronize()
        ev0.record(stream)
        for _ in range(reps):
            m.sb_hrad_predict(taps, HK, n, res, hw, lg3, cls, hws, stream)
        ev1.record(stream)
        torch.cuda.synchronize()
        hrad_out = {"k_layers": HK, "ms_per_step_with_tap": round(tap_ms, 4),
                    "predict_us": round(ev0.elapsed_time(ev1) * 1e3 / reps, 2),
                    "w1_bytes": 256 * din * 4, "class": int(cls.item())}
        del taps

    # The draft side (Section "Branch Resampling"): one drafting round of the
    # 68M draft on its own prefix cache of the same length, k_max = B and
    # depth k (a near-flat q at the branch point gives the verify step's B),
    # then the branch-point candidates and the draft sampler on their own.
    # Not part of `value`.
    draft_out = round_out = None
    if not args.no_draft:
        dshape = synth.SHAPES["draft68m"]
        dm = api.Model(dshape, api.synth_tensors(dshape, seed=1), device=dev)
        DK, DD = B, kd
        R = 1 + DK * DD
        TRUNK = 4
        dk_, dv_ = dm.new_kv(kv_len + max(R, TRUNK + (B + 1) * DD) + 8)
        fill_prefix(dshape, dk_, dv_)
        du = torch.from_numpy(synth.uniforms(R, 31)).to(dev)
        dtok = torch.full((R,), root, dtype=torch.int32, device=dev)
        dq = torch.empty((R, dshape.vocab), dtype=torch.float32, device=dev)
        dws = dm.draft_round_workspace(DK, DD, kv_len)

        def draft_round():
            return dm.sb_draft_round(dk_, dv_, kv_len, DK, "wor", DD, 1.0, du, dtok, dq, dws, stream)
        for _ in range(2):
            draft_round()
        torch.cuda.synchronize()
        reps = 20
        ev0.record(stream)
        for _ in range(reps):
            bd, _, _ = draft_round()
        ev1.record(stream)
        torch.cuda.synchronize()
        round_ms = ev0.elapsed_time(ev1) / reps
        V = dshape.vocab
        cq = dq[0].contiguous()
        cxb = dtok[1:2].clone()
        ccount = torch.empty(1, dtype=torch.int32, device=dev)
        ctok = torch.empty(16, dtype=torch.int32, device=dev)
        crows = torch.empty((16, V), dtype=torch.float32, device=dev)
        cws = torch.empty(api.sb_branch_workspace_bytes(), dtype=torch.uint8, device=dev)
        cu = torch.from_numpy(synth.uniforms(16, 32)).to(dev)
        # device time per call: 50 calls captured in a HIP graph and replayed
        # (the Python binding's own cost per call is larger than the kernels')
        def graph_us(call, reps=50, replays=10):
            gs = torch.cuda.Stream()
            gs.wait_stream(stream)
            with torch.cuda.stream(gs):
                call(gs)
            gs.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=gs):
                for _ in range(reps):
                    call(gs)
            g.replay()
            torch.cuda.synchronize()
            ev0.record(stream)
            for _ in range(replays):
                g.replay()
            ev1.record(stream)
            torch.cuda.synchronize()
            return round(ev0.elapsed_time(ev1) * 1e3 / (reps * replays), 2)
        cand_us = {}
        for mode in ("topk", "iid", "wor"):
            cand_us[mode] = graph_us(lambda st, mode=mode: api.sb_branch_candidates(
                cq, cxb, 6, mode, cu, ccount, ctok, crows, cws, st))
        cand_b = int(ccount.item())
        src = list(range(1, 1 + B))
        dst = list(range(1, 1 + B))
        dsws = torch.empty(api.sb_draft_sample_workspace_bytes(V, B), dtype=torch.uint8, device=dev)
        samp_us = graph_us(lambda st: api.sb_draft_sample(logits, stats, src, 1.0, du, dtok, dq, dst,
                                                          dsws, st))
        # One whole round of Algorithm 2 (sb_spec_round): the 68M draft
        # drafts a chain (confidence threshold 0: always trunk_max - 1 = 3
        # drafts, a length independent of the drafted values), the target
        # verifies that chain on one stream while the draft spawns B + 1
        # candidates' worth of branches at x_b (k_max = B + 1 gives B
        # branches at a near-flat q) and extends them to depth k on another;
        # then Algorithm 1 at the chain's last row and both rollbacks.  Timed
        # on one stream and on two (default priorities); the results must
        # not change.  Random weights on both sides, so the mechanics and
        # the time are the point, not the acceptance.
        RK = B + 1
        rparams = api.round_params(RK, "wor", DD, TRUNK, 0.0, 1.0)
        rbuf = api.RoundBuffers(m, dm, rparams, kv_len, kv_len, dev)
        RR = TRUNK + RK * DD
        r_ud = torch.from_numpy(synth.uniforms(RR, 51)).to(dev)
        r_uw = torch.from_numpy(synth.uniforms(TRUNK + 1, 52)).to(dev)
        r_us = torch.from_numpy(synth.uniforms(RK + 1, 53)).to(dev)
        rbuf.tokens[0] = root
        sv, sd = torch.cuda.Stream(), torch.cuda.Stream()

        def round_on(vs, ds):
            vs.wait_stream(stream)
            ds.wait_stream(stream)
            got = api.sb_spec_round(m, k_, v_, kv_len, dm, dk_, dv_, kv_len, r_ud, r_uw, r_us, rbuf,
                                    vs, ds)
            stream.wait_stream(vs)
            return got
        times, outs = {}, {}
        for name, (vs, ds) in (("serial", (stream, stream)), ("overlapped", (sv, sd))):
            for _ in range(2):
                round_on(vs, ds)
            torch.cuda.synchronize()
            ev0.record(stream)
            for _ in range(reps):
                rc, rb, rpar = round_on(vs, ds)
            ev1.record(stream)
            torch.cuda.synchronize()
            times[name] = ev0.elapsed_time(ev1) / reps
            outs[name] = (api.decode_round(rbuf.round), api.decode_result(rbuf.walk),
                          rbuf.tokens.cpu().tolist(), rbuf.new_lens.cpu().tolist())
        if outs["serial"] != outs["overlapped"]:
            raise RuntimeError("the two-stream round changed a result")
        # the target's part alone: the chain's forward and its walk
        cpar = list(range(-1, rc))

        def verify_chain():
            m.sb_verify_forward(k_, v_, kv_len, rbuf.tokens, cpar, 1.0, rbuf.logits, rbuf.stats, ws,
                                stream)
            api.sb_accept_resample(rbuf.tokens, cpar, rbuf.logits, rbuf.stats, 1.0, rbuf.q, r_uw,
                                   rbuf.walk, sws, stream)
        verify_chain()
        torch.cuda.synchronize()
        ev0.record(stream)
        for _ in range(reps):
            verify_chain()
        ev1.record(stream)
        torch.cuda.synchronize()
        vc_ms = ev0.elapsed_time(ev1) / reps
        # the draft's part alone: the chain, then the branches
        dws_r = dm.draft_round_workspace(RK, DD, kv_len, TRUNK)
        xb_r = torch.empty(1, dtype=torch.int32, device=dev)

        def draft_part(with_branches):
            c_ = dm.sb_draft_chain(dk_, dv_, kv_len, TRUNK, 0.0, 1.0, r_ud, rbuf.tokens, rbuf.q, xb_r,
                                   dws_r, stream)
            if with_branches:
                dm.sb_draft_branches(dk_, dv_, kv_len, c_, xb_r, RK, "wor", DD, 1.0, r_ud[TRUNK:],
                                     rbuf.tokens, rbuf.q, dws_r, stream)
        part_ms = {}
        for wb in (False, True):
            draft_part(wb)
            torch.cuda.synchronize()
            ev0.record(stream)
            for _ in range(reps):
                draft_part(wb)
            ev1.record(stream)
            torch.cuda.synchronize()
            part_ms[wb] = ev0.elapsed_time(ev1) / reps
        br_ms = part_ms[True] - part_ms[False]
        ro = outs["serial"][0]
        saved = times["serial"] - times["overlapped"]
        round_out = {"trunk_max": TRUNK, "confidence": 0.0, "k_max": RK, "depth": DD,
                     "mode": "wor", "chain": rc, "branches": rb, "draft_rows": int(len(rpar)),
                     "n_trunk": ro["n_trunk"], "kept": ro["kept"],
                     "committed": ro["n_trunk"] + 1,
                     "serial_ms": round(times["serial"], 4),
                     "overlapped_ms": round(times["overlapped"], 4),
                     "verify_chain_ms": round(vc_ms, 4),
                     "draft_chain_ms": round(part_ms[False], 4),
                     "draft_branches_ms": round(br_ms, 4),
                     "saved_ms": round(saved, 4),
                     # the most two streams can save is the shorter of the
                     # two concurrent parts
                     "hidden_frac": round(saved / min(vc_ms, br_ms), 3)}
        draft_out = {"shape": f"{dshape.name}: {dshape.n_layers} layers, hidden {dshape.hidden}, "
                              f"{dshape.n_heads}x{dshape.head_dim} heads, ffn {dshape.ffn}, "
                              f"vocab {V}, bf16",
                     "round": f"k_max={DK}, depth={DD}, without replacement, T=1, prefix {P}",
                     "round_ms": round(round_ms, 4), "branches": bd,
                     "round_plus_verify_ms": round(round_ms + ms_per_step, 4),
                     "candidates_us_k6": cand_us, "candidates_B": cand_b,
                     "candidates_bytes_k6_wor": 4 * V * (1 + cand_b),
                     "sample_us": samp_us, "sample_rows": B,
                     "sample_bytes": 2 * 4 * V * B}
        del dm, dk_, dv_, dq, crows

    if args.copy_calibration:
        # a plain device copy of known size, for scaling the HBM byte counters
        src = torch.empty(COPY_BYTES, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    nbytes = algorithmic_bytes(shape, kv_len, n)
    k_avg_ms = k_ms / max(1, k_launches)
    achieved = nbytes["gate_up_launch"] / (k_avg_ms * 1e-3) / 1e9
    verified = (n - 1) / (ms_per_step * 1e-3)
    out = {
        "metric": "verified tokens/s per verify step + % HBM roofline, 7B-shape bf16, B=4 k=8",
        "value": round(verified, 1),
        "unit": "verified tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic: seeded N(0,0.02) bf16 weights, seeded N(0,1) prefix KV, "
                "drafts drawn from alpha*p+(1-alpha)*softmax(N(0,1)/0.7)",
        "config": {"workload": f"{shape.name} verify step: {tree_desc}, prefix {P}",
                   "rows": n, "prefix": P, "branches": B,
                   "depth": kd if args.tree == "branch" else args.trunk + args.fork_depth,
                   "alpha": args.alpha},
        "step_hbm": {"bytes": nbytes["step"],
                     "achieved_gbs": round(nbytes["step"] / (ms_per_step * 1e-3) / 1e9, 1),
                     "frac": round(nbytes["step"] / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                     "ms_per_step_median": round(ms_median, 4),
                     "ms_forward_and_accept": round(ms_no_rollback, 4),
                     "ms_per_step_with_kernel_events": round(evented_ms, 4),
                     "ms_per_step_graph_replay": None if graph_ms is None else round(graph_ms, 4)},
        "roofline": {"bound": "hbm", "scope": "per kernel: the dominant kernel of the step "
                     "(the step as a whole is step_hbm)",
                     "kernel": f"k_gemm (gate/up + SwiGLU), {k_launches} launches",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": measured_traffic(args.workload),
                     "avg_us": round(k_avg_ms * 1e3, 2)},
        "accepted": r["n_accepted"],
    }
    if hrad_out is not None:
        out["hrad"] = hrad_out
    if draft_out is not None:
        out["draft"] = draft_out
        out["overlap"] = round_out

    if not args.no_alpha_sweep:
        # committed tokens per step under the q mixture of each alpha: every
        # sample draws a fresh draft tree (its own seed) and its own uniforms,
        # verifies it and walks it
        sweep = {}
        n_samples = 16
        for a in (0.3, 0.6, 0.9):
            lens = []
            for smp in range(n_samples):
                toks_a, q_a = make_drafts(api, synth, m, k_, v_, kv_len, root, parents, a,
                                          w.q_temp, 1000 + smp)
                dt, dq = torch.from_numpy(toks_a).to(dev), torch.from_numpy(q_a).to(dev)
                m.sb_verify_forward(k_, v_, kv_len, dt, parents, 1.0, logits, stats, ws, stream)
                du = torch.from_numpy(synth.uniforms(n, 100 + smp)).to(dev)
                api.sb_accept_resample(dt, parents, logits, stats, 1.0, dq, du, res, sws, stream)
                lens.append(api.decode_result(res)["n_accepted"] + 1)
            mean = float(np.mean(lens))
            sweep[str(a)] = {"mean_committed": round(mean, 3),
                             "stderr": round(float(np.std(lens, ddof=1) / np.sqrt(n_samples)), 3),
                             "samples": n_samples,
                             "committed_tokens_per_s": round(mean / (ms_per_step * 1e-3), 1)}
        out["alpha_sweep"] = sweep

    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample ...")
        cb = cpu_baseline(shape, host_bits, kv_host, kv_len, inp, args.cpu_layers)
        out["cpu_baseline"] = {k: (round(v, 3) if isinstance(v, float) else v)
                               for k, v in cb.items() if k != "step_s"}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
