"""Host logic of bench.py, on the CPU: the one-GPU guard, the step's
algorithmic bytes against published parameter counts and KV sizes, the
kernel classes of a verify step, and the parsing of kernel traces (a
synthetic trace in rocprofv3's CSV format)."""
import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2506_01979_amd import synth  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU" in json.loads(r.stdout.strip().splitlines()[-1])["error"]


# Total parameter counts of the published models whose shapes the workloads
# use (embedding table, LM head, projections and RMSNorm gains): LLaMA-7B,
# Llama-2-13B, Llama-3-70B.
PUBLISHED_PARAMS = [("llama7b", 6_738_415_616), ("llama13b", 13_015_864_320),
                    ("llama70b", 70_553_706_496)]


@pytest.mark.parametrize("name,params", PUBLISHED_PARAMS)
def test_weight_bytes_match_the_published_parameter_counts(name, params):
    """The step reads every projection and the LM head once in bf16, the
    RMSNorm gains in fp32 and only the n embedding rows it gathers: adding
    back the rest of the embedding table gives the published total."""
    sh = synth.SHAPES[name]
    n = 33
    b = bench.algorithmic_bytes(sh, 2047, n)
    gains = (2 * sh.n_layers + 1) * sh.hidden
    matrix_bytes = b["weights"] - 4 * gains - n * sh.hidden * 2
    assert matrix_bytes % 2 == 0
    assert matrix_bytes // 2 + sh.vocab * sh.hidden + gains == params
    # the per-class launch bytes with no token rows are the weight streams:
    # every layer's four projections plus the LM head again give the total
    c = bench.class_bytes(sh, 0, 0, split_down=0)
    per_layer = c["qkv"] + c["o"] + c["gate_up"] + c["down"]
    assert (sh.n_layers * per_layer + c["lm_head"]) // 2 + sh.vocab * sh.hidden + gains == params


@pytest.mark.parametrize("name,per_token", [("llama7b", 512 * 1024), ("llama13b", 800 * 1024),
                                            ("llama70b", 320 * 1024)])
def test_prefix_kv_bytes_per_token(name, per_token):
    """bf16 K and V of every layer: 512 KiB per token for LLaMA-7B (32
    layers x 4096), 800 KiB for 13B (40 x 5120), 320 KiB for the 70B's 8
    grouped KV heads (80 x 1024)."""
    sh = synth.SHAPES[name]
    for P in (1, 2047, 8191):
        b = bench.algorithmic_bytes(sh, P, 33)
        assert b["prefix_kv"] == P * per_token
        assert b["step"] == b["weights"] + b["prefix_kv"] + 33 * per_token + 33 * sh.vocab * 8
    assert bench.class_bytes(sh, 2047, 33)["attn"] == (2047 + 33) * per_token // sh.n_layers + \
        33 * sh.q_dim * 2


FUSED_LAYER = ["k_rmsnorm_pack<1>", "k_gemm<0, 3, 3>", "k_attn<128, 3, 2, false>",
               "k_attn_merge_reg<128, 8>", "k_gemm<4, 3, 1>", "k_gemm<2, 3, 6>",
               "k_gemm<1, 3, 4>"]
UNFUSED_LAYER = ["k_rmsnorm_pack<1>", "k_gemm<0, 3, 3>", "k_attn<128, 3, 2, false>",
                 "k_attn_merge_reg<128, 8>", "k_gemm<1, 3, 1>", "k_rmsnorm_pack<1>",
                 "k_gemm<2, 3, 6>", "k_gemm<1, 3, 4>"]


@pytest.mark.parametrize("layer,want", [
    (FUSED_LAYER, ["norm", "qkv", "attn", "attn_merge", "o", "gate_up", "down"]),
    (UNFUSED_LAYER, ["norm", "qkv", "attn", "attn_merge", "o", "norm", "gate_up", "down"]),
])
def test_kernel_classes_of_a_layer(layer, want):
    prev, got = "", []
    for name in layer * 2:
        prev = bench.kernel_class(f"void sb::(anonymous namespace)::{name}(sb::GemmArgs)", prev)
        got.append(prev)
    assert got == want * 2
    assert bench.kernel_class("void k_embed_meta<unsigned short>(...)", "") == "embed"
    assert bench.kernel_class("void k_softmax_stats_reg<8>(...)", "lm_head") == "stats"
    assert bench.kernel_class("k_walk(int, ...)", "stats") == "accept_walk"
    assert bench.kernel_class("void k_rollback<unsigned short>(...)", "accept_walk") == "rollback"
    assert bench.kernel_class("void k_gemm<3, 3, 8>(sb::GemmArgs)", "norm") == "lm_head"
    assert bench.kernel_class("void k_gemm_wide<2, 9>(sb::GemmArgs)", "o") == "gate_up"
    assert bench.kernel_class("void k_gemm_wide<1, 9>(sb::GemmArgs)", "gate_up") == "down"


def _write_trace(d, n_steps, n_layers):
    """A kernel trace of n_steps verify steps, each after a launch that is
    no part of a step, in which every kernel of class c lasts dur[c]
    microseconds."""
    dur = {"embed": 5, "norm": 4, "qkv": 20, "attn": 12, "attn_merge": 5, "o": 11,
           "gate_up": 33, "down": 17, "lm_head": 43, "stats": 10, "walk": 17, "rollback": 5}
    names = {"embed": "k_embed_meta<unsigned short>", "lm_head": "k_gemm<3, 3, 8>",
             "stats": "k_softmax_stats_reg<8>", "walk": "k_walk", "rollback": "k_rollback<unsigned short>"}
    classes = ["norm", "qkv", "attn", "attn_merge", "o", "gate_up", "down"]
    rows, t = [], 1_000_000
    for s in range(n_steps):
        seq = [("other", "k_pack")] + [("embed", names["embed"])]
        for _ in range(n_layers):
            seq += list(zip(classes, FUSED_LAYER))
        seq += [("norm", "k_rmsnorm_pack<1>"), ("lm_head", names["lm_head"]),
                ("stats", names["stats"]), ("walk", names["walk"]), ("rollback", names["rollback"])]
        for c, name in seq:
            us = dur.get(c, 2)
            rows.append({"Kernel_Name": f"void sb::(anonymous namespace)::{name}(...)",
                         "Start_Timestamp": t, "End_Timestamp": t + us * 1000})
            t += us * 1000 + 2000
    os.makedirs(os.path.join(d, "run"), exist_ok=True)
    with open(os.path.join(d, "run", "run_kernel_trace.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        w.writeheader()
        w.writerows(rows)
    with open(os.path.join(d, "run", "run_kernel_stats.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Name", "Calls", "AverageNs", "MinNs", "MaxNs",
                                          "Percentage"])
        w.writeheader()
        w.writerow({"Name": "k_gemm<2, 3, 6>", "Calls": n_steps * n_layers, "AverageNs": 33000,
                    "MinNs": 33000, "MaxNs": 33000, "Percentage": 20.0})
    return dur


def test_trace_summary_counts_the_last_five_steps(tmp_path):
    n_layers = 3
    dur = _write_trace(str(tmp_path), 7, n_layers)
    text = bench.trace_summary(str(tmp_path), "llama7b_b4k8_p2048")
    table = {}
    for line in text.split("Whole-run")[0].splitlines():
        cells = [c.strip() for c in line.split("|")]
        if len(cells) == 8 and cells[1] not in ("class", "---", "total", ""):
            table[cells[1]] = (int(cells[3]), float(cells[4]), float(cells[6]))
    per_step = {"norm": n_layers + 1, "qkv": n_layers, "attn": n_layers, "attn_merge": n_layers,
                "o": n_layers, "gate_up": n_layers, "down": n_layers, "lm_head": 1, "stats": 1,
                "accept_walk": 1, "rollback": 1, "embed": 1}
    assert set(table) == set(per_step)
    for c, k in per_step.items():
        us = dur["walk" if c == "accept_walk" else c]
        launches, avg, total = table[c]
        assert launches == k and avg == us and total == pytest.approx(k * us, abs=0.05), c
    assert "Last 5 complete steps" in text
    # the draft-generation launch before each step is no part of a step
    assert "k_pack" not in text.split("Whole-run")[0]
