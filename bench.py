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
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0   # MI355X HBM3E, vendor figure
DOMINANT = "gate_up"    # kernel class holding the most bytes per step


def log(*a):
    print(*a, file=sys.stderr, flush=True)


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


def partial_tree(B: int, k: int, depth: int):
    """Rows of the B x k tree with depth < `depth`, in ascending row order,
    with parents re-indexed; returns (rows, parents)."""
    rows = [0] + [1 + b * k + t for b in range(B) for t in range(depth - 1)]
    rows.sort()
    pos = {r: i for i, r in enumerate(rows)}
    full = [-1] + [0 if t == 0 else 1 + b * k + t - 1 for b in range(B) for t in range(k)]
    return rows, [-1] + [pos[full[r]] for r in rows[1:]]


def make_drafts(api, synth, m, k_, v_, kv_len, root_tok, B, kd, alpha, q_temp, seed):
    """Drafts generated depth by depth: q = alpha * p_target + (1 - alpha) *
    softmax(N(0,1)/q_temp); the root's children are i.i.d. draws from one q."""
    import torch

    V = m.shape.vocab
    n = 1 + B * kd
    g = np.random.default_rng(seed)
    qrand = synth.softmax_rows(synth.random_logits(n, V, 1.0 / q_temp, seed=seed + 7))
    tokens = np.zeros(n, dtype=np.int32)
    tokens[0] = root_tok
    q = np.zeros((n, V), dtype=np.float32)
    for depth in range(1, kd + 1):
        rows, par = partial_tree(B, kd, depth)
        nr = len(rows)
        logits = torch.empty((nr, V), dtype=torch.float32, device="cuda")
        stats = api.new_stats(nr)
        m.sb_verify_forward(k_, v_, kv_len, torch.from_numpy(tokens[rows]).cuda(), par, 1.0,
                            logits, stats, m.workspace(nr, kv_len))
        lg = logits.cpu().numpy().astype(np.float64)
        lg -= lg.max(axis=1, keepdims=True)
        p = np.exp(lg)
        p /= p.sum(axis=1, keepdims=True)
        for b in range(B):
            row = 1 + b * kd + depth - 1
            parent = 0 if depth == 1 else row - 1
            pr = p[rows.index(parent)]
            qr = qrand[1] if depth == 1 else qrand[row]   # root children share one q
            qq = alpha * pr + (1 - alpha) * qr.astype(np.float64)
            qq /= qq.sum()
            q[row] = qq.astype(np.float32)
            tokens[row] = g.choice(V, p=qq)
    return tokens, q


def cpu_baseline(shape, host_bits, kv_host, kv_len, inp, n_layers_sample: int) -> dict:
    """The oracle as it stands, on the host cores: a bf16-emulation forward of
    the first layers of the same model (plus embedding, final norm and LM
    head) and the accept walk, extrapolated to the full depth per layer."""
    from oracle import decoder, sampling
    from paper_2506_01979_amd import synth

    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        cores = len(os.sched_getaffinity(0))

    def weights(nl):
        d = {"embed": synth.bits_to_f32(host_bits[("embed", None)]),
             "lm_head": synth.bits_to_f32(host_bits[("lm_head", None)]),
             "final_norm": synth.norm_gain(shape), "layers": []}
        for l in range(nl):
            lw = {n: synth.bits_to_f32(host_bits[(n, l)]) for n in synth.LAYER_MATS}
            lw["attn_norm"] = synth.norm_gain(shape)
            lw["mlp_norm"] = synth.norm_gain(shape)
            d["layers"].append(lw)
        return d

    Kp = [synth.bits_to_f32(kv_host[l][0]) for l in range(n_layers_sample)]
    Vp = [synth.bits_to_f32(kv_host[l][1]) for l in range(n_layers_sample)]
    times = {}
    for nl in (0, n_layers_sample):
        sh = shape.with_layers(nl)   # 0 layers: embedding, final norm, LM head only
        W = weights(nl)
        t0 = time.perf_counter()
        lg, _, _ = decoder.tree_forward(sh, W, Kp, Vp, kv_len, inp["tokens"], inp["parents"],
                                        "bf16")
        t1 = time.perf_counter()
        r = sampling.accept_resample(inp["tokens"], inp["parents"], lg.astype(np.float32), 1.0,
                                     inp["q"], inp["u"])
        t2 = time.perf_counter()
        times[nl] = (t1 - t0, t2 - t1)
        del W
    head, walk = times[0]
    per_layer = max(0.0, times[n_layers_sample][0] - head) / n_layers_sample
    step_s = head + walk + per_layer * shape.n_layers
    n_draft = len(inp["parents"]) - 1
    return {"value": n_draft / step_s, "unit": "verified tokens/s", "cores": int(cores),
            "kind": "oracle",
            "sample": (f"oracle bf16-emulation forward of layers 0..{n_layers_sample - 1} of "
                       f"{shape.n_layers} (+ embedding, final norm, LM head) and the accept walk "
                       f"on the same inputs; step time = head {head:.2f}s + walk {walk:.3f}s + "
                       f"{shape.n_layers} x per-layer {per_layer:.2f}s"),
            "step_s": step_s}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="llama7b_b4k8_p2048")
    ap.add_argument("--alpha", type=float, default=0.6)
    ap.add_argument("--cpu-layers", type=int, default=4)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-alpha-sweep", action="store_true")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print(json.dumps({"error": "this build runs on one GPU; --gpus must be 1"}), flush=True)
        sys.exit(2)

    import torch

    from paper_2506_01979_amd import api, synth

    w = synth.WORKLOADS[args.workload]
    shape = w.shape
    B, kd, P = w.branches, w.depth, w.prefix
    kv_len, n = w.kv_len, w.n_rows
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

    cap = kv_len + n + 16
    k_, v_ = m.new_kv(cap)
    kv_host = {}
    for l in range(shape.n_layers):
        kb = synth.synthetic_kv(shape, l, kv_len, kv_len, 0, as_bits=True)
        vb = synth.synthetic_kv(shape, l, kv_len, kv_len, 1, as_bits=True)
        k_[l, :, :kv_len] = torch.from_numpy(kb.view(np.int16)).view(torch.bfloat16).to(dev)
        v_[l, :, :, :kv_len] = torch.from_numpy(vb.view(np.int16)).view(torch.bfloat16).to(dev).transpose(1, 2)
        if l < args.cpu_layers:
            kv_host[l] = (kb, vb)
    log(f"prefix KV ready ({kv_len} slots) at {time.time() - t0:.1f}s")

    parents = synth.branch_parents(B, kd)
    root = int(synth.prefix_tokens(shape.vocab, P)[-1])
    tokens, q = make_drafts(api, synth, m, k_, v_, kv_len, root, B, kd, args.alpha, w.q_temp, 11)
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

    def step():
        m.sb_verify_forward(k_, v_, kv_len, d_tok, parents, 1.0, logits, stats, ws, stream)
        api.sb_accept_resample(d_tok, parents, logits, stats, 1.0, d_q, d_u, res, sws, stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    m.sb_timer_start(DOMINANT, args.steps * shape.n_layers)
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    total_ms = ev0.elapsed_time(ev1)
    k_ms, k_launches = m.sb_timer_stop()
    ms_per_step = total_ms / args.steps

    # same loop without the per-kernel events, for the clean step time
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    clean_ms = ev0.elapsed_time(ev1) / args.steps

    # rollback, timed on its own
    new_len = torch.zeros(1, dtype=torch.int32, device=dev)
    ev0.record(stream)
    m.sb_kv_rollback(k_, v_, kv_len, res, new_len, stream)
    ev1.record(stream)
    torch.cuda.synchronize()
    rollback_ms = ev0.elapsed_time(ev1)
    r = api.decode_result(res)

    nbytes = algorithmic_bytes(shape, kv_len, n)
    k_avg_ms = k_ms / max(1, k_launches)
    achieved = nbytes["gate_up_launch"] / (k_avg_ms * 1e-3) / 1e9
    verified = B * kd / (ms_per_step * 1e-3)
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
        "config": {"workload": f"{shape.name} verify step: B={B} branches x k={kd} drafts, "
                               f"prefix {P}", "rows": n, "prefix": P, "branches": B,
                   "depth": kd, "alpha": args.alpha},
        "roofline": {"bound": "hbm", "kernel": f"k_gemm (gate/up + SwiGLU), {k_launches} launches",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                     "avg_us": round(k_avg_ms * 1e3, 2)},
        "step_hbm": {"bytes": nbytes["step"],
                     "achieved_gbs": round(nbytes["step"] / (ms_per_step * 1e-3) / 1e9, 1),
                     "frac": round(nbytes["step"] / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                     "ms_per_step_without_kernel_events": round(clean_ms, 4)},
        "rollback_ms": round(rollback_ms, 4),
        "accepted": r["n_accepted"],
    }

    if not args.no_alpha_sweep:
        sweep = {}
        for a in (0.3, 0.6, 0.9):
            toks_a, q_a = make_drafts(api, synth, m, k_, v_, kv_len, root, B, kd, a, w.q_temp, 21)
            dt, dq = torch.from_numpy(toks_a).to(dev), torch.from_numpy(q_a).to(dev)
            m.sb_verify_forward(k_, v_, kv_len, dt, parents, 1.0, logits, stats, ws, stream)
            lens = []
            for s in range(32):
                du = torch.from_numpy(synth.uniforms(n, 100 + s)).to(dev)
                api.sb_accept_resample(dt, parents, logits, stats, 1.0, dq, du, res, sws, stream)
                lens.append(api.decode_result(res)["n_accepted"] + 1)
            mean = float(np.mean(lens))
            sweep[str(a)] = {"mean_committed": round(mean, 3),
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
