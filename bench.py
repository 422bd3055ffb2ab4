#!/usr/bin/env python3
"""Benchmark of the PRISM drafting hot path on one MI355X.

One benchmark step = one prism_draft_chain call: K = 5 greedy draft steps of
the Llama-3-8B-shaped drafter (hidden 4096, 32/8 heads x 128, SwiGLU 14336,
vocab 128256, step-1 feature 3 x 4096), batch 1, prior context 2048, bf16,
every step with its own parameter set.  Weights and inputs are seeded
synthetic tensors already resident in HBM when timing starts.

Printed (one JSON line): drafted tokens/s, per-draft-step microseconds (the
call time / K, and each step between its own HIP events), the roofline of
the dominant kernel (the LM-head GEMV with fused top-k, timed with HIP
events around each of its launches), and the CPU oracle timed on a bounded
sample of the same workload.  The same line carries, under "bs16", the
batch-16 half of the metric (same weights, ragged contexts 512-4096, paged
KV), and under "llama3_70b_bs32" the 70B-shaped batch-32 chain with the
bf16 MFMA fraction of its weight products.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0       # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0   # dense MFMA
COPY_BYTES = 256 << 20      # counter-calibration copy
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_lmhead_traffic.json")


def kernel_source_digest(read=None):
    """Digest of the LM-head kernel's code (its sources without // comments
    and blank lines), so that the counter figures go stale with the code but
    not with its documentation."""
    import hashlib
    h = hashlib.sha256()
    for f in ("gemm.hip", "device.h", "internal.h", "plan.h"):
        if read is None:
            with open(os.path.join(ROOT, "paper_2602_01762_amd", "csrc", f)) as fh:
                text = fh.read()
        else:
            text = read(f)
        for line in text.splitlines():
            code = line.split("//", 1)[0].rstrip()
            if code:
                h.update(code.encode() + b"\n")
    return h.hexdigest()[:16]


def lm_traffic(cfg):
    """HBM bytes per LM-head launch measured with FETCH_SIZE / WRITE_SIZE
    counter runs (profiles/k_lmhead_traffic.json), or None when they were
    taken on other kernel sources or another workload."""
    try:
        with open(TRAFFIC_FILE) as fh:
            t = json.load(fh)
    except (OSError, ValueError):
        return None
    if t.get("source_digest") != kernel_source_digest() or t.get("workload") != cfg.name:
        return None
    return t.get("bytes_per_launch")

WORKLOADS = {
    "8b_bs1": "llama3_8b_bf16_chain_bs1",
    "8b_bs16": "llama3_8b_bf16_chain_bs16_paged",
    "8b_tree": "llama3_8b_bf16_tree_bs4",
    "70b_bs32": "llama3_70b_bf16_chain_bs32",
    "8b_bs1_catchup": "llama3_8b_bf16_chain_bs1_catchup4",
    "8b_bs16_catchup": "llama3_8b_bf16_chain_bs16_paged_catchup",
    "8b_bs1_t1": "llama3_8b_bf16_chain_bs1_t1",
    "l2_7b_bs1": "llama2_7b_bf16_chain_bs1",
    "l2_7b_bs1_m1": "llama2_7b_bf16_chain_bs1_m1",
    "l2_7b_bs1_m2": "llama2_7b_bf16_chain_bs1_m2",
}


def lm_workgroups(cfg, rows):
    """Workgroups of one LM-head launch (the library's plan: 16-id vocab tiles,
    4 waves per workgroup, tiles per wave by rows)."""
    tiles, nkb = cfg.vocab // 16, cfg.hidden // 32
    if rows == 1 and cfg.dtype == "bf16" and nkb % 16 == 0:
        nt = 4 if tiles % 16 == 0 and nkb % 16 == 0 and tiles // 4 >= 1024 else 1
    elif rows <= 32 and tiles % 8 == 0:
        nt = 8
    elif tiles % 4 == 0:
        nt = 4
    else:
        nt = 2 if tiles % 2 == 0 else 1
    return (tiles // nt + 3) // 4


def lm_topk_pass(cfg, rows):
    """Whether the LM head stores fp32 logits and a separate pass reduces them
    to the top-k partials (the library's rule: greedy top-k > 1 on the MFMA
    tiles, i.e. more than one row or fp32 weights)."""
    gemv = rows == 1 and cfg.dtype == "bf16" and (cfg.hidden // 32) % 16 == 0
    return max(1, cfg.tree_width) > 1 and not gemv and not cfg.temperature


def lm_head_bytes(cfg, rows):
    """Algorithmic HBM bytes of one LM-head launch: the [V, H] weight stream,
    the normalised input rows (a hi/lo pair of bf16 planes, or fp32), and
    either the per-workgroup partials (max, sum and k values and ids per row)
    or, when a separate pass takes the top-k, the fp32 logits rows."""
    es = 2 if cfg.dtype == "bf16" else 4
    k = max(1, cfg.tree_width)
    base = cfg.vocab * cfg.hidden * es + rows * cfg.hidden * 4
    if lm_topk_pass(cfg, rows):
        return base + rows * cfg.vocab * 4
    return base + rows * lm_workgroups(cfg, rows) * (2 + 2 * k) * 4


def step_weight_bytes(cfg, s):
    """Weight bytes one pass of set s reads as the method defines it: every
    matrix of the set once, the fusion FC over [E(x) ; f], and the LM head."""
    es = 2 if cfg.dtype == "bf16" else 4
    H, I, d = cfg.hidden, cfg.ffn, cfg.head_dim
    F = cfg.set_feat_width(s)
    return es * (H * (H + F) + cfg.qkv_dim * H + H * cfg.n_q_heads * d + 3 * H * I + cfg.vocab * H)


def uses_embed_table(cfg, rows):
    """Whether a pass takes the fusion FC's embedding half from the per-set
    table (the library's rule: bf16 contexts whose hidden size is a multiple
    of 64, at any row count)."""
    return cfg.dtype == "bf16" and cfg.hidden % 64 == 0


def step_streamed_bytes(cfg, s, rows):
    """Weight bytes a pass of set s streams from HBM: as step_weight_bytes,
    except that with the embedding table the FC reads only its feature
    columns plus one fp32 table row per row."""
    b = step_weight_bytes(cfg, s)
    if uses_embed_table(cfg, rows):
        es = 2 if cfg.dtype == "bf16" else 4
        b -= es * cfg.hidden * cfg.hidden - rows * cfg.hidden * 4
    return b


def pass_rows(cfg, k):
    """Rows of chain step k (0-based): the batch, or every accepted token of
    the batch at step 1 of a catch-up chain."""
    if k == 0 and cfg.n_new:
        return cfg.batch * cfg.n_new[1]
    return cfg.batch


VERIFY_WORKLOADS = {
    # the verification step of Sec. 2 on synthetic target logits, 8B vocabulary
    "verify_bs16": dict(mode="chain", batch=16, K=5, temperature=1.0),
    "verify_bs16_greedy": dict(mode="chain", batch=16, K=5, temperature=0.0),
    "verify_tree_bs4": dict(mode="tree", batch=4, nodes=60),
}


def verify_bench(args):
    """Time the verification call and report it against the HBM roofline of
    its logits stream (every logits row read once)."""
    import torch
    from synth import L3_8B_BS16, make_verify_chain, make_verify_tree_targets
    from paper_2602_01762_amd import Drafter
    spec = VERIFY_WORKLOADS[args.workload]
    torch.cuda.set_device(0)
    cfg = L3_8B_BS16          # context of the 8B vocabulary (verification needs no weights)
    dr = Drafter(cfg)
    V, B = cfg.vocab, spec["batch"]
    if spec["mode"] == "chain":
        K, T = spec["K"], spec["temperature"]
        d = make_verify_chain(V, B, K, seed=0, device="cuda")
        dlg, uni = (d["draft_logits"], d["uniforms"]) if T > 0 else (None, None)
        call = lambda: dr.verify_chain(d["target_logits"], d["draft_tokens"], T, dlg, uni)
        rows = B * (K + 1) + (B * K if T > 0 else 0)
        name = "verify_chain_8b_vocab_bs%d_k%d_t%g" % (B, K, T)
    else:
        v = spec["nodes"]
        g = torch.Generator(device="cuda")
        g.manual_seed(0)
        tokens = torch.randint(0, V, (B, v), generator=g, device="cuda", dtype=torch.int32)
        parent = torch.tensor([[j - 1 for j in range(v)]] * B, dtype=torch.int32, device="cuda")
        tl = make_verify_tree_targets(tokens, parent, V, seed=0)
        call = lambda: dr.verify_tree(tl, tokens, parent)
        rows = B * (v + 1)
        name = "verify_tree_8b_vocab_bs%d_nodes%d" % (B, v)
    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        call()
    e1.record()
    torch.cuda.synchronize()
    assert dr.device_status() == 0
    us = e0.elapsed_time(e1) * 1e3 / args.steps
    nbytes = rows * V * 4
    gbs = nbytes / (us * 1e-6) / 1e9
    res = {"metric": "verification call latency", "value": round(us, 2), "unit": "us",
           "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "ms_per_step": round(us / 1e3, 5), "higher_is_better": False, "scaling": "weak",
           "vs_baseline": None, "dtype": "f32", "data": "synthetic target / draft logits",
           "config": {"workload": name, "batch": B, "vocab": V},
           "roofline": {"kernel": "k_rows_stats + k_verify_* (logits stream)", "bound": "hbm",
                        "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                        "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None,
                        "algorithmic_bytes_per_launch": nbytes}}
    dr.close()
    print(json.dumps(res), flush=True)


def product_flops(cfg, s, rows):
    """Multiply-add flops (2 per weight element per row) of the weight
    products of one pass of set s over `rows` rows, as the method defines
    them: the whole fusion FC, QKV, O, gate/up, down and the LM head."""
    es = 2 if cfg.dtype == "bf16" else 4
    return 2 * rows * step_weight_bytes(cfg, s) // es


def mfma_ceiling(rows):
    """Largest bf16 MFMA fraction a product can reach while it streams each
    weight from HBM once: 2 * rows flops per 2-byte weight = rows flop/B,
    times 8 TB/s, over the 2.5 PFLOP/s dense peak."""
    return rows * HBM_PEAK_GBS * 1e9 / (BF16_PEAK_TFLOPS * 1e12)


def cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def make_call(cfg, dr, inp):
    """The drafting call of a workload on preallocated outputs."""
    import torch
    tree = cfg.mode == "tree"
    b = dr.batch(inp)
    out = dr.tree_buffers(cfg.batch, cfg.n_steps, debug=False) if tree else \
        dr.chain_buffers(cfg.batch, cfg.n_steps)
    if tree:
        return lambda: dr.tree(inp, out=out, batch=b)
    if cfg.n_new:      # step 1 prefills every accepted token
        return lambda: dr.chain_catchup(inp, out=out, batch=b)
    if cfg.temperature:    # stochastic drafting: draws and their log p_draft
        out["logp"] = torch.empty((cfg.batch, cfg.n_steps), dtype=torch.float32, device="cuda")
        return lambda: dr.chain_sample(inp, cfg.temperature, out=out, batch=b)
    return lambda: dr.chain(inp, out=out, batch=b)


def profiled(dr, call, what, steps):
    """Per-call lists of event-pair milliseconds of the classes `what`
    (eager launches on the stream, each pair around one launch or pass)."""
    import torch
    from paper_2602_01762_amd import binding
    binding.prism_profile_enable(dr.ctx, what)
    call()
    torch.cuda.synchronize()
    runs = []
    for _ in range(steps):
        call()
        runs.append(binding.prism_profile_pairs(dr.ctx))
    binding.prism_profile_enable(dr.ctx, 0)
    return runs


def measure(cfg, w, inp, args, gemm=False):
    """Time one workload: the timed region, per-call spread, per-step and
    LM-head event timings, and (gemm) the weight products' time."""
    import numpy as np
    import torch
    from paper_2602_01762_amd import Drafter, binding
    dr = Drafter(cfg)
    if cfg.f_map is not None:
        dr.set_step_map(cfg.fmap)
    dr.load(w)
    torch.cuda.synchronize()
    tree = cfg.mode == "tree"
    call = make_call(cfg, dr, inp)
    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()
    print("bench: %s: timing %d calls" % (cfg.name, args.steps), file=sys.stderr, flush=True)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_wall = time.perf_counter()
    e0.record()
    for _ in range(args.steps):
        call()
    e1.record()
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    total_ms = e0.elapsed_time(e1)
    ms_per_call = total_ms / args.steps
    K = cfg.n_steps
    drafted = cfg.batch * K if not tree else cfg.batch * cfg.tree_nodes
    assert dr.device_status() == 0
    m = {"ms_per_call": ms_per_call, "value": drafted * args.steps / (total_ms / 1e3),
         "wall_s": t_wall}

    # per-call distribution: a second pass of the same number of calls, each
    # between its own pair of events (kept out of the timed region above)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    for a0, a1 in ev:
        a0.record()
        call()
        a1.record()
    torch.cuda.synchronize()
    per_call = np.array([a0.elapsed_time(a1) for a0, a1 in ev])
    m["call_ms"] = {"median": round(float(np.median(per_call)), 4),
                    "p10": round(float(np.percentile(per_call, 10)), 4),
                    "p90": round(float(np.percentile(per_call, 90)), 4)}

    # each forward pass between its own events (eager launches): per-step us
    runs = profiled(dr, call, binding.PRISM_PROFILE_PASSES, args.steps)
    m["per_step_us"] = [round(float(np.mean([r[k] for r in runs])) * 1e3, 2) for k in range(K)]
    # dominant kernel: HIP events around every LM-head launch (same kernels,
    # launched directly on the stream so the events bracket each launch)
    runs = profiled(dr, call, binding.PRISM_PROFILE_LMHEAD, args.steps)
    lm_ms = [x for r in runs for x in r]
    rows = cfg.batch if not tree else cfg.batch * cfg.tree_width
    lm_us = float(np.mean(lm_ms)) * 1e3
    lm_b = lm_head_bytes(cfg, rows)
    achieved = lm_b / (lm_us * 1e-6) / 1e9
    kname = ("k_lmhead (LM head, fp32 logits stored; top-k by k_lm_topk)" if lm_topk_pass(cfg, rows)
             else "k_lmhead (LM head GEMV + fused top-k partials)" if rows == 1 and cfg.dtype == "bf16"
             else "k_lmhead (LM head MFMA tiles + fused top-k partials)")
    m["roofline"] = {"kernel": kname, "bound": "hbm",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": lm_traffic(cfg),
                     "avg_launch_us": round(lm_us, 2), "launches_timed": len(lm_ms),
                     "algorithmic_bytes_per_launch": lm_b}
    chain_bytes = sum(step_weight_bytes(cfg, cfg.fmap[k]) for k in range(K))
    streamed = sum(step_streamed_bytes(cfg, cfg.fmap[k], pass_rows(cfg, k)) for k in range(K))
    m["weight_bytes_per_step_call"] = chain_bytes
    m["weight_bytes_streamed_per_step_call"] = streamed
    m["whole_call_hbm_frac_weights_only"] = round(streamed / (ms_per_call * 1e-3) / 1e9
                                                  / HBM_PEAK_GBS, 4)
    if gemm:
        # the weight products (LM head included) between their own events
        runs = profiled(dr, call, binding.PRISM_PROFILE_PRODUCTS | binding.PRISM_PROFILE_LMHEAD,
                        args.steps)
        g_ms = float(np.mean([sum(r) for r in runs]))
        flops = sum(product_flops(cfg, cfg.fmap[k], pass_rows(cfg, k)) for k in range(K))
        tf = flops / (g_ms * 1e-3) / 1e12
        m["gemm"] = {"flops_per_call": flops, "ms_per_call": round(g_ms, 4),
                     "launches_per_call": len(runs[0]), "achieved_tflops": round(tf, 1),
                     "peak_tflops": BF16_PEAK_TFLOPS, "mfma_frac": round(tf / BF16_PEAK_TFLOPS, 4),
                     "mfma_frac_ceiling_at_hbm_peak": round(mfma_ceiling(cfg.batch), 4),
                     "note": "algorithmic flops (2 per weight element per row, the whole fusion "
                             "FC) over the summed event time of the product and LM-head "
                             "launches; streaming each weight once caps MFMA use at the "
                             "ceiling given"}
    dr.close()
    return m


def sub_result(cfg, m):
    """A secondary workload's figures inside the one JSON line."""
    out = {"workload": cfg.name, "batch": cfg.batch, "draft_steps": cfg.n_steps,
           "prior_context": cfg.max_ctx if cfg.ctx_range is None else list(cfg.ctx_range),
           "ms_per_call": round(m["ms_per_call"], 4),
           "per_draft_step_us": round(m["ms_per_call"] * 1e3 / cfg.n_steps, 2),
           "per_step_us": m["per_step_us"], "value": round(m["value"], 1),
           "unit": "drafted tokens/s", "call_ms": m["call_ms"],
           "whole_call_hbm_frac_weights_only": m["whole_call_hbm_frac_weights_only"],
           "roofline": m["roofline"]}
    if "gemm" in m:
        out["gemm"] = m["gemm"]
    return out


def tree_cycle_bench(args):
    print(json.dumps(tree_cycle_measure(args)), flush=True)


def tree_cycle_measure(args):
    """One tree speculation cycle on the 8B shapes: the drafter's tree call
    (batch 4, D 6, w 8, v 60), the target model's pass over the root and the
    60 nodes of each tree under the tree mask (one transformer layer of the
    8B shape with its own weights and the shared-shape LM head, the 4 x 61
    rows in one pass), and greedy tree verification of its logits."""
    import numpy as np
    import torch
    from synth import L3_8B_TREE, make_inputs, make_weights, scoring_target
    from paper_2602_01762_amd import Drafter
    torch.cuda.set_device(0)
    cfg, tcfg = L3_8B_TREE, scoring_target(L3_8B_TREE)
    print("bench: %s + %s, generating weights" % (cfg.name, tcfg.name), file=sys.stderr, flush=True)
    w, inp = make_weights(cfg, "cuda"), make_inputs(cfg, "cuda")
    wt, it = make_weights(tcfg.with_(seed=7), "cuda"), make_inputs(tcfg, "cuda")
    it.features.zero_()
    dr, tdr = Drafter(cfg), Drafter(tcfg, max_batch=64)
    dr.load(w)
    tdr.load(wt)
    tree = dr.tree_buffers(cfg.batch, cfg.n_steps, debug=False)
    b, tb = dr.batch(inp), tdr.batch(it)
    lg = torch.empty((cfg.batch, cfg.tree_nodes + 1, cfg.vocab), dtype=torch.float32, device="cuda")
    parts = {"draft": lambda: dr.tree(inp, out=tree, batch=b),
             "score": lambda: tdr.score_tree(it, tree["tokens"], tree["depth"], tree["mask"],
                                             out=lg, batch=tb),
             "verify": lambda: tdr.verify_tree(lg, tree["tokens"], tree["parent"])}
    cycle = lambda: [f() for f in parts.values()]
    for _ in range(args.warmup):
        cycle()
    torch.cuda.synchronize()
    ev = lambda: torch.cuda.Event(enable_timing=True)
    t = {}
    for name, f in list(parts.items()) + [("cycle", cycle)]:
        e0, e1 = ev(), ev()
        e0.record()
        for _ in range(args.steps):
            f()
        e1.record()
        torch.cuda.synchronize()
        t[name] = e0.elapsed_time(e1) * 1e3 / args.steps
    assert dr.device_status() == 0 and tdr.device_status() == 0
    rps = cfg.tree_nodes + 1
    rows = cfg.batch * rps
    # the scoring passes (bf16: whole trees, up to 256 rows each): per pass
    # the layer's weights (FC over [E(x) ; 0], QKV, O, gate/up, down) and the
    # LM head; the logits rows written
    per_pass = 256 // rps * rps if tcfg.dtype == "bf16" else 64
    npass = -(-rows // per_pass)
    es = 2 if tcfg.dtype == "bf16" else 4
    lm_bytes = es * tcfg.vocab * tcfg.hidden
    n_lm = npass
    layer_bytes = step_weight_bytes(tcfg, 0) - 2 * tcfg.hidden * tcfg.hidden - lm_bytes
    score_bytes = npass * layer_bytes + n_lm * lm_bytes + rows * cfg.vocab * 4
    score_params = (layer_bytes + lm_bytes) // es
    res = {"metric": "tree speculation cycle latency (draft tree + target scoring + verify)",
           "value": round(t["cycle"], 2), "unit": "us", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": round(t["cycle"] / 1e3, 5),
           "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
           "data": "synthetic (seeded random-init drafter and one-layer target)",
           "config": {"workload": "llama3_8b_tree_bs4_score_verify", "batch": cfg.batch,
                      "depth": cfg.n_steps, "width": cfg.tree_width, "nodes": cfg.tree_nodes,
                      "target_rows": rows, "target_passes": npass, "target_lm_head_launches": n_lm},
           "part_us": {k: round(v, 2) for k, v in t.items() if k != "cycle"},
           "score_hbm_frac": round(score_bytes / (t["score"] * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
           # the passes are MFMA work (244 rows): every row meets every weight
           # of the layer and the LM head once, as an exact hi/lo bf16 pair of
           # activations, so the MFMAs execute 4 flops per row and weight
           "score_mfma_frac_executed": round(4 * rows * score_params / (t["score"] * 1e-6) / 1e12
                                             / BF16_PEAK_TFLOPS, 4),
           "score_bytes_per_call": score_bytes}
    dr.close()
    tdr.close()
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="8b_bs1",
                    choices=sorted(WORKLOADS) + sorted(VERIFY_WORKLOADS) + ["8b_tree_cycle"])
    ap.add_argument("--cpu-baseline", type=int, default=1,
                    help="time the CPU oracle on a bounded sample (0 = skip)")
    ap.add_argument("--secondary", type=int, default=1,
                    help="with the default workload, also time the batch-16 chain and the "
                         "70B batch-32 chain (0 = skip)")
    ap.add_argument("--calibrate-copy", type=int, default=0,
                    help="also run a plain 256 MiB device copy (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures the single-GPU drafting path; --gpus %d is not supported "
              "(the path has no cross-GPU component)." % args.gpus, file=sys.stderr)
        sys.exit(2)

    if args.workload in VERIFY_WORKLOADS:
        return verify_bench(args)
    if args.workload == "8b_tree_cycle":
        return tree_cycle_bench(args)

    import torch
    from synth import CONFIGS, L3_70B_BS32, L3_8B_BS16, make_inputs, make_weights

    cfg = CONFIGS[WORKLOADS[args.workload]]
    torch.cuda.set_device(0)
    print("bench: %s, generating weights" % cfg.name, file=sys.stderr, flush=True)
    w = make_weights(cfg, "cuda")
    inp = make_inputs(cfg, "cuda")
    m = measure(cfg, w, inp, args, gemm=cfg.batch >= 16)
    K = cfg.n_steps
    res = {
        "metric": "drafted tokens/s + per-draft-step µs (8B shape, bs=1/16); % HBM/MFMA peak",
        "value": round(m["value"], 1), "unit": "drafted tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(m["ms_per_call"], 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": cfg.dtype,
        "data": "synthetic (seeded random-init weights N(0,0.02), features N(0,1), prior KV N(0,1))",
        "config": {"workload": cfg.name, "batch": cfg.batch, "draft_steps": K,
                   "prior_context": cfg.max_ctx if cfg.ctx_range is None else list(cfg.ctx_range),
                   "kv_block": cfg.kv_block_size, "mode": cfg.mode,
                   "accepted_tokens_step1": list(cfg.n_new) if cfg.n_new else 1,
                   "temperature": cfg.temperature or 0.0},
        "per_draft_step_us": round(m["ms_per_call"] * 1e3 / K, 2),
        "per_step_us": m["per_step_us"],
        "call_ms": m["call_ms"],
        "weight_bytes_per_step_call": m["weight_bytes_per_step_call"],
        "weight_bytes_streamed_per_step_call": m["weight_bytes_streamed_per_step_call"],
        "whole_call_hbm_frac_weights_only": m["whole_call_hbm_frac_weights_only"],
        "wall_s": round(m["wall_s"], 4),
        "roofline": m["roofline"],
    }
    if "gemm" in m:
        res["gemm"] = m["gemm"]
    print("bench: gpu done %.3f ms/call" % m["ms_per_call"], file=sys.stderr, flush=True)
    if args.calibrate_copy:
        # a copy of known size: its FETCH_SIZE / WRITE_SIZE counters give the
        # KiB-per-byte scale of the same counters on the LM-head kernel
        src = torch.empty(COPY_BYTES // 2, dtype=torch.bfloat16, device="cuda").normal_()
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
    if args.cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(cfg, w, inp)
    if args.secondary and args.workload == "8b_bs1":
        # the other half of the metric (batch 16, same weights) and the 70B
        # batch-32 chain whose products the MFMA figure is quoted on
        inp16 = make_inputs(L3_8B_BS16, "cuda")
        res["bs16"] = sub_result(L3_8B_BS16, measure(L3_8B_BS16, w, inp16, args))
        del w, inp, inp16
        torch.cuda.empty_cache()
        print("bench: %s, generating weights" % L3_70B_BS32.name, file=sys.stderr, flush=True)
        w70 = make_weights(L3_70B_BS32, "cuda")
        inp70 = make_inputs(L3_70B_BS32, "cuda")
        res["llama3_70b_bs32"] = sub_result(L3_70B_BS32, measure(L3_70B_BS32, w70, inp70, args,
                                                                 gemm=True))
        del w70, inp70
        torch.cuda.empty_cache()
        # the tree speculation cycle (draft tree, target scoring, verification)
        t = tree_cycle_measure(args)
        res["tree_cycle"] = {"workload": t["config"]["workload"], "us_per_cycle": t["value"],
                             "part_us": t["part_us"],
                             "score_mfma_frac_executed": t["score_mfma_frac_executed"],
                             "target_rows": t["config"]["target_rows"],
                             "target_passes": t["config"]["target_passes"]}
    print(json.dumps(res), flush=True)


def cpu_baseline(cfg, w, inp):
    """The oracle, as it is, on the host cores: full drafting calls of one
    sequence of the same workload, repeated until about 10 s have passed."""
    import numpy as np
    from oracle import Oracle
    from oracle import _native
    from synth import host_inputs, host_weights
    seqs = [0]
    hw = host_weights(w)
    hi = host_inputs(inp, cfg, seqs)
    orc = Oracle(cfg, hw)
    _native.lib()
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    n, t0 = 0, time.perf_counter()
    while True:
        if cfg.mode == "tree":
            orc.tree(hi, seqs=seqs)
        else:
            orc.chain(hi, seqs=seqs, catchup=bool(cfg.n_new), temperature=cfg.temperature,
                      uniforms=hi.get("uniforms"))
        n += 1
        el = time.perf_counter() - t0
        if el >= 10.0 or n >= 200:
            break
    drafted = n * (cfg.n_steps if cfg.mode == "chain" else cfg.tree_nodes)
    return {"value": round(drafted / el, 3), "unit": "drafted tokens/s", "cores": threads,
            "cpu_model": cpu_model(), "kind": "oracle",
            "sample": "%d full %s calls of sequence 0 (%d draft steps each), fp64 arithmetic on "
                      "the stored (bf16) tensors, %.1f s" % (n, cfg.mode, cfg.n_steps, el)}


if __name__ == "__main__":
    main()
