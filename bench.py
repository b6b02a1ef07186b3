"""Benchmark of the refinement step on one MI355X.

A step is one refinement pass (non-causal forward over prompt+draft, fused
top-1/confidence reduction over the vocabulary, threshold edit) over one batch
of synthetic input resident in HBM.  Prints one JSON line with the throughput
in refined (draft) positions per second, the roofline of the dominant kernel
measured with HIP events inside the timed region, and the CPU oracle timed on
a bounded sample of the same workload.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16 = 2.5e15        # MI355X dense bf16 MFMA, FLOP/s
PEAK_HBM = 8.0e12         # MI355X HBM3E, B/s
METRIC = "refined positions/sec per refinement step (1 GPU); MFMA % of bf16 peak"


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gemm_expert_gate_up_mini_moe_hbm_traffic.md")
GEMM_SOURCES = ("gemm.hip", "common.h", "kernels.h", "engine.hip")


def kernel_source_digest():
    """sha256 over the sources that define the GEMM kernels and their launches."""
    import hashlib
    h = hashlib.sha256()
    for f in GEMM_SOURCES:
        with open(os.path.join(ROOT, "paper_2608_02625_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def recorded_traffic(kernel, workload):
    """HBM bytes per launch measured with the FETCH_SIZE / WRITE_SIZE counters
    (scaled by a copy of known size), or None when they were taken on other
    sources, another kernel or another workload."""
    if workload != "mini_moe" or not os.path.exists(TRAFFIC_FILE):
        return None
    vals = {}
    with open(TRAFFIC_FILE) as fh:
        for line in fh:
            k, sep, v = line.strip().partition(": ")
            if sep and k in ("kernel", "traffic_bytes_per_launch", "source_digest"):
                vals[k] = v
    if vals.get("kernel") != kernel or vals.get("source_digest") != kernel_source_digest():
        return None
    return float(vals["traffic_bytes_per_launch"])


def step_flops(shape, B, P, D):
    """Algorithmic FLOPs of one pass: active experts only, LM head on draft
    rows only.  Only the draft rows leave the last block, so there the prompt
    rows need nothing but their K and V projections (the library still
    computes their Q, attention and O product, which is not counted)."""
    S = P + D
    T = B * S
    R = B * D
    d, hd, H, KV = shape.d_model, shape.head_dim, shape.n_heads, shape.n_kv_heads
    if shape.n_experts:
        ffn = d * shape.n_experts + (shape.top_k + shape.n_shared_experts) * 3 * d * shape.expert_ffn_dim
    else:
        ffn = 3 * d * shape.ffn_dim
    per_tok = d * (H + 2 * KV) * hd + H * hd * d + ffn
    body = 2 * T * per_tok * (shape.n_layers - 1) + 4 * T * S * H * hd * (shape.n_layers - 1)
    last = 2 * T * d * 2 * KV * hd + 2 * R * (d * H * hd + H * hd * d + ffn) + 4 * R * S * H * hd
    head = 2 * R * d * shape.vocab
    return body + last + head


def expert_rows_per_launch(shape, B, P, D):
    """Mean rows of one expert-GEMM launch over a pass: every row of every
    block, except the last block, whose FFN runs on the B*D draft rows only
    (when there is a prompt)."""
    T = B * (P + D)
    kr = shape.top_k + shape.n_shared_experts
    last = B * D if P > 0 else T
    return (T * (shape.n_layers - 1) + last) * kr / shape.n_layers


def kernel_flops(name, shape, B, P, D):
    """Algorithmic FLOPs of one launch of a named GEMM kernel (for the expert
    GEMMs the mean over one pass's launches)."""
    T = B * (P + D)
    d = shape.d_model
    if name == "gemm_expert_gate_up":
        return 2 * expert_rows_per_launch(shape, B, P, D) * d * 2 * shape.expert_ffn_dim
    if name == "gemm_expert_down":
        return 2 * expert_rows_per_launch(shape, B, P, D) * shape.expert_ffn_dim * d
    if name == "gemm_lm_head":
        return 2 * B * D * d * shape.vocab
    if name == "gemm_qkv":
        return 2 * T * d * (shape.n_heads + 2 * shape.n_kv_heads) * shape.head_dim
    if name == "gemm_o":
        return 2 * T * shape.n_heads * shape.head_dim * d
    if name == "attention":
        return 4 * T * (P + D) * shape.n_heads * shape.head_dim
    raise KeyError(name)


def library_reference(shape, B, P, D, launches, reps=20):
    """The vendor libraries on the same shapes, for context: torch.matmul
    (hipBLASLt; plain bf16 output, none of the fused epilogues) and torch's
    scaled_dot_product_attention, each beside the per-launch time of the
    library kernel doing that product in a refinement pass (`launches`: the
    (kernel, ms) pairs of one profiled pass, in launch order).  The expert
    GEMMs are set against one dense GEMM over all routed rows (no padding, no
    gather), beside the mean launch of the blocks whose FFN runs on every row."""
    import numpy as np
    import torch
    import torch.nn.functional as F

    S, T, R = P + D, B * (P + D), B * D
    d, hd, H, KV = shape.d_model, shape.head_dim, shape.n_heads, shape.n_kv_heads

    def ours(name, first_n=None):
        ms = [m for (n, m) in launches if n == name]
        ms = ms[:first_n] if first_n else ms
        return round(float(np.mean(ms)) * 1e3, 1) if ms else None

    def timed(fn):
        for _ in range(3):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / reps

    gemms = [("gemm_qkv", T, (H + 2 * KV) * hd, d), ("gemm_o", T, d, H * hd)]
    if shape.n_experts:
        kr = shape.top_k + shape.n_shared_experts
        F_ = shape.expert_ffn_dim
        gemms += [("gemm_expert_gate_up", T * kr, 2 * F_, d), ("gemm_expert_down", T * kr, d, F_)]
    gemms.append(("gemm_lm_head", R, shape.vocab, d))
    out = {}
    for name, M, N, K in gemms:
        a = torch.randn(M, K, device="cuda", dtype=torch.bfloat16)
        b = torch.randn(N, K, device="cuda", dtype=torch.bfloat16)
        us = timed(lambda: torch.matmul(a, b.t()))
        del a, b
        first = shape.n_layers - 1 if name.startswith("gemm_expert") and P > 0 else None
        out[name] = {"library": "torch.matmul", "M": M, "N": N, "K": K, "library_us": round(us, 1),
                     "library_tflops": round(2 * M * N * K / us / 1e6, 1), "ours_us": ours(name, first)}
    q = torch.randn(B, H, S, hd, device="cuda", dtype=torch.bfloat16)
    k = torch.randn(B, KV, S, hd, device="cuda", dtype=torch.bfloat16)
    v = torch.randn(B, KV, S, hd, device="cuda", dtype=torch.bfloat16)
    try:
        us = timed(lambda: F.scaled_dot_product_attention(q, k, v, enable_gqa=True))
        out["attention"] = {"library": "scaled_dot_product_attention", "B": B, "H": H, "KV": KV, "S": S, "hd": hd,
                            "library_us": round(us, 1), "library_tflops": round(4 * B * H * S * S * hd / us / 1e6, 1),
                            "ours_us": ours("attention")}
    except RuntimeError as e:                      # no fused attention kernel for this shape
        out["attention"] = {"library": "scaled_dot_product_attention", "error": str(e)[:200],
                            "ours_us": ours("attention")}
    del q, k, v
    return out


def cpu_baseline(w, layers_sample=1):
    """Oracle time for one batch row: `layers_sample` layers + the LM-head
    reduction over that row's draft positions, extrapolated to all layers.
    Weight generation is kept out of the timed region: the sampled layers run
    once untimed first, which generates and caches the weights of exactly the
    experts the sample routes to, then run again timed."""
    import numpy as np
    import oracle
    from oracle.refine import layer_forward, lm_head_reduce
    from workloads import make_inputs

    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    shape = w.model
    W = oracle.OracleWeights(shape, w.weight_seed, cache_layers=True)
    prompt, draft, mask = make_inputs(w, batch=1)
    tokens = np.concatenate([prompt, np.where(mask, shape.mask_id, draft)], 1).astype(np.int32)
    x0 = W.embed_rows(tokens).astype(np.float64)
    layers = [W.layer(l % shape.n_layers) for l in range(layers_sample)]
    W.lm_head()
    x = x0
    for L in layers:                           # untimed: generates the weights the sample uses
        x, _ = layer_forward(shape, L, x)
    x = x0
    t0 = time.perf_counter()
    for L in layers:
        x, _ = layer_forward(shape, L, x)
    t1 = time.perf_counter()
    lm_head_reduce(W, x[0, w.prompt_len:])
    t2 = time.perf_counter()
    per_layer = (t1 - t0) / layers_sample
    t_row = per_layer * shape.n_layers + (t2 - t1)
    return {
        "value": w.draft_len / t_row,
        "unit": "refined positions/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": (f"batch row 0 of {w.name} ({w.seq_len} tokens): {layers_sample} of {shape.n_layers} "
                   f"layers timed ({per_layer:.2f} s/layer) + LM-head reduction over {w.draft_len} draft "
                   f"positions ({t2 - t1:.2f} s), extrapolated to {shape.n_layers} layers; float64 NumPy; "
                   f"weights generated in an untimed pass of the same layers first"),
    }


def bench_local(args, w, R, tokens0):
    """Local refinement: a step is one pass over every chunk of the draft
    (prompt ‖ chunk, the chunk at its positions in the full sequence).  The
    roofline row is the gate/up expert GEMM of the chunk calls."""
    import dataclasses
    import numpy as np
    import torch
    shape = w.model
    B, P, D = w.batch, w.prompt_len, w.draft_len
    L = min(args.local_span, D)
    chunks = [(c0, torch.tensor(np.concatenate([tokens0[:, :P], tokens0[:, P + c0:P + min(c0 + L, D)]], 1),
                                device="cuda")) for c0 in range(0, D, L)]

    def one_step():
        for c0, t in chunks:
            R.refine_step_span(t, P, c0, w.threshold, w.threshold, workspace_draft_len=D)

    for _ in range(args.warmup):
        one_step()
    kname = "gemm_expert_gate_up"
    R.set_profiling(kname)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        one_step()
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / args.steps
    kt = [ms for (n, ms) in R.profile_read() if n == kname]
    R.set_profiling(None)
    flops = sum(step_flops(shape, B, P, t.shape[1] - P) for _, t in chunks)
    # launches cycle through the chunks in order (one per layer per chunk call)
    per_chunk = [kernel_flops(kname, shape, B, P, t.shape[1] - P) for _, t in chunks]
    k_flops = float(np.mean([per_chunk[(i // shape.n_layers) % len(chunks)] for i in range(len(kt))]))
    k_avg_ms = float(np.mean(kt))
    achieved = k_flops / (k_avg_ms * 1e-3) / 1e12
    out = {
        "metric": f"refined positions/sec per local refinement pass (chunks of {L})",
        "value": B * D / (ms_step * 1e-3), "unit": "refined positions/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name, "batch": B, "prompt_len": P, "draft_len": D, "local_span": L,
                   "chunks": len(chunks)},
        "step_mfma_frac": flops / (ms_step * 1e-3) / PEAK_BF16,
        "roofline": {"kernel": kname + " (chunk calls)", "bound": "mfma", "achieved": achieved,
                     "peak": PEAK_BF16 / 1e12, "unit": "TFLOP/s", "frac": achieved / (PEAK_BF16 / 1e12),
                     "traffic": None, "launches": len(kt), "avg_ms": k_avg_ms, "flops_per_launch": k_flops},
    }
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a bounded sample", file=sys.stderr, flush=True)
        cb = cpu_baseline(dataclasses.replace(w, draft_len=L))
        cb["sample"] = f"one chunk call ({P} prompt + {L} chunk tokens): " + cb["sample"]
        out["cpu_baseline"] = cb
    print(json.dumps(out), flush=True)


def cpu_baseline_draft(w, block, steps_avg):
    """Oracle time of one drafting step on block 0 of batch row 0 (prompt +
    one block under the block mask): one layer timed, extrapolated to all
    layers, plus the LM-head reduction of the block's rows; scaled to drafted
    positions per second with the GPU run's average steps per block."""
    import numpy as np
    import oracle
    from oracle.refine import layer_forward, lm_head_reduce
    from workloads import make_inputs

    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    shape = w.model
    W = oracle.OracleWeights(shape, w.weight_seed, cache_layers=True)
    prompt, _, _ = make_inputs(w, batch=1)
    P = w.prompt_len
    tokens = np.concatenate([prompt, np.full((1, block), shape.mask_id, dtype=np.int32)], 1)
    lim = oracle.block_key_limit(P, P + block, block)
    x = W.embed_rows(tokens).astype(np.float64)
    L0 = W.layer(0)
    W.lm_head()
    layer_forward(shape, L0, x, key_limit=lim)     # untimed: generates the weights the step uses
    t0 = time.perf_counter()
    x, _ = layer_forward(shape, L0, x, key_limit=lim)
    t1 = time.perf_counter()
    lm_head_reduce(W, x[0, P:])
    t2 = time.perf_counter()
    t_step = (t1 - t0) * shape.n_layers + (t2 - t1)
    return {
        "value": block / (steps_avg * t_step),
        "unit": "drafted positions/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": (f"one drafting step on block 0 of batch row 0 of {w.name} ({P} prompt + {block} block "
                   f"tokens, block-causal): 1 of {shape.n_layers} layers timed ({t1 - t0:.2f} s), LM-head "
                   f"reduction of {block} rows ({t2 - t1:.2f} s); {steps_avg:.2f} steps per block as on the "
                   f"GPU; later blocks cost the oracle more (it recomputes the prefix); float64 NumPy; weights "
                   f"generated in an untimed pass of the same layer first"),
    }


def bench_draft(args, w, R, prompt_np):
    """Block-AR drafting: a step is one whole draft of the batch (prefill of
    the prompt, then every block's denoising steps; the first step of a block
    also commits the previous block's K/V).  The dominant kernel, the
    routed-expert gate/up GEMM of a block window, streams every expert's
    weights once per launch: HBM-bound."""
    import numpy as np
    import torch
    shape = w.model
    B, P, D = w.batch, w.prompt_len, w.draft_len
    b, s, tau = args.draft_block, args.draft_steps, args.draft_threshold
    prompt = torch.tensor(prompt_np, device="cuda")
    R.draft_workspace(B, P, D, b)
    for _ in range(args.warmup):
        R.draft(prompt, D, b, s, tau)
    torch.cuda.synchronize()
    print(f"[bench] draft warmup done; timing {args.steps} drafts", file=sys.stderr, flush=True)
    kname = "gemm_expert_gate_up"
    R.set_profiling(kname)
    stats = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        _, st = R.draft(prompt, D, b, s, tau)
        stats.append(st)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    launches = [ms for (n, ms) in R.profile_read() if n == kname]
    R.set_profiling(None)
    ms_draft = (t1 - t0) * 1e3 / args.steps
    n_blocks = -(-D // b)
    steps_run = stats[-1]["steps_run"]
    L = shape.n_layers
    # per draft: prefill (layers 0..L-2 reach the experts), then steps x L
    per_call = (L - 1 if P else 0) + steps_run * L
    assert len(launches) == per_call * args.steps, (len(launches), per_call)
    win = []
    for c in range(args.steps):
        seg = launches[c * per_call:(c + 1) * per_call]
        win.extend(seg[(L - 1 if P else 0):])                 # block windows only
    k_avg_ms = float(np.mean(win))
    G = shape.n_experts + shape.n_shared_experts
    F, d = shape.expert_ffn_dim, shape.d_model

    def gu_bytes(T):                 # every expert's weights, gathered rows, output
        rows = T * (shape.top_k + shape.n_shared_experts)
        return G * 2 * F * d * 2 + rows * d * 2 + rows * F * 2

    # the first step of blocks 1.. carries two blocks of rows
    n_two = (n_blocks - 1) * L
    n_one = steps_run * L - n_two
    k_bytes = (n_one * gu_bytes(B * b) + n_two * gu_bytes(2 * B * b)) / (n_one + n_two)
    achieved = k_bytes / (k_avg_ms * 1e-3) / 1e9
    passes = (1 if P else 0) + steps_run
    out = {
        "metric": f"drafted positions/sec per block-AR draft (b{b}, s{s}, t{tau})",
        "value": B * D / (ms_draft * 1e-3), "unit": "drafted positions/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_draft, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"{w.name} draft", "batch": B, "prompt_len": P, "draft_len": D, "block_len": b,
                   "steps_per_block": s, "threshold": tau},
        "draft_stats": {"steps_run": steps_run, "block_steps": stats[-1]["block_steps"],
                        "window_passes": passes, "ms_per_window_pass": ms_draft / passes},
        "roofline": {"kernel": kname + " (block window)", "bound": "hbm", "achieved": achieved,
                     "peak": PEAK_HBM / 1e9, "unit": "GB/s", "frac": achieved / (PEAK_HBM / 1e9),
                     "traffic": None, "launches": len(win), "avg_ms": k_avg_ms, "bytes_per_launch": k_bytes},
    }
    if args.kernel_table:
        R.set_profiling("*")
        R.draft(prompt, D, b, s, tau)
        rows_ = R.profile_read()
        R.set_profiling(None)
        agg = {}
        for n, ms in rows_:
            a = agg.setdefault(n, [0, 0.0])
            a[0] += 1
            a[1] += ms
        out["kernel_table_ms"] = {n: round(v[1], 4) for n, v in sorted(agg.items(), key=lambda kv: -kv[1][1])}
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a bounded sample", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline_draft(w, b, steps_run / n_blocks)
    print(json.dumps(out), flush=True)


def bench_cascade(args, w, R, prompt_np):
    """Two-model cascade: a step is one whole dlm_cascade of the batch (block-AR
    draft with the drafter, then up to n refinement passes with the refiner).
    `value` uses the model time the library reports (drafting + refinement,
    the timing convention of Sec. 5.3 / App. A); the roofline row is the
    refiner's gate/up expert GEMM."""
    import dataclasses
    import numpy as np
    import torch
    from paper_2608_02625_amd import Refiner, cascade
    from workloads import MODELS
    shape = w.model
    B, P, D = w.batch, w.prompt_len, w.draft_len
    b, s, tau = args.draft_block, args.draft_steps, args.draft_threshold
    n_ref, t_ref = args.refine_steps, args.refine_threshold
    dshape = MODELS[args.drafter]
    print(f"[bench] drafter {args.drafter}: loading synthetic weights", file=sys.stderr, flush=True)
    Rd = Refiner(dshape.as_dict(), w.weight_seed + 1)
    prompt = torch.tensor(prompt_np, device="cuda")
    for _ in range(args.warmup):
        cascade(Rd, R, prompt, D, b, s, tau, n_ref, t_ref, t_ref)
    torch.cuda.synchronize()
    print(f"[bench] cascade warmup done; timing {args.steps} cascades", file=sys.stderr, flush=True)
    kname = "gemm_expert_gate_up"
    R.set_profiling(kname)
    stats = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        stats.append(cascade(Rd, R, prompt, D, b, s, tau, n_ref, t_ref, t_ref)[1])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    kt = [ms for (n, ms) in R.profile_read() if n == kname]
    R.set_profiling(None)
    ms_wall = (t1 - t0) * 1e3 / args.steps
    ms_model = float(np.mean([st["draft_ms"] + st["refine_ms"] for st in stats]))
    k_avg_ms = float(np.mean(kt))
    k_flops = kernel_flops(kname, shape, B, P, D)
    achieved = k_flops / (k_avg_ms * 1e-3) / 1e12
    last = stats[-1]
    out = {
        "metric": f"cascade positions/sec, draft ({args.drafter}, b{b} s{s} t{tau}) + refine ({w.name}, "
                  f"{D}x{n_ref}, t{t_ref}), model time",
        "value": B * D / (ms_model * 1e-3), "unit": "generated positions/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_wall, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"{w.name} cascade", "drafter": args.drafter, "batch": B, "prompt_len": P,
                   "draft_len": D, "block_len": b, "steps_per_block": s, "draft_threshold": tau,
                   "refine_steps": n_ref, "refine_threshold": t_ref},
        "cascade": {"model_ms": ms_model, "draft_ms": float(np.mean([st["draft_ms"] for st in stats])),
                    "refine_ms": float(np.mean([st["refine_ms"] for st in stats])),
                    "draft_passes": last["draft_passes"], "refine_passes": last["refine_passes"],
                    "passes": last["draft_passes"] + last["refine_passes"],
                    "refine_stop_reason": last["refine_stop_reason"], "refine_stats": last["refine"]},
        "roofline": {"kernel": kname + " (refiner)", "bound": "mfma", "achieved": achieved,
                     "peak": PEAK_BF16 / 1e12, "unit": "TFLOP/s", "frac": achieved / (PEAK_BF16 / 1e12),
                     "traffic": None, "launches": len(kt), "avg_ms": k_avg_ms, "flops_per_launch": k_flops},
    }
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a bounded sample", file=sys.stderr, flush=True)
        wd = dataclasses.replace(w, model=dshape, weight_seed=w.weight_seed + 1)
        cd = cpu_baseline_draft(wd, b, last["draft_passes"] / (-(-D // b)))
        cr = cpu_baseline(w)
        t_ex = D / cd["value"] + last["refine_passes"] * D / cr["value"]
        out["cpu_baseline"] = {"value": D / t_ex, "unit": "generated positions/s", "cores": cr["cores"],
                               "kind": "oracle",
                               "sample": "drafter: " + cd["sample"] + " || refiner: " + cr["sample"] +
                                         f" || combined as D / (D / draft rate + {last['refine_passes']} x D / "
                                         f"refine rate) for one row"}
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="mini_moe")
    ap.add_argument("--batch", type=int, default=0, help="override the workload's batch size")
    ap.add_argument("--kernel", default="gemm_expert_gate_up", help="kernel reported in roofline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--kernel-table", action="store_true", help="also time every kernel (separate pass)")
    ap.add_argument("--library-reference", action="store_true",
                    help="also time torch.matmul / scaled_dot_product_attention on the pass's shapes")
    ap.add_argument("--local-span", type=int, default=0,
                    help="time local refinement instead: one pass over every draft chunk of this many tokens")
    ap.add_argument("--draft", action="store_true",
                    help="time block-AR drafting of the workload's draft length instead")
    ap.add_argument("--draft-block", type=int, default=64)
    ap.add_argument("--draft-steps", type=int, default=16)
    ap.add_argument("--draft-threshold", type=float, default=0.25)
    ap.add_argument("--cascade", action="store_true",
                    help="time the two-model cascade (drafter --drafter, refiner = the workload's model)")
    ap.add_argument("--drafter", default="mini_drafter")
    ap.add_argument("--refine-steps", type=int, default=4)
    ap.add_argument("--refine-threshold", type=float, default=0.20)
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="first run a plain device copy of this many MiB (reference for memory counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}); multi-GPU sharding is not built",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2608_02625_amd import Refiner
    from workloads import WORKLOADS, make_inputs

    w = WORKLOADS[args.workload]
    if args.batch:
        import dataclasses
        w = dataclasses.replace(w, batch=args.batch)
    shape = w.model
    B, P, D = w.batch, w.prompt_len, w.draft_len
    torch.cuda.set_device(0)
    if args.calibrate_copy_mib:
        # A plain elementwise pass (float32 negation) that reads and writes
        # exactly this many MiB: the reference against which the memory
        # counters of the other kernels are scaled.
        n = (args.calibrate_copy_mib << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst
    print(f"[bench] workload {w.name}: B={B} P={P} D={D}; loading synthetic weights", file=sys.stderr, flush=True)
    R = Refiner(shape.as_dict(), w.weight_seed)
    prompt, draft, mask = make_inputs(w)
    tokens0 = np.concatenate([prompt, np.where(mask, shape.mask_id, draft)], 1).astype(np.int32)
    tokens = torch.tensor(tokens0, device="cuda")
    R.workspace(B, P, D)
    torch.cuda.synchronize()

    if args.local_span:
        bench_local(args, w, R, tokens0)
        return
    if args.draft:
        bench_draft(args, w, R, prompt.astype(np.int32))
        return
    if args.cascade:
        bench_cascade(args, w, R, prompt.astype(np.int32))
        return
    for _ in range(args.warmup):
        R.refine_step(tokens, P, w.threshold)
    torch.cuda.synchronize()
    print(f"[bench] warmup done; timing {args.steps} steps", file=sys.stderr, flush=True)

    R.set_profiling(args.kernel)
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record()
    for _ in range(args.steps):
        R.refine_step(tokens, P, w.threshold)
    ev1.record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    launches = R.profile_read()
    R.set_profiling(None)
    wall = t1 - t0
    ms_step = wall * 1e3 / args.steps
    ev_ms_step = ev0.elapsed_time(ev1) / args.steps

    flops = step_flops(shape, B, P, D)
    kt = [ms for (n, ms) in launches if n == args.kernel]
    k_avg_ms = float(np.mean(kt)) if kt else float("nan")
    k_flops = kernel_flops(args.kernel, shape, B, P, D)
    achieved = k_flops / (k_avg_ms * 1e-3) / 1e12
    out = {
        "metric": METRIC,
        "value": B * D / (ms_step * 1e-3),
        "unit": "refined positions/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "batch": B, "prompt_len": P, "draft_len": D,
                   "n_layers": shape.n_layers, "d_model": shape.d_model, "n_experts": shape.n_experts,
                   "top_k": shape.top_k, "vocab": shape.vocab, "threshold": w.threshold},
        "step_mfma_frac": flops / (ms_step * 1e-3) / PEAK_BF16,
        "step_tflops": flops / (ms_step * 1e-3) / 1e12,
        "event_ms_per_step": ev_ms_step,
        "roofline": {"kernel": args.kernel, "bound": "mfma", "achieved": achieved, "peak": PEAK_BF16 / 1e12,
                     "unit": "TFLOP/s", "frac": achieved / (PEAK_BF16 / 1e12),
                     "traffic": recorded_traffic(args.kernel, w.name),
                     "launches": len(kt), "avg_ms": k_avg_ms, "flops_per_launch": k_flops},
    }
    if args.kernel_table or args.library_reference:
        R.set_profiling("*")
        R.refine_step(tokens, P, w.threshold)
        rows = R.profile_read()
        R.set_profiling(None)
        agg = {}
        for n, ms in rows:
            a = agg.setdefault(n, [0, 0.0])
            a[0] += 1
            a[1] += ms
        if args.kernel_table:
            out["kernel_table_ms"] = {n: round(v[1], 4) for n, v in sorted(agg.items(), key=lambda kv: -kv[1][1])}
        if args.library_reference:
            print("[bench] timing the vendor libraries on the same shapes", file=sys.stderr, flush=True)
            out["library_reference"] = library_reference(shape, B, P, D, rows)
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a bounded sample", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(w)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
