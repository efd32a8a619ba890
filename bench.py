#!/usr/bin/env python3
"""Throughput of the FL-GLM server stack on one MI355X.

One step = the server's whole hot path over one client batch: forward through
the N server blocks, then backward (returning every client's input gradient
and accumulating fp32 weight gradients), all through the C ABI
(fl_server_stack_forward / fl_server_stack_backward).  Inputs are resident in
HBM before the timed region; weights, activations and upstream gradients are
seeded synthetic draws with the workload's shapes and distributions.

Prints one JSON line: tokens/s of the whole step, the fraction of the bf16
matrix-core peak it reaches, a per-kernel-class breakdown (HIP events around
every launch during the timed steps), the roofline entry of the dominant
kernel class, and the CPU oracle timed on a bounded sample of the same
workload on this host's cores.
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

import numpy as np  # noqa: E402

import synth  # noqa: E402

DEFAULT_WORKLOAD = "chatglm6b_26blk_ragged_32x1_recompute"
PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}   # dense matrix-core peaks, MI355X
PEAK_HBM_GBS = 8000.0
METRIC = "server-stack fwd+bwd tokens/sec and MFMA util %, ChatGLM-6B shape"
MFMA_CLASSES = ("gemm_nt_bias", "gemm_nt_bias_res", "gemm_nt_bias_gelu", "gemm_tn_acc", "gemm_nn_gelu_bwd",
                "gemm_nn", "attn_fwd", "attn_bwd")
GEMM_CLASSES = MFMA_CLASSES[:6]


def algorithmic_flops(w: synth.Workload, b: synth.Batch) -> dict:
    """Per step: GEMM 24 H^2 per token per block forward, 48 H^2 backward;
    attention 4 H per visible (query, key) pair forward, 8 H backward.
    Recomputation is not counted."""
    H = w.shape.hidden
    T = b.total_tokens
    pairs = 0.0
    for s in range(b.num_seqs):
        L = float(b.seqlens[s])
        P = float(b.prefix_len[s]) if b.mask == "prefix" else 0.0
        pairs += L * (L + 1) / 2 + (P * (P - 1) / 2 if P > 1 else 0.0)
    mult_g = 72 if w.backward else 24
    mult_a = 12 if w.backward else 4
    g = mult_g * H * H * T * w.shape.num_layers
    a = mult_a * H * pairs * w.shape.num_layers
    return {"gemm": g, "attention": a, "total": g + a, "pairs": pairs}


def device_inputs(w: synth.Workload, b: synth.Batch, seed: int):
    """Seeded device-side draws (torch Philox on the GPU) with the workload's
    distributions: weights and biases N(0, 0.02), LayerNorm gains 1 + N(0, 0.02),
    x ~ N(0, 1), dy ~ N(0, dy_std); rounded to bf16 for bf16 workloads."""
    import torch
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    shapes = synth.param_shapes(w.shape)
    gen = torch.Generator(device="cuda")
    params, grads = [], []
    for l in range(w.shape.num_layers):
        gen.manual_seed(seed * 100003 + l)
        p = {}
        for name, shp in shapes.items():
            t = torch.randn(shp, generator=gen, device="cuda", dtype=torch.float32) * 0.02
            if name in ("ln1_g", "ln2_g"):
                t += 1.0
            p[name] = t.to(dt)
            del t
        params.append(p)
        grads.append({k: torch.zeros(v.shape, dtype=torch.float32, device="cuda") for k, v in p.items()})
    gen.manual_seed(seed * 100003 + 99991)
    T, H = b.total_tokens, w.shape.hidden
    x = torch.randn((T, H), generator=gen, device="cuda", dtype=torch.float32).to(dt)
    dy = (torch.randn((T, H), generator=gen, device="cuda", dtype=torch.float32) * w.dy_std).to(dt)
    return params, grads, x, dy


def cpu_baseline(w: synth.Workload, b: synth.Batch, budget_s: float) -> dict:
    """The CPU oracle (float64, numpy BLAS) on a bounded sample: one block's
    forward + recompute + backward over whole sequences of the workload,
    shortest first, until the budget is used; scaled to the full stack depth."""
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max((i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"),
                      default=1)
    except Exception:  # pragma: no cover
        threads = len(os.sched_getaffinity(0))
    one = synth.StackShape(1, w.shape.hidden, w.shape.num_heads, w.shape.ffn_hidden, w.shape.rotary_dim,
                           w.shape.rope_base, w.shape.ln_eps)
    layer = synth.layer_params(w.shape, 0, seed=0, bf16=w.dtype == "bf16")
    order = np.argsort(b.seqlens, kind="stable")
    done_tokens, spent = 0, 0.0
    seqs = []
    for s in order:
        sub = synth.Batch(np.array([0, int(b.seqlens[s])], np.int32), np.array([0, 1], np.int32), b.mask,
                          None if b.prefix_len is None else np.array([int(b.prefix_len[s])], np.int32))
        L = sub.total_tokens
        x = synth.activations(L, w.shape.hidden, seed=1, bf16=w.dtype == "bf16")
        dy = synth.upstream_grad(L, w.shape.hidden, seed=1, bf16=w.dtype == "bf16", std=w.dy_std)
        t0 = time.perf_counter()
        y, xs = oracle.stack_forward([layer], 1, x, sub, one)
        if w.backward:
            oracle.stack_backward([layer], 1, xs, dy, sub, one)
        spent += time.perf_counter() - t0
        done_tokens += L
        seqs.append(L)
        if spent >= budget_s:
            break
    per_block_tok_s = done_tokens / spent
    return {
        "value": per_block_tok_s / w.shape.num_layers,
        "unit": "tokens/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": (f"1 of {w.shape.num_layers} blocks, {'fwd+recompute+bwd' if w.backward else 'fwd'}, float64, "
                   f"{len(seqs)} whole sequence(s) of lengths {seqs} ({done_tokens} tokens) in {spent:.1f} s; "
                   f"tokens/s divided by {w.shape.num_layers} blocks"),
    }


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD, choices=sorted(synth.WORKLOADS))
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-budget", type=float, default=15.0, help="seconds of CPU oracle work")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true", help="time without per-launch events")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(json.dumps({"error": "this build runs the server stack on one GPU only; "
                                   f"--gpus {args.gpus} is not supported (multi-GPU sharding is design-only)"}))
        return 2

    import torch

    from paper_2406_14898_amd import BatchDesc, ServerStack
    from paper_2406_14898_amd import flglm as F

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    w = synth.WORKLOADS[args.workload]
    b = w.batch(seed=args.seed)
    T = b.total_tokens
    print(f"[bench] workload {w.name}: T={T} S={b.num_seqs} C={b.num_clients} maxL={b.max_seqlen}", file=sys.stderr,
          flush=True)
    params, grads, x, dy = device_inputs(w, b, args.seed)
    ss = ServerStack(w.shape.num_layers, w.shape.hidden, w.shape.num_heads, w.shape.ffn_hidden, w.shape.rotary_dim,
                     w.dtype, w.shape.rope_base, w.shape.ln_eps)
    bd = BatchDesc.from_batch(b)
    saved, ws = ss.buffers(bd, w.recompute, with_saved=w.backward)
    y = torch.empty_like(x)
    dx = torch.empty_like(x) if w.backward else None
    stream = torch.cuda.current_stream()

    def step():
        ss.forward(bd, params, x, y, saved, ws, w.recompute, stream)
        if w.backward:
            ss.backward(bd, params, grads, x, saved, dy, dx, ws, w.recompute, stream)

    for i in range(args.warmup):
        step()
        torch.cuda.synchronize()
        print(f"[bench] warmup step {i + 1}/{args.warmup} done", file=sys.stderr, flush=True)
    F.fl_stack_profile(ss.handle, not args.no_profile)
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for i in range(args.steps):
        step()
    end.record(stream)
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / args.steps
    prof = F.profile_table(ss.handle)
    F.fl_stack_profile(ss.handle, False)
    print(f"[bench] timed {args.steps} steps: {ms:.2f} ms/step", file=sys.stderr, flush=True)

    flops = algorithmic_flops(w, b)
    peak = PEAK_TFLOPS[w.dtype]
    tok_s = T / (ms / 1e3)
    kernels = {}
    for name, r in sorted(prof.items(), key=lambda kv: -kv[1]["ms"]):
        per_ms = r["ms"] / r["launches"]
        ent = {"launches": r["launches"], "ms_per_step": round(r["ms"] / args.steps, 3),
               "avg_launch_us": round(per_ms * 1e3, 2)}
        if r["flops"] > 0:
            ent["tflops"] = round(r["flops"] / (r["ms"] / 1e3) / 1e12, 1)
        if r["bytes"] > 0 and name not in MFMA_CLASSES:
            ent["gbs"] = round(r["bytes"] / (r["ms"] / 1e3) / 1e9, 1)
        kernels[name] = ent
    gemm_ms = sum(prof[k]["ms"] for k in GEMM_CLASSES if k in prof)
    gemm_fl = sum(prof[k]["flops"] for k in GEMM_CLASSES if k in prof)
    roofline = None
    if prof:
        dom = max(prof, key=lambda k: prof[k]["ms"])
        r = prof[dom]
        avg_s = r["ms"] / r["launches"] / 1e3
        if dom in MFMA_CLASSES:
            ach = r["flops"] / r["launches"] / avg_s / 1e12
            roofline = {"kernel": dom, "bound": "mfma", "achieved": round(ach, 1), "peak": peak, "unit": "TFLOP/s",
                        "frac": round(ach / peak, 4), "traffic": None}
        else:
            ach = r["bytes"] / r["launches"] / avg_s / 1e9
            roofline = {"kernel": dom, "bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS,
                        "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBS, 4), "traffic": None}

    out = {
        "metric": METRIC,
        "value": round(tok_s, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded device draws: weights N(0,0.02), x N(0,1), dy N(0,%g))" % w.dy_std,
        "config": {"workload": w.name, "clients": b.num_clients, "seqs": b.num_seqs, "total_tokens": T,
                   "max_seqlen": b.max_seqlen, "blocks": w.shape.num_layers, "hidden": w.shape.hidden,
                   "heads": w.shape.num_heads, "ffn": w.shape.ffn_hidden, "mask": w.mask,
                   "backward": w.backward, "recompute": w.recompute, "parallelism": "single GPU"},
        "mfma_util": round(flops["total"] / (ms / 1e3) / (peak * 1e12), 4),
        "gemm_mfma_util": round(gemm_fl / (gemm_ms / 1e3) / (peak * 1e12), 4) if gemm_ms else None,
        "algorithmic_tflop_per_step": round(flops["total"] / 1e12, 3),
        "roofline": roofline,
        "kernels": kernels,
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a bounded sample", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(w, b, args.cpu_budget)
    ss.close()
    print(json.dumps(out))
    return 0


if __name__ == "__main__":
    sys.exit(main())
