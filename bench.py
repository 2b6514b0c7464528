#!/usr/bin/env python3
"""Throughput of the M2R2 dual-stream decode step on one MI355X.

Workload (default): a Phi-3-mini-shaped dense decoder (32 layers, d_model 3072,
32 heads x 96, SwiGLU 8192, vocab 32064), bfloat16 weights and KV cache,
accelerator adapters of rank 16 on all seven projections, batch 1.  Weights
are seeded N(0, 0.02) (norm gains 1.0); a 1024-token random prompt is
prefilled through the chunked slow forward.  One step = one dual-stream decode
step: embedding, 32 layers carrying the slow and the fast row (shared paged
KV cache, exit signal at every layer, OBSERVE-mode gates at every interior
boundary, tau 0.9), final norm, LM head and argmax.  The step is captured in a
HIP graph and replayed; inputs are resident in HBM before timing starts.

Prints one JSON line (see the repository's design notes for every field).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

HBM_PEAK_GBS = 8000.0


def step_bytes(cfg, ctx: float, dual: bool = True) -> float:
    """Algorithmic HBM bytes of one decode step at context length ctx."""
    d, q, F, V, r, L = cfg.d_model, cfg.qdim, cfg.ffn, cfg.vocab, cfg.rank, cfg.n_layers
    ew = 2 if cfg.wdtype == "bf16" else 4
    ek = 2 if cfg.kvdtype == "bf16" else 4
    mats = (3 * q * d + d * q + 2 * F * d + d * F) * ew
    adapters = r * ((d + q) * 3 + (q + d) + (d + F) * 2 + (F + d)) * ew if dual else 0
    norms = 2 * d * 4
    kv = (ctx * 2 * q + 2 * q) * ek
    per_layer = mats + adapters + norms + kv
    return L * per_layer + V * d * ew + d * 4 + d * ew


def gateup_bytes(cfg, dual: bool = True) -> float:
    """Algorithmic bytes of one gate/up launch: both weight matrices, the
    adapter factors it reads (B_g, B_u, and the columns of A_d for the down
    adapter's partial sums), the input rows and the activation it writes."""
    d, F, r = cfg.d_model, cfg.ffn, cfg.rank
    ew = 2 if cfg.wdtype == "bf16" else 4
    rows = 2 if dual else 1
    return 2 * F * d * ew + (3 * F * r * ew if dual else 0) + rows * (d * 4 + F * 4) + d * 4


def cpu_baseline(cfg, weights, ctx: int, budget_s: float):
    """Time the CPU oracle (float32) on the same decode step at the same
    context length; its cache is filled with seeded synthetic content."""
    import synth
    from oracle import Oracle, KVCache
    from threadpoolctl import threadpool_info
    orc = Oracle(cfg, weights, np.float32)
    cache = KVCache(cfg, ctx + 64, np.float32)
    kvs = synth.synthetic_kv(cfg, ctx)
    for l, (K, V) in kvs.items():
        cache.load(l, K, V)
    del kvs
    gates = list(range(1, cfg.n_layers))
    tok, n, t0 = 1, 0, time.perf_counter()
    while True:
        r = orc.decode_step(tok, ctx + n, cache, gates=gates, tau=0.9, mode="observe")
        tok = r.token
        n += 1
        el = time.perf_counter() - t0
        if el >= budget_s or n >= 64:
            break
    threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    return dict(value=n / el, unit="tokens/s", cores=int(threads), kind="oracle",
                sample=f"{n} dual-stream decode steps of the same model in float32 NumPy at context {ctx} "
                       f"(synthetic cache content), {el:.1f} s")


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=256)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="phi3")
    ap.add_argument("--ctx", type=int, default=1024)
    ap.add_argument("--single", action="store_true", help="slow row only (plain decoding on the same kernels)")
    ap.add_argument("--kernel-reps", type=int, default=20, help="graph replays of the instrumented step")
    ap.add_argument("--cpu-budget", type=float, default=20.0, help="seconds of CPU oracle timing (0: skip)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: --gpus {args.gpus} is not supported by this build "
              f"(the multi-GPU sharding is a design note, not an implementation)", file=sys.stderr)
        return 2

    import torch
    import synth
    from paper_2502_02040_amd import Model, PagedKV

    cfg = synth.CONFIGS[args.config]
    dual = not args.single
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    t_setup = time.perf_counter()
    weights = synth.make_weights(cfg)
    n_inst = 2 * args.kernel_reps
    max_ctx = args.ctx + args.warmup + args.steps + n_inst + 32
    model = Model(cfg, weights, max_batch=1, max_chunk=16, max_ctx=max_ctx)
    bps = (max_ctx + 15) // 16
    kv = PagedKV(cfg, 1, max_ctx, block_size=16, block_table=synth.block_table(1, bps, seed=cfg.seed))
    desc = kv.desc()

    # prefill the prompt through the chunked slow forward
    prompt = synth.prompt_ids(cfg, args.ctx)
    pos = torch.zeros(1, dtype=torch.int32, device=dev)
    targets = torch.zeros(16, dtype=torch.int32, device=dev)
    chunk = torch.tensor(prompt, dtype=torch.int32, device=dev)
    for c0 in range(0, args.ctx, 16):
        n = min(16, args.ctx - c0)
        model.verify(chunk[c0:c0 + n], n, pos, desc, targets)
    torch.cuda.synchronize()
    tok = targets[(args.ctx - 1) % 16:(args.ctx - 1) % 16 + 1].clone()

    N = cfg.n_layers
    gates = list(range(1, N)) if dual else []
    sig = torch.zeros(N, dtype=torch.float32, device=dev)
    exb = torch.zeros(1, dtype=torch.int32, device=dev)
    stream = torch.cuda.Stream()

    def step():
        model.decode_step(tok, pos, desc, dual=dual, gates=gates, tau=0.9, mode="observe", next_token=tok,
                          exit_boundary=exb if dual else None, signal=sig if dual else None, advance=True)

    with torch.cuda.stream(stream):
        for _ in range(args.warmup):
            step()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        step()
    torch.cuda.synchronize()
    setup_s = time.perf_counter() - t_setup

    ctx0 = int(pos.item())
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        e0.record(stream)
        for _ in range(args.steps):
            g.replay()
        e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    ms_step = ms / args.steps
    ctx_mean = ctx0 + (args.steps - 1) / 2.0

    # dominant kernel (gate/up projection): HIP events recorded on the launch
    # stream around each of its launches in further steps of the same decode
    # (launched directly: HIP does not time events recorded inside a graph)
    model.timing_enable("gateup")
    with torch.cuda.stream(stream):
        for _ in range(args.kernel_reps):
            step()
    k_ms, k_n = model.timing_read()
    model.timing_enable(None)
    errs = model.device_errors()
    if errs:
        print(f"device error bits {errs}", file=sys.stderr)
        return 1
    k_avg_ms = k_ms / max(k_n, 1)
    kb = gateup_bytes(cfg, dual)
    achieved = kb / (k_avg_ms * 1e-3) / 1e9
    sb = step_bytes(cfg, ctx_mean, dual)
    step_gbs = sb / (ms_step * 1e-3) / 1e9

    cpu = None
    if args.cpu_budget > 0:
        cpu = cpu_baseline(cfg, weights, args.ctx, args.cpu_budget)

    line = {
        "metric": "decode tokens/s at batch 1 + achieved HBM GB/s of dual-stream layer step",
        "value": round(1000.0 / ms_step, 3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if cfg.wdtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": f"{'dual' if dual else 'single'}-stream decode step, {cfg.name}-shaped "
                               f"{cfg.n_layers}L d{cfg.d_model} {cfg.n_heads}x{cfg.head_dim} ffn{cfg.ffn} "
                               f"vocab{cfg.vocab} rank{cfg.rank}, {cfg.wdtype} weights/KV, batch 1, "
                               f"KV context {args.ctx} (+{args.warmup + args.steps} decoded), HIP graph replay",
                   "batch": 1, "kv_context": args.ctx, "dual_stream": dual},
        "step_hbm_gbs": round(step_gbs, 1),
        "step_bytes": int(sb),
        "step_roofline_frac": round(step_gbs / HBM_PEAK_GBS, 4),
        "roofline": {"bound": "hbm", "kernel": "gate/up projection (k_gateup)",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                     "avg_kernel_us": round(k_avg_ms * 1e3, 3), "bytes_per_launch": int(kb),
                     "launches_timed": k_n},
        "cpu_baseline": cpu,
        "setup_s": round(setup_s, 1),
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
