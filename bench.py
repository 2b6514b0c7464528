#!/usr/bin/env python3
"""Throughput of the M2R2 decode path on one MI355X.

Default workload (``--mode dense``): a Phi-3-mini-shaped dense decoder (32
layers, d_model 3072, 32 heads x 96, SwiGLU 8192, vocab 32064), bfloat16
weights and KV cache, accelerator adapters of rank 16 on all seven
projections, batch 1.  Weights are seeded N(0, 0.02) (norm gains 1.0); a
1024-token random prompt is prefilled through the chunked slow forward.  One
step = one dual-stream decode step: embedding, 32 layers carrying the slow
and the fast row (shared paged KV cache, exit signal at every layer,
OBSERVE-mode gates at every interior boundary, tau 0.9), final norm, LM head
and argmax.  The step is captured in a HIP graph and replayed; inputs are
resident in HBM before timing starts.  Prints one JSON line.

Other measurements (one JSON line each, same fields where they apply):
  --mode batch  the same model, 8 sequences with 4096-token paged contexts
                (block 16, shuffled block table, seeded synthetic cache content)
  --mode spec   self-speculative decoding: drafts of 4 tokens from the fast
                stream exiting at layer 8, verified as 5-token chunks on the
                slow stream; 512 tokens from a 128-token prompt, against plain
                greedy decoding on the same kernels (and the token streams are
                checked to be equal)
  --mode exit   EXIT-mode dynamic compute: the dual-stream step with gates at
                every interior boundary in EXIT mode, for a sweep of exit
                thresholds tau (the token comes from the fast row at the first
                gate whose signal reaches tau; the skipped layers only fill
                their cache entries from the slow row), tokens/s against the
                mean exit boundary; --gate-every K puts the gates every K
                layers, --arla decides them with the latent-attention exit
                router (seeded synthetic weights)
  --mode moe    OLMoE-shaped mixture of experts (16 layers, d 2048, 64 experts
                of width 1024, top 8, vocab 50304) with every expert in pinned
                host memory and a 16-slot HBM cache per layer, fed a
                teacher-forced Zipf token stream: the five placement
                strategies of the paper's comparison (fixed experts, LRU, LRU
                with random preload, previous-layer speculation on the slow
                stream alone; M2R2 ahead-of-time prefetch from the fast
                stream) and an all-resident cache, with per-layer miss rates
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

HBM_PEAK_GBS = 8000.0
METRIC = "decode tokens/s at batch 1 + achieved HBM GB/s of dual-stream layer step"


# ----------------------------------------------------------------------------
# algorithmic bytes
# ----------------------------------------------------------------------------

def layer_weight_bytes(cfg, dual: bool = True) -> float:
    d, q, F, r = cfg.d_model, cfg.qdim, cfg.ffn, cfg.rank
    ew = 2 if cfg.wdtype == "bf16" else 4
    mats = (3 * q * d + d * q + 2 * F * d + d * F) * ew
    if getattr(cfg, "fast_mlp_adapter", False):
        # FLOPs-optimised fast stream: q, k, v, o adapters and the MLP adapter
        # (its selected keys/values are cache bytes the slow row reads anyway)
        adapters = r * ((d + q) * 3 + (q + d) + 2 * d) * ew if dual else 0
    else:
        adapters = r * ((d + q) * 3 + (q + d) + (d + F) * 2 + (F + d)) * ew if dual else 0
    return mats + adapters + 2 * d * 4


def step_bytes(cfg, ctx: float, dual: bool = True, batch: int = 1) -> float:
    """Algorithmic HBM bytes of one decode step: every weight once, the KV
    cache of every sequence once (context ctx each), the new KV entries."""
    d, q, V, L = cfg.d_model, cfg.qdim, cfg.vocab, cfg.n_layers
    ew = 2 if cfg.wdtype == "bf16" else 4
    ek = 2 if cfg.kvdtype == "bf16" else 4
    kv = batch * (ctx * 2 * q + 2 * q) * ek
    return L * (layer_weight_bytes(cfg, dual) + kv) + V * d * ew + d * 4 + batch * d * ew


def gateup_bytes(cfg, rows: int, fast_rows: int) -> float:
    """Algorithmic bytes of one gate/up launch: both weight matrices, the
    adapter factors it reads (B_g, B_u, and the columns of A_d for the down
    adapter's partial sums) when fast rows are present, the input rows and the
    activations it writes."""
    d, F, r = cfg.d_model, cfg.ffn, cfg.rank
    ew = 2 if cfg.wdtype == "bf16" else 4
    return 2 * F * d * ew + (3 * F * r * ew if fast_rows else 0) + rows * (d * 4 + F * 4) + d * 4


def attn_bytes(cfg, batch: int, ctx: float) -> float:
    """Algorithmic bytes of one attention launch: the cached keys and values
    of every sequence plus the new entries."""
    ek = 2 if cfg.kvdtype == "bf16" else 4
    return batch * (ctx + 1) * 2 * cfg.qdim * ek


def expert_gateup_bytes(cfg) -> float:
    ew = 2 if cfg.wdtype == "bf16" else 4
    return cfg.top_k * 2 * cfg.expert_ffn * cfg.d_model * ew + cfg.d_model * 4 * 2 + cfg.top_k * cfg.expert_ffn * 4


def moe_token_bytes(cfg, ctx: float) -> float:
    """HBM bytes of one MoE decode token with every chosen expert resident:
    attention weights, KV, the router, the k experts, the LM head."""
    d, q, L, r = cfg.d_model, cfg.qdim, cfg.n_layers, cfg.rank
    ew = 2 if cfg.wdtype == "bf16" else 4
    ek = 2 if cfg.kvdtype == "bf16" else 4
    attn = (3 * q * d + d * q) * ew + (ctx * 2 * q + 2 * q) * ek
    experts = cfg.top_k * 3 * cfg.expert_ffn * d * ew + cfg.n_experts * d * ew
    return L * (attn + experts + 2 * d * 4) + cfg.vocab * d * ew


# ----------------------------------------------------------------------------
# measured HBM traffic (profiler byte counters), valid for the sources it was
# taken from
# ----------------------------------------------------------------------------

ROOT = os.path.dirname(os.path.abspath(__file__))
GATEUP_COUNTERS = "kr_gateup_phi3_dual_ctx1024_hbm_counters.md"
STEP_COUNTERS = "kp_step_phi3_dual_ctx1024_hbm_counters.md"


def sources_digest() -> str:
    """sha256 over the HIP sources and the C header the library is built from."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2502_02040_amd", "csrc")
    files = [os.path.join(csrc, f) for f in sorted(os.listdir(csrc)) if f.endswith((".h", ".hip"))]
    files.append(os.path.join(ROOT, "include", "m2r2.h"))
    for f in files:
        h.update(os.path.basename(f).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def stored_traffic(name: str):
    """HBM bytes per launch recorded in profiles/<name> (FETCH_SIZE and
    WRITE_SIZE per dispatch, each scaled by a copy-kernel calibration), or
    None when the file is missing or the sources changed since the counters
    were taken."""
    path = os.path.join(ROOT, "profiles", name)
    if not os.path.exists(path):
        return None
    fields = {}
    with open(path) as fh:
        for line in fh:
            if ":" in line and line.split(":", 1)[0].strip() in ("sources_sha256", "hbm_bytes_per_launch"):
                k, v = line.split(":", 1)
                fields[k.strip()] = v.strip().strip("`")
    if fields.get("sources_sha256") != sources_digest() or "hbm_bytes_per_launch" not in fields:
        return None
    return int(float(fields["hbm_bytes_per_launch"]))


# ----------------------------------------------------------------------------
# CPU baseline: the oracle timed on the host cores
# ----------------------------------------------------------------------------

def _blas():
    """BLAS threads NumPy uses (the cores the oracle runs on) and the BLAS
    library behind it."""
    from threadpoolctl import threadpool_info
    b = [i for i in threadpool_info() if i.get("user_api") == "blas"]
    threads = max([i.get("num_threads", 1) for i in b] or [1])
    names = sorted({f"{i.get('internal_api', '?')} {i.get('version') or ''}".strip() for i in b})
    return int(threads), ", ".join(names) or "none"


def _cpu_line(value: float, unit: str, sample: str, **extra) -> dict:
    threads, blas = _blas()
    d = dict(value=value, unit=unit, cores=threads, kind="oracle", sample=sample, host_cpus=os.cpu_count(), blas=blas)
    d.update(extra)
    return d


def cpu_baseline(cfg, weights, ctx: int, budget_s: float, *, seqs: int = 1):
    """Time the CPU oracle (float32) on the same decode step at the same
    context length; its cache is filled with seeded synthetic content.  With
    seqs > 1 (a batch of independent sequences) the oracle steps one of them:
    its sequences run one after another on the same cores, so the aggregate
    rate is the per-sequence rate."""
    import synth
    from oracle import Oracle, KVCache
    orc = Oracle(cfg, weights, np.float32)
    room = 256   # decode steps the cache has room for (each step appends one position)
    cache = KVCache(cfg, ctx + room, np.float32)
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
        if el >= budget_s or n >= room:
            break
    what = f"one of the {seqs} sequences' " if seqs > 1 else ""
    return _cpu_line(n / el, "tokens/s", f"{n} dual-stream decode steps of {what}the same model in float32 NumPy at "
                                         f"context {ctx} (synthetic cache content), {el:.1f} s")


def cpu_moe_baseline(cfg, ctx: int, budget_s: float):
    """The oracle (float32) on one dual-stream MoE decode step at context ctx
    with every expert available (the step as the method defines it, its
    expert placement aside).  Expert weights are generated on first use: an
    untimed first run generates the experts the step routes to, then the
    same step (same token and position) is repeated for the budget."""
    import synth
    from oracle import Oracle, KVCache
    spec = {n: (sh, k) for n, sh, k in synth.tensor_specs(cfg)}
    orc = Oracle(cfg, synth.make_weights(cfg, names=[n for n in spec if ".E" not in n]), np.float32)

    class Lazy(dict):
        def __missing__(self, name):
            sh, kind = spec[name]
            v = np.asarray(synth.make_tensor(cfg, name, sh, kind), np.float32)
            self[name] = v
            return v

    orc.w = Lazy(orc.w)
    cache = KVCache(cfg, ctx + 8, np.float32)
    for l, (K, V) in synth.synthetic_kv(cfg, ctx).items():
        cache.load(l, K, V)
    orc.decode_step(1, ctx, cache)   # untimed: generates the routed experts
    n, t0 = 0, time.perf_counter()
    while True:
        orc.decode_step(1, ctx, cache)
        n += 1
        el = time.perf_counter() - t0
        if el >= budget_s or n >= 4096:
            break
    return _cpu_line(n / el, "tokens/s", f"one dual-stream MoE decode step in float32 NumPy at context {ctx} (every "
                                         f"expert available), repeated {n} times in {el:.1f} s after an untimed first "
                                         f"run that generated the experts it routes to")


def cpu_spec_baseline(cfg, weights, plen: int, gamma: int, exit_layer: int, budget_s: float):
    """The oracle (float32) on the speculative workload: greedy decoding after
    the prompt, then draft + verify rounds from there, each for half the
    budget; returns the speculative rate with the greedy rate beside it."""
    import synth
    from oracle import Oracle, KVCache
    from oracle.decoder import argmax_first
    orc = Oracle(cfg, weights, np.float32)
    cache = KVCache(cfg, plen + 64 * (gamma + 2) + 64, np.float32)
    tok = argmax_first(orc.slow_chunk(list(synth.prompt_ids(cfg, plen)), 0, cache)[-1])
    pos, n, t0 = plen, 0, time.perf_counter()
    while True:
        tok = argmax_first(orc.slow_chunk([tok], pos, cache)[-1])
        pos, n = pos + 1, n + 1
        el_g = time.perf_counter() - t0
        if el_g >= budget_s / 2 or n >= 32:
            break
    toks = rounds = 0
    t0 = time.perf_counter()
    while True:
        d = orc.draft(tok, pos, cache, exit_layer, gamma)
        y = [argmax_first(z) for z in orc.slow_chunk([tok] + d, pos, cache)]
        a = 0
        while a < gamma and d[a] == y[a]:
            a += 1
        tok = y[a]
        pos, toks, rounds = pos + a + 1, toks + a + 1, rounds + 1
        el_s = time.perf_counter() - t0
        if el_s >= budget_s / 2 or rounds >= 16:
            break
    return _cpu_line(toks / el_s, "tokens/s",
                     f"float32 NumPy after a {plen}-token prompt: {n} greedy tokens in {el_g:.1f} s, then {rounds} "
                     f"draft+verify rounds (gamma {gamma}, exit layer {exit_layer}) giving {toks} tokens in {el_s:.1f} s",
                     greedy_value=round(n / el_g, 3))


# ----------------------------------------------------------------------------
# shared helpers
# ----------------------------------------------------------------------------

def dense_capacity(ctx: int, warmup: int, steps: int, kernel_reps: int) -> int:
    """Cache capacity (max_ctx) of the dense and exit runs: room for the
    decoded tokens, rounded up to a multiple of 512 past the prompt, so that
    runs of different lengths share one launch configuration (the parity test
    of the benched configuration builds its model with this capacity)."""
    need = ctx + warmup + steps + 2 * kernel_reps + 32
    return max(ctx + 512, (need + 511) // 512 * 512)


def _progress(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def _line(**kw):
    base = {"metric": METRIC, "n_gpus": 1, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
            "data": "synthetic"}
    base.update(kw)
    print(json.dumps(base), flush=True)


def _prefill(model, prompt, pos, desc, dev):
    """Chunked slow forward of the prompt (chunks of 16); returns the first token."""
    import torch
    targets = torch.zeros(16, dtype=torch.int32, device=dev)
    chunk = torch.tensor(np.asarray(prompt, np.int32), dtype=torch.int32, device=dev)
    n_all = len(prompt)
    for c0 in range(0, n_all, 16):
        n = min(16, n_all - c0)
        model.verify(chunk[c0:c0 + n], n, pos, desc, targets)
    torch.cuda.synchronize()
    i = (n_all - 1) % 16
    return targets[i:i + 1].clone()


def _time_graph(g, stream, steps, per_step=None):
    """Milliseconds of `steps` back-to-back replays of the graph, from HIP
    events on its stream; with `per_step` (a list) an event is also recorded
    after every replay and the single replays' durations are appended."""
    import torch
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1 if per_step is not None else 2)]
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        ev[0].record(stream)
        for i in range(steps):
            g.replay()
            if per_step is not None:
                ev[i + 1].record(stream)
        if per_step is None:
            ev[1].record(stream)
    torch.cuda.synchronize()
    if per_step is not None:
        per_step.extend(ev[i].elapsed_time(ev[i + 1]) for i in range(steps))
    return ev[0].elapsed_time(ev[-1])


def _pcts(xs):
    """p10 / p50 / p90 of per-step milliseconds."""
    import numpy as np
    return {k: round(float(np.percentile(xs, q)), 5) for k, q in (("p10", 10), ("p50", 50), ("p90", 90))}


def _kernel_avg_ms(model, kernel, stream, fn, reps):
    """Average duration of one kernel class over `reps` direct calls of fn,
    from HIP events recorded on the launch stream around each launch."""
    import torch
    model.timing_enable(kernel)
    with torch.cuda.stream(stream):
        for _ in range(reps):
            fn()
    k_ms, k_n = model.timing_read()
    model.timing_enable(None)
    return k_ms / max(k_n, 1), k_n


# ----------------------------------------------------------------------------
# modes
# ----------------------------------------------------------------------------

def run_dense(args) -> int:
    import torch
    import synth
    from paper_2502_02040_amd import Model, PagedKV

    cfg = synth.CONFIGS[args.config]
    dual = not args.single
    dev = torch.device("cuda:0")
    t_setup = time.perf_counter()
    weights = synth.make_weights(cfg)
    max_ctx = dense_capacity(args.ctx, args.warmup, args.steps, args.kernel_reps)
    model = Model(cfg, weights, max_batch=1, max_chunk=16, max_ctx=max_ctx)
    _progress(f"dense: model ready after {time.perf_counter() - t_setup:.1f} s")
    bps = (max_ctx + 15) // 16
    kv = PagedKV(cfg, 1, max_ctx, block_size=16, block_table=synth.block_table(1, bps, seed=cfg.seed))
    desc = kv.desc()
    pos = torch.zeros(1, dtype=torch.int32, device=dev)
    tok = _prefill(model, synth.prompt_ids(cfg, args.ctx), pos, desc, dev)

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
    per = []
    ms = _time_graph(g, stream, args.steps, per)
    ms_step = ms / args.steps
    ctx_mean = ctx0 + (args.steps - 1) / 2.0

    # dominant kernel: the one-launch decode step (every layer and the head
    # in one kernel) when the model's shape has it, timed with HIP events on
    # the launch stream around direct launches; otherwise the gate/up kernel
    # of the per-kernel path, every layer's launch back to back
    reps = max(1, args.kernel_reps)
    k_avg_ms, k_n = _kernel_avg_ms(model, "step", stream, step, reps)
    torch.cuda.synchronize()
    ctx_k = int(pos.item()) - (reps - 1) / 2.0 - 1
    if k_n > 0:
        kb = step_bytes(cfg, ctx_k, dual)
        kname = "one-launch decode step (kp_step): all layers and the LM head"
        traffic = stored_traffic(STEP_COUNTERS) if (args.config == "phi3" and dual) else None
    else:
        k_avg_ms = sum(model.time_gateup_layers(dual, stream=stream) for _ in range(reps)) / reps
        k_n = reps * cfg.n_layers
        kb = gateup_bytes(cfg, 2 if dual else 1, 1 if dual else 0)
        kname = "gate/up projection, one output row per wave (kr_gateup)"
        traffic = stored_traffic(GATEUP_COUNTERS) if (args.config == "phi3" and dual) else None
    errs = model.device_errors()
    if errs:
        print(f"device error bits {errs}", file=sys.stderr)
        return 1
    achieved = kb / (k_avg_ms * 1e-3) / 1e9
    sb = step_bytes(cfg, ctx_mean, dual)
    step_gbs = sb / (ms_step * 1e-3) / 1e9

    cpu = cpu_baseline(cfg, weights, args.ctx, args.cpu_budget) if args.cpu_budget > 0 else None
    _line(value=round(1000.0 / ms_step, 3), unit="tokens/s", steps=args.steps, warmup=args.warmup,
          ms_per_step=round(ms_step, 5), ms_per_step_pcts=_pcts(per), dtype="bf16" if cfg.wdtype == "bf16" else "f32",
          config={"workload": f"{'dual' if dual else 'single'}-stream decode step, {cfg.name}-shaped "
                              f"{cfg.n_layers}L d{cfg.d_model} {cfg.n_heads}x{cfg.head_dim} ffn{cfg.ffn} "
                              f"vocab{cfg.vocab} rank{cfg.rank}, {cfg.wdtype} weights/KV, batch 1, "
                              f"KV context {args.ctx} (+{args.warmup + args.steps} decoded), HIP graph replay",
                  "batch": 1, "kv_context": args.ctx, "dual_stream": dual},
          step_hbm_gbs=round(step_gbs, 1), step_bytes=int(sb), step_roofline_frac=round(step_gbs / HBM_PEAK_GBS, 4),
          roofline={"bound": "hbm", "kernel": kname, "achieved": round(achieved, 1),
                    "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                    "traffic": traffic, "avg_kernel_us": round(k_avg_ms * 1e3, 3), "bytes_per_launch": int(kb),
                    "launches_timed": k_n},
          cpu_baseline=cpu, setup_s=round(setup_s, 1))
    return 0


def run_batch(args) -> int:
    """8 sequences, 4096-token contexts in a paged cache with seeded content."""
    import torch
    import synth
    from paper_2502_02040_amd import Model, PagedKV

    cfg = synth.CONFIGS[args.config]
    B, ctx = args.batch, args.ctx
    dual = not args.single
    dev = torch.device("cuda:0")
    t_setup = time.perf_counter()
    weights = synth.make_weights(cfg)
    max_ctx = ctx + args.warmup + args.steps + 2 * args.kernel_reps + 16
    model = Model(cfg, weights, max_batch=B, max_chunk=16, max_ctx=max_ctx)
    del weights
    bps = (max_ctx + 15) // 16
    kv = PagedKV(cfg, B, max_ctx, block_size=16, block_table=synth.block_table(B, bps, seed=3))
    gen = torch.Generator(device=dev)
    gen.manual_seed(cfg.seed)
    _progress("batch: model ready, filling the cache")
    for t in (kv.k, kv.v):   # synthetic N(0, 1) cache content, every position
        t.copy_(torch.randn(t.shape, generator=gen, device=dev, dtype=torch.float32).to(t.dtype))
    kv.seq_lens.fill_(ctx)
    pos = torch.full((B,), ctx, dtype=torch.int32, device=dev)
    tok = torch.tensor(synth.prompt_ids(cfg, B, stream="batch"), dtype=torch.int32, device=dev)
    desc = kv.desc()
    N = cfg.n_layers
    gates = list(range(1, N)) if dual else []
    sig = torch.zeros(B * N, dtype=torch.float32, device=dev)
    exb = torch.zeros(B, dtype=torch.int32, device=dev)
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
    ctx0 = int(pos[0].item())
    per = []
    ms = _time_graph(g, stream, args.steps, per)
    ms_step = ms / args.steps
    ctx_mean = ctx0 + (args.steps - 1) / 2.0
    k_avg_ms, k_n = _kernel_avg_ms(model, "attn", stream, step, args.kernel_reps)
    errs = model.device_errors()
    if errs:
        print(f"device error bits {errs}", file=sys.stderr)
        return 1
    ab = attn_bytes(cfg, B, ctx0 + args.steps + args.kernel_reps / 2)
    achieved = ab / (k_avg_ms * 1e-3) / 1e9
    sb = step_bytes(cfg, ctx_mean, dual, batch=B)
    step_gbs = sb / (ms_step * 1e-3) / 1e9
    del model
    torch.cuda.empty_cache()
    cpu = cpu_baseline(cfg, synth.make_weights(cfg), ctx, args.cpu_budget, seqs=B) if args.cpu_budget > 0 else None
    _line(metric="batched decode tokens/s (aggregate) + achieved HBM GB/s of the dual-stream step",
          value=round(B * 1000.0 / ms_step, 3), unit="tokens/s", steps=args.steps, warmup=args.warmup,
          ms_per_step=round(ms_step, 5), ms_per_step_pcts=_pcts(per), dtype="bf16" if cfg.wdtype == "bf16" else "f32",
          config={"workload": f"{'dual' if dual else 'single'}-stream decode step, {cfg.name}-shaped model, batch {B}, "
                              f"paged KV context {ctx} per sequence (block 16, shuffled table, seeded N(0,1) "
                              f"content), HIP graph replay", "batch": B, "kv_context": ctx, "dual_stream": dual},
          step_hbm_gbs=round(step_gbs, 1), step_bytes=int(sb), step_roofline_frac=round(step_gbs / HBM_PEAK_GBS, 4),
          roofline={"bound": "hbm", "kernel": "split-context attention, 128-token splits (ks_attn)", "achieved": round(achieved, 1),
                    "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                    "traffic": None, "avg_kernel_us": round(k_avg_ms * 1e3, 3), "bytes_per_launch": int(ab),
                    "launches_timed": k_n},
          cpu_baseline=cpu, setup_s=round(setup_s, 1))
    return 0


SPEC_TIE_REL = 2e-3   # near-tie bound: logit gap <= 2e-3 x max |logit|


def _teacher_forced_greedy(model, cfg, prompt, max_ctx, tokens):
    """Greedy decoding teacher-forced on `tokens` (the speculative output,
    untimed): at every position the slow stream's argmax on the same prefix,
    the logit gap between that argmax and the token taken there, and the
    largest |logit|."""
    import torch
    from paper_2502_02040_amd import PagedKV
    dev = torch.device("cuda:0")
    kv = PagedKV(cfg, 1, max_ctx, block_size=16)
    desc = kv.desc()
    pos = torch.zeros(1, dtype=torch.int32, device=dev)
    first = _prefill(model, prompt, pos, desc, dev)
    n = len(tokens)
    feed = torch.tensor(tokens, dtype=torch.int32, device=dev)
    logits = torch.zeros(cfg.vocab, dtype=torch.float32, device=dev)
    nxt = torch.zeros(1, dtype=torch.int32, device=dev)
    arg = torch.zeros(n, dtype=torch.int32, device=dev)
    gap = torch.zeros(n, dtype=torch.float32, device=dev)
    amax = torch.zeros(n, dtype=torch.float32, device=dev)
    arg[0:1].copy_(first)
    for i in range(n - 1):
        model.decode_step(feed[i:i + 1], pos, desc, dual=False, next_token=nxt, logits=logits, advance=True)
        arg[i + 1:i + 2].copy_(nxt)
        gap[i + 1] = logits.max() - logits[feed[i + 1].long()]
        amax[i + 1] = logits.abs().max()
    torch.cuda.synchronize()
    return arg.cpu().numpy(), gap.cpu().numpy(), amax.cpu().numpy()


def run_spec(args) -> int:
    """Draft + verify against plain greedy decoding on the same kernels."""
    import torch
    import synth
    from paper_2502_02040_amd import Model, PagedKV

    base = synth.CONFIGS[args.config]
    gamma, kL, n_new, plen = args.gamma, args.exit_layer, args.new_tokens, args.prompt
    dev = torch.device("cuda:0")
    results = []
    for lam in args.decay:
        _progress(f"spec: decay {lam}")
        cfg = base
        weights = synth.make_weights(cfg, decay=None if lam == 1.0 else (kL, lam), adapter_scale=args.adapter_scale)
        max_ctx = plen + n_new + 12 * (gamma + 1) + 16
        model = Model(cfg, weights, max_batch=1, max_chunk=16, max_ctx=max_ctx)
        del weights
        prompt = synth.prompt_ids(cfg, plen)
        stream = torch.cuda.Stream()

        # plain greedy: slow-only decode steps, one graph per step
        kv = PagedKV(cfg, 1, max_ctx, block_size=16)
        desc = kv.desc()
        pos = torch.zeros(1, dtype=torch.int32, device=dev)
        tok = _prefill(model, prompt, pos, desc, dev)
        first = int(tok.item())
        hist = torch.zeros(n_new + 8, dtype=torch.int32, device=dev)
        hist[0] = first
        k_i = torch.zeros(1, dtype=torch.int64, device=dev)

        def greedy_step():
            model.decode_step(tok, pos, desc, dual=False, next_token=tok, advance=True)

        with torch.cuda.stream(stream):
            greedy_step()   # warm-up (position plen)
        torch.cuda.synchronize()
        pos.fill_(plen)
        kv.seq_lens.fill_(plen)
        tok.fill_(first)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            greedy_step()
        torch.cuda.synchronize()
        pos.fill_(plen)
        kv.seq_lens.fill_(plen)
        tok.fill_(first)
        greedy_tokens = [first]
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        out_buf = torch.zeros(n_new, dtype=torch.int32, device=dev)
        with torch.cuda.stream(stream):
            e0.record(stream)
            for i in range(n_new - 1):
                g.replay()
                out_buf[i:i + 1].copy_(tok, non_blocking=True)
            e1.record(stream)
        torch.cuda.synchronize()
        greedy_ms = e0.elapsed_time(e1)
        greedy_tokens += out_buf[:n_new - 1].cpu().tolist()
        greedy_tps = (n_new - 1) / (greedy_ms * 1e-3)

        _progress(f"spec: greedy {greedy_tps:.1f} tokens/s")
        # speculative: a round = gamma draft passes + one verify of gamma+1 rows
        kv2 = PagedKV(cfg, 1, max_ctx, block_size=16)
        desc2 = kv2.desc()
        pos2 = torch.zeros(1, dtype=torch.int32, device=dev)
        t2 = _prefill(model, prompt, pos2, desc2, dev)
        assert int(t2.item()) == first
        chunk = torch.zeros(gamma + 1, dtype=torch.int32, device=dev)
        targets = torch.zeros(gamma + 1, dtype=torch.int32, device=dev)
        n_acc = torch.zeros(1, dtype=torch.int32, device=dev)
        max_rounds = n_new + 1
        rec_t = torch.zeros((max_rounds, gamma + 1), dtype=torch.int32, device=dev)
        rec_n = torch.zeros(max_rounds, dtype=torch.int32, device=dev)

        def spec_round():
            model.draft(chunk, pos2, kL, gamma, desc2, chunk[1:])
            model.verify(chunk, gamma + 1, pos2, desc2, targets, n_acc, chunk[0:1])

        chunk[0] = first
        with torch.cuda.stream(stream):
            spec_round()   # warm-up, then restart from the prompt
        torch.cuda.synchronize()
        pos2.fill_(plen)
        kv2.seq_lens.fill_(plen)
        chunk.zero_()
        chunk[0] = first
        gs = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gs, stream=stream):
            spec_round()
        torch.cuda.synchronize()
        pos2.fill_(plen)
        kv2.seq_lens.fill_(plen)
        chunk.zero_()
        chunk[0] = first
        # rounds are replayed in groups; the host checks the count between groups
        produced, rounds = 1, 0
        e0.record(stream)
        with torch.cuda.stream(stream):
            while produced < n_new:
                grp = max(1, min(32, (n_new - produced + gamma) // (gamma + 1)))
                for _ in range(grp):
                    gs.replay()
                    rec_t[rounds].copy_(targets, non_blocking=True)
                    rec_n[rounds:rounds + 1].copy_(n_acc, non_blocking=True)
                    rounds += 1
                produced = 1 + int((rec_n[:rounds] + 1).sum().item())
        e1.record(stream)
        torch.cuda.synchronize()
        spec_ms = e0.elapsed_time(e1)
        rt, rn = rec_t[:rounds].cpu().numpy(), rec_n[:rounds].cpu().numpy()
        spec_tokens = [first]
        for r in range(rounds):
            spec_tokens += rt[r, :rn[r] + 1].tolist()
        spec_tokens = spec_tokens[:n_new]
        alpha = float(rn.sum()) / (rounds * gamma)
        spec_tps = (produced - 1) / (spec_ms * 1e-3)   # tokens after the first, as for greedy
        # model speedup from the measured pass times
        kv3 = PagedKV(cfg, 1, max_ctx, block_size=16)
        d3 = kv3.desc()
        p3 = torch.zeros(1, dtype=torch.int32, device=dev)
        _prefill(model, prompt, p3, d3, dev)
        ch3 = torch.zeros(gamma + 1, dtype=torch.int32, device=dev)
        gd, gv = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
        with torch.cuda.graph(gd, stream=stream):
            model.draft(ch3, p3, kL, gamma, d3, ch3[1:])
        with torch.cuda.graph(gv, stream=stream):
            model.verify(ch3, gamma + 1, p3, d3, targets)   # prefill form: keeps the position fixed below
        torch.cuda.synchronize()
        t_draft = _time_graph(gd, stream, 20) / 20 / gamma
        p3.fill_(plen)
        t_verify = _time_graph(gv, stream, 10) / 10   # each replay advances the context by gamma+1
        t_step = greedy_ms / (n_new - 1)
        E = sum(alpha ** i for i in range(gamma + 1))
        s_model = E * t_step / (gamma * t_draft + t_verify)
        # lossless, teacher-forced: every speculative token is the greedy
        # argmax on the same prefix, except at near-ties of the greedy logits
        # (the verification chunk runs other kernels, whose fp32 sums round
        # differently), which are counted
        div = next((i for i, (a, b) in enumerate(zip(spec_tokens, greedy_tokens)) if a != b), None)
        arg, gap, amax = _teacher_forced_greedy(model, cfg, prompt, max_ctx, spec_tokens)
        diffs = [i for i in range(len(spec_tokens)) if int(arg[i]) != spec_tokens[i]]
        ties = [i for i in diffs if gap[i] <= SPEC_TIE_REL * amax[i]]
        results.append(dict(decay=lam, adapter_scale=args.adapter_scale, alpha=round(alpha, 4), rounds=rounds,
                            tokens=len(spec_tokens),
                            lossless=len(diffs) == len(ties), tokens_checked=len(spec_tokens),
                            differences_from_teacher_forced_greedy=len(diffs), near_tie_exceptions=len(ties),
                            first_difference_free_running=div,
                            max_difference_logit_gap=round(float(max([gap[i] for i in diffs] or [0.0])), 7),
                            greedy_tps=round(greedy_tps, 2), spec_tps=round(spec_tps, 2),
                            speedup=round(spec_tps / greedy_tps, 4), model_speedup=round(s_model, 4),
                            ms_draft_token=round(t_draft, 4), ms_verify=round(t_verify, 4),
                            ms_greedy_step=round(t_step, 4)))
        del model, kv, kv2, kv3
        torch.cuda.empty_cache()
        if len(diffs) > len(ties):
            bad = [i for i in diffs if i not in ties]
            print(f"speculative tokens differ from the teacher-forced greedy argmax at {bad[:8]} (decay {lam}) "
                  f"beyond near-ties", file=sys.stderr)
    main_r = results[0]
    cpu = None
    if args.cpu_budget > 0:
        _progress("spec: CPU oracle baseline")
        cpu = cpu_spec_baseline(base, synth.make_weights(base), plen, gamma, kL, args.cpu_budget)
    _line(metric="self-speculative decode tokens/s at batch 1 (draft from the fast stream, verify on the slow stream)",
          value=main_r["spec_tps"], unit="tokens/s", steps=main_r["rounds"], warmup=1,
          ms_per_step=round(1000.0 / main_r["spec_tps"], 5), dtype="bf16" if base.wdtype == "bf16" else "f32",
          config={"workload": f"{base.name}-shaped model, prompt {plen}, {n_new} generated tokens, gamma {gamma}, "
                              f"draft exit layer {kL}; rounds captured as HIP graphs",
                  "batch": 1, "gamma": gamma, "exit_layer": kL},
          baseline_greedy_tps=main_r["greedy_tps"], results=results, roofline=None, cpu_baseline=cpu)
    return 0 if all(r["lossless"] for r in results) else 1


def run_exit(args) -> int:
    """EXIT-mode dual-stream decoding at the dense configuration: tokens/s and
    the mean exit boundary for each threshold tau (tau > 1 never exits)."""
    import torch
    import synth
    from paper_2502_02040_amd import Model, PagedKV

    cfg = synth.CONFIGS[args.config]
    dev = torch.device("cuda:0")
    weights = synth.make_weights(cfg)
    max_ctx = args.ctx + args.warmup + args.steps + 32
    model = Model(cfg, weights, max_batch=1, max_chunk=16, max_ctx=max_ctx)
    del weights
    N = cfg.n_layers
    gates = list(range(args.gate_every, N, args.gate_every))
    if args.arla:
        model.set_arla(synth.arla_weights(cfg))
    prompt = synth.prompt_ids(cfg, args.ctx)
    stream = torch.cuda.Stream()
    results = []
    for tau in args.taus:
        bps = (max_ctx + 15) // 16
        kv = PagedKV(cfg, 1, max_ctx, block_size=16, block_table=synth.block_table(1, bps, seed=cfg.seed))
        desc = kv.desc()
        pos = torch.zeros(1, dtype=torch.int32, device=dev)
        tok = _prefill(model, prompt, pos, desc, dev)
        exb = torch.zeros(1, dtype=torch.int32, device=dev)
        hist = torch.zeros(args.steps, dtype=torch.int32, device=dev)

        def step():
            model.decode_step(tok, pos, desc, dual=True, gates=gates, tau=tau, mode="exit", next_token=tok,
                              exit_boundary=exb, advance=True)

        with torch.cuda.stream(stream):
            for _ in range(args.warmup):
                step()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            step()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(stream):
            e0.record(stream)
            for i in range(args.steps):
                g.replay()
                hist[i:i + 1].copy_(exb, non_blocking=True)   # the same small copy at every tau
            e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / args.steps
        b = hist.cpu().numpy()
        errs = model.device_errors()
        if errs:
            print(f"device error bits {errs}", file=sys.stderr)
            return 1
        results.append(dict(tau=tau, ms_per_step=round(ms, 5), tokens_per_s=round(1000.0 / ms, 2),
                            mean_exit_boundary=round(float(b.mean()), 3), exit_rate=round(float((b < N).mean()), 4)))
        _progress(f"exit: tau {tau}: {results[-1]}")
        del kv
    base = next((r for r in results if r["exit_rate"] == 0.0), results[0])
    for r in results:
        r["speedup"] = round(base["ms_per_step"] / r["ms_per_step"], 4)
    main_r = min(results, key=lambda r: r["ms_per_step"])
    signal = ("latent-attention exit router (seeded synthetic weights, 64-wide)" if args.arla
              else "cosine signal")
    _line(metric="EXIT-mode dual-stream decode tokens/s at batch 1 (tau sweep)", value=main_r["tokens_per_s"],
          unit="tokens/s", steps=args.steps, warmup=args.warmup, ms_per_step=main_r["ms_per_step"],
          dtype="bf16" if cfg.wdtype == "bf16" else "f32",
          config={"workload": f"{cfg.name}-shaped dual-stream step in EXIT mode, gates every {args.gate_every} "
                              f"layer(s), {signal}, KV context {args.ctx}, HIP graph replay; value = the fastest tau",
                  "batch": 1, "kv_context": args.ctx, "gates": gates},
          results=results, roofline=None, cpu_baseline=None)
    return 0


def run_moe(args) -> int:
    """OLMoE-shaped model with its experts in pinned host memory."""
    import torch
    import synth
    from paper_2502_02040_amd import Model, PagedKV
    from paper_2502_02040_amd.binding import pack_expert_store

    cfg = synth.CONFIGS["olmoe"]
    dev = torch.device("cuda:0")
    t_setup = time.perf_counter()
    names = [n for n, _, _ in synth.tensor_specs(cfg) if ".E" not in n]
    spec = {n: (s, k) for n, s, k in synth.tensor_specs(cfg)}

    def expert_source(l, e):
        return tuple(synth.make_tensor(cfg, f"L{l}.E{e}.{m}", *spec[f"L{l}.E{e}.{m}"]) for m in ("wg", "wu", "wd"))

    store = pack_expert_store(cfg, expert_source, threads=16)
    variant = {"router_coherent": True} if args.router_coherent else {}
    gen_s = time.perf_counter() - t_setup
    _progress(f"moe: {cfg.n_layers * cfg.n_experts} experts packed into pinned host memory in {gen_s:.1f} s")
    plen, steps, C = args.prompt, args.steps, args.slots
    max_ctx = plen + steps + args.warmup + 16
    prompt = synth.prompt_ids(cfg, plen)
    # decode inputs: a teacher-forced token stream with natural-text (Zipf)
    # frequencies, so that routing varies from token to token as it does on
    # text (greedy tokens of random weights fall into short cycles)
    stream_ids = torch.tensor(synth.zipf_ids(cfg, args.warmup + steps), dtype=torch.int32, device=dev)
    table = synth.preload_table(cfg, args.warmup + steps)
    E = cfg.n_experts
    runs = []
    want = set(x for x in args.moe_runs.split(",") if x)

    def prefix(model, pos, desc, nxt, dual):
        for t in prompt:   # prefill with slow-only steps (not timed)
            model.decode_step(torch.tensor([int(t)], dtype=torch.int32, device=dev), pos, desc, dual=False,
                              next_token=nxt, advance=True)
        for i in range(args.warmup):
            model.decode_step(stream_ids[i:i + 1], pos, desc, dual=dual, next_token=nxt, advance=True)

    # the true routing of the timed steps (untimed pass, every expert
    # resident): the table of the oracle-predictor run, an upper bound on
    # prediction (Sec. 3.3 reports accuracy against it implicitly)
    true_table = None
    if not want or "oracle" in want:
        _progress("moe: recording the true routing")
        w = synth.make_weights(cfg, names=names, **variant)
        model = Model(cfg, w, max_batch=1, max_chunk=16, max_ctx=max_ctx, expert_slots=E, expert_store=store)
        del w
        kv = PagedKV(cfg, 1, max_ctx, block_size=16)
        desc = kv.desc()
        pos = torch.zeros(1, dtype=torch.int32, device=dev)
        nxt = torch.zeros(1, dtype=torch.int32, device=dev)
        prefix(model, pos, desc, nxt, False)
        rec = torch.zeros((steps, cfg.n_layers * cfg.top_k), dtype=torch.int32, device=dev)
        for i in range(steps):
            j = args.warmup + i
            model.decode_step(stream_ids[j:j + 1], pos, desc, dual=False, next_token=nxt, advance=True,
                              slow_experts=rec[i])
        torch.cuda.synchronize()
        true_table = rec.cpu().numpy().reshape(steps, cfg.n_layers, cfg.top_k)
        del model, kv
        torch.cuda.empty_cache()
    # the four strategies the paper compares with (Sec. 3.3) run the slow
    # stream alone; M2R2 runs both rows
    for label, slots, policy, dual in (
            ("fixed experts, no replacement", C, "fixed", False),
            ("on-demand LRU", C, "on_demand", False),
            ("LRU + random preload", C, "random_preload", False),
            ("previous-layer residual speculation", C, "previous_layer", False),
            ("M2R2 ahead-of-time prefetch", C, "ahead_of_time", True),
            ("oracle predictor: the true routing of the next layer preloaded after each layer", C, "oracle", False),
            ("all experts resident", E, "on_demand", True)):
        if want and policy not in want and not (policy == "on_demand" and slots == E and "resident" in want):
            continue
        _progress(f"moe: {label}")
        w = synth.make_weights(cfg, names=names, **variant)
        model = Model(cfg, w, max_batch=1, max_chunk=16, max_ctx=max_ctx, expert_slots=slots, expert_store=store)
        del w
        model.moe_set_preload_table(true_table if policy == "oracle" else table)
        model.moe_set_policy("random_preload" if policy == "oracle" else policy)
        kv = PagedKV(cfg, 1, max_ctx, block_size=16)
        desc = kv.desc()
        pos = torch.zeros(1, dtype=torch.int32, device=dev)
        nxt = torch.zeros(1, dtype=torch.int32, device=dev)
        prefix(model, pos, desc, nxt, dual)
        torch.cuda.synchronize()
        model.moe_reset()   # the preload table restarts at its row 0: the same draws as the replay
        stream = torch.cuda.current_stream()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        e0.record(stream)
        for i in range(steps):
            j = args.warmup + i
            model.decode_step(stream_ids[j:j + 1], pos, desc, dual=dual, next_token=nxt, advance=True)
        e1.record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        ms = e0.elapsed_time(e1)
        st = model.moe_stats()
        k_avg_ms, k_n = _kernel_avg_ms(model, "expert_gateup", stream,
                                       lambda: model.decode_step(stream_ids[0:1], pos, desc, dual=dual,
                                                                 next_token=nxt, advance=True), 4)
        n_use = st["hits"] + st["misses"]
        runs.append(dict(run=label, slots=slots, policy=policy, dual_stream=dual,
                         tokens_per_s=round(steps * 1000.0 / ms, 3), ms_per_token=round(ms / steps, 4),
                         wall_s=round(wall, 3), hit_rate=round(st["hits"] / max(n_use, 1), 4),
                         misses_per_token=round(st["misses"] / steps, 3),
                         prefetch_issued=st["prefetch_issued"], prefetch_used=st["prefetch_used"],
                         prefetch_wasted=st["prefetch_wasted"],
                         pred_accuracy=round(st["pred_correct"] / st["pred_total"], 4) if st["pred_total"] else None,
                         h2d_gb=round(st["h2d_bytes"] / 1e9, 3), copy_waits=st["copy_waits"],
                         host_wait_ms_per_token=round(st["host_wait_ns"] / 1e6 / steps, 4),
                         layer_miss_rate=[round(m / (steps * cfg.top_k), 4) for m in st["layer_misses"]],
                         expert_gateup_us=round(k_avg_ms * 1e3, 3)))
        del model, kv
        torch.cuda.empty_cache()
    resident = next((r for r in runs if r["slots"] == E), None)
    for r in runs:
        r["stall_ms_per_token_vs_resident"] = (round(r["ms_per_token"] - resident["ms_per_token"], 4)
                                               if resident else None)
    kb = expert_gateup_bytes(cfg)
    m2 = next((r for r in runs if r["policy"] == "ahead_of_time"), resident or runs[-1])
    # the expert kernel's rate from the all-resident run when it ran (no
    # copies beside it), else from the headline run
    kref = resident or m2
    achieved = kb / (kref["expert_gateup_us"] * 1e-6) / 1e9
    cpu = None
    if args.cpu_budget > 0:
        _progress("moe: CPU oracle baseline")
        cpu = cpu_moe_baseline(cfg, plen, args.cpu_budget)
    _line(metric="MoE decode tokens/s at batch 1 with experts in host memory (HBM expert cache, AoT prefetch)",
          value=m2["tokens_per_s"], unit="tokens/s", steps=steps, warmup=args.warmup,
          ms_per_step=m2["ms_per_token"], dtype="bf16",
          config={"workload": f"olmoe-shaped {cfg.n_layers}L d{cfg.d_model} {cfg.n_heads}x{cfg.head_dim} "
                              f"E{cfg.n_experts} top{cfg.top_k} Fe{cfg.expert_ffn} vocab{cfg.vocab} rank{cfg.rank}, "
                              f"experts in pinned host memory, {C} HBM slots per layer, prompt {plen}, "
                              f"{steps} teacher-forced Zipf-token decode steps"
                              + (", routers shared + 0.5 x noise per layer (router-coherent variant)"
                                 if args.router_coherent else ""), "batch": 1, "slots": C,
                  "router_coherent": bool(args.router_coherent)},
          token_bytes_all_hits=int(moe_token_bytes(cfg, plen + steps / 2)), runs=runs,
          roofline={"bound": "hbm", "kernel": "expert gate/up (k_moe_gateup)", "achieved": round(achieved, 1),
                    "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                    "traffic": None, "avg_kernel_us": kref["expert_gateup_us"], "timed_in": kref["run"],
                    "bytes_per_launch": int(kb)},
          cpu_baseline=cpu, setup_s=round(gen_s, 1))
    return 0


def run_copy(args) -> int:
    """A plain device-to-device copy of a known size, for scaling the HBM
    byte counters of the profiler (FETCH_SIZE / WRITE_SIZE per dispatch)."""
    import torch
    n = 1 << 30
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    a.fill_(1)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = args.steps or 8
    e0.record()
    for _ in range(reps):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    _line(metric="device copy GB/s (read + write) for profiler counter calibration", value=round(2 * n / ms / 1e6, 1),
          unit="GB/s", steps=reps, warmup=0, ms_per_step=round(ms, 5), dtype="u8",
          config={"workload": f"copy of {n} bytes"}, bytes_read=n, bytes_written=n, roofline=None, cpu_baseline=None)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--mode", choices=("dense", "batch", "spec", "exit", "moe", "copy"), default="dense")
    ap.add_argument("--taus", type=float, nargs="*", default=[2.0, 0.99, 0.985, 0.98, 0.97, 0.95, 0.9],
                    help="exit mode: thresholds (above 1: never exits)")
    ap.add_argument("--steps", type=int, default=None)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="phi3")
    ap.add_argument("--ctx", type=int, default=None, help="KV context (dense: 1024, batch: 4096)")
    ap.add_argument("--batch", type=int, default=8, help="sequences (batch mode)")
    ap.add_argument("--single", action="store_true", help="slow row only (plain decoding on the same kernels)")
    ap.add_argument("--kernel-reps", type=int, default=20, help="direct steps timed for the dominant kernel")
    ap.add_argument("--cpu-budget", type=float, default=20.0, help="seconds of CPU oracle timing (0: skip)")
    ap.add_argument("--gamma", type=int, default=4)
    ap.add_argument("--exit-layer", type=int, default=8)
    ap.add_argument("--new-tokens", type=int, default=512)
    ap.add_argument("--prompt", type=int, default=128)
    ap.add_argument("--decay", type=float, nargs="*", default=[1.0, 0.1],
                    help="spec mode: scale of wo/wd in layers >= exit layer (1.0 = plain weights)")
    ap.add_argument("--slots", type=int, default=16, help="moe mode: HBM expert slots per layer")
    ap.add_argument("--router-coherent", action="store_true",
                    help="moe mode: routers drawn as shared + 0.5 x noise per layer (a labelled structured variant)")
    ap.add_argument("--moe-runs", default="",
                    help="moe mode: comma-separated policies to run (default: all), e.g. ahead_of_time,oracle")
    ap.add_argument("--adapter-scale", type=float, default=1.0,
                    help="spec mode: scale of the adapter factors (a labelled structured variant; 0: p == h)")
    ap.add_argument("--gate-every", type=int, default=1, help="exit mode: a gate every this many layers")
    ap.add_argument("--arla", action="store_true",
                    help="exit mode: decide the gates with the latent-attention exit router")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: --gpus {args.gpus} is not supported "
              f"(sharding the step across GPUs is not implemented)", file=sys.stderr)
        return 2
    import torch
    torch.cuda.set_device(0)
    if args.mode == "dense":
        args.steps = args.steps or 256
        args.ctx = args.ctx or 1024
        return run_dense(args)
    if args.mode == "batch":
        args.steps = args.steps or 64
        args.ctx = args.ctx or 4096
        return run_batch(args)
    if args.mode == "spec":
        return run_spec(args)
    if args.mode == "exit":
        args.steps = args.steps or 128
        args.ctx = args.ctx or 1024
        return run_exit(args)
    if args.mode == "copy":
        return run_copy(args)
    args.steps = args.steps or 256
    args.warmup = min(args.warmup, 4)
    return run_moe(args)


if __name__ == "__main__":
    sys.exit(main())
