"""GPU parity at the benchmarked sizes of the dense model (Phi-3-mini shape:
32 layers, d 3072, 32 heads x 96, SwiGLU 8192, vocab 32064, rank 16, bf16),
through the C ABI and in the launch configuration bench.py times, against the
float64 oracle on sampled outputs:

  * the dual-stream step at batch 1 (OBSERVE gates at every boundary) after
    a 16-token prompt, and at context 1024 (seeded synthetic cache content)
    in the cache capacity the benchmark uses, so the attention runs with the
    same splits as in the timed step; and in EXIT mode (the token from the fast row at the first gate whose signal
    reaches tau, the skipped layers' cache filled from the slow row);
  * a draft of 4 tokens from the fast stream exiting at layer 8 and the
    verification of the 5-token chunk;
  * one dual-stream step of 8 sequences with 4096-token paged contexts (seeded
    synthetic cache content), checked on two of the sequences.

The oracle's weights are the same seeded arrays the GPU consumes."""
import numpy as np
import pytest
import torch

import synth
from oracle import KVCache, Oracle
from oracle.decoder import argmax_first, round_to_cache
from paper_2502_02040_amd import Model, PagedKV
from tests.gpu_harness import Tally, oracle_draft_logits, pick_tau, shuffled_table, track

pytestmark = pytest.mark.gpu

CFG = synth.CONFIGS["phi3"]
TOL = 2e-2
PROMPT = 16
CTX_B = 4096


@pytest.fixture(scope="module")
def world():
    w = synth.make_weights(CFG)
    model = track(Model(CFG, w, max_batch=8, max_chunk=16, max_ctx=CTX_B + 16))
    orc = Oracle(CFG, w)
    yield model, orc, w
    del model, orc
    torch.cuda.empty_cache()


def _prefill(model, orc, kv, cache, prompt, t):
    dev = torch.device("cuda")
    pos = torch.zeros(1, dtype=torch.int32, device=dev)
    targets = torch.zeros(16, dtype=torch.int32, device=dev)
    chunk = torch.tensor(prompt, dtype=torch.int32, device=dev)
    model.verify(chunk, len(prompt), pos, kv.desc(), targets)
    torch.cuda.synchronize()
    ref = orc.slow_chunk(list(prompt), 0, cache)
    got = targets[:len(prompt)].cpu().numpy()
    for i in range(len(prompt)):
        t.token(int(got[i]), ref[i], TOL, f"prefill row {i}")
    return int(got[-1]), pos


def _check_cache(kv, cache, seq, start, end, t, layers, what):
    for l in layers:
        K, V = kv.read(seq, l, start, end)
        t.rel(K, cache.K[l][start:end], TOL, f"{what} K layer {l}")
        t.rel(V, cache.V[l][start:end], TOL, f"{what} V layer {l}")


def test_phi3_dual_step(world):
    model, orc, _ = world
    t = Tally()
    kv = PagedKV(CFG, 1, 64, block_size=16, block_table=shuffled_table(1, 64, 16, 7))
    cache = KVCache(CFG, 64)
    prompt = list(synth.prompt_ids(CFG, PROMPT))
    tok, pos_d = _prefill(model, orc, kv, cache, prompt, t)
    _check_cache(kv, cache, 0, 0, PROMPT, t, (0, 15, 31), "prefill")
    dev = torch.device("cuda")
    N = CFG.n_layers
    gates = list(range(1, N))
    tok_d = torch.tensor([tok], dtype=torch.int32, device=dev)
    nxt = torch.zeros(1, dtype=torch.int32, device=dev)
    exb = torch.zeros(1, dtype=torch.int32, device=dev)
    sig = torch.zeros(N, dtype=torch.float32, device=dev)
    logits = torch.zeros(CFG.vocab, dtype=torch.float32, device=dev)
    h_out = torch.zeros(CFG.d_model, dtype=torch.float32, device=dev)
    p_out = torch.zeros(CFG.d_model, dtype=torch.float32, device=dev)
    for step in range(3):
        pos = PROMPT + step
        model.decode_step(tok_d, pos_d, kv.desc(), gates=gates, tau=0.9, mode="observe", next_token=nxt,
                          exit_boundary=exb, signal=sig, logits=logits, h_out=h_out, p_out=p_out, advance=True)
        torch.cuda.synchronize()
        r = orc.decode_step(int(tok_d.item()), pos, cache, gates=gates, tau=0.9, mode="observe")
        _compare_observe_step(t, r, logits, h_out, p_out, sig, exb, nxt, gates, 0.9, step)
        _check_cache(kv, cache, 0, pos, pos + 1, t, (0, 7, 31), f"step {step}")
        t.steps += 1
        tok_d.copy_(nxt)
    assert t.steps == 3 and t.compared >= 5


def _compare_observe_step(t, r, logits, h_out, p_out, sig, exb, nxt, gates, tau, step):
    """Outputs of an OBSERVE step (which do not depend on the gate
    decisions); the exit boundary where every gate signal decides it."""
    t.rel(logits.cpu().numpy(), r.logits, TOL, f"step {step} logits")
    t.rel(h_out.cpu().numpy(), r.h, TOL, f"step {step} h")
    t.rel(p_out.cpu().numpy(), r.p, TOL, f"step {step} p")
    t.close(sig.cpu().numpy(), r.signal, TOL, f"step {step} signal")
    if all(abs(r.signal[b - 1] - tau) > TOL for b in gates):
        t.equal(int(exb.item()), r.exit_boundary, f"step {step} exit boundary")
    else:
        t.skipped += 1
    t.token(int(nxt.item()), r.logits, TOL, f"step {step} token")


def test_phi3_dual_step_bench_context(world):
    """The benchmarked configuration: batch 1, context 1024 (seeded N(0,1)
    cache content, shuffled block table), the cache capacity bench.py uses
    (the attention then runs with the splits of the timed step, the context
    spread over all of them), three OBSERVE dual-stream steps."""
    from bench import dense_capacity
    _, orc, w = world
    ctx = 1024
    cap = dense_capacity(ctx, 5, 20, 20)
    assert cap == dense_capacity(ctx, 10, 256, 20)   # the default run shares it
    model = track(Model(CFG, w, max_batch=1, max_chunk=16, max_ctx=cap))
    try:
        t = Tally()
        kv = PagedKV(CFG, 1, cap, block_size=16, block_table=shuffled_table(1, cap, 16, 11))
        cache = KVCache(CFG, cap)
        content = synth.synthetic_kv(CFG, ctx, seq=0, threads=16)
        for l, (K, V) in content.items():
            kv.load(0, l, K, V)
            cache.load(l, K, V)
        del content
        kv.seq_lens.fill_(ctx)
        dev = torch.device("cuda")
        N = CFG.n_layers
        gates = list(range(1, N))
        tok_d = torch.tensor(synth.prompt_ids(CFG, 1, stream="benchctx"), dtype=torch.int32, device=dev)
        pos_d = torch.full((1,), ctx, dtype=torch.int32, device=dev)
        nxt = torch.zeros(1, dtype=torch.int32, device=dev)
        exb = torch.zeros(1, dtype=torch.int32, device=dev)
        sig = torch.zeros(N, dtype=torch.float32, device=dev)
        logits = torch.zeros(CFG.vocab, dtype=torch.float32, device=dev)
        h_out = torch.zeros(CFG.d_model, dtype=torch.float32, device=dev)
        p_out = torch.zeros(CFG.d_model, dtype=torch.float32, device=dev)
        for step in range(3):
            pos = ctx + step
            model.decode_step(tok_d, pos_d, kv.desc(), gates=gates, tau=0.9, mode="observe", next_token=nxt,
                              exit_boundary=exb, signal=sig, logits=logits, h_out=h_out, p_out=p_out, advance=True)
            torch.cuda.synchronize()
            r = orc.decode_step(int(tok_d.item()), pos, cache, gates=gates, tau=0.9, mode="observe")
            assert int(pos_d.item()) == pos + 1 and int(kv.seq_lens[0].item()) == pos + 1
            _compare_observe_step(t, r, logits, h_out, p_out, sig, exb, nxt, gates, 0.9, step)
            _check_cache(kv, cache, 0, pos, pos + 1, t, (0, 13, 31), f"step {step}")
            t.steps += 1
            tok_d.copy_(nxt)
        # per step: logits, h, p, signals and 6 cache slabs element by element;
        # the token and the exit boundary compared or counted as near ties
        assert t.steps == 3 and t.arrays >= 30 and t.compared + t.skipped == 6
        assert model.device_errors() == 0
    finally:
        del model
        torch.cuda.empty_cache()


# EXIT-mode thresholds, in order of preference, and the window around a gate
# signal inside which a threshold is not used: the measured signal errors
# are below 1e-3, so a decision further than 2e-3 from tau is taken alike
EXIT_TAUS = (0.95, 0.945, 0.955, 0.94, 0.96, 0.935, 0.965, 0.93, 0.97)
EXIT_EPS = 2e-3


def test_phi3_exit_step(world):
    """EXIT mode at every interior boundary (tau 0.95, or the nearest
    threshold that every gate signal of the step decides): the exit boundary,
    the fast row's token at the gate, the skipped layers' cache entries filled
    from the slow row, and the signals of the layers that ran."""
    model, orc, _ = world
    t = Tally()
    kv = PagedKV(CFG, 1, 64, block_size=16, block_table=shuffled_table(1, 64, 16, 9))
    cache = KVCache(CFG, 64)
    prompt = list(synth.prompt_ids(CFG, PROMPT, stream="exit"))
    tok, pos_d = _prefill(model, orc, kv, cache, prompt, t)
    dev = torch.device("cuda")
    N, tau = CFG.n_layers, 0.95
    gates = list(range(1, N))
    tok_d = torch.tensor([tok], dtype=torch.int32, device=dev)
    nxt = torch.zeros(1, dtype=torch.int32, device=dev)
    exb = torch.zeros(1, dtype=torch.int32, device=dev)
    sig = torch.zeros(N, dtype=torch.float32, device=dev)
    logits = torch.zeros(CFG.vocab, dtype=torch.float32, device=dev)
    exits = 0
    for step in range(3):
        pos = PROMPT + step
        tau_s = pick_tau(orc, int(tok_d.item()), pos, cache, gates, EXIT_TAUS, EXIT_EPS)
        assert tau_s is not None, f"step {step}: every threshold lies near a gate signal"
        model.decode_step(tok_d, pos_d, kv.desc(), gates=gates, tau=tau_s, mode="exit", next_token=nxt,
                          exit_boundary=exb, signal=sig, logits=logits, advance=True)
        torch.cuda.synchronize()
        r = orc.decode_step(int(tok_d.item()), pos, cache, gates=gates, tau=tau_s, mode="exit")
        t.equal(int(exb.item()), r.exit_boundary, f"step {step} exit boundary")
        exits += r.exit_boundary < N
        ran = list(range(min(r.exit_boundary, N)))
        t.close(sig.cpu().numpy()[ran], r.signal[ran], TOL, f"step {step} signal")
        t.rel(logits.cpu().numpy(), r.logits, TOL, f"step {step} logits")
        t.token(int(nxt.item()), r.logits, TOL, f"step {step} token")
        skipped = [l for l in (r.exit_boundary, (r.exit_boundary + N) // 2, N - 1) if l < N]
        _check_cache(kv, cache, 0, pos, pos + 1, t, sorted(set([0] + skipped)), f"step {step}")
        t.steps += 1
        tok_d.copy_(nxt)
    assert t.steps == 3 and exits >= 1


def test_phi3_arla_exit_step(world):
    """EXIT mode decided by the latent-attention exit router (Sec. 2.3.1) at
    gates 8, 16 and 24 (intervals of eight fast states), bias 1.5 on the
    last gate's readout so that some steps exit: boundary, token, signals of
    the layers that ran and the skipped layers' cache entries."""
    model, orc, _ = world
    N, tau, gates = CFG.n_layers, 0.7, [8, 16, 24]
    a = synth.arla_weights(CFG)
    a["b_out"][24] = 1.5
    model.set_arla(a)
    try:
        t = Tally()
        kv = PagedKV(CFG, 1, 64, block_size=16, block_table=shuffled_table(1, 64, 16, 4))
        cache = KVCache(CFG, 64)
        prompt = list(synth.prompt_ids(CFG, PROMPT, stream="arla"))
        tok, pos_d = _prefill(model, orc, kv, cache, prompt, t)
        dev = torch.device("cuda")
        tok_d = torch.tensor([tok], dtype=torch.int32, device=dev)
        nxt = torch.zeros(1, dtype=torch.int32, device=dev)
        exb = torch.zeros(1, dtype=torch.int32, device=dev)
        sig = torch.zeros(N, dtype=torch.float32, device=dev)
        logits = torch.zeros(CFG.vocab, dtype=torch.float32, device=dev)
        for step in range(3):
            pos = PROMPT + step
            tau_s = pick_tau(orc, int(tok_d.item()), pos, cache, gates, (tau, 0.69, 0.71, 0.68, 0.72, 0.66, 0.74),
                             EXIT_EPS, arla=a)
            assert tau_s is not None, f"step {step}: every threshold lies near a gate score"
            model.decode_step(tok_d, pos_d, kv.desc(), gates=gates, tau=tau_s, mode="exit", next_token=nxt,
                              exit_boundary=exb, signal=sig, logits=logits, advance=True)
            torch.cuda.synchronize()
            r = orc.decode_step(int(tok_d.item()), pos, cache, gates=gates, tau=tau_s, mode="exit", arla=a)
            t.equal(int(exb.item()), r.exit_boundary, f"step {step} exit boundary")
            ran = list(range(min(r.exit_boundary, N)))
            t.close(sig.cpu().numpy()[ran], r.signal[ran], TOL, f"step {step} signal")
            t.rel(logits.cpu().numpy(), r.logits, TOL, f"step {step} logits")
            t.token(int(nxt.item()), r.logits, TOL, f"step {step} token")
            skipped = [l for l in (r.exit_boundary, N - 1) if l < N]
            _check_cache(kv, cache, 0, pos, pos + 1, t, sorted(set([0] + skipped)), f"step {step}")
            t.steps += 1
            tok_d.copy_(nxt)
        assert t.steps == 3
    finally:
        model.set_arla(None)


def test_phi3_draft_and_verify(world):
    """gamma = 4 drafts from the fast stream exiting at layer 8, then the
    5-row verification chunk through all 32 layers."""
    model, orc, _ = world
    gamma, kL = 4, 8
    t = Tally()
    kv = PagedKV(CFG, 1, 64, block_size=16, block_table=shuffled_table(1, 64, 16, 9))
    cache = KVCache(CFG, 64)
    prompt = list(synth.prompt_ids(CFG, PROMPT, stream="spec"))
    tok, pos_d = _prefill(model, orc, kv, cache, prompt, t)
    dev = torch.device("cuda")
    buf = torch.zeros(gamma + 1, dtype=torch.int32, device=dev)
    buf[0] = tok
    targets = torch.zeros(gamma + 1, dtype=torch.int32, device=dev)
    n_acc = torch.zeros(1, dtype=torch.int32, device=dev)
    model.draft(buf[0:1], pos_d, kL, gamma, kv.desc(), buf[1:])
    torch.cuda.synchronize()
    drafts = buf[1:].cpu().numpy().tolist()
    _, ref_z = oracle_draft_logits(orc, tok, PROMPT, cache, kL, gamma, drafts_fed=drafts)
    for j in range(gamma):
        t.token(drafts[j], ref_z[j], TOL, f"draft {j}")
    model.verify(buf, gamma + 1, pos_d, kv.desc(), targets, n_accepted=n_acc, bonus=buf[0:1])
    torch.cuda.synchronize()
    tg = targets.cpu().numpy().tolist()
    ref = orc.slow_chunk([tok] + drafts, PROMPT, cache)
    for i in range(gamma + 1):
        t.token(tg[i], ref[i], TOL, f"target {i}")
    j = 0
    while j < gamma and drafts[j] == tg[j]:
        j += 1
    t.equal(int(n_acc.item()), j, "accepted")
    t.equal(int(buf[0].item()), tg[j], "bonus")
    assert int(pos_d.item()) == PROMPT + j + 1 == int(kv.seq_lens[0].item())
    _check_cache(kv, cache, 0, PROMPT, PROMPT + j + 1, t, (0, 8, 31), "verify")
    assert t.compared >= 2 + gamma + 1


def test_batch8_long_context_step(world):
    """8 sequences, 4096-token contexts each (seeded N(0,1) cache content,
    shuffled block table), one dual-stream step; sequences 0 and 5 are
    recomputed by the oracle."""
    model, orc, _ = world
    B, sampled = 8, (0, 5)
    t = Tally()
    max_ctx = CTX_B + 16
    bps = (max_ctx + 15) // 16
    kv = PagedKV(CFG, B, max_ctx, block_size=16, block_table=synth.block_table(B, bps, seed=3))
    caches = {}
    for s in range(B):
        content = synth.synthetic_kv(CFG, CTX_B, seq=s, threads=16)
        for l, (K, V) in content.items():
            kv.load(s, l, K, V)
        if s in sampled:
            c = KVCache(CFG, max_ctx)
            for l, (K, V) in content.items():
                c.load(l, K, V)
            caches[s] = c
        del content
    kv.seq_lens.fill_(CTX_B)
    dev = torch.device("cuda")
    toks = synth.prompt_ids(CFG, B, stream="batch")
    tok_d = torch.tensor(toks, dtype=torch.int32, device=dev)
    pos_d = torch.full((B,), CTX_B, dtype=torch.int32, device=dev)
    N = CFG.n_layers
    gates = list(range(1, N))
    nxt = torch.zeros(B, dtype=torch.int32, device=dev)
    sig = torch.zeros(B * N, dtype=torch.float32, device=dev)
    logits = torch.zeros(B * CFG.vocab, dtype=torch.float32, device=dev)
    h_out = torch.zeros(B * CFG.d_model, dtype=torch.float32, device=dev)
    p_out = torch.zeros(B * CFG.d_model, dtype=torch.float32, device=dev)
    model.decode_step(tok_d, pos_d, kv.desc(), gates=gates, tau=0.9, mode="observe", next_token=nxt, signal=sig,
                      logits=logits, h_out=h_out, p_out=p_out, advance=True)
    torch.cuda.synchronize()
    assert pos_d.cpu().numpy().tolist() == [CTX_B + 1] * B
    L = logits.cpu().numpy().reshape(B, -1)
    Hh = h_out.cpu().numpy().reshape(B, -1)
    Pp = p_out.cpu().numpy().reshape(B, -1)
    S = sig.cpu().numpy().reshape(B, N)
    for s in sampled:
        r = orc.decode_step(int(toks[s]), CTX_B, caches[s], gates=gates, tau=0.9, mode="observe")
        t.rel(L[s], r.logits, TOL, f"seq {s} logits")
        t.rel(Hh[s], r.h, TOL, f"seq {s} h")
        t.rel(Pp[s], r.p, TOL, f"seq {s} p")
        t.close(S[s], r.signal, TOL, f"seq {s} signal")
        t.token(int(nxt[s].item()), r.logits, TOL, f"seq {s} token")
        _check_cache(kv, caches[s], s, CTX_B, CTX_B + 1, t, (0, 16, 31), f"seq {s}")
        t.steps += 1
    assert t.steps == len(sampled)
