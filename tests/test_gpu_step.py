"""GPU parity of the dual-stream decode step, the chunked slow forward and the
self-speculative draft/verify, through the C ABI, against the CPU oracle.

Inputs are the seeded synthetic weights and prompts of synth; the paged
cache uses a shuffled block table.  Sizes: the tiny float32 decoder (2
layers, d 256, 4 heads x 64; one sequence runs the one-launch step), a small
bfloat16 decoder (3 layers, d 192, 2 heads x 96, ffn 320: tiles of 16 rows
leave ragged tails in the LM head, vocab 1000; rows not whole 1 KB pieces:
the multi-kernel path) and a small bfloat16 decoder with head_dim 128 (3
layers, d 512, 4 heads; the one-launch step)."""
import numpy as np
import pytest
import torch

import synth
from tests.gpu_harness import Pair, Tally, oracle_draft_logits, pick_tau

pytestmark = pytest.mark.gpu

CASES = ["tiny", "small_bf16", "small_rw"]


TAU_ALTERNATIVES = (0.45, 0.55, 0.4, 0.6, 0.35, 0.65, 0.3, 0.7)


def _decode_run(name, *, mode, tau, gates, n_steps, adapter_scale=1.0, block_size=16, prompt_len=16, arla=None,
                max_ctx=None):
    """Prefill, then n_steps dual-stream decode steps compared with the
    oracle step by step (teacher-forced on the GPU's tokens).  In OBSERVE
    mode the outputs do not depend on the gate decisions (p restarts from h
    at every gate), so a signal within tol of tau only leaves the exit
    boundary uncompared.  In EXIT mode the threshold of each step is `tau`,
    or the first alternative that every gate signal of the step decides
    clearly, so every step is compared in full."""
    cfg = synth.CONFIGS[name]
    w = synth.make_weights(cfg, adapter_scale=adapter_scale)
    pair = Pair(cfg, w, max_ctx=max_ctx or prompt_len + n_steps + 8, block_size=block_size, table_seed=3)
    if arla is not None:
        pair.model.set_arla(arla)
    t = Tally()
    prompt = list(synth.prompt_ids(cfg, prompt_len))
    tok = pair.prefill(prompt, tally=t)
    pair.check_cache(0, 0, prompt_len, t, "prefill")
    dev = pair.dev
    N = cfg.n_layers
    tok_d = torch.tensor([tok], dtype=torch.int32, device=dev)
    pos_d = torch.tensor([prompt_len], dtype=torch.int32, device=dev)
    nxt = torch.zeros(1, dtype=torch.int32, device=dev)
    exb = torch.zeros(1, dtype=torch.int32, device=dev)
    sig = torch.zeros(N, dtype=torch.float32, device=dev)
    logits = torch.zeros(cfg.vocab, dtype=torch.float32, device=dev)
    h_out = torch.zeros(cfg.d_model, dtype=torch.float32, device=dev)
    p_out = torch.zeros(cfg.d_model, dtype=torch.float32, device=dev)
    exits = 0
    for step in range(n_steps):
        pos = prompt_len + step
        tk = int(tok_d.item())
        tau_s = tau
        if mode == "exit" and gates:
            tau_s = pick_tau(pair.orc, tk, pos, pair.caches[0], gates, (tau,) + TAU_ALTERNATIVES, pair.tol, arla=arla)
            assert tau_s is not None, f"step {step}: every threshold lies within tol of a gate signal"
        pair.model.decode_step(tok_d, pos_d, pair.kv.desc(), gates=gates, tau=tau_s, mode=mode, next_token=nxt,
                               exit_boundary=exb, signal=sig, logits=logits, h_out=h_out, p_out=p_out, advance=True)
        torch.cuda.synchronize()
        r = pair.orc.decode_step(tk, pos, pair.caches[0], gates=gates, tau=tau_s, mode=mode, arla=arla)
        assert int(pos_d.item()) == pos + 1 and int(pair.kv.seq_lens[0].item()) == pos + 1
        if mode == "off" or all(abs(r.signal[b - 1] - tau_s) > pair.tol for b in gates):
            t.equal(int(exb.item()), r.exit_boundary, f"step {step}: exit boundary")
        else:
            t.skipped += 1
        t.rel(logits.cpu().numpy(), r.logits, pair.tol, f"step {step} logits")
        t.rel(h_out.cpu().numpy(), r.h, pair.tol, f"step {step} h")
        t.rel(p_out.cpu().numpy(), r.p, pair.tol, f"step {step} p")
        ran = [l for l in range(N) if not (mode == "exit" and r.exit_boundary < N and l >= r.exit_boundary)]
        t.close(sig.cpu().numpy()[ran], r.signal[ran], pair.tol, f"step {step} signal")
        t.token(int(nxt.item()), r.logits, pair.tol, f"step {step} token")
        pair.check_cache(0, pos, pos + 1, t, f"step {step}")
        t.steps += 1
        exits += r.exit_boundary < N
        tok_d.copy_(nxt)
    return t, exits, pair


def _one_launch_steps(pair):
    """Launches of the one-launch step kernel in one more decode step."""
    dev = pair.dev
    pos = pair.kv.seq_lens[:1].clone()
    tok = torch.zeros(1, dtype=torch.int32, device=dev)
    pair.model.timing_enable("step")
    pair.model.decode_step(tok, pos, pair.kv.desc(), gates=[1], tau=0.5, mode="observe", next_token=tok,
                           advance=False)
    torch.cuda.synchronize()
    n = pair.model.timing_read()[1]
    pair.model.timing_enable(None)
    return n


@pytest.mark.parametrize("name", CASES)
def test_dual_step_observe(name):
    """OBSERVE mode at every interior boundary: slow token, fast state,
    per-layer signal and the paged cache match the oracle step by step."""
    cfg = synth.CONFIGS[name]
    gates = list(range(1, cfg.n_layers))
    t, _, pair = _decode_run(name, mode="observe", tau=0.9, gates=gates, n_steps=12)
    assert t.steps == 12 and t.compared >= 12
    # which path one sequence took: the one-launch step where the shape has it
    assert _one_launch_steps(pair) == (0 if name == "small_bf16" else 1)


@pytest.mark.parametrize("name", CASES)
@pytest.mark.parametrize("tau", [-1.0, 0.5])
def test_dual_step_exit(name, tau):
    """EXIT mode: the token comes from the fast row at the gate and the
    skipped layers' cache entries are projected from the slow row."""
    t, exits, _ = _decode_run(name, mode="exit", tau=tau, gates=[1], n_steps=8)
    assert t.steps == 8 and t.compared >= 8
    if tau < 0:
        assert exits == 8


@pytest.mark.parametrize("name", ["tiny", "small_rw"])
@pytest.mark.parametrize("mode,tau,gates", [("observe", 0.9, None), ("exit", 0.5, [1])])
def test_one_sequence_on_the_multi_kernel_path(name, mode, tau, gates, monkeypatch):
    """The shapes that have the one-launch step, with it switched off: one
    sequence runs the multi-kernel path (one launch per phase and layer),
    which must match the oracle as well."""
    monkeypatch.setenv("M2R2_ONE_LAUNCH", "0")
    cfg = synth.CONFIGS[name]
    t, _, pair = _decode_run(name, mode=mode, tau=tau, gates=gates or list(range(1, cfg.n_layers)), n_steps=6)
    assert t.steps == 6 and t.compared >= 6
    assert _one_launch_steps(pair) == 0


def _arla(name, bias=0.0):
    cfg = synth.CONFIGS[name]
    a = synth.arla_weights(cfg)
    a["b_out"][:] = bias
    return a


@pytest.mark.parametrize("name", CASES)
@pytest.mark.parametrize("gate_set", ["last", "all"])
def test_arla_signal_observe(name, gate_set):
    """Latent-attention exit router (Sec. 2.3.1): in OBSERVE mode the router
    score at every gate and every other signal match the oracle.  Gates at
    the last boundary only: one interval from the embedding over two layers
    (three-layer shapes); at every boundary: the later intervals start from
    the slow state the fast row restarts from."""
    cfg = synth.CONFIGS[name]
    gates = [cfg.n_layers - 1] if gate_set == "last" else list(range(1, cfg.n_layers))
    t, _, _ = _decode_run(name, mode="observe", tau=0.5, gates=gates, n_steps=6, arla=_arla(name))
    assert t.steps == 6 and t.compared >= 6


@pytest.mark.parametrize("name", CASES)
@pytest.mark.parametrize("bias", [-40.0, 40.0, 0.0])
def test_arla_exit(name, bias):
    """EXIT mode decided by the router at every interior boundary: a large
    bias forces (or forbids) the exit at the first gate; bias 0 leaves it to
    the latent attention."""
    cfg = synth.CONFIGS[name]
    gates = list(range(1, cfg.n_layers))
    t, exits, _ = _decode_run(name, mode="exit", tau=0.5, gates=gates, n_steps=5, arla=_arla(name, bias))
    assert t.steps == 5 and t.compared >= 5
    if bias > 0:
        assert exits == 5
    if bias < 0:
        assert exits == 0


def test_arla_switched_off_restores_cosine_signal():
    cfg = synth.CONFIGS["tiny"]
    w = synth.make_weights(cfg)
    pair = Pair(cfg, w, max_ctx=32, table_seed=3)
    pair.model.set_arla(_arla("tiny", 40.0))
    pair.model.set_arla(None)
    t = Tally()
    tok = pair.prefill(list(synth.prompt_ids(cfg, 8)), tally=t)
    dev = pair.dev
    nxt = torch.zeros(1, dtype=torch.int32, device=dev)
    exb = torch.zeros(1, dtype=torch.int32, device=dev)
    sig = torch.zeros(cfg.n_layers, dtype=torch.float32, device=dev)
    pos_d = torch.tensor([8], dtype=torch.int32, device=dev)
    pair.model.decode_step(torch.tensor([tok], dtype=torch.int32, device=dev), pos_d, pair.kv.desc(), gates=[1],
                           tau=2.0, mode="exit", next_token=nxt, exit_boundary=exb, signal=sig, advance=True)
    torch.cuda.synchronize()
    r = pair.orc.decode_step(tok, 8, pair.caches[0], gates=[1], tau=2.0, mode="exit")
    assert int(exb.item()) == cfg.n_layers == r.exit_boundary
    assert abs(float(sig[0]) - r.signal[0]) <= pair.tol


@pytest.mark.parametrize("name", CASES)
def test_decode_to_cache_capacity(name):
    """The last steps fill the cache exactly: positions 250..255 of a 256-slot
    cache (two 128-token attention splits, the last block's last slot)."""
    t, _, _ = _decode_run(name, mode="observe", tau=0.9, gates=[1], n_steps=6, prompt_len=250, max_ctx=256)
    assert t.steps == 6 and t.compared >= 6


@pytest.mark.parametrize("name", CASES)
def test_zero_adapters_fast_row_tracks_slow_row(name):
    """P1 on the GPU: zero adapters, no gates -> the GPU's p equals the
    oracle's h within tolerance, every step (the oracle's p equals its h up to
    the rounding of the cache precision)."""
    cfg = synth.CONFIGS[name]
    w = synth.make_weights(cfg, adapter_scale=0.0)
    pair = Pair(cfg, w, max_ctx=32, table_seed=3)
    t = Tally()
    tok = pair.prefill(list(synth.prompt_ids(cfg, 9)), tally=t)
    dev = pair.dev
    tok_d = torch.tensor([tok], dtype=torch.int32, device=dev)
    pos_d = torch.tensor([9], dtype=torch.int32, device=dev)
    nxt = torch.zeros(1, dtype=torch.int32, device=dev)
    h_out = torch.zeros(cfg.d_model, dtype=torch.float32, device=dev)
    p_out = torch.zeros(cfg.d_model, dtype=torch.float32, device=dev)
    for step in range(4):
        pair.model.decode_step(tok_d, pos_d, pair.kv.desc(), mode="off", next_token=nxt, h_out=h_out, p_out=p_out,
                               advance=True)
        torch.cuda.synchronize()
        r = pair.orc.decode_step(int(tok_d.item()), 9 + step, pair.caches[0], mode="off")
        # the slow row reads its own key/value back from the cache (rounded to
        # the cache precision), the fast row uses its exact ones
        assert np.linalg.norm(r.p - r.h) <= (4e-3 if cfg.kvdtype == "bf16" else 1e-6) * np.linalg.norm(r.h)
        t.rel(p_out.cpu().numpy(), r.h, pair.tol, f"step {step} p vs h")
        t.rel(h_out.cpu().numpy(), r.h, pair.tol, f"step {step} h")
        t.steps += 1
        tok_d.copy_(nxt)
    assert t.steps == 4


@pytest.mark.parametrize("block_size", [1, 16, 64])
def test_block_size_and_table_invariance(block_size):
    """P8: results do not depend on the block size or the block-table
    permutation: every block size matches the (unpaged) oracle step by step."""
    t, _, _ = _decode_run("tiny", mode="observe", tau=0.9, gates=[1], n_steps=4, block_size=block_size)
    assert t.steps == 4 and t.compared >= 4


@pytest.mark.parametrize("name", CASES)
def test_single_stream_step(name):
    """dual = 0: the slow row alone (plain decoding on the same kernels)."""
    cfg = synth.CONFIGS[name]
    w = synth.make_weights(cfg)
    pair = Pair(cfg, w, max_ctx=40)
    t = Tally()
    prompt = list(synth.prompt_ids(cfg, 9))
    tok = pair.prefill(prompt, tally=t)
    dev = pair.dev
    tok_d = torch.tensor([tok], dtype=torch.int32, device=dev)
    pos_d = torch.tensor([len(prompt)], dtype=torch.int32, device=dev)
    nxt = torch.zeros(1, dtype=torch.int32, device=dev)
    logits = torch.zeros(cfg.vocab, dtype=torch.float32, device=dev)
    for step in range(6):
        pos = len(prompt) + step
        pair.model.decode_step(tok_d, pos_d, pair.kv.desc(), dual=False, next_token=nxt, logits=logits, advance=True)
        torch.cuda.synchronize()
        ref = pair.orc.slow_chunk([int(tok_d.item())], pos, pair.caches[0])[0]
        t.rel(logits.cpu().numpy(), ref, pair.tol, f"step {step}")
        t.token(int(nxt.item()), ref, pair.tol)
        pair.check_cache(0, pos, pos + 1, t)
        t.steps += 1
        tok_d.copy_(nxt)
    assert t.steps == 6


@pytest.mark.parametrize("name", CASES)
@pytest.mark.parametrize("gamma,exit_layer", [(3, 1), (4, 2)])
def test_draft_and_verify(name, gamma, exit_layer):
    """Draft from the fast row exiting at `exit_layer`, verify on the slow
    stream: drafts, targets and the acceptance bookkeeping match the oracle."""
    cfg = synth.CONFIGS[name]
    if exit_layer > cfg.n_layers:
        pytest.skip("exit layer beyond depth")
    w = synth.make_weights(cfg)
    pair = Pair(cfg, w, max_ctx=64)
    t = Tally()
    prompt = list(synth.prompt_ids(cfg, 11))
    tok = pair.prefill(prompt, tally=t)
    dev = pair.dev
    buf = torch.zeros(gamma + 1, dtype=torch.int32, device=dev)   # [last, d1..d_gamma]
    buf[0] = tok
    pos_d = torch.tensor([len(prompt)], dtype=torch.int32, device=dev)
    targets = torch.zeros(gamma + 1, dtype=torch.int32, device=dev)
    n_acc = torch.zeros(1, dtype=torch.int32, device=dev)
    pos = len(prompt)
    for rnd in range(4):
        last = int(buf[0].item())
        pair.model.draft(buf[0:1], pos_d, exit_layer, gamma, pair.kv.desc(), buf[1:])
        torch.cuda.synchronize()
        drafts = buf[1:].cpu().numpy().tolist()
        # oracle drafts from the same state, teacher-forced on the GPU's drafts:
        # every draft is compared under the margin rule
        _, ref_z = oracle_draft_logits(pair.orc, last, pos, pair.caches[0], exit_layer, gamma, drafts_fed=drafts)
        for j in range(gamma):
            t.token(drafts[j], ref_z[j], pair.tol, f"round {rnd} draft {j}")
        # draft cache entries (fast k/v of layers < exit_layer at pos..pos+gamma-1) are scratch: not compared
        pair.model.verify(buf, gamma + 1, pos_d, pair.kv.desc(), targets, n_accepted=n_acc, bonus=buf[0:1])
        torch.cuda.synchronize()
        tg = targets.cpu().numpy().tolist()
        ref = pair.orc.slow_chunk([last] + drafts, pos, pair.caches[0])
        for i in range(gamma + 1):
            t.token(tg[i], ref[i], pair.tol, f"round {rnd} target {i}")
        j = 0
        while j < gamma and drafts[j] == tg[j]:
            j += 1
        t.equal(int(n_acc.item()), j, f"round {rnd} accepted")
        t.equal(int(buf[0].item()), tg[j], f"round {rnd} bonus")
        assert int(pos_d.item()) == pos + j + 1 == int(pair.kv.seq_lens[0].item())
        pair.check_cache(0, pos, pos + j + 1, t, f"round {rnd}")
        t.steps += 1
        pos += j + 1
    assert t.steps == 4
    # drafts and targets: 4 rounds of 2 * gamma + 1 margin-ruled decisions, most of them decided
    assert t.compared >= 4 * (gamma + 1)


@pytest.mark.parametrize("name", CASES)
@pytest.mark.parametrize("chunks,B", [("1", 3), ("2", 3), ("4", 3), ("1", 8)])
def test_batched_dual_step(name, chunks, B, monkeypatch):
    """Three (eight) sequences with different context lengths decoded
    together (two rows each: the batched short-chain attention with one, two
    or four 128-token chunks per split, and the 8-row (16-row) tile GEMVs):
    every sequence's logits, h, p, signal, token and cache entry match the
    oracle step by step."""
    monkeypatch.setenv("M2R2_ATTN_CHUNKS", chunks)
    cfg = synth.CONFIGS[name]
    w = synth.make_weights(cfg)
    n_steps = 4
    lens = [5, 19, 37, 2, 11, 30, 8, 23][:B]
    pair = Pair(cfg, w, max_ctx=64, table_seed=5, max_batch=B, n_seqs=B)
    t = Tally()
    toks = [pair.prefill(list(synth.prompt_ids(cfg, n, stream=f"b{s}")), seq=s, tally=t) for s, n in enumerate(lens)]
    dev = pair.dev
    N = cfg.n_layers
    gates = list(range(1, N))
    tok_d = torch.tensor(toks, dtype=torch.int32, device=dev)
    pos_d = torch.tensor(lens, dtype=torch.int32, device=dev)
    nxt = torch.zeros(B, dtype=torch.int32, device=dev)
    sig = torch.zeros(B * N, dtype=torch.float32, device=dev)
    logits = torch.zeros(B * cfg.vocab, dtype=torch.float32, device=dev)
    h_out = torch.zeros(B * cfg.d_model, dtype=torch.float32, device=dev)
    p_out = torch.zeros(B * cfg.d_model, dtype=torch.float32, device=dev)
    for step in range(n_steps):
        pair.model.decode_step(tok_d, pos_d, pair.kv.desc(), gates=gates, tau=0.9, mode="observe", next_token=nxt,
                               signal=sig, logits=logits, h_out=h_out, p_out=p_out, advance=True)
        torch.cuda.synchronize()
        L = logits.cpu().numpy().reshape(B, -1)
        Hh, Pp = h_out.cpu().numpy().reshape(B, -1), p_out.cpu().numpy().reshape(B, -1)
        S = sig.cpu().numpy().reshape(B, N)
        got = nxt.cpu().numpy().tolist()
        for s in range(B):
            pos = lens[s] + step
            # OBSERVE mode: the outputs do not depend on the gate decisions
            r = pair.orc.decode_step(int(tok_d[s].item()), pos, pair.caches[s], gates=gates, tau=0.9, mode="observe")
            t.rel(L[s], r.logits, pair.tol, f"step {step} seq {s} logits")
            t.rel(Hh[s], r.h, pair.tol, f"step {step} seq {s} h")
            t.rel(Pp[s], r.p, pair.tol, f"step {step} seq {s} p")
            t.close(S[s], r.signal, pair.tol, f"step {step} seq {s} signal")
            t.token(got[s], r.logits, pair.tol, f"step {step} seq {s} token")
            pair.check_cache(s, pos, pos + 1, t, f"step {step} seq {s}")
            t.steps += 1
        assert pos_d.cpu().numpy().tolist() == [n + step + 1 for n in lens]
        tok_d.copy_(nxt)
    assert t.steps == n_steps * B and t.compared >= 3 * B
