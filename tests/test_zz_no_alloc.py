"""The no-allocation decode step (m2r2_decode_step_noalloc: the step's
per-call scratch in the library's static device array) against the ordinary
decode step (scratch in the context's workspace), through the C ABI: two
contexts over the same weights, identical paged caches and inputs; two calls
in a row, the second with fewer sequences than the first.  Floating-point
outputs must agree within the parity tolerance (the row statistics are summed
with atomics whose order varies, so the two are not bitwise equal); tokens and
exit boundaries exactly where the logit margin and the gate signals decide
them.  Also: a context whose scratch exceeds the static maximum is refused
before anything is enqueued."""
import numpy as np
import pytest
import torch

import synth
from paper_2502_02040_amd import M2R2Error, Model, PagedKV
from tests.gpu_harness import Tally, shuffled_table, tol_of, token_decidable, track

pytestmark = pytest.mark.gpu


def _prefill(model, kv, cfg, lens):
    dev = torch.device("cuda")
    targets = torch.zeros(16, dtype=torch.int32, device=dev)
    for s, n in enumerate(lens):
        prompt = torch.tensor(synth.prompt_ids(cfg, n, stream=f"noalloc{s}"), dtype=torch.int32, device=dev)
        pos = torch.zeros(1, dtype=torch.int32, device=dev)
        for c0 in range(0, n, 16):
            k = min(16, n - c0)
            model.verify(prompt[c0:c0 + k], k, pos, kv.desc(s), targets)
    torch.cuda.synchronize()


@pytest.mark.parametrize("name", ["tiny", "small_bf16"])
def test_noalloc_step_matches_decode_step(name):
    cfg = synth.CONFIGS[name]
    w = synth.make_weights(cfg)
    tol = tol_of(cfg)
    N, B, max_ctx = cfg.n_layers, 3, 64
    lens = [5, 19, 11]
    dev = torch.device("cuda")
    sides = []
    for _ in range(2):
        m = track(Model(cfg, w, max_batch=B, max_chunk=16, max_ctx=max_ctx))
        kv = PagedKV(cfg, B, max_ctx, block_size=16, block_table=shuffled_table(B, max_ctx, 16, 5))
        _prefill(m, kv, cfg, lens)
        sides.append((m, kv, torch.tensor(lens, dtype=torch.int32, device=dev)))
    t = Tally()
    gates = list(range(1, N))
    for call, batch in enumerate((3, 1)):   # the second call decodes fewer sequences
        toks = torch.tensor(synth.prompt_ids(cfg, batch, stream=f"noalloc_call{call}"), dtype=torch.int32,
                            device=dev)
        res = []
        for k, (m, kv, pos) in enumerate(sides):
            o = dict(nxt=torch.zeros(batch, dtype=torch.int32, device=dev),
                     exb=torch.zeros(batch, dtype=torch.int32, device=dev),
                     sig=torch.zeros(batch * N, dtype=torch.float32, device=dev),
                     logits=torch.zeros(batch * cfg.vocab, dtype=torch.float32, device=dev),
                     h=torch.zeros(batch * cfg.d_model, dtype=torch.float32, device=dev),
                     p=torch.zeros(batch * cfg.d_model, dtype=torch.float32, device=dev))
            m.decode_step(toks, pos[:batch], kv.desc(), gates=gates, tau=0.9, mode="observe", next_token=o["nxt"],
                          exit_boundary=o["exb"], signal=o["sig"], logits=o["logits"], h_out=o["h"], p_out=o["p"],
                          advance=True, noalloc=(k == 1))
            torch.cuda.synchronize()
            res.append({key: v.cpu().numpy() for key, v in o.items()})
        ref, got = res
        L_ref, L_got = ref["logits"].reshape(batch, -1), got["logits"].reshape(batch, -1)
        S_ref, S_got = ref["sig"].reshape(batch, N), got["sig"].reshape(batch, N)
        for s in range(batch):
            t.rel(L_got[s], L_ref[s], tol, f"call {call} seq {s} logits")
            t.rel(got["h"].reshape(batch, -1)[s], ref["h"].reshape(batch, -1)[s], tol, f"call {call} seq {s} h")
            t.rel(got["p"].reshape(batch, -1)[s], ref["p"].reshape(batch, -1)[s], tol, f"call {call} seq {s} p")
            t.close(S_got[s], S_ref[s], tol, f"call {call} seq {s} signal")
            if token_decidable(L_ref[s], tol):
                t.equal(int(got["nxt"][s]), int(ref["nxt"][s]), f"call {call} seq {s} token")
            else:
                t.skipped += 1
            if all(abs(S_ref[s][b - 1] - 0.9) > tol for b in gates):
                t.equal(int(got["exb"][s]), int(ref["exb"][s]), f"call {call} seq {s} exit boundary")
            else:
                t.skipped += 1
            p0 = lens[s] + call
            for l in range(N):
                Kr, Vr = sides[0][1].read(s, l, p0, p0 + 1)
                Kg, Vg = sides[1][1].read(s, l, p0, p0 + 1)
                t.rel(Kg, Kr, tol, f"call {call} seq {s} K layer {l}")
                t.rel(Vg, Vr, tol, f"call {call} seq {s} V layer {l}")
            t.steps += 1
        assert sides[0][2].cpu().tolist() == sides[1][2].cpu().tolist()
    assert t.steps == 3 + 1 and t.compared >= 4
    for m, _, _ in sides:
        m.sync_check()


def test_noalloc_refuses_scratch_above_the_static_maximum():
    """32 heads of width 128 with 8 sequences and long contexts: the attention
    partials alone need about 170 MB of scratch, above the 32 MiB array."""
    cfg = synth.ModelConfig("noalloc_big", n_layers=1, d_model=64, n_heads=32, head_dim=128, ffn=64, vocab=64,
                            rank=32, wdtype="f32", kvdtype="f32", seed=29)
    w = synth.make_weights(cfg)
    m = track(Model(cfg, w, max_batch=8, max_chunk=16, max_ctx=8192))
    kv = PagedKV(cfg, 1, 64, block_size=16)
    dev = torch.device("cuda")
    tok = torch.zeros(1, dtype=torch.int32, device=dev)
    pos = torch.zeros(1, dtype=torch.int32, device=dev)
    nxt = torch.zeros(1, dtype=torch.int32, device=dev)
    with pytest.raises(M2R2Error) as e:
        m.decode_step(tok, pos, kv.desc(), next_token=nxt, noalloc=True)
    assert e.value.status == -2 and "static maximum" in str(e.value)
    m.sync_check()
