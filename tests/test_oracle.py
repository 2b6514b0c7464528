"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

Nothing here touches the GPU.  Each test names the passage or identity that
fixes the expected value:
  * brute force: a scalar-loop restatement (tests/bruteforce.py) on tiny shapes;
  * library routines: torch's rms_norm / silu / scaled-dot-product attention /
    bfloat16 conversion, and the HuggingFace Llama decoder for the slow stream;
  * invariants of the method (zero adapters collapse Eq. 2 onto Eq. 1,
    speculative decoding is lossless, the exit path at a gate equals a
    truncated decoder);
  * closed forms (RoPE is a rotation depending on relative position only).
"""
import math

import numpy as np
import pytest
import torch

import synth
from oracle import (Oracle, KVCache, rms_norm, rope, attend, silu, topk_desc, round_to_cache)
from tests.bruteforce import BruteDecoder

MICRO = synth.CONFIGS["micro"]
MICRO_MOE = synth.CONFIGS["micro_moe"]
TINY = synth.CONFIGS["tiny"]


def _weights(cfg, **kw):
    return synth.make_weights(cfg, threads=4, **kw)


# ---------------------------------------------------------------------------
# Elementary operations against library routines / closed forms
# ---------------------------------------------------------------------------

def test_rms_norm_matches_torch():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 37))
    g = rng.standard_normal(37)
    ref = torch.nn.functional.rms_norm(torch.tensor(x), (37,), torch.tensor(g), eps=1e-5).numpy()
    np.testing.assert_allclose(rms_norm(x, g, 1e-5), ref, rtol=1e-13, atol=1e-14)
    # closed form: with unit gain the output has mean square 1 (up to eps)
    y = rms_norm(x, np.ones(37), 0.0)
    np.testing.assert_allclose(np.mean(y * y, axis=-1), 1.0, rtol=1e-13)


def test_silu_matches_torch():
    x = np.linspace(-30, 30, 1001)
    np.testing.assert_allclose(silu(x), torch.nn.functional.silu(torch.tensor(x)).numpy(), rtol=1e-14, atol=1e-300)


def test_attend_matches_torch_sdpa():
    rng = np.random.default_rng(1)
    H, T, hd = 3, 9, 8
    q = rng.standard_normal((H, hd))
    K = rng.standard_normal((T, H, hd))
    V = rng.standard_normal((T, H, hd))
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.tensor(q)[:, None, :], torch.tensor(K).permute(1, 0, 2), torch.tensor(V).permute(1, 0, 2))[:, 0]
    np.testing.assert_allclose(attend(q, K, V), ref.numpy(), rtol=1e-12, atol=1e-13)
    # one key: attention returns its value
    np.testing.assert_allclose(attend(q, K[:1], V[:1]), V[0], rtol=0, atol=1e-15)


def test_rope_is_relative_rotation():
    rng = np.random.default_rng(2)
    H, hd = 2, 16
    q = rng.standard_normal((H, hd))
    k = rng.standard_normal((H, hd))
    # norm preserving
    np.testing.assert_allclose(np.linalg.norm(rope(q, 37, 1e4), axis=-1), np.linalg.norm(q, axis=-1), rtol=1e-13)
    # q_m . k_n depends only on m - n
    d1 = np.sum(rope(q, 10, 1e4) * rope(k, 3, 1e4), axis=-1)
    d2 = np.sum(rope(q, 107, 1e4) * rope(k, 100, 1e4), axis=-1)
    np.testing.assert_allclose(d1, d2, rtol=1e-11)
    # position 0 is the identity
    np.testing.assert_allclose(rope(q, 0, 1e4), q, rtol=0, atol=0)
    # pair (0, hd/2) at the first frequency rotates by exactly `pos` radians
    e = np.zeros((1, hd)); e[0, 0] = 1.0
    r = rope(e, 0.5, 1e4)
    np.testing.assert_allclose([r[0, 0], r[0, hd // 2]], [math.cos(0.5), math.sin(0.5)], rtol=1e-15)


def test_topk_is_stable_descending_sort():
    rng = np.random.default_rng(3)
    for _ in range(50):
        v = rng.integers(0, 5, size=17).astype(np.float64)   # many ties
        ref = np.argsort(-v, kind="stable")[:6]
        np.testing.assert_array_equal(topk_desc(v, 6), ref)


def test_bf16_rounding_matches_torch_and_ties_to_even():
    rng = np.random.default_rng(4)
    x = (rng.standard_normal(10000) * 10.0 ** rng.integers(-6, 6, 10000)).astype(np.float32)
    ref = torch.tensor(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(round_to_cache(x.astype(np.float64), "bf16"), ref)
    # exact midpoints between neighbouring bf16 values go to the even mantissa
    one_ulp = 2.0 ** -7
    assert round_to_cache(np.array([1.0 + one_ulp / 2]), "bf16")[0] == 1.0
    assert round_to_cache(np.array([1.0 + 3 * one_ulp / 2]), "bf16")[0] == 1.0 + 2 * one_ulp


# ---------------------------------------------------------------------------
# Whole decode step against the scalar-loop restatement (P5)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("mode,tau", [("observe", 2.0), ("observe", -1.0), ("exit", -1.0), ("exit", 0.3),
                                      ("off", 0.0)])
@pytest.mark.parametrize("kvdtype", ["f32", "f64"])
def test_decode_step_matches_bruteforce(mode, tau, kvdtype):
    cfg = MICRO.replace(kvdtype=kvdtype)
    w = _weights(cfg)
    orc = Oracle(cfg, w)
    bf = BruteDecoder(cfg, w)
    cache = KVCache(cfg, 16)
    tok = 3
    for pos in range(6):
        r = orc.decode_step(tok, pos, cache, gates=[1], tau=tau, mode=mode)
        b = bf.step(tok, pos, gates=[1], tau=tau, mode=mode)
        np.testing.assert_allclose(r.logits, b["logits"], rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(r.h, b["h"], rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(r.p, b["p"], rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(r.signal, b["signal"], rtol=1e-12, atol=1e-13)
        assert r.exit_boundary == b["exit_boundary"]
        for l in range(cfg.n_layers):
            np.testing.assert_allclose(cache.K[l][pos].reshape(-1), bf.K[l][pos], rtol=1e-12, atol=1e-13)
            np.testing.assert_allclose(cache.V[l][pos].reshape(-1), bf.V[l][pos], rtol=1e-12, atol=1e-13)
        tok = r.token


@pytest.mark.parametrize("mode", ["observe", "off"])
def test_moe_decode_step_matches_bruteforce(mode):
    cfg = MICRO_MOE
    w = _weights(cfg)
    orc = Oracle(cfg, w)
    bf = BruteDecoder(cfg, w)
    cache = KVCache(cfg, 16)
    tok = 5
    for pos in range(5):
        r = orc.decode_step(tok, pos, cache, mode=mode)
        b = bf.step(tok, pos, mode=mode)
        np.testing.assert_allclose(r.logits, b["logits"], rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(r.p, b["p"], rtol=1e-12, atol=1e-13)
        np.testing.assert_array_equal(r.slow_experts, np.array(b["experts"]))
        for lp in range(cfg.n_layers):
            if lp in b["preds"]:
                np.testing.assert_array_equal(r.pred_experts[lp], b["preds"][lp])
            else:
                assert (r.pred_experts[lp] == -1).all()
        tok = r.token


# ---------------------------------------------------------------------------
# Slow stream == a standard decoder (library implementation)
# ---------------------------------------------------------------------------

def _llama(cfg, w, n_layers=None):
    from transformers import LlamaConfig, LlamaForCausalLM
    n_layers = cfg.n_layers if n_layers is None else n_layers
    lc = LlamaConfig(vocab_size=cfg.vocab, hidden_size=cfg.d_model, intermediate_size=cfg.ffn,
                     num_hidden_layers=n_layers, num_attention_heads=cfg.n_heads, num_key_value_heads=cfg.n_heads,
                     head_dim=cfg.head_dim, rms_norm_eps=cfg.rms_eps, rope_theta=cfg.rope_theta,
                     tie_word_embeddings=False, attention_bias=False, mlp_bias=False,
                     max_position_embeddings=4096)
    lc._attn_implementation = "eager"
    m = LlamaForCausalLM(lc).double().eval()
    sd = {"model.embed_tokens.weight": w["embed"], "model.norm.weight": w["final_norm"], "lm_head.weight": w["lm_head"]}
    for l in range(n_layers):
        p = f"model.layers.{l}."
        sd.update({p + "self_attn.q_proj.weight": w[f"L{l}.wq"], p + "self_attn.k_proj.weight": w[f"L{l}.wk"],
                   p + "self_attn.v_proj.weight": w[f"L{l}.wv"], p + "self_attn.o_proj.weight": w[f"L{l}.wo"],
                   p + "mlp.gate_proj.weight": w[f"L{l}.wg"], p + "mlp.up_proj.weight": w[f"L{l}.wu"],
                   p + "mlp.down_proj.weight": w[f"L{l}.wd"], p + "input_layernorm.weight": w[f"L{l}.attn_norm"],
                   p + "post_attention_layernorm.weight": w[f"L{l}.mlp_norm"]})
    m.load_state_dict({k: torch.tensor(np.asarray(v, np.float64)) for k, v in sd.items()}, strict=True)
    return m


# HuggingFace's rotary embedding evaluates its angles in float32, so agreement
# with the float64 oracle is at the 1e-7 level; real wiring errors are O(1).
LLAMA_RTOL, LLAMA_ATOL = 1e-5, 2e-6


def _llama_logits(m, ids):
    with torch.no_grad():
        return m(torch.tensor([list(ids)])).logits[0].numpy()


def test_slow_stream_is_the_standard_decoder():
    """Eq. 1 with pre-norm RMSNorm, RoPE and SwiGLU == HuggingFace Llama."""
    cfg = TINY.replace(kvdtype="f64")
    w = _weights(cfg)
    orc = Oracle(cfg, w)
    ids = list(synth.prompt_ids(cfg, 12))
    ref = _llama_logits(_llama(cfg, w), ids)
    got = orc.slow_chunk(ids, 0, KVCache(cfg, 32))
    np.testing.assert_allclose(got, ref, rtol=LLAMA_RTOL, atol=LLAMA_ATOL)


def test_never_exit_dual_step_tokens_equal_standard_decoder():
    """P2: tau > 1 (no exit) -> the dual step emits the standard decoder's tokens."""
    cfg = TINY.replace(kvdtype="f64")
    w = _weights(cfg)
    orc = Oracle(cfg, w)
    m = _llama(cfg, w)
    prompt = list(synth.prompt_ids(cfg, 8))
    cache = KVCache(cfg, 64)
    logits = orc.slow_chunk(prompt, 0, cache)
    seq = prompt + [int(np.argmax(logits[-1]))]
    for _ in range(6):
        r = orc.decode_step(seq[-1], len(seq) - 1, cache, gates=[1], tau=1.5, mode="exit")
        assert r.exit_boundary == cfg.n_layers
        ref = _llama_logits(m, seq)[-1]
        np.testing.assert_allclose(r.logits, ref, rtol=LLAMA_RTOL, atol=LLAMA_ATOL)
        seq.append(r.token)


def test_exit_at_gate_equals_truncated_decoder():
    """P3: zero adapters, tau = -1, EXIT at gate b -> head(h_b) (Eq. 4 with p = h)."""
    cfg = TINY.replace(kvdtype="f64", n_layers=3)
    w = _weights(cfg, adapter_scale=0.0)
    orc = Oracle(cfg, w)
    ids = list(synth.prompt_ids(cfg, 6))
    for b in (1, 2):
        cache = KVCache(cfg, 16)
        orc.slow_chunk(ids[:-1], 0, cache)
        r = orc.decode_step(ids[-1], len(ids) - 1, cache, gates=[b], tau=-1.0, mode="exit")
        assert r.exit_boundary == b
        # truncated decoder: the first b layers, then the final norm and LM head;
        # the earlier positions of the truncated model see the same first-b-layer cache
        ref = _llama_logits(_llama(cfg, w, n_layers=b), ids)[-1]
        np.testing.assert_allclose(r.logits, ref, rtol=LLAMA_RTOL, atol=LLAMA_ATOL)


def test_zero_adapters_collapse_fast_stream():
    """P1: with zero adapters f_hat = f and g_hat = g, so p == h exactly."""
    cfg = TINY.replace(kvdtype="f64")
    w = _weights(cfg, adapter_scale=0.0)
    orc = Oracle(cfg, w)
    cache = KVCache(cfg, 32)
    tok = 7
    for pos in range(5):
        r = orc.decode_step(tok, pos, cache, mode="off")
        np.testing.assert_array_equal(r.p, r.h)
        tok = r.token


def test_fast_row_at_position_zero_is_decoder_with_merged_adapters():
    """At t = 0 the fast row sees only itself, so Eq. 2 with linear adapters is
    a standard decoder whose weights are W + B A (LoRA merge identity)."""
    cfg = TINY.replace(kvdtype="f64")
    w = _weights(cfg)
    orc = Oracle(cfg, w)
    merged = dict(w)
    for l in range(cfg.n_layers):
        for pr, nm in (("q", "wq"), ("k", "wk"), ("v", "wv"), ("o", "wo"), ("g", "wg"), ("u", "wu"), ("d", "wd")):
            merged[f"L{l}.{nm}"] = (w[f"L{l}.{nm}"].astype(np.float64) +
                                    w[f"L{l}.B_{pr}"].astype(np.float64) @ w[f"L{l}.A_{pr}"].astype(np.float64))
    tok = 42
    r = orc.decode_step(tok, 0, KVCache(cfg, 4), mode="off")
    ref_logits = _llama_logits(_llama(cfg, merged), [tok])[0]
    # the fast row's logits: apply the head to p
    np.testing.assert_allclose(orc.head_logits(r.p), ref_logits, rtol=LLAMA_RTOL, atol=LLAMA_ATOL)


# ---------------------------------------------------------------------------
# Chunked forward, speculative decoding
# ---------------------------------------------------------------------------

def test_chunk_forward_equals_sequential_steps():
    """P12: a causal chunk equals the same rows decoded one at a time."""
    cfg = TINY
    w = _weights(cfg)
    orc = Oracle(cfg, w)
    ids = list(synth.prompt_ids(cfg, 9))
    c1, c2 = KVCache(cfg, 32), KVCache(cfg, 32)
    a = orc.slow_chunk(ids, 0, c1)
    b = np.stack([orc.slow_chunk([t], i, c2)[0] for i, t in enumerate(ids)])
    np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-13)
    # and the dual step's slow logits are the same rows
    c3 = KVCache(cfg, 32)
    orc.slow_chunk(ids[:-1], 0, c3)
    r = orc.decode_step(ids[-1], len(ids) - 1, c3, mode="off")
    np.testing.assert_allclose(r.logits, a[-1], rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("gamma,exit_layer", [(1, 1), (3, 1), (4, 2)])
def test_speculative_equals_greedy(gamma, exit_layer):
    """P4: draft-then-verify under greedy acceptance is lossless."""
    cfg = TINY.replace(n_layers=3)
    w = _weights(cfg)
    orc = Oracle(cfg, w)
    prompt = list(synth.prompt_ids(cfg, 6))
    ref = orc.greedy(prompt, 14)
    got, st = orc.spec_generate(prompt, 14, gamma=gamma, exit_layer=exit_layer)
    assert got == ref
    bad, st2 = orc.spec_generate(prompt, 14, gamma=gamma, exit_layer=exit_layer, corrupt_drafts=True)
    assert bad == ref and st2["accepted"] == 0


def test_full_depth_draft_with_zero_adapters_is_always_accepted():
    """P4b: exit layer N and zero adapters -> drafts are the verifier's tokens."""
    cfg = TINY.replace(kvdtype="f64", n_layers=2)
    w = _weights(cfg, adapter_scale=0.0)
    orc = Oracle(cfg, w)
    prompt = list(synth.prompt_ids(cfg, 5))
    got, st = orc.spec_generate(prompt, 13, gamma=3, exit_layer=cfg.n_layers)
    assert got == orc.greedy(prompt, 13)
    assert st["accepted"] == st["drafted"]


def test_fp32_oracle_close_to_fp64():
    """P13: the float32 oracle (used for CPU timing) agrees with float64."""
    cfg = TINY
    w = _weights(cfg)
    a, b = Oracle(cfg, w, np.float64), Oracle(cfg, w, np.float32)
    ids = list(synth.prompt_ids(cfg, 6))
    la = a.slow_chunk(ids, 0, KVCache(cfg, 16, np.float64))
    lb = b.slow_chunk(ids, 0, KVCache(cfg, 16, np.float32))
    assert np.linalg.norm(la - lb) / np.linalg.norm(la) < 1e-5
