"""Pins of the MoE parts of the oracle: the slow MoE stream against a library
MoE decoder, the speculation from the previous layer's residual state against
the library decoder's own hidden states, and the expert-cache simulations
against a textbook LRU, hand-worked traces and the special cases the policies
fix."""
from collections import OrderedDict

import numpy as np
import pytest
import torch

import synth
from oracle import Oracle, KVCache, simulate_expert_cache, simulate_fixed_experts

MOE = synth.ModelConfig("moe_pin", n_layers=3, d_model=64, n_heads=2, head_dim=32, ffn=0, vocab=50, rank=4,
                        wdtype="f32", kvdtype="f64", n_experts=8, top_k=2, expert_ffn=32, seed=21)


def _qwen2moe(cfg, w):
    """HuggingFace Qwen2-MoE with its extras disabled (zero q/k/v biases, zero
    shared expert, no top-k renormalisation): softmax router over all experts,
    top-k, combine with the raw probabilities."""
    from transformers import Qwen2MoeConfig, Qwen2MoeForCausalLM
    c = Qwen2MoeConfig(vocab_size=cfg.vocab, hidden_size=cfg.d_model, intermediate_size=cfg.expert_ffn,
                       moe_intermediate_size=cfg.expert_ffn, shared_expert_intermediate_size=cfg.expert_ffn,
                       num_hidden_layers=cfg.n_layers, num_attention_heads=cfg.n_heads,
                       num_key_value_heads=cfg.n_heads, num_experts=cfg.n_experts, num_experts_per_tok=cfg.top_k,
                       norm_topk_prob=False, decoder_sparse_step=1, mlp_only_layers=[], tie_word_embeddings=False,
                       rms_norm_eps=cfg.rms_eps, rope_theta=cfg.rope_theta, max_position_embeddings=1024)
    c._attn_implementation = "eager"
    c._experts_implementation = "eager"   # the per-expert loop (the grouped kernel has no float64)
    m = Qwen2MoeForCausalLM(c).double().eval()
    sd = {k: torch.zeros_like(v) for k, v in m.state_dict().items()}
    T = lambda a: torch.tensor(np.asarray(a, np.float64))
    sd["model.embed_tokens.weight"] = T(w["embed"])
    sd["model.norm.weight"] = T(w["final_norm"])
    sd["lm_head.weight"] = T(w["lm_head"])
    for l in range(cfg.n_layers):
        p = f"model.layers.{l}."
        for nm, key in (("wq", "q_proj"), ("wk", "k_proj"), ("wv", "v_proj"), ("wo", "o_proj")):
            sd[p + f"self_attn.{key}.weight"] = T(w[f"L{l}.{nm}"])
        sd[p + "input_layernorm.weight"] = T(w[f"L{l}.attn_norm"])
        sd[p + "post_attention_layernorm.weight"] = T(w[f"L{l}.mlp_norm"])
        sd[p + "mlp.gate.weight"] = T(w[f"L{l}.router"])
        sd[p + "mlp.experts.gate_up_proj"] = T(np.stack([np.concatenate([w[f"L{l}.E{e}.wg"], w[f"L{l}.E{e}.wu"]])
                                                         for e in range(cfg.n_experts)]))
        sd[p + "mlp.experts.down_proj"] = T(np.stack([w[f"L{l}.E{e}.wd"] for e in range(cfg.n_experts)]))
    m.load_state_dict(sd, strict=True)
    return m


def test_moe_slow_stream_matches_library_moe_decoder():
    cfg = MOE
    w = synth.make_weights(cfg, threads=4)
    ids = list(synth.prompt_ids(cfg, 10))
    with torch.no_grad():
        ref = _qwen2moe(cfg, w)(torch.tensor([ids])).logits[0].numpy()
    got = Oracle(cfg, w).slow_chunk(ids, 0, KVCache(cfg, 16))
    # the library evaluates rotary angles and router softmax in float32
    np.testing.assert_allclose(got, ref, rtol=1e-5, atol=2e-6)


def test_previous_layer_prediction_matches_library_hidden_states():
    """The previous-layer strategy of Sec. 3.3: layer l+1's router applied to
    the residual entering layer l's MLP.  The residual is captured from the
    library decoder (input of its post-attention norm) and fed to the
    library's own norm and router of layer l+1."""
    cfg = MOE
    N, K = cfg.n_layers, cfg.top_k
    w = synth.make_weights(cfg, threads=4)
    ids = list(synth.prompt_ids(cfg, 10))
    m = _qwen2moe(cfg, w)
    seen = {}
    hooks = [m.model.layers[l].post_attention_layernorm.register_forward_hook(
        lambda mod, inp, out, l=l: seen.__setitem__(l, inp[0][0, -1].detach().clone())) for l in range(N)]
    ref = {}
    with torch.no_grad():
        m(torch.tensor([ids]))
        for hk in hooks:
            hk.remove()
        for l in range(N - 1):
            nxt = m.model.layers[l + 1]
            z = nxt.mlp.gate(nxt.post_attention_layernorm(seen[l][None]))[0]
            ref[l + 1] = z[0].numpy()
    orc = Oracle(cfg, w)
    cache = KVCache(cfg, 16)
    orc.slow_chunk(ids[:-1], 0, cache)
    r = orc.decode_step(ids[-1], len(ids) - 1, cache)
    assert np.all(r.prev_pred_experts[0] == -1)
    for l in range(1, N):
        np.testing.assert_allclose(r.prev_pred_logits[l], ref[l], rtol=1e-6, atol=1e-9)
        assert set(r.prev_pred_experts[l]) == set(np.argsort(-ref[l])[:K].tolist())


def test_previous_layer_prediction_with_a_repeated_router_is_the_layers_own_choice():
    """If layer l+1 has layer l's router and norm gain, the prediction for
    l+1 equals the experts layer l itself chose (the same vector is routed)."""
    cfg = MOE
    w = dict(synth.make_weights(cfg, threads=4))
    for l in range(1, cfg.n_layers):
        w[f"L{l}.router"] = w["L0.router"]
        w[f"L{l}.mlp_norm"] = w["L0.mlp_norm"]
    orc = Oracle(cfg, w)
    cache = KVCache(cfg, 16)
    ids = list(synth.prompt_ids(cfg, 6))
    orc.slow_chunk(ids[:-1], 0, cache)
    r = orc.decode_step(ids[-1], len(ids) - 1, cache)
    for l in range(cfg.n_layers - 1):
        assert list(r.prev_pred_experts[l + 1]) == list(r.slow_experts[l])


def test_moe_dual_step_slow_logits_equal_chunk_forward():
    cfg = MOE
    w = synth.make_weights(cfg, threads=4)
    orc = Oracle(cfg, w)
    ids = list(synth.prompt_ids(cfg, 7))
    full = orc.slow_chunk(ids, 0, KVCache(cfg, 16))
    c = KVCache(cfg, 16)
    orc.slow_chunk(ids[:-1], 0, c)
    r = orc.decode_step(ids[-1], len(ids) - 1, c, mode="off")
    np.testing.assert_allclose(r.logits, full[-1], rtol=1e-12, atol=1e-13)
    # predictions exist exactly for layers 2i+2, 2i+3 below N
    assert (r.pred_experts[:2] == -1).all() and (r.pred_experts[2:] >= 0).all()


def _zero_expert_down(cfg, w):
    """The same weights with every expert's down projection zeroed: each MoE
    layer then adds nothing to the slow residual."""
    w = dict(w)
    for l in range(cfg.n_layers):
        for e in range(cfg.n_experts):
            w[f"L{l}.E{e}.wd"] = np.zeros_like(w[f"L{l}.E{e}.wd"])
    return w


def _library_layer_outputs(m, ids, N):
    """Residual leaving each decoder layer of the library model, last position."""
    seen = {}
    hooks = [m.model.layers[l].register_forward_hook(
        lambda mod, inp, out, l=l: seen.__setitem__(l, out[0, -1].detach().clone())) for l in range(N)]
    with torch.no_grad():
        m(torch.tensor([ids]))
    for hk in hooks:
        hk.remove()
    return seen


def _library_router_logits(m, l, x):
    """Layer l's own norm and router of the library model applied to residual x."""
    with torch.no_grad():
        lay = m.model.layers[l]
        return lay.mlp.gate(lay.post_attention_layernorm(x[None]))[0][0].numpy()


def _check_predictions_against_library(cfg, r, m, after):
    """Sec. 2.3.3 schedule: the fast state after layer i predicts the experts
    of layers 2i+2 and 2i+3 (each with that layer's own norm gain and router);
    layers 0 and 1 get no prediction.  `after[i]` is the library's residual
    after layer i that the fast state must equal.  (The library evaluates
    rotary angles in float32: values agree to about 1e-6; the top-k margins
    of these seeded routers are far larger, so the expert lists must be
    identical.)"""
    N, K = cfg.n_layers, cfg.top_k
    assert np.all(r.pred_experts[:2] == -1)
    checked = 0
    for i in range(N):
        for lp in (2 * i + 2, 2 * i + 3):
            if lp >= N:
                continue
            z = _library_router_logits(m, lp, after[i])
            np.testing.assert_allclose(r.pred_logits[lp], z, rtol=1e-5, atol=2e-6)
            order = np.argsort(-z, kind="stable")[:K]
            assert list(r.pred_experts[lp]) == order.tolist(), f"layer {lp}"
            checked += 1
    assert checked == N - 2


def test_zero_adapters_and_silent_experts_keep_fast_state_on_slow_state():
    """With zero adapters and zero expert down projections every MoE layer
    leaves both rows unchanged and the fast row's attention equals the slow
    row's, so p == h bitwise after every layer.  The predictions for layers
    2i+2 and 2i+3 are then the library decoder's own router choices on its
    residual after layer i (a multi-token prompt: the fast row attends to a
    real slow cache)."""
    cfg = MOE.replace(n_layers=6)
    w = _zero_expert_down(cfg, synth.make_weights(cfg, threads=4, adapter_scale=0.0))
    ids = list(synth.prompt_ids(cfg, 7))
    m = _qwen2moe(cfg, w)
    after = _library_layer_outputs(m, ids, cfg.n_layers)
    orc = Oracle(cfg, w)
    c = KVCache(cfg, 16)
    orc.slow_chunk(ids[:-1], 0, c)
    r = orc.decode_step(ids[-1], len(ids) - 1, c, mode="off")
    np.testing.assert_array_equal(r.p, r.h)
    for i in range(cfg.n_layers):
        np.testing.assert_allclose(r.fast_states[i], after[i].numpy(), rtol=1e-5, atol=2e-6)
    _check_predictions_against_library(cfg, r, m, after)


def test_zero_adapter_fast_stream_at_position_zero_is_the_attention_only_decoder():
    """With zero adapters and real experts the fast row differs from the slow
    one: its MLP is the (zero) adapter alone.  At position 0 it attends only
    to itself, so it is exactly the library decoder with the expert down
    projections zeroed, run on the one token; its predictions are that
    decoder's router choices on its residual after layer i."""
    cfg = MOE.replace(n_layers=6)
    w = synth.make_weights(cfg, threads=4, adapter_scale=0.0)
    tok = int(synth.prompt_ids(cfg, 1)[0])
    m = _qwen2moe(cfg, _zero_expert_down(cfg, w))
    after = _library_layer_outputs(m, [tok], cfg.n_layers)
    orc = Oracle(cfg, w)
    r = orc.decode_step(tok, 0, KVCache(cfg, 4), mode="off")
    assert np.linalg.norm(r.p - r.h) > 1e-3 * np.linalg.norm(r.h)   # the experts moved the slow row
    for i in range(cfg.n_layers):
        np.testing.assert_allclose(r.fast_states[i], after[i].numpy(), rtol=1e-5, atol=2e-6)
    _check_predictions_against_library(cfg, r, m, after)


# ---------------------------------------------------------------------------
# Expert cache simulation
# ---------------------------------------------------------------------------

def _textbook_lru(trace, E, C):
    """OrderedDict LRU per layer, warm start 0..C-1 (0 oldest); within a layer
    step the resident experts are touched first, then the missing ones are loaded."""
    T, N, K = trace.shape
    caches = [OrderedDict((e, None) for e in range(C)) for _ in range(N)]
    hits = misses = 0
    for t in range(T):
        for l in range(N):
            od = caches[l]
            need = [int(e) for e in trace[t, l]]
            for e in need:
                if e in od:
                    od.move_to_end(e)
                    hits += 1
            for e in need:
                if e not in od:
                    misses += 1
                    od.popitem(last=False)
                    od[e] = None
    return hits, misses


@pytest.mark.parametrize("E,K,C", [(8, 2, 2), (8, 2, 3), (16, 4, 6), (64, 8, 16)])
def test_cache_sim_without_prediction_is_textbook_lru(E, K, C):
    rng = np.random.default_rng(E * 100 + C)
    T, N = 40, 5
    # skewed expert popularity so that both hits and misses occur
    pop = rng.dirichlet(np.ones(E) * 0.3)
    trace = np.stack([[rng.choice(E, K, replace=False, p=pop) for _ in range(N)] for _ in range(T)])
    st = simulate_expert_cache(trace, None, E, C)
    h, m = _textbook_lru(trace, E, C)
    assert (st.hits, st.misses) == (h, m)
    assert st.loads == m and st.prefetch_issued == 0


def test_cache_sim_special_cases():
    rng = np.random.default_rng(5)
    E, K, N, T = 16, 4, 8, 30
    trace = np.stack([[rng.choice(E, K, replace=False) for _ in range(N)] for _ in range(T)])
    # every expert resident: all hits, nothing moves
    st = simulate_expert_cache(trace, trace, E, E)
    assert st.misses == 0 and st.hits == T * N * K and st.loads == 0
    # a perfect predictor: every predicted layer (l >= 2) hits
    pred = trace.copy()
    pred[:, :2] = -1
    st = simulate_expert_cache(trace, pred, E, K)
    assert st.per_layer_misses[2:] == [0] * (N - 2)
    assert st.pred_correct == st.pred_total == T * (N - 2) * K
    assert st.prefetch_used + st.prefetch_wasted <= st.prefetch_issued
    # C < K is rejected
    with pytest.raises(ValueError):
        simulate_expert_cache(trace, None, E, K - 1)


def test_cache_sim_worked_example():
    """Hand-worked trace: E=4, K=1, C=2, one layer."""
    trace = np.array([[[2]], [[0]], [[2]], [[1]], [[3]], [[1]]])
    # start: resident {0 (oldest), 1}
    # t0 need 2: miss, evict 0 -> {1, 2}; t1 need 0: miss, evict 1 -> {2, 0};
    # t2 need 2: hit -> {0, 2}; t3 need 1: miss, evict 0 -> {2, 1};
    # t4 need 3: miss, evict 2 -> {1, 3}; t5 need 1: hit
    st = simulate_expert_cache(trace, None, 4, 2)
    assert (st.hits, st.misses) == (2, 4)


def test_next_layer_schedule_worked_example():
    """Hand-worked trace for predictions applied to layer i+1 after layer i:
    E=4, K=1, C=2, two layers, both caches start as {0 (oldest), 1}."""
    slow = np.array([[[2], [3]], [[2], [0]], [[1], [3]]])
    pred = np.array([[[-1], [3]], [[-1], [1]], [[-1], [3]]])
    # t0: L0 needs 2: miss, evict 0 -> {1, 2}; predict L1 {3}: load, evict 0 -> {1, 3*}
    #     L1 needs 3: hit (prefetch used)
    # t1: L0 needs 2: hit; predict L1 {1}: resident, refreshed -> {3, 1}
    #     L1 needs 0: miss; victims exclude predicted 1 -> evict 3 -> {1, 0}
    # t2: L0 needs 1: hit; predict L1 {3}: load, evict 1 (older than 0) -> {0, 3*}
    #     L1 needs 3: hit (prefetch used)
    st = simulate_expert_cache(slow, pred, 4, 2, schedule="next")
    assert (st.hits, st.misses) == (4, 2)
    assert st.per_layer_misses == [1, 1]
    assert (st.prefetch_issued, st.prefetch_used, st.prefetch_wasted) == (2, 2, 0)
    assert (st.pred_correct, st.pred_total) == (2, 3)
    assert st.loads == 4


def test_next_layer_schedule_special_cases():
    rng = np.random.default_rng(9)
    E, K, N, T = 16, 4, 6, 25
    trace = np.stack([[rng.choice(E, K, replace=False) for _ in range(N)] for _ in range(T)])
    # a perfect predictor for layer i+1: every layer but the first hits, even with C = K
    pred = trace.copy()
    pred[:, 0] = -1
    st = simulate_expert_cache(trace, pred, E, K, schedule="next")
    assert st.per_layer_misses[1:] == [0] * (N - 1)
    assert st.prefetch_used == st.prefetch_issued
    # without predictions both schedules are plain LRU
    a = simulate_expert_cache(trace, None, E, 6, schedule="next")
    b = simulate_expert_cache(trace, None, E, 6, schedule="aot")
    assert a == b
    with pytest.raises(ValueError):
        simulate_expert_cache(trace, pred, E, K, schedule="later")


def test_fixed_experts_closed_form():
    """Fixed experts: a use is a hit exactly when the expert is one of the
    first C-K, and every other use is a copy."""
    rng = np.random.default_rng(11)
    E, K, N, T, C = 12, 3, 4, 30, 7
    trace = np.stack([[rng.choice(E, K, replace=False) for _ in range(N)] for _ in range(T)])
    st = simulate_fixed_experts(trace, E, C)
    low = trace < C - K
    assert st.hits == int(low.sum()) and st.misses == int((~low).sum()) == st.loads
    assert st.per_layer_misses == [int((~low[:, l]).sum()) for l in range(N)]
    assert st.prefetch_issued == st.pred_total == 0
    # C = K leaves nothing fixed; C = E keeps E-K experts, so only the top ids miss
    assert simulate_fixed_experts(trace, E, K).misses == trace.size
    st = simulate_fixed_experts(np.array([[[0, 9], [11, 10]]]), 12, 12)
    assert (st.hits, st.misses) == (2, 2)
    with pytest.raises(ValueError):
        simulate_fixed_experts(trace, E, K - 1)
