"""Pins of the oracle's latent-attention exit router (Sec. 2.3.1, ARLA; Fig.
4a), with no GPU: closed forms of the attention (one state; keys that carry no
information), the same computation composed from torch's library routines
(rms_norm, linear, scaled-dot-product attention, sigmoid), and which fast
states enter each gate's interval inside the decode step."""
import dataclasses

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import synth
from oracle import ARLA_DIM, KVCache, Oracle, arla_score

EPS = 1e-5
CFG = synth.ModelConfig("arla_pin", n_layers=7, d_model=96, n_heads=2, head_dim=48, ffn=160, vocab=64, rank=4,
                        wdtype="f32", kvdtype="f64", seed=31)


def _unit(x):
    return x / np.sqrt(np.mean(x * x) + EPS)


def _sig(z):
    return 1.0 / (1.0 + np.exp(-z))


def _rand(rng, d, n):
    wq, wk, wv = (rng.standard_normal((ARLA_DIM, d)) * 0.2 for _ in range(3))
    w = rng.standard_normal(ARLA_DIM) / 8
    states = [rng.standard_normal(d) * (1 + i) for i in range(n)]
    return wq, wk, wv, w, states


def test_single_state_is_the_readout_of_its_value():
    """One state: the softmax weight is 1, so the score is the readout of v."""
    rng = np.random.default_rng(0)
    wq, wk, wv, w, states = _rand(rng, 40, 1)
    got = arla_score(wq, wk, wv, w, 0.3, states, EPS)
    assert got == pytest.approx(_sig(w @ (wv @ _unit(states[0])) + 0.3), rel=1e-12)


def test_keys_without_information_average_the_values():
    """All keys equal (W_K = 0): uniform attention over the interval."""
    rng = np.random.default_rng(1)
    wq, _, wv, w, states = _rand(rng, 40, 5)
    got = arla_score(wq, np.zeros_like(wq), wv, w, -0.2, states, EPS)
    mean_v = np.mean([wv @ _unit(x) for x in states], axis=0)
    assert got == pytest.approx(_sig(w @ mean_v - 0.2), rel=1e-12)


@pytest.mark.parametrize("n", [1, 3, 8])
def test_matches_library_composition(n):
    """rms_norm -> three linear maps -> scaled-dot-product attention of the
    last state's query (scale 1/sqrt(64), torch's default) -> linear -> sigmoid."""
    rng = np.random.default_rng(10 + n)
    wq, wk, wv, w, states = _rand(rng, 72, n)
    T = lambda a: torch.tensor(np.asarray(a, np.float64))
    X = F.rms_norm(T(np.stack(states)), (72,), eps=EPS)
    q = F.linear(X[-1:], T(wq))
    K, V = F.linear(X, T(wk)), F.linear(X, T(wv))
    o = F.scaled_dot_product_attention(q[None], K[None], V[None])[0, 0]
    ref = torch.sigmoid(F.linear(o, T(w[None]), T([0.05]))).item()
    assert arla_score(wq, wk, wv, w, 0.05, states, EPS) == pytest.approx(ref, rel=1e-10)


def test_score_does_not_depend_on_the_scale_of_the_states():
    rng = np.random.default_rng(4)
    wq, wk, wv, w, states = _rand(rng, 64, 4)
    a = arla_score(wq, wk, wv, w, 0.0, states, 0.0)
    b = arla_score(wq, wk, wv, w, 0.0, [3.7 * x for x in states], 0.0)
    assert a == pytest.approx(b, rel=1e-12)


def _prompt():
    return [int(t) for t in synth.prompt_ids(CFG, 6)]


def _step(arla, gates, mode="observe", tau=2.0, cfg=CFG):
    w = synth.make_weights(cfg, threads=2)
    orc = Oracle(cfg, w)
    cache = KVCache(cfg, 16)
    ids = _prompt()
    orc.slow_chunk(ids[:-1], 0, cache)
    return orc.decode_step(ids[-1], len(ids) - 1, cache, gates=gates, tau=tau, mode=mode, arla=arla)


def _slow_state_at(b):
    """The slow residual entering layer b, from a model cut after layer b-1
    (synth draws every tensor from its own name, so the first b layers are
    the same tensors)."""
    cut = dataclasses.replace(CFG, n_layers=b)
    return _step(None, [], mode="off", cfg=cut).h


def _arla_f64():
    a = {k: np.asarray(v, np.float64) for k, v in synth.arla_weights(CFG).items()}
    a["b_out"][:] = np.arange(CFG.n_layers) * 0.1
    return a


def test_decode_step_interval_bookkeeping():
    """Gates 2 and 5 of 7 layers, keys without information (uniform
    attention): the signal at gate 2 averages the values of the embedding
    (where p starts) and the fast states after layers 0, 1; at gate 5 those
    of the slow state entering layer 2 (where p restarts) and the fast states
    after layers 2, 3, 4.  Other layers keep the cosine signal."""
    a = _arla_f64()
    a["wk"][:] = 0.0
    plain = _step(None, [2, 5])
    r = _step(a, [2, 5])
    fs = r.fast_states
    emb = synth.make_weights(CFG, names=["embed"])["embed"][_prompt()[-1]].astype(np.float64)
    for b, states in ((2, [emb, fs[0], fs[1]]), (5, [_slow_state_at(2), fs[2], fs[3], fs[4]])):
        mean_v = np.mean([a["wv"][b] @ _unit(x) for x in states], axis=0)
        assert r.signal[b - 1] == pytest.approx(_sig(a["w_out"][b] @ mean_v + a["b_out"][b]), rel=1e-10)
    others = [l for l in range(CFG.n_layers) if l not in (1, 4)]
    np.testing.assert_allclose(r.signal[others], plain.signal[others], rtol=1e-12)
    # observe mode restarts p at every gate whatever the signal: same states, same logits
    np.testing.assert_allclose(r.logits, plain.logits, rtol=1e-12)


def test_decode_step_interval_matches_arla_score():
    """With informative keys, the signal at gates 1, 3 and 6 is arla_score
    over the interval assembled outside the step: the restart state (the
    embedding, then the slow state entering the previous gate), then the fast
    states after the interval's layers."""
    a = _arla_f64()
    r = _step(a, [1, 3, 6])
    fs = r.fast_states
    emb = synth.make_weights(CFG, names=["embed"])["embed"][_prompt()[-1]].astype(np.float64)
    cases = ((1, [emb, fs[0]]), (3, [_slow_state_at(1), fs[1], fs[2]]),
             (6, [_slow_state_at(3), fs[3], fs[4], fs[5]]))
    for b, states in cases:
        want = arla_score(a["wq"][b], a["wk"][b], a["wv"][b], a["w_out"][b], float(a["b_out"][b]), states, EPS)
        assert r.signal[b - 1] == pytest.approx(want, rel=1e-12)
        # the restart state matters: the interval without it scores differently
        assert abs(arla_score(a["wq"][b], a["wk"][b], a["wv"][b], a["w_out"][b], float(a["b_out"][b]),
                              states[1:], EPS) - want) > 1e-6


def test_decode_step_exit_follows_the_router():
    """EXIT mode: the step stops at the first gate whose router score reaches tau."""
    a = {k: np.asarray(v, np.float64) for k, v in synth.arla_weights(CFG).items()}
    a["b_out"][:] = -50.0
    a["b_out"][4] = 50.0          # only gate 4 can fire
    r = _step(a, [2, 4, 6], mode="exit", tau=0.5)
    assert r.exit_boundary == 4
    assert r.signal[3] > 0.99 and r.signal[1] < 0.01
    off = _step(a, [2, 4, 6], mode="off")
    assert off.exit_boundary == CFG.n_layers
