"""Pins of the oracle's latent-attention exit router (Sec. 2.3.1, ARLA; Fig.
4a), with no GPU: closed forms of the attention (one state; keys that carry no
information), the same computation composed from torch's library routines
(rms_norm, linear, scaled-dot-product attention, sigmoid), and which fast
states enter each gate's interval inside the decode step."""
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


def _step(arla, gates, mode="observe", tau=2.0):
    w = synth.make_weights(CFG, threads=2)
    orc = Oracle(CFG, w)
    cache = KVCache(CFG, 16)
    ids = list(synth.prompt_ids(CFG, 6))
    orc.slow_chunk(ids[:-1], 0, cache)
    return orc.decode_step(ids[-1], len(ids) - 1, cache, gates=gates, tau=tau, mode=mode, arla=arla)


def test_decode_step_uses_the_states_since_the_previous_gate():
    """Gates 2 and 5 of 7 layers, keys without information: the signal at
    gate 2 averages the values of the fast states after layers 0, 1; at gate
    5 those after layers 2, 3, 4.  Other layers keep the cosine signal."""
    a = synth.arla_weights(CFG)
    a = {k: np.asarray(v, np.float64) for k, v in a.items()}
    a["wk"][:] = 0.0
    a["b_out"][:] = np.arange(CFG.n_layers) * 0.1
    plain = _step(None, [2, 5])
    r = _step(a, [2, 5])
    fs = r.fast_states
    for b, lay in ((2, [0, 1]), (5, [2, 3, 4])):
        mean_v = np.mean([a["wv"][b] @ _unit(fs[l]) for l in lay], axis=0)
        assert r.signal[b - 1] == pytest.approx(_sig(a["w_out"][b] @ mean_v + a["b_out"][b]), rel=1e-10)
    others = [l for l in range(CFG.n_layers) if l not in (1, 4)]
    np.testing.assert_allclose(r.signal[others], plain.signal[others], rtol=1e-12)
    # observe mode restarts p at every gate whatever the signal: same states, same logits
    np.testing.assert_allclose(r.logits, plain.logits, rtol=1e-12)


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
