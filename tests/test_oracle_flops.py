"""Pins of the oracle's FLOPs-optimised fast stream (Sec. 2.5) on the CPU.

  * the context selection is the prefix of a plain stable sort of the slow
    row's scores (ties to the lower position), checked by brute force;
  * a whole decode step matches the scalar-loop restatement of
    tests/bruteforce.py, which sorts the scores with Python's ``sorted``;
  * with every head kept, the context not limited, the full fast MLP and no
    low-rank head the step is the memory-bound form bit for bit;
  * pruned heads do not reach the fast row, and neither do cached values
    outside the selection, while a selected value does;
  * the low-rank head with identity/LM-head factors is the LM head.
"""
import math

import numpy as np
import pytest

import synth
from oracle import KVCache, Oracle, select_top, top_gap
from tests.bruteforce import BruteDecoder

MICRO_F = synth.CONFIGS["micro_flops"]
TINY_F = synth.CONFIGS["tiny_flops"]


def _weights(cfg, **kw):
    return synth.make_weights(cfg, threads=4, **kw)


# ---------------------------------------------------------------------------
# Context selection
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("n,k", [(1, 1), (5, 3), (40, 8), (40, 64), (100, 1), (64, 64), (65, 64)])
def test_select_top_is_the_prefix_of_a_stable_sort(n, k):
    rng = np.random.default_rng(n * 131 + k)
    for trial in range(20):
        # integer-valued scores: many exact ties, also at the boundary
        s = rng.integers(-4, 5, size=n).astype(np.float64)
        got = select_top(s, k)
        want = sorted(sorted(range(n), key=lambda t: (-s[t], t))[:k]) if n > k else list(range(n))
        assert got.tolist() == want
        if n > k:
            kept = set(want)
            # every kept score is at least every dropped one
            assert min(s[t] for t in kept) >= max(s[t] for t in range(n) if t not in kept)
            srt = sorted(s.tolist(), reverse=True)
            assert top_gap(s, k) == srt[k - 1] - srt[k]
        else:
            assert top_gap(s, k) == math.inf


def test_select_top_without_a_limit_keeps_everything():
    s = np.array([3.0, -1.0, 2.0])
    assert select_top(s, 0).tolist() == [0, 1, 2]
    assert select_top(np.zeros(0), 4).tolist() == []


# ---------------------------------------------------------------------------
# Whole step against the scalar-loop restatement
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("mode,tau", [("observe", 2.0), ("exit", -1.0), ("exit", 0.3), ("off", 0.0)])
@pytest.mark.parametrize("kvdtype", ["f32", "f64"])
def test_flops_decode_step_matches_bruteforce(mode, tau, kvdtype):
    """micro_flops: 2 heads of which the fast row keeps 1, top-3 context,
    adapter-only MLP, rank-3 head.  Positions 0..7 cover contexts below,
    at and above the limit."""
    cfg = MICRO_F.replace(kvdtype=kvdtype)
    w = _weights(cfg)
    orc = Oracle(cfg, w)
    bf = BruteDecoder(cfg, w)
    cache = KVCache(cfg, 16)
    tok = 5
    exits = 0
    for pos in range(8):
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
        # the pruned head never selects; the kept one selects once the context exceeds 3
        assert np.all(np.isinf(r.topk_gap[:, 1]))
        assert np.all(np.isinf(r.topk_gap[:, 0])) == (pos <= 3)
        exits += r.exit_boundary < cfg.n_layers
        tok = r.token
    if mode == "exit" and tau < 0:
        assert exits == 8


# ---------------------------------------------------------------------------
# Reduction to the memory-bound form
# ---------------------------------------------------------------------------

def test_all_heads_whole_context_full_mlp_is_the_memory_bound_step():
    """fast_heads = H and a context limit above every position, with the
    full fast MLP and the LM head: the FLOPs-form code path gives the
    memory-bound step exactly (same weights: the configs share their seed)."""
    base = synth.CONFIGS["tiny"].replace(kvdtype="f64")
    red = base.replace(name="tiny_red", fast_heads=base.n_heads, fast_topk=1000)
    assert red.is_flops and not red.fast_mlp_adapter and not red.head_rank
    w = _weights(base)
    a, b = Oracle(base, w), Oracle(red, w)
    ca, cb = KVCache(base, 24), KVCache(red, 24)
    tok = 11
    for pos in range(10):
        for mode, tau in (("observe", 0.5), ("exit", 0.999)):
            ra = a.decode_step(tok, pos, ca, gates=[1], tau=tau, mode=mode)
            rb = b.decode_step(tok, pos, cb, gates=[1], tau=tau, mode=mode)
            for x, y in ((ra.logits, rb.logits), (ra.h, rb.h), (ra.p, rb.p), (ra.signal, rb.signal)):
                np.testing.assert_allclose(y, x, rtol=1e-13, atol=1e-14)
            assert ra.exit_boundary == rb.exit_boundary
        tok = ra.token


def test_adapter_only_mlp_with_zero_factor_adds_nothing():
    """The fast MLP of the FLOPs form is the adapter alone: with A_m = 0 the
    fast state after the MLP equals the state after attention (checked via
    the layer function on one position)."""
    cfg = TINY_F.replace(kvdtype="f64")
    w = _weights(cfg)
    w0 = dict(w)
    for l in range(cfg.n_layers):
        w0[f"L{l}.A_m"] = np.zeros_like(w[f"L{l}.A_m"])
    orc = Oracle(cfg, w0)
    rng = np.random.default_rng(3)
    p = rng.standard_normal(cfg.d_model)
    h = rng.standard_normal(cfg.d_model)
    K = rng.standard_normal((12, cfg.n_heads, cfg.head_dim))
    V = rng.standard_normal((12, cfg.n_heads, cfg.head_dim))
    out, _ = orc._fast_layer_flops(0, p, h, 12, K, V)
    # attention part alone: rebuild with the MLP removed from the sum
    q, k, v = orc._qkv(0, p, 12, fast=True)
    qs, _, _ = orc._qkv(0, h, 12, fast=False)
    o = np.zeros_like(q)
    for j in range(cfg.fast_heads):
        s = K[:, j] @ qs[j] / math.sqrt(cfg.head_dim)
        sel = select_top(s, cfg.fast_topk)
        sc = np.concatenate([K[sel, j] @ q[j], [k[j] @ q[j]]]) / math.sqrt(cfg.head_dim)
        e = np.exp(sc - sc.max())
        o[j] = (e / e.sum()) @ np.concatenate([V[sel, j], v[j][None]])
    p1 = p + orc._attn_out(0, o, fast=True)
    np.testing.assert_allclose(out, p1, rtol=1e-13, atol=1e-14)


# ---------------------------------------------------------------------------
# What reaches the fast row
# ---------------------------------------------------------------------------

def _first_layer_fast_state(cfg, w, K=None, V=None, pos=12):
    """Fast state after layer 0 (mode off), with layer 0's cache positions
    [0, pos) set to K, V."""
    orc = Oracle(cfg, w)
    cache = KVCache(cfg, pos + 4)
    rng = np.random.default_rng(7)
    for l in range(cfg.n_layers):
        Kl = rng.standard_normal((pos, cfg.n_heads, cfg.head_dim))
        Vl = rng.standard_normal((pos, cfg.n_heads, cfg.head_dim))
        if l == 0 and K is not None:
            Kl, Vl = K, V
        cache.load(l, Kl, Vl)
    r = orc.decode_step(9, pos, cache, mode="off")
    return r.fast_states[0], r


def test_pruned_heads_do_not_reach_the_fast_row():
    cfg = TINY_F.replace(kvdtype="f64")
    w = _weights(cfg)
    hd, nh = cfg.head_dim, cfg.fast_heads
    base, rb = _first_layer_fast_state(cfg, w)
    rng = np.random.default_rng(5)
    # rows of B_q, B_k, B_v and columns of A_o of a pruned head
    w2 = dict(w)
    pr = slice(nh * hd, (nh + 1) * hd)
    for nm in ("B_q", "B_k", "B_v"):
        a = w[f"L0.{nm}"].copy()
        a[pr] += rng.standard_normal(a[pr].shape)
        w2[f"L0.{nm}"] = a
    a = w["L0.A_o"].copy()
    a[:, pr] += rng.standard_normal(a[:, pr].shape)
    w2["L0.A_o"] = a
    got, rg = _first_layer_fast_state(cfg, w2)
    np.testing.assert_array_equal(got, base)
    np.testing.assert_array_equal(rg.h, rb.h)
    # the same perturbation on a kept head moves the fast row
    w3 = dict(w)
    kp = slice(0, hd)
    a = w["L0.B_q"].copy()
    a[kp] += rng.standard_normal(a[kp].shape)
    w3["L0.B_q"] = a
    moved, _ = _first_layer_fast_state(cfg, w3)
    assert np.max(np.abs(moved - base)) > 1e-6


def test_values_outside_the_selection_do_not_reach_the_fast_row():
    cfg = TINY_F.replace(kvdtype="f64")
    w = _weights(cfg)
    rng = np.random.default_rng(9)
    pos = 30
    K = rng.standard_normal((pos, cfg.n_heads, cfg.head_dim))
    V = rng.standard_normal((pos, cfg.n_heads, cfg.head_dim))
    base, r = _first_layer_fast_state(cfg, w, K, V, pos)
    # the selection of every kept head at layer 0, from the slow query
    orc = Oracle(cfg, w)
    qs, _, _ = orc._qkv(0, w["embed"][9].astype(np.float64), pos, fast=False)
    chosen = set()
    for j in range(cfg.fast_heads):
        chosen |= set(select_top(K[:, j] @ qs[j] / math.sqrt(cfg.head_dim), cfg.fast_topk).tolist())
    assert len(chosen) < pos
    out = [t for t in range(pos) if t not in chosen]
    V2 = V.copy()
    V2[out, :cfg.fast_heads] += 10.0
    same, _ = _first_layer_fast_state(cfg, w, K, V2, pos)
    np.testing.assert_array_equal(same, base)
    V3 = V.copy()
    V3[sorted(chosen)[0], :cfg.fast_heads] += 10.0
    moved, _ = _first_layer_fast_state(cfg, w, K, V3, pos)
    assert np.max(np.abs(moved - base)) > 1e-6


def test_low_rank_head_with_identity_factors_is_the_lm_head():
    cfg = TINY_F.replace(kvdtype="f64", head_rank=TINY_F.d_model)
    w = _weights(TINY_F)
    w = dict(w)
    w["head_A"] = np.eye(cfg.d_model)
    w["head_B"] = w["lm_head"].astype(np.float64)
    orc = Oracle(cfg, w)
    x = np.random.default_rng(2).standard_normal(cfg.d_model)
    np.testing.assert_allclose(orc.fast_head_logits(x), orc.head_logits(x), rtol=1e-12, atol=1e-13)


def test_fast_only_draft_is_refused():
    cfg = MICRO_F
    orc = Oracle(cfg, _weights(cfg))
    with pytest.raises(ValueError):
        orc.draft(1, 0, KVCache(cfg, 8), 1, 2)
