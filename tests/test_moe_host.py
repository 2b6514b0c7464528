"""Host-side parts of the mixture-of-experts path, no GPU needed: the C
library's expert-cache policies (replayed on routing traces) against the
oracle's cache simulations, and the packed expert layout."""
import numpy as np
import pytest

import synth
from oracle import simulate_expert_cache, simulate_fixed_experts
from paper_2502_02040_amd import binding as B

FIELDS = ("hits", "misses", "prefetch_issued", "prefetch_used", "prefetch_wasted", "loads", "pred_correct",
          "pred_total")


def _trace(rng, T, N, E, K, *, correlated=0.0):
    """Random routing trace: distinct experts per (token, layer); predictions
    for layers >= 2 that copy the true choice with probability `correlated`."""
    slow = np.stack([np.stack([rng.permutation(E)[:K] for _ in range(N)]) for _ in range(T)]).astype(np.int32)
    pred = np.full_like(slow, -1)
    for t in range(T):
        for l in range(2, N):
            p = rng.permutation(E)[:K]
            keep = rng.random(K) < correlated
            cand = [e for e in slow[t, l] if e not in p]
            for j in range(K):
                if keep[j] and cand:
                    p[j] = cand.pop()
            if len(set(p.tolist())) == K:
                pred[t, l] = p
    return slow, pred


def _oracle(slow, pred, E, C, prefetch):
    st = simulate_expert_cache(slow, pred, E, C, prefetch=prefetch)
    d = {f: getattr(st, f) for f in FIELDS}
    d["layer_misses"] = list(st.per_layer_misses)
    return d


def _lib(slow, pred, E, C, prefetch):
    T, N, K = slow.shape
    d = B.cache_replay(N, E, K, C, slow, pred, prefetch)
    return {f: d[f] for f in FIELDS + ("layer_misses",)}


@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("C", [3, 5, 8, 12])
@pytest.mark.parametrize("prefetch", [False, True])
def test_policy_replay_matches_cache_simulation(seed, C, prefetch):
    rng = np.random.default_rng(seed)
    E, K, N, T = 12, 3, 7, 40
    slow, pred = _trace(rng, T, N, E, K, correlated=0.5)
    assert _lib(slow, pred, E, C, prefetch) == _oracle(slow, pred, E, C, prefetch)


@pytest.mark.parametrize("seed", [0, 1])
@pytest.mark.parametrize("C", [3, 6, 12])
@pytest.mark.parametrize("policy", ["random_preload", "previous_layer"])
def test_next_layer_policies_replay_matches_cache_simulation(seed, C, policy):
    """Both comparison strategies that preload for layer i+1 after layer i."""
    rng = np.random.default_rng(seed + 10)
    E, K, N, T = 12, 3, 7, 40
    slow, pred = _trace(rng, T, N, E, K, correlated=0.6)
    pred[:, 1] = slow[:, 1]          # layer 1 gets a prediction too under this schedule
    st = simulate_expert_cache(slow, pred, E, C, schedule="next")
    want = {f: getattr(st, f) for f in FIELDS}
    want["layer_misses"] = list(st.per_layer_misses)
    assert _lib(slow, pred, E, C, policy) == want
    assert want["prefetch_issued"] > 0 or C == E


@pytest.mark.parametrize("C", [3, 5, 12])
def test_fixed_policy_replay_matches_simulation(C):
    rng = np.random.default_rng(C)
    E, K, N, T = 12, 3, 5, 30
    slow, pred = _trace(rng, T, N, E, K)
    st = simulate_fixed_experts(slow, E, C)
    got = _lib(slow, pred, E, C, "fixed")
    want = {f: getattr(st, f) for f in FIELDS}
    want["layer_misses"] = list(st.per_layer_misses)
    assert got == want


def test_replay_rejects_unknown_policy():
    slow = np.zeros((1, 2, 2), np.int32)
    slow[..., 1] = 1
    out = B.MoeCounters()
    assert B.lib().m2r2_expert_cache_replay(2, 4, 2, 2, 1, slow.ctypes.data, None, 5, B.ctypes.byref(out)) != 0


def test_policy_replay_without_predictions_matches():
    rng = np.random.default_rng(7)
    slow, _ = _trace(rng, 50, 5, 16, 4)
    assert _lib(slow, None, 16, 6, True) == _oracle(slow, None, 16, 6, True)


def test_all_resident_cache_never_misses():
    rng = np.random.default_rng(3)
    slow, pred = _trace(rng, 20, 6, 10, 3)
    d = B.cache_replay(6, 10, 3, 10, slow, pred, True)
    assert d["misses"] == 0 and d["hits"] == slow.size


def test_true_predictions_make_every_predicted_layer_hit():
    rng = np.random.default_rng(4)
    T, N, E, K = 30, 8, 16, 4
    slow, _ = _trace(rng, T, N, E, K)
    pred = np.full_like(slow, -1)
    pred[:, 2:] = slow[:, 2:]
    d = B.cache_replay(N, E, K, K, slow, pred, True)
    assert all(d["layer_misses"][l] == 0 for l in range(2, N))
    assert d["pred_correct"] == d["pred_total"] == T * (N - 2) * K


def test_replay_rejects_bad_arguments():
    slow = np.zeros((1, 2, 2), np.int32)
    slow[..., 1] = 1
    with pytest.raises(B.M2R2Error):
        B.cache_replay(2, 4, 2, 1, slow)          # slots < top_k
    bad = slow.copy()
    bad[0, 0, 0] = 9
    with pytest.raises(B.M2R2Error):
        B.cache_replay(2, 4, 2, 2, bad)          # expert id out of range


def _unpack(buf, rows, K, wdtype):
    """Row-major matrix read back from the tile-packed layout: 16-row tiles,
    K cut into MFMA steps of 32 (bf16) or 16 (f32) elements, each step a
    1 KB block where lane l holds row l % 16, elements [EPL*(l//16), +EPL)."""
    kstep = 32 if wdtype == "bf16" else 16
    epl = kstep // 4
    dt = np.uint16 if wdtype == "bf16" else np.float32
    a = np.frombuffer(buf, dtype=dt)
    tiles, S = (rows + 15) // 16, K // kstep
    a = a[:tiles * S * 64 * epl].reshape(tiles, S, 4, 16, epl)      # tile, step, lane group, row, elem
    out = a.transpose(0, 3, 1, 2, 4).reshape(tiles * 16, S * kstep)
    return out[:rows]


@pytest.mark.parametrize("wdtype", ["bf16", "f32"])
def test_pack_expert_layout(wdtype):
    cfg = synth.ModelConfig("pk", n_layers=1, d_model=64, n_heads=1, head_dim=64, ffn=0, vocab=8, rank=2,
                            wdtype=wdtype, n_experts=2, top_k=1, expert_ffn=96, seed=3)
    rng = np.random.default_rng(0)
    g, u = rng.standard_normal((2, 96, 64)).astype(np.float32)
    d = rng.standard_normal((64, 96)).astype(np.float32)
    eb = B.expert_bytes(cfg)
    esz = 2 if wdtype == "bf16" else 4
    assert eb == (2 * 96 * 64 + 64 * 96) * esz
    dst = np.zeros(eb, np.uint8)
    c = B.make_config(cfg)
    mats = [B._host_matrix(x, wdtype) for x in (g, u, d)]
    B._check(B.lib().m2r2_pack_expert(B.ctypes.byref(c), mats[0].ctypes.data, mats[1].ctypes.data,
                                      mats[2].ctypes.data, dst.ctypes.data), "pack")
    m = 96 * 64 * esz
    np.testing.assert_array_equal(_unpack(dst[:m].tobytes(), 96, 64, wdtype), mats[0])
    np.testing.assert_array_equal(_unpack(dst[m:2 * m].tobytes(), 96, 64, wdtype), mats[1])
    np.testing.assert_array_equal(_unpack(dst[2 * m:].tobytes(), 64, 96, wdtype), mats[2])
