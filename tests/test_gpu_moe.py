"""GPU parity of the mixture-of-experts decode step (Sec. 2.3.3) through the
C ABI against the CPU oracle: the slow row's routed experts, the fast row's
adapter-only MLP and its expert predictions for layers 2i+2 and 2i+3 (or,
under the previous-layer strategy of Sec. 3.3, layer i+1's router on the slow
row), the hidden states, logits and cache; and the HBM expert cache's
counters, under each of the five placement strategies, against the oracle's
cache simulations replayed on the GPU's own routing trace.

Sizes: a bfloat16 model with 6 layers, d 256, 2 heads x 128, 16 experts of
width 96, top-4 (caches of 5 and 16 slots), a float32 model with 5 layers,
d 128, 2 heads x 64, 8 experts of width 64, top-2 (both on the tile GEMVs),
and a bfloat16 model with 4 layers, d 512, 4 heads x 128, rank 8 (rows of
whole 1 KB pieces: the row-per-wave q/k/v, o and head kernels and the
short-chain attention)."""
import numpy as np
import pytest
import torch

import synth
from oracle import KVCache, Oracle, simulate_expert_cache, simulate_fixed_experts
from paper_2502_02040_amd import Model, PagedKV
from tests.gpu_harness import Tally, shuffled_table, tol_of, track

pytestmark = pytest.mark.gpu

FIELDS = ("hits", "misses", "prefetch_issued", "prefetch_used", "prefetch_wasted", "loads", "pred_correct",
          "pred_total")


class MoePair:
    def __init__(self, name, *, slots, max_ctx=64, policy="ahead_of_time", weights=None):
        cfg = synth.CONFIGS[name]
        self.cfg = cfg
        self.tol = tol_of(cfg)
        self.w = weights if weights is not None else synth.make_weights(cfg)
        self.model = track(Model(cfg, self.w, max_batch=1, max_chunk=16, max_ctx=max_ctx, expert_slots=slots))
        self.policy = policy
        if policy == "random_preload":
            self.table = synth.preload_table(cfg, 64)
            self.model.moe_set_preload_table(self.table)
        self.model.moe_set_policy(policy)
        self.kv = PagedKV(cfg, 1, max_ctx, block_size=16, block_table=shuffled_table(1, max_ctx, 16, 5))
        self.orc = Oracle(cfg, self.w)
        self.cache = KVCache(cfg, max_ctx)
        self.dev = torch.device("cuda")
        N, K = cfg.n_layers, cfg.top_k
        self.slow = torch.zeros(N * K, dtype=torch.int32, device=self.dev)
        self.pred = torch.zeros(N * K, dtype=torch.int32, device=self.dev)

    def prefill(self, prompt, t: Tally):
        """Slow-only decode steps on the GPU, the chunked slow forward in the oracle."""
        ref = self.orc.slow_chunk(list(prompt), 0, self.cache)
        pos = torch.zeros(1, dtype=torch.int32, device=self.dev)
        nxt = torch.zeros(1, dtype=torch.int32, device=self.dev)
        for i, tok in enumerate(prompt):
            tk = torch.tensor([tok], dtype=torch.int32, device=self.dev)
            self.model.decode_step(tk, pos, self.kv.desc(), dual=False, next_token=nxt, advance=True)
            torch.cuda.synchronize()
            t.token(int(nxt.item()), ref[i], self.tol, f"prefill row {i}")
        for l in range(self.cfg.n_layers):
            K, V = self.kv.read(0, l, 0, len(prompt))
            t.rel(K, self.cache.K[l][:len(prompt)], self.tol, f"prefill K layer {l}")
            t.rel(V, self.cache.V[l][:len(prompt)], self.tol, f"prefill V layer {l}")
        return int(nxt.item())

    def run(self, n_steps, *, mode="observe", gates=(), tau=2.0, prompt_len=12, check=True):
        cfg, N, K = self.cfg, self.cfg.n_layers, self.cfg.top_k
        t = Tally()
        prompt = list(synth.prompt_ids(cfg, prompt_len))
        tok = self.prefill(prompt, t)
        self.model.moe_reset()
        dev = self.dev
        tok_d = torch.tensor([tok], dtype=torch.int32, device=dev)
        pos_d = torch.tensor([prompt_len], dtype=torch.int32, device=dev)
        nxt = torch.zeros(1, dtype=torch.int32, device=dev)
        exb = torch.zeros(1, dtype=torch.int32, device=dev)
        sig = torch.zeros(N, dtype=torch.float32, device=dev)
        logits = torch.zeros(cfg.vocab, dtype=torch.float32, device=dev)
        h_out = torch.zeros(cfg.d_model, dtype=torch.float32, device=dev)
        p_out = torch.zeros(cfg.d_model, dtype=torch.float32, device=dev)
        slow_tr, pred_tr, outs = [], [], []
        for step in range(n_steps):
            pos = prompt_len + step
            self.model.decode_step(tok_d, pos_d, self.kv.desc(), gates=gates, tau=tau, mode=mode, next_token=nxt,
                                   exit_boundary=exb, signal=sig, logits=logits, h_out=h_out, p_out=p_out,
                                   advance=True, slow_experts=self.slow, pred_experts=self.pred)
            torch.cuda.synchronize()
            gs = self.slow.cpu().numpy().reshape(N, K)
            gp = self.pred.cpu().numpy().reshape(N, K)
            slow_tr.append(gs)
            pred_tr.append(gp)
            outs.append(logits.cpu().numpy().copy())
            if not check:
                tok_d.copy_(nxt)
                continue
            r = self.orc.decode_step(int(tok_d.item()), pos, self.cache, gates=gates, tau=tau, mode=mode)
            # expert choices, in order, where the router margins decide them
            ran = r.slow_experts.shape[0]
            diverged = False
            for l in range(ran):
                decided = t.experts(gs[l], r.slow_experts[l], r.router_logits[l], K, self.tol,
                                    f"step {step} layer {l}: slow experts")
                if not decided and set(gs[l]) != set(r.slow_experts[l]):
                    diverged = True   # a near tie went the other way: the two sides now differ
                    break
            if diverged:
                t.skipped += 1
                break
            assert np.all(gs[ran:] == -1), f"step {step}: layers after the exit report experts"
            prev = self.policy == "previous_layer"
            ref_pred = r.prev_pred_experts if prev else r.pred_experts
            ref_logits = r.prev_pred_logits if prev else r.pred_logits
            for l in range(N):
                if ref_pred[l][0] < 0:
                    assert np.all(gp[l] == -1), f"step {step} layer {l}: unexpected prediction"
                else:
                    t.experts(gp[l], ref_pred[l], ref_logits[l], K, self.tol, f"step {step} layer {l}: predicted")
            if mode == "off" or all(abs(r.signal[b - 1] - tau) > self.tol for b in gates):
                t.equal(int(exb.item()), r.exit_boundary, f"step {step}: exit boundary")
            else:
                assert mode == "observe", "an EXIT-mode test must pick a threshold the signals decide"
                t.skipped += 1
            t.rel(logits.cpu().numpy(), r.logits, self.tol, f"step {step} logits")
            t.rel(h_out.cpu().numpy(), r.h, self.tol, f"step {step} h")
            t.rel(p_out.cpu().numpy(), r.p, self.tol, f"step {step} p")
            got_sig = sig.cpu().numpy()
            lr = [l for l in range(N) if not (mode == "exit" and r.exit_boundary < N and l >= r.exit_boundary)]
            t.close(got_sig[lr], r.signal[lr], self.tol, f"step {step} signal")
            t.token(int(nxt.item()), r.logits, self.tol, f"step {step} token")
            for l in range(N):
                K_, V_ = self.kv.read(0, l, pos, pos + 1)
                t.rel(K_, self.cache.K[l][pos:pos + 1], self.tol, f"step {step} K layer {l}")
                t.rel(V_, self.cache.V[l][pos:pos + 1], self.tol, f"step {step} V layer {l}")
            t.steps += 1
            tok_d.copy_(nxt)
        return t, slow_tr, pred_tr, outs


@pytest.mark.parametrize("name,slots", [("small_moe", 5), ("small_moe", 16), ("small_moe_f32", 3),
                                        ("small_moe_rw", 6)])
def test_moe_dual_step_observe(name, slots):
    cfg = synth.CONFIGS[name]
    p = MoePair(name, slots=slots)
    t, *_ = p.run(10, mode="observe", gates=list(range(1, cfg.n_layers)), tau=0.9)
    assert t.steps >= 6 and t.compared >= 6 * t.steps


@pytest.mark.parametrize("name", ["small_moe_f32", "small_moe_rw"])
@pytest.mark.parametrize("resident", [False, True])
def test_moe_exit_mode_fills_skipped_layers(name, resident):
    """EXIT mode: the layers after the exit run no MLP and still fill their
    cache entries.  With every expert resident the host never sees the exit
    (the token is enqueued whole): the expert kernels skip themselves and the
    down projection's launch adds the slow row's statistics instead."""
    cfg = synth.CONFIGS[name]
    p = MoePair(name, slots=cfg.n_experts if resident else 4, policy="on_demand" if resident else "ahead_of_time")
    t, slow_tr, _, _ = p.run(6, mode="exit", gates=[2], tau=-1.0)
    assert t.steps == 6 and t.compared >= 6
    assert all(np.all(s[2:] == -1) for s in slow_tr)
    if resident:
        st = p.model.moe_stats()
        assert st["hits"] == 6 * 2 * cfg.top_k and st["misses"] == 0 and st["host_wait_ns"] == 0


@pytest.mark.parametrize("name", ["small_moe", "small_moe_f32", "small_moe_rw"])
def test_resident_cache_enqueues_whole_tokens(name):
    """As many slots as experts under the LRU policy: every expert is taken
    from its slot on the device and the host never waits for routing.  The
    outputs match the oracle, and the hits the expert kernels count equal the
    routed layers times top_k."""
    cfg = synth.CONFIGS[name]
    p = MoePair(name, slots=cfg.n_experts, policy="on_demand")
    t, slow_tr, *_ = p.run(8, mode="observe", gates=list(range(1, cfg.n_layers)), tau=0.9)
    assert t.steps >= 6 and t.compared >= 6 * t.steps
    st = p.model.moe_stats()
    routed = sum(int(np.sum(s[:, 0] >= 0)) for s in slow_tr)
    assert routed == len(slow_tr) * cfg.n_layers
    assert st["hits"] == routed * cfg.top_k
    assert st["misses"] == 0 and st["loads"] == 0 and st["host_wait_ns"] == 0


def test_moe_previous_layer_predictions_match_oracle():
    """Under the previous-layer strategy the step reports, for layer l+1, the
    top-k of layer l+1's router on the slow row entering layer l's MLP."""
    cfg = synth.CONFIGS["small_moe"]
    p = MoePair("small_moe", slots=5, policy="previous_layer")
    t, *_ = p.run(8, mode="observe", gates=list(range(1, cfg.n_layers)), tau=0.9)
    assert t.steps >= 6 and t.compared >= 6 * t.steps


POLICY_NAMES = ["ahead_of_time", "on_demand", "fixed", "random_preload", "previous_layer"]


@pytest.mark.parametrize("policy", POLICY_NAMES)
def test_expert_cache_counters_match_simulation(policy):
    """The runtime's hits, misses, prefetches and prediction accuracy equal
    the oracle's cache simulation replayed on the GPU's own routing trace."""
    p = MoePair("small_moe", slots=5, policy=policy)
    T = 16
    _, slow_tr, pred_tr, _ = p.run(T, check=False)
    slow = np.stack(slow_tr)
    E = p.cfg.n_experts
    if policy == "fixed":
        st = simulate_fixed_experts(slow, E, 5)
    elif policy == "random_preload":
        st = simulate_expert_cache(slow, p.table[:T], E, 5, schedule="next")
    elif policy == "previous_layer":
        st = simulate_expert_cache(slow, np.stack(pred_tr), E, 5, schedule="next")
    else:
        st = simulate_expert_cache(slow, np.stack(pred_tr), E, 5, prefetch=policy == "ahead_of_time")
    got = p.model.moe_stats()
    for f in FIELDS:
        assert got[f] == getattr(st, f), f"{f}: {got[f]} != {getattr(st, f)}"
    assert got["layer_misses"] == list(st.per_layer_misses)
    assert got["h2d_bytes"] == got["loads"] * p.model.expert_bytes
    if policy in ("ahead_of_time", "random_preload", "previous_layer"):
        assert got["prefetch_issued"] > 0


@pytest.mark.parametrize("policy", ["ahead_of_time", "fixed", "random_preload", "previous_layer"])
def test_small_cache_gives_the_same_outputs_as_all_resident(policy):
    """Copies into a 4-slot cache deliver the same expert weights as an
    all-resident cache under every placement strategy: logits and routing are
    bitwise equal (the predictions too, where both runs make the same kind)."""
    w = synth.make_weights(synth.CONFIGS["small_moe"])
    a = MoePair("small_moe", slots=4, weights=w, policy=policy)
    _, sa, pa, oa = a.run(8, check=False)
    b = MoePair("small_moe", slots=16, weights=w, policy="ahead_of_time" if policy != "previous_layer" else policy)
    _, sb, pb, ob = b.run(8, check=False)
    assert a.model.moe_stats()["misses"] > 0 and b.model.moe_stats()["misses"] == 0
    for i in range(8):
        np.testing.assert_array_equal(sa[i], sb[i])
        if policy in ("ahead_of_time", "previous_layer"):
            np.testing.assert_array_equal(pa[i], pb[i])
        np.testing.assert_array_equal(oa[i], ob[i])


def test_external_prefetch_makes_experts_resident():
    p = MoePair("small_moe", slots=4, policy="on_demand")
    p.model.moe_reset()
    p.model.prefetch_experts(3, [9, 10, 11])
    torch.cuda.synchronize()
    st = p.model.moe_stats()
    assert st["prefetch_issued"] == 3 and st["loads"] == 3
    p.model.prefetch_experts(3, [9, 10, 11], priority=True)   # already resident: refreshed, no copy
    assert p.model.moe_stats()["loads"] == 3


@pytest.mark.parametrize("name", ["small_moe", "small_moe_rw"])
@pytest.mark.parametrize("policy", ["on_demand", "ahead_of_time", "fixed", "previous_layer"])
def test_device_slot_table_matches_host_slots(name, policy, monkeypatch):
    """Expert kernels that read their slots from the device table (launched
    before the host has seen the routing) give the same routing, predictions
    and cache counters, and the same logits, as kernels launched by the host
    with its own slots after every routing decision.  (The logits are equal
    to float rounding: the row-per-wave kernels add their row statistics
    with atomics, whose order varies from run to run.)"""
    w = synth.make_weights(synth.CONFIGS[name])
    monkeypatch.setenv("M2R2_MOE_DEVICE_SLOTS", "0")
    a = MoePair(name, slots=5, weights=w, policy=policy)
    _, sa, pa, oa = a.run(10, check=False)
    monkeypatch.delenv("M2R2_MOE_DEVICE_SLOTS")
    b = MoePair(name, slots=5, weights=w, policy=policy)
    _, sb, pb, ob = b.run(10, check=False)
    for i in range(10):
        np.testing.assert_array_equal(sa[i], sb[i])
        np.testing.assert_array_equal(pa[i], pb[i])
        np.testing.assert_allclose(oa[i], ob[i], rtol=1e-4, atol=1e-4 * np.max(np.abs(oa[i])))
    ga, gb = a.model.moe_stats(), b.model.moe_stats()
    for f in FIELDS + ("h2d_bytes", "layer_misses"):
        assert ga[f] == gb[f], f
