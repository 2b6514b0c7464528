"""Deterministic simulation of the per-layer HBM expert cache with
least-recently-used eviction and ahead-of-time (AoT) prefetch.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Policy (Sec. 2.3.3 and Appendix B of the paper: LRU experts are replaced by
speculated ones, predictions for layers 2i+2 and 2i+3 are issued while layer
i computes, and experts still missing when a layer's MLP starts are loaded on
demand).  The paper leaves the bookkeeping open; the reading used here:

  1. every layer owns ``C`` slots; the cache starts warm with experts
     0..C-1 resident, expert 0 the least recently used;
  2. a global counter stamps every use and every insertion;
  3. when layer i runs with needed set S (router order): first every needed
     expert that is resident is refreshed (in S order), then each missing one
     is loaded on demand (in S order) into the slot with the smallest stamp
     among experts that are neither needed now nor predicted for this layer
     earlier in the same token (if every resident expert is one of those, the
     smallest stamp among those not needed now);
  4. after layer i, if predictions are enabled, for each predicted layer
     L in (2i+2, 2i+3) below N and each predicted expert (in order): a
     resident one is refreshed, a missing one is inserted into the slot with
     the smallest stamp among experts not predicted for L in this token;
  5. "hit" is logical: resident (or in flight) when the layer's MLP starts.

The baselines the paper compares against (Sec. 3.3) reuse these rules:
  * least-recently-used alone: no predictions;
  * random preload and speculation from the previous layer's residual state:
    the predictions for layer i+1 (random experts, or the top-k of layer
    i+1's router applied to the slow row that enters layer i's MLP) are
    applied after layer i (``schedule="next"``), instead of the fast row's
    predictions for 2i+2 and 2i+3 (``schedule="aot"``);
  * experts fixed in HBM without replacement (``simulate_fixed_experts``):
    the paper does not say which experts are fixed or where a missing one
    goes; the reading here keeps the first C-K experts of every layer
    resident for good and copies every other needed expert, at every use,
    into one of K staging slots, so that the HBM budget is the same C slots.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Sequence

import numpy as np


@dataclasses.dataclass
class CacheStats:
    hits: int = 0
    misses: int = 0
    prefetch_issued: int = 0
    prefetch_used: int = 0
    prefetch_wasted: int = 0      # prefetched experts evicted before any use
    loads: int = 0                # every host-to-device expert copy (misses + prefetches)
    pred_correct: int = 0         # |P_l ∩ S_l| summed over predicted layers
    pred_total: int = 0           # |P_l| summed over predicted layers
    per_layer_misses: Optional[List[int]] = None

    @property
    def hit_rate(self) -> float:
        n = self.hits + self.misses
        return self.hits / n if n else 1.0


class _Layer:
    def __init__(self, C: int, clock: List[int]):
        self.stamp: Dict[int, int] = {e: e - C for e in range(C)}   # expert -> last stamp
        self.prefetched: Dict[int, bool] = {}
        self.C = C
        self.clock = clock

    def tick(self) -> int:
        self.clock[0] += 1
        return self.clock[0]

    def victim(self, protect, fallback) -> int:
        cands = [e for e in self.stamp if e not in protect] or [e for e in self.stamp if e not in fallback]
        return min(cands, key=lambda e: self.stamp[e])

    def insert(self, e: int, protect, stats: CacheStats, fallback=()) -> None:
        if len(self.stamp) >= self.C:
            v = self.victim(protect, fallback)
            if self.prefetched.pop(v, False):
                stats.prefetch_wasted += 1
            del self.stamp[v]
        self.stamp[e] = self.tick()
        stats.loads += 1


def simulate_expert_cache(slow: np.ndarray, pred: Optional[np.ndarray], n_experts: int, slots: int,
                          *, prefetch: bool = True, schedule: str = "aot") -> CacheStats:
    """Run the policy over a trace.

    ``slow[t, l]``: experts used by layer l at token t (router order).
    ``pred[t, l]``: experts predicted for layer l at token t (row of -1 when
    layer l has no prediction), or None.  With ``schedule="aot"`` the
    predictions for layers L=2i+2, 2i+3 are applied right after layer i of
    the same token; with ``schedule="next"`` those for layer L=i+1.
    """
    T, N, K = slow.shape
    if slots < K or slots > n_experts:
        raise ValueError("need top_k <= slots <= n_experts")
    if schedule not in ("aot", "next"):
        raise ValueError(f"schedule {schedule!r}")
    clock = [0]
    layers = [_Layer(slots, clock) for _ in range(N)]
    st = CacheStats(per_layer_misses=[0] * N)
    use_pred = prefetch and pred is not None
    for t in range(T):
        predicted: Dict[int, List[int]] = {}
        for i in range(N):
            L = layers[i]
            need = [int(e) for e in slow[t, i]]
            protect = set(need) | set(predicted.get(i, ()))
            if i in predicted:
                st.pred_total += len(predicted[i])
                st.pred_correct += len(set(predicted[i]) & set(need))
            for e in need:
                if e in L.stamp:
                    st.hits += 1
                    if L.prefetched.pop(e, False):
                        st.prefetch_used += 1
                    L.stamp[e] = L.tick()
            for e in need:
                if e not in L.stamp:
                    st.misses += 1
                    st.per_layer_misses[i] += 1
                    L.insert(e, protect, st, fallback=set(need))
            if use_pred:
                for Lp in ((2 * i + 2, 2 * i + 3) if schedule == "aot" else (i + 1,)):
                    if Lp >= N:
                        continue
                    P = [int(e) for e in pred[t, Lp] if e >= 0]
                    predicted[Lp] = P
                    tgt = layers[Lp]
                    for e in P:
                        if e in tgt.stamp:
                            tgt.stamp[e] = tgt.tick()
                        else:
                            tgt.insert(e, set(P), st)
                            tgt.prefetched[e] = True
                            st.prefetch_issued += 1
    return st


def simulate_fixed_experts(slow: np.ndarray, n_experts: int, slots: int) -> CacheStats:
    """Experts fixed in HBM without replacement (Sec. 3.3, first strategy).

    Experts 0..C-K-1 of every layer stay resident; every other needed expert
    is a miss and is copied into a staging slot each time a layer needs it.
    """
    T, N, K = slow.shape
    if slots < K or slots > n_experts:
        raise ValueError("need top_k <= slots <= n_experts")
    fixed = slots - K
    st = CacheStats(per_layer_misses=[0] * N)
    for t in range(T):
        for i in range(N):
            for e in slow[t, i]:
                if int(e) < fixed:
                    st.hits += 1
                else:
                    st.misses += 1
                    st.per_layer_misses[i] += 1
                    st.loads += 1
    return st
