"""Helpers shared by the GPU parity tests: run the HIP path through the C ABI
and the oracle side by side on the same seeded inputs, teacher-forced on the
GPU's tokens, and compare under one rule:

  * hidden states, logits and cache slabs: per array the norm-wise error
    ||x_gpu - x_ref|| / ||x_ref|| <= tol, and per row (the last axis) every
    element |x_gpu - x_ref| <= tol * max|x_ref row|; tol = 1e-4 for float32
    weights, 2e-2 for bfloat16 weights;
  * a token (argmax) is compared only when the oracle's top-2 margin exceeds
    2 * eps * max|z| (eps = tol); an expert list position by position where
    the router logits on both sides of it are further apart than that bound;
  * an exit decision is compared only when |signal - tau| > tol.
Comparisons not made are counted (``skipped``), never dropped silently; every
test asserts a minimum number of comparisons, and the session ends with a
table of every test's counts and worst errors.
"""
from __future__ import annotations

import copy
import dataclasses
import weakref
from typing import List, Optional, Sequence

import numpy as np
import torch

import synth
from oracle import Oracle, KVCache
from oracle.decoder import argmax_first, round_to_cache
from paper_2502_02040_amd import Model, PagedKV

# (test id, Tally) of the session, printed at its end by conftest
TALLIES: List = []
CURRENT_TEST = [None]
# models whose sticky device error bits are checked after every GPU test
_MODELS: List[weakref.ref] = []


def track(model):
    """Check `model`'s device error bits after every GPU test while it lives."""
    _MODELS.append(weakref.ref(model))
    return model


def live_models():
    alive = [r() for r in _MODELS]
    _MODELS[:] = [r for r, m in zip(list(_MODELS), alive) if m is not None]
    return [m for m in alive if m is not None]


def tol_of(cfg) -> float:
    return 2e-2 if cfg.wdtype == "bf16" else 1e-4


def rel(a, b) -> float:
    a = np.asarray(a, np.float64).reshape(-1)
    b = np.asarray(b, np.float64).reshape(-1)
    n = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / (n if n > 0 else 1.0))


def elem_ratio(a, b) -> float:
    """Largest |a - b| of a row (the last axis) over the largest |b| of that row."""
    b = np.asarray(b, np.float64)
    a = np.asarray(a, np.float64).reshape(b.shape)
    rows_a = a.reshape(-1, b.shape[-1]) if b.ndim > 1 else a.reshape(1, -1)
    rows_b = b.reshape(-1, b.shape[-1]) if b.ndim > 1 else b.reshape(1, -1)
    err = np.max(np.abs(rows_a - rows_b), axis=1)
    scale = np.maximum(np.max(np.abs(rows_b), axis=1), 1e-30)
    return float(np.max(err / scale))


def token_decidable(logits: np.ndarray, eps: float) -> bool:
    z = np.sort(np.asarray(logits, np.float64))
    return (z[-1] - z[-2]) > 2 * eps * np.max(np.abs(z))


@dataclasses.dataclass
class Tally:
    compared: int = 0       # decisions compared (tokens, expert positions, exit boundaries, acceptance)
    arrays: int = 0         # arrays compared element by element (states, logits, signals, cache slabs)
    skipped: int = 0        # decisions not compared (near ties)
    steps: int = 0          # decode steps or rounds whose outputs were compared in full
    worst: float = 0.0      # largest norm-wise relative error
    worst_elem: float = 0.0  # largest element error relative to its row's largest reference value

    def __post_init__(self):
        TALLIES.append((CURRENT_TEST[0], self))

    def rel(self, got, ref, tol, what=""):
        ref = np.asarray(ref, np.float64)
        got = np.asarray(got, np.float64)
        assert got.size == ref.size, f"{what}: {got.shape} vs {ref.shape}"
        e, el = rel(got, ref), elem_ratio(got, ref)
        self.worst = max(self.worst, e)
        self.worst_elem = max(self.worst_elem, el)
        self.arrays += 1
        assert e <= tol, f"{what}: relative error {e:.3e} > {tol:.1e}"
        assert el <= tol, f"{what}: element error {el:.3e} of the row's largest value > {tol:.1e}"

    def close(self, got, ref, tol, what=""):
        """Absolute element-wise bound (signals, which lie in [-1, 1])."""
        got = np.asarray(got, np.float64).reshape(-1)
        ref = np.asarray(ref, np.float64).reshape(-1)
        e = float(np.max(np.abs(got - ref))) if ref.size else 0.0
        self.worst_elem = max(self.worst_elem, e)
        self.arrays += 1
        assert e <= tol, f"{what}: max abs error {e:.3e} > {tol:.1e}"

    def token(self, got: int, logits_ref: np.ndarray, eps: float, what=""):
        if token_decidable(logits_ref, eps):
            self.compared += 1
            assert got == int(np.argmax(logits_ref)), f"{what}: token {got} != {int(np.argmax(logits_ref))}"
        else:
            self.skipped += 1

    def equal(self, got, ref, what=""):
        """An exact (integer) result."""
        self.compared += 1
        assert got == ref, f"{what}: {got} != {ref}"

    def experts(self, got: Sequence[int], ref: Sequence[int], logits_ref: np.ndarray, k: int, eps: float,
                what="") -> bool:
        """Expert list in descending router order (lowest id on ties).
        Position j is decided when the oracle's sorted logits j-1|j and j|j+1
        are both further apart than the bound; a run of undecided positions
        is compared as a set, provided the logits around the run decide it.
        Returns True when the chosen set is decided (and so compared)."""
        z = np.sort(np.asarray(logits_ref, np.float64))[::-1]
        bound = 2 * eps * np.max(np.abs(z))
        gap = [z[j] - z[j + 1] > bound for j in range(min(k, len(z) - 1))]   # gap[j]: between j and j+1
        set_ok = k >= len(z) or gap[k - 1]
        got, ref = [int(x) for x in got], [int(x) for x in ref]
        j = 0
        while j < k:
            e = j
            while e < k - 1 and not gap[e]:
                e += 1
            # positions j..e form a group bounded by decided gaps (or the list ends)
            closed = (j == 0 or gap[j - 1]) and (e == k - 1 and set_ok or e < k - 1 and gap[e])
            if closed:
                self.compared += 1
                if e == j:
                    assert got[j] == ref[j], f"{what}: position {j}: {got[j]} != {ref[j]}"
                else:
                    assert sorted(got[j:e + 1]) == sorted(ref[j:e + 1]), f"{what}: positions {j}..{e}"
            else:
                self.skipped += 1
            j = e + 1
        return set_ok


def shuffled_table(n_seqs: int, max_ctx: int, block_size: int, seed: int) -> np.ndarray:
    bps = (max_ctx + block_size - 1) // block_size
    return synth.block_table(n_seqs, bps, seed=seed, shuffle=True)


def pick_tau(orc: Oracle, token: int, pos: int, cache: KVCache, gates: Sequence[int], candidates: Sequence[float],
             eps: float, arla=None) -> Optional[float]:
    """First threshold of `candidates` that every gate signal of this step
    decides clearly (|s - tau| > eps).  The signals up to the exit do not
    depend on tau (every gate that does not fire restarts p from h), so an
    OBSERVE step of the oracle on a copy of the cache gives them."""
    r = orc.decode_step(token, pos, copy.deepcopy(cache), gates=gates, tau=2.0, mode="observe", arla=arla)
    s = [r.signal[b - 1] for b in gates]
    for tau in candidates:
        if all(abs(x - tau) > eps for x in s):
            return tau
    return None


def oracle_draft_logits(orc: Oracle, token: int, pos: int, cache: KVCache, exit_layer: int, gamma: int,
                        drafts_fed: Optional[Sequence[int]] = None):
    """The oracle's draft (Sec. 2.3.2) with the logits of every draft
    position.  With `drafts_fed` (the GPU's drafts) draft j+1 starts from
    drafts_fed[j] (teacher forcing), so one near tie does not end the
    comparison."""
    cfg = orc.cfg
    scK = [np.zeros((gamma, cfg.n_heads, cfg.head_dim)) for _ in range(exit_layer)]
    scV = [np.zeros((gamma, cfg.n_heads, cfg.head_dim)) for _ in range(exit_layer)]
    out, zs, tok = [], [], token
    for j in range(gamma):
        p = orc.w["embed"][tok].copy()
        for l in range(exit_layer):
            ctxK = np.concatenate([cache.K[l][:pos], scK[l][:j]], axis=0)
            ctxV = np.concatenate([cache.V[l][:pos], scV[l][:j]], axis=0)
            p, (k, v) = orc._fast_layer(l, p, pos + j, ctxK, ctxV)
            scK[l][j] = round_to_cache(k, cfg.kvdtype)
            scV[l][j] = round_to_cache(v, cfg.kvdtype)
        z = orc.head_logits(p)
        out.append(argmax_first(z))
        zs.append(z)
        tok = drafts_fed[j] if drafts_fed is not None else out[-1]
    return out, zs


class Pair:
    """A GPU model and the oracle over the same weights, one sequence."""

    def __init__(self, cfg, weights, *, max_ctx: int, block_size: int = 16, table_seed: int = 0, max_batch: int = 1,
                 n_seqs: int = 1):
        self.cfg = cfg
        self.tol = tol_of(cfg)
        self.model = track(Model(cfg, weights, max_batch=max_batch, max_chunk=16, max_ctx=max_ctx))
        self.kv = PagedKV(cfg, n_seqs, max_ctx, block_size=block_size,
                          block_table=shuffled_table(n_seqs, max_ctx, block_size, table_seed))
        self.orc = Oracle(cfg, weights)
        self.max_ctx = max_ctx
        self.caches = [KVCache(cfg, max_ctx) for _ in range(n_seqs)]
        self.dev = torch.device("cuda")

    def prefill(self, prompt: Sequence[int], seq: int = 0, tally: Optional[Tally] = None) -> int:
        """Chunked slow forward of the prompt on both sides; returns the GPU's first token."""
        pos = torch.zeros(1, dtype=torch.int32, device=self.dev)
        targets = torch.zeros(16, dtype=torch.int32, device=self.dev)
        ref = self.orc.slow_chunk(list(prompt), 0, self.caches[seq])
        tok = None
        for c0 in range(0, len(prompt), 16):
            chunk = torch.tensor(list(prompt[c0:c0 + 16]), dtype=torch.int32, device=self.dev)
            n = chunk.numel()
            self.model.verify(chunk, n, pos, self.kv.desc(seq), targets)
            torch.cuda.synchronize()
            got = targets[:n].cpu().numpy()
            if tally is not None:
                for i in range(n):
                    tally.token(int(got[i]), ref[c0 + i], self.tol, f"prefill row {c0 + i}")
            tok = int(got[n - 1])
        assert int(pos.item()) == len(prompt)
        assert int(self.kv.seq_lens[seq].item()) == len(prompt)
        return tok

    def check_cache(self, seq: int, start: int, end: int, tally: Tally, what: str = "") -> None:
        for l in range(self.cfg.n_layers):
            K, V = self.kv.read(seq, l, start, end)
            tally.rel(K, self.caches[seq].K[l][start:end], self.tol, f"{what} K layer {l}")
            tally.rel(V, self.caches[seq].V[l][start:end], self.tol, f"{what} V layer {l}")
