"""Helpers shared by the GPU parity tests: run the HIP path through the C ABI
and the oracle side by side on the same seeded inputs, teacher-forced on the
GPU's tokens, and compare under one rule:

  * hidden states and logits: per-row ||x_gpu - x_ref|| / ||x_ref|| <= tol,
    tol = 1e-4 for float32 weights, 2e-2 for bfloat16 weights;
  * a token (argmax) is compared only when the oracle's top-2 margin exceeds
    2 * eps * max|z| (eps = tol); skipped comparisons are counted;
  * an exit decision is compared only when |signal - tau| > tol.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence

import numpy as np
import torch

import synth
from oracle import Oracle, KVCache
from paper_2502_02040_amd import Model, PagedKV


def tol_of(cfg) -> float:
    return 2e-2 if cfg.wdtype == "bf16" else 1e-4


def rel(a, b) -> float:
    a = np.asarray(a, np.float64).reshape(-1)
    b = np.asarray(b, np.float64).reshape(-1)
    n = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / (n if n > 0 else 1.0))


def token_decidable(logits: np.ndarray, eps: float) -> bool:
    z = np.sort(np.asarray(logits, np.float64))
    return (z[-1] - z[-2]) > 2 * eps * np.max(np.abs(z))


@dataclasses.dataclass
class Tally:
    compared: int = 0
    skipped: int = 0
    worst: float = 0.0

    def rel(self, got, ref, tol, what=""):
        e = rel(got, ref)
        self.worst = max(self.worst, e)
        assert e <= tol, f"{what}: relative error {e:.3e} > {tol:.1e}"

    def token(self, got: int, logits_ref: np.ndarray, eps: float, what=""):
        if token_decidable(logits_ref, eps):
            self.compared += 1
            assert got == int(np.argmax(logits_ref)), f"{what}: token {got} != {int(np.argmax(logits_ref))}"
        else:
            self.skipped += 1


def shuffled_table(n_seqs: int, max_ctx: int, block_size: int, seed: int) -> np.ndarray:
    bps = (max_ctx + block_size - 1) // block_size
    return synth.block_table(n_seqs, bps, seed=seed, shuffle=True)


class Pair:
    """A GPU model and the oracle over the same weights, one sequence."""

    def __init__(self, cfg, weights, *, max_ctx: int, block_size: int = 16, table_seed: int = 0, max_batch: int = 1,
                 n_seqs: int = 1):
        self.cfg = cfg
        self.tol = tol_of(cfg)
        self.model = Model(cfg, weights, max_batch=max_batch, max_chunk=16, max_ctx=max_ctx)
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
