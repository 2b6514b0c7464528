"""CPU oracle for the M2R2 decode path (arXiv 2502.02040).

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow NumPy statement of
what the decode path computes, in float64 by default.  Only the test suite,
the package smoke check and the CPU-baseline leg of the benchmark may import
it.  It shares no code with the HIP implementation: its only input-side
dependency is ``synth`` (seeded shapes, weights and prompts, which carry none
of the method's arithmetic).

Where the paper fixes a plain definition, the oracle is that definition
written out:
  * the slow stream is a standard pre-norm decoder (Eq. 1);
  * self-speculative decoding must reproduce plain greedy decoding;
  * ahead-of-time expert loading must reproduce MoE decoding with every
    expert available (the cache is simulated separately).
Where the method is a heuristic (the accelerated stream of Eq. 2 with its
shared KV cache, the exit signal, the fast-residual expert prediction and the
LRU/prefetch policy) the oracle follows the steps in the paper's order.

Every function is pinned by a CPU test (adapters set to zero collapse the
fast stream onto the slow one; never-exit reproduces a scalar-loop decoder;
speculative output equals greedy output; brute force on tiny shapes; the
textbook LRU).  Quantities that depend on trained weights (acceptance rates,
hit rates of real routers) are parity unpinned and are not claimed.
"""
from .decoder import (Oracle, KVCache, StepResult, rms_norm, rope, attend, silu, topk_desc,
                      round_to_cache, arla_score, ARLA_DIM, select_top, top_gap)
from .cache_sim import simulate_expert_cache, simulate_fixed_experts, CacheStats

__all__ = ["Oracle", "KVCache", "StepResult", "rms_norm", "rope", "attend", "silu", "topk_desc",
           "round_to_cache", "simulate_expert_cache", "simulate_fixed_experts", "CacheStats", "arla_score",
           "ARLA_DIM", "select_top", "top_gap"]
