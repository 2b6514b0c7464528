"""Seeded synthetic inputs for the M2R2 decode path.

This module is shared by the CPU oracle and the HIP path *as a source of
inputs only*: model shapes, seeded weight tensors, prompts and synthetic KV
caches.  It holds none of the method's arithmetic (no normalisation, attention,
adapters, routing or decoding) so that the two sides stay independent.

Weights follow one recipe for every configuration: each named tensor has its
own PCG64 stream keyed by ``(seed, crc32(name))`` so values never depend on the
order in which tensors are generated; matrices, embeddings, the LM head and
both adapter factors are N(0, 0.02) in float32; norm gains are 1.0.  For
bfloat16 configurations every float32 sample is rounded to the nearest
bfloat16 (ties to even) and both sides consume the rounded values.
"""
from __future__ import annotations

import dataclasses
import os
import zlib
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, Iterable, List, Optional, Tuple

import numpy as np

__all__ = [
    "ModelConfig", "CONFIGS", "tensor_specs", "make_weights", "make_tensor",
    "bf16_round", "bf16_bits", "bf16_bits_to_f32", "prompt_ids", "synthetic_kv",
    "block_table", "pool_threads",
]

PROJ_DENSE = ("q", "k", "v", "o", "g", "u", "d")
PROJ_MOE = ("q", "k", "v", "o", "m")


@dataclasses.dataclass(frozen=True)
class ModelConfig:
    """Shape and storage precision of a decoder-only transformer with an
    accelerated residual stream.

    ``wdtype``/``kvdtype`` are ``"f32"`` or ``"bf16"``.  ``n_experts == 0``
    means a dense SwiGLU MLP of width ``ffn``; otherwise each layer holds
    ``n_experts`` SwiGLU experts of width ``expert_ffn`` with top-``top_k``
    routing, and the accelerated stream uses a rank-``rank`` adapter in place
    of the MLP.
    """
    name: str
    n_layers: int
    d_model: int
    n_heads: int
    head_dim: int
    ffn: int
    vocab: int
    rank: int
    wdtype: str = "f32"
    kvdtype: str = "f32"
    rms_eps: float = 1e-5
    rope_theta: float = 10000.0
    n_experts: int = 0
    top_k: int = 0
    expert_ffn: int = 0
    seed: int = 0
    # FLOPs-optimised accelerated stream (dense models; all zero / False:
    # the memory-bound form): the fast row uses the first ``fast_heads``
    # heads, each attending to ``fast_topk`` cached positions; its MLP is the
    # rank-``rank`` adapter ``m`` alone; its tokens come from a rank-
    # ``head_rank`` head ``head_A [head_rank][d]``, ``head_B [vocab][head_rank]``
    fast_heads: int = 0
    fast_topk: int = 0
    fast_mlp_adapter: bool = False
    head_rank: int = 0

    @property
    def qdim(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def is_moe(self) -> bool:
        return self.n_experts > 0

    @property
    def is_flops(self) -> bool:
        return bool(self.fast_heads or self.fast_topk or self.fast_mlp_adapter or self.head_rank)

    def replace(self, **kw) -> "ModelConfig":
        return dataclasses.replace(self, **kw)


CONFIGS: Dict[str, ModelConfig] = {
    # Tiny dense decoder, fp32 (parity configuration).
    "tiny": ModelConfig("tiny", n_layers=2, d_model=256, n_heads=4, head_dim=64, ffn=1024, vocab=1024,
                        rank=8, wdtype="f32", kvdtype="f32", seed=1),
    # Phi-3-mini-shaped dense decoder, bf16.
    "phi3": ModelConfig("phi3", n_layers=32, d_model=3072, n_heads=32, head_dim=96, ffn=8192, vocab=32064,
                        rank=16, wdtype="bf16", kvdtype="bf16", seed=2),
    # OLMoE-shaped sparse MoE decoder, bf16.
    "olmoe": ModelConfig("olmoe", n_layers=16, d_model=2048, n_heads=16, head_dim=128, ffn=0, vocab=50304,
                         rank=16, wdtype="bf16", kvdtype="bf16", n_experts=64, top_k=8, expert_ffn=1024, seed=5),
    # Small shapes used by tests (cover ragged tiles and both precisions).
    "micro": ModelConfig("micro", n_layers=2, d_model=8, n_heads=2, head_dim=4, ffn=16, vocab=11, rank=2,
                         wdtype="f32", kvdtype="f32", seed=11),
    "small_bf16": ModelConfig("small_bf16", n_layers=3, d_model=192, n_heads=2, head_dim=96, ffn=320, vocab=1000,
                              rank=4, wdtype="bf16", kvdtype="bf16", seed=7),
    "micro_moe": ModelConfig("micro_moe", n_layers=6, d_model=16, n_heads=2, head_dim=8, ffn=0, vocab=23, rank=2,
                             wdtype="f32", kvdtype="f32", n_experts=8, top_k=2, expert_ffn=8, seed=13),
    "small_moe": ModelConfig("small_moe", n_layers=6, d_model=256, n_heads=2, head_dim=128, ffn=0, vocab=777,
                             rank=4, wdtype="bf16", kvdtype="bf16", n_experts=16, top_k=4, expert_ffn=96, seed=17),
    "small_moe_f32": ModelConfig("small_moe_f32", n_layers=5, d_model=128, n_heads=2, head_dim=64, ffn=0,
                                 vocab=300, rank=4, wdtype="f32", kvdtype="f32", n_experts=8, top_k=2,
                                 expert_ffn=64, seed=19),
    # a dense bfloat16 decoder whose rows are whole 1 KB pieces (d 512,
    # ffn 1024): the one-launch decode step at head_dim 128
    "small_rw": ModelConfig("small_rw", n_layers=3, d_model=512, n_heads=4, head_dim=128, ffn=1024, vocab=1000,
                            rank=8, wdtype="bf16", kvdtype="bf16", seed=31),
    # rows of whole 1 KB pieces: the one- and two-row q/k/v, o and head kernels
    "small_moe_rw": ModelConfig("small_moe_rw", n_layers=4, d_model=512, n_heads=4, head_dim=128, ffn=0, vocab=1000,
                                rank=8, wdtype="bf16", kvdtype="bf16", n_experts=16, top_k=4, expert_ffn=96, seed=23),
}
# FLOPs-optimised fast stream on the same shapes: a quarter of the heads
# (half for the small decoders), top-64 positions (8 at test sizes), the
# adapter-only MLP and a low-rank head for the fast row's tokens
CONFIGS["phi3_flops"] = CONFIGS["phi3"].replace(name="phi3_flops", fast_heads=8, fast_topk=64, fast_mlp_adapter=True,
                                                head_rank=64)
CONFIGS["tiny_flops"] = CONFIGS["tiny"].replace(name="tiny_flops", fast_heads=2, fast_topk=8, fast_mlp_adapter=True,
                                                head_rank=16)
CONFIGS["small_bf16_flops"] = CONFIGS["small_bf16"].replace(name="small_bf16_flops", fast_heads=1, fast_topk=8,
                                                            fast_mlp_adapter=True, head_rank=16)
CONFIGS["small_rw_flops"] = CONFIGS["small_rw"].replace(name="small_rw_flops", fast_heads=2, fast_topk=8,
                                                        fast_mlp_adapter=True, head_rank=32)
CONFIGS["micro_flops"] = CONFIGS["micro"].replace(name="micro_flops", fast_heads=1, fast_topk=3, fast_mlp_adapter=True,
                                                  head_rank=3)


# ----------------------------------------------------------------------------
# bfloat16 storage helpers (input preparation only)
# ----------------------------------------------------------------------------

def bf16_bits(a: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest, ties to even."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + r) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def bf16_round(a: np.ndarray) -> np.ndarray:
    """Values of ``a`` rounded to the nearest bfloat16, returned as float32."""
    return bf16_bits_to_f32(bf16_bits(a))


# ----------------------------------------------------------------------------
# Tensor inventory
# ----------------------------------------------------------------------------

def _adapter_dims(cfg: ModelConfig, proj: str) -> Tuple[int, int]:
    d, q, f = cfg.d_model, cfg.qdim, cfg.ffn
    return {"q": (d, q), "k": (d, q), "v": (d, q), "o": (q, d), "g": (d, f), "u": (d, f), "d": (f, d),
            "m": (d, d)}[proj]


def tensor_specs(cfg: ModelConfig) -> List[Tuple[str, Tuple[int, ...], str]]:
    """Every weight tensor as ``(name, shape, kind)`` with kind in
    {"normal", "ones"}.  Matrices are stored ``[d_out][d_in]``; adapter
    factors are ``A [rank][d_in]`` and ``B [d_out][rank]``."""
    d, q, r = cfg.d_model, cfg.qdim, cfg.rank
    specs: List[Tuple[str, Tuple[int, ...], str]] = [("embed", (cfg.vocab, d), "normal")]
    for l in range(cfg.n_layers):
        p = f"L{l}."
        specs += [(p + "attn_norm", (d,), "ones"), (p + "wq", (q, d), "normal"), (p + "wk", (q, d), "normal"),
                  (p + "wv", (q, d), "normal"), (p + "wo", (d, q), "normal"), (p + "mlp_norm", (d,), "ones")]
        if cfg.is_moe:
            specs.append((p + "router", (cfg.n_experts, d), "normal"))
            for e in range(cfg.n_experts):
                fe = cfg.expert_ffn
                specs += [(p + f"E{e}.wg", (fe, d), "normal"), (p + f"E{e}.wu", (fe, d), "normal"),
                          (p + f"E{e}.wd", (d, fe), "normal")]
            projs = PROJ_MOE
        else:
            specs += [(p + "wg", (cfg.ffn, d), "normal"), (p + "wu", (cfg.ffn, d), "normal"),
                      (p + "wd", (d, cfg.ffn), "normal")]
            projs = PROJ_MOE if cfg.fast_mlp_adapter else PROJ_DENSE
        for pr in projs:
            din, dout = _adapter_dims(cfg, pr)
            specs += [(p + f"A_{pr}", (r, din), "normal"), (p + f"B_{pr}", (dout, r), "normal")]
    specs += [("final_norm", (d,), "ones"), ("lm_head", (cfg.vocab, d), "normal")]
    if cfg.head_rank:
        specs += [("head_A", (cfg.head_rank, d), "normal"), ("head_B", (cfg.vocab, cfg.head_rank), "normal")]
    return specs


def _stream(seed: int, name: str) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, zlib.crc32(name.encode())])))


def make_tensor(cfg: ModelConfig, name: str, shape: Tuple[int, ...], kind: str, *,
                adapter_scale: float = 1.0, decay: Optional[Tuple[int, float]] = None,
                router_coherent: bool = False, embed_scale: float = 1.0) -> np.ndarray:
    """One weight tensor as float32 (already rounded to bf16 for bf16 configs).

    Variants used by the structured experiments:
      * ``adapter_scale`` multiplies both adapter factors (0 gives a fast
        stream identical to the slow one);
      * ``decay=(layer, lam)`` scales ``wo`` and ``wd`` of layers >= layer by
        ``lam`` (a shrinking late-layer update);
      * ``router_coherent`` draws router ``l`` as ``shared + 0.5 * noise_l``;
      * ``embed_scale`` multiplies the token embedding (a larger one keeps the
        token's identity visible in the residual stream through the layers,
        as in trained models, instead of a residual dominated by the context
        average that the attention layers add).
    """
    if kind == "ones":
        a = np.ones(shape, np.float32)
    else:
        a = np.empty(shape, np.float32)
        _stream(cfg.seed, name).standard_normal(out=a, dtype=np.float32)
        if router_coherent and name.endswith(".router"):
            shared = np.empty(shape, np.float32)
            _stream(cfg.seed, "router.shared").standard_normal(out=shared, dtype=np.float32)
            a = shared + np.float32(0.5) * a
        a *= np.float32(0.02)
        if name == "embed":
            a *= np.float32(embed_scale)
        base = name.split(".")[-1]
        if base.startswith("A_") or base.startswith("B_"):
            a *= np.float32(adapter_scale)
        if decay is not None and name.startswith("L") and base in ("wo", "wd"):
            layer = int(name[1:name.index(".")])
            if layer >= decay[0]:
                a *= np.float32(decay[1])
    if cfg.wdtype == "bf16":
        a = bf16_round(a)
    return a


def pool_threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def make_weights(cfg: ModelConfig, *, names: Optional[Iterable[str]] = None, threads: Optional[int] = None,
                 **variant) -> Dict[str, np.ndarray]:
    """All (or the named) weight tensors of ``cfg`` as float32 arrays."""
    specs = tensor_specs(cfg)
    if names is not None:
        want = set(names)
        specs = [s for s in specs if s[0] in want]
    threads = threads or pool_threads()
    out: Dict[str, np.ndarray] = {}
    with ThreadPoolExecutor(threads) as ex:
        for (name, _, _), arr in zip(specs, ex.map(lambda s: make_tensor(cfg, *s, **variant), specs)):
            out[name] = arr
    return out


def prompt_ids(cfg: ModelConfig, n: int, *, seed: Optional[int] = None, stream: str = "prompt") -> np.ndarray:
    """``n`` token ids drawn uniformly from ``[0, vocab)``."""
    g = _stream(cfg.seed if seed is None else seed, stream)
    return g.integers(0, cfg.vocab, size=n, dtype=np.int64).astype(np.int32)


def synthetic_kv(cfg: ModelConfig, length: int, *, seq: int = 0, layers: Optional[Iterable[int]] = None,
                 threads: int = 1) -> Dict[int, Tuple[np.ndarray, np.ndarray]]:
    """Seeded stand-in KV cache content: per layer ``(K, V)`` each
    ``[length][n_heads][head_dim]`` drawn N(0, 1) and stored in the cache dtype."""
    layers = list(range(cfg.n_layers) if layers is None else layers)

    def one(lw):
        l, which = lw
        a = np.empty((length, cfg.n_heads, cfg.head_dim), np.float32)
        _stream(cfg.seed, f"kv.{seq}.{l}.{which}").standard_normal(out=a, dtype=np.float32)
        return bf16_round(a) if cfg.kvdtype == "bf16" else a

    jobs = [(l, w) for l in layers for w in ("K", "V")]
    with ThreadPoolExecutor(max(1, threads)) as ex:
        arrs = list(ex.map(one, jobs))
    return {l: (arrs[2 * i], arrs[2 * i + 1]) for i, l in enumerate(layers)}


def block_table(n_seqs: int, blocks_per_seq: int, *, seed: int = 0, shuffle: bool = True) -> np.ndarray:
    """A ``[n_seqs][blocks_per_seq]`` table of distinct physical block ids in
    ``[0, n_seqs*blocks_per_seq)``, optionally shuffled (seeded)."""
    ids = np.arange(n_seqs * blocks_per_seq, dtype=np.int32)
    if shuffle:
        _stream(seed, "block_table").shuffle(ids)
    return ids.reshape(n_seqs, blocks_per_seq)


def preload_table(cfg: ModelConfig, n_tokens: int, *, seed: Optional[int] = None) -> np.ndarray:
    """``[n_tokens][n_layers][top_k]`` expert ids for the random-preload cache
    strategy: in every row ``top_k`` distinct experts drawn uniformly from
    ``[0, n_experts)`` (row 0 of each token, layer 0, is never used)."""
    g = _stream(cfg.seed if seed is None else seed, "preload")
    keys = g.random((n_tokens, cfg.n_layers, cfg.n_experts))
    return np.argsort(keys, axis=-1, kind="stable")[..., :cfg.top_k].astype(np.int32)


def zipf_ids(cfg: ModelConfig, n: int, *, s: float = 1.0, seed: Optional[int] = None,
             stream: str = "zipf") -> np.ndarray:
    """``n`` token ids whose frequencies follow Zipf's law, the rank-frequency
    shape of natural text: the id of rank r (a seeded permutation of the
    vocabulary) is drawn with probability proportional to r**-s."""
    g = _stream(cfg.seed if seed is None else seed, stream)
    p = np.arange(1, cfg.vocab + 1, dtype=np.float64) ** -s
    p /= p.sum()
    perm = g.permutation(cfg.vocab)
    return perm[g.choice(cfg.vocab, size=n, p=p)].astype(np.int32)


def arla_weights(cfg: ModelConfig, *, dim: int = 64, seed: Optional[int] = None) -> Dict[str, np.ndarray]:
    """Weights of the latent-attention exit router, one block per boundary b
    (block 0 unused): ``wq``, ``wk``, ``wv`` [n_layers, dim, d] N(0, 0.02) in
    the weight dtype (as float32), ``w_out`` [n_layers, dim] N(0, 1/dim) and
    ``b_out`` [n_layers] zero, float32."""
    s = cfg.seed if seed is None else seed
    out: Dict[str, np.ndarray] = {}
    for nm in ("wq", "wk", "wv"):
        a = _stream(s, f"arla.{nm}").standard_normal((cfg.n_layers, dim, cfg.d_model), dtype=np.float32)
        a *= np.float32(0.02)
        out[nm] = bf16_round(a) if cfg.wdtype == "bf16" else a
    out["w_out"] = (_stream(s, "arla.w_out").standard_normal((cfg.n_layers, dim), dtype=np.float32)
                    * np.float32(1.0 / np.sqrt(dim))).astype(np.float32)
    out["b_out"] = np.zeros(cfg.n_layers, np.float32)
    return out
