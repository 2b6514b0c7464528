"""ctypes binding of ``libm2r2.so`` (include/m2r2.h).

Argument marshalling only: every step of the decode path runs in the HIP
kernels behind the C ABI.  torch is used for device memory (weights,
workspace, KV pages) and for stream handles.  If the library is not built
this module raises on use: there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_float, c_int32, c_size_t, c_void_p
from typing import Dict, Optional, Sequence

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libm2r2.so")

F32, BF16 = 0, 1
EXIT_OFF, EXIT_OBSERVE, EXIT_EXIT = 0, 1, 2
MODES = {"off": EXIT_OFF, "observe": EXIT_OBSERVE, "exit": EXIT_EXIT}
PROJ = ("q", "k", "v", "o", "g", "u", "d")

# include/m2r2.h: the decode path's boundary
EXPORTS = ("m2r2_workspace_size", "m2r2_create", "m2r2_destroy", "m2r2_decode_step", "m2r2_draft", "m2r2_verify",
           "m2r2_device_errors", "m2r2_sync_check", "m2r2_decode_step_noalloc",
           "m2r2_last_error", "m2r2_expert_bytes", "m2r2_pack_expert", "m2r2_moe_set_policy", "m2r2_prefetch_experts",
           "m2r2_moe_reset", "m2r2_moe_stats", "m2r2_expert_cache_replay", "m2r2_moe_set_preload_table",
           "m2r2_set_arla")
# include/m2r2_measure.h: measurement hooks
MEASURE_EXPORTS = ("m2r2_timing_enable", "m2r2_timing_read", "m2r2_time_gateup_layers")
KERNEL_CLASSES = {"qkv": 0, "attn": 1, "oproj": 2, "gateup": 3, "down": 4, "head": 5, "embed": 6, "attn_merge": 7,
                  "expert_gateup": 8, "expert_down": 9, "router": 10, "step": 11}
MOE_ON_DEMAND, MOE_AHEAD_OF_TIME, MOE_FIXED, MOE_RANDOM_PRELOAD, MOE_PREVIOUS_LAYER = 0, 1, 2, 3, 4
POLICIES = {"on_demand": MOE_ON_DEMAND, "ahead_of_time": MOE_AHEAD_OF_TIME, "fixed": MOE_FIXED,
            "random_preload": MOE_RANDOM_PRELOAD, "previous_layer": MOE_PREVIOUS_LAYER}


class Config(ctypes.Structure):
    _fields_ = [("n_layers", c_int32), ("d_model", c_int32), ("n_heads", c_int32), ("head_dim", c_int32),
                ("ffn", c_int32), ("vocab", c_int32), ("rank", c_int32), ("wdtype", c_int32), ("kvdtype", c_int32),
                ("rms_eps", c_float), ("rope_theta", c_float), ("n_experts", c_int32), ("top_k", c_int32),
                ("expert_ffn", c_int32), ("expert_slots", c_int32), ("fast_heads", c_int32), ("fast_topk", c_int32),
                ("fast_mlp_adapter", c_int32), ("head_rank", c_int32)]


class LayerWeights(ctypes.Structure):
    _fields_ = [("attn_norm", c_void_p), ("wq", c_void_p), ("wk", c_void_p), ("wv", c_void_p), ("wo", c_void_p),
                ("mlp_norm", c_void_p), ("wg", c_void_p), ("wu", c_void_p), ("wd", c_void_p),
                ("A", c_void_p * 7), ("B", c_void_p * 7), ("router", c_void_p), ("A_m", c_void_p), ("B_m", c_void_p)]


class Weights(ctypes.Structure):
    _fields_ = [("embed", c_void_p), ("final_norm", c_void_p), ("lm_head", c_void_p),
                ("layers", POINTER(LayerWeights)), ("experts_h", c_void_p), ("head_a", c_void_p),
                ("head_b", c_void_p)]


class KV(ctypes.Structure):
    _fields_ = [("k_pages", c_void_p), ("v_pages", c_void_p), ("block_table_d", c_void_p), ("seq_lens_d", c_void_p),
                ("num_blocks", c_int32), ("block_size", c_int32), ("max_blocks_per_seq", c_int32)]


class Exit(ctypes.Structure):
    _fields_ = [("gates_h", POINTER(c_int32)), ("n_gates", c_int32), ("tau", c_float), ("mode", c_int32)]


class StepOut(ctypes.Structure):
    _fields_ = [("next_token_d", c_void_p), ("exit_boundary_d", c_void_p), ("signal_d", c_void_p),
                ("logits_d", c_void_p), ("h_out_d", c_void_p), ("p_out_d", c_void_p), ("advance", c_int32),
                ("slow_experts_d", c_void_p), ("pred_experts_d", c_void_p)]


_I64 = ctypes.c_int64
COUNTER_FIELDS = ("hits", "misses", "prefetch_issued", "prefetch_used", "prefetch_wasted", "loads", "pred_correct",
                  "pred_total", "h2d_bytes", "copy_waits", "host_wait_ns", "copies_failed")


class Arla(ctypes.Structure):
    _fields_ = [("wq", c_void_p), ("wk", c_void_p), ("wv", c_void_p), ("w_out", c_void_p), ("b_out", c_void_p)]


class MoeCounters(ctypes.Structure):
    _fields_ = [(f, _I64) for f in COUNTER_FIELDS] + [("layer_misses", _I64 * 128)]

    def as_dict(self, n_layers: int) -> dict:
        d = {f: int(getattr(self, f)) for f in COUNTER_FIELDS}
        d["layer_misses"] = [int(self.layer_misses[i]) for i in range(n_layers)]
        return d


_lib = None


def lib() -> ctypes.CDLL:
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2502_02040_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        L.m2r2_workspace_size.argtypes = [POINTER(Config), c_int32, c_int32, c_int32, POINTER(c_size_t)]
        L.m2r2_create.argtypes = [POINTER(Config), POINTER(Weights), c_int32, c_int32, c_int32, c_void_p, c_size_t,
                                  POINTER(c_void_p)]
        L.m2r2_destroy.argtypes = [c_void_p]
        L.m2r2_destroy.restype = None
        L.m2r2_decode_step.argtypes = [c_void_p, c_int32, c_int32, c_void_p, c_void_p, POINTER(KV), POINTER(Exit),
                                       POINTER(StepOut), c_void_p]
        L.m2r2_decode_step_noalloc.argtypes = [c_void_p, c_int32, c_int32, c_void_p, c_void_p, POINTER(KV),
                                               POINTER(Exit), POINTER(StepOut), c_void_p]
        L.m2r2_draft.argtypes = [c_void_p, c_void_p, c_void_p, c_int32, c_int32, POINTER(KV), c_void_p, c_void_p]
        L.m2r2_verify.argtypes = [c_void_p, c_void_p, c_int32, c_void_p, POINTER(KV), c_void_p, c_void_p, c_void_p,
                                  c_void_p]
        L.m2r2_timing_enable.argtypes = [c_void_p, c_int32]
        L.m2r2_timing_read.argtypes = [c_void_p, POINTER(ctypes.c_double), POINTER(c_int32)]
        L.m2r2_time_gateup_layers.argtypes = [c_void_p, c_int32, c_void_p, POINTER(ctypes.c_double)]
        L.m2r2_device_errors.argtypes = [c_void_p, c_void_p, POINTER(c_int32)]
        L.m2r2_sync_check.argtypes = [c_void_p, c_void_p]
        L.m2r2_last_error.restype = ctypes.c_char_p
        L.m2r2_expert_bytes.argtypes = [POINTER(Config), POINTER(c_size_t)]
        L.m2r2_pack_expert.argtypes = [POINTER(Config), c_void_p, c_void_p, c_void_p, c_void_p]
        L.m2r2_moe_set_policy.argtypes = [c_void_p, c_int32]
        L.m2r2_prefetch_experts.argtypes = [c_void_p, c_int32, POINTER(c_int32), c_int32, c_int32, c_void_p]
        L.m2r2_moe_reset.argtypes = [c_void_p]
        L.m2r2_moe_set_preload_table.argtypes = [c_void_p, c_void_p, c_int32]
        L.m2r2_set_arla.argtypes = [c_void_p, c_void_p]
        L.m2r2_moe_stats.argtypes = [c_void_p, POINTER(MoeCounters)]
        L.m2r2_expert_cache_replay.argtypes = [c_int32, c_int32, c_int32, c_int32, c_int32, c_void_p, c_void_p,
                                               c_int32, POINTER(MoeCounters)]
        for f in ("m2r2_workspace_size", "m2r2_create", "m2r2_decode_step", "m2r2_draft", "m2r2_verify",
                  "m2r2_timing_enable", "m2r2_timing_read", "m2r2_time_gateup_layers", "m2r2_device_errors",
                  "m2r2_sync_check", "m2r2_decode_step_noalloc", "m2r2_expert_bytes",
                  "m2r2_pack_expert", "m2r2_moe_set_policy", "m2r2_prefetch_experts", "m2r2_moe_reset",
                  "m2r2_moe_stats", "m2r2_expert_cache_replay", "m2r2_moe_set_preload_table", "m2r2_set_arla"):
            getattr(L, f).restype = c_int32
        _lib = L
    return _lib


class M2R2Error(RuntimeError):
    def __init__(self, status: int, where: str):
        msg = lib().m2r2_last_error().decode()
        super().__init__(f"{where} failed with status {status}: {msg}")
        self.status = status


def _check(st: int, where: str) -> None:
    if st != 0:
        raise M2R2Error(st, where)


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> int:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def make_config(cfg, expert_slots: Optional[int] = None) -> Config:
    slots = cfg.n_experts if expert_slots is None else expert_slots
    return Config(cfg.n_layers, cfg.d_model, cfg.n_heads, cfg.head_dim, cfg.ffn, cfg.vocab, cfg.rank,
                  BF16 if cfg.wdtype == "bf16" else F32, BF16 if cfg.kvdtype == "bf16" else F32,
                  cfg.rms_eps, cfg.rope_theta, cfg.n_experts, cfg.top_k, cfg.expert_ffn, slots,
                  getattr(cfg, "fast_heads", 0), getattr(cfg, "fast_topk", 0), int(getattr(cfg, "fast_mlp_adapter", 0)),
                  getattr(cfg, "head_rank", 0))


def workspace_size(cfg, max_batch: int, max_chunk: int, max_ctx: int, expert_slots: Optional[int] = None) -> int:
    n = c_size_t(0)
    _check(lib().m2r2_workspace_size(ctypes.byref(make_config(cfg, expert_slots)), max_batch, max_chunk, max_ctx,
                                     ctypes.byref(n)), "m2r2_workspace_size")
    return n.value


def expert_bytes(cfg) -> int:
    n = c_size_t(0)
    _check(lib().m2r2_expert_bytes(ctypes.byref(make_config(cfg)), ctypes.byref(n)), "m2r2_expert_bytes")
    return n.value


def _host_matrix(a: np.ndarray, wdtype: str) -> np.ndarray:
    """A weight matrix in its storage dtype (bf16 bit patterns or float32)."""
    if wdtype == "bf16":
        u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
        return ((u + (((u >> 16) & 1) + np.uint32(0x7FFF))) >> 16).astype(np.uint16)
    return np.ascontiguousarray(a, dtype=np.float32)


def pack_expert_store(cfg, expert_source, *, threads: int = 8):
    """Pinned host tensor holding every expert of every layer in the packed
    layout of the C library; ``expert_source(l, e)`` returns the row-major
    (gate, up, down) matrices of expert e of layer l."""
    import torch
    from concurrent.futures import ThreadPoolExecutor
    eb = expert_bytes(cfg)
    store = torch.empty(cfg.n_layers * cfg.n_experts * eb, dtype=torch.uint8, pin_memory=True)
    base = store.data_ptr()
    c = make_config(cfg)

    def one(le):
        l, e = le
        g, u, d = (_host_matrix(x, cfg.wdtype) for x in expert_source(l, e))
        _check(lib().m2r2_pack_expert(ctypes.byref(c), g.ctypes.data, u.ctypes.data, d.ctypes.data,
                                      base + (l * cfg.n_experts + e) * eb), "m2r2_pack_expert")

    jobs = [(l, e) for l in range(cfg.n_layers) for e in range(cfg.n_experts)]
    with ThreadPoolExecutor(threads) as ex:
        list(ex.map(one, jobs))
    return store


def cache_replay(n_layers: int, n_experts: int, top_k: int, slots: int, slow: np.ndarray,
                 pred: Optional[np.ndarray] = None, prefetch=True) -> dict:
    """Host-only replay of the library's expert-cache policy on a trace
    ``slow[t][l][k]`` (and predictions of the same shape, -1 where none).
    ``prefetch``: a policy name, or a bool (ahead of time / on demand)."""
    policy = POLICIES[prefetch] if isinstance(prefetch, str) else (MOE_AHEAD_OF_TIME if prefetch else MOE_ON_DEMAND)
    slow = np.ascontiguousarray(slow, dtype=np.int32)
    pr = None if pred is None else np.ascontiguousarray(pred, dtype=np.int32)
    out = MoeCounters()
    _check(lib().m2r2_expert_cache_replay(n_layers, n_experts, top_k, slots, slow.shape[0], slow.ctypes.data,
                                          None if pr is None else pr.ctypes.data, policy,
                                          ctypes.byref(out)), "m2r2_expert_cache_replay")
    return out.as_dict(n_layers)


class PagedKV:
    """Paged slow-stream KV cache in device memory (caller-owned, per the ABI):
    pages ``[n_layers][num_blocks][H][block_size][hd]``, one block table
    ``[n_seqs][max_blocks_per_seq]`` shared by all layers."""

    def __init__(self, cfg, n_seqs: int, max_ctx: int, *, block_size: int = 16, block_table=None,
                 num_blocks: Optional[int] = None, device="cuda"):
        import torch
        self.cfg = cfg
        self.block_size = block_size
        self.max_blocks_per_seq = (max_ctx + block_size - 1) // block_size
        if block_table is None:
            block_table = np.arange(n_seqs * self.max_blocks_per_seq, dtype=np.int32).reshape(
                n_seqs, self.max_blocks_per_seq)
        block_table = np.asarray(block_table, np.int32)
        assert block_table.shape == (n_seqs, self.max_blocks_per_seq)
        self.num_blocks = int(num_blocks if num_blocks is not None else block_table.max() + 1)
        dt = torch.bfloat16 if cfg.kvdtype == "bf16" else torch.float32
        shape = (cfg.n_layers, self.num_blocks, cfg.n_heads, block_size, cfg.head_dim)
        self.k = torch.zeros(shape, dtype=dt, device=device)
        self.v = torch.zeros(shape, dtype=dt, device=device)
        self.block_table_np = block_table
        self.block_table = torch.tensor(block_table, device=device)
        self.seq_lens = torch.zeros(n_seqs, dtype=torch.int32, device=device)

    def desc(self, seq: int = 0) -> KV:
        """Descriptor whose first sequence is block-table row `seq`."""
        return KV(self.k.data_ptr(), self.v.data_ptr(), self.block_table[seq:].data_ptr(),
                  self.seq_lens[seq:].data_ptr(), self.num_blocks, self.block_size, self.max_blocks_per_seq)

    def _index(self, seq: int, positions: np.ndarray):
        blk = self.block_table_np[seq][positions // self.block_size]
        return blk, positions % self.block_size

    def load(self, seq: int, layer: int, K: np.ndarray, V: np.ndarray, start: int = 0) -> None:
        """Store ``K/V [T][H][hd]`` at positions start.. of a sequence."""
        import torch
        blk, slot = self._index(seq, np.arange(start, start + K.shape[0]))
        bi = torch.tensor(blk, device=self.k.device, dtype=torch.long)
        si = torch.tensor(slot, device=self.k.device, dtype=torch.long)
        self.k[layer, bi, :, si, :] = torch.tensor(np.asarray(K, np.float32)).to(self.k.dtype).to(self.k.device)
        self.v[layer, bi, :, si, :] = torch.tensor(np.asarray(V, np.float32)).to(self.v.dtype).to(self.v.device)

    def read(self, seq: int, layer: int, start: int, end: int):
        """K/V of positions [start, end) as float64 arrays ``[T][H][hd]``."""
        import torch
        blk, slot = self._index(seq, np.arange(start, end))
        bi = torch.tensor(blk, device=self.k.device, dtype=torch.long)
        si = torch.tensor(slot, device=self.k.device, dtype=torch.long)
        return (self.k[layer, bi, :, si, :].double().cpu().numpy(), self.v[layer, bi, :, si, :].double().cpu().numpy())


class Model:
    """Weights resident in HBM plus a context of the C library."""

    def __init__(self, cfg, weights: Dict[str, np.ndarray], *, max_batch: int = 1, max_chunk: int = 16,
                 max_ctx: int = 2048, device: str = "cuda", expert_slots: Optional[int] = None,
                 expert_store=None, expert_source=None):
        """For a mixture-of-experts ``cfg`` the experts live in pinned host
        memory: ``expert_store`` (from pack_expert_store), else one is packed
        from ``expert_source(l, e)`` or, by default, from ``weights``."""
        import torch
        self.cfg = cfg
        self.expert_slots = cfg.n_experts if expert_slots is None else expert_slots
        self.device = device
        self.max_batch, self.max_chunk, self.max_ctx = max_batch, max_chunk, max_ctx
        wdt = torch.bfloat16 if cfg.wdtype == "bf16" else torch.float32
        self._keep = []

        def up(name, dt=wdt):
            t = torch.from_numpy(np.ascontiguousarray(weights[name], dtype=np.float32)).to(device=device, dtype=dt)
            self._keep.append(t)
            return t.data_ptr()

        # projection matrices: m2r2_create packs them into the workspace (for
        # chunks of more than two rows); one- and two-row calls stream these
        # row-major copies, so they live as long as the context
        def up_t(name):
            t = torch.from_numpy(np.ascontiguousarray(weights[name], dtype=np.float32)).to(device=device, dtype=wdt)
            self._keep.append(t)
            return t.data_ptr()

        self._layers = (LayerWeights * cfg.n_layers)()
        for l in range(cfg.n_layers):
            p = f"L{l}."
            L = self._layers[l]
            L.attn_norm = up(p + "attn_norm", torch.float32)
            L.mlp_norm = up(p + "mlp_norm", torch.float32)
            L.wq, L.wk, L.wv, L.wo = up_t(p + "wq"), up_t(p + "wk"), up_t(p + "wv"), up_t(p + "wo")
            if cfg.is_moe:
                L.router = up_t(p + "router")
            else:
                L.wg, L.wu, L.wd = up_t(p + "wg"), up_t(p + "wu"), up_t(p + "wd")
            if p + "A_m" in weights:   # the adapter-only fast MLP (mixture of experts, FLOPs-optimised form)
                L.A_m, L.B_m = up(p + "A_m"), up(p + "B_m")
            for i, pr in enumerate(PROJ):
                if (cfg.is_moe or getattr(cfg, "fast_mlp_adapter", False)) and i >= 4:
                    break
                if p + f"A_{pr}" in weights:
                    L.A[i] = up_t(p + f"A_{pr}") if i < 3 else up(p + f"A_{pr}")
                    L.B[i] = up(p + f"B_{pr}")
        self.expert_store = None
        self.expert_bytes = expert_bytes(cfg) if cfg.is_moe else 0
        if cfg.is_moe:
            if expert_store is None:
                src = expert_source or (lambda l, e: (weights[f"L{l}.E{e}.wg"], weights[f"L{l}.E{e}.wu"],
                                                      weights[f"L{l}.E{e}.wd"]))
                expert_store = pack_expert_store(cfg, src)
            self.expert_store = expert_store
        hr = getattr(cfg, "head_rank", 0)
        self._w = Weights(up("embed"), up("final_norm", torch.float32), up_t("lm_head"), self._layers,
                          None if self.expert_store is None else self.expert_store.data_ptr(),
                          up("head_A") if hr else None, up("head_B") if hr else None)
        self.ws_bytes = workspace_size(cfg, max_batch, max_chunk, max_ctx, self.expert_slots)
        self.workspace = torch.empty(self.ws_bytes + 256, dtype=torch.uint8, device=device)
        base = self.workspace.data_ptr()
        ws_ptr = (base + 255) & ~255
        self._ctx = c_void_p()
        _check(lib().m2r2_create(ctypes.byref(make_config(cfg, self.expert_slots)), ctypes.byref(self._w), max_batch,
                                 max_chunk, max_ctx, ws_ptr, self.ws_bytes, ctypes.byref(self._ctx)), "m2r2_create")
        torch.cuda.synchronize()

    def __del__(self):
        try:
            if getattr(self, "_ctx", None) and self._ctx.value:
                lib().m2r2_destroy(self._ctx)
                self._ctx = c_void_p()
        except Exception:
            pass

    # -- calls ------------------------------------------------------------------
    def decode_step(self, tokens, positions, kv: KV, *, dual: bool = True, gates: Sequence[int] = (),
                    tau: float = 2.0, mode: str = "observe", next_token=None, exit_boundary=None, signal=None,
                    logits=None, h_out=None, p_out=None, advance: bool = False, slow_experts=None,
                    pred_experts=None, stream=None, noalloc: bool = False) -> None:
        """One decode step; ``noalloc`` calls m2r2_decode_step_noalloc (the
        step's scratch in the library's static device array)."""
        g = (c_int32 * max(1, len(gates)))(*gates)
        ex = Exit(ctypes.cast(g, POINTER(c_int32)), len(gates), tau, MODES[mode])
        out = StepOut(_ptr(next_token), _ptr(exit_boundary), _ptr(signal), _ptr(logits), _ptr(h_out), _ptr(p_out),
                      1 if advance else 0, _ptr(slow_experts), _ptr(pred_experts))
        B = tokens.numel()
        fn = lib().m2r2_decode_step_noalloc if noalloc else lib().m2r2_decode_step
        _check(fn(self._ctx, B, 1 if dual else 0, tokens.data_ptr(), positions.data_ptr(), ctypes.byref(kv),
                  ctypes.byref(ex), ctypes.byref(out), _stream(stream)),
               "m2r2_decode_step_noalloc" if noalloc else "m2r2_decode_step")

    def draft(self, last_token, positions, exit_layer: int, gamma: int, kv: KV, drafts, *, stream=None) -> None:
        _check(lib().m2r2_draft(self._ctx, last_token.data_ptr(), positions.data_ptr(), exit_layer, gamma,
                                ctypes.byref(kv), drafts.data_ptr(), _stream(stream)), "m2r2_draft")

    def verify(self, chunk, n: int, positions, kv: KV, targets, n_accepted=None, bonus=None, *, stream=None) -> None:
        _check(lib().m2r2_verify(self._ctx, chunk.data_ptr(), n, positions.data_ptr(), ctypes.byref(kv),
                                 targets.data_ptr(), _ptr(n_accepted), _ptr(bonus), _stream(stream)), "m2r2_verify")

    def timing_enable(self, kernel: Optional[str]) -> None:
        _check(lib().m2r2_timing_enable(self._ctx, -1 if kernel is None else KERNEL_CLASSES[kernel]),
               "m2r2_timing_enable")

    def timing_read(self):
        """(summed kernel milliseconds, launches) of the current record."""
        ms, n = ctypes.c_double(0.0), c_int32(0)
        _check(lib().m2r2_timing_read(self._ctx, ctypes.byref(ms), ctypes.byref(n)), "m2r2_timing_read")
        return ms.value, n.value

    def time_gateup_layers(self, dual: bool = True, *, stream=None) -> float:
        """Average milliseconds of one gate/up launch, the kernel of every
        layer launched back to back between one pair of events (waits)."""
        ms = ctypes.c_double(0.0)
        _check(lib().m2r2_time_gateup_layers(self._ctx, int(bool(dual)), _stream(stream), ctypes.byref(ms)),
               "m2r2_time_gateup_layers")
        return ms.value

    # -- mixture of experts --------------------------------------------------------
    def moe_set_policy(self, policy: str) -> None:
        _check(lib().m2r2_moe_set_policy(self._ctx, POLICIES[policy]), "m2r2_moe_set_policy")

    def prefetch_experts(self, layer: int, ids: Sequence[int], *, priority: bool = False, stream=None) -> None:
        a = (c_int32 * max(1, len(ids)))(*[int(i) for i in ids])
        _check(lib().m2r2_prefetch_experts(self._ctx, layer, ctypes.cast(a, POINTER(c_int32)), len(ids),
                                           1 if priority else 0, None if stream is None else stream.cuda_stream),
               "m2r2_prefetch_experts")

    def moe_reset(self) -> None:
        _check(lib().m2r2_moe_reset(self._ctx), "m2r2_moe_reset")

    def moe_set_preload_table(self, ids: np.ndarray) -> None:
        """Random-preload draws ``[n_tokens][n_layers][top_k]``."""
        a = np.ascontiguousarray(ids, dtype=np.int32)
        if a.ndim != 3 or a.shape[1:] != (self.cfg.n_layers, self.cfg.top_k):
            raise ValueError(f"preload table of shape {a.shape}")
        _check(lib().m2r2_moe_set_preload_table(self._ctx, a.ctypes.data, a.shape[0]), "m2r2_moe_set_preload_table")

    def set_arla(self, weights: Optional[dict]) -> None:
        """Latent-attention exit router (``synth.arla_weights`` layout), or
        None to return to the cosine signal.  The weights are copied to the
        device and kept as long as the model."""
        import torch
        if weights is None:
            _check(lib().m2r2_set_arla(self._ctx, None), "m2r2_set_arla")
            return
        wdt = torch.bfloat16 if self.cfg.wdtype == "bf16" else torch.float32
        ts = {k: torch.from_numpy(np.ascontiguousarray(weights[k], dtype=np.float32)).to(
            device=self.device, dtype=wdt if k in ("wq", "wk", "wv") else torch.float32) for k in
            ("wq", "wk", "wv", "w_out", "b_out")}
        self._arla = ts
        a = Arla(*(ts[k].data_ptr() for k in ("wq", "wk", "wv", "w_out", "b_out")))
        _check(lib().m2r2_set_arla(self._ctx, ctypes.byref(a)), "m2r2_set_arla")

    def moe_stats(self) -> dict:
        out = MoeCounters()
        _check(lib().m2r2_moe_stats(self._ctx, ctypes.byref(out)), "m2r2_moe_stats")
        return out.as_dict(self.cfg.n_layers)

    def sync_check(self, stream=None) -> None:
        """Raise M2R2Error if the enqueued work failed or set a device error bit."""
        _check(lib().m2r2_sync_check(self._ctx, _stream(stream)), "m2r2_sync_check")

    def device_errors(self, stream=None) -> int:
        bits = c_int32(0)
        _check(lib().m2r2_device_errors(self._ctx, _stream(stream), ctypes.byref(bits)), "m2r2_device_errors")
        return bits.value
