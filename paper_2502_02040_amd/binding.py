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

EXPORTS = ("m2r2_workspace_size", "m2r2_create", "m2r2_destroy", "m2r2_decode_step", "m2r2_draft", "m2r2_verify",
           "m2r2_timing_enable", "m2r2_timing_read", "m2r2_device_errors", "m2r2_last_error")
KERNEL_CLASSES = {"qkv": 0, "attn": 1, "oproj": 2, "gateup": 3, "down": 4, "head": 5, "embed": 6, "attn_merge": 7}


class Config(ctypes.Structure):
    _fields_ = [("n_layers", c_int32), ("d_model", c_int32), ("n_heads", c_int32), ("head_dim", c_int32),
                ("ffn", c_int32), ("vocab", c_int32), ("rank", c_int32), ("wdtype", c_int32), ("kvdtype", c_int32),
                ("rms_eps", c_float), ("rope_theta", c_float)]


class LayerWeights(ctypes.Structure):
    _fields_ = [("attn_norm", c_void_p), ("wq", c_void_p), ("wk", c_void_p), ("wv", c_void_p), ("wo", c_void_p),
                ("mlp_norm", c_void_p), ("wg", c_void_p), ("wu", c_void_p), ("wd", c_void_p),
                ("A", c_void_p * 7), ("B", c_void_p * 7)]


class Weights(ctypes.Structure):
    _fields_ = [("embed", c_void_p), ("final_norm", c_void_p), ("lm_head", c_void_p),
                ("layers", POINTER(LayerWeights))]


class KV(ctypes.Structure):
    _fields_ = [("k_pages", c_void_p), ("v_pages", c_void_p), ("block_table_d", c_void_p), ("seq_lens_d", c_void_p),
                ("num_blocks", c_int32), ("block_size", c_int32), ("max_blocks_per_seq", c_int32)]


class Exit(ctypes.Structure):
    _fields_ = [("gates_h", POINTER(c_int32)), ("n_gates", c_int32), ("tau", c_float), ("mode", c_int32)]


class StepOut(ctypes.Structure):
    _fields_ = [("next_token_d", c_void_p), ("exit_boundary_d", c_void_p), ("signal_d", c_void_p),
                ("logits_d", c_void_p), ("h_out_d", c_void_p), ("p_out_d", c_void_p), ("advance", c_int32)]


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
        L.m2r2_draft.argtypes = [c_void_p, c_void_p, c_void_p, c_int32, c_int32, POINTER(KV), c_void_p, c_void_p]
        L.m2r2_verify.argtypes = [c_void_p, c_void_p, c_int32, c_void_p, POINTER(KV), c_void_p, c_void_p, c_void_p,
                                  c_void_p]
        L.m2r2_timing_enable.argtypes = [c_void_p, c_int32]
        L.m2r2_timing_read.argtypes = [c_void_p, POINTER(ctypes.c_double), POINTER(c_int32)]
        L.m2r2_device_errors.argtypes = [c_void_p, c_void_p, POINTER(c_int32)]
        L.m2r2_last_error.restype = ctypes.c_char_p
        for f in ("m2r2_workspace_size", "m2r2_create", "m2r2_decode_step", "m2r2_draft", "m2r2_verify",
                  "m2r2_timing_enable", "m2r2_timing_read", "m2r2_device_errors"):
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


def make_config(cfg) -> Config:
    return Config(cfg.n_layers, cfg.d_model, cfg.n_heads, cfg.head_dim, cfg.ffn, cfg.vocab, cfg.rank,
                  BF16 if cfg.wdtype == "bf16" else F32, BF16 if cfg.kvdtype == "bf16" else F32,
                  cfg.rms_eps, cfg.rope_theta)


def workspace_size(cfg, max_batch: int, max_chunk: int, max_ctx: int) -> int:
    n = c_size_t(0)
    _check(lib().m2r2_workspace_size(ctypes.byref(make_config(cfg)), max_batch, max_chunk, max_ctx, ctypes.byref(n)),
           "m2r2_workspace_size")
    return n.value


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
                 max_ctx: int = 2048, device: str = "cuda"):
        import torch
        self.cfg = cfg
        self.device = device
        self.max_batch, self.max_chunk, self.max_ctx = max_batch, max_chunk, max_ctx
        wdt = torch.bfloat16 if cfg.wdtype == "bf16" else torch.float32
        self._keep = []

        def up(name, dt=wdt):
            t = torch.from_numpy(np.ascontiguousarray(weights[name], dtype=np.float32)).to(device=device, dtype=dt)
            self._keep.append(t)
            return t.data_ptr()

        # projection matrices (and the q/k/v adapter-down factors) are read by
        # m2r2_create only: it packs them into the workspace
        self._transient = []

        def up_t(name):
            t = torch.from_numpy(np.ascontiguousarray(weights[name], dtype=np.float32)).to(device=device, dtype=wdt)
            self._transient.append(t)
            return t.data_ptr()

        self._layers = (LayerWeights * cfg.n_layers)()
        for l in range(cfg.n_layers):
            p = f"L{l}."
            L = self._layers[l]
            L.attn_norm = up(p + "attn_norm", torch.float32)
            L.mlp_norm = up(p + "mlp_norm", torch.float32)
            L.wq, L.wk, L.wv, L.wo = up_t(p + "wq"), up_t(p + "wk"), up_t(p + "wv"), up_t(p + "wo")
            L.wg, L.wu, L.wd = up_t(p + "wg"), up_t(p + "wu"), up_t(p + "wd")
            for i, pr in enumerate(PROJ):
                if p + f"A_{pr}" in weights:
                    L.A[i] = up_t(p + f"A_{pr}") if i < 3 else up(p + f"A_{pr}")
                    L.B[i] = up(p + f"B_{pr}")
        self._w = Weights(up("embed"), up("final_norm", torch.float32), up_t("lm_head"), self._layers)
        self.ws_bytes = workspace_size(cfg, max_batch, max_chunk, max_ctx)
        self.workspace = torch.empty(self.ws_bytes + 256, dtype=torch.uint8, device=device)
        base = self.workspace.data_ptr()
        ws_ptr = (base + 255) & ~255
        self._ctx = c_void_p()
        _check(lib().m2r2_create(ctypes.byref(make_config(cfg)), ctypes.byref(self._w), max_batch, max_chunk, max_ctx,
                                 ws_ptr, self.ws_bytes, ctypes.byref(self._ctx)), "m2r2_create")
        torch.cuda.synchronize()
        self._transient = []   # packed copies live in the workspace

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
                    logits=None, h_out=None, p_out=None, advance: bool = False, stream=None) -> None:
        g = (c_int32 * max(1, len(gates)))(*gates)
        ex = Exit(ctypes.cast(g, POINTER(c_int32)), len(gates), tau, MODES[mode])
        out = StepOut(_ptr(next_token), _ptr(exit_boundary), _ptr(signal), _ptr(logits), _ptr(h_out), _ptr(p_out),
                      1 if advance else 0)
        B = tokens.numel()
        _check(lib().m2r2_decode_step(self._ctx, B, 1 if dual else 0, tokens.data_ptr(), positions.data_ptr(),
                                      ctypes.byref(kv), ctypes.byref(ex), ctypes.byref(out), _stream(stream)),
               "m2r2_decode_step")

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

    def device_errors(self, stream=None) -> int:
        bits = c_int32(0)
        _check(lib().m2r2_device_errors(self._ctx, _stream(stream), ctypes.byref(bits)), "m2r2_device_errors")
        return bits.value
