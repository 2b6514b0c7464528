"""Plain NumPy statement of the M2R2 decode path.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Notation follows the paper: ``h`` is the slow residual stream, ``p`` the
accelerated residual stream, layers are 0-indexed and gate boundary ``b``
sits after layer ``b-1``.

Readings of the paper taken here (each one is also listed with its
justification in the design notes of the repository):
  * Slow stream (Eq. 1) is a pre-norm decoder layer with RMSNorm (the paper
    omits normalisation, footnote to Eq. 1), rotate-half RoPE, scaled
    dot-product attention with H_kv = H, and a SwiGLU MLP.
  * Accelerated stream (Eq. 2, Sec. 2.2): the same base layer plus linear
    rank-r adapters ``(x A^T) B^T`` added to every projection (q, k, v, o,
    gate, up, down) with scale 1; the MLP acts on ``p + A_hat(p)`` as the body
    of Eq. 2 writes (the ``g(h_i)`` in its where-clause is read as a typo).
    For MoE models the fast MLP is the adapter alone (Sec. 2.3.3).
  * Shared KV cache (Sec. 2.2): the fast query attends to the slow cache for
    positions < t plus its own key/value at t; the fast stream never writes the
    cache.  Values read back from a cache are rounded to the cache precision.
  * ``p <- h`` at the start of the pass and at every gate (Fig. 3 caption).
  * Exit signal: cosine between the fast state entering and leaving a layer
    (the directional shift of Sec. 2.1 applied to the fast stream), standing in
    for the trained ARLA router; exit iff signal >= tau at a gate.
  * When a token exits at gate b (Eq. 4), its token comes from the final norm
    and LM head applied to ``p`` at the gate, and the skipped layers' cache
    entries at t are projected from the slow ``h`` at the gate.
  * FLOPs-optimised fast stream (Sec. 2.5), for dense models whose config
    sets it: the fast row keeps only the first ``fast_heads`` heads (q, k, v
    and the o input of the others are zero); fast head j attends to the
    ``fast_topk`` cached positions with the largest scores of the slow row's
    head j at the same layer (all positions when there are no more than
    that; ties to the lower position), plus its own key/value; its MLP is the
    rank-r adapter ``m`` alone, as for MoE layers; a token it emits comes
    from the final norm and a rank-``head_rank`` head ``head_A``, ``head_B``.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

MODES = ("off", "observe", "exit")


# ----------------------------------------------------------------------------
# Elementary operations (each the textbook definition)
# ----------------------------------------------------------------------------

def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm along the last axis: x / sqrt(mean(x^2) + eps) * g."""
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * g


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def rope(x: np.ndarray, pos, theta: float) -> np.ndarray:
    """Rotate-half rotary embedding of ``x[..., H, hd]`` at position(s) ``pos``.

    Pair (i, i + hd/2) of each head is rotated by angle ``pos * theta^(-2i/hd)``.
    ``pos`` is a scalar or an array broadcastable to ``x.shape[:-2]``.
    """
    hd = x.shape[-1]
    half = hd // 2
    inv = theta ** (-(2.0 * np.arange(half, dtype=np.float64)) / hd)
    ang = np.asarray(pos, dtype=np.float64)[..., None, None] * inv  # [..., 1, half]
    c, s = np.cos(ang).astype(x.dtype), np.sin(ang).astype(x.dtype)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def attend(q: np.ndarray, K: np.ndarray, V: np.ndarray) -> np.ndarray:
    """Single-query multi-head attention: q [H, hd], K/V [T, H, hd] -> [H, hd]."""
    hd = q.shape[-1]
    s = np.einsum("hd,thd->ht", q, K) / math.sqrt(hd)   # a Python float keeps q's precision
    s = s - s.max(axis=-1, keepdims=True)
    w = np.exp(s)
    w = w / w.sum(axis=-1, keepdims=True)
    return np.einsum("ht,thd->hd", w, V)


def topk_desc(v: np.ndarray, k: int) -> np.ndarray:
    """Indices of the k largest entries, by descending value, ties to the lower index."""
    order = np.lexsort((np.arange(v.shape[-1]), -v))
    return order[:k]


def select_top(scores: np.ndarray, k: int) -> np.ndarray:
    """Positions of the ``k`` largest scores in increasing position order
    (every position when there are no more than ``k``; ``k <= 0``: all)."""
    n = scores.shape[0]
    if k <= 0 or n <= k:
        return np.arange(n)
    return np.sort(topk_desc(scores, k))


def top_gap(scores: np.ndarray, k: int) -> float:
    """Distance between the k-th and the (k+1)-th largest score: how far the
    selection of ``select_top`` is from a tie (inf when it takes everything)."""
    n = scores.shape[0]
    if k <= 0 or n <= k:
        return math.inf
    srt = np.sort(scores)[::-1]
    return float(srt[k - 1] - srt[k])


def argmax_first(v: np.ndarray) -> int:
    """Index of the maximum, lowest index on ties."""
    return int(np.argmax(v))


def round_to_cache(x: np.ndarray, kvdtype: str) -> np.ndarray:
    """Value of ``x`` once stored in the cache precision, returned in x's dtype.

    bf16: nearest value with 8 significant bits, ties to even (computed with
    frexp/rint so that float64 inputs round once).  f32: nearest float32.
    f64: unchanged (used by tests that need exact identities).
    """
    if kvdtype == "f64":
        return x.copy()
    if kvdtype == "f32":
        return x.astype(np.float32).astype(x.dtype)
    if kvdtype == "bf16":
        m, e = np.frexp(x)
        return np.ldexp(np.rint(np.ldexp(m, 8)), e - 8).astype(x.dtype)
    raise ValueError(kvdtype)


ARLA_DIM = 64   # latent width of the exit router (the value the paper uses)


def arla_score(wq: np.ndarray, wk: np.ndarray, wv: np.ndarray, w_out: np.ndarray, b_out: float,
               states: Sequence[np.ndarray], eps: float) -> float:
    """Exit probability of the accelerated-residual latent-attention router
    (Sec. 2.3.1, ARLA; Fig. 4a) at a gate.

    ``states`` are the fast residuals of the interval that ends at the gate,
    oldest first: the state the fast stream restarts from at the previous
    gate, then the state after each layer up to the gate.  Each is
    RMS-normalised without a gain, then projected to the latent space
    (``wk``, ``wv``: [64, d]).  Every state has a query too, but the decision
    is one probability taken at the gate, so attention runs causally over the
    interval and only the output at its newest state is read: the query is
    the projection (``wq``) of the last state, its softmax attention (scale
    1/sqrt(64)) pools the values, and a linear readout with a sigmoid gives
    the probability.  (The paper does not fix the pooling, the normalisation
    or the readout; these are the readings used throughout.)
    """
    U = [x / np.sqrt(np.mean(x * x) + eps) for x in states]
    q = wq @ U[-1]
    K = np.stack([wk @ u for u in U])
    V = np.stack([wv @ u for u in U])
    z = K @ q / np.sqrt(ARLA_DIM)
    a = np.exp(z - z.max())
    a = a / a.sum()
    o = a @ V
    return float(1.0 / (1.0 + np.exp(-(w_out @ o + b_out))))


def cosine(a: np.ndarray, b: np.ndarray) -> float:
    return float(np.dot(a, b) / (np.linalg.norm(a) * np.linalg.norm(b)))


# ----------------------------------------------------------------------------
# Cache
# ----------------------------------------------------------------------------

class KVCache:
    """Slow-stream KV cache of one sequence: per layer K, V ``[T_max, H, hd]``."""

    def __init__(self, cfg, max_len: int, dtype=np.float64):
        self.cfg = cfg
        self.K = [np.zeros((max_len, cfg.n_heads, cfg.head_dim), dtype) for _ in range(cfg.n_layers)]
        self.V = [np.zeros((max_len, cfg.n_heads, cfg.head_dim), dtype) for _ in range(cfg.n_layers)]

    def write(self, l: int, pos, k: np.ndarray, v: np.ndarray) -> None:
        self.K[l][pos] = round_to_cache(k, self.cfg.kvdtype)
        self.V[l][pos] = round_to_cache(v, self.cfg.kvdtype)

    def load(self, l: int, K: np.ndarray, V: np.ndarray, start: int = 0) -> None:
        """Place given cache content (already in cache precision) at [start, start+len)."""
        n = K.shape[0]
        self.K[l][start:start + n] = K
        self.V[l][start:start + n] = V


@dataclasses.dataclass
class StepResult:
    token: int
    logits: np.ndarray
    exit_boundary: int
    signal: np.ndarray          # [N] cos(p_in, p_out) per layer (nan where not computed)
    h: np.ndarray               # slow state fed to the head (final layer, or gate on exit)
    p: np.ndarray               # fast state at the end (gate state on exit)
    slow_experts: Optional[np.ndarray] = None   # [N, K] (MoE)
    slow_probs: Optional[np.ndarray] = None     # [N, E] router probabilities (MoE)
    pred_experts: Optional[np.ndarray] = None   # [N, K], -1 where no prediction (MoE)
    pred_logits: Optional[np.ndarray] = None    # [N, E] fast-router logits (MoE)
    prev_pred_experts: Optional[np.ndarray] = None   # [N, K] layer l's top-k from the slow row entering layer l-1's MLP
    prev_pred_logits: Optional[np.ndarray] = None    # [N, E] the logits behind prev_pred_experts
    fast_states: Optional[np.ndarray] = None    # [N, d] p after each layer (before a gate's restart), nan if not run
    router_logits: Optional[np.ndarray] = None  # [N, E] slow-router logits (MoE)
    topk_gap: Optional[np.ndarray] = None       # [N, H] FLOPs mode: top_gap of each fast head's selection (inf: none)


# ----------------------------------------------------------------------------
# The decoder
# ----------------------------------------------------------------------------

class Oracle:
    """Reference decoder over a weight dictionary produced by ``synth``."""

    def __init__(self, cfg, weights: Dict[str, np.ndarray], dtype=np.float64):
        self.cfg = cfg
        self.dtype = dtype
        self.w = {k: np.asarray(v, dtype=dtype) for k, v in weights.items()}

    # -- pieces ---------------------------------------------------------------
    def _W(self, l: int, name: str) -> np.ndarray:
        return self.w[f"L{l}.{name}"]

    def _adapter(self, l: int, proj: str, x: np.ndarray) -> np.ndarray:
        """Rank-r accelerator adapter (x A^T) B^T of one projection."""
        return (x @ self._W(l, f"A_{proj}").T) @ self._W(l, f"B_{proj}").T

    def _qkv(self, l: int, x: np.ndarray, pos, fast: bool):
        """Projections of the normed input ``x`` ([..., d]) to roped q, k and v ([..., H, hd])."""
        cfg = self.cfg
        u = rms_norm(x, self._W(l, "attn_norm"), cfg.rms_eps)
        q = u @ self._W(l, "wq").T
        k = u @ self._W(l, "wk").T
        v = u @ self._W(l, "wv").T
        if fast:
            q = q + self._adapter(l, "q", u)
            k = k + self._adapter(l, "k", u)
            v = v + self._adapter(l, "v", u)
        shp = x.shape[:-1] + (cfg.n_heads, cfg.head_dim)
        q, k, v = q.reshape(shp), k.reshape(shp), v.reshape(shp)
        return rope(q, pos, cfg.rope_theta), rope(k, pos, cfg.rope_theta), v

    def _attn_out(self, l: int, o: np.ndarray, fast: bool) -> np.ndarray:
        o = o.reshape(o.shape[:-2] + (-1,))
        y = o @ self._W(l, "wo").T
        if fast:
            y = y + self._adapter(l, "o", o)
        return y

    def _dense_mlp(self, l: int, x: np.ndarray, fast: bool) -> np.ndarray:
        m = rms_norm(x, self._W(l, "mlp_norm"), self.cfg.rms_eps)
        g = m @ self._W(l, "wg").T
        u = m @ self._W(l, "wu").T
        if fast:
            g = g + self._adapter(l, "g", m)
            u = u + self._adapter(l, "u", m)
        a = silu(g) * u
        y = a @ self._W(l, "wd").T
        if fast:
            y = y + self._adapter(l, "d", a)
        return y

    def router_logits(self, l: int, x: np.ndarray) -> np.ndarray:
        """Router logits of layer l for residual ``x`` (router input = mlp-normed x)."""
        m = rms_norm(x, self._W(l, "mlp_norm"), self.cfg.rms_eps)
        return m @ self._W(l, "router").T

    def _moe_mlp(self, l: int, x: np.ndarray):
        """Slow-stream MoE MLP for one row: softmax over all experts, top-k,
        combine with the unrenormalised probabilities."""
        cfg = self.cfg
        m = rms_norm(x, self._W(l, "mlp_norm"), cfg.rms_eps)
        z = m @ self._W(l, "router").T
        pz = np.exp(z - z.max())
        pz = pz / pz.sum()
        S = topk_desc(pz, cfg.top_k)
        y = np.zeros_like(x)
        for e in S:
            g = m @ self._W(l, f"E{e}.wg").T
            u = m @ self._W(l, f"E{e}.wu").T
            y = y + pz[e] * ((silu(g) * u) @ self._W(l, f"E{e}.wd").T)
        return y, S, pz, z

    def _fast_moe_mlp(self, l: int, x: np.ndarray) -> np.ndarray:
        """Fast-stream MLP of an MoE layer (or of a dense layer in the FLOPs-
        optimised form): the rank-r adapter alone."""
        m = rms_norm(x, self._W(l, "mlp_norm"), self.cfg.rms_eps)
        return self._adapter(l, "m", m)

    def head_logits(self, x: np.ndarray) -> np.ndarray:
        return rms_norm(x, self.w["final_norm"], self.cfg.rms_eps) @ self.w["lm_head"].T

    def fast_head_logits(self, x: np.ndarray) -> np.ndarray:
        """Logits of a token the fast row emits: the low-rank head of the
        FLOPs-optimised form when the config has one, else the LM head."""
        if not self.cfg.head_rank:
            return self.head_logits(x)
        u = rms_norm(x, self.w["final_norm"], self.cfg.rms_eps)
        return (u @ self.w["head_A"].T) @ self.w["head_B"].T

    # -- one layer, one position, slow row --------------------------------------
    def _slow_layer(self, l: int, h: np.ndarray, pos: int, cache: KVCache, moe_out=None) -> np.ndarray:
        q, k, v = self._qkv(l, h, pos, fast=False)
        cache.write(l, pos, k, v)
        o = attend(q, cache.K[l][:pos + 1], cache.V[l][:pos + 1])
        h1 = h + self._attn_out(l, o, fast=False)
        if self.cfg.is_moe:
            y, S, pz, z = self._moe_mlp(l, h1)
            if moe_out is not None:
                moe_out.append((S, pz, z, h1))
            return h1 + y
        return h1 + self._dense_mlp(l, h1, fast=False)

    # -- one layer, one position, fast row ---------------------------------------
    def _fast_layer(self, l: int, p: np.ndarray, pos: int, ctxK: np.ndarray, ctxV: np.ndarray):
        """Fast row of layer l at position ``pos`` attending to the context
        ``ctxK/ctxV`` (positions < pos, cache precision) plus its own k/v.
        Returns the new p and the row's own (k, v) before any rounding."""
        q, k, v = self._qkv(l, p, pos, fast=True)
        K = np.concatenate([ctxK, k[None]], axis=0)
        V = np.concatenate([ctxV, v[None]], axis=0)
        o = attend(q, K, V)
        p1 = p + self._attn_out(l, o, fast=True)
        if self.cfg.is_moe:
            return p1 + self._fast_moe_mlp(l, p1), (k, v)
        return p1 + self._dense_mlp(l, p1, fast=True), (k, v)

    def _fast_layer_flops(self, l: int, p: np.ndarray, h: np.ndarray, pos: int, ctxK: np.ndarray,
                          ctxV: np.ndarray):
        """Fast row of layer l in the FLOPs-optimised form (Sec. 2.5).  The
        slow row's query of the same layer (from ``h``, the slow state
        entering it) scores the cached context; fast head j < fast_heads
        attends to the positions ``select_top`` keeps for slow head j plus its
        own key/value; the other heads contribute nothing.  Returns the new p
        and the selection gaps of the heads [H]."""
        cfg = self.cfg
        nh = cfg.fast_heads or cfg.n_heads
        qs, _, _ = self._qkv(l, h, pos, fast=False)
        q, k, v = self._qkv(l, p, pos, fast=True)
        o = np.zeros_like(q)
        gaps = np.full(cfg.n_heads, math.inf)
        for j in range(nh):
            s = ctxK[:, j] @ qs[j] / math.sqrt(cfg.head_dim)
            sel = select_top(s, cfg.fast_topk)
            gaps[j] = top_gap(s, cfg.fast_topk)
            Kj = np.concatenate([ctxK[sel, j], k[j][None]], axis=0)
            Vj = np.concatenate([ctxV[sel, j], v[j][None]], axis=0)
            o[j] = attend(q[j][None], Kj[:, None], Vj[:, None])[0]
        p1 = p + self._attn_out(l, o, fast=True)
        if cfg.fast_mlp_adapter:
            return p1 + self._fast_moe_mlp(l, p1), gaps
        return p1 + self._dense_mlp(l, p1, fast=True), gaps

    def _kv_fill(self, l: int, h: np.ndarray, pos: int, cache: KVCache) -> None:
        """Cache entry of a skipped layer: projected from the slow state at the gate."""
        _, k, v = self._qkv(l, h, pos, fast=False)
        cache.write(l, pos, k, v)

    # -- the dual-stream decode step -------------------------------------------------
    def decode_step(self, token: int, pos: int, cache: KVCache, *, gates: Sequence[int] = (),
                    tau: float = 2.0, mode: str = "observe", arla: Optional[Dict[str, np.ndarray]] = None
                    ) -> StepResult:
        """One decode step carrying the slow row ``h`` and the fast row ``p``.

        ``gates`` are boundaries b in [1, N-1]; at a gate the signal of layer
        b-1 is compared with ``tau``: the first gate with signal >= tau is
        recorded as the exit boundary; in ``exit`` mode the step stops there,
        otherwise (and whenever the test fails) ``p`` restarts from ``h``.

        With ``arla`` (arrays ``wq``, ``wk``, ``wv`` [N, 64, d], ``w_out``
        [N, 64], ``b_out`` [N]; block b belongs to boundary b) the signal at a
        gate b is ``arla_score`` over the interval from the previous gate g
        (or the start, g = 0) to b instead of the cosine of layer b-1: the
        state p restarts from at g (h there; the embedding for g = 0), then
        p after each of the layers g .. b-1.
        """
        cfg = self.cfg
        assert mode in MODES
        N = cfg.n_layers
        gates = set(int(b) for b in gates)
        h = self.w["embed"][token].copy()
        p = h.copy()
        signal = np.full(N, np.nan)
        exit_b = N
        moe_rec: List = []
        pred = np.full((N, max(cfg.top_k, 1)), -1, np.int64)
        pred_logits = np.full((N, max(cfg.n_experts, 1)), np.nan)
        self._fast_states = np.full((N, cfg.d_model), np.nan)
        self._topk_gap = np.full((N, cfg.n_heads), np.inf) if cfg.is_flops else None
        # the gate's interval: the state p (re)starts from, then p after each layer
        interval: List[np.ndarray] = [h.copy()]
        for l in range(N):
            p_in = p
            # fast row first: it sees the cache before the slow row writes position pos
            if cfg.is_flops:
                assert not cfg.is_moe, "the FLOPs-optimised form is defined here for dense models"
                p, self._topk_gap[l] = self._fast_layer_flops(l, p, h, pos, cache.K[l][:pos], cache.V[l][:pos])
            else:
                p, _ = self._fast_layer(l, p, pos, cache.K[l][:pos], cache.V[l][:pos])
            h = self._slow_layer(l, h, pos, cache, moe_rec)
            self._fast_states[l] = p
            interval.append(p)
            signal[l] = cosine(p_in, p)
            if arla is not None and mode != "off" and (l + 1) in gates:
                b = l + 1
                signal[l] = arla_score(arla["wq"][b], arla["wk"][b], arla["wv"][b], arla["w_out"][b],
                                       float(arla["b_out"][b]), interval, cfg.rms_eps)
            if cfg.is_moe:
                for lp in (2 * l + 2, 2 * l + 3):
                    if lp < N:
                        z = self.router_logits(lp, p)
                        pred_logits[lp] = z
                        pred[lp] = topk_desc(z, cfg.top_k)
            b = l + 1
            if b in gates:
                interval = [h.copy()]   # p restarts from h at the gate (when the step goes on)
            if mode != "off" and b in gates:
                fired = signal[l] >= tau
                if fired and exit_b == N:
                    exit_b = b
                if mode == "exit" and fired:
                    for l2 in range(b, N):
                        self._kv_fill(l2, h, pos, cache)
                    logits = self.fast_head_logits(p)
                    return self._result(logits, exit_b, signal, h, p, moe_rec, pred, pred_logits)
                p = h.copy()
        logits = self.head_logits(h)
        return self._result(logits, exit_b, signal, h, p, moe_rec, pred, pred_logits)

    def _result(self, logits, exit_b, signal, h, p, moe_rec, pred, pred_logits) -> StepResult:
        cfg = self.cfg
        r = StepResult(token=argmax_first(logits), logits=logits, exit_boundary=exit_b, signal=signal, h=h, p=p,
                       fast_states=self._fast_states, topk_gap=self._topk_gap)
        if cfg.is_moe:
            n = len(moe_rec)
            r.slow_experts = np.array([m[0] for m in moe_rec]).reshape(n, cfg.top_k)
            r.slow_probs = np.array([m[1] for m in moe_rec]).reshape(n, cfg.n_experts)
            r.router_logits = np.array([m[2] for m in moe_rec]).reshape(n, cfg.n_experts)
            r.pred_experts = pred
            r.pred_logits = pred_logits
            # speculation from the previous layer's residual state (the comparison
            # strategy of Sec. 3.3): layer l+1's router on the slow row that enters
            # layer l's MLP
            N = cfg.n_layers
            r.prev_pred_experts = np.full((N, cfg.top_k), -1, np.int64)
            r.prev_pred_logits = np.full((N, cfg.n_experts), np.nan)
            for l in range(n):
                if l + 1 < N:
                    z = self.router_logits(l + 1, moe_rec[l][3])
                    r.prev_pred_logits[l + 1] = z
                    r.prev_pred_experts[l + 1] = topk_desc(z, cfg.top_k)
        return r

    # -- slow-only chunk forward (prefill and verification) ------------------------------
    def slow_chunk(self, tokens: Sequence[int], pos0: int, cache: KVCache, *, record_moe=None) -> np.ndarray:
        """Slow stream over ``tokens`` at positions pos0.. (causal); writes
        their cache entries and returns the logits of every row ``[n, V]``."""
        cfg = self.cfg
        n = len(tokens)
        H = self.w["embed"][np.asarray(tokens)].copy()
        pos = pos0 + np.arange(n)
        for l in range(cfg.n_layers):
            q, k, v = self._qkv(l, H, pos, fast=False)
            cache.write(l, slice(pos0, pos0 + n), k, v)
            o = np.stack([attend(q[i], cache.K[l][:pos0 + i + 1], cache.V[l][:pos0 + i + 1]) for i in range(n)])
            H1 = H + self._attn_out(l, o, fast=False)
            if cfg.is_moe:
                Y = np.zeros_like(H1)
                for i in range(n):
                    y, S, pz, z = self._moe_mlp(l, H1[i])
                    Y[i] = y
                    if record_moe is not None:
                        record_moe.append((i, l, S))
                H = H1 + Y
            else:
                H = H1 + self._dense_mlp(l, H1, fast=False)
        return self.head_logits(H)

    # -- fast-only draft ------------------------------------------------------------------
    def draft(self, token: int, pos: int, cache: KVCache, exit_layer: int, gamma: int) -> List[int]:
        """Greedy draft of ``gamma`` tokens from the fast row run through layers
        0..exit_layer-1 (fast stream at rate N/exit_layer).  The fast k/v of
        earlier draft positions are kept, in cache precision, in a scratch area
        that later drafts attend to; the slow cache is not modified."""
        cfg = self.cfg
        if cfg.is_flops:
            raise ValueError("a fast-only draft has no slow-row scores: the FLOPs-optimised form is the "
                             "dual-stream step's")
        scK = [np.zeros((gamma, cfg.n_heads, cfg.head_dim), self.dtype) for _ in range(exit_layer)]
        scV = [np.zeros((gamma, cfg.n_heads, cfg.head_dim), self.dtype) for _ in range(exit_layer)]
        out = []
        tok = token
        for j in range(gamma):
            p = self.w["embed"][tok].copy()
            for l in range(exit_layer):
                ctxK = np.concatenate([cache.K[l][:pos], scK[l][:j]], axis=0)
                ctxV = np.concatenate([cache.V[l][:pos], scV[l][:j]], axis=0)
                p, (k, v) = self._fast_layer(l, p, pos + j, ctxK, ctxV)
                scK[l][j] = round_to_cache(k, cfg.kvdtype)
                scV[l][j] = round_to_cache(v, cfg.kvdtype)
            tok = argmax_first(self.head_logits(p))
            out.append(tok)
        return out

    # -- generation loops -------------------------------------------------------------------
    def greedy(self, prompt: Sequence[int], n_new: int, *, max_len: Optional[int] = None) -> List[int]:
        """Plain greedy decoding on the slow stream: ``n_new`` generated ids."""
        max_len = max_len or (len(prompt) + n_new + 1)
        cache = KVCache(self.cfg, max_len, self.dtype)
        logits = self.slow_chunk(prompt, 0, cache)
        out = [argmax_first(logits[-1])]
        pos = len(prompt)
        while len(out) < n_new:
            logits = self.slow_chunk([out[-1]], pos, cache)
            out.append(argmax_first(logits[-1]))
            pos += 1
        return out

    def spec_generate(self, prompt: Sequence[int], n_new: int, *, gamma: int, exit_layer: int,
                      corrupt_drafts: bool = False, max_len: Optional[int] = None):
        """Self-speculative greedy decoding: draft ``gamma`` tokens from the
        fast stream exiting at ``exit_layer``, verify them in one slow chunk,
        keep the longest matching prefix plus the verifier's next token.

        Returns ``(tokens, stats)`` with stats = dict(rounds, drafted, accepted).
        ``corrupt_drafts`` replaces every draft by (draft + 1) mod V so that
        none can be accepted (exercises the rejection path)."""
        cfg = self.cfg
        max_len = max_len or (len(prompt) + n_new + gamma + 2)
        cache = KVCache(cfg, max_len, self.dtype)
        logits = self.slow_chunk(prompt, 0, cache)
        out = [argmax_first(logits[-1])]
        pos = len(prompt)          # position of out[-1], whose cache entry is not written yet
        rounds = drafted = accepted = 0
        while len(out) < n_new:
            d = self.draft(out[-1], pos, cache, exit_layer, gamma)
            if corrupt_drafts:
                d = [(x + 1) % cfg.vocab for x in d]
            logits = self.slow_chunk([out[-1]] + d, pos, cache)
            y = [argmax_first(z) for z in logits]
            n = 0
            while n < gamma and d[n] == y[n]:
                n += 1
            new = d[:n] + [y[n]]
            rounds += 1
            drafted += gamma
            accepted += n
            out.extend(new)
            pos += n + 1
        return out[:n_new], dict(rounds=rounds, drafted=drafted, accepted=accepted)
