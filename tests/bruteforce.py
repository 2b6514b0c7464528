"""Scalar-loop restatement of one decode step, for tiny shapes only.

Written independently of ``oracle/`` (plain Python floats and loops, the
``math`` module, no NumPy linear algebra) so that a wiring mistake in the
vectorised oracle (a transposed weight, a wrong head slice, a RoPE pair index,
an adapter on the wrong projection, the wrong keys for the fast query) shows
up as a mismatch.  It follows the paper's equations directly: Eq. 1 for the
slow row, Eq. 2 with low-rank adapters for the fast row, the shared KV cache
of Sec. 2.2, re-initialisation at gates (Fig. 3 caption) and the exit of Eq. 4,
and the FLOPs-optimised fast stream of Sec. 2.5 (pruned heads, a context
chosen by sorting the slow row's scores, the adapter-only MLP and the
low-rank head).
"""
from __future__ import annotations

import math
from typing import Dict, List, Sequence

import numpy as np


def _f(a) -> List:
    """Nested Python lists of floats."""
    return np.asarray(a, dtype=np.float64).tolist()


def mv(W: List[List[float]], x: List[float]) -> List[float]:
    out = []
    for row in W:
        s = 0.0
        for j in range(len(x)):
            s += row[j] * x[j]
        out.append(s)
    return out


def add(a, b):
    return [a[i] + b[i] for i in range(len(a))]


def rms(x, g, eps):
    ms = 0.0
    for v in x:
        ms += v * v
    ms /= len(x)
    inv = 1.0 / math.sqrt(ms + eps)
    return [x[i] * inv * g[i] for i in range(len(x))]


def rot(vec, pos, H, hd, theta):
    out = list(vec)
    half = hd // 2
    for hh in range(H):
        base = hh * hd
        for i in range(half):
            ang = pos * theta ** (-2.0 * i / hd)
            c, s = math.cos(ang), math.sin(ang)
            a, b = vec[base + i], vec[base + half + i]
            out[base + i] = a * c - b * s
            out[base + half + i] = b * c + a * s
    return out


def mha(q, keys, vals, H, hd):
    """q: flat [H*hd]; keys/vals: lists of flat [H*hd] rows."""
    out = [0.0] * (H * hd)
    for hh in range(H):
        sl = range(hh * hd, (hh + 1) * hd)
        sc = []
        for k in keys:
            s = 0.0
            for d in sl:
                s += q[d] * k[d]
            sc.append(s / math.sqrt(hd))
        mx = max(sc)
        e = [math.exp(s - mx) for s in sc]
        tot = sum(e)
        for j, v in enumerate(vals):
            wgt = e[j] / tot
            for d in sl:
                out[d] += wgt * v[d]
    return out


def one_head(q, keys, vals, hh, hd):
    """Attention of head hh alone over the given rows: its hd outputs."""
    sl = range(hh * hd, (hh + 1) * hd)
    sc = []
    for k in keys:
        s = 0.0
        for d in sl:
            s += q[d] * k[d]
        sc.append(s / math.sqrt(hd))
    mx = max(sc)
    e = [math.exp(s - mx) for s in sc]
    tot = sum(e)
    out = [0.0] * hd
    for j, v in enumerate(vals):
        for i, d in enumerate(sl):
            out[i] += e[j] / tot * v[d]
    return out


def silu(x):
    return x / (1.0 + math.exp(-x))


def store(x, kvdtype):
    if kvdtype == "f64":
        return list(x)
    if kvdtype == "f32":
        return [float(np.float32(v)) for v in x]
    raise ValueError(kvdtype)


class BruteDecoder:
    """One sequence, dense or MoE, dual stream, f32/f64 cache only."""

    def __init__(self, cfg, weights: Dict[str, np.ndarray]):
        self.cfg = cfg
        self.W = {k: _f(v) for k, v in weights.items()}
        self.K: List[List[List[float]]] = [[] for _ in range(cfg.n_layers)]
        self.V: List[List[List[float]]] = [[] for _ in range(cfg.n_layers)]

    def lora(self, l, proj, x):
        return mv(self.W[f"L{l}.B_{proj}"], mv(self.W[f"L{l}.A_{proj}"], x))

    def qkv(self, l, x, pos, fast):
        c = self.cfg
        u = rms(x, self.W[f"L{l}.attn_norm"], c.rms_eps)
        q, k, v = mv(self.W[f"L{l}.wq"], u), mv(self.W[f"L{l}.wk"], u), mv(self.W[f"L{l}.wv"], u)
        if fast:
            q, k, v = add(q, self.lora(l, "q", u)), add(k, self.lora(l, "k", u)), add(v, self.lora(l, "v", u))
        return rot(q, pos, c.n_heads, c.head_dim, c.rope_theta), rot(k, pos, c.n_heads, c.head_dim, c.rope_theta), v

    def mlp(self, l, x, fast):
        c = self.cfg
        m = rms(x, self.W[f"L{l}.mlp_norm"], c.rms_eps)
        if c.is_moe:
            if fast:
                return self.lora(l, "m", m), None
            z = mv(self.W[f"L{l}.router"], m)
            mx = max(z)
            e = [math.exp(v - mx) for v in z]
            tot = sum(e)
            pr = [v / tot for v in e]
            order = sorted(range(len(pr)), key=lambda i: (-pr[i], i))[:c.top_k]
            y = [0.0] * len(x)
            for ex in order:
                g = mv(self.W[f"L{l}.E{ex}.wg"], m)
                u = mv(self.W[f"L{l}.E{ex}.wu"], m)
                a = [silu(g[i]) * u[i] for i in range(len(g))]
                y = add(y, [pr[ex] * v for v in mv(self.W[f"L{l}.E{ex}.wd"], a)])
            return y, order
        g, u = mv(self.W[f"L{l}.wg"], m), mv(self.W[f"L{l}.wu"], m)
        if fast:
            g, u = add(g, self.lora(l, "g", m)), add(u, self.lora(l, "u", m))
        a = [silu(g[i]) * u[i] for i in range(len(g))]
        y = mv(self.W[f"L{l}.wd"], a)
        if fast:
            y = add(y, self.lora(l, "d", a))
        return y, None

    def head(self, x):
        return mv(self.W["lm_head"], rms(x, self.W["final_norm"], self.cfg.rms_eps))

    def fast_head(self, x):
        if not self.cfg.head_rank:
            return self.head(x)
        return mv(self.W["head_B"], mv(self.W["head_A"], rms(x, self.W["final_norm"], self.cfg.rms_eps)))

    def fast_attention_flops(self, l, q_slow, qp, kp, vp, pos):
        """FLOPs-optimised fast attention (Sec. 2.5): head hh < fast_heads
        keeps the fast_topk cached positions whose slow-row score (head hh)
        is largest, by a plain sort on (-score, position); other heads give 0."""
        c = self.cfg
        hd = c.head_dim
        nh = c.fast_heads or c.n_heads
        out = [0.0] * (c.n_heads * hd)
        for hh in range(nh):
            sc = []
            for t in range(pos):
                s = 0.0
                for d in range(hh * hd, (hh + 1) * hd):
                    s += q_slow[d] * self.K[l][t][d]
                sc.append(s / math.sqrt(hd))
            keep = list(range(pos))
            if 0 < c.fast_topk < pos:
                keep = sorted(sorted(range(pos), key=lambda t: (-sc[t], t))[:c.fast_topk])
            o = one_head(qp, [self.K[l][t] for t in keep] + [kp], [self.V[l][t] for t in keep] + [vp], hh, hd)
            out[hh * hd:(hh + 1) * hd] = o
        return out

    def step(self, token: int, pos: int, gates: Sequence[int] = (), tau: float = 2.0, mode: str = "observe"):
        """Returns dict(logits, h, p, signal, exit_boundary, experts)."""
        c = self.cfg
        N = c.n_layers
        h = list(self.W["embed"][token])
        p = list(h)
        signal = [float("nan")] * N
        exit_b = N
        experts = []
        preds = {}
        for l in range(N):
            assert len(self.K[l]) == pos
            p_in = p
            # slow row: its own k/v go through the cache
            q, k, v = self.qkv(l, h, pos, fast=False)
            self.K[l].append(store(k, c.kvdtype))
            self.V[l].append(store(v, c.kvdtype))
            o = mha(q, self.K[l], self.V[l], c.n_heads, c.head_dim)
            h1 = add(h, mv(self.W[f"L{l}.wo"], o))
            y, order = self.mlp(l, h1, fast=False)
            experts.append(order)
            h = add(h1, y)
            # fast row: slow cache before pos, then its own k/v
            qp, kp, vp = self.qkv(l, p, pos, fast=True)
            if c.is_flops:
                op = self.fast_attention_flops(l, q, qp, kp, vp, pos)
            else:
                op = mha(qp, self.K[l][:pos] + [kp], self.V[l][:pos] + [vp], c.n_heads, c.head_dim)
            p1 = add(add(p, mv(self.W[f"L{l}.wo"], op)), self.lora(l, "o", op))
            if c.fast_mlp_adapter:
                yp = self.lora(l, "m", rms(p1, self.W[f"L{l}.mlp_norm"], c.rms_eps))
            else:
                yp, _ = self.mlp(l, p1, fast=True)
            p = add(p1, yp)
            dot = sum(p_in[i] * p[i] for i in range(len(p)))
            na = math.sqrt(sum(v * v for v in p_in))
            nb = math.sqrt(sum(v * v for v in p))
            signal[l] = dot / (na * nb)
            if c.is_moe:
                for lp in (2 * l + 2, 2 * l + 3):
                    if lp < N:
                        z = mv(self.W[f"L{lp}.router"], rms(p, self.W[f"L{lp}.mlp_norm"], c.rms_eps))
                        preds[lp] = sorted(range(len(z)), key=lambda i: (-z[i], i))[:c.top_k]
            b = l + 1
            if mode != "off" and b in set(gates):
                if signal[l] >= tau and exit_b == N:
                    exit_b = b
                if mode == "exit" and signal[l] >= tau:
                    for l2 in range(b, N):
                        _, k2, v2 = self.qkv(l2, h, pos, fast=False)
                        self.K[l2].append(store(k2, c.kvdtype))
                        self.V[l2].append(store(v2, c.kvdtype))
                    return dict(logits=self.fast_head(p), h=h, p=p, signal=signal, exit_boundary=exit_b,
                                experts=experts, preds=preds)
                p = list(h)
        return dict(logits=self.head(h), h=h, p=p, signal=signal, exit_boundary=exit_b, experts=experts,
                    preds=preds)
