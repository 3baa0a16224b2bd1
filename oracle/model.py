"""Llama-style decoder used as the target model M (oracle side).

The paper runs pretrained instruction models (Section 4); the workloads here are
random-initialised decoders of the same family, so the layer is the standard
pre-norm block:

    a   = RMSNorm(x) * g_attn,           RMSNorm(x) = x / sqrt(mean(x^2) + eps)
    q,k,v = Wq a, Wk a, Wv a              (heads of size D; Hkv key/value heads)
    q,k <- RoPE(q, pos), RoPE(k, pos)     rotate-half form, frequencies theta^(-2j/D)
    h   = x + Wo Attn(q, K, V)
    x'  = h + W_down( SiLU(W_gate b) * (W_up b) ),   b = RMSNorm(h) * g_ffn
    logits = W_lm (RMSNorm(x_last) * g_final)

Weights arrive as bf16 bit patterns (uint16) or float32 and are widened to
float64 exactly; every operation is then float64.  The KV cache holds rotated
keys, as a serving engine's prefix cache does (Section 3 reuses it across the
probe and the sampling stage).
"""
from __future__ import annotations

import numpy as np

from .attention import attend


def widen(a: np.ndarray) -> np.ndarray:
    """Exact float64 view of a bf16-bit-pattern (uint16) or float32 array."""
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return np.asarray(a, dtype=np.float64)


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    x = np.asarray(x, np.float64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * widen(g)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def rope(x: np.ndarray, pos: int, theta: float) -> np.ndarray:
    """Rotate-half rotary embedding of x [H][D] at integer position pos: the pair
    (x_j, x_{j+D/2}) is rotated by the angle pos * theta^(-2j/D)."""
    d = x.shape[-1]
    half = d // 2
    freq = theta ** (-(2.0 * np.arange(half)) / d)
    ang = pos * freq
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def linear(w: np.ndarray, x: np.ndarray, chunk_rows: int = 8192) -> np.ndarray:
    """y = x W^T for x [n][in] (or [in]) and W [out][in]; W widened per row-chunk."""
    x = np.asarray(x, np.float64)
    vec = x.ndim == 1
    x2 = x[None, :] if vec else x
    out = np.empty((x2.shape[0], w.shape[0]))
    for r0 in range(0, w.shape[0], chunk_rows):
        wc = widen(w[r0:r0 + chunk_rows])
        out[:, r0:r0 + wc.shape[0]] = x2 @ wc.T
    return out[0] if vec else out


class KVCache:
    """Per-layer K/V of one token sequence: lists of [Hkv][D] float64 rows."""

    def __init__(self, n_layers: int):
        self.k = [[] for _ in range(n_layers)]
        self.v = [[] for _ in range(n_layers)]

    @classmethod
    def from_arrays(cls, ks, vs):
        c = cls(len(ks))
        for l, (k, v) in enumerate(zip(ks, vs)):
            c.k[l] = list(widen(k))
            c.v[l] = list(widen(v))
        return c

    def length(self) -> int:
        return len(self.k[0]) if self.k else 0

    def arrays(self, layer: int):
        return np.asarray(self.k[layer]), np.asarray(self.v[layer])


class Decoder:
    """The target model M over synthetic weights (see synth.Weights)."""

    def __init__(self, weights):
        self.W = weights
        w = weights.w
        self.cfg = w
        self.hq, self.hkv, self.d = w.n_heads, w.n_kv_heads, w.head_dim

    # one transformer block for n new tokens, given the K/V visible to each
    def _block(self, l, x, positions, visible):
        """x [n][d_model]; positions [n]; visible(t, k_new, v_new) -> (K, V) the
        t-th new token attends to.  Returns (x', k_new, v_new)."""
        L = self.W.layers[l]
        c = self.cfg
        a = rmsnorm(x, L["attn_norm"], c.rms_eps)
        q = linear(L["wq"], a).reshape(-1, self.hq, self.d)
        k = linear(L["wk"], a).reshape(-1, self.hkv, self.d)
        v = linear(L["wv"], a).reshape(-1, self.hkv, self.d)
        for t, pos in enumerate(positions):
            q[t] = rope(q[t], pos, c.rope_theta)
            k[t] = rope(k[t], pos, c.rope_theta)
        o = np.empty_like(q)
        for t in range(len(positions)):
            K, V = visible(t, k, v)
            o[t] = attend(q[t], K, V)
        h = x + linear(L["wo"], o.reshape(len(positions), -1))
        b = rmsnorm(h, L["ffn_norm"], c.rms_eps)
        f = silu(linear(L["w_gate"], b)) * linear(L["w_up"], b)
        return h + linear(L["w_down"], f), k, v

    def logits(self, x_last: np.ndarray) -> np.ndarray:
        return linear(self.W.lm_head, rmsnorm(x_last, self.W.final_norm, self.cfg.rms_eps))

    def embed(self, tokens) -> np.ndarray:
        return widen(self.W.embed[np.asarray(tokens)])

    def prefill(self, tokens, cache: KVCache, start_pos: int | None = None, taps: dict | None = None) -> np.ndarray:
        """Causal forward of a prompt segment appended to `cache` (which holds
        positions [0, start_pos)); returns the last position's logits.  taps,
        when given, receives the last position's residual stream: taps[0] the
        embedding, taps[l] the output of block l (1-based)."""
        tokens = np.asarray(tokens)
        start = cache.length() if start_pos is None else start_pos
        assert start == cache.length()
        pos = np.arange(start, start + len(tokens))
        x = self.embed(tokens)
        if taps is not None:
            taps[0] = x[-1].copy()
        for l in range(self.cfg.n_layers):
            Kc, Vc = cache.arrays(l)
            Kc = Kc.reshape(-1, self.hkv, self.d)
            Vc = Vc.reshape(-1, self.hkv, self.d)

            def visible(t, k, v, Kc=Kc, Vc=Vc):
                return (np.concatenate([Kc, k[:t + 1]]), np.concatenate([Vc, v[:t + 1]]))

            x, k, v = self._block(l, x, pos, visible)
            cache.k[l].extend(list(k))
            cache.v[l].extend(list(v))
            if taps is not None:
                taps[l + 1] = x[-1].copy()
        return self.logits(x[-1])

    def decode(self, token: int, prefix: KVCache, tail: KVCache) -> np.ndarray:
        """One decode step of a row whose context is `prefix` (shared, read
        only) followed by its own `tail` (appended to).  Returns logits."""
        pos = prefix.length() + tail.length()
        x = self.embed([token])
        for l in range(self.cfg.n_layers):
            Kp, Vp = prefix.arrays(l)
            Kt, Vt = tail.arrays(l)
            parts_k = [a.reshape(-1, self.hkv, self.d) for a in (Kp, Kt) if len(a)]
            parts_v = [a.reshape(-1, self.hkv, self.d) for a in (Vp, Vt) if len(a)]

            def visible(t, k, v):
                return (np.concatenate(parts_k + [k[:1]]), np.concatenate(parts_v + [v[:1]]))

            x, k, v = self._block(l, x, [pos], visible)
            tail.k[l].append(k[0])
            tail.v[l].append(v[0])
        return self.logits(x[0])
