"""Grouped-query decode attention over a shared prompt KV plus a per-row tail.

Section 3 reuses the prompt's KV cache for the greedy probe and for every
sampled continuation; each decoding row therefore attends to the prompt
positions it shares with all other rows of that prompt and to the positions it
generated itself.  For query head h the key/value head is h // G with
G = Hq / Hkv, and the scores are scaled by 1/sqrt(D):

    o_h = sum_j softmax_j(q_h . k_{g,j} / sqrt(D)) v_{g,j}

where j runs over the prompt positions followed by the row's own positions.
float64 throughout.
"""
from __future__ import annotations

import numpy as np


def softmax(s: np.ndarray) -> np.ndarray:
    e = np.exp(s - s.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def attend(q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """q [Hq][D]; k, v [n][Hkv][D] -> o [Hq][D]."""
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    hq, d = q.shape
    hkv = k.shape[1]
    g = hq // hkv
    out = np.empty((hq, d))
    for h in range(hq):
        kh = k[:, h // g, :]
        s = kh @ q[h] / np.sqrt(d)
        out[h] = softmax(s) @ v[:, h // g, :]
    return out


def attend_prefix_tail(q, k_prefix, v_prefix, k_tail, v_tail) -> np.ndarray:
    """Attention of one row over its prompt prefix followed by its own tail."""
    k = np.concatenate([np.asarray(k_prefix, np.float64), np.asarray(k_tail, np.float64)], axis=0)
    v = np.concatenate([np.asarray(v_prefix, np.float64), np.asarray(v_tail, np.float64)], axis=0)
    return attend(q, k, v)
