"""Decode attention over a paged cache, in float64 numpy (test infrastructure only).

Secondary check of the repack: attention that walks a request's new block table over the
repacked cache must equal dense attention over only the request's live tokens taken from
the cache before the pass. This is the consumer the slot mapping of Sec. 3.4 serves; the
paper keeps the attention kernel unchanged and relies on it reading relocated tokens
through the token table.

Attention for query head h with GQA group G = Hq / H reads KV head h // G:
  out[h] = softmax(q[h] . K[:, h//G]^T / sqrt(D)) @ V[:, h//G]
"""
from __future__ import annotations

import numpy as np


def dense_decode(q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """q [Hq, D]; k, v [n, H, D] -> [Hq, D] in float64."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    Hq, D = q.shape
    H = k.shape[1]
    G = Hq // H
    out = np.zeros((Hq, D), dtype=np.float64)
    if k.shape[0] == 0:
        return out
    for h in range(Hq):
        s = k[:, h // G, :] @ q[h] / np.sqrt(D)
        w = np.exp(s - s.max())
        w /= w.sum()
        out[h] = w @ v[:, h // G, :]
    return out


def paged_decode(q: np.ndarray, k_plane: np.ndarray, v_plane: np.ndarray, block_table,
                 num_tokens: int, S: int) -> np.ndarray:
    """Attention over the first `num_tokens` slots of `block_table` (slot = b*S + off).
    k_plane, v_plane: [num_blocks*S, H, D] element arrays of one layer."""
    slots = [int(block_table[p // S]) * S + p % S for p in range(num_tokens)]
    return dense_decode(q, k_plane[slots], v_plane[slots])
