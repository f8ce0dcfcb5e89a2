"""Slot mapping and decode attention over a paged cache, in float64 numpy (test
infrastructure only: nothing in the product path imports this module).

Slot mapping (Sec. 3.4): with a token table, a token's attention slot is no longer
block_id * S + offset of its logical position; the mapping consults the table instead. For
each request it lists the slots of the live tokens in logical order; dead tokens are left out
(Sec. 3.2: an evicted token is excluded from later slot mappings).

Decode attention (the consumer the slot mapping serves; the paper keeps the attention kernel
unchanged and relies on it reading relocated tokens through the token table). For query head
h with GQA group G = Hq / H reading KV head h // G, over the request's slots s_1..s_c:
  out[h] = softmax(scale * q[h] . K[s_j, h//G]) @ V[s_j, h//G],  scale = 1/sqrt(D) by default
and zeros for a request with no slots.
"""
from __future__ import annotations

import numpy as np


def dense_decode(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale=None) -> np.ndarray:
    """q [Hq, D]; k, v [n, H, D] -> [Hq, D] in float64."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    Hq, D = q.shape
    H = k.shape[1]
    G = Hq // H
    scale = 1.0 / np.sqrt(D) if scale is None else float(scale)
    out = np.zeros((Hq, D), dtype=np.float64)
    if k.shape[0] == 0:
        return out
    for h in range(Hq):
        s = (k[:, h // G, :] @ q[h]) * scale
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


def slot_mapping(token_slot, tok_indptr, seq_lens):
    """Token table -> slot mapping: per request, the slots of its live tokens (token_slot
    >= 0) in logical order, as CSR (slot_indptr [R+1], slots)."""
    token_slot = np.asarray(token_slot, dtype=np.int64)
    indptr = [0]
    slots = []
    for r in range(len(seq_lens)):
        a = int(tok_indptr[r])
        ts = token_slot[a:a + int(seq_lens[r])]
        live = ts[ts >= 0]
        slots.extend(int(x) for x in live)
        indptr.append(len(slots))
    return np.asarray(indptr, dtype=np.int64), np.asarray(slots, dtype=np.int64)


def slot_table(token_slot, tok_indptr, seq_lens, reserve: int):
    """The slot mapping laid out with room for `reserve` more slots per request (the
    append-only translation cache of Sec. 3.2): (slot_start [R+1], slot_count [R], slots),
    request r's live slots at slots[slot_start[r] ..][:slot_count[r]], unused room -1."""
    indptr, packed = slot_mapping(token_slot, tok_indptr, seq_lens)
    counts = np.diff(indptr)
    start = np.concatenate([[0], np.cumsum(counts + reserve)]).astype(np.int64)
    slots = np.full(int(start[-1]), -1, dtype=np.int64)
    for r in range(len(counts)):
        slots[start[r]:start[r] + counts[r]] = packed[indptr[r]:indptr[r + 1]]
    return start, counts.astype(np.int64), slots


def append_to_table(start, count, slots, new_slots_per_request):
    """Append each request's new slots after its current ones if its region has room;
    returns (count, slots, overflowed) with overflowing requests left unchanged."""
    count = np.array(count, dtype=np.int64)
    slots = np.array(slots, dtype=np.int64)
    overflow = False
    for r, new in enumerate(new_slots_per_request):
        n = len(new)
        if n == 0:
            continue
        if count[r] + n > start[r + 1] - start[r]:
            overflow = True
            continue
        slots[start[r] + count[r]:start[r] + count[r] + n] = new
        count[r] += n
    return count, slots, overflow


def decode_batch(q: np.ndarray, k_plane: np.ndarray, v_plane: np.ndarray, slot_indptr,
                 slots, scale=None) -> np.ndarray:
    """Decode attention of every request through a slot mapping. q [R, Hq, D]; k_plane,
    v_plane [num_slots, H, D] (one layer's K and V planes as values) -> [R, Hq, D]."""
    q = np.asarray(q, dtype=np.float64)
    out = np.zeros(q.shape, dtype=np.float64)
    for r in range(q.shape[0]):
        sl = np.asarray(slots[int(slot_indptr[r]):int(slot_indptr[r + 1])], dtype=np.int64)
        out[r] = dense_decode(q[r], k_plane[sl], v_plane[sl], scale)
    return out
