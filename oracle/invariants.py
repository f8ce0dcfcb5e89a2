"""Convention-free checks of a repack pass against the paper's invariants (test only).

These accept any valid packing - they do not assume which free blocks are taken, in which
request order, or which requests the headroom admits - so they pin the oracle (and any
implementation) independently of the readings frozen in the header.

  I1  token conservation (Sec. 3.5): the ordered live tokens of each request and their K/V
      payloads are identical before and after; checked as in Sec. 5.8 by hashing
      (logical position, payload) in logical order.
  I2  unique mapping (Sec. 3.5): every live token has exactly one valid (block, offset) inside
      its request's table, and no slot is referenced twice.
  I4  layout-aware planning (Sec. 3.5): a repacked request ends with strictly fewer blocks.
  Relocation planning (Sec. 3.3.3): ceil(live / S) destinations, filled in logical order,
      each block completely before the next; destinations come from the free pool.
  Sec. 3.3.4: only the old blocks of repacked requests are released.
  Sec. 2.3.1: the waste ratio F over allocated blocks does not increase.
  Bytes outside the moved rows are unchanged (out-of-place relocation, Sec. 3.3.2).
"""
from __future__ import annotations

import hashlib
from collections import Counter
from typing import Optional

import numpy as np


def _fail(msg: str):
    raise AssertionError(msg)


def _waste(tables, live_slot_lists, S):
    total_blocks = 0
    total_live = 0
    for table, slots in zip(tables, live_slot_lists):
        total_blocks += len(table)
        total_live += len(slots)
    if total_blocks == 0:
        return 0.0
    return 1.0 - total_live / (total_blocks * S)


def check_invariants(seq_lens, tok_indptr, bt_indptr, block_ids, live, free_list, S: int,
                     num_blocks: int, token_slot, new_bt_indptr, new_block_ids, freed,
                     used: int, kv_before: Optional[np.ndarray] = None,
                     kv_after: Optional[np.ndarray] = None, inplace: bool = False) -> None:
    """Raise AssertionError naming the first violated invariant. With inplace=True the
    destinations of a repacked request must be the leading blocks of its own table, its other
    blocks must be released, and the free list must stay untouched."""
    R = len(seq_lens)
    live = np.asarray(live, dtype=np.uint8)
    token_slot = np.asarray(token_slot, dtype=np.int64)
    free_list = np.asarray(free_list, dtype=np.int64)
    all_live_slots = []
    old_tables, new_tables, old_live_slots, new_live_slots = [], [], [], []
    repacked = []
    for r in range(R):
        n = int(seq_lens[r])
        a = int(tok_indptr[r])
        bt = [int(x) for x in block_ids[bt_indptr[r]:bt_indptr[r + 1]]]
        nbt = [int(x) for x in new_block_ids[new_bt_indptr[r]:new_bt_indptr[r + 1]]]
        old_tables.append(bt)
        new_tables.append(nbt)
        lv = live[a:a + n] != 0
        ts = token_slot[a:a + n]
        c = int(lv.sum())
        if np.any(ts[~lv] != -1):
            _fail(f"I2: request {r} has a dead token with a slot")
        if len(set(nbt)) != len(nbt):
            _fail(f"I2: request {r} table repeats a block")
        pos_of_block = {b: i for i, b in enumerate(nbt)}
        seq_pos = []
        for p in np.nonzero(lv)[0]:
            s = int(ts[p])
            if s < 0 or s >= num_blocks * S:
                _fail(f"I2: request {r} token {p} slot {s} out of range")
            if s // S not in pos_of_block:
                _fail(f"I2: request {r} token {p} slot outside its block table")
            seq_pos.append(pos_of_block[s // S] * S + s % S)
            all_live_slots.append(s)
        old_slots = [bt[p // S] * S + p % S for p in np.nonzero(lv)[0]]
        old_live_slots.append(old_slots)
        new_live_slots.append([int(ts[p]) for p in np.nonzero(lv)[0]])
        moved = nbt != bt
        repacked.append(moved)
        if moved:
            if len(nbt) >= len(bt):
                _fail(f"I4: request {r} repacked without a strict block reduction")
            if len(nbt) * S < c or (len(nbt) - 1) * S >= c:
                _fail(f"3.3.3: request {r} uses {len(nbt)} blocks for {c} live tokens")
            if seq_pos != list(range(c)):
                _fail(f"3.3.3: request {r} live tokens not filled in order, block by block")
        else:
            if [int(ts[p]) for p in np.nonzero(lv)[0]] != old_slots:
                _fail(f"request {r} kept its table but its token slots changed")
    if len(set(all_live_slots)) != len(all_live_slots):
        _fail("I2: a slot is referenced by two live tokens")

    if inplace:
        # destinations are the request's own leading blocks; the rest is released
        for r in range(R):
            if repacked[r] and new_tables[r] != old_tables[r][:len(new_tables[r])]:
                _fail(f"in place: request {r} destinations are not its leading blocks")
        if Counter(int(x) for x in freed) != Counter(
                b for r in range(R) if repacked[r] for b in old_tables[r][len(new_tables[r]):]):
            _fail("in place: freed blocks are not the released tails of repacked requests")
        consumed = 0
    else:
        # destinations come from the free pool, freed = old blocks of repacked requests
        if used < 0 or used > len(free_list):
            _fail("3.3.2: more destinations than the free list holds")
        dest_blocks = Counter(b for r in range(R) if repacked[r] for b in new_tables[r])
        if dest_blocks != Counter(int(x) for x in free_list[:used]):
            _fail("3.3.3: destination blocks are not the consumed free-list entries")
        if Counter(int(x) for x in freed) != Counter(b for r in range(R) if repacked[r]
                                                     for b in old_tables[r]):
            _fail("3.3.4: freed blocks are not exactly the old blocks of repacked requests")
        consumed = used
    before = Counter(b for t in old_tables for b in t) + Counter(int(x) for x in free_list)
    after = Counter(b for t in new_tables for b in t) + Counter(int(x) for x in freed) + \
        Counter(int(x) for x in free_list[consumed:])
    if before != after:
        _fail("block conservation: tables + pool differ before and after")
    if _waste(new_tables, new_live_slots, S) > _waste(old_tables, old_live_slots, S) + 1e-12:
        _fail("2.3.1: waste ratio increased")

    if kv_before is None or kv_after is None:
        return
    kv_before = np.asarray(kv_before)
    kv_after = np.asarray(kv_after)
    touched = np.zeros(kv_before.shape[1], dtype=bool)
    for r in range(R):
        h0, h1 = hashlib.sha256(), hashlib.sha256()
        a = int(tok_indptr[r])
        lv = np.nonzero(live[a:a + int(seq_lens[r])])[0]
        for i, p in enumerate(lv):
            so, sn = old_live_slots[r][i], new_live_slots[r][i]
            h0.update(int(p).to_bytes(8, "little"))
            h0.update(np.ascontiguousarray(kv_before[:, so, :]).tobytes())
            h1.update(int(p).to_bytes(8, "little"))
            h1.update(np.ascontiguousarray(kv_after[:, sn, :]).tobytes())
            if so != sn:
                touched[sn] = True
        if h0.digest() != h1.digest():
            _fail(f"I1: request {r} live tokens or payloads changed")
    if not np.array_equal(kv_after[:, ~touched, :], kv_before[:, ~touched, :]):
        _fail("bytes outside the moved rows changed")
