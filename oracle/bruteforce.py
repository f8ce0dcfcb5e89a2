"""Per-token pure-Python repack for tiny inputs (test infrastructure only).

An independent, literal walk through relocation planning (Sec. 3.3.3) and headroom-aware
admission (Sec. 3.3.2) on Python lists, used to pin the vectorised oracle. It shares no
code with repack.py: no scans, no ceil formula, no fancy indexing.

  - A request's destination count is found by search: the fewest blocks whose S slots each
    can hold all of its live tokens.
  - The plan is dropped unless that count is strictly below the blocks the request holds.
  - Destinations are handed out from the free list in request order while enough remain;
    after the first refusal no later request receives any.
  - The destination slots are listed block by block, offset by offset, and the i-th live
    token (in logical order) takes the i-th slot.
  - Rows move from the old slot to the new slot in every plane; everything else stays.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence


def brute_repack(seq_lens: Sequence[int], block_tables: Sequence[Sequence[int]],
                 live_masks: Sequence[Sequence[int]], free_list: Sequence[int], S: int,
                 planes: Optional[List[Dict[int, bytes]]] = None, inplace: bool = False):
    """Returns a dict with token_slot (list per request), admitted, new_tables, freed, used,
    src_plan (flat list) and, if `planes` (slot -> row bytes per plane) is given, the new
    planes. With inplace=True a request that gains blocks reuses its own leading blocks as
    destinations (no free list, nothing deferred) and releases the blocks it no longer
    fills. Moves are applied one token at a time, in logical order: a token only moves to
    an earlier or equal slot position, and every slot it overwrites has already been read."""
    free = list(free_list)
    handed_out = 0
    refused = False
    token_slot: List[List[int]] = []
    admitted: List[int] = []
    new_tables: List[List[int]] = []
    freed: List[int] = []
    src_plan: List[int] = []
    moves = []  # (old slot, new slot)

    for r in range(len(seq_lens)):
        n = seq_lens[r]
        table = list(block_tables[r])
        live = list(live_masks[r])
        old_slot = []
        for p in range(n):
            old_slot.append(table[p // S] * S + p % S)
        live_positions = [p for p in range(n) if live[p]]

        blocks = 0
        while blocks * S < len(live_positions):
            blocks += 1

        plan_ok = blocks < len(table)
        if plan_ok and not inplace and (refused or handed_out + blocks > len(free)):
            refused = True
            plan_ok = False
        if not plan_ok:
            admitted.append(0)
            new_tables.append(table)
            token_slot.append([old_slot[p] if live[p] else -1 for p in range(n)])
            continue

        if inplace:
            dest = table[:blocks]
        else:
            dest = free[handed_out:handed_out + blocks]
        handed_out += blocks
        dest_slots = []
        for blk in dest:
            for off in range(S):
                dest_slots.append(blk * S + off)
        slots = [-1] * n
        for i, p in enumerate(live_positions):
            slots[p] = dest_slots[i]
            moves.append((old_slot[p], dest_slots[i]))
        for i in range(len(dest_slots)):
            src_plan.append(old_slot[live_positions[i]] if i < len(live_positions) else -1)
        admitted.append(1)
        new_tables.append(dest)
        token_slot.append(slots)
        freed.extend(table[blocks:] if inplace else table)

    out = dict(token_slot=token_slot, admitted=admitted, new_tables=new_tables, freed=freed,
               used=handed_out, src_plan=src_plan,
               live_count=[sum(1 for x in m if x) for m in live_masks])
    if planes is not None:
        new_planes = []
        for plane in planes:
            q = dict(plane)
            for old, new in moves:
                # out of place the source is untouched; in place it is read from the plane
                # being built, which the logical order keeps valid (see the docstring)
                q[new] = q[old] if inplace else plane[old]
            new_planes.append(q)
        out["planes"] = new_planes
    return out


def brute_plan_partial(seq_lens: Sequence[int], block_tables: Sequence[Sequence[int]],
                       live_masks: Sequence[Sequence[int]], slots: Sequence[Sequence[int]],
                       free_list: Sequence[int], S: int, theta=(1, 4), max_live=None,
                       max_sources=1 << 30, min_eligible=1, free_watermark=-1,
                       pinned: Sequence[int] = (), planes: Optional[List[Dict[int, bytes]]] = None):
    """Literal walk of the partial pass (Sec. 3.3.1-3.3.4) on Python lists, sharing no code
    with planner.py: live tokens per block are counted one slot at a time, the waste ratio is
    compared as a fraction, candidates are collected block by block while a budget counter
    runs down, destinations are handed out slot by slot. Returns a dict of lists."""
    from fractions import Fraction
    R = len(seq_lens)
    holders: Dict[int, int] = {}
    for t in block_tables:
        for b in t:
            holders[b] = holders.get(b, 0) + 1
    live_at = set()
    for r in range(R):
        for p in range(seq_lens[r]):
            if live_masks[r][p]:
                live_at.add(slots[r][p])
    count = {b: 0 for b in holders}
    for b in holders:
        for off in range(S):
            if b * S + off in live_at:
                count[b] += 1
    total_live = sum(count.values())
    n_alloc = len(holders)
    waste = Fraction(0) if n_alloc == 0 else 1 - Fraction(total_live, n_alloc * S)
    theta_f = Fraction(theta[0], theta[1])
    if max_live is None:
        # a block is low-utilisation when its own waste exceeds theta_F
        ok = lambda b: 1 - Fraction(count[b], S) > theta_f  # noqa: E731
    else:
        ok = lambda b: count[b] <= max_live  # noqa: E731
    pinned_set = set(pinned)
    candidates = [[b for b in block_tables[r] if holders[b] == 1 and b not in pinned_set
                   and ok(b)] for r in range(R)]
    n_cand = sum(len(c) for c in candidates)
    go = (n_alloc > 0 and waste > theta_f and n_cand >= min_eligible
          and (free_watermark < 0 or len(free_list) <= free_watermark))

    chosen = [[] for _ in range(R)]
    if go:
        left = max_sources
        for r in range(R):
            for b in candidates[r]:
                if left > 0:
                    chosen[r].append(b)
                left -= 1
    free = list(free_list)
    handed = 0
    refused = False
    admitted, new_tables, freed, token_slot, src_plan = [], [], [], [], []
    moves = []
    for r in range(R):
        moving = [p for p in range(seq_lens[r])
                  if live_masks[r][p] and slots[r][p] // S in chosen[r]]
        blocks = 0
        while blocks * S < len(moving):
            blocks += 1
        good = len(chosen[r]) > 0 and blocks < len(chosen[r])
        if good and (refused or handed + blocks > len(free)):
            refused = True
            good = False
        out = [slots[r][p] if live_masks[r][p] else -1 for p in range(seq_lens[r])]
        if not good:
            admitted.append(0)
            new_tables.append(list(block_tables[r]))
            token_slot.append(out)
            continue
        dest = free[handed:handed + blocks]
        handed += blocks
        dest_slots = [blk * S + off for blk in dest for off in range(S)]
        for i, p in enumerate(moving):
            out[p] = dest_slots[i]
            moves.append((slots[r][p], dest_slots[i]))
        src_plan.extend(slots[r][moving[i]] if i < len(moving) else -1
                        for i in range(len(dest_slots)))
        admitted.append(1)
        new_tables.append([b for b in block_tables[r] if b not in chosen[r]] + dest)
        freed.extend(b for b in block_tables[r] if b in chosen[r])
        token_slot.append(out)
    out = dict(triggered=go, count=count, chosen=[len(c) for c in chosen], admitted=admitted,
               new_tables=new_tables, freed=freed, token_slot=token_slot, used=handed,
               src_plan=src_plan)
    if planes is not None:
        new_planes = []
        for plane in planes:
            q = dict(plane)
            for old, new in moves:
                q[new] = plane[old]
            new_planes.append(q)
        out["planes"] = new_planes
    return out
