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
