"""Numpy oracle of the paper's partial reclamation pass (test infrastructure only).

Where oracle/repack.py takes every block of a request as a source, this follows the four
stages of the reclamation backend of Sec. 3.3 as the paper states them, in its order:

  P1  eligibility     - Sec. 3.3.1 and Sec. 2.3.1: n_b = live tokens in block b, u_b = n_b / S,
                        F = 1 - sum(n_b) / (N * S) over the N allocated blocks.
  P2  trigger         - Sec. 3.3.2: reclamation is attempted only when F > theta_F, enough
                        low-utilisation blocks exist and the free-block count is near its low
                        watermark.
  P3  planning        - Sec. 3.3.3: per request, its eligible low-utilisation source blocks
                        (at most B source blocks considered in the round), their live tokens
                        T_live, ceil(T_live / S) destinations, a plan only if that is fewer
                        blocks than the sources; admission only if the free list can supply
                        the destinations (Sec. 3.3.2).
  P4  move list       - Sec. 3.3.3: the live tokens of the sources in logical order, assigned
                        sequentially to the destination slots, each destination block filled
                        before the next; applying it updates the token table (Sec. 3.2).
  P5  copy            - the rows of every plane move to their destination slots.
  P6  release         - Sec. 3.3.4: the emptied source blocks are freed.
  Shared prefix       - I4 of Sec. 3.5 and Sec. 5.7: blocks in more than one request's table
                        (and blocks the caller pins) are never sources.

Inputs are a token table rather than a positional layout: slot_in[t] is the current slot of
logical token t (-1 when it holds none), so passes can follow each other (tokens of a
partially repacked request are no longer in block-table order).

Readings where the paper gives no number or order (frozen in the C header as well):
  * a block is a low-utilisation source candidate iff it is in exactly one table, is not
    pinned and n_b <= max_live_per_source (default: its own waste exceeds theta_F,
    n_b < (1 - theta_F) * S);
  * a sufficient number of low-utilisation blocks: at least min_eligible candidates; a free
    count close to the low watermark: free-list length <= free_watermark (a negative
    watermark drops the condition);
    F > theta_F is evaluated exactly as (N*S - sum n_b) * den > num * N*S;
  * B counts the blocks considered: candidates are taken in request order, table order
    within a request, until B are taken, whether or not the request's plan is then admitted;
  * admission is the prefix rule of the full pass: destinations come from the front of the
    free list in request order, and after the first request that does not fit no later one
    is admitted;
  * a repacked request's new table is its unselected blocks in their order followed by its
    destination blocks; the freed list is its selected sources in table order;
  * dead tokens map to -1 in the output token table.
KV is opaque bytes: kv[plane, slot, :] is one token's row in one plane.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

from oracle.repack import OracleInputError


@dataclasses.dataclass
class PlannerParams:
    theta_num: int = 1            # theta_F = theta_num / theta_den (0.25, Sec. 3.3.2)
    theta_den: int = 4
    max_live_per_source: Optional[int] = None  # None: n_b < (1 - theta_F) * S
    max_sources: int = 1 << 30    # B
    min_eligible: int = 1
    free_watermark: int = -1      # < 0: no watermark condition

    def max_live(self, S: int) -> int:
        if self.max_live_per_source is not None:
            return int(self.max_live_per_source)
        # largest n with n * den < (den - num) * S
        lim = (self.theta_den - self.theta_num) * S
        return (lim - 1) // self.theta_den if lim > 0 else -1


@dataclasses.dataclass
class PlannerResult:
    n_b: dict                  # block -> live tokens, every block in some table
    refs: dict                 # block -> number of tables holding it
    live_total: int            # sum of n_b over the distinct allocated blocks
    allocated: int             # N
    eligible: int              # candidate blocks over all requests
    triggered: bool
    src_count: np.ndarray      # int32 [R] sources considered per request (k_r)
    moved_live: np.ndarray     # int64 [R] T_live of the considered sources
    need: np.ndarray           # int64 [R]
    token_slot: np.ndarray     # int32 [T]
    live_count: np.ndarray     # int32 [R]
    admitted: np.ndarray       # int32 [R]
    dst_indptr: np.ndarray     # int32 [R+1]
    new_bt_indptr: np.ndarray  # int32 [R+1]
    new_block_ids: np.ndarray  # int32
    src_plan: np.ndarray       # int32 [used*S]
    freed_indptr: np.ndarray   # int32 [R+1]
    freed: np.ndarray          # int32 [n_freed]
    used: int
    n_admitted: int
    n_freed: int
    tokens_moved: int
    kv: Optional[np.ndarray] = None


def waste_ratio_exceeds(live_total: int, allocated: int, S: int, num: int, den: int) -> bool:
    """F > num/den with F = 1 - live_total / (allocated * S), in exact integers."""
    cap = allocated * S
    return cap > 0 and (cap - live_total) * den > num * cap


def plan_partial(seq_lens, tok_indptr, bt_indptr, block_ids, live, slot_in, free_list,
                 block_size: int, num_blocks: int, params: PlannerParams = PlannerParams(),
                 pinned=None, kv: Optional[np.ndarray] = None) -> PlannerResult:
    S = int(block_size)
    seq_lens = np.asarray(seq_lens, dtype=np.int64)
    tok_indptr = np.asarray(tok_indptr, dtype=np.int64)
    bt_indptr = np.asarray(bt_indptr, dtype=np.int64)
    block_ids = np.asarray(block_ids, dtype=np.int64)
    live = np.asarray(live, dtype=np.uint8)
    slot_in = np.asarray(slot_in, dtype=np.int64)
    free_list = np.asarray(free_list, dtype=np.int64)
    pinned = np.zeros(num_blocks, dtype=bool) if pinned is None else \
        np.asarray(pinned, dtype=bool)
    R = len(seq_lens)
    if len(tok_indptr) != R + 1 or len(bt_indptr) != R + 1 or len(slot_in) != len(live):
        raise OracleInputError("shape", "indptr arrays need R+1 entries, slot_in one per token")
    if len(block_ids) and (block_ids.min() < 0 or block_ids.max() >= num_blocks):
        raise OracleInputError("block_range", "block table")
    for r in range(R):
        if int(tok_indptr[r + 1]) - int(tok_indptr[r]) != int(seq_lens[r]):
            raise OracleInputError("tok_len", f"request {r}")
    tables = [block_ids[bt_indptr[r]:bt_indptr[r + 1]] for r in range(R)]
    tokens = [(int(tok_indptr[r]), int(tok_indptr[r + 1])) for r in range(R)]

    # P1: per-block live tokens. A slot counts once even if several requests hold it live
    # (shared-prefix blocks).
    refs = {}
    for t in tables:
        for b in t:
            refs[int(b)] = refs.get(int(b), 0) + 1
    live_slots = {}
    for r in range(R):
        a, e = tokens[r]
        own = set(int(b) for b in tables[r])
        for t in range(a, e):
            if live[t]:
                s = int(slot_in[t])
                if s < 0 or s >= num_blocks * S or s // S not in own:
                    raise OracleInputError("slot", f"request {r} live token {t - a} slot {s}")
                holders = live_slots.setdefault(s, [])
                if r in holders or (holders and refs[s // S] == 1):
                    raise OracleInputError("slot", f"slot {s} held twice (I2, Sec. 3.5)")
                holders.append(r)
    n_b = {b: 0 for b in refs}
    for s in live_slots:
        n_b[s // S] += 1
    live_total = sum(n_b.values())
    allocated = len(refs)

    # P2: trigger
    max_live = params.max_live(S)
    candidate = {b: refs[b] == 1 and not pinned[b] and n_b[b] <= max_live for b in refs}
    eligible_per_req = [[int(b) for b in t if candidate[int(b)]] for t in tables]
    eligible = sum(len(x) for x in eligible_per_req)
    triggered = (waste_ratio_exceeds(live_total, allocated, S, params.theta_num,
                                     params.theta_den)
                 and eligible >= params.min_eligible
                 and (params.free_watermark < 0 or len(free_list) <= params.free_watermark))

    # P3: sources under the bound B, T_live, need, profit, admission
    src_count = np.zeros(R, dtype=np.int64)
    moved_live = np.zeros(R, dtype=np.int64)
    need = np.zeros(R, dtype=np.int64)
    admitted = np.zeros(R, dtype=bool)
    dst_off = np.zeros(R, dtype=np.int64)
    if triggered:
        budget = int(params.max_sources)
        for r in range(R):
            k = min(len(eligible_per_req[r]), max(budget, 0))
            budget -= len(eligible_per_req[r])
            src_count[r] = k
            moved_live[r] = sum(n_b[b] for b in eligible_per_req[r][:k])
        need = (moved_live + S - 1) // S
        profitable = (src_count > 0) & (need < src_count)
        o = 0
        for r in range(R):
            if not profitable[r]:
                continue
            dst_off[r] = o
            admitted[r] = o + need[r] <= len(free_list)
            o += int(need[r])
    used = int((need * admitted).sum())
    if used and (free_list[:used].min() < 0 or free_list[:used].max() >= num_blocks):
        raise OracleInputError("block_range", "free list")

    # P4: move list, token table, new tables, source plan; P6: released sources
    token_slot = np.full(len(live), -1, dtype=np.int64)
    live_count = np.zeros(R, dtype=np.int64)
    dst_indptr = np.zeros(R + 1, dtype=np.int64)
    dst_indptr[1:] = np.cumsum(need * admitted)
    src_plan = np.full(used * S, -1, dtype=np.int64)
    new_tables, freed_lists = [], []
    moves = []
    for r in range(R):
        a, e = tokens[r]
        lv = live[a:e] != 0
        live_count[r] = lv.sum()
        token_slot[a:e] = np.where(lv, slot_in[a:e], -1)
        if not admitted[r]:
            new_tables.append(tables[r])
            freed_lists.append(np.zeros(0, np.int64))
            continue
        chosen = set(eligible_per_req[r][:src_count[r]])
        dest = free_list[dst_indptr[r]:dst_indptr[r + 1]]
        q = 0
        for t in range(a, e):                      # logical order
            if lv[t - a] and int(slot_in[t]) // S in chosen:
                new = int(dest[q // S]) * S + q % S
                src_plan[dst_indptr[r] * S + q] = slot_in[t]
                moves.append((int(slot_in[t]), new))
                token_slot[t] = new
                q += 1
        assert q == moved_live[r]
        new_tables.append(np.concatenate([[b for b in tables[r] if int(b) not in chosen],
                                          dest]).astype(np.int64))
        freed_lists.append(np.asarray([b for b in tables[r] if int(b) in chosen], np.int64))

    new_bt_indptr = np.zeros(R + 1, dtype=np.int64)
    new_bt_indptr[1:] = np.cumsum([len(t) for t in new_tables])
    freed_indptr = np.zeros(R + 1, dtype=np.int64)
    freed_indptr[1:] = np.cumsum([len(x) for x in freed_lists])

    # P5: copy
    kv_out = None
    if kv is not None:
        kv_out = kv.copy()
        if moves:
            src = np.asarray([m[0] for m in moves])
            dst = np.asarray([m[1] for m in moves])
            kv_out[:, dst, :] = kv[:, src, :]

    i32 = lambda x: np.asarray(x, dtype=np.int32)  # noqa: E731
    cat = lambda xs: np.concatenate(xs) if xs else np.zeros(0, np.int64)  # noqa: E731
    return PlannerResult(
        n_b=n_b, refs=refs, live_total=live_total, allocated=allocated, eligible=eligible,
        triggered=bool(triggered), src_count=i32(src_count), moved_live=moved_live, need=need,
        token_slot=i32(token_slot), live_count=i32(live_count), admitted=i32(admitted),
        dst_indptr=i32(dst_indptr), new_bt_indptr=i32(new_bt_indptr),
        new_block_ids=i32(cat(new_tables)), src_plan=i32(src_plan),
        freed_indptr=i32(freed_indptr), freed=i32(cat(freed_lists)), used=used,
        n_admitted=int(admitted.sum()), n_freed=int(freed_indptr[-1]),
        tokens_moved=int((moved_live * admitted).sum()), kv=kv_out)


def positional_slots(seq_lens, tok_indptr, bt_indptr, block_ids, S: int) -> np.ndarray:
    """slot_in of a positional layout: logical position p of a request sits at
    block_table[p // S] * S + p % S (Sec. 2.1, Sec. 3.4)."""
    out = np.full(int(tok_indptr[-1]) if len(tok_indptr) else 0, -1, dtype=np.int64)
    for r in range(len(seq_lens)):
        a = int(tok_indptr[r])
        bt = np.asarray(block_ids[bt_indptr[r]:bt_indptr[r + 1]], dtype=np.int64)
        p = np.arange(int(seq_lens[r]))
        out[a:a + len(p)] = bt[p // S] * S + p % S
    return out
