"""Vectorised numpy oracle of one vToken repack pass (test infrastructure only).

Every step follows the paper ("vToken", arXiv 2608.13263) in its own order and notation:

  O1  token table scan  - Sec. 3.2 (per-request token table) and Sec. 3.3.3 (live tokens are
                          assigned in logical order): rank(p) = #live tokens before p.
  O2  need and gain     - Sec. 3.3.3: ceil(T_live / S) destination blocks; a plan exists only
                          when it releases more blocks than it consumes (I4, Sec. 3.5).
  O3  admission         - Sec. 3.3.2: a plan is admitted only if the headroom can provide its
                          destinations, otherwise it is deferred.
  O4  token table       - Sec. 3.3.3 sequential fill, each destination block filled before the
                          next; Sec. 3.2 apply_moves; Sec. 3.4 slot = block_id * S + offset.
  O5  copy              - Sec. 3.3 (lazy compaction, out-of-place relocation, Sec. 3.3.2).
  O6  freed blocks      - Sec. 3.3.4: sources go back to the pool after the commit.

Readings of points the paper leaves open (the same readings are frozen in the C header):
destinations are consumed front to back from the free list by requests in ascending
order; every block of a request is a source; an unprofitable or deferred request keeps its
layout; once one profitable request is deferred, later ones are deferred too; dead tokens
map to -1; tail slots of the last destination block and all other bytes keep their prior
contents; freed = all old blocks of admitted requests, requests ascending, table order.

In-place mode (an extension, not in the paper): the destinations of a repacked request are
its own first ceil(T_live / S) blocks instead of free blocks, every profitable request is
repacked (no headroom is needed), and the freed blocks are the tail of its old table. The
token table, fill order and copy are the same (O1, O2, O4, O5); the copy reads every source
before it writes (the definition of a move), whatever order an implementation uses.

KV is handled as opaque bytes: kv[plane, slot, :] is the row of one token in one plane
(plane = 2*layer + {0: K, 1: V}), so the oracle is independent of the element type.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np


class OracleInputError(ValueError):
    """Inputs that violate the paged-layout contract; `reason` names the check."""

    def __init__(self, reason: str, msg: str):
        super().__init__(f"{reason}: {msg}")
        self.reason = reason


@dataclasses.dataclass
class OracleResult:
    token_slot: np.ndarray     # int32 [T]
    live_count: np.ndarray     # int32 [R]
    admitted: np.ndarray       # int32 [R]
    dst_indptr: np.ndarray     # int32 [R+1]
    new_bt_indptr: np.ndarray  # int32 [R+1]
    new_block_ids: np.ndarray  # int32 [new_bt_indptr[R]]
    src_plan: np.ndarray       # int32 [used*S]
    freed_indptr: np.ndarray   # int32 [R+1]
    freed: np.ndarray          # int32 [n_freed]
    used: int
    n_admitted: int
    n_freed: int
    kv: Optional[np.ndarray] = None  # uint8 [P][num_blocks*S][row_bytes] after the pass


def slot_of_position(block_table: np.ndarray, positions: np.ndarray, S: int) -> np.ndarray:
    """Slot of logical positions in a paged layout: the block holding position p is
    block_table[p // S] and its offset is p % S (Sec. 2.1); slot = block_id * S + offset
    (Sec. 3.4)."""
    positions = np.asarray(positions, dtype=np.int64)
    return np.asarray(block_table, dtype=np.int64)[positions // S] * S + positions % S


def exclusive_live_rank(live: np.ndarray) -> np.ndarray:
    """O1: for every position p, the number of live tokens strictly before p."""
    lv = np.asarray(live, dtype=np.int64)
    return np.cumsum(lv) - lv


def plan_requests(live_count: np.ndarray, old_blocks: np.ndarray, free_len: int, S: int):
    """O2 and O3 for all requests.

    need_r       = ceil(c_r / S)                      destinations of a full-request plan
    profitable_r = need_r < m_r                       strict block reduction (I4)
    o_r          = sum of need over earlier profitable requests  (position in the free list)
    admitted_r   = profitable_r and o_r + need_r <= f (headroom can supply all destinations)
    """
    c = np.asarray(live_count, dtype=np.int64)
    m = np.asarray(old_blocks, dtype=np.int64)
    need = (c + S - 1) // S
    profitable = need < m
    e = np.where(profitable, need, 0)
    o = np.concatenate([[0], np.cumsum(e)[:-1]]) if len(e) else np.zeros(0, np.int64)
    admitted = profitable & (o + need <= free_len)
    return need, profitable, admitted, o


def _validate(seq_lens, tok_indptr, bt_indptr, block_ids, live, S, num_blocks):
    R = len(seq_lens)
    if len(tok_indptr) != R + 1 or len(bt_indptr) != R + 1:
        raise OracleInputError("shape", "indptr arrays must have R+1 entries")
    T, M = len(live), len(block_ids)
    for r in range(R):
        n = int(seq_lens[r])
        a, b = int(tok_indptr[r]), int(tok_indptr[r + 1])
        if n < 0 or a < 0 or b > T or b - a != n:
            raise OracleInputError("tok_len", f"request {r}")
        a, b = int(bt_indptr[r]), int(bt_indptr[r + 1])
        if a < 0 or b > M or b - a != (n + S - 1) // S:
            raise OracleInputError("bt_len", f"request {r}")
        bt = np.asarray(block_ids[a:b], dtype=np.int64)
        if len(bt) and (bt.min() < 0 or bt.max() >= num_blocks):
            raise OracleInputError("block_range", f"request {r}")


def oracle_repack(seq_lens, tok_indptr, bt_indptr, block_ids, live, free_list, block_size: int,
                  num_blocks: int, kv: Optional[np.ndarray] = None,
                  inplace: bool = False) -> OracleResult:
    """One repack pass over host arrays; returns every output of the pass.

    kv, if given, is uint8 [P][num_blocks*S][row_bytes] and is not modified; the result
    holds a modified copy. With inplace=True the free list is ignored and each repacked
    request's destinations are its own first blocks (see the module docstring); `used` then
    counts destination blocks."""
    S = int(block_size)
    seq_lens = np.asarray(seq_lens, dtype=np.int64)
    tok_indptr = np.asarray(tok_indptr, dtype=np.int64)
    bt_indptr = np.asarray(bt_indptr, dtype=np.int64)
    block_ids = np.asarray(block_ids, dtype=np.int64)
    live = np.asarray(live, dtype=np.uint8)
    free_list = np.asarray(free_list, dtype=np.int64)
    R = len(seq_lens)
    _validate(seq_lens, tok_indptr, bt_indptr, block_ids, live, S, num_blocks)
    f = len(free_list)

    # O1: per-request exclusive scan of the live mask
    rank = np.full(len(live), -1, dtype=np.int64)
    live_count = np.zeros(R, dtype=np.int64)
    for r in range(R):
        a, b = tok_indptr[r], tok_indptr[r + 1]
        lv = live[a:b] != 0
        rank[a:b] = np.where(lv, exclusive_live_rank(lv), -1)
        live_count[r] = lv.sum()

    # O2 + O3: need, profitability, headroom admission
    old_blocks = bt_indptr[1:] - bt_indptr[:-1]
    need, profitable, admitted, o = plan_requests(live_count, old_blocks, f, S)
    if inplace:
        admitted = profitable  # destinations are the request's own blocks: nothing to defer
    used = int((need * admitted).sum())
    if not inplace:
        consumed = free_list[:used]
        if used and (consumed.min() < 0 or consumed.max() >= num_blocks):
            raise OracleInputError("block_range", "free list")

    # O4: destination tables, token table and source plan
    dst_indptr = np.zeros(R + 1, dtype=np.int64)
    dst_indptr[1:] = np.cumsum(need * admitted)
    new_len = np.where(admitted, need, old_blocks)
    new_bt_indptr = np.zeros(R + 1, dtype=np.int64)
    new_bt_indptr[1:] = np.cumsum(new_len)
    new_block_ids = np.zeros(int(new_bt_indptr[-1]), dtype=np.int64)
    token_slot = np.full(len(live), -1, dtype=np.int64)
    src_plan = np.full(used * S, -1, dtype=np.int64)
    moves_old, moves_new = [], []
    for r in range(R):
        a, b = tok_indptr[r], tok_indptr[r + 1]
        bt = block_ids[bt_indptr[r]:bt_indptr[r + 1]]
        rk = rank[a:b]
        live_pos = np.nonzero(rk >= 0)[0]
        old_slots = slot_of_position(bt, live_pos, S)
        if admitted[r]:
            dest = bt[:need[r]] if inplace else free_list[dst_indptr[r]:dst_indptr[r + 1]]
            new_block_ids[new_bt_indptr[r]:new_bt_indptr[r + 1]] = dest
            new_slots = slot_of_position(dest, rk[live_pos], S)
            token_slot[a + live_pos] = new_slots
            src_plan[dst_indptr[r] * S + rk[live_pos]] = old_slots
            moves_old.append(old_slots)
            moves_new.append(new_slots)
        else:
            new_block_ids[new_bt_indptr[r]:new_bt_indptr[r + 1]] = bt
            token_slot[a + live_pos] = old_slots

    # O6: freed = old blocks of every admitted request (in-place: the ones past its need)
    first_freed = need if inplace else np.zeros(R, dtype=np.int64)
    freed_indptr = np.zeros(R + 1, dtype=np.int64)
    freed_indptr[1:] = np.cumsum((old_blocks - first_freed) * admitted)
    freed = np.concatenate([block_ids[bt_indptr[r] + first_freed[r]:bt_indptr[r + 1]]
                            for r in range(R) if admitted[r]] or [np.zeros(0, np.int64)])

    # O5: out-of-place copy of every live row in every plane
    kv_out = None
    if kv is not None:
        kv_out = kv.copy()
        if moves_old:
            src = np.concatenate(moves_old)
            dst = np.concatenate(moves_new)
            kv_out[:, dst, :] = kv[:, src, :]

    i32 = lambda x: np.asarray(x, dtype=np.int32)  # noqa: E731
    return OracleResult(
        token_slot=i32(token_slot), live_count=i32(live_count), admitted=i32(admitted),
        dst_indptr=i32(dst_indptr), new_bt_indptr=i32(new_bt_indptr),
        new_block_ids=i32(new_block_ids), src_plan=i32(src_plan),
        freed_indptr=i32(freed_indptr), freed=i32(freed), used=used,
        n_admitted=int(admitted.sum()), n_freed=int(freed_indptr[-1]), kv=kv_out)


# Status codes of the layout check (the values of include/vtoken.h's status enum).
LAYOUT_OK, LAYOUT_BLOCK_RANGE, LAYOUT_DUPLICATE = 0, -10, -14


def check_layout(block_ids, free_list, num_blocks: int) -> int:
    """The full pass's layout precondition, checked one id at a time.

    Every block of an admitted request is a source and goes back to the pool after the copy
    (O6; Sec. 3.3.3, Sec. 3.3.4), and destinations are taken from the free list (O3): so each
    block id may be held by at most one block table or free-list entry, or a block would be
    released twice, or written as a destination while a table still holds it (the token
    table's injectivity, I2 of Sec. 3.5). Ids outside [0, num_blocks) are reported first
    (LAYOUT_BLOCK_RANGE), then any id seen twice (LAYOUT_DUPLICATE); else LAYOUT_OK."""
    ids = [int(b) for b in block_ids] + [int(b) for b in free_list]
    for b in ids:
        if b < 0 or b >= num_blocks:
            return LAYOUT_BLOCK_RANGE
    seen = set()
    for b in ids:
        if b in seen:
            return LAYOUT_DUPLICATE
        seen.add(b)
    return LAYOUT_OK


def oracle_repack_inputs(inp, kv: Optional[np.ndarray] = None,
                         inplace: bool = False) -> OracleResult:
    """oracle_repack over a RepackInputs-like object (attribute access only)."""
    return oracle_repack(inp.seq_lens, inp.tok_indptr, inp.bt_indptr, inp.block_ids, inp.live,
                         inp.free_list, inp.shape.block_size, inp.num_blocks, kv, inplace)


def block_live_counts(block_table: np.ndarray, slots_of_live: np.ndarray, S: int) -> np.ndarray:
    """n_b of Sec. 2.3.1 for each block of a table: live tokens whose slot lies in it."""
    bt = np.asarray(block_table, dtype=np.int64)
    blocks = np.asarray(slots_of_live, dtype=np.int64) // S
    counts = {int(b): 0 for b in bt}
    for b in blocks:
        counts[int(b)] += 1
    return np.array([counts[int(b)] for b in bt], dtype=np.int64)


def waste_ratio(n_b: np.ndarray, S: int) -> float:
    """Intra-block waste ratio of Sec. 2.3.1: F = 1 - sum(n_i) / (N * S) over N allocated
    blocks with n_i valid tokens each (0 for an empty allocation)."""
    n_b = np.asarray(n_b, dtype=np.float64)
    if n_b.size == 0:
        return 0.0
    return float(1.0 - n_b.sum() / (n_b.size * S))


def capacity_blocks(num_tokens: int, S: int) -> int:
    """Blocks a request of `num_tokens` resident tokens occupies: ceil(L / B) (Sec. 5.4)."""
    return -(-int(num_tokens) // int(S))


def max_concurrency(pool_blocks: int, blocks_per_request: int) -> int:
    """Largest C with C * blocks_per_request <= pool_blocks (the capacity model of Sec. 5.4)."""
    return int(pool_blocks) // int(blocks_per_request)


def kv_bytes_per_token(num_layers: int, hidden_kv: int, dtype_bytes: int) -> int:
    """KV bytes of one token: 2 * L * (H * D) * dtype_size (Sec. 2.1)."""
    return 2 * int(num_layers) * int(hidden_kv) * int(dtype_bytes)
