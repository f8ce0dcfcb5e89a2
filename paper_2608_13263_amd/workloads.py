"""Seeded synthetic inputs for the KV repack: paged caches, block tables and liveness.

This module only builds inputs. It holds none of the repack's arithmetic (no scan, no
admission, no packing); both the HIP path and the CPU oracle take its arrays as given.

The paper evaluates on ShareGPT / LongBench prompts with Llama-3.1-8B and Mistral-7B
(Sec. 5.1). Those datasets and models are not used here: the generators below reproduce
the shapes that matter to the repack - the KV geometry, request-length mix, physical
scatter of blocks in the pool, and the liveness pattern an eviction policy leaves
behind (Random, H2O, Scissorhands; Sec. 2.2 and the policy-adapter figure of Sec. 4).

Physical scatter: the block pool is a seeded permutation of [0, num_blocks); requests
take consecutive chunks of it as block tables and the rest, in permuted order, is the
free list. Lengths are integer-uniform and inclusive. Seeds go into numpy's PCG64.
"""
from __future__ import annotations

import dataclasses
import collections
import math
from typing import Callable, Dict, List, Optional, Sequence

import numpy as np

__all__ = [
    "KVShape",
    "RepackInputs",
    "CONFIGS",
    "make",
    "from_masks",
    "tiny_cache",
    "llama3_8b_random",
    "llama3_8b_h2o",
    "llama3_70b_h2o",
    "ScissorhandsStream",
    "next_wave",
    "kv_host",
    "kv_device",
    "bernoulli_live",
    "random_live",
    "h2o_live",
    "slot_limit_inputs",
]


@dataclasses.dataclass(frozen=True)
class KVShape:
    """Geometry of a paged KV cache (Sec. 2.1: per-token bytes 2*L*H*D*dtype)."""

    num_layers: int
    num_kv_heads: int
    head_dim: int
    block_size: int
    dtype: str  # "fp16", "bf16" or "fp8_e4m3"

    @property
    def elem_bytes(self) -> int:
        return {"fp16": 2, "bf16": 2, "fp8_e4m3": 1}[self.dtype]

    @property
    def row_bytes(self) -> int:
        """Bytes of one token's row in one plane: H * D * elem_bytes."""
        return self.num_kv_heads * self.head_dim * self.elem_bytes

    @property
    def num_planes(self) -> int:
        """Planes of the cache: one K and one V plane per layer."""
        return 2 * self.num_layers

    @property
    def token_bytes(self) -> int:
        """KV bytes of one token over all layers, K and V (Sec. 2.1)."""
        return self.num_planes * self.row_bytes

    @property
    def block_bytes(self) -> int:
        """Bytes one block id stands for over all planes."""
        return self.token_bytes * self.block_size


@dataclasses.dataclass
class RepackInputs:
    """One batch of requests over one paged pool (host arrays, CSR layout)."""

    name: str
    shape: KVShape
    num_blocks: int
    seq_lens: np.ndarray   # int32 [R]
    tok_indptr: np.ndarray  # int32 [R+1]
    bt_indptr: np.ndarray   # int32 [R+1]
    block_ids: np.ndarray   # int32 [M]
    live: np.ndarray        # uint8 [T]
    free_list: np.ndarray   # int32 [f]
    seed: int = 0
    note: str = ""
    # token-table inputs of the partial pass: current slot of every token (-1: none) and
    # blocks the caller protects; None for a positional layout
    slot_in: Optional[np.ndarray] = None   # int32 [T]
    pinned: Optional[np.ndarray] = None    # uint8 [num_blocks]

    def slots(self) -> np.ndarray:
        """slot_in, or the positional slots block_table[p // S] * S + p % S (Sec. 3.4)."""
        if self.slot_in is not None:
            return self.slot_in
        S = self.shape.block_size
        out = np.empty(self.num_tokens, dtype=np.int32)
        for r in range(self.num_reqs):
            a, n = int(self.tok_indptr[r]), int(self.seq_lens[r])
            bt = self.request_blocks(r).astype(np.int64)
            p = np.arange(n)
            out[a:a + n] = bt[p // S] * S + p % S
        return out

    @property
    def num_reqs(self) -> int:
        return int(self.seq_lens.shape[0])

    @property
    def num_tokens(self) -> int:
        return int(self.live.shape[0])

    @property
    def num_bt_entries(self) -> int:
        return int(self.block_ids.shape[0])

    def request_live(self, r: int) -> np.ndarray:
        return self.live[self.tok_indptr[r]:self.tok_indptr[r + 1]]

    def request_blocks(self, r: int) -> np.ndarray:
        return self.block_ids[self.bt_indptr[r]:self.bt_indptr[r + 1]]

    def pool_bytes(self) -> int:
        return self.num_blocks * self.shape.block_bytes


def _blocks_for(n: int, block_size: int) -> int:
    # a request of n tokens occupies ceil(n / S) blocks of a paged layout (Sec. 2.1)
    return (int(n) + block_size - 1) // block_size


def _assemble(name: str, shape: KVShape, rng: np.random.Generator, seq_lens: Sequence[int],
              masks: Sequence[np.ndarray], free_blocks: int, seed: int,
              note: str = "") -> RepackInputs:
    """Lay requests out in a shuffled pool of len(tables) + free_blocks blocks."""
    S = shape.block_size
    seq_lens = np.asarray(seq_lens, dtype=np.int64)
    blocks_per_req = np.array([_blocks_for(n, S) for n in seq_lens], dtype=np.int64)
    M = int(blocks_per_req.sum())
    num_blocks = M + int(free_blocks)
    perm = rng.permutation(num_blocks).astype(np.int32)
    tok_indptr = np.zeros(len(seq_lens) + 1, dtype=np.int64)
    tok_indptr[1:] = np.cumsum(seq_lens)
    bt_indptr = np.zeros(len(seq_lens) + 1, dtype=np.int64)
    bt_indptr[1:] = np.cumsum(blocks_per_req)
    live = np.concatenate([np.asarray(m, dtype=np.uint8) for m in masks]) if len(masks) else \
        np.zeros(0, dtype=np.uint8)
    assert live.shape[0] == tok_indptr[-1]
    return RepackInputs(
        name=name, shape=shape, num_blocks=num_blocks,
        seq_lens=seq_lens.astype(np.int32), tok_indptr=tok_indptr.astype(np.int32),
        bt_indptr=bt_indptr.astype(np.int32), block_ids=perm[:M].copy(),
        live=live, free_list=perm[M:].copy(), seed=seed, note=note)


# ----------------------------------------------------------------------------------------
# Liveness stand-ins for the eviction policies the paper evaluates (Sec. 2.2, Sec. 4).
# ----------------------------------------------------------------------------------------

def bernoulli_live(rng: np.random.Generator, n: int, keep: float, sink: int = 0) -> np.ndarray:
    """Each token live with probability `keep`; the first `sink` tokens always live."""
    live = (rng.random(n) < keep).astype(np.uint8)
    live[:min(sink, n)] = 1
    return live


def random_live(rng: np.random.Generator, n: int, keep: float, recent: int) -> np.ndarray:
    """Random policy: floor(keep*n) victims-survivors sampled uniformly without replacement
    from the evictable range [0, n - recent), plus the last `recent` tokens live."""
    live = np.zeros(n, dtype=np.uint8)
    evictable = max(n - recent, 0)
    k = min(int(math.floor(keep * n)), evictable)
    if k > 0:
        live[rng.choice(evictable, size=k, replace=False)] = 1
    live[evictable:] = 1
    return live


def h2o_live(rng: np.random.Generator, n: int, keep: float, recent: int,
             zipf_s: float = 1.1) -> np.ndarray:
    """H2O-style: cumulative attention hits drawn as n samples of a Zipf(s) law over
    positions (P(p) proportional to (p+1)^-s); keep the top floor(keep*n) positions of
    [0, n - recent) by (hits desc, position asc), plus the last `recent` tokens."""
    live = np.zeros(n, dtype=np.uint8)
    evictable = max(n - recent, 0)
    if n > 0:
        w = np.arange(1, n + 1, dtype=np.float64) ** (-zipf_s)
        hits = np.bincount(rng.choice(n, size=n, p=w / w.sum()), minlength=n)
        k = min(int(math.floor(keep * n)), evictable)
        if k > 0:
            pos = np.arange(evictable)
            order = np.lexsort((pos, -hits[:evictable]))
            live[order[:k]] = 1
    live[evictable:] = 1
    return live


# ----------------------------------------------------------------------------------------
# The workloads.
# ----------------------------------------------------------------------------------------

def tiny_cache(seed: int = 101) -> RepackInputs:
    """1 layer, 2 KV heads, head_dim 64, fp16, block 16; 8 requests of U[100,500] tokens in a
    shuffled 512-block pool; Bernoulli(0.5) liveness with the first 4 tokens live."""
    rng = np.random.Generator(np.random.PCG64(seed))
    shape = KVShape(1, 2, 64, 16, "fp16")
    lens = rng.integers(100, 500, size=8, endpoint=True)
    masks = [bernoulli_live(rng, int(n), 0.5, sink=4) for n in lens]
    M = sum(_blocks_for(n, 16) for n in lens)
    return _assemble("tiny", shape, rng, lens, masks, 512 - M, seed,
                     "fp16 1x2x64, S=16, 8 req U[100,500], Bernoulli 0.5 + 4 sink, 512-block pool")


def llama3_8b_random(seed: int = 201, num_reqs: int = 64, num_layers: int = 32,
                     len_range=(2048, 8192), keep: float = 0.3, recent: int = 64,
                     slack_blocks: int = 1024, pool_bytes: Optional[int] = None,
                     block_size: int = 16) -> RepackInputs:
    """Llama-3-8B KV geometry (32 layers, 8 KV heads, head_dim 128, bf16, block 16 unless
    `block_size` says otherwise); 64 requests of U[2048,8192] tokens; Random policy keeping 30%
    of the evictable tokens plus the last 64. The free pool holds keep*M + R*(recent/S + 1) +
    slack blocks, or, with `pool_bytes`, every block of a pool of that size (a serving engine's
    whole KV cache) that the requests do not hold."""
    rng = np.random.Generator(np.random.PCG64(seed))
    S = int(block_size)
    shape = KVShape(num_layers, 8, 128, S, "bf16")
    lens = rng.integers(len_range[0], len_range[1], size=num_reqs, endpoint=True)
    masks = [random_live(rng, int(n), keep, recent) for n in lens]
    M = sum(_blocks_for(n, S) for n in lens)
    free = int(math.ceil(keep * M)) + num_reqs * (recent // S + 1) + slack_blocks
    note = ""
    if pool_bytes is not None:
        free = max(free, int(pool_bytes // shape.block_bytes) - M)
        note = f", {(M + free) * shape.block_bytes / 2**30:.0f} GiB pool"
    name = "llama3_8b_random" if S == 16 else f"llama3_8b_random_s{S}"
    return _assemble(name, shape, rng, lens, masks, free, seed,
                     f"bf16 {num_layers}x8x128, S={S}, {num_reqs} req U{list(len_range)}, "
                     f"Random keep {keep} + last {recent}{note}")


def llama3_8b_h2o(seed: int = 301, num_reqs: int = 128, num_layers: int = 32,
                  len_range=(4096, 16384), keep: float = 0.2, recent: int = 128,
                  slack_blocks: int = 1024) -> RepackInputs:
    """Llama-3-8B geometry; 128 requests of U[4096,16384] tokens; H2O-style liveness: Zipf(1.1)
    attention hits, top 20% by score plus a 128-token recent window."""
    rng = np.random.Generator(np.random.PCG64(seed))
    shape = KVShape(num_layers, 8, 128, 16, "bf16")
    lens = rng.integers(len_range[0], len_range[1], size=num_reqs, endpoint=True)
    masks = [h2o_live(rng, int(n), keep, recent) for n in lens]
    M = sum(_blocks_for(n, 16) for n in lens)
    free = int(math.ceil(keep * M)) + num_reqs * (recent // 16 + 1) + slack_blocks
    return _assemble("llama3_8b_h2o", shape, rng, lens, masks, free, seed,
                     f"bf16 {num_layers}x8x128, S=16, {num_reqs} req U{list(len_range)}, "
                     f"H2O Zipf(1.1) keep {keep} + last {recent}")


def llama3_70b_h2o(seed: int = 501, keep: float = 0.3, dtype: str = "fp8_e4m3",
                   num_reqs: int = 32, num_layers: int = 80, num_kv_heads: int = 8,
                   len_range=(16384, 65536), recent: int = 128,
                   pool_bytes: Optional[int] = None, resident_frac: float = 0.8) -> RepackInputs:
    """Llama-3-70B KV geometry (80 layers, 8 KV heads, head_dim 128, block 32) in fp8 (OCP
    e4m3) or bf16; up to 32 requests of U[16384,65536] tokens; H2O-style Zipf liveness at
    keep ratio k plus the last 128 tokens.

    The literal batch does not fit one GPU (bf16 averages ~400 GiB resident). Fit rule: with
    a device budget `pool_bytes`, keep the longest request prefix whose blocks take at most
    `resident_frac` of the pool; every remaining block is free."""
    rng = np.random.Generator(np.random.PCG64(seed))
    shape = KVShape(num_layers, num_kv_heads, 128, 32, dtype)
    lens = rng.integers(len_range[0], len_range[1], size=num_reqs, endpoint=True)
    if pool_bytes is None:
        pool_blocks = sum(_blocks_for(n, 32) for n in lens) * 2
    else:
        pool_blocks = int(pool_bytes // shape.block_bytes)
    keep_n, used = 0, 0
    for n in lens:
        b = _blocks_for(n, 32)
        if used + b > resident_frac * pool_blocks:
            break
        keep_n += 1
        used += b
    lens = lens[:keep_n]
    masks = [h2o_live(rng, int(n), keep, recent) for n in lens]
    heads = "" if num_kv_heads == 8 else f"_h{num_kv_heads}"
    return _assemble(f"llama3_70b_h2o_{dtype}_k{keep}{heads}", shape, rng, lens, masks,
                     pool_blocks - used, seed,
                     f"{dtype} {num_layers}x{num_kv_heads}x128, S=32, {keep_n} of {num_reqs} "
                     f"req U{list(len_range)}, H2O keep {keep} + last {recent}")


def next_wave(inp: RepackInputs, admitted, live_count, new_bt_indptr, new_block_ids,
              used: int, freed) -> RepackInputs:
    """The caller's side between two passes over one batch ("waves"): apply a pass's outputs
    and re-submit. A repacked request keeps only its live tokens, in order, all live, in its
    new block table; every other request is unchanged; the free list becomes the unconsumed
    entries followed by the freed blocks. A pool too small for every destination at once
    defers the later requests (prefix admission) to the next wave."""
    R = inp.num_reqs
    admitted = np.asarray(admitted)[:R]
    live_count = np.asarray(live_count, dtype=np.int64)[:R]
    new_bt_indptr = np.asarray(new_bt_indptr, dtype=np.int64)
    new_block_ids = np.asarray(new_block_ids, dtype=np.int32)
    lens, masks, tables = [], [], []
    for r in range(R):
        if admitted[r]:
            n = int(live_count[r])
            lens.append(n)
            masks.append(np.ones(n, dtype=np.uint8))
            tables.append(new_block_ids[new_bt_indptr[r]:new_bt_indptr[r + 1]])
        else:
            lens.append(int(inp.seq_lens[r]))
            masks.append(inp.request_live(r))
            tables.append(inp.request_blocks(r))
    seq_lens = np.asarray(lens, dtype=np.int64)
    tok_indptr = np.zeros(R + 1, dtype=np.int64)
    tok_indptr[1:] = np.cumsum(seq_lens)
    bt_indptr = np.zeros(R + 1, dtype=np.int64)
    bt_indptr[1:] = np.cumsum([len(t) for t in tables])
    free = np.concatenate([np.asarray(inp.free_list, dtype=np.int32)[int(used):],
                           np.asarray(freed, dtype=np.int32)])
    return RepackInputs(
        name=inp.name, shape=inp.shape, num_blocks=inp.num_blocks,
        seq_lens=seq_lens.astype(np.int32), tok_indptr=tok_indptr.astype(np.int32),
        bt_indptr=bt_indptr.astype(np.int32),
        block_ids=(np.concatenate(tables) if tables else np.zeros(0)).astype(np.int32),
        live=(np.concatenate(masks) if masks else np.zeros(0)).astype(np.uint8),
        free_list=free.astype(np.int32), seed=inp.seed, note=inp.note)


def from_masks(masks: Sequence[Sequence[int]], shape: KVShape, free_blocks: int,
               seed: int = 0, name: str = "custom") -> RepackInputs:
    """Inputs from explicit per-request live masks (edge cases: empty, all-dead, ragged)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    masks = [np.asarray(m, dtype=np.uint8) for m in masks]
    return _assemble(name, shape, rng, [len(m) for m in masks], masks, free_blocks, seed)


class ScissorhandsStream:
    """Scissorhands-style repeated repack over a long decode (Sec. 2.2; policy figure, Sec. 4).

    The caller's side of a serving loop, as inputs for the repack:
      decode()   every request appends `decode_steps` tokens (blocks from the front of the
                 free list once its last block is full), each resident live token's
                 persistence score grows by Binomial(decode_steps, min(1, 1/sqrt(1+age))),
                 and liveness keeps the top floor(budget * L) - |window| live non-window
                 tokens by (score desc, logical position asc) plus the live tokens of the last
                 `window` positions; everything else is evicted. An evicted token stays dead.
      inputs()   the current layout as RepackInputs (a request's tokens in slot order).
      commit()   apply one pass's outputs: repacked requests keep only their live tokens, in
                 order, in their new block table; the free list becomes the unconsumed
                 entries followed by the freed blocks.
    A round is decode() followed by passes ("waves") until a pass repacks nothing: a pool
    too small for every destination at once defers the later requests to the next wave.

    Initial state (before the first round): logical length L0 ~ U[len_range] - decode_steps; the
    request was packed by the previous round, holding a sorted random subset of
    [0, L0 - window) of size floor(budget * L0) - window plus the window [L0 - window, L0),
    with persistence scores Binomial(2 * decode_steps, min(1, 1/sqrt(1+age))).
    The pool has `pool_blocks` blocks (default: twice the resident blocks), shuffled.
    """

    def __init__(self, seed: int = 401, num_reqs: int = 256, num_layers: int = 32,
                 len_range=(2048, 32768), budget: float = 0.25, window: int = 256,
                 decode_steps: int = 512, pool_blocks: Optional[int] = None,
                 num_kv_heads: int = 8, head_dim: int = 128, block_size: int = 16):
        self.rng = np.random.Generator(np.random.PCG64(seed))
        self.seed = seed
        self.shape = KVShape(num_layers, num_kv_heads, head_dim, block_size, "bf16")
        self.budget, self.window, self.decode_steps = budget, window, decode_steps
        S = block_size
        L_end = self.rng.integers(len_range[0], len_range[1], size=num_reqs, endpoint=True)
        self.L = (L_end - decode_steps).astype(np.int64)
        self.pos: List[np.ndarray] = []
        self.score: List[np.ndarray] = []
        self.alive: List[np.ndarray] = []
        for L0 in self.L:
            L0 = int(L0)
            older = max(L0 - window, 0)
            kept = min(max(int(math.floor(budget * L0)) - window, 0), older)
            sel = np.sort(self.rng.choice(older, size=kept, replace=False)) if kept else \
                np.zeros(0, dtype=np.int64)
            pos = np.concatenate([sel.astype(np.int64), np.arange(older, L0, dtype=np.int64)])
            p = np.minimum(1.0, 1.0 / np.sqrt(1.0 + (L0 - pos)))
            self.pos.append(pos)
            self.score.append(self.rng.binomial(2 * decode_steps, p).astype(np.int64))
            self.alive.append(np.ones(len(pos), dtype=bool))
        resident = sum(_blocks_for(len(p), S) for p in self.pos)
        self.num_blocks = int(pool_blocks) if pool_blocks is not None else 2 * resident
        if self.num_blocks < resident:
            raise ValueError("pool smaller than the resident blocks")
        perm = self.rng.permutation(self.num_blocks).astype(np.int32)
        self.tables: List[np.ndarray] = []
        o = 0
        for pos in self.pos:
            b = _blocks_for(len(pos), S)
            self.tables.append(perm[o:o + b].copy())
            o += b
        self.free = perm[o:].copy()
        self.round = 0
        self.wave = 0

    def decode(self) -> None:
        S = self.shape.block_size
        free = list(self.free)
        for r in range(len(self.pos)):
            L = int(self.L[r])
            fresh = np.arange(L, L + self.decode_steps, dtype=np.int64)
            self.pos[r] = np.concatenate([self.pos[r], fresh])
            self.score[r] = np.concatenate([self.score[r], np.zeros(len(fresh), np.int64)])
            self.alive[r] = np.concatenate([self.alive[r], np.ones(len(fresh), dtype=bool)])
            grow = _blocks_for(len(self.pos[r]), S) - len(self.tables[r])
            if grow > len(free):
                raise RuntimeError("pool exhausted while appending decoded tokens")
            if grow > 0:
                self.tables[r] = np.concatenate([self.tables[r],
                                                 np.asarray(free[:grow], dtype=np.int32)])
                free = free[grow:]
            L += self.decode_steps
            self.L[r] = L
            pos, alive = self.pos[r], self.alive[r]
            p = np.minimum(1.0, 1.0 / np.sqrt(1.0 + (L - pos)))
            self.score[r] = self.score[r] + np.where(alive, self.rng.binomial(
                self.decode_steps, p), 0)
            win = alive & (pos >= L - self.window)
            cand = np.nonzero(alive & ~win)[0]
            k = max(int(math.floor(self.budget * L)) - int(win.sum()), 0)
            new_alive = win.copy()
            if k > 0 and len(cand):
                order = np.lexsort((pos[cand], -self.score[r][cand]))
                new_alive[cand[order[:k]]] = True
            self.alive[r] = new_alive
        self.free = np.asarray(free, dtype=np.int32)
        self.round += 1
        self.wave = 0

    def inputs(self) -> RepackInputs:
        seq_lens = np.array([len(p) for p in self.pos], dtype=np.int64)
        tok_indptr = np.zeros(len(seq_lens) + 1, dtype=np.int64)
        tok_indptr[1:] = np.cumsum(seq_lens)
        bt_indptr = np.zeros(len(seq_lens) + 1, dtype=np.int64)
        bt_indptr[1:] = np.cumsum([len(t) for t in self.tables])
        return RepackInputs(
            name="llama3_8b_scissorhands", shape=self.shape, num_blocks=self.num_blocks,
            seq_lens=seq_lens.astype(np.int32), tok_indptr=tok_indptr.astype(np.int32),
            bt_indptr=bt_indptr.astype(np.int32),
            block_ids=np.concatenate(self.tables).astype(np.int32) if self.tables else
            np.zeros(0, np.int32),
            live=np.concatenate(self.alive).astype(np.uint8) if self.alive else
            np.zeros(0, np.uint8),
            free_list=self.free.copy(), seed=self.seed,
            note=f"Scissorhands budget {self.budget} window {self.window}, "
                 f"{len(self.pos)} req, round {self.round} wave {self.wave}")

    def commit(self, admitted, new_bt_indptr, new_block_ids, used: int, freed) -> None:
        """Apply one pass's outputs (admitted [R], new tables in CSR, consumed free-list
        entries, freed blocks)."""
        for r in range(len(self.pos)):
            if not admitted[r]:
                continue
            keep = np.nonzero(self.alive[r])[0]
            self.pos[r] = self.pos[r][keep]
            self.score[r] = self.score[r][keep]
            self.alive[r] = np.ones(len(keep), dtype=bool)
            self.tables[r] = np.asarray(new_block_ids[new_bt_indptr[r]:new_bt_indptr[r + 1]],
                                        dtype=np.int32)
        self.free = np.concatenate([self.free[int(used):],
                                    np.asarray(freed, dtype=np.int32)]).astype(np.int32)
        self.wave += 1

    def resident_blocks(self) -> int:
        return sum(len(t) for t in self.tables)


def token_table_inputs(seed: int = 601, shape: Optional[KVShape] = None, num_reqs: int = 64,
                       len_range=(2048, 8192), keep: float = 0.3, recent: int = 64,
                       shared_groups: int = 0, group_size: int = 4, prefix_tokens: int = 0,
                       shuffled_frac: float = 0.5, dropped_frac: float = 0.1,
                       pin_tail: bool = True, free_blocks: Optional[int] = None,
                       name: str = "token_table") -> RepackInputs:
    """Requests as token tables, the input of the partial pass.

    Request r has L_r ~ U[len_range] logical tokens in its own blocks of a shuffled pool,
    positional (token p at block_table[p // S] * S + p % S) except that for a fraction
    `shuffled_frac` of requests the tokens are permuted over the occupied slots (a layout left
    by earlier passes: token order no longer follows table order). Liveness is the Random
    policy (keep a fraction `keep` of the evictable tokens plus the last `recent`); a fraction
    `dropped_frac` of the dead tokens hold no slot any more (-1, their slot left empty).
    `shared_groups` groups of `group_size` requests share their first `prefix_tokens` tokens
    (rounded down to whole blocks): one set of blocks at the front of every member's table,
    every member's first tokens on the same slots, liveness drawn per member. With `pin_tail`
    each request's last table block (where decoding appends) is pinned."""
    rng = np.random.Generator(np.random.PCG64(seed))
    shape = shape or KVShape(2, 8, 128, 16, "bf16")
    S = shape.block_size
    R = int(num_reqs)
    lens = rng.integers(len_range[0], len_range[1], size=R, endpoint=True).astype(np.int64)
    prefix = (int(prefix_tokens) // S) * S
    groups = []
    members = rng.permutation(R)
    for g in range(int(shared_groups)):
        grp = members[g * group_size:(g + 1) * group_size]
        if len(grp) >= 2 and prefix > 0:
            groups.append([int(x) for x in grp])
            lens[grp] = np.maximum(lens[grp], prefix + 1)
    group_of = {r: gi for gi, grp in enumerate(groups) for r in grp}
    own_blocks = [_blocks_for(int(lens[r]) - (prefix if r in group_of else 0), S)
                  for r in range(R)]
    M_shared = len(groups) * (prefix // S)
    M_own = int(sum(own_blocks))
    if free_blocks is None:
        free_blocks = int(math.ceil(keep * M_own)) + R * (recent // S + 1) + 256
    num_blocks = M_shared + M_own + int(free_blocks)
    perm = rng.permutation(num_blocks).astype(np.int64)
    o = 0
    shared_tables = []
    for _ in groups:
        shared_tables.append(perm[o:o + prefix // S])
        o += prefix // S
    tables, slots, lives = [], [], []
    for r in range(R):
        n = int(lens[r])
        own = perm[o:o + own_blocks[r]]
        o += own_blocks[r]
        sh = shared_tables[group_of[r]] if r in group_of else perm[:0]
        table = np.concatenate([sh, own])
        p0 = prefix if r in group_of else 0
        pos = np.arange(n - p0)
        own_slots = own[pos // S] * S + pos % S
        if rng.random() < shuffled_frac:
            own_slots = own_slots[rng.permutation(len(own_slots))]
        sl = np.concatenate([sh[np.arange(p0) // S] * S + np.arange(p0) % S, own_slots])
        lv = random_live(rng, n, keep, recent)
        dead = np.nonzero(lv == 0)[0]
        drop = dead[rng.random(len(dead)) < dropped_frac]
        sl = sl.copy()
        sl[drop] = -1
        tables.append(table)
        slots.append(sl)
        lives.append(lv)
    seq_lens = lens.astype(np.int32)
    tok_indptr = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    bt_indptr = np.concatenate([[0], np.cumsum([len(t) for t in tables])]).astype(np.int32)
    pinned = np.zeros(num_blocks, dtype=np.uint8)
    if pin_tail:
        for t in tables:
            if len(t):
                pinned[int(t[-1])] = 1
    return RepackInputs(
        name=name, shape=shape, num_blocks=num_blocks, seq_lens=seq_lens,
        tok_indptr=tok_indptr, bt_indptr=bt_indptr,
        block_ids=np.concatenate(tables).astype(np.int32) if tables else np.zeros(0, np.int32),
        live=np.concatenate(lives).astype(np.uint8) if lives else np.zeros(0, np.uint8),
        free_list=perm[o:].astype(np.int32), seed=seed,
        slot_in=np.concatenate(slots).astype(np.int32) if slots else np.zeros(0, np.int32),
        pinned=pinned,
        note=f"{shape.dtype} {shape.num_layers}x{shape.num_kv_heads}x{shape.head_dim}, S={S}, "
             f"{R} req U{list(len_range)} as token tables ({shuffled_frac:.0%} permuted), "
             f"Random keep {keep} + last {recent}, {len(groups)} shared prefixes of {prefix} "
             f"tokens x {group_size}")


class PartialStream:
    """The Scissorhands-style serving loop of ScissorhandsStream, driven by the partial pass:
    requests are token tables, so a pass can move a few low-utilisation blocks of a request
    and leave the rest in place.

      decode()   as in ScissorhandsStream: `decode_steps` tokens appended per request (into the
                 free slots of its append block, then blocks from the front of the free list,
                 each becoming the append block), persistence scores, eviction to
                 floor(budget * L) plus the window.
      inputs()   the token tables as RepackInputs (slot_in set); every request's append block
                 is pinned.
      commit()   apply one pass's outputs: token slots from the new token table, tokens that
                 lost their slot dropped, the new tables, the free list = unconsumed entries
                 followed by the released sources.
    The initial state is ScissorhandsStream's (same seed, same draws)."""

    def __init__(self, **kw):
        base = ScissorhandsStream(**kw)
        self.base_kw = kw
        self.rng = base.rng
        self.seed = base.seed
        self.shape = base.shape
        self.budget, self.window, self.decode_steps = base.budget, base.window, base.decode_steps
        self.L = base.L
        self.pos, self.score, self.alive = base.pos, base.score, base.alive
        self.tables = [list(int(b) for b in t) for t in base.tables]
        self.num_blocks = base.num_blocks
        self.free = list(int(b) for b in base.free)
        S = self.shape.block_size
        self.slot = []
        self.fill = {}
        self.tail = []
        for pos, t in zip(self.pos, self.tables):
            i = np.arange(len(pos))
            tb = np.asarray(t, dtype=np.int64)
            self.slot.append(tb[i // S] * S + i % S)
            for j, b in enumerate(t):
                self.fill[b] = min(S, len(pos) - j * S)
            self.tail.append(t[-1] if t else None)
        self.round = 0
        self.wave = 0

    def decode(self) -> None:
        S = self.shape.block_size
        for r in range(len(self.pos)):
            L = int(self.L[r])
            new_slots = []
            for _ in range(self.decode_steps):
                last = self.tail[r]
                if last is None or self.fill[last] >= S:
                    if not self.free:
                        raise RuntimeError("pool exhausted while appending decoded tokens")
                    last = self.free.pop(0)
                    self.tables[r].append(last)
                    self.fill[last] = 0
                    self.tail[r] = last
                new_slots.append(last * S + self.fill[last])
                self.fill[last] += 1
            fresh = np.arange(L, L + self.decode_steps, dtype=np.int64)
            self.pos[r] = np.concatenate([self.pos[r], fresh])
            self.slot[r] = np.concatenate([self.slot[r], np.asarray(new_slots, np.int64)])
            self.score[r] = np.concatenate([self.score[r], np.zeros(len(fresh), np.int64)])
            self.alive[r] = np.concatenate([self.alive[r], np.ones(len(fresh), dtype=bool)])
            L += self.decode_steps
            self.L[r] = L
            pos, alive = self.pos[r], self.alive[r]
            p = np.minimum(1.0, 1.0 / np.sqrt(1.0 + (L - pos)))
            self.score[r] = self.score[r] + np.where(alive, self.rng.binomial(
                self.decode_steps, p), 0)
            win = alive & (pos >= L - self.window)
            cand = np.nonzero(alive & ~win)[0]
            k = max(int(math.floor(self.budget * L)) - int(win.sum()), 0)
            new_alive = win.copy()
            if k > 0 and len(cand):
                order = np.lexsort((pos[cand], -self.score[r][cand]))
                new_alive[cand[order[:k]]] = True
            self.alive[r] = new_alive
        self.round += 1
        self.wave = 0

    def inputs(self) -> RepackInputs:
        seq_lens = np.array([len(p) for p in self.pos], dtype=np.int64)
        tok_indptr = np.concatenate([[0], np.cumsum(seq_lens)]).astype(np.int32)
        bt_indptr = np.concatenate([[0], np.cumsum([len(t) for t in self.tables])]).astype(
            np.int32)
        pinned = np.zeros(self.num_blocks, dtype=np.uint8)
        for b in self.tail:
            if b is not None:
                pinned[b] = 1
        return RepackInputs(
            name="llama3_8b_scissorhands_partial", shape=self.shape, num_blocks=self.num_blocks,
            seq_lens=seq_lens.astype(np.int32), tok_indptr=tok_indptr, bt_indptr=bt_indptr,
            block_ids=np.asarray([b for t in self.tables for b in t], dtype=np.int32),
            live=np.concatenate(self.alive).astype(np.uint8) if self.alive else
            np.zeros(0, np.uint8),
            free_list=np.asarray(self.free, dtype=np.int32), seed=self.seed,
            slot_in=np.concatenate(self.slot).astype(np.int32) if self.slot else
            np.zeros(0, np.int32),
            pinned=pinned,
            note=f"Scissorhands budget {self.budget} window {self.window}, {len(self.pos)} req, "
                 f"token tables, round {self.round} wave {self.wave}")

    def commit(self, token_slot, new_bt_indptr, new_block_ids, used: int, sources) -> None:
        """Apply one partial pass's outputs (token table [T], new tables in CSR, consumed
        free-list entries, released sources)."""
        S = self.shape.block_size
        a = 0
        for r in range(len(self.pos)):
            n = len(self.pos[r])
            ts = np.asarray(token_slot[a:a + n], dtype=np.int64)
            a += n
            keep = ts >= 0
            self.pos[r] = self.pos[r][keep]
            self.score[r] = self.score[r][keep]
            self.alive[r] = self.alive[r][keep]
            self.slot[r] = ts[keep]
            old = self.tables[r]
            new = [int(b) for b in new_block_ids[new_bt_indptr[r]:new_bt_indptr[r + 1]]]
            fresh = [b for b in new if b not in set(old)]
            if fresh:
                counts = collections.Counter(int(s) // S for s in self.slot[r])
                for b in fresh:
                    self.fill[b] = counts.get(b, 0)
            self.tables[r] = new
        for b in sources:
            self.fill.pop(int(b), None)
        self.free = self.free[int(used):] + [int(b) for b in sources]
        self.wave += 1

    def resident_blocks(self) -> int:
        return sum(len(t) for t in self.tables)


def block_copy_inputs(shape: KVShape, num_reqs: int, num_blocks: Optional[int] = None,
                      name: str = "block_copy", note: str = "") -> RepackInputs:
    """Reference inputs for the copy's streaming ceiling (not a paper workload): each request
    holds 3 consecutive blocks of which the first two are fully live and the third fully dead,
    and the free list follows them in address order, so a repack copies whole blocks from
    contiguous sources to contiguous destinations. The pool has `num_blocks` blocks (at least
    the 5 per request it needs plus 1024); the blocks past those stay free."""
    S = shape.block_size
    R = int(num_reqs)
    M = 3 * R
    nb = max(M + 2 * R + 1024, int(num_blocks or 0))
    live = np.tile(np.concatenate([np.ones(2 * S, np.uint8), np.zeros(S, np.uint8)]), R)
    return RepackInputs(
        name=name, shape=shape, num_blocks=nb, seq_lens=np.full(R, 3 * S, dtype=np.int32),
        tok_indptr=(np.arange(R + 1) * 3 * S).astype(np.int32),
        bt_indptr=(np.arange(R + 1) * 3).astype(np.int32),
        block_ids=np.arange(M, dtype=np.int32), live=live,
        free_list=np.arange(M, nb, dtype=np.int32), seed=0,
        note=note or f"{R} req of 3 consecutive blocks (2 live, 1 dead), sequential free list")


def llama3_8b_block_copy(num_reqs: int = 3277, num_layers: int = 32,
                         pool_bytes: Optional[int] = None) -> RepackInputs:
    """The block-copy reference in the Llama-3-8B geometry with the bytes of the Llama-3-8B
    Random workload (3,277 requests: 27.5 GB per pass); with `pool_bytes` the pool is that
    large."""
    shape = KVShape(num_layers, 8, 128, 16, "bf16")
    nb = int(pool_bytes // shape.block_bytes) if pool_bytes is not None else None
    inp = block_copy_inputs(shape, num_reqs, nb, name="llama3_8b_block_copy")
    inp.note = (f"bf16 {num_layers}x8x128, S=16, {num_reqs} req of 3 consecutive blocks (2 live, "
                f"1 dead), sequential free list, {inp.num_blocks * shape.block_bytes / 2**30:.0f} "
                f"GiB pool")
    return inp


def llama3_8b_shared_prefix(seed: int = 701, num_reqs: int = 64, num_layers: int = 32,
                            groups: int = 16, group_size: int = 4, prefix_tokens: int = 1024,
                            pool_bytes: Optional[int] = None) -> RepackInputs:
    """Prefix caching (Sec. 5.7) in the Llama-3-8B geometry: 64 requests of U[2048, 8192]
    tokens as token tables, 16 groups of 4 sharing their first 1024 tokens (one set of
    blocks per group, at the front of every member's table), Random keep 0.3 + last 64 drawn
    per request, append blocks pinned. With `pool_bytes` the free list fills a pool that
    large (the same request lengths; placement and liveness are drawn over that pool)."""
    shape = KVShape(num_layers, 8, 128, 16, "bf16")
    kw = dict(seed=seed, shape=shape, num_reqs=num_reqs, len_range=(2048, 8192), keep=0.3,
              recent=64, shared_groups=groups, group_size=group_size,
              prefix_tokens=prefix_tokens, name="llama3_8b_shared_prefix")
    inp = token_table_inputs(**kw)
    if pool_bytes is not None:
        held = inp.num_blocks - len(inp.free_list)
        free = max(int(pool_bytes // shape.block_bytes) - held, len(inp.free_list))
        inp = token_table_inputs(free_blocks=free, **kw)
    inp.note += f", {inp.num_blocks * shape.block_bytes / 2**30:.0f} GiB pool"
    return inp


SLOT_LIMIT = 2 ** 31 - 1   # slots are int32 on the device: num_blocks * S <= 2^31 - 1


def slot_limit_inputs(shape: KVShape, masks: Sequence[Sequence[int]], seed: int,
                      top_block: str = "source", spare: int = 1024,
                      name: str = "slot_limit") -> RepackInputs:
    """The largest pool a cache of block size S can have: num_blocks = (2^31 - 1) // S, so
    slot indices come within S of 2^31. The requests' tables and `spare` free blocks are a
    seeded permutation of the top blocks of the pool; the pool's last block is moved to the
    head of the first request's table (top_block="source") or of the free list
    ("destination")."""
    if top_block not in ("source", "destination"):
        raise ValueError("top_block is 'source' or 'destination'")
    S = shape.block_size
    num_blocks = SLOT_LIMIT // S
    rng = np.random.Generator(np.random.PCG64(seed))
    masks = [np.asarray(m, dtype=np.uint8) for m in masks]
    seq_lens = np.array([len(m) for m in masks], dtype=np.int64)
    M = int(sum(_blocks_for(n, S) for n in seq_lens))
    ids = (num_blocks - (M + spare) + rng.permutation(M + spare)).astype(np.int64)
    i = int(np.nonzero(ids == num_blocks - 1)[0][0])
    j = 0 if top_block == "source" else M
    ids[[i, j]] = ids[[j, i]]
    tok_indptr = np.concatenate([[0], np.cumsum(seq_lens)])
    bt_indptr = np.concatenate([[0], np.cumsum([_blocks_for(n, S) for n in seq_lens])])
    live = np.concatenate(masks) if len(masks) else np.zeros(0, dtype=np.uint8)
    return RepackInputs(
        name=name, shape=shape, num_blocks=num_blocks, seq_lens=seq_lens.astype(np.int32),
        tok_indptr=tok_indptr.astype(np.int32), bt_indptr=bt_indptr.astype(np.int32),
        block_ids=ids[:M].astype(np.int32), live=live, free_list=ids[M:].astype(np.int32),
        seed=seed, note=f"{num_blocks} blocks of {S} slots, tables and free list at the top, "
                        f"last block as {top_block}")


CONFIGS: Dict[str, Callable[..., RepackInputs]] = {
    "tiny": tiny_cache,
    "llama3_8b_random": llama3_8b_random,
    "llama3_8b_h2o": llama3_8b_h2o,
    "llama3_70b_h2o": llama3_70b_h2o,
    "llama3_8b_block_copy": llama3_8b_block_copy,
    "llama3_8b_shared_prefix": llama3_8b_shared_prefix,
}


def make(name: str, **kw) -> RepackInputs:
    return CONFIGS[name](**kw)


# ----------------------------------------------------------------------------------------
# KV payloads. The repack copies opaque bytes; values only matter to the attention check.
# ----------------------------------------------------------------------------------------

def kv_host(shape: KVShape, num_blocks: int, seed: int) -> np.ndarray:
    """Random KV bytes on the host, uint8 [2L][num_blocks*S][row_bytes]."""
    rng = np.random.Generator(np.random.PCG64(seed))
    n = shape.num_planes * num_blocks * shape.block_size * shape.row_bytes
    return rng.integers(0, 256, size=n, dtype=np.uint8).reshape(
        shape.num_planes, num_blocks * shape.block_size, shape.row_bytes)


def torch_dtype(shape: KVShape):
    import torch
    return {"fp16": torch.float16, "bf16": torch.bfloat16,
            "fp8_e4m3": torch.float8_e4m3fn}[shape.dtype]


def kv_device(shape: KVShape, num_blocks: int, seed: int, device="cuda"):
    """KV values ~N(0,1) in the cache dtype on `device`, [2L][num_blocks][S][H][D]
    (fp8 values are N(0,1) draws rounded to OCP e4m3)."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    dims = (shape.num_planes, num_blocks, shape.block_size, shape.num_kv_heads, shape.head_dim)
    out = torch.empty(dims, dtype=torch_dtype(shape), device=device)
    # fill plane by plane to bound the temporary
    for p in range(shape.num_planes):
        if shape.dtype == "fp8_e4m3":
            out[p].copy_(torch.randn(dims[1:], generator=g, device=device,
                                     dtype=torch.float16).to(torch.float8_e4m3fn))
        else:
            out[p].normal_(generator=g)
    return out
