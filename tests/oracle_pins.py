"""Pins of the CPU oracle: checks that do not call back into the code they check.

Each pin takes the oracle module to check (oracle.repack, or a copy of it with a planted
mistake) and raises AssertionError when the module disagrees with what the paper or the
mathematics fixes:

  worked_example  hand-derived expected outputs of a 5-request pass (tests/golden)
  paper_numbers   block counts and capacities printed in Sec. 5.4, bytes in Sec. 2.1 and 4
  bruteforce      the independent per-token walk of oracle.bruteforce on tiny inputs
  invariants      convention-free invariants I1, I2, I4 (oracle.invariants)
  reductions      textbook special cases: brute-force counting scan, S=1 stream compaction,
                  all-live identity, all-dead release, the two forms of the waste ratio
"""
from __future__ import annotations

import itertools

import numpy as np

from conftest import read_golden
from oracle.bruteforce import brute_repack
from oracle.invariants import check_invariants


def _csr(masks, tables):
    seq_lens = np.array([len(m) for m in masks], dtype=np.int64)
    tok_indptr = np.concatenate([[0], np.cumsum(seq_lens)]).astype(np.int64)
    bt_indptr = np.concatenate([[0], np.cumsum([len(t) for t in tables])]).astype(np.int64)
    live = np.concatenate([np.asarray(m, np.uint8) for m in masks]) if masks else \
        np.zeros(0, np.uint8)
    block_ids = np.concatenate([np.asarray(t, np.int64) for t in tables]) if tables else \
        np.zeros(0, np.int64)
    if block_ids.size == 0:
        block_ids = np.zeros(0, np.int64)
    return seq_lens, tok_indptr, bt_indptr, block_ids, live


def _kv(num_planes, num_slots, row_bytes, seed):
    rng = np.random.default_rng(seed)
    return rng.integers(0, 256, size=(num_planes, num_slots, row_bytes), dtype=np.uint8)


def random_case(rng, S, max_reqs=3, max_len=12, p_live=None):
    """Random tiny batch: lengths, masks, block tables drawn from a shuffled pool."""
    R = int(rng.integers(0, max_reqs + 1))
    lens = [int(rng.integers(0, max_len + 1)) for _ in range(R)]
    masks = []
    for n in lens:
        p = rng.random() if p_live is None else p_live
        masks.append((rng.random(n) < p).astype(np.uint8))
    m = [(n + S - 1) // S for n in lens]
    extra = int(rng.integers(0, sum(m) + 3))
    nb = sum(m) + extra
    perm = rng.permutation(nb)
    tables, o = [], 0
    for b in m:
        tables.append(list(perm[o:o + b]))
        o += b
    free = list(perm[o:])
    f = int(rng.integers(0, len(free) + 1))
    return masks, tables, free[:f], nb


def run_case(mod, masks, tables, free, S, nb, kv=None):
    seq_lens, tok_indptr, bt_indptr, block_ids, live = _csr(masks, tables)
    return mod.oracle_repack(seq_lens, tok_indptr, bt_indptr, block_ids, live,
                             np.asarray(free, np.int64), S, nb, kv)


# -------------------------------------------------------------------------------------------

def pin_worked_example(mod):
    g = read_golden("worked_example.txt")
    S = int(g["block_size"][0])
    nb = int(g["num_blocks"][0])
    masks = [r["live"] for r in g["req"]]
    tables = [r["table"] for r in g["req"]]
    free = [int(x) for x in g["free_list"]]
    kv = _kv(2, nb * S, 8, 7)
    res = run_case(mod, masks, tables, free, S, nb, kv)
    ints = lambda k: [int(x) for x in g[k]]  # noqa: E731
    for key in ("live_count", "admitted", "dst_indptr", "new_bt_indptr", "new_block_ids",
                "token_slot", "src_plan", "freed_indptr", "freed"):
        got = [int(x) for x in getattr(res, key)]
        assert got == ints(key), f"worked example: {key} = {got}, expected {ints(key)}"
    assert res.used == int(g["used"][0]), "worked example: used"
    assert res.n_admitted == sum(ints("admitted")), "worked example: n_admitted"
    assert res.n_freed == len(ints("freed")), "worked example: n_freed"
    expect = kv.copy()
    for mv in g["moves"]:
        old, new = (int(x) for x in mv.split(":"))
        expect[:, new, :] = kv[:, old, :]
    assert np.array_equal(res.kv, expect), "worked example: KV bytes"


def pin_paper_numbers(mod):
    g = read_golden("paper_numbers.txt")
    v = lambda k: int(g[k][0])  # noqa: E731
    S = v("block_size")
    full, packed = v("full_blocks_per_request"), v("packed_blocks_per_request")
    # a request whose full context fills `full` blocks and whose H2O-retained tokens fill
    # `packed` blocks when packed
    n, c = full * S, packed * S
    rng = np.random.default_rng(5)
    live = np.zeros(n, np.uint8)
    live[rng.choice(n, size=c, replace=False)] = 1
    perm = rng.permutation(full + packed + 4)
    res = run_case(mod, [live], [list(perm[:full])], list(perm[full:]), S, full + packed + 4)
    assert res.new_bt_indptr[1] - res.new_bt_indptr[0] == packed, "packed footprint"
    assert res.n_freed == full, "blocks released"
    assert res.used == packed, "destinations consumed"
    # an all-live request of the same length keeps its full footprint
    res_full = run_case(mod, [np.ones(n, np.uint8)], [list(perm[:full])], list(perm[full:]),
                        S, full + packed + 4)
    assert res_full.new_bt_indptr[1] == full and res_full.n_admitted == 0, "full retention"
    assert mod.capacity_blocks(n, S) == full and mod.capacity_blocks(c, S) == packed
    assert mod.max_concurrency(v("pool_blocks_035"), full) == v("max_c_full_035")
    assert 6 * full == v("six_full_requests_blocks") > v("pool_blocks_035")
    assert mod.max_concurrency(v("pool_blocks_050"), full) == v("max_c_full_050")
    assert mod.max_concurrency(v("pool_blocks_050"), packed) == v("max_c_vtoken_050")
    assert mod.max_concurrency(v("pool_blocks_035"), packed) >= v("min_c_vtoken_035")
    b = mod.kv_bytes_per_token(v("llama13b_layers"), v("llama13b_hidden"),
                               v("llama13b_dtype_bytes"))
    assert abs(b / 1e6 - float(g["llama13b_mb_per_token"][0])) < 0.05, "Sec. 2.1 per-token KV"
    assert b * 32 * 1024 > v("llama13b_gb_at_32k_more_than") * 1e9, "Sec. 2.1 32K context"
    b8 = mod.kv_bytes_per_token(v("llama8b_layers"), v("llama8b_kv_heads") * v("llama8b_head_dim"),
                                2) * v("seq_tokens")
    table = v("entry_bytes") * v("seq_tokens")
    assert table == v("table_kb") * 1024 and table / b8 < 1e-3, "Sec. 4 metadata footprint"
    assert abs(b8 / 2 ** 30 - 2.0) < 0.1, "Sec. 4 ~2 GB fp16 KV at 16K tokens"


def _compare_brute(mod, masks, tables, free, S, nb, with_kv=True):
    P, RB = 2, 3
    kv = _kv(P, nb * S, RB, 11) if with_kv else None
    res = run_case(mod, masks, tables, free, S, nb, kv)
    planes = None
    if with_kv:
        planes = [{s: bytes(kv[p, s]) for s in range(nb * S)} for p in range(P)]
    bf = brute_repack([len(m) for m in masks], tables, masks, free, S, planes)
    ts = [int(x) for x in res.token_slot]
    assert ts == [s for req in bf["token_slot"] for s in req], "brute force: token_slot"
    assert [int(x) for x in res.admitted] == bf["admitted"], "brute force: admitted"
    assert [int(x) for x in res.live_count] == bf["live_count"], "brute force: live_count"
    assert [int(x) for x in res.new_block_ids] == [b for t in bf["new_tables"] for b in t], \
        "brute force: new block tables"
    lens = [len(t) for t in bf["new_tables"]]
    assert [int(x) for x in res.new_bt_indptr] == [0] + list(itertools.accumulate(lens)), \
        "brute force: new_bt_indptr"
    assert [int(x) for x in res.freed] == bf["freed"], "brute force: freed"
    assert res.used == bf["used"], "brute force: used"
    assert [int(x) for x in res.src_plan] == bf["src_plan"], "brute force: src_plan"
    if with_kv:
        for p in range(P):
            got = [bytes(res.kv[p, s]) for s in range(nb * S)]
            assert got == [bf["planes"][p][s] for s in range(nb * S)], "brute force: KV"


def pin_bruteforce(mod, exhaustive_max_len=9, random_cases=300, seed=0):
    # exhaustive single-request masks, every block size, free-list lengths around the need
    for S in (1, 2, 3, 4, 16):
        for n in range(0, exhaustive_max_len + 1):
            m = (n + S - 1) // S
            table = list(range(m))
            pool = list(range(m, 2 * m + 2))
            for bits in itertools.product((0, 1), repeat=n):
                c = sum(bits)
                need = (c + S - 1) // S
                for f in sorted({0, max(need - 1, 0), need, need + 1}):
                    _compare_brute(mod, [list(bits)], [table], pool[:f], S, 2 * m + 2,
                                   with_kv=(n <= 6))
    rng = np.random.default_rng(seed)
    for i in range(random_cases):
        S = int(rng.choice([1, 2, 3, 4, 5, 16]))
        masks, tables, free, nb = random_case(rng, S, max_reqs=4, max_len=14)
        _compare_brute(mod, masks, tables, free, S, nb)


def pin_invariants(mod, cases=200, seed=1):
    rng = np.random.default_rng(seed)
    for i in range(cases):
        S = int(rng.choice([1, 2, 4, 7, 16]))
        masks, tables, free, nb = random_case(rng, S, max_reqs=5, max_len=60)
        kv = _kv(3, nb * S, 4, i)
        res = run_case(mod, masks, tables, free, S, nb, kv)
        seq_lens, tok_indptr, bt_indptr, block_ids, live = _csr(masks, tables)
        check_invariants(seq_lens, tok_indptr, bt_indptr, block_ids, live, np.asarray(free),
                         S, nb, res.token_slot, res.new_bt_indptr, res.new_block_ids,
                         res.freed, res.used, kv, res.kv)
        # with a pool large enough for everyone, every profitable request is repacked, so no
        # request may keep more blocks than its live tokens need (Sec. 3.3.3 minimal count)
        big = list(range(nb, nb + sum(len(t) for t in tables) + 1))
        res2 = run_case(mod, masks, tables, big, S, nb + len(big))
        for r, msk in enumerate(masks):
            c = int(np.sum(msk))
            nbt = res2.new_bt_indptr[r + 1] - res2.new_bt_indptr[r]
            assert nbt == min(len(tables[r]), -(-c // S)), "minimal block count with ample pool"


def pin_reductions(mod, seed=2):
    rng = np.random.default_rng(seed)
    # exclusive scan by brute-force counting
    for n in (0, 1, 2, 5, 64, 200):
        lv = (rng.random(n) < 0.4).astype(np.uint8)
        expect = [sum(int(x) for x in lv[:p]) for p in range(n)]
        assert [int(x) for x in mod.exclusive_live_rank(lv)] == expect, "scan vs counting"
    # S = 1: the packed rows are boolean-mask stream compaction of the live rows
    for trial in range(20):
        n = int(rng.integers(1, 40))
        lv = (rng.random(n) < 0.5).astype(np.uint8)
        lv[0] = 0  # at least one dead token so the plan is profitable
        nb = 2 * n + 1
        perm = rng.permutation(nb)
        table, free = list(perm[:n]), list(perm[n:])
        kv = _kv(2, nb, 5, trial)
        res = run_case(mod, [lv], [table], free, 1, nb, kv)
        new_table = [int(x) for x in res.new_block_ids]
        packed = res.kv[:, new_table, :]
        assert np.array_equal(packed, kv[:, table, :][:, lv.astype(bool), :]), "S=1 compaction"
    # all live: nothing to gain, identity; all dead: every block released, empty table
    for S in (1, 4, 16):
        for n in (0, 1, S, 3 * S + 1):
            m = (n + S - 1) // S
            table = list(range(m))
            free = list(range(m, 2 * m + 1))
            kv = _kv(1, (2 * m + 1) * S, 2, n)
            res = run_case(mod, [np.ones(n, np.uint8)], [table], free, S, 2 * m + 1, kv)
            assert res.n_admitted == 0 and np.array_equal(res.kv, kv), "all-live identity"
            assert [int(x) for x in res.new_block_ids] == table
            res = run_case(mod, [np.zeros(n, np.uint8)], [table], free, S, 2 * m + 1, kv)
            assert res.n_freed == m and res.new_bt_indptr[1] == 0 and res.used == 0, \
                "all-dead release"
            assert res.n_admitted == (1 if m > 0 else 0)
            assert np.array_equal(res.kv, kv), "all-dead moves nothing"
    # waste ratio: 1 - sum(n_i)/(N*S) equals 1 - mean(u_i) with u_i = n_i / S (Sec. 2.3.1)
    for trial in range(10):
        S = int(rng.integers(1, 33))
        n_b = rng.integers(0, S + 1, size=int(rng.integers(1, 50)))
        assert abs(mod.waste_ratio(n_b, S) - (1.0 - float(np.mean(n_b / S)))) < 1e-12
    assert mod.waste_ratio([16, 8, 4, 0], 16) == 1.0 - 28 / 64
    # per-block live counts of a hand-made table
    assert list(mod.block_live_counts([5, 2], [20, 21, 23, 9], 4)) == [3, 1]


def pin_layout(mod):
    """Hand-derived codes of the full pass's layout precondition (0 ok, -10 an id outside
    the pool, reported first, -14 an id held twice)."""
    nb = 10
    cases = [
        ([], [], 0),
        ([0, 1, 2], [3, 4], 0),
        ([0, 1, 1], [3], -14),                          # twice in one table
        ([0, 5], [5, 6], -14),                          # held and free
        ([2], [7, 7], -14),                             # twice in the free list
        ([0, 10], [1], -10),                            # past the pool
        ([0, 1], [-1, 1], -10),                         # negative and a repeat: range first
        ([3], [9], 0),                                  # the pool's last block, once
        ([9, 8, 7, 6, 5, 4, 3, 2, 1, 0], [], 0),        # the whole pool, once each
    ]
    for tables, free, code in cases:
        got = mod.check_layout(tables, free, nb)
        assert got == code, f"check_layout({tables}, {free}) = {got}, expected {code}"


ALL_PINS = (pin_worked_example, pin_paper_numbers, pin_reductions, pin_invariants,
            pin_bruteforce, pin_layout)
