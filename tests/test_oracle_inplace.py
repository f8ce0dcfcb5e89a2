"""The in-place mode of the oracle (destinations = a request's own leading blocks) against
the per-token brute force, the convention-free invariants, and a hand-derived example."""
import itertools

import numpy as np

import oracle.repack as R
import oracle_pins as P
from oracle.bruteforce import brute_repack
from oracle.invariants import check_invariants


def _run(masks, tables, free, S, nb, kv=None):
    seq_lens, tok_indptr, bt_indptr, block_ids, live = P._csr(masks, tables)
    return R.oracle_repack(seq_lens, tok_indptr, bt_indptr, block_ids, live,
                           np.asarray(free, np.int64), S, nb, kv, inplace=True)


def _compare(masks, tables, free, S, nb):
    kv = P._kv(2, nb * S, 3, 21)
    res = _run(masks, tables, free, S, nb, kv)
    planes = [{s: bytes(kv[p, s]) for s in range(nb * S)} for p in range(2)]
    bf = brute_repack([len(m) for m in masks], tables, masks, free, S, planes, inplace=True)
    assert [int(x) for x in res.token_slot] == [s for q in bf["token_slot"] for s in q]
    assert [int(x) for x in res.admitted] == bf["admitted"]
    assert [int(x) for x in res.new_block_ids] == [b for t in bf["new_tables"] for b in t]
    assert [int(x) for x in res.freed] == bf["freed"]
    assert [int(x) for x in res.src_plan] == bf["src_plan"]
    assert res.used == bf["used"]
    for p in range(2):
        assert [bytes(res.kv[p, s]) for s in range(nb * S)] == \
            [bf["planes"][p][s] for s in range(nb * S)]
    seq_lens, tok_indptr, bt_indptr, block_ids, live = P._csr(masks, tables)
    check_invariants(seq_lens, tok_indptr, bt_indptr, block_ids, live, np.asarray(free), S, nb,
                     res.token_slot, res.new_bt_indptr, res.new_block_ids, res.freed, res.used,
                     kv, res.kv, inplace=True)
    return res


def test_inplace_exhaustive_small():
    for S in (1, 2, 3, 4):
        for n in range(0, 9):
            m = (n + S - 1) // S
            for bits in itertools.product((0, 1), repeat=n):
                _compare([list(bits)], [list(range(m))], [], S, m + 1)


def test_inplace_random_multi_request():
    rng = np.random.default_rng(3)
    for _ in range(300):
        S = int(rng.choice([1, 2, 4, 5, 16]))
        masks, tables, free, nb = P.random_case(rng, S, max_reqs=4, max_len=40)
        _compare(masks, tables, free, S, nb)


def test_inplace_hand_example():
    # S = 4, table [7, 2, 5], live 1011001001 (ranks 0..4 at positions 0,2,3,6,9):
    # destinations are blocks 7 and 2; slots 28,29,30,31,8 (position 9 -> rank 4 -> block 2
    # offset 0); sources 28,30,31,10,21; block 5 is released; position 0 stays in place.
    res = _run([[1, 0, 1, 1, 0, 0, 1, 0, 0, 1]], [[7, 2, 5]], [9, 3], 4, 16,
               P._kv(1, 64, 2, 5))
    assert [int(x) for x in res.token_slot] == [28, -1, 29, 30, -1, -1, 31, -1, -1, 8]
    assert [int(x) for x in res.new_block_ids] == [7, 2]
    assert [int(x) for x in res.freed] == [5]
    assert [int(x) for x in res.src_plan] == [28, 30, 31, 10, 21, -1, -1, -1]
    assert res.used == 2 and res.n_admitted == 1


def test_inplace_ignores_free_list_and_admits_every_profitable_request():
    rng = np.random.default_rng(9)
    masks = [list((rng.random(50) < 0.3).astype(int)) for _ in range(5)]
    tables = [list(range(4 * i, 4 * i + 4)) for i in range(5)]
    a = _run(masks, tables, [], 16, 20)
    b = _run(masks, tables, [100, 101], 16, 102)
    assert a.n_admitted == 5 and b.n_admitted == 5
    assert np.array_equal(a.token_slot, b.token_slot)
