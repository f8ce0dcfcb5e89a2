"""The CPU oracle against its pins (no GPU)."""
import pytest

import oracle.repack as oracle_repack_mod
import oracle_pins


def test_worked_example():
    oracle_pins.pin_worked_example(oracle_repack_mod)


def test_paper_numbers():
    oracle_pins.pin_paper_numbers(oracle_repack_mod)


def test_textbook_reductions():
    oracle_pins.pin_reductions(oracle_repack_mod)


def test_invariants_random():
    oracle_pins.pin_invariants(oracle_repack_mod, cases=300)


def test_bruteforce_exhaustive_and_random():
    oracle_pins.pin_bruteforce(oracle_repack_mod, exhaustive_max_len=9, random_cases=400)


def test_brute_force_itself_on_worked_example():
    """The brute force is pinned too: it reproduces the hand-derived example."""
    from conftest import read_golden
    from oracle.bruteforce import brute_repack
    g = read_golden("worked_example.txt")
    masks = [r["live"] for r in g["req"]]
    tables = [r["table"] for r in g["req"]]
    bf = brute_repack([len(m) for m in masks], tables, masks, [int(x) for x in g["free_list"]],
                      int(g["block_size"][0]))
    assert [s for req in bf["token_slot"] for s in req] == [int(x) for x in g["token_slot"]]
    assert bf["freed"] == [int(x) for x in g["freed"]]
    assert bf["src_plan"] == [int(x) for x in g["src_plan"]]
    assert bf["used"] == int(g["used"][0])


def test_invariant_checker_rejects_bad_packings():
    """The convention-free checker itself catches broken outputs of the worked example."""
    import numpy as np
    from oracle.invariants import check_invariants
    g_res = oracle_pins.run_case
    masks = [[1, 0, 1, 1, 0, 0, 1, 0, 0, 1]]
    tables = [[7, 2, 5]]
    free = [9, 3]
    kv = oracle_pins._kv(2, 16 * 4, 4, 3)
    res = g_res(oracle_repack_mod, masks, tables, free, 4, 16, kv)
    seq_lens, tok_indptr, bt_indptr, block_ids, live = oracle_pins._csr(masks, tables)
    args = (seq_lens, tok_indptr, bt_indptr, block_ids, live, np.asarray(free), 4, 16)

    def check(ts=res.token_slot, nbi=res.new_bt_indptr, nb=res.new_block_ids, fr=res.freed,
              used=res.used, kv_after=res.kv):
        check_invariants(*args, ts, nbi, nb, fr, used, kv, kv_after)

    check()
    bad = res.token_slot.copy(); bad[[0, 2]] = bad[[2, 0]]
    with pytest.raises(AssertionError):
        check(ts=bad)                       # order broken
    bad_kv = res.kv.copy(); bad_kv[1, 37, 0] ^= 1
    with pytest.raises(AssertionError):
        check(kv_after=bad_kv)              # payload changed (I1)
    bad_kv = res.kv.copy(); bad_kv[0, 63, 0] ^= 1
    with pytest.raises(AssertionError):
        check(kv_after=bad_kv)              # a byte outside the moved rows changed
    with pytest.raises(AssertionError):
        check(fr=res.freed[:-1])            # a source block not released


# ---- the full pass's layout precondition (each block id held at most once) ----

def test_check_layout_hand_cases():
    oracle_pins.pin_layout(oracle_repack_mod)


def test_check_layout_on_generated_layouts():
    """Every generated workload is a permutation of the pool split into tables and free list;
    planting one repeated id in any position gives the duplicate code."""
    import numpy as np
    from oracle.repack import check_layout
    from paper_2608_13263_amd import workloads as W
    inp = W.tiny_cache(101)
    assert check_layout(inp.block_ids, inp.free_list, inp.num_blocks) == 0
    rng = np.random.default_rng(4)
    ids = np.concatenate([inp.block_ids, inp.free_list])
    for _ in range(20):
        i, j = rng.choice(len(ids), size=2, replace=False)
        bad = ids.copy()
        bad[j] = bad[i]
        M = len(inp.block_ids)
        assert check_layout(bad[:M], bad[M:], inp.num_blocks) == -14
