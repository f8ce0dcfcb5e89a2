"""Property-based checks of the repack oracle (hypothesis): on generated batches - any
number of requests with any masks, any block size, a shuffled pool and a free list of any
length - the vectorised oracle equals the independent per-token walk of oracle.bruteforce
output for output (KV bytes included), satisfies the convention-free invariants, and its
layout precondition holds on every generated pool."""
import numpy as np
from hypothesis import given, settings
from hypothesis import strategies as st

import oracle.repack as R
import oracle_pins as P
from oracle.invariants import check_invariants


@st.composite
def batches(draw):
    S = draw(st.sampled_from([1, 2, 3, 4, 5, 16]))
    masks = draw(st.lists(st.lists(st.integers(0, 1), max_size=40), max_size=5))
    M = sum(-(-len(m) // S) for m in masks)
    f = draw(st.integers(0, M + 3))
    perm = draw(st.permutations(list(range(M + f))))
    tables, o = [], 0
    for m in masks:
        k = -(-len(m) // S)
        tables.append(perm[o:o + k])
        o += k
    return masks, tables, perm[o:], S, M + f


@settings(max_examples=150, deadline=None)
@given(batches())
def test_oracle_equals_brute_force(case):
    masks, tables, free, S, nb = case
    P._compare_brute(R, masks, tables, free, S, max(nb, 1))


@settings(max_examples=150, deadline=None)
@given(batches())
def test_oracle_invariants_and_layout(case):
    masks, tables, free, S, nb = case
    nb = max(nb, 1)
    seq_lens, tok_indptr, bt_indptr, block_ids, live = P._csr(masks, tables)
    assert R.check_layout(block_ids, free, nb) == R.LAYOUT_OK
    kv = P._kv(2, nb * S, 3, 5)
    res = R.oracle_repack(seq_lens, tok_indptr, bt_indptr, block_ids, live,
                          np.asarray(free, np.int64), S, nb, kv)
    check_invariants(seq_lens, tok_indptr, bt_indptr, block_ids, live, np.asarray(free), S,
                     nb, res.token_slot, res.new_bt_indptr, res.new_block_ids, res.freed,
                     res.used, kv, res.kv)
