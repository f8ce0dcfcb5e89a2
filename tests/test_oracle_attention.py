"""Pins of the slot-mapping and decode-attention oracle (oracle/attention.py) against facts
the definitions fix, independent of the oracle's own code, plus planted mistakes that the
pins must catch.

  slot mapping   the hand-derived worked example (tests/golden/worked_example.txt, Sec. 3.4:
                 slots of live tokens in logical order) and the per-token brute force
  decode         closed forms: one key -> its value row; equal keys or scale 0 -> mean of the
                 values; two keys -> logistic weight; GQA head h reads KV head h // G; order
                 invariance over the keys; a paged walk over a block table equals the dense
                 sequence it spells; an empty request -> zeros
"""
import os
import sys
import types

import numpy as np
import pytest

from conftest import read_golden
from oracle import attention as A
from oracle.bruteforce import brute_repack
from oracle.repack import oracle_repack

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle",
                   "attention.py")


def _csr(masks, tables):
    seq_lens = [len(m) for m in masks]
    tok_indptr = np.concatenate([[0], np.cumsum(seq_lens)]).astype(np.int64)
    bt_indptr = np.concatenate([[0], np.cumsum([len(t) for t in tables])]).astype(np.int64)
    block_ids = np.asarray([b for t in tables for b in t], dtype=np.int64)
    live = np.asarray([x for m in masks for x in m], dtype=np.uint8)
    return np.asarray(seq_lens, np.int64), tok_indptr, bt_indptr, block_ids, live


def pin_slot_mapping_worked_example(mod):
    g = read_golden("worked_example.txt")
    S, nb = int(g["block_size"][0]), int(g["num_blocks"][0])
    masks = [r["live"] for r in g["req"]]
    tables = [r["table"] for r in g["req"]]
    seq_lens, tok_indptr, bt_indptr, block_ids, live = _csr(masks, tables)
    res = oracle_repack(seq_lens, tok_indptr, bt_indptr, block_ids, live,
                        np.asarray([int(x) for x in g["free_list"]]), S, nb)
    indptr, slots = mod.slot_mapping(res.token_slot, tok_indptr, seq_lens)
    assert [int(x) for x in indptr] == [int(x) for x in g["slot_indptr"]], "slot_indptr"
    assert [int(x) for x in slots] == [int(x) for x in g["slots"]], "slots"


def pin_slot_mapping_bruteforce(mod, cases=200, seed=5):
    rng = np.random.default_rng(seed)
    for _ in range(cases):
        S = int(rng.integers(1, 5))
        R = int(rng.integers(0, 4))
        masks, tables = [], []
        nb = 0
        for _r in range(R):
            n = int(rng.integers(0, 12))
            masks.append([int(x) for x in rng.random(n) < rng.random()])
            m = -(-n // S)
            tables.append(list(range(nb, nb + m)))
            nb += m
        free = list(range(nb, nb + int(rng.integers(0, nb + 2))))
        nb += len(free)
        seq_lens, tok_indptr, bt_indptr, block_ids, live = _csr(masks, tables)
        res = oracle_repack(seq_lens, tok_indptr, bt_indptr, block_ids, live,
                            np.asarray(free, np.int64), S, max(nb, 1))
        brute = brute_repack(seq_lens, tables, masks, free, S)
        indptr, slots = mod.slot_mapping(res.token_slot, tok_indptr, seq_lens)
        expect = [s for ts in brute["token_slot"] for s in ts if s != -1]
        assert [int(x) for x in slots] == expect, "slot mapping differs from the brute force"
        counts = [sum(m) for m in masks]
        assert [int(x) for x in np.diff(indptr)] == counts, "slot counts are the live counts"


def pin_one_key(mod):
    rng = np.random.default_rng(0)
    q = rng.standard_normal((4, 8))
    k = rng.standard_normal((1, 2, 8))
    v = rng.standard_normal((1, 2, 8))
    out = mod.dense_decode(q, k, v)
    for h in range(4):
        assert np.array_equal(out[h], v[0, h // 2]), "one key: output is its value row"


def pin_equal_keys_and_zero_scale(mod):
    rng = np.random.default_rng(1)
    q = rng.standard_normal((2, 6))
    v = rng.standard_normal((5, 1, 6))
    k = np.repeat(rng.standard_normal((1, 1, 6)), 5, axis=0)
    mean = v[:, 0, :].mean(axis=0)
    out = mod.dense_decode(q, k, v)
    assert np.allclose(out, mean[None, :], atol=1e-12), "equal keys: mean of the values"
    k2 = rng.standard_normal((5, 1, 6))
    out0 = mod.dense_decode(q, k2, v, scale=0.0)
    assert np.allclose(out0, mean[None, :], atol=1e-12), "scale 0: mean of the values"


def pin_two_keys_logistic(mod):
    # two keys with scores a and b: weight of the first is 1 / (1 + e^(b - a))
    D = 4
    q = np.array([[1.0, 0.0, 0.0, 0.0]])
    k = np.zeros((2, 1, D))
    k[0, 0, 0], k[1, 0, 0] = 3.0, 1.0
    v = np.zeros((2, 1, D))
    v[0, 0, 1], v[1, 0, 2] = 1.0, 1.0
    scale = 0.5
    a, b = 3.0 * scale, 1.0 * scale
    w0 = 1.0 / (1.0 + np.exp(b - a))
    out = mod.dense_decode(q, k, v, scale=scale)
    assert abs(out[0, 1] - w0) < 1e-14 and abs(out[0, 2] - (1 - w0)) < 1e-14, "two keys"
    out_default = mod.dense_decode(q, k, v)
    w0d = 1.0 / (1.0 + np.exp((1.0 - 3.0) / np.sqrt(D)))
    assert abs(out_default[0, 1] - w0d) < 1e-14, "default scale is 1/sqrt(D)"


def pin_gqa_mapping(mod):
    # KV head j holds values that are all j + 1 and keys that differ per head; query head h
    # must read KV head h // G
    H, G, D, n = 2, 4, 4, 3
    rng = np.random.default_rng(3)
    k = rng.standard_normal((n, H, D))
    v = np.zeros((n, H, D))
    for j in range(H):
        v[:, j, :] = j + 1
    out = mod.dense_decode(rng.standard_normal((H * G, D)), k, v)
    for h in range(H * G):
        assert np.allclose(out[h], h // G + 1), f"GQA: head {h} reads KV head {h // G}"
    # and the keys of that head decide the weights: distinct values per token
    v2 = rng.standard_normal((n, H, D))
    q = rng.standard_normal((H * G, D))
    out2 = mod.dense_decode(q, k, v2)
    for h in range(H * G):
        s = k[:, h // G, :] @ q[h] / np.sqrt(D)
        w = np.exp(s) / np.exp(s).sum()
        assert np.allclose(out2[h], w @ v2[:, h // G, :], atol=1e-12), f"GQA keys, head {h}"


def pin_order_invariance_and_paging(mod):
    rng = np.random.default_rng(4)
    S, H, D, n = 4, 2, 8, 11
    q = rng.standard_normal((2 * H, D))
    k = rng.standard_normal((n, H, D))
    v = rng.standard_normal((n, H, D))
    ref = mod.dense_decode(q, k, v)
    perm = rng.permutation(n)
    assert np.allclose(mod.dense_decode(q, k[perm], v[perm]), ref, atol=1e-12), "order"
    # place the sequence in scattered blocks; the paged walk must read it back
    table = [5, 1, 7]
    kp = rng.standard_normal((8 * S, H, D))
    vp = rng.standard_normal((8 * S, H, D))
    for p in range(n):
        kp[table[p // S] * S + p % S] = k[p]
        vp[table[p // S] * S + p % S] = v[p]
    assert np.allclose(mod.paged_decode(q, kp, vp, table, n, S), ref, atol=1e-12), "paged"
    # and the batched form through a slot mapping, with an empty request in the middle
    slots = [table[p // S] * S + p % S for p in range(n)]
    indptr = [0, n, n, n + 1]
    qb = np.stack([q, q, q])
    out = mod.decode_batch(qb, kp, vp, indptr, slots + [slots[3]])
    assert np.allclose(out[0], ref, atol=1e-12), "batched: first request"
    assert np.array_equal(out[1], np.zeros_like(ref)), "batched: empty request -> zeros"
    for h in range(2 * H):
        assert np.allclose(out[2][h], v[3, h // 2], atol=1e-12), "batched: one-key request"


def pin_slot_table(mod):
    """The append-only slot table: hand-derived layout of the worked example with room for two
    more slots per request; reserve 0 is the packed mapping; appends equal the mapping of the
    extended token table, and a full region is left unchanged."""
    g = read_golden("worked_example.txt")
    S, nb = int(g["block_size"][0]), int(g["num_blocks"][0])
    masks = [r["live"] for r in g["req"]]
    tables = [r["table"] for r in g["req"]]
    seq_lens, tok_indptr, bt_indptr, block_ids, live = _csr(masks, tables)
    res = oracle_repack(seq_lens, tok_indptr, bt_indptr, block_ids, live,
                        np.asarray([int(x) for x in g["free_list"]]), S, nb)
    start, count, slots = mod.slot_table(res.token_slot, tok_indptr, seq_lens, 2)
    assert [int(x) for x in start] == [0, 7, 14, 16, 20, 24], "slot table starts"
    assert [int(x) for x in count] == [5, 5, 0, 2, 2], "slot table counts"
    assert [int(x) for x in slots] == [36, 37, 38, 39, 12, -1, -1, 16, 17, 18, 19, 44, -1, -1,
                                       -1, -1, 48, 49, -1, -1, 56, 63, -1, -1], "slot table"
    i0, p0 = mod.slot_mapping(res.token_slot, tok_indptr, seq_lens)
    s0, c0, t0 = mod.slot_table(res.token_slot, tok_indptr, seq_lens, 0)
    assert list(s0) == list(i0) and list(t0) == list(p0) and list(c0) == list(np.diff(i0))
    new = [[60, 61], [], [62, 63], [50, 51, 52], [53]]     # request 3 overflows (2 + 3 > 4)
    cnt, sl, overflow = mod.append_to_table(start, count, slots, new)
    assert overflow, "a full region must be reported"
    assert [int(x) for x in cnt] == [7, 5, 2, 2, 3], "counts after the appends"
    flat = [[int(x) for x in sl[start[r]:start[r] + cnt[r]]] for r in range(5)]
    assert flat == [[36, 37, 38, 39, 12, 60, 61], [16, 17, 18, 19, 44], [62, 63], [48, 49],
                    [56, 63, 53]], "appended regions"


ALL_PINS = [pin_slot_mapping_worked_example, pin_slot_mapping_bruteforce, pin_slot_table,
            pin_one_key,
            pin_equal_keys_and_zero_scale, pin_two_keys_logistic, pin_gqa_mapping,
            pin_order_invariance_and_paging]


@pytest.mark.parametrize("pin", ALL_PINS, ids=lambda p: p.__name__)
def test_attention_oracle_pin(pin):
    pin(A)


MUTATIONS = {
    "no_scale": ("s = (k[:, h // G, :] @ q[h]) * scale", "s = k[:, h // G, :] @ q[h]"),
    "scale_sqrt_missing": ("scale = 1.0 / np.sqrt(D) if", "scale = 1.0 / D if"),
    "gqa_modulo": ("k[:, h // G, :] @ q[h]", "k[:, h % H, :] @ q[h]"),
    "value_head_modulo": ("out[h] = w @ v[:, h // G, :]", "out[h] = w @ v[:, h % H, :]"),
    "no_normalisation": ("w /= w.sum()", "w /= 1.0"),
    "dead_slots_kept": ("live = ts[ts >= 0]", "live = ts"),
    "inclusive_indptr": ("indptr.append(len(slots))", "indptr.append(len(slots) + 1)"),
    "reversed_order": ("slots.extend(int(x) for x in live)",
                       "slots.extend(int(x) for x in live[::-1])"),
    "paged_transposed": ("int(block_table[p // S]) * S + p % S",
                         "int(block_table[p % S]) * S + p // S"),
    "batch_slot_window": ("slots[int(slot_indptr[r]):int(slot_indptr[r + 1])]",
                          "slots[int(slot_indptr[r]):int(slot_indptr[r + 1]) - 1]"),
    "reserve_ignored": ("np.cumsum(counts + reserve)", "np.cumsum(counts)"),
    "append_overwrites": ("slots[start[r] + count[r]:start[r] + count[r] + n] = new",
                          "slots[start[r]:start[r] + n] = new"),
    "append_past_region": ("if count[r] + n > start[r + 1] - start[r]:",
                           "if count[r] + n > start[r + 1] - start[r] + 1:"),
}


def _mutant(name, old, new):
    src = open(SRC).read()
    assert src.count(old) >= 1, f"mutation {name}: pattern not found"
    mod = types.ModuleType(f"attention_mutant_{name}")
    mod.__file__ = SRC
    sys.modules[mod.__name__] = mod
    exec(compile(src.replace(old, new, 1), SRC, "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_attention_pins_catch_mutation(name):
    mod = _mutant(name, *MUTATIONS[name])
    caught = False
    for pin in ALL_PINS:
        try:
            pin(mod)
        except Exception:
            caught = True
            break
    assert caught, f"no pin catches the planted mistake '{name}'"
