"""Pins of the partial-pass oracle (oracle/planner.py), each a function of the module under
test so that planted mistakes (tests/test_oracle_planner.py) can be run through them:

  pin_worked_example   the hand-derived example of tests/golden/partial_example.txt
  pin_full_reduction   with every block a candidate, no bound B and the trigger forced, the
                       partial pass on a positional layout is the full-request pass of
                       oracle/repack.py output for output (an independent oracle pinned on
                       its own)
  pin_bruteforce       the literal per-token walk of oracle/bruteforce.py on random token
                       tables with shared and pinned blocks and random parameters
  pin_invariants       convention-free properties (I1, I2, I4, candidates only, bound B,
                       untouched tokens keep their slots, F does not increase, conservation)
"""
from __future__ import annotations

import hashlib
from collections import Counter
from fractions import Fraction

import numpy as np

from conftest import GOLDEN
from oracle.bruteforce import brute_plan_partial
from oracle.repack import oracle_repack
import os


def read_partial_golden():
    head, cases, cur = {"req": []}, [], None
    with open(os.path.join(GOLDEN, "partial_example.txt")) as fh:
        for line in fh:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *vals = line.split()
            if key == "case":
                cur = {"name": vals[0], "B": int(vals[2]), "theta": (int(vals[4]), int(vals[5])),
                       "watermark": int(vals[7]), "min_eligible": int(vals[9])}
            elif key == "end":
                cases.append(cur)
                cur = None
            elif cur is not None:
                cur[key] = vals
            elif key == "req":
                i, j, k = vals.index("live"), vals.index("slots"), vals.index("table")
                head["req"].append(dict(live=[int(x) for x in vals[i + 1:j]],
                                        slots=[int(x) for x in vals[j + 1:k]],
                                        table=[int(x) for x in vals[k + 1:]]))
            else:
                head[key] = vals
    return head, cases


def csr(masks, slots, tables):
    seq_lens = np.asarray([len(m) for m in masks], np.int64)
    tok_indptr = np.concatenate([[0], np.cumsum(seq_lens)]).astype(np.int64)
    bt_indptr = np.concatenate([[0], np.cumsum([len(t) for t in tables])]).astype(np.int64)
    block_ids = np.asarray([b for t in tables for b in t], np.int64)
    live = np.asarray([x for m in masks for x in m], np.uint8)
    slot_in = np.asarray([x for s in slots for x in s], np.int64)
    return seq_lens, tok_indptr, bt_indptr, block_ids, live, slot_in


def run(mod, masks, slots, tables, free, S, nb, pinned=(), kv=None, **params):
    seq_lens, tok_indptr, bt_indptr, block_ids, live, slot_in = csr(masks, slots, tables)
    pin = np.zeros(nb, bool)
    pin[list(pinned)] = True
    return mod.plan_partial(seq_lens, tok_indptr, bt_indptr, block_ids, live, slot_in,
                            np.asarray(free, np.int64), S, nb, mod.PlannerParams(**params),
                            pinned=pin, kv=kv)


def pin_worked_example(mod):
    head, cases = read_partial_golden()
    S, nb = int(head["block_size"][0]), int(head["num_blocks"][0])
    masks = [r["live"] for r in head["req"]]
    slots = [r["slots"] for r in head["req"]]
    tables = [r["table"] for r in head["req"]]
    free = [int(x) for x in head["free_list"]]
    pinned = [int(x) for x in head["pinned"]]
    rng = np.random.default_rng(3)
    kv = rng.integers(0, 256, size=(2, nb * S, 8), dtype=np.uint8)
    ints = lambda c, k: [int(x) for x in c[k]]  # noqa: E731
    for c in cases:
        res = run(mod, masks, slots, tables, free, S, nb, pinned, kv, theta_num=c["theta"][0],
                  theta_den=c["theta"][1], max_sources=c["B"], min_eligible=c["min_eligible"],
                  free_watermark=c["watermark"])
        tag = f"partial example {c['name']}"
        if c["theta"] == (1, 4):
            assert res.live_total == int(head["live_total"][0]), f"{tag}: live_total"
            assert res.allocated == int(head["allocated"][0]), f"{tag}: allocated"
            assert res.eligible == int(head["eligible"][0]), f"{tag}: eligible"
        assert int(res.triggered) == int(c["triggered"][0]), f"{tag}: triggered"
        assert res.used == int(c["used"][0]), f"{tag}: used"
        for key in ("src_count", "admitted", "dst_indptr", "token_slot", "src_plan",
                    "new_bt_indptr", "new_block_ids", "freed_indptr", "freed"):
            if key in c:
                got = [int(x) for x in getattr(res, key)]
                assert got == ints(c, key), f"{tag}: {key} = {got}, expected {ints(c, key)}"
        if "moves" in c:
            expect = kv.copy()
            for mv in c["moves"]:
                old, new = (int(x) for x in mv.split(":"))
                expect[:, new, :] = kv[:, old, :]
            assert np.array_equal(res.kv, expect), f"{tag}: KV bytes"


def pin_full_reduction(mod, cases=150, seed=11):
    rng = np.random.default_rng(seed)
    for _ in range(cases):
        S = int(rng.choice([1, 2, 3, 4, 16]))
        R = int(rng.integers(0, 5))
        masks, tables, nb = [], [], 0
        for _r in range(R):
            n = int(rng.integers(0, 40))
            masks.append((rng.random(n) < rng.random()).astype(int).tolist())
            m = -(-n // S)
            tables.append(list(range(nb, nb + m)))
            nb += m
        free = list(range(nb, nb + int(rng.integers(0, nb + 2))))
        nb = max(nb + len(free), 1)
        perm = rng.permutation(nb)
        tables = [[int(perm[b]) for b in t] for t in tables]
        free = [int(perm[b]) for b in free]
        slots = [[t[p // S] * S + p % S for p in range(len(m))] for m, t in zip(masks, tables)]
        kv = rng.integers(0, 256, size=(2, nb * S, 4), dtype=np.uint8)
        seq_lens, tok_indptr, bt_indptr, block_ids, live, _ = csr(masks, slots, tables)
        full = oracle_repack(seq_lens, tok_indptr, bt_indptr, block_ids, live,
                             np.asarray(free, np.int64), S, nb, kv)
        part = run(mod, masks, slots, tables, free, S, nb, (), kv, theta_num=-1, theta_den=1,
                   max_sources=1 << 30, min_eligible=0, free_watermark=-1)
        for key in ("token_slot", "admitted", "dst_indptr", "new_bt_indptr", "new_block_ids",
                    "src_plan", "freed_indptr", "freed", "live_count"):
            a = [int(x) for x in getattr(full, key)]
            b = [int(x) for x in getattr(part, key)]
            assert a == b, f"full reduction: {key} {b} vs full pass {a}"
        assert part.used == full.used, "full reduction: used"
        assert np.array_equal(part.kv, full.kv), "full reduction: KV bytes"


def random_table_case(rng):
    """Random token tables: private blocks with tokens at arbitrary distinct slots (a history
    of earlier passes), optional shared prefix blocks held by several requests, pinned blocks,
    dead tokens with and without slots."""
    S = int(rng.choice([1, 2, 3, 4, 5, 8]))
    R = int(rng.integers(0, 5))
    nb_total = 64
    pool = [int(x) for x in rng.permutation(nb_total)]
    nxt = 0
    shared_tables, shared_slots, shared_live = [], [], []
    if R >= 2 and rng.random() < 0.5:
        k = int(rng.integers(1, 3))
        shared_tables = pool[nxt:nxt + k]
        nxt += k
        ns = int(rng.integers(1, k * S + 1))
        shared_slots = [b * S + o for b in shared_tables for o in range(S)][:ns]
    sharers = set(rng.choice(R, size=min(R, int(rng.integers(2, 4))), replace=False).tolist()) \
        if shared_tables else set()
    masks, slots, tables = [], [], []
    for r in range(R):
        m = int(rng.integers(0, 5))
        own = pool[nxt:nxt + m]
        nxt += m
        cap = [b * S + o for b in own for o in range(S)]
        used = int(rng.integers(0, len(cap) + 1))
        chosen = [cap[i] for i in sorted(rng.choice(len(cap), size=used, replace=False))] \
            if used else []
        if rng.random() < 0.5:
            chosen = [chosen[i] for i in rng.permutation(len(chosen))]  # non-positional
        sl, lv = [], []
        if r in sharers:
            sl += list(shared_slots)
            lv += (rng.random(len(shared_slots)) < 0.7).astype(int).tolist()
        for s in chosen:
            sl.append(s)
            lv.append(int(rng.random() < rng.random()))
        for _ in range(int(rng.integers(0, 3))):       # tokens compacted away earlier
            pos = int(rng.integers(0, len(sl) + 1))
            sl.insert(pos, -1)
            lv.insert(pos, 0)
        masks.append(lv)
        slots.append(sl)
        tables.append((shared_tables if r in sharers else []) + own)
    free = pool[nxt:nxt + int(rng.integers(0, 8))]
    pinned = [b for t in tables for b in t if rng.random() < 0.1]
    theta = [(1, 4), (0, 1), (1, 2), (-1, 1), (3, 4), (2, 3)][int(rng.integers(0, 6))]
    params = dict(theta_num=theta[0], theta_den=theta[1],
                  max_live_per_source=None if rng.random() < 0.6 else int(rng.integers(0, S + 1)),
                  max_sources=int(rng.choice([0, 1, 2, 3, 5, 1 << 30])),
                  min_eligible=int(rng.choice([0, 1, 3])),
                  free_watermark=int(rng.choice([-1, len(free), max(len(free) - 1, 0)])))
    return S, nb_total, masks, slots, tables, free, pinned, params


def pin_bruteforce(mod, cases=400, seed=12):
    rng = np.random.default_rng(seed)
    for _ in range(cases):
        S, nb, masks, slots, tables, free, pinned, params = random_table_case(rng)
        planes = [{s: bytes(rng.integers(0, 256, 4, dtype=np.uint8)) for s in range(nb * S)}
                  for _p in range(2)]
        kv = np.stack([np.stack([np.frombuffer(pl[s], np.uint8) for s in range(nb * S)])
                       for pl in planes])
        res = run(mod, masks, slots, tables, free, S, nb, pinned, kv, **params)
        brute = brute_plan_partial([len(m) for m in masks], tables, masks, slots, free, S,
                                   theta=(params["theta_num"], params["theta_den"]),
                                   max_live=params["max_live_per_source"],
                                   max_sources=params["max_sources"],
                                   min_eligible=params["min_eligible"],
                                   free_watermark=params["free_watermark"], pinned=pinned,
                                   planes=planes)
        tag = f"brute force (S={S}, params={params})"
        assert res.triggered == brute["triggered"], f"{tag}: triggered"
        assert [int(x) for x in res.src_count] == brute["chosen"], f"{tag}: sources"
        assert [int(x) for x in res.admitted] == brute["admitted"], f"{tag}: admitted"
        assert res.used == brute["used"], f"{tag}: used"
        flat = [x for ts in brute["token_slot"] for x in ts]
        assert [int(x) for x in res.token_slot] == flat, f"{tag}: token table"
        tabs = [[int(x) for x in res.new_block_ids[res.new_bt_indptr[r]:res.new_bt_indptr[r + 1]]]
                for r in range(len(masks))]
        assert tabs == brute["new_tables"], f"{tag}: new tables"
        assert [int(x) for x in res.freed] == brute["freed"], f"{tag}: freed"
        assert [int(x) for x in res.src_plan] == brute["src_plan"], f"{tag}: source plan"
        for p, pl in enumerate(brute["planes"]):
            got = [bytes(res.kv[p, s]) for s in range(nb * S)]
            assert got == [pl[s] for s in range(nb * S)], f"{tag}: plane {p}"
        for b, c in brute["count"].items():
            assert res.n_b[b] == c, f"{tag}: n_b of block {b}"


def _waste(tables, live_slots_by_block, S):
    blocks = set(b for t in tables for b in t)
    if not blocks:
        return Fraction(0)
    live = sum(len(live_slots_by_block.get(b, ())) for b in blocks)
    return 1 - Fraction(live, len(blocks) * S)


def pin_invariants(mod, cases=300, seed=13):
    """Properties any valid partial pass has, whatever its conventions."""
    rng = np.random.default_rng(seed)
    for _ in range(cases):
        S, nb, masks, slots, tables, free, pinned, params = random_table_case(rng)
        kv = rng.integers(0, 256, size=(2, nb * S, 4), dtype=np.uint8)
        res = run(mod, masks, slots, tables, free, S, nb, pinned, kv, **params)
        R = len(masks)
        refs = Counter(b for t in tables for b in t)
        lv_by_block = {}
        for m, sl in zip(masks, slots):
            for x, s in zip(m, sl):
                if x:
                    lv_by_block.setdefault(s // S, set()).add(s)
        n_b = {b: len(lv_by_block.get(b, ())) for b in refs}
        new_tables, a = [], 0
        total_sources = 0
        for r in range(R):
            nt = [int(x) for x in res.new_block_ids[res.new_bt_indptr[r]:res.new_bt_indptr[r + 1]]]
            new_tables.append(nt)
            n = len(masks[r])
            ts = [int(x) for x in res.token_slot[a:a + n]]
            h0, h1 = hashlib.sha256(), hashlib.sha256()
            for p in range(n):
                if masks[r][p]:
                    if ts[p] < 0 or ts[p] // S not in nt:
                        raise AssertionError("I2: live token without a slot in its table")
                    h0.update(p.to_bytes(4, "little") + kv[:, slots[r][p]].tobytes())
                    h1.update(p.to_bytes(4, "little") + res.kv[:, ts[p]].tobytes())
                elif ts[p] != -1:
                    raise AssertionError("dead token keeps a slot")
            if h0.digest() != h1.digest():
                raise AssertionError(f"I1: request {r} tokens or payloads changed")
            gone = [b for b in tables[r] if b not in nt]
            if res.admitted[r]:
                if len(nt) >= len(tables[r]):
                    raise AssertionError("I4: repacked request without a block reduction")
                for b in gone:
                    if refs[b] != 1 or b in pinned:
                        raise AssertionError("I4 / Sec. 5.7: a shared or pinned block moved")
                    if n_b[b] > mod.PlannerParams(**params).max_live(S):
                        raise AssertionError("a source above the utilisation bound")
                for p in range(n):
                    if masks[r][p] and slots[r][p] // S not in gone and ts[p] != slots[r][p]:
                        raise AssertionError("a token outside the sources moved")
                total_sources += len(gone)
            elif nt != list(tables[r]) or any(
                    masks[r][p] and ts[p] != slots[r][p] for p in range(n)):
                raise AssertionError("a request that was not repacked changed")
            a += n
        if total_sources > max(params["max_sources"], 0):
            raise AssertionError("more sources than the bound B")
        live_slots = [int(x) for x in res.token_slot if x >= 0]
        owners = Counter(live_slots)
        for s, c in owners.items():
            if c > 1 and refs.get(s // S, 0) < 2:
                raise AssertionError("I2: two tokens share a private slot")
        used = res.used
        dest = Counter(b for r in range(R) if res.admitted[r]
                       for b in new_tables[r] if b not in tables[r])
        if dest != Counter(free[:used]):
            raise AssertionError("destinations are not the consumed free-list entries")
        before = Counter(b for t in tables for b in t) + Counter(free)
        after = Counter(b for t in new_tables for b in t) + Counter(int(x) for x in res.freed) \
            + Counter(free[used:])
        if before != after:
            raise AssertionError("block conservation")
        new_lv = {}
        for s in set(live_slots):
            new_lv.setdefault(s // S, set()).add(s)
        if _waste(new_tables, new_lv, S) > _waste(tables, lv_by_block, S):
            raise AssertionError("the waste ratio increased")
        moved = set(b for r in range(R) if res.admitted[r] for b in tables[r]
                    if b not in new_tables[r])
        touched = np.zeros(nb * S, bool)
        for r in range(R):
            for b in new_tables[r]:
                if b not in tables[r]:
                    touched[b * S:(b + 1) * S] = True
        if not np.array_equal(res.kv[:, ~touched], kv[:, ~touched]):
            raise AssertionError("bytes outside the destination blocks changed")
        assert len(moved) == int(res.freed_indptr[-1])


ALL_PINS = [pin_worked_example, pin_full_reduction, pin_bruteforce, pin_invariants]
