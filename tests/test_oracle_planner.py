"""Pins of the partial-pass oracle and planted mistakes they must catch (CPU only)."""
import os
import sys
import types

import numpy as np
import pytest

import planner_pins
from oracle import planner as P

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle",
                   "planner.py")


@pytest.mark.parametrize("pin", planner_pins.ALL_PINS, ids=lambda p: p.__name__)
def test_planner_oracle_pin(pin):
    pin(P)


MUTATIONS = {
    "waste_non_strict": ("(cap - live_total) * den > num * cap",
                         "(cap - live_total) * den >= num * cap"),
    "utilisation_strict": ("n_b[b] <= max_live", "n_b[b] < max_live"),
    "max_live_off_by_one": ("return (lim - 1) // self.theta_den", "return lim // self.theta_den"),
    "shared_blocks_allowed": ("refs[b] == 1 and not pinned[b]", "refs[b] >= 1 and not pinned[b]"),
    "pins_ignored": ("refs[b] == 1 and not pinned[b]", "refs[b] == 1 and True"),
    "min_eligible_strict": ("eligible >= params.min_eligible", "eligible > params.min_eligible"),
    "watermark_strict": ("len(free_list) <= params.free_watermark",
                         "len(free_list) < params.free_watermark"),
    "profit_non_strict": ("(need < src_count)", "(need <= src_count)"),
    "floor_need": ("need = (moved_live + S - 1) // S", "need = moved_live // S"),
    "dead_keep_slots": ("token_slot[a:e] = np.where(lv, slot_in[a:e], -1)",
                        "token_slot[a:e] = slot_in[a:e]"),
    "destinations_first": ("np.concatenate([[b for b in tables[r] if int(b) not in chosen],\n"
                           "                                          dest])",
                           "np.concatenate([dest, [b for b in tables[r] if int(b) not in "
                           "chosen]])"),
    "freed_unselected": ("freed_lists.append(np.asarray([b for b in tables[r] if int(b) in chosen]",
                         "freed_lists.append(np.asarray([b for b in tables[r] if int(b) not in "
                         "chosen]"),
    "shared_live_counted_twice": ("for s in live_slots:\n        n_b[s // S] += 1",
                                  "for s in live_slots:\n        n_b[s // S] += "
                                  "len(live_slots[s])"),
    "dead_tokens_counted": ("if live[t]:\n                s = int(slot_in[t])",
                            "if live[t] or slot_in[t] >= 0:\n                s = int(slot_in[t])"),
    "budget_ignored": ("k = min(len(eligible_per_req[r]), max(budget, 0))",
                       "k = len(eligible_per_req[r])"),
    "no_deferral": ("admitted[r] = o + need[r] <= len(free_list)", "admitted[r] = True"),
}


def _mutant(name, old, new):
    src = open(SRC).read()
    assert src.count(old) >= 1, f"mutation {name}: pattern not found"
    mod = types.ModuleType(f"planner_mutant_{name}")
    mod.__file__ = SRC
    sys.modules[mod.__name__] = mod
    exec(compile(src.replace(old, new, 1), SRC, "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planner_pins_catch_mutation(name):
    mod = _mutant(name, *MUTATIONS[name])
    for pin in planner_pins.ALL_PINS:
        try:
            if pin is planner_pins.pin_bruteforce:
                pin(mod, cases=200)
            elif pin is planner_pins.pin_invariants:
                pin(mod, cases=150)
            elif pin is planner_pins.pin_full_reduction:
                pin(mod, cases=60)
            else:
                pin(mod)
        except Exception:
            return
    raise AssertionError(f"no pin catches the planted mistake '{name}'")


def test_brute_plan_partial_itself_on_worked_example():
    """The partial pass's brute-force walk is pinned on its own, not only against
    plan_partial: every case of the hand-derived example (tests/golden/partial_example.txt)
    is reproduced output for output, KV moves included."""
    from oracle.bruteforce import brute_plan_partial
    head, cases = planner_pins.read_partial_golden()
    S, nb = int(head["block_size"][0]), int(head["num_blocks"][0])
    masks = [r["live"] for r in head["req"]]
    slots = [r["slots"] for r in head["req"]]
    tables = [r["table"] for r in head["req"]]
    free = [int(x) for x in head["free_list"]]
    pinned = [int(x) for x in head["pinned"]]
    planes = [{s: bytes([s % 251, p]) for s in range(nb * S)} for p in range(2)]
    ints = lambda c, k: [int(x) for x in c[k]]  # noqa: E731
    for c in cases:
        tag = f"brute force, partial example {c['name']}"
        bf = brute_plan_partial([len(m) for m in masks], tables, masks, slots, free, S,
                                theta=c["theta"], max_sources=c["B"],
                                min_eligible=c["min_eligible"], free_watermark=c["watermark"],
                                pinned=pinned, planes=planes)
        assert int(bf["triggered"]) == int(c["triggered"][0]), f"{tag}: triggered"
        assert bf["used"] == int(c["used"][0]), f"{tag}: used"
        flat = {"admitted": bf["admitted"], "src_count": bf["chosen"],
                "token_slot": [s for req in bf["token_slot"] for s in req],
                "src_plan": bf["src_plan"], "freed": bf["freed"],
                "new_block_ids": [b for t in bf["new_tables"] for b in t]}
        for key, got in flat.items():
            if key in c:
                assert [int(x) for x in got] == ints(c, key), f"{tag}: {key}"
        if "new_bt_indptr" in c:
            lens = [0] + [len(t) for t in bf["new_tables"]]
            assert list(np.cumsum(lens)) == ints(c, "new_bt_indptr"), f"{tag}: new tables"
        if "moves" in c:
            expect = [dict(p) for p in planes]
            for mv in c["moves"]:
                old, new = (int(x) for x in mv.split(":"))
                for p in range(2):
                    expect[p][new] = planes[p][old]
            assert bf["planes"] == expect, f"{tag}: KV moves"
