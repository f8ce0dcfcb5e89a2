"""Plant plausible mistakes in a copy of the oracle (on the CPU) and show that the pins catch
every one of them: a dropped term, an off-by-one, a wrong comparison, a transposed index,
swapped operands."""
import os
import sys
import types

import pytest

import oracle_pins

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle",
                   "repack.py")

MUTATIONS = {
    "inclusive_scan": ("return np.cumsum(lv) - lv", "return np.cumsum(lv)"),
    "floor_need": ("need = (c + S - 1) // S", "need = c // S"),
    "non_strict_gain": ("profitable = need < m", "profitable = need <= m"),
    "strict_headroom": ("(o + need <= free_len)", "(o + need < free_len)"),
    "no_prefix_offset": ("o = np.concatenate([[0], np.cumsum(e)[:-1]])", "o = np.cumsum(e)"),
    "offset_uses_all_needs": ("e = np.where(profitable, need, 0)", "e = need"),
    "transposed_slot": ("[positions // S] * S + positions % S",
                        "[positions % S] * S + positions // S"),
    "swapped_copy": ("kv_out[:, dst, :] = kv[:, src, :]", "kv_out[:, src, :] = kv[:, dst, :]"),
    "freed_wrong_requests": ("for r in range(R) if admitted[r]]",
                             "for r in range(R) if not admitted[r]]"),
    "plan_new_slots": ("src_plan[dst_indptr[r] * S + rk[live_pos]] = old_slots",
                       "src_plan[dst_indptr[r] * S + rk[live_pos]] = new_slots"),
    "deferred_gets_moved": ("if admitted[r]:\n            dest", "if profitable[r]:\n            dest"),
    "dead_tokens_kept": ("lv = live[a:b] != 0", "lv = live[a:b] >= 0"),
    "layout_ignores_free_list": ("ids = [int(b) for b in block_ids] + [int(b) for b in free_list]",
                                 "ids = [int(b) for b in block_ids]"),
    "layout_upper_bound": ("if b < 0 or b >= num_blocks:", "if b < 0 or b > num_blocks:"),
    "layout_no_negative": ("if b < 0 or b >= num_blocks:", "if b >= num_blocks:"),
}


def _mutant(name, old, new):
    src = open(SRC).read()
    assert src.count(old) >= 1, f"mutation {name}: pattern not found"
    mod = types.ModuleType(f"oracle_mutant_{name}")
    mod.__file__ = SRC
    sys.modules[mod.__name__] = mod
    exec(compile(src.replace(old, new, 1), SRC, "exec"), mod.__dict__)
    return mod


def _pins_fail(mod):
    for pin in oracle_pins.ALL_PINS:
        try:
            if pin is oracle_pins.pin_bruteforce:
                pin(mod, exhaustive_max_len=6, random_cases=100)
            elif pin is oracle_pins.pin_invariants:
                pin(mod, cases=60)
            else:
                pin(mod)
        except Exception:
            return True
    return False


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch_mutation(name):
    old, new = MUTATIONS[name]
    mod = _mutant(name, old, new)
    try:
        assert _pins_fail(mod), f"no pin caught the planted mistake {name!r}"
    finally:
        sys.modules.pop(mod.__name__, None)


def test_unmutated_copy_passes():
    mod = _mutant("none", "import numpy as np", "import numpy as np")
    try:
        assert not _pins_fail(mod)
    finally:
        sys.modules.pop(mod.__name__, None)
