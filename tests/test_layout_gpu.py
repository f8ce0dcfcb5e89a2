"""vtoken_check_layout through the C ABI against oracle.repack.check_layout: the full pass's
layout precondition (every block id in the pool and held at most once over the block tables
and the free list). Bit-exact status on generated layouts, on planted faults of every kind
(a repeated id inside one table, across tables, held and free, twice free; ids outside the
pool, alone and together with a repeat), on empty input, on a 2^27-block pool with the fault
at its last block, and on a clean call right after a failing one (the workspace is cleared by
the call)."""
import numpy as np
import pytest

from gpu_helpers import torch
from oracle.repack import check_layout
from paper_2608_13263_amd import workloads as W

pytestmark = pytest.mark.gpu


def _B():
    from paper_2608_13263_amd import binding as B
    return B


def _run(block_ids, free_list, num_blocks, label, workspace=None):
    """One request of block size 1 holding every table id (the check reads only block_ids
    and free_list); returns the device status."""
    t = torch()
    B = _B()
    block_ids = np.asarray(block_ids, dtype=np.int64)
    free_list = np.asarray(free_list, dtype=np.int64)
    M = len(block_ids)
    print(f"[gpu] layout {label}: num_blocks={num_blocks} M={M} f={len(free_list)}", flush=True)
    kv = t.empty((2, num_blocks, 1, 1, 8), dtype=t.float16, device="cuda")   # 16-byte rows
    cache = B.KVCache(kv, 1, 1, 8, 1)
    batch = B.Batch.from_host([M], [0, M], [0, M], block_ids, np.zeros(M, np.uint8), free_list)
    status = B.check_layout(cache, batch, workspace=workspace)
    t.cuda.synchronize()
    return int(status.item())


def _plant(rng, ids, M, kind, num_blocks):
    ids = ids.copy()
    f = len(ids) - M
    if kind == "table_twice" and M >= 2:
        i, j = rng.choice(M, size=2, replace=False)
        ids[j] = ids[i]
    elif kind == "held_and_free" and M >= 1 and f >= 1:
        ids[M + rng.integers(f)] = ids[rng.integers(M)]
    elif kind == "free_twice" and f >= 2:
        i, j = M + rng.choice(f, size=2, replace=False)
        ids[j] = ids[i]
    elif kind == "past_pool":
        ids[rng.integers(len(ids))] = num_blocks + int(rng.integers(0, 3))
    elif kind == "negative":
        ids[rng.integers(len(ids))] = -1 - int(rng.integers(0, 5))
    elif kind == "range_and_repeat" and len(ids) >= 3:
        i, j, k = rng.choice(len(ids), size=3, replace=False)
        ids[j] = ids[i]
        ids[k] = num_blocks
    return ids


@pytest.mark.parametrize("maker", ["tiny", "llama3_8b_random", "token_tables"])
def test_generated_layouts_pass(maker):
    inp = {"tiny": lambda: W.tiny_cache(101),
           "llama3_8b_random": lambda: W.llama3_8b_random(241, num_layers=1),
           "token_tables": lambda: W.token_table_inputs(651, num_reqs=12,
                                                        len_range=(100, 900))}[maker]()
    want = check_layout(inp.block_ids, inp.free_list, inp.num_blocks)
    assert want == 0
    assert _run(inp.block_ids, inp.free_list, inp.num_blocks, maker) == want


def test_shared_prefix_tables_fail():
    """Token tables with shared prefixes hold blocks in several tables: the full pass must
    not run on them (the partial pass keeps such blocks in place)."""
    inp = W.token_table_inputs(652, num_reqs=12, len_range=(200, 900), shared_groups=2,
                               group_size=3, prefix_tokens=64)
    assert check_layout(inp.block_ids, inp.free_list, inp.num_blocks) == -14
    assert _run(inp.block_ids, inp.free_list, inp.num_blocks, "shared prefixes") == -14


KINDS = ["none", "table_twice", "held_and_free", "free_twice", "past_pool", "negative",
         "range_and_repeat"]


@pytest.mark.parametrize("seed", range(28))
def test_random_layouts_match_oracle(seed):
    rng = np.random.default_rng(900 + seed)
    num_blocks = int(rng.choice([1, 31, 32, 33, 100, 1000, 4097, 70000]))
    total = int(rng.integers(0, num_blocks + 1))
    ids = rng.permutation(num_blocks)[:total].astype(np.int64)
    M = int(rng.integers(0, total + 1))
    kind = KINDS[seed % len(KINDS)]
    ids = _plant(rng, ids, M, kind, num_blocks) if total else ids
    want = check_layout(ids[:M], ids[M:], num_blocks)
    assert _run(ids[:M], ids[M:], num_blocks, f"random {seed} {kind}") == want


def test_empty_and_large_pool():
    assert _run([], [], 5, "empty") == 0
    nb = 1 << 27
    top = np.arange(nb - 5000, nb, dtype=np.int64)
    assert _run(top[:3000], top[3000:], nb, "2^27 blocks") == 0
    bad = top.copy()
    bad[10] = nb - 1                                   # the pool's last block held twice
    assert check_layout(bad[:3000], bad[3000:], nb) == -14
    assert _run(bad[:3000], bad[3000:], nb, "2^27 blocks, last block twice") == -14


def test_clean_call_after_a_failing_one():
    """Both calls share one workspace: the second starts from the bits and flags the first
    left, and must clear them itself."""
    t = torch()
    ws = t.empty(3, dtype=t.int32, device="cuda")          # 12 bytes: 64 blocks
    ids = np.arange(64, dtype=np.int64)
    bad = ids.copy()
    bad[5] = 7
    assert _run(bad[:40], bad[40:], 64, "repeat", ws) == -14
    assert _run(ids[:40], ids[40:], 64, "clean after repeat", ws) == 0
    bad[50] = 64
    assert _run(bad[:40], bad[40:], 64, "range and repeat", ws) == -10
    assert _run(ids[:40], ids[40:], 64, "clean after range", ws) == 0
