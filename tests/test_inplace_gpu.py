"""In-place mode through the C ABI vs the oracle's in-place mode: bit-exact on every output
and every KV byte. Overlap-heavy masks check the block-order hazard rule: a destination
block is written only after every read of its own and earlier destination blocks."""
import numpy as np
import pytest

from gpu_helpers import assert_kv_equal, assert_plan_equal, full_parity, gpu_pass, kv_bytes, torch
from oracle.repack import oracle_repack_inputs
from paper_2608_13263_amd import workloads as W

pytestmark = pytest.mark.gpu


def test_inplace_tiny():
    full_parity(W.tiny_cache(101), seed=1, inplace=True)


def test_inplace_llama3_8b_random_two_layers():
    full_parity(W.llama3_8b_random(201, num_layers=2, num_reqs=8), seed=3, inplace=True)


def test_inplace_llama3_8b_h2o_one_layer():
    full_parity(W.llama3_8b_h2o(301, num_layers=1, num_reqs=6), seed=4, inplace=True)


@pytest.mark.parametrize("dtype", ["fp8_e4m3", "bf16"])
def test_inplace_llama3_70b_shape(dtype):
    # bf16 at S = 32 stages 64 KiB blocks (single LDS buffer), fp8 32 KiB (double buffer)
    inp = W.llama3_70b_h2o(501, keep=0.3, dtype=dtype, num_layers=2, num_reqs=3,
                           len_range=(3000, 7000))
    full_parity(inp, seed=5, inplace=True)


def _overlap_masks(S, rng):
    n = 9 * S + 3
    return [
        [0] + [1] * (n - 1),                      # every row shifts by one slot
        [1] * S + [0] + [1] * (n - S - 1),        # identity first block, then a one-slot shift
        [0] * S + [1] * (n - S),                  # every row moves back by a whole block
        list((rng.random(n) < 0.97).astype(int)),  # few holes: long overlapping chains
        list((rng.random(n) < 0.5).astype(int)),
        [1] * (n - 1) + [0],                      # only the tail is dead: pure identity
        [],
        [0] * 40,
        [1] * 33,
    ]


@pytest.mark.parametrize("S", [1, 2, 16, 32, 48, 128])
def test_inplace_overlap_masks(S):
    rng = np.random.default_rng(100 + S)
    shape = W.KVShape(1, 2, 64, S, "fp16")
    inp = W.from_masks(_overlap_masks(S, rng), shape, free_blocks=4, seed=S)
    full_parity(inp, seed=S, inplace=True)


@pytest.mark.parametrize("heads,dim,dtype", [(3, 8, "fp16"), (1, 8, "fp16"), (5, 48, "bf16"),
                                             (8, 128, "bf16"), (1, 128, "fp8_e4m3")])
def test_inplace_row_geometries(heads, dim, dtype):
    rng = np.random.default_rng(heads * 100 + dim)
    shape = W.KVShape(2, heads, dim, 16, dtype)
    masks = [list((rng.random(int(n)) < 0.6).astype(int)) for n in rng.integers(1, 400, 10)]
    full_parity(W.from_masks(masks, shape, free_blocks=0, seed=4), seed=8, inplace=True)


def test_inplace_second_pass_moves_nothing():
    """After a pass, the packed layout (live tokens only) needs no further repack."""
    t = torch()
    from paper_2608_13263_amd import binding as B
    inp = W.llama3_8b_random(212, num_layers=2, num_reqs=6, len_range=(500, 2500))
    kv = W.kv_device(inp.shape, inp.num_blocks, 6)
    before = kv_bytes(kv, inp.shape)
    orc = oracle_repack_inputs(inp, before, inplace=True)
    gpu = gpu_pass(inp, kv, inplace=True)
    assert_plan_equal(gpu, orc)
    assert_kv_equal(kv_bytes(kv, inp.shape), orc.kv)
    # second pass over the committed layout
    R = inp.num_reqs
    masks, tables = [], []
    for r in range(R):
        a = int(inp.tok_indptr[r])
        lv = inp.live[a:a + int(inp.seq_lens[r])]
        nbt = orc.new_block_ids[orc.new_bt_indptr[r]:orc.new_bt_indptr[r + 1]]
        masks.append(np.ones(int(lv.sum()), np.uint8) if orc.admitted[r] else lv)
        tables.append(nbt)
    nxt = W.RepackInputs(
        name="second pass", shape=inp.shape, num_blocks=inp.num_blocks,
        seq_lens=np.array([len(m) for m in masks], np.int32),
        tok_indptr=np.concatenate([[0], np.cumsum([len(m) for m in masks])]).astype(np.int32),
        bt_indptr=np.concatenate([[0], np.cumsum([len(x) for x in tables])]).astype(np.int32),
        block_ids=np.concatenate(tables).astype(np.int32),
        live=np.concatenate(masks).astype(np.uint8),
        free_list=np.concatenate([inp.free_list, orc.freed]).astype(np.int32))
    snap = kv_bytes(kv, inp.shape)
    gpu2 = gpu_pass(nxt, kv, inplace=True, label="in-place second pass")
    orc2 = oracle_repack_inputs(nxt, snap, inplace=True)
    assert_plan_equal(gpu2, orc2)
    assert_kv_equal(kv_bytes(kv, inp.shape), snap)
    del kv
    t.cuda.empty_cache()


@pytest.mark.parametrize("variant", [1, 2, 3, 4])
@pytest.mark.parametrize("S", [16, 32])
def test_inplace_staging_variants(variant, S):
    # LDS double buffer, LDS single buffer, registers: identical bytes
    rng = np.random.default_rng(300 + S)
    shape = W.KVShape(2, 8, 128, S, "bf16")
    masks = _overlap_masks(S, rng) + [list((rng.random(int(n)) < 0.7).astype(int))
                                      for n in rng.integers(50, 900, 6)]
    full_parity(W.from_masks(masks, shape, free_blocks=0, seed=7), seed=11, inplace=True,
                variant=variant)


@pytest.mark.parametrize("S", [1, 2, 16, 32, 48, 64])
def test_inplace_pipelined_variant(S):
    """Variant 4 (reads of the next moving block in flight while one is written, plans staged
    32 blocks at a time): overlap-heavy masks, chains far longer than 32 blocks with identity
    blocks between moving ones, and rows that do not fill the last unit round."""
    rng = np.random.default_rng(400 + S)
    shape = W.KVShape(1, 3, 8, S, "fp16")            # 48-byte rows: chunks of 3*S units
    n = 80 * S + 5
    long_masks = [
        [0] + [1] * (n - 1),                                        # 80-block shifting chain
        [1] * (40 * S) + [0] + [1] * (n - 40 * S - 1),              # 40 identity blocks first
        ([1] * S + [0] * (S // 2 + 1) + [1] * (S // 2)) * 30,       # alternating blocks
        list((rng.random(n) < 0.9).astype(int)),
    ]
    inp = W.from_masks(_overlap_masks(S, rng) + long_masks, shape, free_blocks=4, seed=S)
    full_parity(inp, seed=S, inplace=True, variant=4)
    shape2 = W.KVShape(2, 4, 128, S, "bf16")                  # 1 KiB rows, chunks <= 64 KiB
    masks2 = _overlap_masks(S, rng) + [list((rng.random(int(m)) < 0.6).astype(int))
                                       for m in rng.integers(50, 60 * S, 4)]
    full_parity(W.from_masks(masks2, shape2, free_blocks=0, seed=9), seed=12, inplace=True,
                variant=4)


@pytest.mark.parametrize("R", [255, 256, 257, 700])
def test_inplace_pipelined_many_requests(R):
    """Variant 4 hands chains out longest first when there are at most 256 requests and in
    request order above that; both sides of the switch, with equal chain lengths (ties broken by
    request index) and requests that move nothing."""
    rng = np.random.default_rng(500 + R)
    S = 16
    shape = W.KVShape(1, 2, 16, S, "fp16")
    masks = []
    for i in range(R):
        n = int(rng.integers(1, 6 * S))
        kind = i % 4
        if kind == 0:
            m = [1] * n                                           # nothing moves
        elif kind == 1:
            m = [0] + [1] * (3 * S)                               # equal lengths: ties
        else:
            m = list((rng.random(n) < 0.6).astype(int))
        masks.append(m)
    full_parity(W.from_masks(masks, shape, free_blocks=0, seed=R), seed=R, inplace=True,
                variant=4)


@pytest.mark.parametrize("built", ["in_place", "out_of_place"])
def test_copy_rejects_a_plan_of_the_other_mode(built):
    """A plan carries its mode (counters[4]): the out-of-place copy handed an in-place plan,
    or the in-place copy handed an out-of-place plan, copies nothing and sets the status word
    to VTOKEN_ERR_PLAN_MODE; the free call that follows then releases nothing. A plan of the
    right mode on the same cache is unaffected."""
    t = torch()
    from paper_2608_13263_amd import binding as B
    inp = W.llama3_8b_random(201, num_layers=2, num_reqs=6)
    sh = inp.shape
    print(f"[gpu] plan-mode mismatch: {built} plan to the other copy", flush=True)
    kv = W.kv_device(sh, inp.num_blocks, 11)
    before = kv.clone()
    cache = B.KVCache(kv, sh.num_layers, sh.num_kv_heads, sh.head_dim, sh.block_size)
    batch = B.Batch.from_inputs(inp)
    plan = B.Plan.allocate(batch, sh.block_size, inplace=True)
    freed = t.full((max(inp.num_bt_entries, 1),), -9, dtype=t.int32, device="cuda")
    if built == "in_place":
        B.build_token_table_inplace(cache, batch, plan)
        t.cuda.synchronize()
        assert plan.counters.cpu().tolist()[3:] == [0, 2]
        B.repack(cache, batch, plan)
    else:
        B.build_token_table(cache, batch, plan)
        t.cuda.synchronize()
        assert plan.counters.cpu().tolist()[3:] == [0, 1]
        B.repack_inplace(cache, batch, plan)
    B.free_blocks(batch, plan, freed=freed)
    t.cuda.synchronize()
    assert int(plan.counters[1]) > 0, "the plan admitted requests"
    assert int(plan.counters[3]) == B.STATUS_CODE["VTOKEN_ERR_PLAN_MODE"]
    assert t.equal(kv, before), "a mismatched copy wrote KV bytes"
    assert bool((freed == -9).all()), "blocks were released after the failed copy"
    # the same cache through the matching copy equals the oracle
    del before
    full_parity(inp, seed=11, inplace=built == "in_place")
