"""Parity at the largest pool the boundary accepts.

Slots are int32 on the device, so a cache holds at most num_blocks * S <= 2^31 - 1 slots
(VTOKEN_ERR_SHAPE above that). These tests build that pool, (2^31 - 1) // S blocks, put the
requests' tables and the free blocks at its top and the pool's very last block in the path
(the head of a table, a source; the head of the free list, a destination; the head of a
table repacked in place, a destination in place). Slot indices then come within S of 2^31 and
byte offsets into a plane exceed 2^35.

Repack and partial pass: rows are 16 bytes (one layer, one KV head of 16 one-byte elements);
every row of every plane holds its own slot index and plane as two int64 tags, so after a pass
every row of the 64 GiB cache is checked: a row the oracle moves holds its source's tags,
every other row its own. Metadata outputs are compared element by element with the oracle.

Decode: a 128 GiB fp8 cache (head_dim 32), random values in the requests' blocks, decode
through the positional slots before the pass and through the device slot mapping after it,
both against the float64 oracle over the live rows (same tolerance as the other decode
tests), and the two decodes bit-identical."""
import gc

import numpy as np
import pytest

from gpu_helpers import (assert_partial_equal, assert_plan_equal, gpu_partial, gpu_pass,
                         oracle_moves, oracle_params, torch)
from oracle.attention import decode_batch, slot_mapping
from oracle.planner import plan_partial
from oracle.repack import oracle_repack_inputs
from paper_2608_13263_amd import workloads as W

pytestmark = pytest.mark.gpu

ATOL, RTOL = 1e-4, 1e-4


def _label(msg):
    print(f"[gpu] {msg}", flush=True)


def _release():
    t = torch()
    gc.collect()
    t.cuda.synchronize()
    t.cuda.empty_cache()


def _masks(S, rng, first_live):
    """Requests of ragged lengths and mixed densities; the first request's token S - 1 (the
    last row of its first block) is live when first_live, its token 0 dead otherwise."""
    m0 = (rng.random(2500) < 0.35).astype(np.uint8)
    if first_live:
        m0[S - 1] = 1
    else:
        m0[0] = 0
    return [m0, np.zeros(40, np.uint8), np.ones(17, np.uint8),
            W.bernoulli_live(rng, 5000, 0.3, sink=4), np.ones(1, np.uint8),
            W.bernoulli_live(rng, 2000, 0.05), np.zeros(0, np.uint8),
            (rng.random(777) < 0.6).astype(np.uint8)]


def _tagged_cache(shape, num_blocks):
    """uint8 [2L][num_blocks][S][H][D] with 16-byte rows; row s of plane p holds the int64
    pair (s, s + (p + 1) * 2^40). Returns the cache and its int64 view [P][slots][2]."""
    t = torch()
    assert shape.row_bytes == 16
    P, n = shape.num_planes, num_blocks * shape.block_size
    kv = t.empty((P, num_blocks, shape.block_size, shape.num_kv_heads, shape.head_dim),
                 dtype=t.uint8, device="cuda")
    tags = kv.view(-1).view(t.int64).view(P, n, 2)
    ar = t.arange(n, dtype=t.int64, device="cuda")
    for p in range(P):
        tags[p, :, 0].copy_(ar)
        tags[p, :, 1].copy_(ar)
        tags[p, :, 1].add_((p + 1) << 40)
    del ar
    return kv, tags


def _check_tags(tags, src, dst):
    """Every row: a moved row holds its source's tags, every other row its own."""
    t = torch()
    P, n, _ = tags.shape
    expect = t.arange(n, dtype=t.int64, device="cuda")
    expect[t.from_numpy(dst).cuda()] = t.from_numpy(src).cuda()
    for p in range(P):
        assert t.equal(tags[p, :, 0], expect), f"plane {p}: slot tags differ"
        expect.add_((p + 1) << 40)
        assert t.equal(tags[p, :, 1], expect), f"plane {p}: plane tags differ"
        expect.sub_((p + 1) << 40)
    del expect


CASES = [
    # (mode, S, role of the pool's last block)
    ("out_of_place", 16, "source"),
    ("out_of_place", 16, "destination"),
    ("out_of_place", 1, "source"),
    ("out_of_place", 1, "destination"),
    ("in_place", 16, "source"),
    ("in_place", 1, "source"),
]


@pytest.mark.parametrize("mode,S,top", CASES, ids=[f"{m}_S{s}_{r}" for m, s, r in CASES])
def test_repack_at_slot_limit(mode, S, top):
    inplace = mode == "in_place"
    shape = W.KVShape(1, 1, 16, S, "fp8_e4m3")
    rng = np.random.default_rng(7000 + S)
    # the last block is live at its last row when it is a source out of place; in place it
    # is the first block of the first request, whose token 0 is dead, so rows move into it
    masks = _masks(S, rng, first_live=not inplace)
    inp = W.slot_limit_inputs(shape, masks, seed=7100 + S, top_block=top,
                              name=f"slot_limit_{mode}_S{S}_{top}")
    nb = inp.num_blocks
    assert nb * S <= W.SLOT_LIMIT < (nb + 1) * S
    _label(f"{inp.name}: {nb} blocks, {nb * S} slots, "
           f"{nb * S * shape.token_bytes / 2**30:.1f} GiB cache")
    orc = oracle_repack_inputs(inp, inplace=inplace)
    kv, tags = _tagged_cache(shape, nb)
    gpu = gpu_pass(inp, kv, label=inp.name, inplace=inplace)
    assert_plan_equal(gpu, orc)
    src, dst = oracle_moves(orc, inp, inplace)
    top_slot = nb * S - 1
    if inplace or top == "destination":
        assert top_slot in set(dst.tolist()), "the pool's last slot receives a row"
    else:
        assert top_slot in set(src.tolist()), "the pool's last slot is read"
    _check_tags(tags, src, dst)
    _label(f"{inp.name}: {len(src)} rows moved, every row of every plane checked")
    del kv, tags
    _release()


def test_partial_pass_at_slot_limit():
    """The paper's partial pass over the largest pool: per-block live bitmaps and counts for
    all 134M blocks, trigger forced (theta_F = 0), sources and destinations at the top."""
    from paper_2608_13263_amd import binding as B
    S = 16
    shape = W.KVShape(1, 1, 16, S, "fp8_e4m3")
    rng = np.random.default_rng(7300)
    inp = W.slot_limit_inputs(shape, _masks(S, rng, first_live=True), seed=7301,
                              top_block="source", name="slot_limit_partial")
    params = B.PlannerParams(theta=(0, 1))
    _label(f"{inp.name}: {inp.num_blocks} blocks")
    orc = plan_partial(inp.seq_lens, inp.tok_indptr, inp.bt_indptr, inp.block_ids, inp.live,
                       inp.slots(), inp.free_list, S, inp.num_blocks, oracle_params(params))
    assert orc.used > 0
    kv, tags = _tagged_cache(shape, inp.num_blocks)
    g = gpu_partial(inp, kv, params, label=inp.name)
    assert_partial_equal(g, orc, inp)
    src, dst = oracle_moves(orc, inp)
    assert inp.num_blocks * S - 1 in set(src.tolist()), "the pool's last slot is read"
    _check_tags(tags, src, dst)
    _label(f"{inp.name}: {len(src)} rows moved by the partial pass, every row checked")
    del kv, tags
    _release()


def _fp8_rows(n, D, seed):
    """n random fp8 e4m3 rows of D elements (N(0,1) rounded on the CPU) as uint8 [n][D]."""
    t = torch()
    g = t.Generator().manual_seed(seed)
    return t.randn((n, D), generator=g).to(t.float8_e4m3fn).view(t.uint8).numpy()


def _as_values(rows_u8):
    t = torch()
    return t.from_numpy(np.ascontiguousarray(rows_u8)).view(t.float8_e4m3fn).double().numpy()


def test_decode_at_slot_limit():
    """Decode over a 128 GiB fp8 cache at the slot limit, G = 1 and G = 8, before the pass
    (positional slots at the top of the pool) and after it (the device slot mapping; the
    pool's last block is the first destination)."""
    t = torch()
    from paper_2608_13263_amd import binding as B
    S, D = 16, 32
    shape = W.KVShape(1, 1, D, S, "fp8_e4m3")
    rng = np.random.default_rng(7400)
    masks = [(rng.random(3000) < 0.4).astype(np.uint8), np.ones(1025, np.uint8),
             (rng.random(40) < 0.5).astype(np.uint8), np.ones(S, np.uint8)]
    inp = W.slot_limit_inputs(shape, masks, seed=7401, top_block="destination",
                              name="slot_limit_decode")
    nb = inp.num_blocks
    _label(f"{inp.name}: {nb} blocks, {nb * S * shape.token_bytes / 2**30:.1f} GiB cache")
    kv = t.zeros((2, nb, S, 1, D), dtype=t.uint8, device="cuda")
    rows = kv.view(2, nb * S, D)
    old = inp.slots().astype(np.int64)                     # positional slot of every token
    kv_rows = [_fp8_rows(len(old), D, 7402), _fp8_rows(len(old), D, 7403)]
    idx = t.from_numpy(old).cuda()
    for p in range(2):
        rows[p][idx] = t.from_numpy(kv_rows[p]).cuda()

    # the oracle's inputs: every request's live rows in logical order (compact slots)
    live_tok = np.nonzero(inp.live)[0]
    k_vals = _as_values(kv_rows[0][live_tok])[:, None, :]
    v_vals = _as_values(kv_rows[1][live_tok])[:, None, :]
    counts = [int(inp.request_live(r).sum()) for r in range(inp.num_reqs)]
    c_indptr = np.concatenate([[0], np.cumsum(counts)])
    c_slots = np.arange(len(live_tok))
    max_tokens = max(counts)

    orc = oracle_repack_inputs(inp)
    ref_indptr, ref_slots = slot_mapping(orc.token_slot, inp.tok_indptr, inp.seq_lens)
    assert nb * S - 1 in set(ref_slots.tolist()), "the pool's last slot is decoded"

    cache = B.KVCache(kv, 1, 1, D, S)
    old_indptr = t.from_numpy(c_indptr.astype(np.int32)).cuda()
    old_slots = t.from_numpy(old[live_tok].astype(np.int32)).cuda()
    qs = {G: rng.standard_normal((inp.num_reqs, G, D)).astype(np.float32) for G in (1, 8)}
    before = {}
    for G, q in qs.items():
        out = B.paged_decode(cache, t.from_numpy(q).cuda(), old_indptr, old_slots, 0,
                             max_tokens, kv_dtype=B.KV_FP8_E4M3)
        before[G] = out.cpu().numpy()
        ref = decode_batch(q, k_vals, v_vals, c_indptr, c_slots)
        np.testing.assert_allclose(before[G].astype(np.float64), ref, atol=ATOL, rtol=RTOL)

    batch = B.Batch.from_inputs(inp)
    plan = B.Plan.allocate(batch, S)
    B.run_pass(cache, batch, plan)
    indptr, slots = B.build_slot_mapping(batch, plan)
    t.cuda.synchronize()
    assert np.array_equal(indptr.cpu().numpy(), ref_indptr)
    assert np.array_equal(slots.cpu().numpy()[:int(ref_indptr[-1])], ref_slots)
    for G, q in qs.items():
        out = B.paged_decode(cache, t.from_numpy(q).cuda(), indptr, slots, 0, max_tokens,
                             kv_dtype=B.KV_FP8_E4M3)
        assert np.array_equal(out.cpu().numpy(), before[G]), f"G={G}: decode changed"
    _label(f"{inp.name}: decode at G = 1 and 8 before and after the pass")
    del kv, rows, cache, plan, batch
    _release()
