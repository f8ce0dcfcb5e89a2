"""HIP path vs CPU oracle through the C ABI: bit-exact on every output and every KV byte.

Sizes here finish in seconds on the oracle yet span many 32 KiB copy items, several scan
tiles and ragged tails; the full Llama-3-8B-shaped cache is covered in
test_parity_full_gpu.py."""
import numpy as np
import pytest

from gpu_helpers import (assert_kv_equal, assert_plan_equal, full_parity, gpu_pass, kv_bytes,
                         plan_to_host, torch)
from oracle.repack import oracle_repack_inputs
from paper_2608_13263_amd import workloads as W

pytestmark = pytest.mark.gpu


def test_tiny_cache():
    full_parity(W.tiny_cache(101), seed=1)


def test_tiny_cache_copy_and_free_in_one_launch():
    full_parity(W.tiny_cache(101), seed=1, fused=True)


def test_tiny_cache_other_seed():
    full_parity(W.tiny_cache(7), seed=2)


def test_llama3_8b_random_two_layers():
    full_parity(W.llama3_8b_random(201, num_layers=2, num_reqs=8), seed=3)


def test_llama3_8b_h2o_one_layer():
    full_parity(W.llama3_8b_h2o(301, num_layers=1, num_reqs=6), seed=4)


@pytest.mark.parametrize("dtype", ["fp8_e4m3", "bf16"])
def test_llama3_70b_shape_block32(dtype):
    # S = 32; bf16 rows make 64 KiB chunks (two copy rounds per item), fp8 rows 32 KiB
    inp = W.llama3_70b_h2o(501, keep=0.3, dtype=dtype, num_layers=2, num_reqs=3,
                           len_range=(3000, 7000))
    full_parity(inp, seed=5)


@pytest.mark.parametrize("dtype", ["fp8_e4m3", "bf16"])
@pytest.mark.parametrize("keep", [0.1, 0.6])
def test_llama3_70b_keep_ratios(keep, dtype):
    # every KV byte of every plane; the full-size caches of all six variants run in
    # test_parity_full_gpu.py as waves
    inp = W.llama3_70b_h2o(502, keep=keep, dtype=dtype, num_layers=1, num_reqs=3,
                           len_range=(2000, 5000))
    full_parity(inp, seed=6)


def _edge_masks(S, rng):
    return [
        [],                                       # empty request: nothing to do
        [0] * 37,                                 # all dead: every block released
        [1] * 40,                                 # all live: unprofitable, unchanged
        [1],                                      # single token
        list((rng.random(2 * S) < 0.5).astype(int)),  # exact multiple of S
        list((rng.random(3 * S + 5) < 0.3).astype(int)),  # ragged tail
        [1] + [0] * (4 * S) + [1],                # two live tokens far apart
        list((rng.random(7 * S + 3) < 0.9).astype(int)),  # mostly live
    ]


@pytest.mark.parametrize("fused", [False, True], ids=["three_calls", "repack_free"])
@pytest.mark.parametrize("S", [1, 2, 16, 32, 48, 128, 256, 1000])
def test_edge_masks_block_sizes(S, fused):
    # S = 48 (not a power of two, several copy rounds), S = 128 and 256 (plan read from
    # memory; 64 KiB chunks: two parts) and S = 1000 (not a power of two, 250 KiB chunks: eight
    # parts, the last one partial)
    rng = np.random.default_rng(S)
    shape = W.KVShape(1, 2, 64, S, "fp16")
    inp = W.from_masks(_edge_masks(S, rng), shape, free_blocks=64, seed=S)
    full_parity(inp, seed=S, fused=fused)


@pytest.mark.parametrize("heads,dim,dtype", [(3, 8, "fp16"), (1, 8, "fp16"), (1, 16, "fp8_e4m3"),
                                             (5, 48, "bf16"), (1, 128, "fp8_e4m3")])
def test_row_geometries(heads, dim, dtype):
    # rows of 48 B (3 units, not a power of two), 16 B (one unit), 16 B fp8, 480 B, 128 B
    rng = np.random.default_rng(heads * 1000 + dim)
    shape = W.KVShape(2, heads, dim, 16, dtype)
    masks = [list((rng.random(int(n)) < 0.4).astype(int)) for n in rng.integers(1, 300, 12)]
    full_parity(W.from_masks(masks, shape, free_blocks=80, seed=3), seed=9)


@pytest.mark.parametrize("fused", [False, True], ids=["three_calls", "repack_free"])
@pytest.mark.parametrize("free_blocks", [0, 1, 3, 6])
def test_headroom_deferral(free_blocks, fused):
    # a short free list: the admitted requests are a prefix of the profitable ones
    rng = np.random.default_rng(11)
    shape = W.KVShape(1, 2, 64, 16, "fp16")
    masks = [list((rng.random(int(n)) < 0.3).astype(int)) for n in rng.integers(40, 120, 8)]
    inp = W.from_masks(masks, shape, free_blocks=free_blocks, seed=5)
    gpu, orc = full_parity(inp, seed=12, fused=fused)
    assert orc.used <= free_blocks


@pytest.mark.parametrize("fused", [False, True], ids=["three_calls", "repack_free"])
def test_empty_free_list_releases_dead_requests(fused):
    """No free block at all: only requests with no live token are admitted (they need no
    destination), so nothing is copied, yet their blocks are released."""
    shape = W.KVShape(1, 2, 64, 16, "fp16")
    # two requests with no live token first (admitted: 4 + 2 blocks released), then two that
    # need destinations (deferred)
    masks = [[0] * 50, [0] * 17, [1, 0] * 30, [1] * 5 + [0] * 40]
    inp = W.from_masks(masks, shape, free_blocks=0, seed=2)
    gpu, orc = full_parity(inp, seed=3, fused=fused)
    assert orc.used == 0 and orc.n_freed == 4 + 2 and gpu["n_admitted"] == 2


@pytest.mark.parametrize("fused", [False, True], ids=["three_calls", "repack_free"])
def test_no_requests(fused):
    shape = W.KVShape(1, 2, 64, 16, "fp16")
    full_parity(W.from_masks([], shape, free_blocks=8, seed=1), seed=1, fused=fused)


def test_nan_payloads_are_copied_bit_exactly():
    t = torch()
    inp = W.llama3_8b_random(203, num_layers=1, num_reqs=4, len_range=(300, 900))
    kv = W.kv_device(inp.shape, inp.num_blocks, 0)
    g = t.Generator(device="cuda")
    g.manual_seed(5)
    raw = kv.view(t.uint8)
    raw.copy_(t.randint(0, 256, raw.shape, generator=g, device="cuda", dtype=t.uint8))
    assert t.isnan(kv.float()).any()
    before = kv_bytes(kv, inp.shape)
    orc = oracle_repack_inputs(inp, before)
    gpu = gpu_pass(inp, kv)
    assert_plan_equal(gpu, orc)
    assert_kv_equal(kv_bytes(kv, inp.shape), orc.kv)


@pytest.mark.parametrize("variant,order,grid", [(v, 0, 0) for v in range(7)] + [
    (0, 1, 0), (0, 2, 0), (4, 1, 1), (1, 2, 7), (2, 1, 3), (5, 2, 1), (6, 1, 2048)])
def test_copy_variants_agree(variant, order, grid):
    # every cache policy, both work orders, persistent grids down to one workgroup
    inp = W.llama3_8b_random(204, num_layers=2, num_reqs=6, len_range=(500, 2500))
    full_parity(inp, seed=13, variant=variant, order=order, grid=grid)


@pytest.mark.parametrize("order", [1, 2])
def test_copy_grid_around_item_count(order):
    """Grids just below, at, just above and three times the pass's work items (destination
    blocks x planes, 32 KiB parts): below, the grid-stride loop takes the rest; above, the
    items are spread over the grid and the workgroups without one leave. Bytes and metadata
    equal the oracle's every time."""
    inp = W.llama3_8b_random(205, num_layers=2, num_reqs=6, len_range=(500, 2500))
    items = oracle_repack_inputs(inp).used * inp.shape.num_planes
    assert items > 8
    for grid in (items - 1, items, items + 1, 3 * items):
        print(f"[gpu] copy grid {grid} for {items} items, order {order}", flush=True)
        full_parity(inp, seed=14, variant=0, order=order, grid=grid)


def test_repack_is_idempotent():
    t = torch()
    from paper_2608_13263_amd import binding as B
    inp = W.llama3_8b_random(205, num_layers=2, num_reqs=6, len_range=(500, 2500))
    kv = W.kv_device(inp.shape, inp.num_blocks, 3)
    before = kv_bytes(kv, inp.shape)
    orc = oracle_repack_inputs(inp, before)
    cache = B.KVCache(kv, 2, 8, 128, 16)
    batch = B.Batch.from_inputs(inp)
    plan = B.Plan.allocate(batch, 16)
    print("[gpu] idempotence: two passes on unchanged inputs", flush=True)
    for _ in range(2):
        B.run_pass(cache, batch, plan)
        t.cuda.synchronize()
        assert_kv_equal(kv_bytes(kv, inp.shape), orc.kv)


def test_side_stream_and_stream_order():
    """All three calls on a non-default stream; a consumer on the default stream that waits
    on an event recorded after free_blocks sees the packed cache (invariant I3)."""
    t = torch()
    from paper_2608_13263_amd import binding as B
    inp = W.llama3_8b_random(206, num_layers=2, num_reqs=6, len_range=(500, 2500))
    kv = W.kv_device(inp.shape, inp.num_blocks, 4)
    before = kv_bytes(kv, inp.shape)
    orc = oracle_repack_inputs(inp, before)
    cache = B.KVCache(kv, 2, 8, 128, 16)
    batch = B.Batch.from_inputs(inp)
    plan = B.Plan.allocate(batch, 16)
    side = t.cuda.Stream()
    side.wait_stream(t.cuda.current_stream())
    print("[gpu] side stream pass", flush=True)
    with t.cuda.stream(side):
        B.run_pass(cache, batch, plan, stream=side)
        done = t.cuda.Event()
        done.record(side)
    t.cuda.current_stream().wait_event(done)
    snap = kv.clone()          # runs on the default stream, after the event
    t.cuda.synchronize()
    assert_kv_equal(kv_bytes(snap, inp.shape), orc.kv)


# ------------------------------------------------------------------------------------------
# device-detected errors: status word set, no KV byte written
# ------------------------------------------------------------------------------------------

@pytest.fixture(params=["small", "large", "large_repack_free", "many"])
def error_batch(request):
    """A batch under the one-launch planning bound (8192 tokens, 24 requests), one above it
    (count launch + plan launch) and one of more requests than the plan workgroups admit
    themselves (600: count, admission and plan launches): every device-detected error is
    checked on each path, and with the copy and the freed list in one launch."""
    lens = {"small": (300, 900), "many": (40, 120)}.get(request.param, (4000, 6000))
    R = 600 if request.param == "many" else 5
    make = lambda: W.llama3_8b_random(207, num_layers=1, num_reqs=R, len_range=lens)  # noqa
    return make, request.param.endswith("repack_free")


def _error_case(mutate, expect, batch):
    t = torch()
    from paper_2608_13263_amd import binding as B
    make, fused = batch
    inp = make()
    mutate(inp)
    kv = W.kv_device(inp.shape, inp.num_blocks, 5)
    before = kv_bytes(kv, inp.shape)
    gpu = gpu_pass(inp, kv, label=f"error case {expect}", fused=fused)
    assert gpu["status"] == B.STATUS_CODE[expect]
    assert gpu["used"] == 0 and gpu["n_admitted"] == 0 and gpu["n_freed"] == 0
    assert_kv_equal(kv_bytes(kv, inp.shape), before)


def test_error_block_id_out_of_range(error_batch):
    def m(inp):
        inp.block_ids[3] = inp.num_blocks
    _error_case(m, "VTOKEN_ERR_BLOCK_RANGE", error_batch)


def test_error_negative_block_id(error_batch):
    def m(inp):
        inp.block_ids[-1] = -2
    _error_case(m, "VTOKEN_ERR_BLOCK_RANGE", error_batch)


def test_error_free_list_entry_out_of_range(error_batch):
    def m(inp):
        inp.free_list[0] = inp.num_blocks + 5
    _error_case(m, "VTOKEN_ERR_BLOCK_RANGE", error_batch)


def test_error_block_table_length(error_batch):
    def m(inp):
        inp.bt_indptr[2] += 1
    _error_case(m, "VTOKEN_ERR_BT_LEN", error_batch)


def test_error_token_range(error_batch):
    def m(inp):
        inp.seq_lens[1] += 1
    _error_case(m, "VTOKEN_ERR_TOK_LEN", error_batch)


@pytest.mark.parametrize("batch_kind", ["one_launch", "count_plan", "admission"])
@pytest.mark.parametrize("inplace", [False, True], ids=["out_of_place", "in_place"])
def test_pass_graph_replay(inplace, batch_kind):
    """The whole pass (build, copy, free) captured once in a HIP graph over fixed buffers and
    replayed: before each replay new liveness is written into the captured live-mask buffer
    and the KV bytes are whatever the previous replay left; every replay equals the oracle on
    those inputs, with unrelated eager work between replays. No kernel of the pass needs a
    memset: the admission kernel rewrites every counter."""
    import dataclasses
    t = torch()
    from paper_2608_13263_amd import binding as B
    # the table build as one launch (8 requests), as count and plan launches (40) and with the
    # admission in a launch of its own (600 short requests)
    R, lens, layers = {"one_launch": (8, (300, 1500), 2), "count_plan": (40, (300, 1500), 1),
                       "admission": (600, (40, 120), 1)}[batch_kind]
    inp = W.llama3_8b_random(231, num_layers=layers, num_reqs=R, len_range=lens)
    sh = inp.shape
    kv = W.kv_device(sh, inp.num_blocks, 21)
    cache = B.KVCache(kv, sh.num_layers, sh.num_kv_heads, sh.head_dim, sh.block_size)
    batch = B.Batch.from_inputs(inp)
    plan = B.Plan.allocate(batch, sh.block_size, inplace=inplace)
    print(f"[gpu] pass graph replay inplace={inplace}: R={inp.num_reqs} T={inp.num_tokens}",
          flush=True)

    side = t.cuda.Stream()
    side.wait_stream(t.cuda.current_stream())
    with t.cuda.stream(side):          # eager run before capture (also a first check)
        first_before = kv_bytes(kv, sh)
        B.run_pass(cache, batch, plan, inplace=inplace)
    t.cuda.current_stream().wait_stream(side)
    t.cuda.synchronize()
    orc = oracle_repack_inputs(inp, first_before, inplace=inplace)
    assert_plan_equal(plan_to_host(plan, inp), orc)
    assert_kv_equal(kv_bytes(kv, sh), orc.kv)

    graph = t.cuda.CUDAGraph()
    with t.cuda.graph(graph):
        B.run_pass(cache, batch, plan, inplace=inplace)

    rng = np.random.default_rng(7)
    for step in range(3):
        live = (rng.random(inp.num_tokens) < (0.2, 0.5, 0.8)[step]).astype(np.uint8)
        cur = dataclasses.replace(inp, live=live)
        batch.live.copy_(t.from_numpy(live).to(batch.live.device))
        t.cuda.synchronize()
        before = kv_bytes(kv, sh)
        noise = t.randn(256, 256, device="cuda")
        noise = noise @ noise                     # unrelated eager work between replays
        graph.replay()
        t.cuda.synchronize()
        orc = oracle_repack_inputs(cur, before, inplace=inplace)
        assert_plan_equal(plan_to_host(plan, cur), orc)
        assert_kv_equal(kv_bytes(kv, sh), orc.kv)
        assert orc.n_admitted > 0


def _random_case(seed):
    """A random small geometry, batch and pool: block sizes 1..128 (powers of two and not),
    1-8 KV heads, head_dim 8..256, fp16 / bf16 / fp8 rows (multiples of 16 bytes), ragged
    requests at random densities, free lists from empty (deferral) to ample."""
    rng = np.random.default_rng(seed)
    dtype = ["fp16", "bf16", "fp8_e4m3"][int(rng.integers(3))]
    e = 1 if dtype == "fp8_e4m3" else 2
    while True:
        S = int(rng.choice([1, 2, 3, 4, 5, 7, 8, 16, 24, 32, 48, 64, 96, 128]))
        H = int(rng.integers(1, 9))
        D = int(rng.choice([8, 16, 24, 32, 64, 96, 128, 256]))
        row = H * D * e
        if row % 16 == 0 and S * row <= 64 * 1024:
            break
    R = int(rng.integers(1, 13))
    masks = []
    for _ in range(R):
        n = int(rng.integers(0, 12 * S + 40))
        masks.append((rng.random(n) < rng.random()).astype(int).tolist())
    M = sum(-(-len(m) // S) for m in masks)
    free = int(rng.integers(0, M + 8))
    layers = int(rng.integers(1, 3))
    inp = W.from_masks(masks, W.KVShape(layers, H, D, S, dtype), free_blocks=free, seed=seed,
                       name=f"fuzz{seed}")
    return inp


@pytest.mark.parametrize("seed", range(40))
def test_random_geometries(seed):
    """Seeded random geometries and batches, out of place and in place, bit-exact."""
    inp = _random_case(1000 + seed)
    full_parity(inp, seed=seed)
    full_parity(inp, seed=seed, inplace=True)
    full_parity(inp, seed=seed, fused=True)


def _random_large_case(seed):
    """A random batch of 200-1500 requests (either side of the separate admission, short and
    long requests), block sizes 1-96, small rows, a free list from a tenth of the requests'
    blocks (deferral) to ample."""
    rng = np.random.default_rng(seed)
    S = int(rng.choice([1, 3, 8, 16, 24, 32, 48, 96]))
    R = int(rng.integers(200, 1501))
    top = int(rng.choice([60, 400, 3000]))
    masks = [(rng.random(int(n)) < rng.random()).astype(int).tolist()
             for n in rng.integers(0, top, size=R)]
    M = sum(-(-len(m) // S) for m in masks)
    free = int(M * rng.choice([0.1, 0.5, 2.0]))
    return W.from_masks(masks, W.KVShape(1, 1, 8, S, "fp16"), free_blocks=free, seed=seed,
                        name=f"fuzz_large{seed}")


@pytest.mark.parametrize("seed", range(8))
def test_random_large_batches(seed):
    """Seeded random large batches, out of place (three calls and repack_free) and in place,
    bit-exact."""
    inp = _random_large_case(5000 + seed)
    full_parity(inp, seed=seed)
    full_parity(inp, seed=seed, fused=True)
    full_parity(inp, seed=seed, inplace=True)


@pytest.mark.parametrize("extra", [0, 1], ids=["at_token_bound", "past_token_bound"])
def test_small_batch_planning_bound_tokens(extra):
    """8192 tokens are planned by the one-launch kernel, 8193 by the count and plan launches:
    both equal the oracle on the same requests (the last one a token longer)."""
    rng = np.random.default_rng(40 + extra)
    lens = [700] * 10 + [8192 - 7000 + extra]
    masks = [(rng.random(n) < 0.4).astype(int).tolist() for n in lens]
    M = sum(-(-n // 16) for n in lens)
    inp = W.from_masks(masks, W.KVShape(1, 2, 64, 16, "fp16"), free_blocks=M, seed=extra,
                       name=f"bound_tokens_{extra}")
    assert inp.num_tokens == 8192 + extra
    full_parity(inp, seed=3)


@pytest.mark.parametrize("mode", ["three_calls", "repack_free", "in_place"])
@pytest.mark.parametrize("S,R", [(24, 340), (48, 340), (24, 700)])
def test_large_batch_block_size_not_power_of_two(S, R, mode):
    """Past the one-launch bounds (340 or 700 requests, over 16384 tokens) with a block size
    that is not a power of two, so the plan launch divides positions by S: 340 requests of
    ~48 blocks with S = 48 (~1,536 tokens) are admitted by every plan workgroup itself, whose
    destinations reach past the free-list head it stages in LDS; with S = 24 (~768 tokens) and
    with 700 requests the admission runs in a launch of its own before the plan launch."""
    rng = np.random.default_rng(S + R)
    lens = rng.integers(0, 64 * S, size=R)
    masks = [(rng.random(int(n)) < rng.uniform(0.8, 1.0)).astype(int).tolist() for n in lens]
    M = sum(-(-len(m) // S) for m in masks)
    inp = W.from_masks(masks, W.KVShape(1, 1, 8, S, "fp16"), free_blocks=M, seed=S,
                       name=f"large_block{S}_{R}")
    assert inp.num_tokens > 16384 and inp.num_reqs > 256
    gpu, orc = full_parity(inp, seed=S, fused=mode == "repack_free", inplace=mode == "in_place")
    assert orc.n_admitted > 256 and (mode == "in_place" or orc.used > 8192)


@pytest.mark.parametrize("R,lens", [(24, (0, 60)), (25, (0, 60)), (256, (0, 60)), (257, (0, 60)),
                                    (512, (1100, 1400)), (513, (1100, 1400)), (1100, (0, 60)),
                                    (4200, (0, 60))])
def test_planning_bounds_requests(R, lens):
    """24 requests are planned by the one-launch kernel, 25 by the count and plan launches. Up
    to 256 requests every plan workgroup runs the admission itself, and up to 512 when the
    requests average 1024 tokens or more; past that one launch runs the admission before the
    plan launch (1100: several 1024-request rounds; 4200: past the 4096 live counts that launch
    stages in LDS). A third of the blocks the requests hold are free, so the admission defers a
    suffix of the profitable requests."""
    rng = np.random.default_rng(R)
    masks = [(rng.random(int(n)) < 0.5).astype(int).tolist()
             for n in rng.integers(lens[0], lens[1], size=R)]
    M = sum(-(-len(m) // 16) for m in masks)
    inp = W.from_masks(masks, W.KVShape(1, 2, 64, 16, "bf16"), free_blocks=M // 3, seed=R,
                       name=f"bound_requests_{R}")
    gpu, orc = full_parity(inp, seed=4)
    profitable = sum(-(-sum(m) // 16) < -(-len(m) // 16) for m in masks)
    assert 0 < orc.n_admitted < profitable
    full_parity(inp, seed=4, fused=True)
    full_parity(inp, seed=4, inplace=True)
