"""The partial reclamation pass (vtoken_plan_partial + vtoken_repack) through the C ABI
against the CPU oracle of oracle/planner.py: every output bit-exact (per-block n_b and
reference counts, the statistics, sources considered, admission, CSR offsets, token table,
new tables, source plan, released sources) and every KV byte after the copy."""
import numpy as np
import pytest

from gpu_helpers import (assert_partial_equal, gpu_partial, kv_bytes, partial_to_host,
                         run_partial_oracle, torch)
from oracle.repack import oracle_repack_inputs
from paper_2608_13263_amd import workloads as W

pytestmark = pytest.mark.gpu


def _B():
    from paper_2608_13263_amd import binding as B
    return B


def partial_parity(inp, params=None, seed=0, label=""):
    t = torch()
    B = _B()
    params = params or B.PlannerParams()
    kv = W.kv_device(inp.shape, inp.num_blocks, seed)
    before = kv_bytes(kv, inp.shape)
    o = run_partial_oracle(inp, before, params)
    g = gpu_partial(inp, kv, params, label)
    assert_partial_equal(g, o, inp)
    after = kv_bytes(kv, inp.shape)
    if not np.array_equal(after, o.kv):
        diff = np.nonzero((after != o.kv).any(axis=2))
        raise AssertionError(f"KV bytes differ in {len(diff[0])} rows")
    del kv
    t.cuda.empty_cache()
    return g, o


CASES = {
    "tiny_shared": lambda: W.token_table_inputs(
        611, W.KVShape(1, 2, 64, 16, "fp16"), num_reqs=8, len_range=(100, 500),
        shared_groups=1, group_size=3, prefix_tokens=64),
    "llama3_8b_shared": lambda: W.token_table_inputs(
        612, W.KVShape(2, 8, 128, 16, "bf16"), num_reqs=32, len_range=(600, 3000),
        shared_groups=3, group_size=4, prefix_tokens=512),
    "llama3_70b_fp8": lambda: W.token_table_inputs(
        613, W.KVShape(2, 8, 128, 32, "fp8_e4m3"), num_reqs=6, len_range=(2000, 9000),
        keep=0.3, recent=128),
    "block_64": lambda: W.token_table_inputs(
        614, W.KVShape(1, 4, 64, 64, "bf16"), num_reqs=10, len_range=(300, 2000),
        shared_groups=1, group_size=2, prefix_tokens=128),
    "block_1": lambda: W.token_table_inputs(
        615, W.KVShape(1, 2, 32, 1, "fp16"), num_reqs=6, len_range=(20, 300)),
    "positional": lambda: W.token_table_inputs(
        616, W.KVShape(1, 2, 64, 16, "fp16"), num_reqs=12, len_range=(100, 900),
        shuffled_frac=0.0, dropped_frac=0.0, pin_tail=False),
    "many_requests": lambda: W.token_table_inputs(
        617, W.KVShape(1, 1, 64, 4, "fp16"), num_reqs=1500, len_range=(1, 60), recent=4,
        shared_groups=20, group_size=3, prefix_tokens=8),
}


@pytest.mark.parametrize("case", sorted(CASES))
def test_partial_parity_default_params(case):
    g, o = partial_parity(CASES[case](), label=case)
    print(f"[gpu] {case}: triggered={o.triggered} admitted={o.n_admitted} moved={o.tokens_moved} "
          f"released={o.n_freed}", flush=True)


@pytest.mark.parametrize("params", [
    dict(max_sources=5), dict(max_sources=0), dict(max_sources=37),
    dict(theta=(99, 100)), dict(theta=(0, 1)), dict(free_watermark=0),
    dict(free_watermark=100000), dict(min_eligible=100000), dict(max_live_per_source=2),
    dict(max_live_per_source=0), dict(theta=(-1, 1), max_live_per_source=16, min_eligible=0),
], ids=lambda d: ",".join(f"{k}={v}" for k, v in d.items()))
def test_partial_parity_params(params):
    B = _B()
    inp = W.token_table_inputs(621, W.KVShape(1, 2, 64, 16, "bf16"), num_reqs=16,
                               len_range=(200, 1500), shared_groups=2, group_size=3,
                               prefix_tokens=96)
    partial_parity(inp, B.PlannerParams(**params), label=str(params))


@pytest.mark.parametrize("call", ["free_blocks", "repack_free"])
def test_freed_list_refuses_a_partial_plan(call):
    """A partial pass's plan carries its own mode (counters[4] = 3): its released blocks are
    the planner state's sources, so vtoken_free_blocks and vtoken_repack_free refuse it
    (VTOKEN_ERR_PLAN_MODE, nothing released; vtoken_repack_free copies nothing either), while
    vtoken_repack copies it (every other test of this file)."""
    t = torch()
    B = _B()
    inp = CASES["tiny_shared"]()
    sh = inp.shape
    print(f"[gpu] partial plan handed to {call}", flush=True)
    kv = W.kv_device(sh, inp.num_blocks, 3)
    before = kv.clone()
    cache = B.KVCache(kv, sh.num_layers, sh.num_kv_heads, sh.head_dim, sh.block_size)
    batch = B.Batch.from_inputs(inp)
    slot_in = t.from_numpy(np.ascontiguousarray(inp.slots(), dtype=np.int32)).cuda()
    plan = B.Plan.allocate(batch, sh.block_size)
    state = B.PlannerState.allocate(inp.num_blocks, batch, pinned=inp.pinned)
    B.plan_partial(cache, batch, slot_in, plan, state, B.PlannerParams())
    t.cuda.synchronize()
    assert plan.counters.cpu().tolist()[3:] == [0, 3]
    assert int(plan.counters[1]) > 0, "the plan admitted requests"
    freed = t.full((max(inp.num_bt_entries, 1),), -9, dtype=t.int32, device="cuda")
    if call == "free_blocks":
        B.repack(cache, batch, plan)
        t.cuda.synchronize()
        assert int(plan.counters[3]) == 0
        B.free_blocks(batch, plan, freed=freed)
    else:
        B.repack_free(cache, batch, plan, freed=freed)
        t.cuda.synchronize()
        assert t.equal(kv, before), "vtoken_repack_free copied a partial plan"
    t.cuda.synchronize()
    assert int(plan.counters[3]) == B.STATUS_CODE["VTOKEN_ERR_PLAN_MODE"]
    assert bool((freed == -9).all()), "a freed list was written for a partial plan"


@pytest.mark.parametrize("call", ["free_blocks", "repack_free"])
def test_partial_plan_refused_with_no_table_entries(call):
    """The same refusal for a batch whose requests hold no blocks (M = 0): the freed-list
    workgroups of vtoken_repack_free still run and find the partial mode, as vtoken_free_blocks
    does after vtoken_repack."""
    t = torch()
    B = _B()
    inp = W.from_masks([[], [], []], W.KVShape(1, 2, 64, 16, "fp16"), free_blocks=8, seed=1,
                       name="no_table_entries")
    assert inp.num_bt_entries == 0 and inp.num_reqs == 3
    sh = inp.shape
    print(f"[gpu] partial plan of a batch without table entries handed to {call}", flush=True)
    kv = W.kv_device(sh, inp.num_blocks, 3)
    cache = B.KVCache(kv, sh.num_layers, sh.num_kv_heads, sh.head_dim, sh.block_size)
    batch = B.Batch.from_inputs(inp)
    slot_in = t.zeros(1, dtype=t.int32, device="cuda")
    plan = B.Plan.allocate(batch, sh.block_size)
    state = B.PlannerState.allocate(inp.num_blocks, batch)
    B.plan_partial(cache, batch, slot_in, plan, state, B.PlannerParams())
    t.cuda.synchronize()
    assert plan.counters.cpu().tolist()[3:] == [0, 3]
    if call == "free_blocks":
        B.repack(cache, batch, plan)
        t.cuda.synchronize()
        assert int(plan.counters[3]) == 0
        B.free_blocks(batch, plan)
    else:
        B.repack_free(cache, batch, plan)
    t.cuda.synchronize()
    assert int(plan.counters[3]) == B.STATUS_CODE["VTOKEN_ERR_PLAN_MODE"]


def test_partial_pool_short_defers():
    B = _B()
    inp = W.token_table_inputs(622, W.KVShape(1, 2, 64, 16, "fp16"), num_reqs=12,
                               len_range=(300, 1200), free_blocks=30)
    g, o = partial_parity(inp, B.PlannerParams(), label="short pool")
    assert 0 < o.n_admitted < int((o.src_count > 0).sum())


def test_partial_forced_equals_full_pass():
    """Every block a candidate, no bound, trigger forced, positional layout: the partial pass
    must give the full pass's outputs on the GPU too."""
    t = torch()
    B = _B()
    inp = W.token_table_inputs(623, W.KVShape(2, 4, 64, 16, "bf16"), num_reqs=10,
                               len_range=(100, 900), shuffled_frac=0.0, dropped_frac=0.0,
                               pin_tail=False)
    prm = B.PlannerParams(theta=(-1, 1), max_live_per_source=16, min_eligible=0)
    g, _ = partial_parity(inp, prm, seed=4, label="forced")
    kv = W.kv_device(inp.shape, inp.num_blocks, 4)
    before = kv_bytes(kv, inp.shape)
    full = oracle_repack_inputs(inp, before)
    for key in ("token_slot", "admitted", "new_bt_indptr", "new_block_ids", "src_plan",
                "freed_indptr", "freed"):
        assert np.array_equal(np.asarray(g[key], np.int64),
                              np.asarray(getattr(full, key), np.int64)), key
    del kv
    t.cuda.empty_cache()


def test_partial_chained_passes():
    """Pass 2 runs on the token tables pass 1 left (non-positional), as a serving loop does."""
    t = torch()
    B = _B()
    inp = W.token_table_inputs(624, W.KVShape(1, 2, 64, 16, "bf16"), num_reqs=20,
                               len_range=(300, 2000), shared_groups=2, group_size=3,
                               prefix_tokens=64)
    kv = W.kv_device(inp.shape, inp.num_blocks, 6)
    for step in range(3):
        before = kv_bytes(kv, inp.shape)
        prm = B.PlannerParams(max_sources=40)
        o = run_partial_oracle(inp, before, prm)
        g = gpu_partial(inp, kv, prm, label=f"chained pass {step}")
        assert_partial_equal(g, o, inp)
        assert np.array_equal(kv_bytes(kv, inp.shape), o.kv)
        # next state: the new token table and tables; evict a few more tokens
        rng = np.random.default_rng(step)
        live = inp.live.copy()
        live[(rng.random(len(live)) < 0.1)] = 0
        slot = np.asarray(g["token_slot"], np.int32)
        slot[(live == 0) & (rng.random(len(live)) < 0.5)] = -1
        used = g["used"]
        inp = W.RepackInputs(
            name=inp.name, shape=inp.shape, num_blocks=inp.num_blocks, seq_lens=inp.seq_lens,
            tok_indptr=inp.tok_indptr, bt_indptr=np.asarray(g["new_bt_indptr"], np.int32),
            block_ids=np.asarray(g["new_block_ids"], np.int32), live=live,
            free_list=np.concatenate([inp.free_list[used:], g["freed"]]).astype(np.int32),
            seed=inp.seed, slot_in=slot, pinned=inp.pinned)
    del kv
    t.cuda.empty_cache()


@pytest.mark.parametrize("fault", ["slot_range", "duplicate_slot", "block_range"])
def test_partial_device_errors(fault):
    """Inconsistent token tables set the status word; the copy then writes nothing."""
    t = torch()
    B = _B()
    inp = W.token_table_inputs(625, W.KVShape(1, 2, 64, 16, "fp16"), num_reqs=6,
                               len_range=(100, 400), pin_tail=False)
    slot = inp.slots().copy()
    live = inp.live
    first_live = np.nonzero(live)[0]
    code = "VTOKEN_ERR_SLOT"
    if fault == "slot_range":
        slot[first_live[3]] = inp.num_blocks * inp.shape.block_size + 5
    elif fault == "duplicate_slot":
        a, b = first_live[1], first_live[2]       # same request: its first live tokens
        slot[b] = slot[a]
    else:
        inp.block_ids = inp.block_ids.copy()
        inp.block_ids[2] = inp.num_blocks + 3
        code = "VTOKEN_ERR_BLOCK_RANGE"
    inp.slot_in = slot
    kv = W.kv_device(inp.shape, inp.num_blocks, 8)
    before = kv_bytes(kv, inp.shape)
    # an attempt is forced so that the duplicate slot lands in a source
    prm = B.PlannerParams(theta=(-1, 1), max_live_per_source=16, min_eligible=0)
    g = gpu_partial(inp, kv, prm, label=f"fault {fault}")
    assert g["status"] == B.STATUS_CODE[code], (g["status"], code)
    assert np.array_equal(kv_bytes(kv, inp.shape), before), "KV written despite the error"
    del kv
    t.cuda.empty_cache()


def test_two_cache_groups_share_liveness():
    """Multiple KV-cache groups (Sec. 6): one liveness state, group-specific placement. Two
    pools with their own geometry, block tables and token tables are reclaimed with the same
    live mask on the device; each group matches the oracle run on its own placement."""
    t = torch()
    B = _B()
    a = W.token_table_inputs(631, W.KVShape(2, 8, 128, 16, "bf16"), num_reqs=12,
                             len_range=(400, 2000), shared_groups=1, group_size=3,
                             prefix_tokens=128)
    # group b: same requests and liveness, another pool (4 KV heads of 64, block 32)
    b = W.token_table_inputs(632, W.KVShape(1, 4, 64, 32, "fp16"), num_reqs=12,
                             len_range=(400, 2000))
    b.seq_lens, b.tok_indptr, b.live = a.seq_lens, a.tok_indptr, a.live
    b_slots = []
    S = b.shape.block_size
    # lay group b out positionally over fresh tables sized for the shared lengths
    rng = np.random.default_rng(5)
    nb = sum(-(-int(n) // S) for n in a.seq_lens) + 256
    perm = rng.permutation(nb).astype(np.int32)
    o, tables = 0, []
    for n in a.seq_lens:
        m = -(-int(n) // S)
        tables.append(perm[o:o + m])
        p = np.arange(int(n))
        b_slots.append(perm[o:o + m][p // S].astype(np.int64) * S + p % S)
        o += m
    b.num_blocks = nb
    b.bt_indptr = np.concatenate([[0], np.cumsum([len(x) for x in tables])]).astype(np.int32)
    b.block_ids = np.concatenate(tables).astype(np.int32)
    b.free_list = perm[o:].copy()
    b.slot_in = np.concatenate(b_slots).astype(np.int32)
    b.pinned = None
    b.slot_in[a.live == 0] = np.where(rng.random(int((a.live == 0).sum())) < 0.1, -1,
                                      b.slot_in[a.live == 0])
    for inp, seed in ((a, 1), (b, 2)):
        partial_parity(inp, B.PlannerParams(), seed=seed, label=f"group {inp.shape.dtype}")


def test_partial_pass_graph_replay():
    """Planner and copy captured once in a HIP graph and replayed: before each replay new
    liveness (a random subset of the tokens that hold a slot) is written into the captured
    live-mask buffer; every replay equals the oracle on those inputs and the KV bytes the
    previous replay left. The planner clears its state with a kernel, never a memset."""
    import dataclasses
    t = torch()
    B = _B()
    inp = W.token_table_inputs(641, W.KVShape(1, 2, 64, 16, "bf16"), num_reqs=16,
                               len_range=(200, 1500), shared_groups=2, group_size=3,
                               prefix_tokens=96)
    sh = inp.shape
    prm = B.PlannerParams(theta=(-1, 1), max_live_per_source=16, min_eligible=0)
    kv = W.kv_device(sh, inp.num_blocks, 9)
    cache = B.KVCache(kv, sh.num_layers, sh.num_kv_heads, sh.head_dim, sh.block_size)
    batch = B.Batch.from_inputs(inp)
    slot_in = t.from_numpy(np.ascontiguousarray(inp.slots(), dtype=np.int32)).cuda()
    plan = B.Plan.allocate(batch, sh.block_size)
    state = B.PlannerState.allocate(inp.num_blocks, batch, pinned=inp.pinned)
    print(f"[gpu] partial graph replay: R={inp.num_reqs} T={inp.num_tokens}", flush=True)

    def run():
        B.plan_partial(cache, batch, slot_in, plan, state, prm)
        B.repack(cache, batch, plan)

    side = t.cuda.Stream()
    side.wait_stream(t.cuda.current_stream())
    before = kv_bytes(kv, sh)
    with t.cuda.stream(side):
        run()
    t.cuda.current_stream().wait_stream(side)
    t.cuda.synchronize()
    o = run_partial_oracle(inp, before, prm)
    assert_partial_equal(partial_to_host(plan, state, inp), o, inp)
    assert np.array_equal(kv_bytes(kv, sh), o.kv)

    graph = t.cuda.CUDAGraph()
    with t.cuda.graph(graph):
        run()
    rng = np.random.default_rng(3)
    has_slot = inp.slots() >= 0
    for step, keep in enumerate((0.3, 0.6, 0.9)):
        live = (has_slot & (rng.random(inp.num_tokens) < keep)).astype(np.uint8)
        cur = dataclasses.replace(inp, live=live)
        batch.live.copy_(t.from_numpy(live).to(batch.live.device))
        t.cuda.synchronize()
        before = kv_bytes(kv, sh)
        noise = t.randn(256, 256, device="cuda")
        noise = noise @ noise                     # unrelated eager work between replays
        graph.replay()
        t.cuda.synchronize()
        o = run_partial_oracle(cur, before, prm)
        assert_partial_equal(partial_to_host(plan, state, cur), o, cur)
        assert np.array_equal(kv_bytes(kv, sh), o.kv), f"KV bytes, replay {step}"
        assert o.n_admitted > 0


def _random_partial_case(seed):
    """Random geometry, token tables and planner parameters for the partial pass."""
    B = _B()
    rng = np.random.default_rng(seed)
    dtype = ["fp16", "bf16", "fp8_e4m3"][int(rng.integers(3))]
    e = 1 if dtype == "fp8_e4m3" else 2
    while True:
        S = int(rng.choice([1, 2, 3, 4, 8, 16, 24, 32, 64]))
        H = int(rng.integers(1, 9))
        D = int(rng.choice([16, 32, 64, 128]))
        if (H * D * e) % 16 == 0:
            break
    R = int(rng.integers(1, 25))
    lo = int(rng.integers(1, 600))
    inp = W.token_table_inputs(
        seed, W.KVShape(int(rng.integers(1, 3)), H, D, S, dtype), num_reqs=R,
        len_range=(lo, lo + int(rng.integers(0, 1500))), keep=float(rng.uniform(0.05, 0.9)),
        recent=int(rng.integers(0, 4 * S + 1)), shared_groups=int(rng.integers(0, 3)),
        group_size=int(rng.integers(2, 4)), prefix_tokens=int(rng.integers(0, 8 * S + 1)),
        shuffled_frac=float(rng.random()), dropped_frac=float(rng.random() * 0.5),
        pin_tail=bool(rng.integers(2)),
        free_blocks=int(rng.choice([0, 5, 40, 300, 3000])), name=f"partial_fuzz{seed}")
    # mostly parameters under which a pass triggers and moves rows, sometimes the edges
    theta = [(-1, 1), (-1, 1), (0, 1), (1, 4), (1, 2)][int(rng.integers(5))]
    prm = B.PlannerParams(
        theta=theta, max_live_per_source=int(rng.choice([-1, S, S, S // 2, 1, 0])),
        max_sources=int(rng.choice([1 << 40, 1 << 40, 50, 7, 1, 0])),
        min_eligible=int(rng.choice([0, 0, 1, 3])),
        free_watermark=int(rng.choice([-1, -1, -1, 100000, 50, 0])))
    return inp, prm


@pytest.mark.parametrize("seed", range(30))
def test_partial_random_cases(seed):
    """Seeded random geometries (S 1-64 incl. non-powers of two), token tables (shuffled
    layouts, dropped slots, shared prefixes, pins) and planner parameters, bit-exact."""
    inp, prm = _random_partial_case(7000 + seed)
    partial_parity(inp, prm, seed=seed, label=f"fuzz {seed}")
