"""Parity at full size, in the launch configuration the benchmark times.

Each full-size cache is repacked through the C ABI. Then:
  - every metadata output equals the oracle's, element by element;
  - three sampled planes (first, middle, last) equal, byte for byte, the oracle run on their
    pre-call bytes (tracked on the host across the passes of a loop);
  - every plane, every row the oracle moves, byte for byte: out of place the sources are never
    written, so each destination row must equal its source row after the pass; in place each
    destination row must equal its source's pre-call bytes, gathered before the pass;
  - every plane, every other row unchanged: for the 56 GiB Llama-3-8B cache byte for byte
    against a pre-call clone on the device; pools too large to clone by 64-bit weighted row
    checksums taken before and after the pass (rows that do not move only).
Llama-3-70B (all six fp8 / bf16 x keep 0.1 / 0.3 / 0.6 variants) and the Scissorhands loop run
as waves: a pass, its outputs applied, the batch re-submitted, until a pass admits nothing."""
import gc

import numpy as np
import pytest

from gpu_helpers import (assert_kv_equal, assert_partial_equal, assert_plan_equal, gpu_partial,
                         gpu_pass, oracle_moves, run_partial_oracle, torch)
from oracle.repack import oracle_repack_inputs
from paper_2608_13263_amd import workloads as W

pytestmark = pytest.mark.gpu


def _plane_bytes(kv, p, shape):
    t = torch()
    return kv[p].view(t.uint8).reshape(-1, shape.row_bytes)


def _row_sums(kv, p, shape):
    """Weighted 64-bit checksum of every row of plane p (wrapping integer arithmetic)."""
    t = torch()
    x = _plane_bytes(kv, p, shape).view(t.int64)
    w = t.arange(1, x.shape[1] + 1, dtype=t.int64, device=x.device) * 2654435761 + 1
    return (x * w).sum(dim=1)


def run_full(inp, seed, sample_planes, clone=True):
    t = torch()
    shape = inp.shape
    print(f"[gpu] full-size {inp.name}: pool {inp.pool_bytes() / 2**30:.1f} GiB, "
          f"{inp.num_reqs} requests", flush=True)
    orc_meta = oracle_repack_inputs(inp)
    kv = W.kv_device(shape, inp.num_blocks, seed)
    pre = np.stack([_plane_bytes(kv, p, shape).cpu().numpy() for p in sample_planes])
    if clone:
        before = kv.clone()
    else:
        before = t.stack([_row_sums(kv, p, shape) for p in range(shape.num_planes)])
    gpu = gpu_pass(inp, kv, label=f"full-size {inp.name}")
    assert_plan_equal(gpu, orc_meta)

    orc = oracle_repack_inputs(inp, pre)
    post = np.stack([_plane_bytes(kv, p, shape).cpu().numpy() for p in sample_planes])
    assert_kv_equal(post, orc.kv)

    _check_all_planes(kv, before, clone, orc_meta, inp)
    live = int(np.asarray(orc_meta.live_count)[np.asarray(orc_meta.admitted) == 1].sum())
    print(f"[gpu] full-size {inp.name}: {live} live tokens repacked, used {orc_meta.used} "
          f"blocks, freed {orc_meta.n_freed}", flush=True)
    del kv, before
    gc.collect()
    t.cuda.empty_cache()


def _check_all_planes(kv, before, clone, orc_meta, inp, inplace=False, pre_src=None):
    """Every plane after a pass: moved rows byte-exact (out of place against their source rows,
    which the pass never writes; in place against `pre_src`, the sources' pre-call bytes), and
    every other row unchanged (byte-exact against a clone, or by row checksums)."""
    t = torch()
    shape = inp.shape
    src, dst = oracle_moves(orc_meta, inp, inplace)
    src_t = t.from_numpy(src).cuda()
    dst_t = t.from_numpy(dst).cuda()
    for p in range(shape.num_planes):
        plane = _plane_bytes(kv, p, shape)
        if clone:
            cb = _plane_bytes(before, p, shape)
            cb[dst_t] = cb[src_t]
            assert t.equal(plane, cb), f"plane {p} differs"
            continue
        moved = plane[dst_t]
        expect = pre_src[p].to(moved.device) if inplace else plane[src_t]
        assert t.equal(moved, expect), f"plane {p}: a moved row differs from its source"
        del moved, expect
        keep = t.ones(plane.shape[0], dtype=t.bool, device=plane.device)
        keep[dst_t] = False
        assert t.equal(_row_sums(kv, p, shape)[keep], before[p][keep]), \
            f"plane {p}: a row that does not move changed (row checksums)"


def _gather_sources(kv, orc_meta, inp):
    """Pre-call bytes of every row an in-place pass moves, plane by plane (rows moved x row
    bytes each; kept on the device when it has room, else on the host)."""
    t = torch()
    shape = inp.shape
    src, _ = oracle_moves(orc_meta, inp, True)
    src_t = t.from_numpy(src).cuda()
    need = shape.num_planes * len(src) * shape.row_bytes
    free, _ = t.cuda.mem_get_info()
    on_host = need > free - (16 << 30)
    out = []
    for p in range(shape.num_planes):
        g = _plane_bytes(kv, p, shape)[src_t]
        out.append(g.cpu() if on_host else g)
    return out


def test_llama3_8b_random_full_size():
    inp = W.llama3_8b_random(201)
    run_full(inp, seed=1, sample_planes=[0, 31, 63])


def test_llama3_8b_random_full_size_serving_pool():
    # the benchmark's default: the same requests in a pool of 90% of free HBM (~258 GiB)
    inp = W.llama3_8b_random(201, pool_bytes=int(0.9 * _budget()))
    run_full(inp, seed=1, sample_planes=[0, 31, 63], clone=False)


def _budget():
    t = torch()
    free, _ = t.cuda.mem_get_info()
    return free


def test_llama3_8b_h2o_full_size():
    # 128 requests of 4K-16K tokens, ~198 GiB pool
    inp = W.llama3_8b_h2o(301)
    assert inp.pool_bytes() < 0.8 * _budget()
    run_full(inp, seed=2, sample_planes=[0, 33, 63], clone=False)


@pytest.mark.parametrize("dtype", ["bf16", "fp8_e4m3"])
def test_llama3_70b_tensor_parallel_share_full_size(dtype):
    # one GPU's share under 8-way tensor parallelism: one KV head, 256 B / 128 B rows; all 32
    # requests fit the pool
    budget = min(240 * 2 ** 30, int(0.85 * _budget()))
    inp = W.llama3_70b_h2o(501, keep=0.3, dtype=dtype, num_kv_heads=1, pool_bytes=budget)
    assert inp.num_reqs == 32
    run_full(inp, seed=4, sample_planes=[0, 97, 159], clone=False)


LLAMA3_70B_VARIANTS = [(d, k) for d in ("fp8_e4m3", "bf16") for k in (0.1, 0.3, 0.6)]


@pytest.mark.parametrize("dtype,keep", LLAMA3_70B_VARIANTS,
                         ids=[f"{d}_k{k}" for d, k in LLAMA3_70B_VARIANTS])
def test_llama3_70b_h2o_waves_full_size(dtype, keep):
    """The Llama-3-70B cache at full size (fit rule: the requests whose blocks take <= 80% of a
    min(240 GiB, 0.85 x free) pool), as waves: the free list cannot supply every destination at
    once, so the first pass defers requests (Sec. 3.3.2); its outputs are applied and the batch
    re-submitted (unconsumed free entries, then the freed blocks) until a pass admits nothing.
    Every pass: all metadata bit-exact against the oracle, the sampled planes byte-exact
    against the oracle's bytes tracked from the initial snapshot, every moved row of every
    plane byte-exact, every other row unchanged. At the end no profitable request is left
    deferred: each holds ceil(live/S) blocks."""
    t = torch()
    budget = min(240 * 2 ** 30, int(0.85 * _budget()))
    inp = W.llama3_70b_h2o(501, keep=keep, dtype=dtype, pool_bytes=budget)
    shape = inp.shape
    S = shape.block_size
    sample = [0, 81, 159]
    print(f"[gpu] 70B waves {dtype} keep {keep}: pool {inp.pool_bytes() / 2**30:.1f} GiB, "
          f"{inp.num_reqs} requests", flush=True)
    kv = W.kv_device(shape, inp.num_blocks, 3)
    host = np.stack([_plane_bytes(kv, p, shape).cpu().numpy() for p in sample])
    waves = []
    for wave in range(16):
        orc_meta = oracle_repack_inputs(inp)
        before = t.stack([_row_sums(kv, p, shape) for p in range(shape.num_planes)])
        gpu = gpu_pass(inp, kv, label=f"70B {dtype} k{keep} wave {wave}")
        assert_plan_equal(gpu, orc_meta)
        orc = oracle_repack_inputs(inp, host)
        host = orc.kv
        post = np.stack([_plane_bytes(kv, p, shape).cpu().numpy() for p in sample])
        assert_kv_equal(post, host)
        _check_all_planes(kv, before, False, orc_meta, inp)
        del before
        adm = np.asarray(orc_meta.admitted)
        need = -(-np.asarray(orc_meta.live_count, np.int64) // S)
        deferred = int(((need < np.diff(inp.bt_indptr)) & (adm == 0)).sum())
        moved = int(np.asarray(orc_meta.live_count)[adm == 1].sum())
        waves.append((int(orc_meta.n_admitted), deferred, moved))
        print(f"[gpu] 70B {dtype} k{keep} wave {wave}: {orc_meta.n_admitted} admitted, "
              f"{deferred} deferred, {moved} live tokens moved, {orc_meta.used} destinations, "
              f"{orc_meta.n_freed} freed", flush=True)
        if orc_meta.n_admitted == 0:
            break
        inp = W.next_wave(inp, orc_meta.admitted, orc_meta.live_count, orc_meta.new_bt_indptr,
                          orc_meta.new_block_ids, orc_meta.used, orc_meta.freed)
    assert waves[-1][0] == 0 and waves[-1][1] == 0, f"requests left deferred: {waves}"
    for r in range(inp.num_reqs):
        c = int(inp.request_live(r).sum())
        assert len(inp.request_blocks(r)) == -(-c // S)
    del kv
    gc.collect()
    t.cuda.empty_cache()


def test_llama3_8b_scissorhands_rounds_with_waves():
    """256 requests, a repack every 512 decode steps in a pool too small for one pass: each
    round runs passes until one repacks nothing. The stream is driven by the oracle's outputs;
    every pass's GPU outputs must equal the oracle's, the sampled planes must equal the
    oracle's bytes (tracked on the host from the initial snapshot), and every plane must pass
    the all-plane check of that pass (moved rows byte-exact, other rows unchanged)."""
    t = torch()
    budget = min(240 * 2 ** 30, int(0.85 * _budget()))
    shape = W.KVShape(32, 8, 128, 16, "bf16")
    stream = W.ScissorhandsStream(seed=401, pool_blocks=int(budget // shape.block_bytes))
    sample = [0, 27, 63]
    kv = W.kv_device(shape, stream.num_blocks, 4)
    host = np.stack([_plane_bytes(kv, p, shape).cpu().numpy() for p in sample])
    total_moved = 0
    for rnd in range(2):
        stream.decode()
        for wave in range(8):
            inp = stream.inputs()
            orc_meta = oracle_repack_inputs(inp)
            before = t.stack([_row_sums(kv, p, shape) for p in range(shape.num_planes)])
            gpu = gpu_pass(inp, kv, label=f"scissorhands round {rnd} wave {wave}")
            assert_plan_equal(gpu, orc_meta)
            orc = oracle_repack_inputs(inp, host)
            host = orc.kv
            post = np.stack([_plane_bytes(kv, p, shape).cpu().numpy() for p in sample])
            assert_kv_equal(post, host)
            _check_all_planes(kv, before, False, orc_meta, inp)
            del before
            moved = int(np.asarray(orc_meta.live_count)[np.asarray(orc_meta.admitted) == 1].sum())
            total_moved += moved
            print(f"[gpu] round {rnd} wave {wave}: {orc_meta.n_admitted} admitted, {moved} live "
                  f"tokens moved, {orc_meta.used} destinations, {orc_meta.n_freed} freed",
                  flush=True)
            stream.commit(orc_meta.admitted, orc_meta.new_bt_indptr, orc_meta.new_block_ids,
                          orc_meta.used, orc_meta.freed)
            if orc_meta.n_admitted == 0:
                break
        assert wave >= 1, "the pool should force at least two passes per round"
    assert total_moved > 0
    del kv
    gc.collect()
    t.cuda.empty_cache()


def test_llama3_8b_scissorhands_partial_rounds():
    """The same loop driven by the partial pass at full size (token tables, append blocks
    pinned, theta_F = 0.25): rounds until a pass is attempted and admits requests. Every
    pass's GPU outputs equal the oracle's; the sampled planes equal the oracle's bytes
    (tracked on the host); every plane passes the all-plane check of the moves (moved rows
    byte-exact, other rows unchanged)."""
    t = torch()
    from paper_2608_13263_amd import binding as B
    budget = min(240 * 2 ** 30, int(0.85 * _budget()))
    shape = W.KVShape(32, 8, 128, 16, "bf16")
    stream = W.PartialStream(seed=401, pool_blocks=int(budget // shape.block_bytes))
    sample = [0, 40, 63]
    kv = W.kv_device(shape, stream.num_blocks, 5)
    host = np.stack([_plane_bytes(kv, p, shape).cpu().numpy() for p in sample])
    params = B.PlannerParams()
    moved_total = 0
    for rnd in range(6):
        stream.decode()
        for wave in range(8):
            inp = stream.inputs()
            orc_meta = run_partial_oracle(inp, None, params)
            before = t.stack([_row_sums(kv, p, shape) for p in range(shape.num_planes)])
            gpu = gpu_partial(inp, kv, params, label=f"round {rnd} wave {wave}")
            assert_partial_equal(gpu, orc_meta, inp)
            orc = run_partial_oracle(inp, host, params)
            host = orc.kv
            post = np.stack([_plane_bytes(kv, p, shape).cpu().numpy() for p in sample])
            assert_kv_equal(post, host)
            _check_all_planes(kv, before, False, orc_meta, inp)
            del before
            moved_total += orc_meta.tokens_moved
            print(f"[gpu] partial round {rnd} wave {wave}: F {1 - orc_meta.live_total / (16 * max(orc_meta.allocated, 1)):.3f}, "
                  f"attempted {orc_meta.triggered}, {orc_meta.n_admitted} admitted, "
                  f"{orc_meta.tokens_moved} tokens moved, {orc_meta.n_freed} released",
                  flush=True)
            stream.commit(orc_meta.token_slot, orc_meta.new_bt_indptr, orc_meta.new_block_ids,
                          orc_meta.used, orc_meta.freed)
            if orc_meta.n_admitted == 0:
                break
        if moved_total > 0:
            break
    assert moved_total > 0, "no round triggered the partial pass"
    del kv
    gc.collect()
    t.cuda.empty_cache()


def test_llama3_8b_shared_prefix_full_size():
    """The prefix-caching workload the benchmark times (64 requests, 16 groups of 4 sharing
    1024 tokens, 258 GiB pool), one partial pass: every output against the partial-pass
    oracle, the shared blocks neither sources nor touched, sampled planes byte-exact against
    the oracle run on their pre-call bytes, every moved row of every plane byte-exact, other
    rows unchanged by row checksums."""
    t = torch()
    from paper_2608_13263_amd import binding as B
    inp = W.llama3_8b_shared_prefix(701, pool_bytes=int(0.9 * _budget()))
    shape = inp.shape
    sample = [0, 31, 63]
    print(f"[gpu] full-size {inp.name}: pool {inp.pool_bytes() / 2**30:.1f} GiB", flush=True)
    params = B.PlannerParams()
    orc_meta = run_partial_oracle(inp, None, params)
    shared = {b for b, n in orc_meta.refs.items() if n > 1}
    assert len(shared) == 16 * 64 and not shared & set(int(b) for b in orc_meta.freed)
    kv = W.kv_device(shape, inp.num_blocks, 9)
    pre = np.stack([_plane_bytes(kv, p, shape).cpu().numpy() for p in sample])
    before = t.stack([_row_sums(kv, p, shape) for p in range(shape.num_planes)])
    gpu = gpu_partial(inp, kv, params, label=f"full-size {inp.name}")
    assert_partial_equal(gpu, orc_meta, inp)
    orc = run_partial_oracle(inp, pre, params)
    post = np.stack([_plane_bytes(kv, p, shape).cpu().numpy() for p in sample])
    assert_kv_equal(post, orc.kv)
    _check_all_planes(kv, before, False, orc_meta, inp)
    print(f"[gpu] full-size {inp.name}: {orc_meta.tokens_moved} tokens moved, "
          f"{len(shared)} shared blocks kept", flush=True)
    del kv, before
    gc.collect()
    t.cuda.empty_cache()


@pytest.mark.parametrize("config", ["llama3_8b_h2o", "llama3_70b_bf16", "llama3_70b_fp8"])
def test_inplace_full_size(config):
    """In-place mode at full size in the launch configuration the benchmark times: every
    metadata output equals the oracle's in-place mode, sampled planes byte-exact against the
    oracle run on their pre-call bytes, every moved row of every plane byte-exact against its
    source's pre-call bytes (gathered before the pass: the moves apply to the pre-call rows
    all at once, the definition of a move), other rows unchanged by row checksums."""
    t = torch()
    if config == "llama3_8b_h2o":
        inp = W.llama3_8b_h2o(301)
        sample = [0, 33, 63]
    else:
        budget = min(240 * 2 ** 30, int(0.85 * _budget()))
        dtype = "bf16" if config == "llama3_70b_bf16" else "fp8_e4m3"
        inp = W.llama3_70b_h2o(501, keep=0.3, dtype=dtype, pool_bytes=budget)
        sample = [0, 81, 159]
    shape = inp.shape
    print(f"[gpu] in-place full-size {inp.name}: pool {inp.pool_bytes() / 2**30:.1f} GiB",
          flush=True)
    orc_meta = oracle_repack_inputs(inp, inplace=True)
    kv = W.kv_device(shape, inp.num_blocks, 7)
    pre = np.stack([_plane_bytes(kv, p, shape).cpu().numpy() for p in sample])
    before = t.stack([_row_sums(kv, p, shape) for p in range(shape.num_planes)])
    pre_src = _gather_sources(kv, orc_meta, inp)
    gpu = gpu_pass(inp, kv, inplace=True, label=f"in-place full-size {inp.name}")
    assert_plan_equal(gpu, orc_meta)
    orc = oracle_repack_inputs(inp, pre, inplace=True)
    post = np.stack([_plane_bytes(kv, p, shape).cpu().numpy() for p in sample])
    assert_kv_equal(post, orc.kv)
    _check_all_planes(kv, before, False, orc_meta, inp, inplace=True, pre_src=pre_src)
    del pre_src
    src, _ = oracle_moves(orc_meta, inp, True)
    print(f"[gpu] in-place full-size {inp.name}: {orc_meta.n_admitted} requests, {len(src)} rows "
          f"moved per plane", flush=True)
    del kv, before
    gc.collect()
    t.cuda.empty_cache()


@pytest.mark.parametrize("config,G", [("llama3_8b_h2o", 4), ("llama3_70b_fp8", 8)])
def test_decode_full_size_sampled(config, G):
    """Decode over a full cache after a pass, in the launch configuration the decode benchmark
    times (every request, the first and last layers): eight sampled requests against the
    float64 oracle computed one by one from their own K/V rows. Llama-3-8B H2O with 32 query
    heads, Llama-3-70B H2O fp8 with 64."""
    t = torch()
    from oracle.attention import dense_decode, slot_mapping
    from paper_2608_13263_amd import binding as B
    if config == "llama3_8b_h2o":
        inp = W.llama3_8b_h2o(301)
    else:
        budget = min(240 * 2 ** 30, int(0.85 * _budget()))
        inp = W.llama3_70b_h2o(501, keep=0.3, dtype="fp8_e4m3", pool_bytes=budget)
    shape = inp.shape
    S, H, D = shape.block_size, shape.num_kv_heads, shape.head_dim
    kv = W.kv_device(shape, inp.num_blocks, 8)
    orc = oracle_repack_inputs(inp)
    gpu = gpu_pass(inp, kv, label="decode full-size pass")
    assert_plan_equal(gpu, orc)
    cache = B.KVCache(kv, shape.num_layers, H, D, S)
    indptr, slots = slot_mapping(orc.token_slot, inp.tok_indptr, inp.seq_lens)
    d_indptr = t.from_numpy(indptr.astype(np.int32)).cuda()
    d_slots = t.from_numpy(slots.astype(np.int32)).cuda()
    max_tokens = int(np.diff(indptr).max())
    q = t.randn(inp.num_reqs, G * H, D, device="cuda",
                generator=t.Generator(device="cuda").manual_seed(3))
    rng = np.random.default_rng(9)
    sample = rng.choice(inp.num_reqs, size=min(8, inp.num_reqs), replace=False)
    worst = 0.0
    for layer in (0, shape.num_layers - 1):
        out = B.paged_decode(cache, q, d_indptr, d_slots, layer, max_tokens).cpu().numpy()
        kp = kv[2 * layer].reshape(-1, H, D)
        vp = kv[2 * layer + 1].reshape(-1, H, D)
        for r in sample:
            sl = t.from_numpy(slots[indptr[r]:indptr[r + 1]]).cuda()
            k = kp[sl].float().cpu().numpy()
            v = vp[sl].float().cpu().numpy()
            ref = dense_decode(q[r].cpu().numpy().astype(np.float64), k, v)
            np.testing.assert_allclose(out[r], ref, atol=1e-4, rtol=1e-4)
            worst = max(worst, float(np.abs(out[r] - ref).max()))
    print(f"[gpu] decode full-size {inp.name}: {len(sample)} sampled requests x 2 layers, "
          f"max |diff| {worst:.2e}", flush=True)
    del kv
    gc.collect()
    t.cuda.empty_cache()
