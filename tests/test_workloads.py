"""Seeded input generators: determinism, the closed forms of the liveness recipes, and the
oracle's invariants on the workload shapes (no GPU)."""
import hashlib
import math

import numpy as np
import pytest

from paper_2608_13263_amd import workloads as W
from oracle.repack import oracle_repack_inputs
from oracle.invariants import check_invariants


def _digest(inp):
    h = hashlib.sha256()
    for a in (inp.seq_lens, inp.tok_indptr, inp.bt_indptr, inp.block_ids, inp.live,
              inp.free_list):
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def test_same_seed_same_inputs():
    assert _digest(W.tiny_cache(7)) == _digest(W.tiny_cache(7))
    assert _digest(W.tiny_cache(7)) != _digest(W.tiny_cache(8))
    a = W.llama3_8b_random(3, num_layers=1, num_reqs=4)
    b = W.llama3_8b_random(3, num_layers=1, num_reqs=4)
    assert _digest(a) == _digest(b)


def test_pool_is_a_permutation():
    for inp in (W.tiny_cache(), W.llama3_8b_random(num_layers=1, num_reqs=8),
                W.llama3_8b_h2o(num_layers=1, num_reqs=4)):
        allb = np.concatenate([inp.block_ids, inp.free_list])
        assert np.array_equal(np.sort(allb), np.arange(inp.num_blocks))
        for r in range(inp.num_reqs):
            n = int(inp.seq_lens[r])
            assert len(inp.request_blocks(r)) == math.ceil(n / inp.shape.block_size)
            assert len(inp.request_live(r)) == n


def test_tiny_recipe():
    inp = W.tiny_cache()
    assert inp.num_blocks == 512 and inp.num_reqs == 8
    assert inp.shape.row_bytes == 256
    for r in range(8):
        assert 100 <= inp.seq_lens[r] <= 500
        assert inp.request_live(r)[:4].all()


@pytest.mark.parametrize("keep,recent,maker", [(0.3, 64, W.llama3_8b_random),
                                               (0.2, 128, W.llama3_8b_h2o)])
def test_live_count_closed_form(keep, recent, maker):
    inp = maker(num_layers=1, num_reqs=6)
    for r in range(inp.num_reqs):
        n = int(inp.seq_lens[r])
        lv = inp.request_live(r)
        assert int(lv.sum()) == math.floor(keep * n) + recent
        assert lv[n - recent:].all()


def test_h2o_prefers_heavy_hitters():
    rng = np.random.default_rng(0)
    lv = W.h2o_live(rng, 8192, 0.2, 128)
    # Zipf mass concentrates on early positions: the first 64 are all heavy hitters
    assert lv[:64].all()
    assert lv.sum() == math.floor(0.2 * 8192) + 128


def test_70b_fit_rule():
    shape_bytes = W.KVShape(80, 8, 128, 32, "bf16").block_bytes
    inp = W.llama3_70b_h2o(keep=0.3, dtype="bf16", pool_bytes=240 * 2 ** 30)
    resident = len(inp.block_ids)
    assert resident <= 0.8 * inp.num_blocks
    assert inp.num_blocks * shape_bytes <= 240 * 2 ** 30
    assert inp.shape.row_bytes == 2048
    fp8 = W.llama3_70b_h2o(keep=0.3, dtype="fp8_e4m3", pool_bytes=240 * 2 ** 30)
    assert fp8.shape.row_bytes == 1024 and fp8.num_reqs >= inp.num_reqs


@pytest.mark.parametrize("maker,kw", [
    (W.tiny_cache, {}),
    (W.llama3_8b_random, dict(num_layers=1, num_reqs=6, len_range=(200, 900))),
    (W.llama3_8b_h2o, dict(num_layers=1, num_reqs=4, len_range=(300, 1200))),
    (W.llama3_70b_h2o, dict(num_layers=1, num_reqs=3, len_range=(500, 2000))),
])
def test_oracle_invariants_on_workload_shapes(maker, kw):
    inp = maker(**kw)
    kv = W.kv_host(W.KVShape(1, 1, 8, inp.shape.block_size, "fp16"), inp.num_blocks, 1)
    res = oracle_repack_inputs(inp, kv)
    check_invariants(inp.seq_lens, inp.tok_indptr, inp.bt_indptr, inp.block_ids, inp.live,
                     inp.free_list, inp.shape.block_size, inp.num_blocks, res.token_slot,
                     res.new_bt_indptr, res.new_block_ids, res.freed, res.used, kv, res.kv)
    assert res.n_admitted > 0


@pytest.mark.parametrize("S,top", [(16, "source"), (16, "destination"), (1, "source"),
                                   (64, "destination")])
def test_slot_limit_inputs(S, top):
    masks = [np.ones(40, np.uint8), np.zeros(0, np.uint8), (np.arange(300) % 3 == 0)]
    inp = W.slot_limit_inputs(W.KVShape(1, 1, 16, S, "fp8_e4m3"), masks, seed=5, top_block=top)
    nb = inp.num_blocks
    assert nb * S <= 2 ** 31 - 1 < (nb + 1) * S
    ids = np.concatenate([inp.block_ids, inp.free_list]).astype(np.int64)
    assert len(np.unique(ids)) == len(ids) and ids.min() >= nb - len(ids) and ids.max() == nb - 1
    assert list(np.diff(inp.bt_indptr)) == [-(-len(m) // S) for m in masks]
    assert list(inp.seq_lens) == [len(m) for m in masks] and len(inp.free_list) == 1024
    assert (inp.block_ids[0] if top == "source" else inp.free_list[0]) == nb - 1
    with pytest.raises(ValueError):
        W.slot_limit_inputs(inp.shape, masks, seed=5, top_block="middle")


@pytest.mark.parametrize("keep", [0.1, 0.3, 0.6])
def test_waves_pack_every_request(keep):
    """Passes over one batch with a pool too small for every destination at once (the
    Llama-3-70B recipe's deferral, Sec. 3.3.2), each re-submitted through next_wave: the first
    pass defers requests, each later pass admits a prefix of the deferred ones, and when a pass
    admits nothing every request holds exactly ceil(live/S) blocks. Blocks are conserved and
    each request's live rows (tracked as bytes through every pass) keep their logical order."""
    shape = W.KVShape(1, 1, 8, 8, "fp16")           # 16-byte rows
    inp = W.llama3_70b_h2o(501, keep=keep, dtype="fp16", num_layers=1, num_kv_heads=1,
                           len_range=(200, 900), num_reqs=12, resident_frac=0.75)
    inp = W.RepackInputs(**{**inp.__dict__, "shape": W.KVShape(1, 1, 8, 32, "fp16")})
    S = inp.shape.block_size
    rng = np.random.default_rng(1)
    kv = rng.integers(0, 256, size=(2, inp.num_blocks * S, 16), dtype=np.uint8)
    # each live token's payload before any pass, in logical order per request
    want = []
    for r in range(inp.num_reqs):
        p = np.nonzero(inp.request_live(r))[0]
        bt = inp.request_blocks(r).astype(np.int64)
        want.append(kv[:, bt[p // S] * S + p % S].copy())
    # keep only the free blocks the first pass's deferral needs: about half the destinations
    need0 = sum(-(-int(inp.request_live(r).sum()) // S) for r in range(inp.num_reqs))
    inp = W.RepackInputs(**{**inp.__dict__, "free_list": inp.free_list[:max(need0 // 2, 1)]})
    pool = set(inp.block_ids.tolist()) | set(inp.free_list.tolist())
    profitable = sum(-(-int(inp.request_live(r).sum()) // S) < len(inp.request_blocks(r))
                     for r in range(inp.num_reqs))
    admitted_per_wave = []
    for wave in range(64):
        res = oracle_repack_inputs(inp, kv)
        kv = res.kv
        admitted_per_wave.append(int(res.n_admitted))
        if res.n_admitted == 0:
            break
        inp = W.next_wave(inp, res.admitted, res.live_count, res.new_bt_indptr,
                          res.new_block_ids, res.used, res.freed)
        assert set(inp.block_ids.tolist()) | set(inp.free_list.tolist()) == pool
        assert len(inp.block_ids) + len(inp.free_list) == len(pool)
    assert admitted_per_wave[0] < profitable and len(admitted_per_wave) > 2, admitted_per_wave
    assert sum(admitted_per_wave) == profitable
    for r in range(inp.num_reqs):
        c = int(inp.request_live(r).sum())
        assert inp.request_live(r).all() and len(inp.request_blocks(r)) == -(-c // S)
        bt = inp.request_blocks(r).astype(np.int64)
        p = np.arange(c)
        assert np.array_equal(kv[:, bt[p // S] * S + p % S], want[r]), f"request {r}"
