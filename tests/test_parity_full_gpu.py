"""Parity at full size, in the launch configuration the benchmark times.

The whole Llama-3-8B-shaped cache (32 layers, 8 KV heads, head_dim 128, bf16, block 16, 64
requests of 2K-8K tokens, ~56 GiB) is repacked once through the C ABI. Then:
  - every metadata output equals the oracle's, element by element;
  - three sampled planes (first, middle, last) equal the oracle run on their pre-call bytes;
  - every plane: each row the oracle moves equals the pre-call source row, and every other
    byte equals its pre-call value (a device-side comparison against a pre-call clone, using
    the oracle's move list)."""
import numpy as np
import pytest

from gpu_helpers import assert_kv_equal, assert_plan_equal, gpu_pass, torch
from oracle.repack import oracle_repack_inputs
from paper_2608_13263_amd import workloads as W

pytestmark = pytest.mark.gpu


def _moves(orc, inp):
    S = inp.shape.block_size
    sp = np.asarray(orc.src_plan, dtype=np.int64).reshape(orc.used, S)
    g, j = np.nonzero(sp >= 0)
    src = sp[g, j]
    dst = np.asarray(inp.free_list, dtype=np.int64)[g] * S + j
    return src, dst


def _plane_bytes(kv, p, shape):
    t = torch()
    return kv[p].view(t.uint8).reshape(-1, shape.row_bytes)


def run_full(inp, seed, sample_planes):
    t = torch()
    shape = inp.shape
    print(f"[gpu] full-size {inp.name}: pool {inp.pool_bytes() / 2**30:.1f} GiB, "
          f"{inp.num_reqs} requests", flush=True)
    orc_meta = oracle_repack_inputs(inp)
    kv = W.kv_device(shape, inp.num_blocks, seed)
    pre = np.stack([_plane_bytes(kv, p, shape).cpu().numpy() for p in sample_planes])
    clone = kv.clone()
    gpu = gpu_pass(inp, kv, label=f"full-size {inp.name}")
    assert_plan_equal(gpu, orc_meta)

    orc = oracle_repack_inputs(inp, pre)
    post = np.stack([_plane_bytes(kv, p, shape).cpu().numpy() for p in sample_planes])
    assert_kv_equal(post, orc.kv)

    src, dst = _moves(orc_meta, inp)
    src_t = t.from_numpy(src).cuda()
    dst_t = t.from_numpy(dst).cuda()
    for p in range(shape.num_planes):
        cb = _plane_bytes(clone, p, shape)
        cb[dst_t] = cb[src_t]
        assert t.equal(_plane_bytes(kv, p, shape), cb), f"plane {p} differs"
    live = int(np.asarray(orc_meta.live_count)[np.asarray(orc_meta.admitted) == 1].sum())
    print(f"[gpu] full-size {inp.name}: {live} live tokens repacked, used {orc_meta.used} "
          f"blocks, freed {orc_meta.n_freed}", flush=True)
    del kv, clone
    t.cuda.empty_cache()


def test_llama3_8b_random_full_size():
    inp = W.llama3_8b_random(201)
    run_full(inp, seed=1, sample_planes=[0, 31, 63])
