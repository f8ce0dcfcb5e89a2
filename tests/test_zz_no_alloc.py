"""The allocation-free decode entry point (vtoken_paged_decode_noalloc) through the C ABI: its
split partials live in the library-held device array instead of a caller workspace. Two
calls in a row, the second smaller than the first, each must give exactly the outputs of
vtoken_paged_decode with a caller workspace on the same inputs (the same kernels; the array
keeps the first call's partials when the second runs), and the second is also held to the
float64 oracle at the decode's tolerance. A call whose partials exceed the array is refused."""
import numpy as np
import pytest

from gpu_helpers import kv_bytes, torch
from oracle.attention import decode_batch, slot_mapping
from oracle.repack import oracle_repack_inputs
from paper_2608_13263_amd import workloads as W

pytestmark = pytest.mark.gpu

ATOL, RTOL = 1e-4, 1e-4


def _positional_mapping(inp):
    """Slots of the live tokens before any pass (block * S + offset of each live position)."""
    S = inp.shape.block_size
    indptr, slots = [0], []
    for r in range(inp.num_reqs):
        a = int(inp.tok_indptr[r])
        bt = inp.block_ids[inp.bt_indptr[r]:inp.bt_indptr[r + 1]].astype(np.int64)
        pos = np.nonzero(inp.live[a:a + int(inp.seq_lens[r])])[0]
        slots.extend((bt[pos // S] * S + pos % S).tolist())
        indptr.append(len(slots))
    return np.asarray(indptr, np.int64), np.asarray(slots, np.int64)


def _both(B, cache, q, indptr, slots, layer, max_tokens):
    t = torch()
    ref = B.paged_decode(cache, q, indptr, slots, layer, max_tokens)
    out = t.full_like(q, float("nan"))
    B.paged_decode_noalloc(cache, q, indptr, slots, layer, max_tokens, out=out)
    t.cuda.synchronize()
    return ref, out


def test_noalloc_decode_equals_workspace_decode_on_two_calls():
    t = torch()
    from paper_2608_13263_amd import binding as B
    dev = lambda x: t.from_numpy(np.asarray(x, dtype=np.int32)).cuda()  # noqa: E731

    # call 1: Llama-3-8B H2O geometry, one layer, all 128 requests, 32 query heads: partials
    # close to the array's size
    big = W.llama3_8b_h2o(301, num_layers=1)
    sh = big.shape
    kv = W.kv_device(sh, big.num_blocks, 21)
    cache = B.KVCache(kv, sh.num_layers, sh.num_kv_heads, sh.head_dim, sh.block_size)
    indptr, slots = _positional_mapping(big)
    max_tokens = int(np.diff(indptr).max())
    need = B.decode_workspace_bytes(big.num_reqs, 32, sh.head_dim, max_tokens)
    print(f"[gpu] no-alloc decode call 1: {big.num_reqs} requests, max {max_tokens} tokens, "
          f"partials bound {need / 2**20:.1f} MiB of {B.DECODE_SCRATCH_BYTES >> 20}", flush=True)
    assert need > B.DECODE_SCRATCH_BYTES // 2
    q = t.randn(big.num_reqs, 32, sh.head_dim, device="cuda",
                generator=t.Generator(device="cuda").manual_seed(1))
    ref, out = _both(B, cache, q, dev(indptr), dev(slots), 0, max_tokens)
    assert t.equal(ref, out), "call 1 differs from the workspace entry point"
    del kv, cache
    t.cuda.empty_cache()

    # call 2: a smaller batch (fp8, G = 8, 10 requests of split-edge lengths), after a repack
    # pass; the array still holds call 1's partials
    sh2 = W.KVShape(2, 2, 128, 32, "fp8_e4m3")
    masks = [[0] * 50, [0] * 9 + [1], [1] * 255, [1] * 256 + [0] * 7, [1] * 257,
             [1, 1, 0] * 257, [1] * 1023, [0] * 3 + [1] * 1024, [1] * 1025, [1] * 2049]
    M = sum(-(-len(m) // 32) for m in masks)
    small = W.from_masks(masks, sh2, free_blocks=M + 64, seed=5, name="noalloc_small")
    kv2 = W.kv_device(sh2, small.num_blocks, 22)
    orc = oracle_repack_inputs(small, kv_bytes(kv2, sh2))
    cache2 = B.KVCache(kv2, sh2.num_layers, sh2.num_kv_heads, sh2.head_dim, sh2.block_size)
    batch = B.Batch.from_inputs(small)
    plan = B.run_pass(cache2, batch)
    d_indptr, d_slots = B.build_slot_mapping(batch, plan)
    ref_indptr, ref_slots = slot_mapping(orc.token_slot, small.tok_indptr, small.seq_lens)
    max2 = int(np.diff(ref_indptr).max())
    print(f"[gpu] no-alloc decode call 2: {small.num_reqs} requests, max {max2} tokens", flush=True)
    q2 = t.randn(small.num_reqs, 16, 128, device="cuda",
                 generator=t.Generator(device="cuda").manual_seed(2))
    ref2, out2 = _both(B, cache2, q2, d_indptr, d_slots, 1, max2)
    assert t.equal(ref2, out2), "call 2 differs from the workspace entry point"
    vals = t.from_numpy(np.ascontiguousarray(orc.kv)).view(t.float8_e4m3fn).float()
    vals = vals.reshape(orc.kv.shape[0], orc.kv.shape[1], 2, 128).double().numpy()
    want = decode_batch(q2.cpu().numpy(), vals[2], vals[3], ref_indptr, ref_slots)
    np.testing.assert_allclose(out2.cpu().numpy().astype(np.float64), want, atol=ATOL,
                               rtol=RTOL)
    assert np.array_equal(out2[0].cpu().numpy(), np.zeros((16, 128), np.float32))


def test_noalloc_decode_refuses_partials_beyond_the_array():
    t = torch()
    from paper_2608_13263_amd import binding as B
    sh = W.KVShape(1, 8, 128, 16, "bf16")
    kv = t.zeros(sh.num_planes, 64, 16, 8, 128, dtype=t.bfloat16, device="cuda")
    cache = B.KVCache(kv, 1, 8, 128, 16)
    q = t.zeros(4, 32, 128, device="cuda")
    out = t.zeros_like(q)
    indptr = t.zeros(5, dtype=t.int32, device="cuda")
    slots = t.zeros(1, dtype=t.int32, device="cuda")
    # 4 requests x 32 heads x 1000 splits x 130 x 4 B = 63.5 MiB fits; 1100 splits do not
    B.paged_decode_noalloc(cache, q, indptr, slots, 0, 1000 * 128, out=out)
    t.cuda.synchronize()
    assert bool((out == 0).all())
    with pytest.raises(B.VTokenError, match="CAPACITY"):
        B.paged_decode_noalloc(cache, q, indptr, slots, 0, 1100 * 128, out=out)
