"""Secondary check: decode attention that reads the repacked cache through the new token
table equals dense attention over only the live tokens of the cache before the pass.

Reference: float64 dense attention (oracle/attention.py) over the live tokens of each
request in logical order, K/V taken from the pre-call bytes at their old slots. Under test:
float32 attention on the GPU whose keys and values are gathered from the post-call cache
through the slots the HIP path returned (token_slot of the live tokens, which for a
repacked request walks its new block table: slot = block * S + offset, Sec. 3.4). GQA with
G query heads per KV head. Tolerance: 2e-2 absolute and 1e-2 relative (bf16 / fp8 inputs,
fp32 math); fp8 values are dequantised to float32 first."""
import numpy as np
import pytest

from gpu_helpers import gpu_pass, torch
from oracle.attention import dense_decode
from paper_2608_13263_amd import workloads as W

pytestmark = pytest.mark.gpu

ATOL, RTOL = 2e-2, 1e-2


def _check(inp, group, layers, seed=0):
    t = torch()
    sh = inp.shape
    kv = W.kv_device(sh, inp.num_blocks, seed)
    S, H, D = sh.block_size, sh.num_kv_heads, sh.head_dim
    before = kv.float().reshape(sh.num_planes, -1, H, D).cpu().numpy()  # [P][slots][H][D]
    gpu = gpu_pass(inp, kv, label=f"attention check {inp.name}")
    assert gpu["status"] == 0
    after = kv.float().reshape(sh.num_planes, -1, H, D)                  # on the device
    rng = np.random.default_rng(seed)
    worst = 0.0
    for r in range(inp.num_reqs):
        n = int(inp.seq_lens[r])
        a = int(inp.tok_indptr[r])
        bt = inp.block_ids[inp.bt_indptr[r]:inp.bt_indptr[r + 1]].astype(np.int64)
        live = np.nonzero(inp.live[a:a + n])[0]
        old_slots = bt[live // S] * S + live % S
        new_slots = gpu["token_slot"][a + live].astype(np.int64)
        assert (new_slots >= 0).all()
        idx = t.from_numpy(new_slots).cuda()
        for layer in layers:
            q = rng.standard_normal((H * group, D))
            ref = dense_decode(q, before[2 * layer][old_slots], before[2 * layer + 1][old_slots])
            k = after[2 * layer][idx]                # [c][H][D]
            v = after[2 * layer + 1][idx]
            qt = t.from_numpy(q).float().cuda().view(H, group, D).contiguous()
            if len(new_slots) == 0:
                out = np.zeros_like(ref)
            else:
                kt = k.permute(1, 2, 0).contiguous()        # [H][D][c], float32
                vt = v.permute(1, 0, 2).contiguous()        # [H][c][D]
                w = t.softmax(t.bmm(qt, kt) / np.sqrt(D), dim=-1)
                out = t.bmm(w, vt).reshape(H * group, D).cpu().numpy()
            np.testing.assert_allclose(out, ref, atol=ATOL, rtol=RTOL)
            worst = max(worst, float(np.abs(out - ref).max()))
    print(f"[gpu] attention check {inp.name}: max |diff| {worst:.2e}", flush=True)
    del kv
    t.cuda.empty_cache()


def test_attention_llama3_8b_random():
    inp = W.llama3_8b_random(211, num_layers=2, num_reqs=8, len_range=(600, 2400))
    _check(inp, group=4, layers=[0, 1])


def test_attention_llama3_8b_h2o():
    inp = W.llama3_8b_h2o(311, num_layers=2, num_reqs=4, len_range=(1000, 3000))
    _check(inp, group=4, layers=[1])


@pytest.mark.parametrize("dtype", ["fp8_e4m3", "bf16"])
def test_attention_llama3_70b_shape(dtype):
    inp = W.llama3_70b_h2o(511, keep=0.3, dtype=dtype, num_layers=2, num_reqs=3,
                           len_range=(2000, 5000))
    _check(inp, group=8, layers=[0, 1])


def test_attention_tiny():
    _check(W.tiny_cache(101), group=1, layers=[0])
