"""Consumer side of the repack through the C ABI: the attention slot mapping (Sec. 3.4), the
HIP paged decode that reads the cache through it, the relocation-stream / event ordering of
Sec. 3.3.4 and invariant I3 (Sec. 3.5), and graph replay with a mutable slot buffer (Sec. 3.4,
CUDA Graph compatibility).

Parity bars:
  slot mapping   bit-exact against oracle.attention.slot_mapping of the oracle's token table
  decode         against oracle.attention.decode_batch (float64) over the oracle's post-pass
                 cache, |diff| <= 1e-4 + 1e-4 |ref|. The kernel computes in float32 from
                 inputs that are exact in float32 (fp16 / bf16 / e4m3 values): dot products
                 of at most 256 terms of magnitude < 40 err by < 1e-5 before the softmax
                 scale, exp and the normalising sum add a few float32 ulps per weight, so
                 outputs (values of magnitude < 5) err by well under 1e-4.
  decode of one key returns that key's value row exactly, so every fp16, bf16 and e4m3 code
                 is checked bit for bit against torch's CPU conversion
  before/after   decode through the old slots over the old cache and through the new slots
                 over the repacked cache are bit-identical (the same values in the same
                 order), also after the released blocks are overwritten (I1, Sec. 3.5)
"""
import numpy as np
import pytest

from gpu_helpers import kv_bytes, torch
from oracle.attention import append_to_table, decode_batch, slot_mapping, slot_table
from oracle.repack import oracle_repack_inputs
from paper_2608_13263_amd import workloads as W

pytestmark = pytest.mark.gpu

ATOL, RTOL = 1e-4, 1e-4


def _B():
    from paper_2608_13263_amd import binding as B
    return B


def _values(kv_u8: np.ndarray, shape: W.KVShape) -> np.ndarray:
    """uint8 [P][slots][row_bytes] -> float64 [P][slots][H][D] via torch's CPU conversion."""
    t = torch()
    x = t.from_numpy(np.ascontiguousarray(kv_u8)).view(W.torch_dtype(shape)).float()
    return x.reshape(kv_u8.shape[0], kv_u8.shape[1], shape.num_kv_heads,
                     shape.head_dim).double().numpy()


def _old_slot_mapping(inp: W.RepackInputs):
    """Slots of the live tokens in the layout before the pass: slot = block * S + offset of
    the logical position in the request's table (Sec. 3.4), live tokens in order."""
    S = inp.shape.block_size
    indptr, slots = [0], []
    for r in range(inp.num_reqs):
        a = int(inp.tok_indptr[r])
        bt = inp.block_ids[inp.bt_indptr[r]:inp.bt_indptr[r + 1]].astype(np.int64)
        pos = np.nonzero(inp.live[a:a + int(inp.seq_lens[r])])[0]
        slots.extend((bt[pos // S] * S + pos % S).tolist())
        indptr.append(len(slots))
    return np.asarray(indptr, np.int64), np.asarray(slots, np.int64)


def _dev_i32(x):
    t = torch()
    return t.from_numpy(np.ascontiguousarray(x, dtype=np.int32)).cuda()


def _device_pass(inp, kv, inplace=False, stream=None):
    """One repack pass and the slot-mapping refresh, enqueued on `stream`."""
    B = _B()
    sh = inp.shape
    cache = B.KVCache(kv, sh.num_layers, sh.num_kv_heads, sh.head_dim, sh.block_size)
    batch = B.Batch.from_inputs(inp)
    plan = B.Plan.allocate(batch, sh.block_size, inplace=inplace)
    B.run_pass(cache, batch, plan, stream=stream, inplace=inplace)
    indptr, slots = B.build_slot_mapping(batch, plan, stream=stream)
    return cache, batch, plan, indptr, slots


def _label(msg):
    print(f"[gpu] {msg}", flush=True)


# ------------------------------------------------------------------------------------------
# slot mapping
# ------------------------------------------------------------------------------------------
def _edge_inputs():
    sh = W.KVShape(1, 2, 64, 16, "fp16")
    rng = np.random.default_rng(7)
    masks = [[], [0] * 40, [1] * 17, [1, 0] * 600, [0] * 15 + [1],
             (rng.random(3000) < 0.4).astype(int).tolist(), [1]]
    return W.from_masks(masks, sh, free_blocks=400, seed=7, name="edge")


def _many_requests():
    sh = W.KVShape(1, 1, 64, 4, "fp16")
    rng = np.random.default_rng(8)
    masks = [(rng.random(int(n)) < 0.5).astype(int).tolist()
             for n in rng.integers(0, 40, size=1300)]
    return W.from_masks(masks, sh, free_blocks=4000, seed=8, name="many_requests")


SLOT_CASES = {
    "tiny": lambda: W.tiny_cache(101),
    "edge": _edge_inputs,
    "many_requests": _many_requests,
    "llama3_8b_random": lambda: W.llama3_8b_random(221, num_layers=1, num_reqs=16),
    "llama3_70b_fp8": lambda: W.llama3_70b_h2o(521, num_layers=1, num_reqs=4,
                                               len_range=(2000, 9000)),
    # requests of two to three 8192-token compaction tiles with ragged tails
    "long_requests": lambda: W.llama3_70b_h2o(522, num_layers=1, num_reqs=3,
                                              len_range=(17000, 23000)),
}


@pytest.mark.parametrize("inplace", [False, True], ids=["out_of_place", "in_place"])
@pytest.mark.parametrize("case", sorted(SLOT_CASES))
def test_slot_mapping_parity(case, inplace):
    t = torch()
    inp = SLOT_CASES[case]()
    _label(f"slot mapping {case} inplace={inplace}: R={inp.num_reqs} T={inp.num_tokens}")
    kv = W.kv_device(inp.shape, inp.num_blocks, 3)
    orc = oracle_repack_inputs(inp, None, inplace=inplace)
    _, _, plan, indptr, slots = _device_pass(inp, kv, inplace=inplace)
    t.cuda.synchronize()
    assert int(plan.counters[3]) == 0
    ref_indptr, ref_slots = slot_mapping(orc.token_slot, inp.tok_indptr, inp.seq_lens)
    got_indptr = indptr.cpu().numpy().astype(np.int64)
    assert np.array_equal(got_indptr, ref_indptr)
    got = slots.cpu().numpy()[:int(ref_indptr[-1])].astype(np.int64)
    assert np.array_equal(got, ref_slots)


# ------------------------------------------------------------------------------------------
# paged decode parity
# ------------------------------------------------------------------------------------------
def _decode_inputs(dtype, H, D, S, seed):
    """Two layers; live counts 0, 1, 255, 256, 257, 514, 1023, 1024, 1025, 2049 (split edges
    of every geometry: splits hold 32768 / (D * element bytes) tokens, 64 to 1024) and
    Bernoulli(0.5) requests up to 3000 tokens (several splits with ragged tails)."""
    sh = W.KVShape(2, H, D, S, dtype)
    rng = np.random.default_rng(seed)
    masks = [[0] * 50, [0] * 9 + [1], [1] * 255, [1] * 256 + [0] * 7, [1] * 257,
             [1, 1, 0] * 257, [1] * 1023, [0] * 3 + [1] * 1024, [1] * 1025, [1] * 2049]
    masks += [(rng.random(int(n)) < 0.5).astype(int).tolist()
              for n in rng.integers(1, 3000, size=6)]
    M = sum(-(-len(m) // S) for m in masks)
    return W.from_masks(masks, sh, free_blocks=M + 64, seed=seed, name=f"decode_{dtype}")


DECODE_CASES = [
    # dtype, H, D, G, S   (lanes per head row = D / 8; tokens per split = 32768 / (D * bytes))
    ("bf16", 8, 128, 4, 16),   # Llama-3-8B KV geometry
    ("fp16", 2, 64, 1, 16),    # no GQA
    ("bf16", 4, 32, 2, 16),    # 512-token splits (1024 for fp8)
    ("fp16", 4, 128, 8, 16),   # G = 8
    ("bf16", 2, 256, 2, 16),   # 32 lanes per head row, 64-token splits
    ("fp8_e4m3", 8, 128, 8, 32),  # Llama-3-70B fp8 geometry
    ("fp8_e4m3", 2, 64, 2, 16),
    ("fp8_e4m3", 2, 256, 4, 16),
    ("fp8_e4m3", 4, 32, 1, 16),
    ("bf16", 2, 64, 8, 16),    # G = 8 at the other head sizes
    ("bf16", 1, 256, 8, 16),
    ("fp8_e4m3", 2, 32, 8, 16),
]


@pytest.mark.parametrize("dtype,H,D,G,S", DECODE_CASES,
                         ids=[f"{c[0]}_H{c[1]}_D{c[2]}_G{c[3]}" for c in DECODE_CASES])
def test_paged_decode_parity(dtype, H, D, G, S):
    t = torch()
    B = _B()
    inp = _decode_inputs(dtype, H, D, S, seed=31 + D + G)
    sh = inp.shape
    _label(f"paged decode {dtype} H={H} D={D} G={G} S={S}: R={inp.num_reqs}")
    kv = W.kv_device(sh, inp.num_blocks, 5)
    orc = oracle_repack_inputs(inp, kv_bytes(kv, sh))
    cache, _, _, indptr, slots = _device_pass(inp, kv)
    ref_indptr, ref_slots = slot_mapping(orc.token_slot, inp.tok_indptr, inp.seq_lens)
    vals = _values(orc.kv, sh)
    rng = np.random.default_rng(D * G)
    max_tokens = int(np.diff(ref_indptr).max())
    worst = 0.0
    for layer in (0, 1):
        q = rng.standard_normal((inp.num_reqs, H * G, D)).astype(np.float32)
        out = B.paged_decode(cache, t.from_numpy(q).cuda(), indptr, slots, layer, max_tokens)
        got = out.cpu().numpy().astype(np.float64)
        ref = decode_batch(q, vals[2 * layer], vals[2 * layer + 1], ref_indptr, ref_slots)
        np.testing.assert_allclose(got, ref, atol=ATOL, rtol=RTOL)
        assert np.array_equal(got[0], np.zeros_like(got[0])), "no live tokens -> zeros"
        worst = max(worst, float(np.abs(got - ref).max()))
    _label(f"paged decode {dtype} H={H} D={D} G={G}: max |diff| {worst:.2e}")


@pytest.mark.parametrize("seed", range(24))
def test_paged_decode_random_geometries(seed):
    """Seeded random decode geometries: KV heads 1-8, head_dim 32-256, GQA groups 1-8, all
    three dtypes, block sizes 1-64, 1-12 requests of random lengths and densities (splits of
    every geometry with ragged tails), a softmax scale within 2x of 1/sqrt(head_dim)."""
    t = torch()
    B = _B()
    rng = np.random.default_rng(5000 + seed)
    dtype = ["fp16", "bf16", "fp8_e4m3"][int(rng.integers(3))]
    H = int(rng.integers(1, 9))
    D = int(rng.choice([32, 64, 128, 256]))
    G = int(rng.choice([1, 2, 4, 8]))
    S = int(rng.choice([1, 4, 16, 32, 64]))
    R = int(rng.integers(1, 13))
    masks = [(rng.random(int(rng.integers(0, 2600))) < rng.random()).astype(int).tolist()
             for _ in range(R)]
    M = sum(-(-len(m) // S) for m in masks)
    inp = W.from_masks(masks, W.KVShape(2, H, D, S, dtype), free_blocks=M + 16, seed=seed,
                       name=f"decode_fuzz{seed}")
    sh = inp.shape
    _label(f"decode fuzz {seed}: {dtype} H={H} D={D} G={G} S={S} R={R}")
    kv = W.kv_device(sh, inp.num_blocks, seed)
    orc = oracle_repack_inputs(inp, kv_bytes(kv, sh))
    cache, _, _, indptr, slots = _device_pass(inp, kv)
    ref_indptr, ref_slots = slot_mapping(orc.token_slot, inp.tok_indptr, inp.seq_lens)
    vals = _values(orc.kv, sh)
    scale = float(rng.uniform(0.5, 2.0)) / np.sqrt(D)     # around the usual 1/sqrt(D)
    max_tokens = max(int(np.diff(ref_indptr).max()), 1)
    q = rng.standard_normal((R, H * G, D)).astype(np.float32)
    out = B.paged_decode(cache, t.from_numpy(q).cuda(), indptr, slots, 1, max_tokens,
                         scale=scale)
    got = out.cpu().numpy().astype(np.float64)
    ref = decode_batch(q, vals[2], vals[3], ref_indptr, ref_slots, scale=scale)
    np.testing.assert_allclose(got, ref, atol=ATOL, rtol=RTOL)


@pytest.mark.parametrize("dtype,G", [("bf16", 4), ("fp8_e4m3", 8), ("fp16", 1)])
def test_paged_decode_slot_outside_pool_gives_nan(dtype, G):
    """A slot outside the pool (past the end, or negative) is read nowhere: the requests that
    hold one get NaN rows, every other request is unaffected."""
    t = torch()
    B = _B()
    H, D, S = 2, 128, 16
    inp = _decode_inputs(dtype, H, D, S, seed=91 + G)
    sh = inp.shape
    kv = W.kv_device(sh, inp.num_blocks, 7)
    orc = oracle_repack_inputs(inp, kv_bytes(kv, sh))
    cache, _, _, indptr, slots = _device_pass(inp, kv)
    ref_indptr, ref_slots = slot_mapping(orc.token_slot, inp.tok_indptr, inp.seq_lens)
    counts = np.diff(ref_indptr)
    bad = [int(np.nonzero(counts == 1)[0][0]), int(np.nonzero(counts > 600)[0][0])]
    host = slots.cpu().numpy()
    host[ref_indptr[bad[0]]] = inp.num_blocks * S + 3           # past the pool
    host[ref_indptr[bad[1]] + counts[bad[1]] // 2] = -7         # negative, mid-request
    bad_slots = t.from_numpy(host).cuda()
    vals = _values(orc.kv, sh)
    q = np.random.default_rng(4).standard_normal((inp.num_reqs, H * G, D)).astype(np.float32)
    out = B.paged_decode(cache, t.from_numpy(q).cuda(), indptr, bad_slots, 0,
                         int(counts.max()))
    got = out.cpu().numpy().astype(np.float64)
    ref = decode_batch(q, vals[0], vals[1], ref_indptr, ref_slots)
    good = np.ones(inp.num_reqs, bool)
    good[bad] = False
    np.testing.assert_allclose(got[good], ref[good], atol=ATOL, rtol=RTOL)
    assert np.isnan(got[bad]).all()


@pytest.mark.parametrize("dtype,G", [("bf16", 4), ("fp8_e4m3", 8)])
def test_paged_decode_malformed_slot_indptr_gives_nan(dtype, G):
    """A request whose slot range is malformed - slot_indptr[r] < 0, which also makes the
    previous request's count negative - reads no slot and gets NaN rows, also when the
    workspace still holds a previous call's partials for it; the other requests are exact."""
    t = torch()
    B = _B()
    H, D, S = 2, 128, 16
    inp = _decode_inputs(dtype, H, D, S, seed=71 + G)
    sh = inp.shape
    kv = W.kv_device(sh, inp.num_blocks, 9)
    orc = oracle_repack_inputs(inp, kv_bytes(kv, sh))
    cache, _, _, indptr, slots = _device_pass(inp, kv)
    ref_indptr, ref_slots = slot_mapping(orc.token_slot, inp.tok_indptr, inp.seq_lens)
    counts = np.diff(ref_indptr)
    max_tokens = int(counts.max())
    q = np.random.default_rng(6).standard_normal((inp.num_reqs, H * G, D)).astype(np.float32)
    qd = t.from_numpy(q).cuda()
    ws = t.empty(B.decode_workspace_bytes(inp.num_reqs, H * G, D, max_tokens) // 4,
                 dtype=t.float32, device="cuda")
    B.paged_decode(cache, qd, indptr, slots, 0, max_tokens, workspace=ws)   # fills ws
    r = int(np.nonzero(counts[1:] > 600)[0][0]) + 1        # a multi-split request, r >= 1
    bad_indptr = indptr.clone()
    bad_indptr[r] = -5
    _label(f"decode malformed slot_indptr {dtype} G={G}: request {r} (and {r - 1})")
    out = B.paged_decode(cache, qd, bad_indptr, slots, 0, max_tokens, workspace=ws)
    got = out.cpu().numpy().astype(np.float64)
    vals = _values(orc.kv, sh)
    ref = decode_batch(q, vals[0], vals[1], ref_indptr, ref_slots)
    good = np.ones(inp.num_reqs, bool)
    good[[r - 1, r]] = False
    np.testing.assert_allclose(got[good], ref[good], atol=ATOL, rtol=RTOL)
    assert np.isnan(got[~good]).all()


@pytest.mark.parametrize("dtype,G", [("bf16", 4), ("fp8_e4m3", 8)])
def test_paged_decode_max_tokens_too_small(dtype, G):
    """max_tokens below a request's slot count: requests whose slots fit the splits it implies
    are exact, the others get NaN rows (never a silently truncated softmax)."""
    t = torch()
    B = _B()
    H, D, S = 2, 128, 16
    inp = _decode_inputs(dtype, H, D, S, seed=77 + G)
    sh = inp.shape
    kv = W.kv_device(sh, inp.num_blocks, 6)
    orc = oracle_repack_inputs(inp, kv_bytes(kv, sh))
    cache, _, _, indptr, slots = _device_pass(inp, kv)
    ref_indptr, ref_slots = slot_mapping(orc.token_slot, inp.tok_indptr, inp.seq_lens)
    vals = _values(orc.kv, sh)
    split = 32768 // (D * (1 if dtype == "fp8_e4m3" else 2))
    max_tokens = split + 1                       # two splits
    counts = np.diff(ref_indptr)
    fits = counts <= 2 * split
    assert fits.any() and (~fits).any()
    q = np.random.default_rng(3).standard_normal((inp.num_reqs, H * G, D)).astype(np.float32)
    out = B.paged_decode(cache, t.from_numpy(q).cuda(), indptr, slots, 1, max_tokens)
    got = out.cpu().numpy().astype(np.float64)
    ref = decode_batch(q, vals[2], vals[3], ref_indptr, ref_slots)
    np.testing.assert_allclose(got[fits], ref[fits], atol=ATOL, rtol=RTOL)
    assert np.isnan(got[~fits]).all()


@pytest.mark.parametrize("dtype,G,D", [("bf16", 1, 128), ("fp16", 2, 128), ("bf16", 4, 128),
                                     ("fp16", 4, 64), ("bf16", 2, 256), ("fp16", 1, 32)])
def test_paged_decode_long_batch_eight_wave_splits(dtype, G, D):
    """A batch whose longest request spans 64 or more 4-wave splits takes 8-wave split
    workgroups for 16-bit caches at G < 8 (twice the tokens per split): requests of ~18K live
    tokens (~36K at head_dim 32, whose 4-wave split is 512 tokens) and a short one, against
    the float64 oracle."""
    t = torch()
    B = _B()
    H, S = 2, 16
    rng = np.random.default_rng(1700 + 10 * G + D)
    scale = 2 if D == 32 else 1
    masks = [(rng.random(scale * n) < 0.9).astype(np.uint8) for n in (20_000, 19_000, 17_500)]
    masks.append((rng.random(300) < 0.5).astype(np.uint8))
    M = sum(-(-len(m) // S) for m in masks)
    inp = W.from_masks(masks, W.KVShape(1, H, D, S, dtype), free_blocks=M + 16, seed=G,
                       name="decode_long_batch")
    sh = inp.shape
    _label(f"decode 8-wave splits {dtype} G={G} D={D}: {int(inp.live.sum())} live tokens")
    kv = W.kv_device(sh, inp.num_blocks, 12)
    orc = oracle_repack_inputs(inp, kv_bytes(kv, sh))
    cache, _, _, indptr, slots = _device_pass(inp, kv)
    ref_indptr, ref_slots = slot_mapping(orc.token_slot, inp.tok_indptr, inp.seq_lens)
    counts = np.diff(ref_indptr)
    assert counts.max() >= 64 * (32768 // (D * 2))
    vals = _values(orc.kv, sh)
    q = rng.standard_normal((inp.num_reqs, H * G, D)).astype(np.float32)
    out = B.paged_decode(cache, t.from_numpy(q).cuda(), indptr, slots, 0, int(counts.max()))
    got = out.cpu().numpy().astype(np.float64)
    ref = decode_batch(q, vals[0], vals[1], ref_indptr, ref_slots)
    np.testing.assert_allclose(got, ref, atol=ATOL, rtol=RTOL)
    del kv, vals
    t.cuda.empty_cache()


@pytest.mark.parametrize("dtype,G", [("bf16", 4), ("fp16", 1), ("fp8_e4m3", 4)])
def test_paged_decode_split_size_by_bound(dtype, G):
    """The host picks the split size from max_tokens alone (16-bit caches at G < 8: 8-wave
    splits from 64 four-wave splits, 8,192 tokens at head_dim 128). One batch whose longest
    request holds 8,191 live tokens, decoded with the tight bound (4-wave splits), with 8,192
    and 20,000 (8-wave splits for 16-bit caches, most split slots empty), with 15,872 and
    16,384 (62 and 64 splits of 256 tokens: the grid's split count rounded up to 63 below 64,
    kept at 64) and with 65,536: every output within the bar of the float64 oracle, and the
    calls agree to float32 rounding."""
    t = torch()
    B = _B()
    H, D, S = 2, 128, 16
    rng = np.random.default_rng(1800 + G)
    masks = [np.ones(8191, np.uint8), (rng.random(9000) < 0.6).astype(np.uint8),
             (rng.random(700) < 0.5).astype(np.uint8), np.ones(1, np.uint8)]
    M = sum(-(-len(m) // S) for m in masks)
    inp = W.from_masks(masks, W.KVShape(1, H, D, S, dtype), free_blocks=M + 16, seed=G,
                       name="decode_bound")
    sh = inp.shape
    _label(f"decode split size by bound {dtype} G={G}")
    kv = W.kv_device(sh, inp.num_blocks, 13)
    orc = oracle_repack_inputs(inp, kv_bytes(kv, sh))
    cache, _, _, indptr, slots = _device_pass(inp, kv)
    ref_indptr, ref_slots = slot_mapping(orc.token_slot, inp.tok_indptr, inp.seq_lens)
    counts = np.diff(ref_indptr)
    assert counts.max() == 8191
    vals = _values(orc.kv, sh)
    q = rng.standard_normal((inp.num_reqs, H * G, D)).astype(np.float32)
    ref = decode_batch(q, vals[0], vals[1], ref_indptr, ref_slots)
    qd = t.from_numpy(q).cuda()
    outs = []
    for bound in (8191, 8192, 20_000, 15_872, 16_384, 65_536):
        got = B.paged_decode(cache, qd, indptr, slots, 0, bound).cpu().numpy().astype(np.float64)
        np.testing.assert_allclose(got, ref, atol=ATOL, rtol=RTOL, err_msg=f"bound {bound}")
        outs.append(got)
    for got in outs[1:]:
        np.testing.assert_allclose(got, outs[0], atol=1e-5, rtol=1e-5)
    del kv, vals
    t.cuda.empty_cache()


@pytest.mark.parametrize("dtype,G,S", [("bf16", 4, 16), ("fp8_e4m3", 8, 32)])
def test_paged_decode_long_request(dtype, G, S):
    """One request of ~1M live tokens among short ones (a 1.5M-token context, keep 0.7):
    4,100 splits per head (8-wave splits for bf16, 1-byte elements for fp8) merged by the
    combine kernel, after a repack pass, against the float64 oracle."""
    t = torch()
    B = _B()
    H, D = 1, 128
    rng = np.random.default_rng(1500 + G)
    masks = [(rng.random(1_500_000) < 0.7).astype(np.uint8), [1] * 5, [0] * 10,
             (rng.random(3000) < 0.5).astype(np.uint8)]
    M = sum(-(-len(m) // S) for m in masks)
    inp = W.from_masks(masks, W.KVShape(1, H, D, S, dtype), free_blocks=M + 16, seed=G,
                       name="decode_long")
    sh = inp.shape
    _label(f"decode long request {dtype} G={G}: {int(inp.live.sum())} live tokens")
    kv = W.kv_device(sh, inp.num_blocks, 11)
    orc = oracle_repack_inputs(inp, kv_bytes(kv, sh))
    cache, _, _, indptr, slots = _device_pass(inp, kv)
    ref_indptr, ref_slots = slot_mapping(orc.token_slot, inp.tok_indptr, inp.seq_lens)
    counts = np.diff(ref_indptr)
    assert counts[0] > 1_000_000
    vals = _values(orc.kv, sh)
    q = rng.standard_normal((inp.num_reqs, H * G, D)).astype(np.float32)
    out = B.paged_decode(cache, t.from_numpy(q).cuda(), indptr, slots, 0, int(counts.max()))
    got = out.cpu().numpy().astype(np.float64)
    ref = decode_batch(q, vals[0], vals[1], ref_indptr, ref_slots)
    np.testing.assert_allclose(got, ref, atol=ATOL, rtol=RTOL)
    assert np.array_equal(got[2], np.zeros_like(got[2])), "no live tokens -> zeros"
    del kv, vals
    t.cuda.empty_cache()


@pytest.mark.parametrize("dtype", ["fp8_e4m3", "fp16", "bf16"])
def test_decode_one_key_returns_value_codes_exactly(dtype):
    """Requests of one live token with a zero key: softmax weight exactly 1, so the output is
    the value row converted to float32; the value rows hold every finite code of the type
    (non-finite values are outside the kernel's contract)."""
    t = torch()
    B = _B()
    e = 1 if dtype == "fp8_e4m3" else 2
    H, D = (1, 64) if e == 1 else (8, 128)
    per_row = H * D
    codes = np.arange(256 if e == 1 else 65536, dtype=np.uint8 if e == 1 else np.uint16)
    R = len(codes) // per_row
    sh = W.KVShape(1, H, D, 16, dtype)
    num_blocks = R
    raw = np.zeros((2, num_blocks * 16, per_row), dtype=codes.dtype)
    for r in range(R):
        raw[1, r * 16, :] = codes[r * per_row:(r + 1) * per_row]   # V row of slot r*16
    kv = t.from_numpy(raw.view(np.uint8)).cuda().view(W.torch_dtype(sh)).reshape(
        2, num_blocks, 16, H, D).contiguous()
    cache = B.KVCache(kv, 1, H, D, 16)
    indptr = _dev_i32(np.arange(R + 1))
    slots = _dev_i32(np.arange(R) * 16)
    q = t.randn(R, H, D, device="cuda")
    _label(f"one-key decode {dtype}: {len(codes)} codes in {R} requests")
    got = B.paged_decode(cache, q, indptr, slots, 0, 1).cpu().numpy().reshape(R, per_row)
    expect = t.from_numpy(codes.view(np.uint8 if e == 1 else np.int16).copy()).view(
        W.torch_dtype(sh)).float().numpy().reshape(R, per_row)
    # -0.0 comes out as +0.0 (0 + -0 = +0 in the accumulation); == treats them as equal
    finite = np.isfinite(expect)
    same = (got == expect) | ~finite
    assert finite.sum() > 0.9 * finite.size
    bad = np.nonzero(~same.reshape(-1))[0]
    assert len(bad) == 0, (f"{len(bad)} codes differ, first {codes[bad[:5]]}: "
                           f"got {got.reshape(-1)[bad[:5]]} expect {expect.reshape(-1)[bad[:5]]}")


def test_decode_fp8_key_codes():
    """Every e4m3 key code reaches the score exactly: requests of two tokens, token 0 with key
    x * e_0 (x = the code's value), token 1 with a zero key; value rows e_0 and 0; query e_0 at
    scale 1/64. Then out[0] = sigmoid(x / 64), checked against torch's CPU conversion of the
    code (NaN codes excluded)."""
    t = torch()
    B = _B()
    H, D, S = 1, 64, 16
    codes = np.arange(256, dtype=np.uint8)
    codes = codes[(codes & 0x7F) != 0x7F]            # the two NaN codes
    R = len(codes)
    sh = W.KVShape(1, H, D, S, "fp8_e4m3")
    raw = np.zeros((2, R * S, H * D), dtype=np.uint8)
    one = np.frombuffer(t.tensor([1.0]).to(t.float8_e4m3fn).view(t.uint8).numpy().tobytes(),
                        np.uint8)[0]
    for r, code in enumerate(codes):
        raw[0, r * S, 0] = code                        # K of token 0: x at dimension 0
        raw[1, r * S, 0] = one                         # V of token 0: e_0
    kv = t.from_numpy(raw).cuda().view(t.float8_e4m3fn).reshape(2, R, S, H, D).contiguous()
    cache = B.KVCache(kv, 1, H, D, S)
    indptr = _dev_i32(np.arange(R + 1) * 2)
    slots = _dev_i32(np.stack([np.arange(R) * S, np.arange(R) * S + 1], 1).reshape(-1))
    q = t.zeros(R, H, D, device="cuda")
    q[:, :, 0] = 1.0
    _label(f"fp8 key codes: {R} codes")
    got = B.paged_decode(cache, q, indptr, slots, 0, 2, scale=1.0 / 64).cpu().numpy()[:, 0, 0]
    x = t.from_numpy(codes.copy()).view(t.float8_e4m3fn).float().numpy().astype(np.float64)
    expect = 1.0 / (1.0 + np.exp(-x / 64))
    # the weights reach the value product as two 16-bit parts (~2^-17 relative); neighbouring
    # codes differ by >= 1/16 relative, i.e. by >= 1e-4 in the sigmoid of x / 64
    np.testing.assert_allclose(got, expect, rtol=1e-5, atol=1e-7)


# ------------------------------------------------------------------------------------------
# before / after the repack, stream-event ordering, graph replay
# ------------------------------------------------------------------------------------------
def _layout_inputs(seed=41):
    return W.llama3_8b_random(seed, num_layers=4, num_reqs=12, len_range=(600, 3000))


def _scribble_freed(kv, plan, sh):
    """Overwrite every released block in every plane (what a reuse of the block does)."""
    t = torch()
    n = int(plan.counters[2])
    freed = plan.freed[:n].long()
    if n:
        kv.view(sh.num_planes, -1, sh.block_size * sh.num_kv_heads * sh.head_dim)[:, freed] = \
            float("nan")
    return n


@pytest.mark.parametrize("inplace", [False, True], ids=["out_of_place", "in_place"])
def test_decode_bit_identical_across_repack_on_relocation_stream(inplace):
    """The schedule of Sec. 3.3.4: decode on the main stream through the old slots; the
    repack pass and the slot-mapping refresh on a relocation stream (waiting for the main
    stream's decode first, which the in-place mode needs since it overwrites what that decode
    reads); an event recorded on the relocation stream and waited for by the main stream
    before the next decode (I3). Both decodes agree bit for bit, also after the released
    blocks are overwritten."""
    t = torch()
    B = _B()
    inp = _layout_inputs()
    sh = inp.shape
    _label(f"relocation stream inplace={inplace}: R={inp.num_reqs} T={inp.num_tokens}")
    kv = W.kv_device(sh, inp.num_blocks, 9)
    cache = B.KVCache(kv, sh.num_layers, sh.num_kv_heads, sh.head_dim, sh.block_size)
    old_indptr, old_slots = _old_slot_mapping(inp)
    max_tokens = int(np.diff(old_indptr).max())
    q = t.randn(inp.num_reqs, 4 * sh.num_kv_heads, sh.head_dim, device="cuda")
    main = t.cuda.current_stream()
    before = [B.paged_decode(cache, q, _dev_i32(old_indptr), _dev_i32(old_slots), layer,
                             max_tokens) for layer in range(sh.num_layers)]
    reloc = t.cuda.Stream()
    reloc.wait_stream(main)
    with t.cuda.stream(reloc):
        batch = B.Batch.from_inputs(inp)
        plan = B.Plan.allocate(batch, sh.block_size, inplace=inplace)
        B.run_pass(cache, batch, plan, inplace=inplace)
        indptr, slots = B.build_slot_mapping(batch, plan)
        done = t.cuda.Event()
        done.record(reloc)
    main.wait_event(done)
    after = [B.paged_decode(cache, q, indptr, slots, layer, max_tokens)
             for layer in range(sh.num_layers)]
    for a, b in zip(before, after):
        assert t.equal(a, b), "decode changed across the repack"
    assert int(plan.counters[1]) > 0, "the pass repacked nothing"
    n = _scribble_freed(kv, plan, sh)
    again = [B.paged_decode(cache, q, indptr, slots, layer, max_tokens)
             for layer in range(sh.num_layers)]
    for a, b in zip(before, again):
        assert t.equal(a, b), "decode read a released block"
    t.cuda.synchronize()
    _label(f"relocation stream inplace={inplace}: {int(plan.counters[1])} requests repacked, "
           f"{n} blocks released and overwritten")


def test_graph_replay_with_mutable_slot_buffer():
    """Decode captured once in a HIP graph over fixed slot / query / output buffers. The
    repack and the refresh of the slot buffer run outside the graph on a relocation stream;
    the main stream waits for its event before the replay. Every replay equals the eager
    decode of the same state, with unrelated eager work between replays."""
    t = torch()
    B = _B()
    inp = _layout_inputs(43)
    sh = inp.shape
    layer = 2
    _label(f"graph replay: R={inp.num_reqs} T={inp.num_tokens}")
    kv = W.kv_device(sh, inp.num_blocks, 11)
    cache = B.KVCache(kv, sh.num_layers, sh.num_kv_heads, sh.head_dim, sh.block_size)
    old_indptr, old_slots = _old_slot_mapping(inp)
    max_tokens = int(np.diff(old_indptr).max())
    R, Hq, D = inp.num_reqs, 2 * sh.num_kv_heads, sh.head_dim
    slot_indptr = _dev_i32(old_indptr)
    slots = t.zeros(max(inp.num_tokens, 1), dtype=t.int32, device="cuda")
    slots[:len(old_slots)] = _dev_i32(old_slots)
    q = t.randn(R, Hq, D, device="cuda")
    out = t.empty_like(q)
    ws = t.empty(B.decode_workspace_bytes(R, Hq, D, max_tokens) // 4, dtype=t.float32,
                 device="cuda")

    def decode(o):
        return B.paged_decode(cache, q, slot_indptr, slots, layer, max_tokens, out=o,
                              workspace=ws)

    side = t.cuda.Stream()
    side.wait_stream(t.cuda.current_stream())
    with t.cuda.stream(side):
        decode(out)
    t.cuda.current_stream().wait_stream(side)
    graph = t.cuda.CUDAGraph()
    with t.cuda.graph(graph):
        decode(out)

    def replay_and_check(tag):
        eager = decode(t.empty_like(q))
        t.cuda.synchronize()
        noise = t.randn(512, 512, device="cuda")
        noise = noise @ noise
        graph.replay()
        t.cuda.synchronize()
        assert t.equal(out, eager), f"replay differs from eager decode ({tag})"
        return out.clone()

    first = replay_and_check("old layout")
    first_again = replay_and_check("old layout, second replay")
    assert t.equal(first, first_again)

    main = t.cuda.current_stream()
    reloc = t.cuda.Stream()
    reloc.wait_stream(main)     # the slot buffer is read by the replay before
    with t.cuda.stream(reloc):
        batch = B.Batch.from_inputs(inp)
        plan = B.Plan.allocate(batch, sh.block_size)
        B.run_pass(cache, batch, plan)
        B.build_slot_mapping(batch, plan, slot_indptr=slot_indptr, slots=slots)
        done = t.cuda.Event()
        done.record(reloc)
    main.wait_event(done)
    graph.replay()
    t.cuda.synchronize()
    assert t.equal(out, first), "replay after the repack differs"
    assert int(plan.counters[1]) > 0
    assert not np.array_equal(slots.cpu().numpy()[:len(old_slots)], old_slots)
    _scribble_freed(kv, plan, sh)
    replayed = replay_and_check("released blocks overwritten")
    assert t.equal(replayed, first)
    # a new query in the captured input buffer
    q.copy_(t.randn(R, Hq, D, device="cuda"))
    replay_and_check("new query")


def test_slot_table_append_and_decode():
    """The append-only translation cache (Sec. 3.2): rebuilt after a pass with room for 8
    more slots per request, then grown by appends (one request past its room, which must be
    reported and left unchanged); the table equals the oracle's after each step, and decode
    through it equals decode through a packed mapping of the same slot lists, bit for bit."""
    t = torch()
    B = _B()
    inp = _layout_inputs(47)
    sh = inp.shape
    S = sh.block_size
    R = inp.num_reqs
    _label(f"slot table: R={R} T={inp.num_tokens}")
    kv = W.kv_device(sh, inp.num_blocks, 13)
    orc = oracle_repack_inputs(inp, None)
    cache, batch, plan, _, _ = _device_pass(inp, kv)
    start, count, slots = B.build_slot_table(batch, plan, reserve=8)
    t.cuda.synchronize()
    o_start, o_count, o_slots = slot_table(orc.token_slot, inp.tok_indptr, inp.seq_lens, 8)
    assert np.array_equal(start.cpu().numpy().astype(np.int64), o_start)
    assert np.array_equal(count.cpu().numpy()[:R].astype(np.int64), o_count)
    got = slots.cpu().numpy().astype(np.int64)
    for r in range(R):
        a = int(o_start[r])
        assert np.array_equal(got[a:a + o_count[r]], o_slots[a:a + o_count[r]])
    # appends: new tokens in the free blocks the pass did not consume (any valid slots)
    rng = np.random.default_rng(3)
    spare = inp.free_list[int(plan.counters[0]):].astype(np.int64)
    pool = (spare[:, None] * S + np.arange(S)).reshape(-1)
    ks = rng.integers(0, 6, size=R)
    ks[R // 2] = 9                                   # past its room of 8
    new, o = [], 0
    for k in ks:
        new.append(pool[o:o + k])
        o += k
    app_indptr = _dev_i32(np.concatenate([[0], np.cumsum(ks)]))
    app_slots = _dev_i32(np.concatenate(new) if o else np.zeros(1))
    status = B.append_slots(start, count, slots, app_indptr, app_slots)
    t.cuda.synchronize()
    o_count2, o_slots2, overflow = append_to_table(o_start, o_count, o_slots, new)
    assert overflow and int(status[0]) == B.STATUS_CODE["VTOKEN_ERR_CAPACITY"]
    assert np.array_equal(count.cpu().numpy()[:R].astype(np.int64), o_count2)
    got = slots.cpu().numpy().astype(np.int64)
    lists = []
    for r in range(R):
        a = int(o_start[r])
        assert np.array_equal(got[a:a + o_count2[r]], o_slots2[a:a + o_count2[r]])
        lists.append(o_slots2[a:a + o_count2[r]])
    # decode through the table vs through a packed mapping of the same lists
    indptr = np.concatenate([[0], np.cumsum([len(x) for x in lists])])
    packed = np.concatenate(lists)
    max_tokens = int(np.diff(indptr).max())
    q = t.randn(R, 4 * sh.num_kv_heads, sh.head_dim, device="cuda")
    for layer in range(sh.num_layers):
        a_out = B.paged_decode(cache, q, start, slots, layer, max_tokens, slot_count=count)
        b_out = B.paged_decode(cache, q, _dev_i32(indptr), _dev_i32(packed), layer, max_tokens)
        assert t.equal(a_out, b_out), f"layer {layer}: table and packed decode differ"
    del kv
    t.cuda.empty_cache()
