"""Shared helpers of the GPU tests: run one repack pass through the C ABI and compare every
output with the CPU oracle."""
from __future__ import annotations

import numpy as np

from oracle.planner import PlannerParams as OracleParams
from oracle.planner import plan_partial
from oracle.repack import oracle_repack_inputs
from paper_2608_13263_amd import workloads as W


def torch():
    import torch as t
    return t


def kv_bytes(kv, shape: W.KVShape):
    """uint8 host view [2L][num_blocks*S][row_bytes] of a device KV tensor."""
    t = torch()
    n = kv.shape[1] * shape.block_size
    return kv.view(t.uint8).reshape(shape.num_planes, n, shape.row_bytes).cpu().numpy()


def gpu_pass(inp: W.RepackInputs, kv, variant=0, grid=0, order=0, label="", inplace=False,
             fused=False):
    """build_token_table -> repack_ex -> free_blocks on the current stream (fused: the copy and
    the freed list in one launch, vtoken_repack_free); returns host copies of every plan
    output, trimmed to the sizes the counters report."""
    t = torch()
    from paper_2608_13263_amd import binding as B
    print(f"[gpu] {label or inp.name}: R={inp.num_reqs} T={inp.num_tokens} "
          f"M={inp.num_bt_entries} f={len(inp.free_list)} S={inp.shape.block_size} "
          f"row={inp.shape.row_bytes}B planes={inp.shape.num_planes} "
          f"variant={variant} grid={grid} order={order} inplace={inplace} fused={fused}",
          flush=True)
    cache = B.KVCache(kv, inp.shape.num_layers, inp.shape.num_kv_heads, inp.shape.head_dim,
                      inp.shape.block_size)
    batch = B.Batch.from_inputs(inp)
    plan = B.Plan.allocate(batch, inp.shape.block_size, inplace=inplace)
    if inplace:
        B.build_token_table_inplace(cache, batch, plan)
        B.repack_inplace_ex(cache, batch, plan, variant=variant)
    elif fused:
        assert (variant, grid, order) == (0, 0, 0), "the fused call uses the default copy"
        B.build_token_table(cache, batch, plan)
        B.repack_free(cache, batch, plan)
    else:
        B.build_token_table(cache, batch, plan)
        B.repack_ex(cache, batch, plan, variant=variant, grid=grid, order=order)
    if not fused:
        B.free_blocks(batch, plan)
    t.cuda.synchronize()
    return plan_to_host(plan, inp)


def plan_to_host(plan, inp):
    h = {k: getattr(plan, k).cpu().numpy() for k in plan.FIELDS + ("freed",)}
    used, n_adm, n_freed, status = (int(x) for x in h["counters"][:4])
    R, T = inp.num_reqs, inp.num_tokens
    S = inp.shape.block_size
    out = dict(status=status, used=used, n_admitted=n_adm, n_freed=n_freed)
    if status != 0:
        return out
    out.update(token_slot=h["token_slot"][:T], live_count=h["live_count"][:R],
               admitted=h["admitted"][:R], dst_indptr=h["dst_indptr"][:R + 1],
               new_bt_indptr=h["new_bt_indptr"][:R + 1],
               freed_indptr=h["freed_indptr"][:R + 1], src_plan=h["src_plan"][:used * S],
               freed=h["freed"][:n_freed])
    out["new_block_ids"] = h["new_block_ids"][:int(out["new_bt_indptr"][-1])] if R else \
        h["new_block_ids"][:0]
    return out


def assert_plan_equal(gpu: dict, orc) -> None:
    assert gpu["status"] == 0, f"device status {gpu['status']}"
    assert gpu["used"] == orc.used
    assert gpu["n_admitted"] == orc.n_admitted
    assert gpu["n_freed"] == orc.n_freed
    for key in ("token_slot", "live_count", "admitted", "dst_indptr", "new_bt_indptr",
                "new_block_ids", "src_plan", "freed_indptr", "freed"):
        g = np.asarray(gpu[key], dtype=np.int64)
        o = np.asarray(getattr(orc, key), dtype=np.int64)
        assert g.shape == o.shape, f"{key}: shape {g.shape} vs oracle {o.shape}"
        if not np.array_equal(g, o):
            bad = np.nonzero(g != o)[0]
            raise AssertionError(f"{key}: {len(bad)} mismatches, first at {bad[:5]}: "
                                 f"gpu {g[bad[:5]]} oracle {o[bad[:5]]}")


def assert_kv_equal(got: np.ndarray, expect: np.ndarray) -> None:
    if not np.array_equal(got, expect):
        diff = np.nonzero((got != expect).any(axis=2))
        raise AssertionError(f"KV bytes differ in {len(diff[0])} rows; first (plane, slot): "
                             f"{list(zip(diff[0][:5], diff[1][:5]))}")


def full_parity(inp: W.RepackInputs, seed: int = 0, variant=0, grid=0, order=0,
                inplace=False, fused=False):
    """Seeded KV on the device, one pass through the C ABI, every output and every KV byte
    against the oracle run on the pre-call bytes."""
    t = torch()
    kv = W.kv_device(inp.shape, inp.num_blocks, seed)
    before = kv_bytes(kv, inp.shape)
    orc = oracle_repack_inputs(inp, before, inplace=inplace)
    gpu = gpu_pass(inp, kv, variant=variant, grid=grid, order=order, inplace=inplace,
                   fused=fused)
    assert_plan_equal(gpu, orc)
    assert_kv_equal(kv_bytes(kv, inp.shape), orc.kv)
    del kv
    t.cuda.empty_cache()
    return gpu, orc


def oracle_moves(orc, inp, inplace=False):
    """(source slot, destination slot) of every row the oracle moves; the plan's destination
    block g is free_list[g] out of place, the request's own k-th block in place."""
    S = inp.shape.block_size
    sp = np.asarray(orc.src_plan, dtype=np.int64).reshape(orc.used, S)
    g, j = np.nonzero(sp >= 0)
    src = sp[g, j]
    if inplace:
        dest = np.empty(orc.used, dtype=np.int64)
        for r in np.nonzero(np.asarray(orc.admitted))[0]:
            a, b = int(orc.dst_indptr[r]), int(orc.dst_indptr[r + 1])
            n0 = int(orc.new_bt_indptr[r])
            dest[a:b] = orc.new_block_ids[n0:n0 + (b - a)]
    else:
        dest = np.asarray(inp.free_list, dtype=np.int64)
    dst = dest[g] * S + j
    keep = src != dst                       # rows already in place are not moves
    return src[keep], dst[keep]


def gpu_partial(inp, kv, params=None, label=""):
    """plan_partial -> repack on the current stream; host copies of every output, trimmed
    to the sizes the counters report."""
    t = torch()
    from paper_2608_13263_amd import binding as B
    sh = inp.shape
    params = params or B.PlannerParams()
    print(f"[gpu] partial {label or inp.name}: R={inp.num_reqs} T={inp.num_tokens} "
          f"M={inp.num_bt_entries} f={len(inp.free_list)} S={sh.block_size} theta={params.theta} "
          f"B={params.max_sources} wm={params.free_watermark}", flush=True)
    cache = B.KVCache(kv, sh.num_layers, sh.num_kv_heads, sh.head_dim, sh.block_size)
    batch = B.Batch.from_inputs(inp)
    slot_in = t.from_numpy(np.ascontiguousarray(inp.slots(), dtype=np.int32)).cuda()
    plan = B.Plan.allocate(batch, sh.block_size)
    state = B.PlannerState.allocate(inp.num_blocks, batch, pinned=inp.pinned)
    B.plan_partial(cache, batch, slot_in, plan, state, params)
    B.repack(cache, batch, plan)
    t.cuda.synchronize()
    return partial_to_host(plan, state, inp)


def partial_to_host(plan, state, inp):
    """Host copies of the partial pass's outputs, trimmed to the sizes the counters report."""
    sh = inp.shape
    h = {k: getattr(plan, k).cpu().numpy() for k in plan.FIELDS}
    for k in state.FIELDS:
        h[k] = getattr(state, k).cpu().numpy()
    R, T = inp.num_reqs, inp.num_tokens
    used, n_adm, n_freed, status = (int(x) for x in h["counters"][:4])
    out = dict(status=status, used=used, n_admitted=n_adm, n_freed=n_freed)
    if status != 0:
        return out
    out.update(token_slot=h["token_slot"][:T], live_count=h["live_count"][:R],
               admitted=h["admitted"][:R], src_count=h["src_count"][:R],
               dst_indptr=h["dst_indptr"][:R + 1], new_bt_indptr=h["new_bt_indptr"][:R + 1],
               freed_indptr=h["freed_indptr"][:R + 1], src_plan=h["src_plan"][:used * sh.block_size],
               freed=h["sources"][:n_freed], stats=h["stats"][:8], n_b=h["n_b"],
               refs=h["refs"])
    out["new_block_ids"] = h["new_block_ids"][:int(out["new_bt_indptr"][-1])] if R else \
        h["new_block_ids"][:0]
    return out


def oracle_params(p):
    return OracleParams(theta_num=p.theta[0], theta_den=p.theta[1],
                        max_live_per_source=None if p.max_live_per_source < 0
                        else p.max_live_per_source,
                        max_sources=p.max_sources, min_eligible=p.min_eligible,
                        free_watermark=p.free_watermark)


def run_partial_oracle(inp, kv_host, params):
    return plan_partial(inp.seq_lens, inp.tok_indptr, inp.bt_indptr, inp.block_ids, inp.live,
                        inp.slots(), inp.free_list, inp.shape.block_size, inp.num_blocks,
                        oracle_params(params), pinned=inp.pinned, kv=kv_host)


def assert_partial_equal(g, o, inp):
    assert g["status"] == 0, f"device status {g['status']}"
    assert g["used"] == o.used and g["n_admitted"] == o.n_admitted and g["n_freed"] == o.n_freed
    stats = [o.live_total, o.allocated, o.eligible, int(o.triggered),
             int(o.src_count.sum()), o.tokens_moved, o.n_freed, o.used]
    assert [int(x) for x in g["stats"]] == stats, (list(g["stats"]), stats)
    for key in ("token_slot", "live_count", "admitted", "src_count", "dst_indptr",
                "new_bt_indptr", "new_block_ids", "src_plan", "freed_indptr", "freed"):
        a = np.asarray(g[key], dtype=np.int64)
        b = np.asarray(getattr(o, key), dtype=np.int64)
        assert a.shape == b.shape, f"{key}: shape {a.shape} vs oracle {b.shape}"
        if not np.array_equal(a, b):
            bad = np.nonzero(a != b)[0]
            raise AssertionError(f"{key}: {len(bad)} mismatches, first at {bad[:5]}: "
                                 f"gpu {a[bad[:5]]} oracle {b[bad[:5]]}")
    for b, n in o.n_b.items():
        assert int(g["n_b"][b]) == n, f"n_b[{b}]"
        assert int(g["refs"][b]) == o.refs[b], f"refs[{b}]"
