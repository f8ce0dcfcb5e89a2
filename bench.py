#!/usr/bin/env python3
"""Throughput of the vToken KV repack hot path on one MI355X.

One step is one whole repack pass over one batch: vtoken_build_token_table (live-mask scan,
admission, token table, plan), vtoken_repack (gather of every live K/V row of every layer
into packed blocks) and vtoken_free_blocks, all enqueued on one stream. Inputs are resident
in HBM before the timed region. The pass is idempotent on unchanged inputs (out-of-place:
sources are never written), so every timed step does the full work again.

The default workload is the Llama-3-8B-shaped cache: 32 layers, 8 KV heads, head_dim 128,
bf16, block 16, 64 requests of U[2048, 8192] tokens, Random eviction keeping 30% of each
request plus its last 64 tokens, their blocks shuffled through a KV pool of 90% of free HBM
(a serving engine's whole KV cache; --pool-frac 0 packs the pool to the requests' blocks,
their destinations and 1024 spare blocks, 56 GiB).

Prints one JSON line. `value` is repacked KV GB/s over the whole step (read+write bytes of
the live rows: 2 * live tokens * 2*L*H*D*elem_bytes); `roofline` prices the repack kernel
alone against the 8 TB/s HBM peak, timed with HIP events on its launch stream (the build and
free calls are timed separately) and to the practical ceiling measured in the same run:
`ceiling` holds the streaming probe's copy over the pass's bytes in the same pool (the best
copy pattern measured on this memory system), torch's device copy and, with --ceiling all,
the repack kernel copying whole contiguous blocks of the same pool; `cpu_baseline` is the CPU
oracle on a sample of the planes.

--config llama3_70b_h2o runs a round of waves: the Llama-3-70B batch does not get all its
destinations from the free list at once, so each pass defers requests, its outputs are
applied and the batch re-submitted until none is left deferred; every wave's pass is replayed
--steps times (idempotent on unchanged inputs) and the line reports the round's bytes over the
sum of the waves' times.

    python bench.py [--steps K] [--warmup W] [--config NAME] [--variant V] [--grid G]
    python bench.py --mode copy      # plain device-to-device copy of known size
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
HBM_PEAK_GBS = 8000.0
PROFILES = os.path.join(ROOT, "profiles")


def parse_args(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="llama3_8b_random",
                    choices=["llama3_8b_random", "llama3_8b_h2o", "llama3_70b_h2o", "tiny",
                             "llama3_8b_scissorhands", "llama3_8b_block_copy",
                             "llama3_8b_shared_prefix"],
                    help="llama3_8b_block_copy: whole contiguous blocks to contiguous "
                         "destinations in the same-size pool, the copy's streaming ceiling "
                         "(a reference, not a paper workload); llama3_8b_shared_prefix: "
                         "prefix caching, timed as the partial pass")
    ap.add_argument("--seed", type=int, default=None)
    ap.add_argument("--block-size", type=int, default=16,
                    help="llama3_8b_random: tokens per block (the paper's sensitivity study "
                         "uses 16, 32 and 48)")
    ap.add_argument("--keep", type=float, default=0.3, help="keep ratio (70B config)")
    ap.add_argument("--kv-dtype", default="fp8_e4m3", help="70B config: fp8_e4m3 or bf16")
    ap.add_argument("--kv-heads", type=int, default=8,
                    help="70B config: KV heads in the cache (1 = one GPU's share under 8-way "
                         "tensor parallelism: 256 B / 128 B rows)")
    ap.add_argument("--ceiling", default="copy", choices=["none", "copy", "all"],
                    help="practical-ceiling leg after the timed steps: copy = the streaming "
                         "probe's copy over the pass's bytes in the same pool (another kernel) "
                         "and torch's device copy of 4 GiB; all = also the repack kernel on "
                         "whole contiguous blocks of the same pool (adds launches of the "
                         "timed kernel, so a profile of the run would mix the two)")
    ap.add_argument("--variant", type=int, default=0)
    ap.add_argument("--grid", type=int, default=0)
    ap.add_argument("--order", type=int, default=0)
    ap.add_argument("--pool-frac", type=float, default=0.9,
                    help="llama3_8b_random: size the block pool to this fraction of free HBM, "
                         "as a serving engine sizes its KV cache (the paper runs with "
                         "gpu_mem_util 0.90); 0 = the requests' blocks plus their "
                         "destinations plus 1024 spare blocks (56 GiB)")
    ap.add_argument("--partial", action="store_true",
                    help="llama3_8b_scissorhands: drive the loop with the paper's partial pass "
                         "(low-utilisation sources only) instead of whole-request repacks")
    ap.add_argument("--max-sources", type=int, default=1 << 40,
                    help="partial pass: bound B on the source blocks considered per pass")
    ap.add_argument("--inplace", action="store_true",
                    help="in-place mode: destinations are each request's own leading blocks; "
                         "bytes count only the rows that move")
    ap.add_argument("--mode", default="repack",
                    choices=["repack", "copy", "decode", "overlap", "stream", "placement",
                             "plan"],
                    help="decode: the consumer side, paged decode attention of every layer "
                         "through the slot mapping, before and after the repack; overlap: a "
                         "decode step (every layer) on the main stream with the repack pass on "
                         "a relocation stream, against the two one after the other; stream: "
                         "read / write / copy and decode-pattern probes, the memory system's "
                         "streaming ceilings; placement: the minimal 56 GiB pool allocated 4 times, "
                         "repack and write / read probes on each (for counter runs); plan: "
                         "the table build alone on batches of 8 to 3277 requests, short and "
                         "long, either side of its launch bounds")
    ap.add_argument("--q-heads", type=int, default=32, help="decode mode: query heads")
    ap.add_argument("--copy-gib", type=float, default=8.0)
    ap.add_argument("--graph", action="store_true",
                    help="repack mode: also time the whole pass captured once in a HIP graph "
                         "and replayed (graph_ms_per_step; for launch-bound small batches); "
                         "decode mode: the whole decode step (every layer) replayed from a "
                         "graph (after_repack.graph_step_ms)")
    ap.add_argument("--three-calls", action="store_true",
                    help="copy and freed list as two calls (vtoken_repack, vtoken_free_blocks) "
                         "instead of one launch (vtoken_repack_free)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-planes", type=int, default=4,
                    help="planes of the workload the CPU oracle is timed on")
    return ap.parse_args(argv)


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def separate_free(args) -> bool:
    """The copy and the freed list as two calls: asked for, or needed by copy options that
    the one-launch call does not take."""
    return args.three_calls or (args.variant, args.grid, args.order) != (0, 0, 0)


def timed_graph(args, cache, batch, plan):
    """The pass (build, copy, free; the same options as the eager steps) captured once in a
    HIP graph and replayed: warm-up replays, then the mean of `steps` replays between two
    events on the replaying stream."""
    import torch
    from paper_2608_13263_amd import binding as B
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        B.build_token_table(cache, batch, plan)
        if separate_free(args):
            B.repack_ex(cache, batch, plan, args.variant, args.grid, args.order)
            B.free_blocks(batch, plan)
        else:
            B.repack_free(cache, batch, plan)
    for _ in range(max(args.warmup, 1)):
        graph.replay()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(args.steps):
        graph.replay()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / args.steps


def make_workload(args):
    from paper_2608_13263_amd import workloads as W
    if args.config == "llama3_8b_random":
        pool = None
        if args.pool_frac > 0:
            import torch
            free, _ = torch.cuda.mem_get_info()
            pool = int(args.pool_frac * free)
        return W.llama3_8b_random(args.seed if args.seed is not None else 201, pool_bytes=pool,
                                  block_size=args.block_size)
    if args.config == "llama3_8b_h2o":
        return W.llama3_8b_h2o(args.seed if args.seed is not None else 301)
    if args.config == "tiny":
        return W.tiny_cache(args.seed if args.seed is not None else 101)
    if args.config == "llama3_8b_block_copy":
        import torch
        free, _ = torch.cuda.mem_get_info()
        return W.llama3_8b_block_copy(pool_bytes=int(args.pool_frac * free)
                                      if args.pool_frac > 0 else None)
    if args.config == "llama3_8b_shared_prefix":
        import torch
        free, _ = torch.cuda.mem_get_info()
        return W.llama3_8b_shared_prefix(args.seed if args.seed is not None else 701,
                                         pool_bytes=int(args.pool_frac * free)
                                         if args.pool_frac > 0 else None)
    import torch
    free, _ = torch.cuda.mem_get_info()
    budget = min(240 * 2 ** 30, int(0.85 * free))
    return W.llama3_70b_h2o(args.seed if args.seed is not None else 501, keep=args.keep,
                            dtype=args.kv_dtype, num_kv_heads=args.kv_heads, pool_bytes=budget)


_TRAFFIC_RECORD = re.compile(
    r"traffic_record: kernel=(\S+) workload=(\S+) source=(\S+) source_sha256=([0-9a-f]{64}) "
    r"algorithmic_bytes=(\d+) traffic_bytes=(\d+)")


def recorded_traffic(kernel: str, workload: str, bytes_alg: int):
    """HBM bytes per launch of `kernel` on `workload` from the committed rocprofv3 --pmc
    summaries in profiles/ (FETCH_SIZE and WRITE_SIZE, calibrated): a `traffic_record` line
    counts only while its kernel source file still hashes to the recorded SHA-256 and its
    algorithmic bytes equal this run's (the same requests, liveness and layout); else None."""
    for name in sorted(os.listdir(PROFILES)):
        if not name.endswith(".md"):
            continue
        for m in _TRAFFIC_RECORD.finditer(open(os.path.join(PROFILES, name)).read()):
            k, w, src, sha, alg, traffic = m.groups()
            if k != kernel or w != workload or int(alg) != int(bytes_alg):
                continue
            path = os.path.join(ROOT, src)
            if os.path.exists(path) and hashlib.sha256(open(path, "rb").read()).hexdigest() == sha:
                return int(traffic)
    return None


def host_kv_sample(shape, num_blocks: int, planes: int):
    """`planes` planes of host KV for the oracle legs: 64 MiB of random bytes tiled (the
    oracle's cost does not depend on the values)."""
    import numpy as np
    rng = np.random.Generator(np.random.PCG64(17))
    tile = np.frombuffer(rng.bytes(1 << 26), dtype=np.uint8)
    kv = np.empty((planes, num_blocks * shape.block_size, shape.row_bytes), dtype=np.uint8)
    flat = kv.reshape(-1)
    for o in range(0, flat.size, tile.size):
        n = min(tile.size, flat.size - o)
        flat[o:o + n] = tile[:n]
    return kv


def timed_passes(fn, min_seconds: float, max_repeats: int):
    times = []
    while len(times) < max_repeats and sum(times) < min_seconds:
        t0 = time.perf_counter()
        fn()
        times.append(time.perf_counter() - t0)
    return times


def positional_slots(inp):
    """Each token's slot before the pass: its request's block table at its position."""
    import numpy as np
    S = inp.shape.block_size
    out = np.empty(inp.num_tokens, dtype=np.int64)
    for r in range(inp.num_reqs):
        a, n = int(inp.tok_indptr[r]), int(inp.seq_lens[r])
        bt = inp.block_ids[inp.bt_indptr[r]:inp.bt_indptr[r + 1]].astype(np.int64)
        pos = np.arange(n)
        out[a:a + n] = bt[pos // S] * S + pos % S
    return out


def cpu_baseline(inp, planes: int, min_seconds: float = 10.0, max_repeats: int = 8,
                 inplace: bool = False):
    """The CPU oracle as it stands, on the full metadata and `planes` planes of host KV,
    timed over repeated passes until at least `min_seconds` of CPU work. Bytes as on the
    GPU: each moved live row read and written once (in place: rows whose slot changes)."""
    import numpy as np
    from oracle.repack import oracle_repack_inputs
    from paper_2608_13263_amd import workloads as W
    sh = inp.shape
    planes = max(2, min(planes, sh.num_planes)) // 2 * 2
    sample_shape = W.KVShape(planes // 2, sh.num_kv_heads, sh.head_dim, sh.block_size, sh.dtype)
    kv = host_kv_sample(sh, inp.num_blocks, planes)
    times = timed_passes(lambda: oracle_repack_inputs(inp, kv, inplace=inplace), min_seconds,
                         max_repeats)
    dt = sum(times) / len(times)
    res = oracle_repack_inputs(inp, None, inplace=inplace)
    live = int(np.asarray(res.live_count, dtype=np.int64)[np.asarray(res.admitted) == 1].sum())
    rows = live
    if inplace:
        ts = np.asarray(res.token_slot, dtype=np.int64)
        rows = int(((ts != positional_slots(inp)) & (inp.live != 0)).sum())
    bytes_alg = 2 * rows * sample_shape.token_bytes
    ncpu = len(os.sched_getaffinity(0))
    return {"value": round(bytes_alg / dt / 1e9, 3), "unit": "GB/s", "cores": 1,
            "kind": "oracle",
            "sample": f"{inp.name}{' (in place)' if inplace else ''}: full metadata and "
                      f"{planes} of {sh.num_planes} KV planes ({kv.nbytes / 2**30:.1f} GiB "
                      f"host), {live} live tokens, {rows} rows moved; {len(times)} passes of "
                      f"{dt:.2f} s; numpy, single-threaded: 1 core used of {ncpu} available",
            "seconds_per_pass": round(dt, 3),
            "live_tokens_per_ms": round(live * planes / sh.num_planes / (dt * 1e3), 3)}


def cpu_baseline_partial(inp, planes: int, max_sources: int, min_seconds: float = 10.0,
                         max_repeats: int = 8, what: str = "the round's moving pass"):
    """The partial-pass oracle (plan and copy) on one pass that moves rows: full metadata,
    `planes` planes of host KV."""
    import numpy as np
    from oracle.planner import PlannerParams as OracleParams
    from oracle.planner import plan_partial
    from paper_2608_13263_amd import workloads as W
    sh = inp.shape
    planes = max(2, min(planes, sh.num_planes)) // 2 * 2
    sample_shape = W.KVShape(planes // 2, sh.num_kv_heads, sh.head_dim, sh.block_size, sh.dtype)
    kv = host_kv_sample(sh, inp.num_blocks, planes)
    prm = OracleParams(max_sources=max_sources)
    run = lambda: plan_partial(inp.seq_lens, inp.tok_indptr, inp.bt_indptr,  # noqa: E731
                               inp.block_ids, inp.live, inp.slots(), inp.free_list,
                               sh.block_size, inp.num_blocks, prm, pinned=inp.pinned, kv=kv)
    times = timed_passes(run, min_seconds, max_repeats)
    dt = sum(times) / len(times)
    moved = int(run().tokens_moved)
    ncpu = len(os.sched_getaffinity(0))
    return {"value": round(2 * moved * sample_shape.token_bytes / dt / 1e9, 3), "unit": "GB/s",
            "cores": 1, "kind": "oracle",
            "sample": f"{what}: full metadata and {planes} of {sh.num_planes} "
                      f"KV planes ({kv.nbytes / 2**30:.1f} GiB host), {moved} rows moved; "
                      f"{len(times)} passes of {dt:.2f} s; numpy, single-threaded: 1 core used "
                      f"of {ncpu} available",
            "seconds_per_pass": round(dt, 3)}


def cpu_baseline_decode(inp, token_slot, q_heads: int, min_seconds: float = 10.0):
    """The decode oracle (float64, one request at a time) over requests in order until
    `min_seconds`, one layer, random K/V values of the requests' live rows; BLAS held to one
    thread. Bytes as on the GPU: each live token's head rows of K and V."""
    import numpy as np
    from threadpoolctl import threadpool_limits
    from oracle.attention import decode_batch, slot_mapping
    sh = inp.shape
    H, D = sh.num_kv_heads, sh.head_dim
    indptr, slots = slot_mapping(token_slot, inp.tok_indptr, inp.seq_lens)
    rng = np.random.default_rng(5)
    done_tok, done_req, spent = 0, 0, 0.0
    with threadpool_limits(limits=1):
        for r in range(inp.num_reqs):
            n = int(indptr[r + 1] - indptr[r])
            k = rng.standard_normal((n, H, D))
            v = rng.standard_normal((n, H, D))
            q = rng.standard_normal((1, q_heads, D))
            t0 = time.perf_counter()
            decode_batch(q, k, v, np.array([0, n]), np.arange(n))
            spent += time.perf_counter() - t0
            done_tok += n
            done_req += 1
            if spent >= min_seconds:
                break
    bytes_alg = done_tok * 2 * H * D * sh.elem_bytes
    return {"value": round(bytes_alg / spent / 1e9, 3), "unit": "GB/s", "cores": 1,
            "kind": "oracle",
            "sample": f"{done_req} of {inp.num_reqs} requests ({done_tok} live tokens) of one "
                      f"layer, {q_heads} query heads; float64 numpy, BLAS limited to 1 thread",
            "seconds": round(spent, 3)}


def inputs_sha256(inp) -> dict:
    """SHA-256 (first 16 hex digits) of every input array of the pass."""
    import numpy as np
    out = {}
    for k in ("seq_lens", "tok_indptr", "bt_indptr", "block_ids", "live", "free_list"):
        a = np.ascontiguousarray(getattr(inp, k))
        out[k] = hashlib.sha256(a.tobytes()).hexdigest()[:16]
    return out


def streaming_ceiling(args, inp, kv, cache, bytes_alg: int, stream, block_copy: bool,
                      steps: int = 10):
    """The copy's practical ceiling, timed in the same run after the timed steps: the streaming
    probe's plane copy (bench_probe.hip; the repack's work order over contiguous chunks) over
    about the pass's bytes inside the same KV pool; torch's device copy of 4 GiB
    when that much HBM is still free (a library copy, for reference); with `block_copy` the
    repack kernel on whole contiguous blocks (block-copy metadata over the same KV tensor,
    which adds launches of the timed kernel to a profile of the run). The copies overwrite
    bytes of the pool; the copy is value-agnostic."""
    import torch
    out = probe_copy_ceiling(kv, inp.shape.num_planes, bytes_alg, stream, steps)
    if block_copy:
        out.update(block_copy_ceiling(inp, cache, bytes_alg, stream, steps))
    free, _ = torch.cuda.mem_get_info()
    n = 4 << 30
    if free > 2 * n + (1 << 30):
        src = torch.empty(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        src.fill_(3)
        dst.copy_(src)
        cev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(5)]
        for a, b in cev:
            a.record()
            dst.copy_(src)
            b.record()
        torch.cuda.synchronize()
        cms = sum(a.elapsed_time(b) for a, b in cev) / len(cev)
        out["torch_copy_4GiB_GBps"] = round(2 * n / (cms / 1e3) / 1e9, 1)
        del src, dst
    log(f"ceiling: {out}")
    return out


def probe_copy_ceiling(kv, num_planes: int, bytes_alg: int, stream, steps: int = 10):
    """The streaming ceiling of the repack's own work order: bench_probe.hip's plane copy over
    the KV tensor's planes, consecutive workgroups on one 32 KiB chunk index of different
    planes (the repack's block-major order), contiguous chunks from the first half of each plane
    to its second half, about the pass's bytes in all. Read + write bytes per second."""
    import ctypes
    import torch
    lib = probe_library()
    chunk = 32768
    plane_bytes = kv.numel() * kv.element_size() // num_planes
    per_plane = plane_bytes // chunk
    n = min(bytes_alg // 2 // (chunk * num_planes), per_plane // 2)
    if n == 0 or plane_bytes % chunk:
        return {}
    sh = ctypes.c_void_p(stream.cuda_stream)
    call = lambda: lib.vtoken_probe_plane_copy(kv.data_ptr(), plane_bytes, num_planes, 0,  # noqa: E731
                                               per_plane // 2, n, sh)
    for _ in range(3):
        if call() != 0:
            raise SystemExit("probe plane copy refused its arguments")
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    for a, b in evs:
        a.record(stream)
        call()
        b.record(stream)
    torch.cuda.synchronize()
    ms = sum(a.elapsed_time(b) for a, b in evs) / steps
    nbytes = 2 * n * chunk * num_planes
    gbs = nbytes / (ms / 1e3) / 1e9
    return {"probe_copy": "bench_probe.hip plane copy: the repack's work order (consecutive "
                          "workgroups on one chunk of different planes) over contiguous 32 KiB "
                          "chunks of the same KV pool, non-temporal loads, sc1 stores",
            "probe_copy_bytes": nbytes, "probe_copy_ms": round(ms, 4),
            "probe_copy_GBps": round(gbs, 1), "probe_copy_frac": round(gbs / HBM_PEAK_GBS, 4)}


def block_copy_ceiling(inp, cache, bytes_alg: int, stream, steps: int):
    import torch
    from paper_2608_13263_amd import binding as B
    from paper_2608_13263_amd import workloads as W
    sh = inp.shape
    per_req = 2 * 2 * sh.block_size * sh.token_bytes
    R = max(1, min(int(round(bytes_alg / per_req)), (inp.num_blocks - 1024) // 5))
    ref = W.block_copy_inputs(sh, R, inp.num_blocks, name="block_copy")
    cb = B.Batch.from_inputs(ref)
    cp = B.Plan.allocate(cb, sh.block_size)
    B.build_token_table(cache, cb, cp, stream)
    for _ in range(3):
        B.repack(cache, cb, cp, stream)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    for a, b in evs:
        a.record(stream)
        B.repack(cache, cb, cp, stream)
        b.record(stream)
    torch.cuda.synchronize()
    if int(cp.counters[3]) != 0 or int(cp.counters[1]) != R:
        raise SystemExit("block-copy reference: unexpected plan")
    ms = sum(a.elapsed_time(b) for a, b in evs) / steps
    ref_bytes = 2 * R * 2 * sh.block_size * sh.token_bytes
    gbs = ref_bytes / (ms / 1e3) / 1e9
    return {"block_copy": "repack_direct_kernel on whole contiguous blocks of the same pool",
            "block_copy_bytes": ref_bytes, "block_copy_ms": round(ms, 4),
            "block_copy_GBps": round(gbs, 1), "block_copy_frac": round(gbs / HBM_PEAK_GBS, 4)}


def run_copy(args):
    """A plain device-to-device copy of known size: the practical HBM ceiling, and the
    calibration kernel for the FETCH_SIZE / WRITE_SIZE counters."""
    import torch
    n = int(args.copy_gib * 2 ** 30)
    src = torch.empty(n, dtype=torch.uint8, device="cuda")
    src.fill_(3)
    dst = torch.empty_like(src)
    for _ in range(args.warmup):
        dst.copy_(src)
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    for a, b in evs:
        a.record()
        dst.copy_(src)
        b.record()
    torch.cuda.synchronize()
    ms = sum(a.elapsed_time(b) for a, b in evs) / len(evs)
    gbs = 2 * n / (ms / 1e3) / 1e9
    print(json.dumps({"mode": "copy", "bytes_each_way": n, "ms": round(ms, 4),
                      "GBps_read_plus_write": round(gbs, 1),
                      "frac_of_8TBps": round(gbs / HBM_PEAK_GBS, 4)}), flush=True)


PROBE_SOURCE = os.path.join(ROOT, "bench_probe.hip")


def probe_library(rebuild: bool = False):
    """The memory-system probes (bench_probe.hip; measurement tooling, not part of the C ABI)
    as a ctypes library, compiled on demand with the package's hipcc flags into
    _build/libvtoken_probe-<source hash>.so (an existing build of the same source is reused
    unless `rebuild`)."""
    import ctypes
    from paper_2608_13263_amd import build as Bld
    sha = hashlib.sha256(open(PROBE_SOURCE, "rb").read()).hexdigest()[:16]
    path = os.path.join(ROOT, "_build", f"libvtoken_probe-{sha}.so")
    if rebuild or not os.path.exists(path):
        os.makedirs(os.path.dirname(path), exist_ok=True)
        Bld.build_one(path, [PROBE_SOURCE])
    lib = ctypes.CDLL(path)
    vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
    lib.vtoken_probe_read.argtypes = [vp, i64, i32, vp, vp]
    lib.vtoken_probe_write.argtypes = [vp, i64, i32, vp]
    lib.vtoken_probe_copy.argtypes = [vp, vp, i64, i32, vp]
    lib.vtoken_probe_head_read.argtypes = [vp, i64, i32, vp, i64, i32, vp, vp]
    lib.vtoken_probe_plane_copy.argtypes = [vp, i64, i32, i64, i64, i64, vp]
    return lib


def run_plan(args):
    """vtoken_build_token_table alone on synthetic batches either side of its launch bounds
    (one planning launch up to 24 requests and 8192 tokens; count and plan launches, the plan
    workgroups admitting for themselves, up to 256 requests, or 512 averaging 1024 tokens or
    more; a separate admission launch above): the median of 30 calls, each between HIP events
    on the launch stream (a call's launch overhead included). 16-byte rows (the table build
    does not read the cache), Bernoulli(0.5) liveness, free list of every request's blocks."""
    import numpy as np
    import torch
    from paper_2608_13263_amd import binding as B
    from paper_2608_13263_amd import workloads as W
    rng = np.random.default_rng(args.seed if args.seed is not None else 0)
    shapes = [("short", 32, 96, R) for R in (8, 24, 64, 256, 257, 512, 1024, 3277)]
    shapes += [("long", 2048, 8192, R) for R in (64, 128, 256, 512, 1024)]
    stream = torch.cuda.current_stream()
    out = []
    for kind, lo, hi, R in shapes:
        lens = rng.integers(lo, hi + 1, size=R)
        masks = [(rng.random(int(n)) < 0.5).astype(np.int8) for n in lens]
        M = sum(-(-len(m) // 16) for m in masks)
        inp = W.from_masks([m.tolist() for m in masks], W.KVShape(1, 1, 8, 16, "fp16"),
                           free_blocks=M, seed=1, name=f"{kind}_{R}")
        kv = W.kv_device(inp.shape, inp.num_blocks, 0)
        cache = B.KVCache(kv, 1, 1, 8, 16)
        batch = B.Batch.from_inputs(inp)
        plan = B.Plan.allocate(batch, 16)
        for _ in range(5):
            B.build_token_table(cache, batch, plan, stream)
        torch.cuda.synchronize()
        ts = []
        for _ in range(30):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            B.build_token_table(cache, batch, plan, stream)
            b.record(stream)
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b) * 1e3)
        status = int(plan.counters[3])
        if status != 0:
            raise SystemExit(f"device status {B.STATUS.get(status, status)}")
        out.append({"requests": R, "tokens": inp.num_tokens, "kind": kind,
                    "build_us": round(float(np.median(ts)), 1)})
        log(f"plan {kind} R={R} T={inp.num_tokens}: {out[-1]['build_us']} us")
        del kv, cache, batch, plan
    print(json.dumps({"metric": "vtoken_build_token_table time per call (us)", "mode": "plan",
                      "value": None, "unit": "us", "n_gpus": 1, "higher_is_better": False,
                      "data": "synthetic", "cases": out,
                      "config": {"workload": "plan_batches", "row_bytes": 16,
                                 "block_size": 16, "keep": 0.5}}), flush=True)
    return 0


def run_stream(args):
    """Streaming rates of the memory system (bench_probe.hip) in one pool sized as the
    repack benchmark's (90% of free HBM by default): reads, writes and copies of 32 KiB chunks
    and the decode's pattern (256-byte head pieces of 2 KiB token rows through a slot list of
    shuffled 16-token blocks, K and V planes). These are the ceilings the repack and the
    decode are set against; HIP events on the launch stream."""
    import ctypes
    import torch
    lib = probe_library()
    free, _ = torch.cuda.mem_get_info()
    chunk = 32768
    pool = int((args.pool_frac if args.pool_frac > 0 else 0.5) * free)
    # two regions (source at 0, destination at half the pool) of up to 64 GiB, whole multiples
    # of 1024 chunks so that every interleave below divides the chunk count
    region = min(64 * 2 ** 30, pool // 4) // (1024 * chunk) * (1024 * chunk)
    buf = torch.zeros(pool // chunk * chunk, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()
    sh = ctypes.c_void_p(stream.cuda_stream)
    src = buf.data_ptr()
    dst = buf.data_ptr() + (buf.numel() // 2) // chunk * chunk
    log(f"stream probes: pool {buf.numel() / 2**30:.1f} GiB, regions of "
        f"{region / 2**30:.1f} GiB")

    def timed(call, nbytes):
        code = call()
        if code != 0:
            raise SystemExit(f"probe call failed with {code}")
        torch.cuda.synchronize()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(max(args.steps // 4, 3))]
        for a, b in evs:
            a.record(stream)
            call()
            b.record(stream)
        torch.cuda.synchronize()
        ms = sum(a.elapsed_time(b) for a, b in evs) / len(evs)
        return round(nbytes / (ms / 1e3) / 1e9, 1)

    rates = {}
    for nt in (1, 0):
        rates[f"read_{'nt' if nt else 'plain'}"] = timed(
            lambda: lib.vtoken_probe_read(src, region, nt, sink.data_ptr(), sh), region)
    for ways in (1, 64):
        rates[f"write_ways{ways}"] = timed(
            lambda: lib.vtoken_probe_write(dst, region, ways, sh), region)
        rates[f"copy_ways{ways}"] = timed(
            lambda: lib.vtoken_probe_copy(src, dst, region, ways, sh), 2 * region)
    # decode pattern over the source region as a K plane and a V plane of 2 KiB rows
    plane = region // 2
    rows = plane // 2048
    tokens = rows // 64 * 64
    g = torch.Generator().manual_seed(5)
    blocks = torch.randperm(rows // 16, generator=g)
    slots = (blocks.repeat_interleave(16) * 16 + torch.arange(16).repeat(rows // 16))
    slots = slots[:tokens].to(torch.int32).cuda()
    for nt in (1, 0):
        rates[f"head_pieces_{'nt' if nt else 'plain'}"] = timed(
            lambda: lib.vtoken_probe_head_read(src, plane, 2048, slots.data_ptr(), tokens, nt,
                                               sink.data_ptr(), sh), 2 * tokens * 256 * 8)
    best_copy = max(rates["copy_ways1"], rates["copy_ways64"])
    out = {"metric": "streaming rates of the memory system (probe kernels)", "mode": "stream",
           "value": best_copy, "unit": "GB/s", "n_gpus": 1, "higher_is_better": True,
           "data": "synthetic", "rates_GBps": rates,
           "frac_of_8TBps": {k: round(v / HBM_PEAK_GBS, 4) for k, v in rates.items()},
           "config": {"workload": "stream_probes", "pool_gib": round(buf.numel() / 2 ** 30, 1),
                      "region_gib": round(region / 2 ** 30, 2), "chunk_bytes": chunk,
                      "decode_pattern": f"{tokens} tokens x 8 heads x 256 B, K and V planes"}}
    print(json.dumps(out), flush=True)
    return 0


def run_placement(args):
    """The Llama-3-8B Random requests in the minimal pool (their blocks, their destinations and
    1024 spare blocks: 56 GiB), allocated four times in one process (all held; consecutive
    allocations of this size land on placements of two speeds). On each pool, in this order:
    the repack pass (--warmup + --steps, the copy timed with HIP events), the probe write of
    half the pass's bytes (64 chunks apart, the copy's store pattern), the probe read of the
    same bytes. Run under rocprofv3 --pmc, the dispatches of each pool come before those of the
    next, so counters can be set side by side per placement."""
    import ctypes
    import torch
    from paper_2608_13263_amd import binding as B
    from paper_2608_13263_amd import workloads as W
    lib = probe_library()
    inp = W.llama3_8b_random(args.seed if args.seed is not None else 201)
    sh = inp.shape
    stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    batch = B.Batch.from_inputs(inp)
    pools, kvs = [], []
    chunk, unit = 32768, 1024 * 32768

    def timed(fn, n):
        for _ in range(max(args.warmup, 1)):
            fn()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(n)]
        for a, b in evs:
            a.record(stream)
            fn()
            b.record(stream)
        torch.cuda.synchronize()
        return sum(a.elapsed_time(b) for a, b in evs) / n

    for k in range(4):
        kv = W.kv_device(sh, inp.num_blocks, 1 + k)
        kvs.append(kv)
        cache = B.KVCache(kv, sh.num_layers, sh.num_kv_heads, sh.head_dim, sh.block_size)
        plan = B.Plan.allocate(batch, sh.block_size)
        B.build_token_table(cache, batch, plan, stream)
        torch.cuda.synchronize()
        log(f"pool {k}: {inp.pool_bytes() / 2**30:.1f} GiB at {kv.data_ptr():#x}")
        ms = timed(lambda: B.repack(cache, batch, plan, stream), args.steps)
        cnt = plan.counters.cpu().tolist()
        if cnt[3] != 0:
            raise SystemExit(f"device status {B.STATUS.get(cnt[3], cnt[3])}")
        moved = int((plan.live_count[:inp.num_reqs].long() *
                     plan.admitted[:inp.num_reqs].long()).sum())
        bytes_alg = 2 * moved * sh.token_bytes
        total = kv.numel() * kv.element_size()
        region = min(bytes_alg // 2, total // 2) // unit * unit
        dst = kv.data_ptr() + (total // 2) // chunk * chunk
        sink = torch.zeros(1, dtype=torch.int32, device="cuda")
        w_ms = timed(lambda: lib.vtoken_probe_write(dst, region, 64, sp), max(args.steps // 2, 3))
        r_ms = timed(lambda: lib.vtoken_probe_read(kv.data_ptr(), region, 1, sink.data_ptr(), sp),
                     max(args.steps // 2, 3))
        pools.append({"pool": k, "address": hex(kv.data_ptr()), "repack_ms": round(ms, 4),
                      "repack_GBps": round(bytes_alg / (ms / 1e3) / 1e9, 1),
                      "repack_frac": round(bytes_alg / (ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
                      "probe_write_GBps": round(region / (w_ms / 1e3) / 1e9, 1),
                      "probe_read_GBps": round(region / (r_ms / 1e3) / 1e9, 1),
                      "bytes_alg": bytes_alg, "probe_bytes": region})
        log(f"pool {k}: {pools[-1]}")
    out = {"metric": "repack and probe rates on four 56 GiB allocations", "mode": "placement",
           "value": min(p["repack_GBps"] for p in pools), "unit": "GB/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "higher_is_better": True,
           "data": "synthetic", "pools": pools,
           "config": {"workload": inp.name, "recipe": inp.note,
                      "pool_gib": round(inp.pool_bytes() / 2 ** 30, 2)}}
    print(json.dumps(out), flush=True)
    return 0


def gpu_busy_while_host_enqueues():
    """Enqueue a spin kernel of about half a millisecond: the calls enqueued after it (their
    argument marshalling included) are in the queue before it ends, so that events recorded
    after it time the GPU work, not the host, when the GPU was idle before."""
    import torch
    torch.cuda._sleep(1_000_000)


def run_scissorhands(args):
    """Scissorhands-style repeated repack: 256 requests, a repack every 512 decode steps in a
    pool of min(240 GiB, 85% of free HBM). A round is the host-side decode bookkeeping
    followed by passes until one repacks nothing; every pass (build + repack + free) is timed
    with HIP events. One warm-up round, then `--steps` timed rounds (default 4)."""
    import numpy as np
    import torch
    from paper_2608_13263_amd import binding as B
    from paper_2608_13263_amd import workloads as W
    free, _ = torch.cuda.mem_get_info()
    shape = W.KVShape(32, 8, 128, 16, "bf16")
    budget = min(240 * 2 ** 30, int(0.85 * free))
    stream = W.ScissorhandsStream(seed=args.seed if args.seed is not None else 401,
                                  pool_blocks=budget // shape.block_bytes)
    kv = W.kv_device(shape, stream.num_blocks, 1)
    cache = B.KVCache(kv, shape.num_layers, shape.num_kv_heads, shape.head_dim,
                      shape.block_size)
    S = shape.block_size

    def one_round():
        stream.decode()
        passes = []
        while True:
            inp = stream.inputs()
            batch = B.Batch.from_inputs(inp)
            plan = B.Plan.allocate(batch, S, inplace=args.inplace)
            ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True),
                  torch.cuda.Event(enable_timing=True))
            torch.cuda.synchronize()
            gpu_busy_while_host_enqueues()
            ev[0].record()
            if args.inplace:
                B.build_token_table_inplace(cache, batch, plan)
                ev[1].record()
                B.repack_inplace(cache, batch, plan)
                B.free_blocks(batch, plan)
            else:
                B.build_token_table(cache, batch, plan)
                ev[1].record()
                B.repack_free(cache, batch, plan)
            ev[2].record()
            torch.cuda.synchronize()
            cnt = plan.counters.cpu().tolist()
            if cnt[3] != 0:
                raise SystemExit(f"device status {B.STATUS.get(cnt[3], cnt[3])}")
            R = inp.num_reqs
            adm = plan.admitted[:R].cpu().numpy()
            live = plan.live_count[:R].cpu().numpy().astype(np.int64)
            nbi = plan.new_bt_indptr[:R + 1].cpu().numpy()
            nbids = plan.new_block_ids[:int(nbi[-1])].cpu().numpy()
            freed = plan.freed[:cnt[2]].cpu().numpy()
            rows = int((live * adm).sum())
            if args.inplace:   # rows whose slot changes (the rest are already in place)
                ts = plan.token_slot[:inp.num_tokens].cpu().numpy().astype(np.int64)
                rows = int(((ts != positional_slots(inp)) & (inp.live != 0)).sum())
            passes.append(dict(ms=ev[0].elapsed_time(ev[2]), moved=int((live * adm).sum()),
                               rows=rows, admitted=cnt[1], used=cnt[0]))
            # in place no free-list entry is consumed (counters[0] counts own blocks then)
            stream.commit(adm, nbi, nbids, 0 if args.inplace else cnt[0], freed)
            if cnt[1] == 0:
                return passes

    log(f"scissorhands: {len(stream.pos)} requests, pool {stream.num_blocks} blocks = "
        f"{stream.num_blocks * shape.block_bytes / 2**30:.1f} GiB; warm-up round")
    one_round()
    rounds, resident = [], []
    for i in range(args.steps if args.steps != 20 else 4):
        rounds.append(one_round())
        resident.append(stream.resident_blocks())
        log(f"round {i}: " + ", ".join(f"{p['admitted']} req / {p['moved']} tok / "
                                      f"{p['ms']:.2f} ms" for p in rounds[-1]) +
            f"; resident {resident[-1]}")
    moved = sum(p["moved"] for r in rounds for p in r)
    rows = sum(p["rows"] for r in rounds for p in r)
    ms = sum(p["ms"] for r in rounds for p in r)
    bytes_alg = 2 * rows * shape.token_bytes
    value = bytes_alg / (ms / 1e3) / 1e9
    out = {
        "metric": "repacked KV GB/s (read+write) as % of HBM peak; live tokens repacked/ms",
        "mode": "inplace" if args.inplace else "repack",
        "value": round(value, 2), "unit": "GB/s", "n_gpus": 1, "steps": len(rounds),
        "warmup": 1, "ms_per_step": round(ms / len(rounds), 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "u8", "data": "synthetic",
        "pct_of_hbm_peak": round(100 * value / HBM_PEAK_GBS, 2),
        "live_tokens_per_ms": round(moved / ms, 1),
        "config": {"workload": "llama3_8b_scissorhands",
                   "recipe": "bf16 32x8x128, S=16, 256 req, logical length U[2048,32768], "
                             "Scissorhands budget 0.25 + window 256, repack every 512 decode "
                             "steps, passes until one repacks nothing",
                   "pool_gib": round(stream.num_blocks * shape.block_bytes / 2 ** 30, 2),
                   "rounds": [[{k: (round(v, 3) if isinstance(v, float) else v)
                                for k, v in p.items()} for p in r] for r in rounds],
                   "resident_blocks_after_round": resident,
                   "live_tokens_repacked": moved, "rows_moved": rows,
                   "bytes_alg_total": bytes_alg},
        "roofline": None, "cpu_baseline": None,
    }
    print(json.dumps(out), flush=True)
    return 0


def run_partial_stream(args):
    """The Scissorhands loop of run_scissorhands driven by the partial pass: requests are
    token tables, each pass plans on the device (per-block live counts, F > 0.25 trigger,
    low-utilisation unpinned sources, bound B) and copies only the sources' live rows. Plan
    and copy are timed with HIP events; `value` counts the bytes of the rows moved."""
    import numpy as np
    import torch
    from paper_2608_13263_amd import binding as B
    from paper_2608_13263_amd import workloads as W
    free, _ = torch.cuda.mem_get_info()
    shape = W.KVShape(32, 8, 128, 16, "bf16")
    budget = min(240 * 2 ** 30, int(0.85 * free))
    stream = W.PartialStream(seed=args.seed if args.seed is not None else 401,
                             pool_blocks=budget // shape.block_bytes)
    kv = W.kv_device(shape, stream.num_blocks, 1)
    cache = B.KVCache(kv, shape.num_layers, shape.num_kv_heads, shape.head_dim,
                      shape.block_size)
    S = shape.block_size
    params = B.PlannerParams(max_sources=args.max_sources)
    moving_pass = []          # the inputs of the first timed pass that moves rows

    def one_round():
        stream.decode()
        passes = []
        while True:
            inp = stream.inputs()
            batch = B.Batch.from_inputs(inp)
            slot_in = torch.from_numpy(inp.slot_in).cuda()
            plan = B.Plan.allocate(batch, S)
            state = B.PlannerState.allocate(inp.num_blocks, batch, pinned=inp.pinned)
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
            torch.cuda.synchronize()
            gpu_busy_while_host_enqueues()
            ev[0].record()
            B.plan_partial(cache, batch, slot_in, plan, state, params)
            ev[1].record()
            B.repack(cache, batch, plan)
            ev[2].record()
            torch.cuda.synchronize()
            cnt = plan.counters.cpu().tolist()
            if cnt[3] != 0:
                raise SystemExit(f"device status {B.STATUS.get(cnt[3], cnt[3])}")
            st = state.stats.cpu().tolist()
            R = inp.num_reqs
            nbi = plan.new_bt_indptr[:R + 1].cpu().numpy()
            passes.append(dict(plan_ms=ev[0].elapsed_time(ev[1]),
                               copy_ms=ev[1].elapsed_time(ev[2]), moved=int(st[5]),
                               admitted=cnt[1], used=cnt[0], released=cnt[2],
                               F=1.0 - st[0] / max(st[1] * S, 1), attempted=int(st[3])))
            if cnt[1] > 0 and not moving_pass:
                moving_pass.append(inp)
            stream.commit(plan.token_slot[:inp.num_tokens].cpu().numpy(), nbi,
                          plan.new_block_ids[:int(nbi[-1])].cpu().numpy(), cnt[0],
                          state.sources[:cnt[2]].cpu().numpy())
            if cnt[1] == 0:
                return passes

    log(f"scissorhands (partial pass): {len(stream.pos)} requests, pool {stream.num_blocks} "
        f"blocks = {stream.num_blocks * shape.block_bytes / 2**30:.1f} GiB; warm-up round")
    one_round()
    moving_pass.clear()
    rounds, resident = [], []
    for i in range(args.steps if args.steps != 20 else 4):
        rounds.append(one_round())
        resident.append(stream.resident_blocks())
        log(f"round {i}: " + ", ".join(
            f"{p['admitted']} req / {p['moved']} tok / F {p['F']:.3f} / plan {p['plan_ms']:.2f} "
            f"+ copy {p['copy_ms']:.2f} ms" for p in rounds[-1]) + f"; resident {resident[-1]}")
    moved = sum(p["moved"] for r in rounds for p in r)
    ms = sum(p["plan_ms"] + p["copy_ms"] for r in rounds for p in r)
    copy_ms = sum(p["copy_ms"] for r in rounds for p in r)
    bytes_alg = 2 * moved * shape.token_bytes
    value = bytes_alg / (ms / 1e3) / 1e9
    out = {
        "metric": "repacked KV GB/s (read+write) as % of HBM peak; live tokens repacked/ms",
        "mode": "partial", "value": round(value, 2), "unit": "GB/s", "n_gpus": 1,
        "steps": len(rounds), "warmup": 1, "ms_per_step": round(ms / len(rounds), 4),
        "higher_is_better": True, "dtype": "u8", "data": "synthetic",
        "live_tokens_per_ms": round(moved / ms, 1),
        "config": {"workload": "llama3_8b_scissorhands_partial",
                   "recipe": "bf16 32x8x128, S=16, 256 req, logical length U[2048,32768], "
                             "Scissorhands budget 0.25 + window 256, a partial pass every 512 "
                             "decode steps (theta_F 0.25, append blocks pinned), passes until "
                             "one repacks nothing",
                   "max_sources": args.max_sources,
                   "pool_gib": round(stream.num_blocks * shape.block_bytes / 2 ** 30, 2),
                   "rounds": [[{k: (round(v, 4) if isinstance(v, float) else v)
                                for k, v in p.items()} for p in r] for r in rounds],
                   "resident_blocks_after_round": resident,
                   "live_tokens_moved": moved, "bytes_alg_total": bytes_alg},
        "roofline": {"bound": "hbm", "kernel": "repack_direct_kernel",
                     "achieved": round(bytes_alg / (copy_ms / 1e3) / 1e9, 1) if copy_ms else None,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(bytes_alg / (copy_ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4)
                     if copy_ms else None, "traffic": None},
        "cpu_baseline": None if args.no_cpu_baseline or not moving_pass else
        cpu_baseline_partial(moving_pass[0], args.cpu_planes, args.max_sources),
    }
    print(json.dumps(out), flush=True)
    return 0


def run_partial_pass(args):
    """One partial pass (Sec. 3.3) over a token-table workload with shared prefixes (Sec.
    5.7): plan on the device, then copy the selected sources' live rows. Every step re-runs
    the pass on the same inputs (same plan, same rows between the same addresses). Blocks in
    several tables are shared and never move (I4); the run checks that none was a source."""
    import numpy as np
    import torch
    from paper_2608_13263_amd import binding as B
    from paper_2608_13263_amd import workloads as W
    t_setup = time.perf_counter()
    inp = make_workload(args)
    sh = inp.shape
    log(f"{inp.name}: {inp.num_reqs} requests, {inp.num_tokens} tokens, pool "
        f"{inp.num_blocks} blocks = {inp.pool_bytes() / 2**30:.1f} GiB")
    kv = W.kv_device(sh, inp.num_blocks, 1)
    cache = B.KVCache(kv, sh.num_layers, sh.num_kv_heads, sh.head_dim, sh.block_size)
    batch = B.Batch.from_inputs(inp)
    slot_in = torch.from_numpy(np.ascontiguousarray(inp.slots(), dtype=np.int32)).cuda()
    plan = B.Plan.allocate(batch, sh.block_size)
    state = B.PlannerState.allocate(inp.num_blocks, batch, pinned=inp.pinned)
    params = B.PlannerParams(max_sources=args.max_sources)
    stream = torch.cuda.current_stream()

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        B.plan_partial(cache, batch, slot_in, plan, state, params, stream)
        if ev is not None:
            ev[1].record(stream)
        B.repack(cache, batch, plan, stream)
        if ev is not None:
            ev[2].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"setup {time.perf_counter() - t_setup:.1f} s; timing {args.steps} steps")
    evs = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(3))
           for _ in range(args.steps)]
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    step_ms = (time.perf_counter() - t0) * 1e3 / args.steps
    plan_ms = sum(e[0].elapsed_time(e[1]) for e in evs) / args.steps
    copy_ms = sum(e[1].elapsed_time(e[2]) for e in evs) / args.steps
    cnt = plan.counters.cpu().tolist()
    if cnt[3] != 0:
        raise SystemExit(f"device status {B.STATUS.get(cnt[3], cnt[3])}")
    st = state.stats.cpu().tolist()
    moved = int(st[5])
    refs = state.refs.cpu().numpy()
    shared = np.nonzero(refs > 1)[0]
    sources = state.sources[:cnt[2]].cpu().numpy()
    if np.isin(sources, shared).any():
        raise SystemExit("a shared block was selected as a source")
    shared_live = int(state.n_b.cpu().numpy()[shared].sum())
    bytes_alg = 2 * moved * sh.token_bytes
    achieved = bytes_alg / (copy_ms / 1e3) / 1e9 if copy_ms > 0 else None
    log(f"step {step_ms:.3f} ms: plan {plan_ms:.3f} + copy {copy_ms:.3f} ms, {moved} tokens "
        f"moved, {len(shared)} shared blocks kept")
    out = {
        "metric": "repacked KV GB/s (read+write) as % of HBM peak; live tokens repacked/ms",
        "mode": "partial", "value": round(bytes_alg / (step_ms / 1e3) / 1e9, 2), "unit": "GB/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(step_ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "u8",
        "data": "synthetic",
        "pct_of_hbm_peak": round(100 * bytes_alg / (step_ms / 1e3) / 1e9 / HBM_PEAK_GBS, 2),
        "live_tokens_per_ms": round(moved / step_ms, 1), "plan_ms": round(plan_ms, 4),
        "repack_ms": round(copy_ms, 4),
        "config": {"workload": inp.name, "recipe": inp.note, "requests": inp.num_reqs,
                   "tokens": inp.num_tokens, "pool_blocks": inp.num_blocks,
                   "pool_gib": round(inp.pool_bytes() / 2 ** 30, 2),
                   "live_tokens_moved": moved, "triggered": int(st[3]),
                   "F": round(1.0 - st[0] / max(st[1] * sh.block_size, 1), 4),
                   "eligible_blocks": int(st[2]), "sources": cnt[2], "destinations": cnt[0],
                   "admitted": cnt[1], "shared_blocks": int(len(shared)),
                   "shared_live_tokens_kept": shared_live, "max_sources": args.max_sources,
                   "bytes_alg_per_step": bytes_alg},
        "roofline": {"bound": "hbm", "kernel": "repack_direct_kernel",
                     "achieved": round(achieved, 1) if achieved else None,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4) if achieved else None,
                     "traffic": recorded_traffic("repack_direct_kernel", inp.name, bytes_alg)},
        "cpu_baseline": None if args.no_cpu_baseline or moved == 0 else
        cpu_baseline_partial(inp, args.cpu_planes, args.max_sources, what="the pass"),
    }
    print(json.dumps(out), flush=True)
    return 0


def run_waves(args, inp, kv, cache, stream):
    """One round of waves over the batch: pass, apply its outputs (W.next_wave), re-submit,
    until no profitable request is left deferred. Each wave's pass (build, then the copy and
    the freed list in one launch; --three-calls: three calls) is replayed `warmup` + `steps`
    times on unchanged inputs (the same plan and the same rows
    between the same addresses each time) with HIP events on the launch stream; then its
    outputs are read back and applied."""
    import numpy as np
    import torch
    from paper_2608_13263_amd import binding as B
    from paper_2608_13263_amd import workloads as W
    sh = inp.shape
    S = sh.block_size
    first = inp
    waves = []
    for wave in range(64):
        batch = B.Batch.from_inputs(inp)
        plan = B.Plan.allocate(batch, S)
        three = separate_free(args)

        def step(ev=None):
            if ev is not None:
                ev[0].record(stream)
            B.build_token_table(cache, batch, plan, stream)
            if ev is not None:
                ev[1].record(stream)
            if three:
                B.repack_ex(cache, batch, plan, args.variant, args.grid, args.order, stream)
            else:
                B.repack_free(cache, batch, plan, stream=stream)
            if ev is not None:
                ev[2].record(stream)
            if three:
                B.free_blocks(batch, plan, stream=stream)
            if ev is not None:
                ev[3].record(stream)

        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()
        evs = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(4))
               for _ in range(args.steps)]
        # the wave's passes with nothing between the calls, then as many again with events
        # between them for the per-call breakdown
        t0 = time.perf_counter()
        for i in range(args.steps):
            step()
        torch.cuda.synchronize()
        wall = (time.perf_counter() - t0) * 1e3 / args.steps
        for i in range(args.steps):
            step(evs[i])
        torch.cuda.synchronize()
        cnt = plan.counters.cpu().tolist()
        if cnt[3] != 0:
            raise SystemExit(f"wave {wave}: device status {B.STATUS.get(cnt[3], cnt[3])}")
        R = inp.num_reqs
        adm = plan.admitted[:R].cpu().numpy()
        live = plan.live_count[:R].cpu().numpy().astype(np.int64)
        nbi = plan.new_bt_indptr[:R + 1].cpu().numpy()
        nbids = plan.new_block_ids[:int(nbi[-1])].cpu().numpy()
        freed = plan.freed[:cnt[2]].cpu().numpy()
        m = np.diff(inp.bt_indptr.astype(np.int64))
        profitable = -(-live // S) < m
        moved = int((live * adm).sum())
        waves.append(dict(
            admitted=cnt[1], deferred=int((profitable & (adm == 0)).sum()),
            live_tokens_moved=moved, bytes_alg=2 * moved * sh.token_bytes,
            destinations=cnt[0], freed_blocks=cnt[2], free_list=len(inp.free_list),
            step_ms=round(wall, 4),
            repack_ms=round(sum(e[1].elapsed_time(e[2]) for e in evs) / args.steps, 4),
            build_ms=round(sum(e[0].elapsed_time(e[1]) for e in evs) / args.steps, 4),
            free_ms=(round(sum(e[2].elapsed_time(e[3]) for e in evs) / args.steps, 4)
                     if three else None)))
        w = waves[-1]
        log(f"wave {wave}: {w['admitted']} admitted, {w['deferred']} deferred, "
            f"{moved} live tokens, {w['repack_ms']:.3f} ms copy, {w['step_ms']:.3f} ms pass")
        if w["deferred"] == 0:
            break
        if cnt[1] == 0:
            raise SystemExit(f"wave {wave}: requests deferred but none admitted")
        inp = W.next_wave(inp, adm, live, nbi, nbids, cnt[0], freed)
    bytes_alg = sum(w["bytes_alg"] for w in waves)
    moved = sum(w["live_tokens_moved"] for w in waves)
    step_ms = sum(w["step_ms"] for w in waves)
    repack_ms = sum(w["repack_ms"] for w in waves)
    value = bytes_alg / (step_ms / 1e3) / 1e9
    achieved = bytes_alg / (repack_ms / 1e3) / 1e9
    ceiling = None
    if args.ceiling != "none":
        ceiling = streaming_ceiling(args, inp, kv, cache, waves[0]["bytes_alg"], stream,
                                    block_copy=False)
    cpu = None
    if not args.no_cpu_baseline:
        log(f"CPU oracle on {args.cpu_planes} planes of the first wave")
        cpu = cpu_baseline(first, args.cpu_planes)
    out = {
        "metric": "repacked KV GB/s (read+write) as % of HBM peak; live tokens repacked/ms",
        "mode": "waves", "value": round(value, 2), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(step_ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "u8",
        "data": "synthetic", "pct_of_hbm_peak": round(100 * value / HBM_PEAK_GBS, 2),
        "live_tokens_per_ms": round(moved / step_ms, 1), "repack_ms": round(repack_ms, 4),
        "config": {"workload": first.name, "recipe": first.note,
                   "round": "one step = every wave of the round (pass, outputs applied, "
                            "re-submitted) until no request is deferred",
                   "layers": sh.num_layers, "kv_heads": sh.num_kv_heads,
                   "head_dim": sh.head_dim, "block_size": S, "kv_dtype": sh.dtype,
                   "requests": first.num_reqs, "tokens": first.num_tokens,
                   "pool_blocks": first.num_blocks,
                   "pool_gib": round(first.pool_bytes() / 2 ** 30, 2),
                   "live_tokens_repacked": moved, "bytes_alg_per_step": bytes_alg,
                   "waves": waves, "inputs_sha256": inputs_sha256(first)},
        "roofline": {"bound": "hbm", "kernel": "repack_direct_kernel",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                     "practical_ceiling": (ceiling or {}).get("probe_copy_GBps"),
                     "frac_of_practical_ceiling":
                         round(achieved / ceiling["probe_copy_GBps"], 4)
                         if ceiling and ceiling.get("probe_copy_GBps") else None},
        "ceiling": ceiling, "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)
    return 0


def run_inplace(args, inp, kv, cache, batch, plan, stream):
    """In-place mode. The pass is re-run on the same inputs: every step computes the same
    plan and moves the same rows between the same addresses (after the first step the bytes
    it moves are ones it already moved, which does not change the traffic)."""
    import numpy as np
    import torch
    from paper_2608_13263_amd import binding as B
    sh = inp.shape
    S = sh.block_size

    def step(ev=None):
        B.build_token_table_inplace(cache, batch, plan, stream)
        if ev is not None:
            ev[0].record(stream)
        B.repack_inplace_ex(cache, batch, plan, args.variant, stream)
        if ev is not None:
            ev[1].record(stream)
        B.free_blocks(batch, plan, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    step_ms = (time.perf_counter() - t0) * 1e3 / args.steps
    kern = sum(a.elapsed_time(b) for a, b in evs) / args.steps
    cnt = plan.counters.cpu().tolist()
    if cnt[3] != 0:
        raise SystemExit(f"device status {B.STATUS.get(cnt[3], cnt[3])}")
    # rows that move: live tokens of repacked requests whose slot changes
    old_slot = np.empty(inp.num_tokens, dtype=np.int64)
    for r in range(inp.num_reqs):
        a, n = int(inp.tok_indptr[r]), int(inp.seq_lens[r])
        bt = inp.block_ids[inp.bt_indptr[r]:inp.bt_indptr[r + 1]].astype(np.int64)
        pos = np.arange(n)
        old_slot[a:a + n] = bt[pos // S] * S + pos % S
    ts = plan.token_slot[:inp.num_tokens].cpu().numpy().astype(np.int64)
    moved = int(((ts != old_slot) & (inp.live != 0)).sum())
    R = inp.num_reqs
    repacked = int((plan.live_count[:R].long() * plan.admitted[:R].long()).sum())
    bytes_alg = 2 * moved * sh.token_bytes
    pipelined = sh.block_size <= 64 and args.variant in (0, 4)
    inplace_kernel = "repack_inplace_pipe_kernel" if pipelined else "repack_inplace_kernel"
    out = {
        "metric": "repacked KV GB/s (read+write) as % of HBM peak; live tokens repacked/ms",
        "mode": "inplace", "value": round(bytes_alg / (step_ms / 1e3) / 1e9, 2), "unit": "GB/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(step_ms, 4),
        "pct_of_hbm_peak": round(100 * bytes_alg / (step_ms / 1e3) / 1e9 / HBM_PEAK_GBS, 2),
        "live_tokens_per_ms": round(repacked / step_ms, 1), "repack_ms": round(kern, 4),
        "config": {"workload": inp.name, "recipe": inp.note, "live_tokens_repacked": repacked,
                   "rows_moved": moved, "rows_in_place": repacked - moved,
                   "pool_gib": round(inp.pool_bytes() / 2 ** 30, 2),
                   "bytes_alg_per_step": bytes_alg, "admitted": cnt[1], "freed_blocks": cnt[2]},
        "roofline": {"bound": "hbm", "kernel": inplace_kernel,
                     "achieved": round(bytes_alg / (kern / 1e3) / 1e9, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s",
                     "frac": round(bytes_alg / (kern / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
                     "traffic": recorded_traffic(inplace_kernel, inp.name, bytes_alg)},
        "cpu_baseline": None if args.no_cpu_baseline else
        cpu_baseline(inp, args.cpu_planes, inplace=True),
    }
    print(json.dumps(out), flush=True)
    return 0


def run_decode(args, inp, kv, cache, batch, plan, stream):
    """Consumer side: decode attention of every layer for every request, reading the live
    K/V rows through the slot mapping. Timed on the layout before the repack (slots in the
    requests' original blocks) and after it (the repacked blocks), same bytes either way:
    each live token's head row of K and V, per layer."""
    import numpy as np
    import torch
    from paper_2608_13263_amd import binding as B
    sh = inp.shape
    S = sh.block_size
    R, Hq, D = inp.num_reqs, args.q_heads, sh.head_dim
    old_indptr, old_slots = [0], []
    for r in range(R):
        a = int(inp.tok_indptr[r])
        bt = inp.block_ids[inp.bt_indptr[r]:inp.bt_indptr[r + 1]].astype(np.int64)
        pos = np.nonzero(inp.live[a:a + int(inp.seq_lens[r])])[0]
        old_slots.extend((bt[pos // S] * S + pos % S).tolist())
        old_indptr.append(len(old_slots))
    dev = lambda x: torch.from_numpy(np.asarray(x, dtype=np.int32)).cuda()  # noqa: E731
    layouts = {"before_repack": (dev(old_indptr), dev(old_slots))}
    B.run_pass(cache, batch, plan, stream=stream)
    layouts["after_repack"] = B.build_slot_mapping(batch, plan, stream=stream)
    torch.cuda.synchronize()
    live = np.diff(np.asarray(old_indptr))
    max_tokens = int(live.max())
    q = torch.randn(R, Hq, D, device="cuda")
    out = torch.empty_like(q)
    ws = torch.empty(B.decode_workspace_bytes(R, Hq, D, max_tokens) // 4, dtype=torch.float32,
                     device="cuda")
    bytes_layer = int(live.sum()) * 2 * sh.num_kv_heads * D * sh.elem_bytes
    bytes_step = bytes_layer * sh.num_layers
    res = {}
    for name, (indptr, slots) in layouts.items():
        def step(ev=None):
            for layer in range(sh.num_layers):
                if ev is not None:
                    ev[layer][0].record(stream)
                B.paged_decode(cache, q, indptr, slots, layer, max_tokens, out=out,
                               workspace=ws, stream=stream)
                if ev is not None:
                    ev[layer][1].record(stream)
        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()
        evs = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                for _ in range(sh.num_layers)] for _ in range(args.steps)]
        t0 = time.perf_counter()
        for i in range(args.steps):
            step(evs[i])
        torch.cuda.synchronize()
        step_ms = (time.perf_counter() - t0) * 1e3 / args.steps
        call_ms = sum(a.elapsed_time(b) for e in evs for a, b in e) / (args.steps * sh.num_layers)
        res[name] = dict(step_ms=step_ms, call_ms=call_ms,
                         gbs=bytes_step / (step_ms / 1e3) / 1e9,
                         call_gbs=bytes_layer / (call_ms / 1e3) / 1e9)
        log(f"decode {name}: step {step_ms:.3f} ms ({res[name]['gbs']:.0f} GB/s), per layer "
            f"{call_ms * 1e3:.1f} us ({res[name]['call_gbs']:.0f} GB/s)")
        if args.graph and name == "after_repack":
            # the whole decode step (every layer) captured once and replayed
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                for layer in range(sh.num_layers):
                    B.paged_decode(cache, q, indptr, slots, layer, max_tokens, out=out,
                                   workspace=ws)
            for _ in range(max(args.warmup, 1)):
                graph.replay()
            torch.cuda.synchronize()
            g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            g0.record()
            for _ in range(args.steps):
                graph.replay()
            g1.record()
            torch.cuda.synchronize()
            gms = g0.elapsed_time(g1) / args.steps
            res[name]["graph_step_ms"] = gms
            res[name]["graph_gbs"] = bytes_step / (gms / 1e3) / 1e9
            log(f"decode {name} from a HIP graph: step {gms:.3f} ms "
                f"({res[name]['graph_gbs']:.0f} GB/s)")
    after = res["after_repack"]
    out_json = {
        "metric": "paged decode K/V GB/s through the slot mapping (all layers, all requests)",
        "mode": "decode", "value": round(after["gbs"], 2), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(after["step_ms"], 4),
        "higher_is_better": True, "dtype": "f32",
        "config": {"workload": inp.name, "recipe": inp.note, "q_heads": Hq,
                   "live_tokens": int(live.sum()), "max_live_tokens": max_tokens,
                   "bytes_alg_per_layer": bytes_layer,
                   "admitted": int(plan.counters[1])},
        "before_repack": {k: round(v, 4) for k, v in res["before_repack"].items()},
        "after_repack": {k: round(v, 4) for k, v in after.items()},
        "roofline": {"bound": "hbm", "kernel": "vtoken_paged_decode (split + combine)",
                     "achieved": round(after["call_gbs"], 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(after["call_gbs"] / HBM_PEAK_GBS, 4),
                     "traffic": recorded_traffic("vtoken_paged_decode", f"{inp.name}_q{Hq}",
                                                 bytes_layer)},
        "cpu_baseline": None if args.no_cpu_baseline else cpu_baseline_decode(
            inp, plan.token_slot[:inp.num_tokens].cpu().numpy(), Hq),
    }
    print(json.dumps(out_json), flush=True)
    return 0


def run_overlap(args, inp, kv, cache, batch, plan, stream):
    """The paper's relocation schedule (Sec. 3.3.4): the copy runs on its own stream beside
    attention, which keeps reading the old slots (out of place, the sources are never
    written, I3), and the next decode step waits for an event recorded after the pass. Times
    one decode step over every layer and one repack pass, one after the other on one stream
    and concurrently on two, with HIP events; HBM is shared, so the overlap gains only what
    neither saturates."""
    import numpy as np
    import torch
    from paper_2608_13263_amd import binding as B
    sh = inp.shape
    S = sh.block_size
    R, Hq, D = inp.num_reqs, args.q_heads, sh.head_dim
    old_indptr, old_slots = [0], []
    for r in range(R):
        a = int(inp.tok_indptr[r])
        bt = inp.block_ids[inp.bt_indptr[r]:inp.bt_indptr[r + 1]].astype(np.int64)
        pos = np.nonzero(inp.live[a:a + int(inp.seq_lens[r])])[0]
        old_slots.extend((bt[pos // S] * S + pos % S).tolist())
        old_indptr.append(len(old_slots))
    dev = lambda x: torch.from_numpy(np.asarray(x, dtype=np.int32)).cuda()  # noqa: E731
    indptr, slots = dev(old_indptr), dev(old_slots)
    live = np.diff(np.asarray(old_indptr))
    max_tokens = int(live.max())
    q = torch.randn(R, Hq, D, device="cuda")
    out = torch.empty_like(q)
    ws = torch.empty(B.decode_workspace_bytes(R, Hq, D, max_tokens) // 4, dtype=torch.float32,
                     device="cuda")
    reloc = torch.cuda.Stream()

    def decode_step(st):
        for layer in range(sh.num_layers):
            B.paged_decode(cache, q, indptr, slots, layer, max_tokens, out=out, workspace=ws,
                           stream=st)

    def repack_pass(st):
        B.build_token_table(cache, batch, plan, st)
        B.repack_free(cache, batch, plan, stream=st)

    def timed(fn):
        times = []
        for i in range(args.warmup + args.steps):
            torch.cuda.synchronize()
            t0 = torch.cuda.Event(enable_timing=True)
            t1 = torch.cuda.Event(enable_timing=True)
            t0.record(stream)
            fn()
            t1.record(stream)
            torch.cuda.synchronize()
            if i >= args.warmup:
                times.append(t0.elapsed_time(t1))
        return sum(times) / len(times)

    def concurrent():
        reloc.wait_stream(stream)
        repack_pass(reloc)
        decode_step(stream)
        done = torch.cuda.Event()
        done.record(reloc)
        stream.wait_event(done)        # the next decode step would read the new slots

    decode_ms = timed(lambda: decode_step(stream))
    repack_ms = timed(lambda: repack_pass(stream))
    serial_ms = timed(lambda: (decode_step(stream), repack_pass(stream)))
    overlap_ms = timed(concurrent)

    # decode latency under a concurrent copy: the copy (its grid capped at `cap` workgroups,
    # a grid-stride loop covering the rest) starts on the relocation stream, the decode step
    # on the main stream right after; events on both streams time each one and the pair
    def under_copy(cap):
        B.build_token_table(cache, batch, plan, reloc)
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        alone = []
        for i in range(args.warmup + args.steps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(reloc)
            B.repack_ex(cache, batch, plan, 0, cap, 0, reloc)
            b.record(reloc)
            torch.cuda.synchronize()
            if i >= args.warmup:
                alone.append(a.elapsed_time(b))
        dec, cop, both = [], [], []
        for i in range(args.warmup + args.steps):
            torch.cuda.synchronize()
            ev[0].record(reloc)
            B.repack_ex(cache, batch, plan, 0, cap, 0, reloc)
            ev[1].record(reloc)
            ev[2].record(stream)
            decode_step(stream)
            ev[3].record(stream)
            torch.cuda.synchronize()
            if i >= args.warmup:
                dec.append(ev[2].elapsed_time(ev[3]))
                cop.append(ev[0].elapsed_time(ev[1]))
                both.append(max(ev[0].elapsed_time(ev[1]), ev[0].elapsed_time(ev[3])))
        mean = lambda x: sum(x) / len(x)  # noqa: E731
        return {"grid_cap": cap or 1 << 19, "copy_alone_ms": round(mean(alone), 4),
                "decode_alone_ms": round(decode_ms, 4),
                "decode_with_copy_ms": round(mean(dec), 4),
                "copy_with_decode_ms": round(mean(cop), 4),
                "together_ms": round(mean(both), 4),
                "decode_slowdown": round(mean(dec) / decode_ms, 3),
                "copy_slowdown": round(mean(cop) / mean(alone), 3)}

    caps = [0, 1 << 15, 1 << 12, 1 << 10, 1 << 8]
    sweep = [under_copy(c) for c in caps]
    for row in sweep:
        log(f"copy grid cap {row['grid_cap']}: copy alone {row['copy_alone_ms']:.3f} ms, decode "
            f"{row['decode_alone_ms']:.3f} -> {row['decode_with_copy_ms']:.3f} ms beside the "
            f"copy ({row['copy_with_decode_ms']:.3f} ms), both {row['together_ms']:.3f} ms")
    cnt = plan.counters.cpu().tolist()
    if cnt[3] != 0:
        raise SystemExit(f"device status {B.STATUS.get(cnt[3], cnt[3])}")
    dec_bytes = int(live.sum()) * 2 * sh.num_kv_heads * D * sh.elem_bytes * sh.num_layers
    moved = int((plan.live_count[:R].long() * plan.admitted[:R].long()).sum())
    rep_bytes = 2 * moved * sh.token_bytes
    total = dec_bytes + rep_bytes
    res = {
        "metric": "decode step + repack pass: HBM GB/s with the copy on a relocation stream",
        "mode": "overlap", "value": round(total / (overlap_ms / 1e3) / 1e9, 1), "unit": "GB/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(overlap_ms, 4), "higher_is_better": True, "data": "synthetic",
        "config": {"workload": inp.name, "recipe": inp.note, "q_heads": Hq,
                   "decode_bytes": dec_bytes, "repack_bytes": rep_bytes},
        "decode_ms": round(decode_ms, 4), "repack_ms": round(repack_ms, 4),
        "serial_ms": round(serial_ms, 4), "overlap_ms": round(overlap_ms, 4),
        "serial_GBps": round(total / (serial_ms / 1e3) / 1e9, 1),
        "overlap_saving": round(1 - overlap_ms / serial_ms, 4),
        "decode_under_copy": sweep,
        "roofline": {"bound": "hbm", "kernel": "decode split + combine and repack_direct_kernel",
                     "achieved": round(total / (overlap_ms / 1e3) / 1e9, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(total / (overlap_ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
                     "traffic": None},
        "cpu_baseline": None,
    }
    log(f"overlap: decode {decode_ms:.3f} ms, repack {repack_ms:.3f} ms, serial "
        f"{serial_ms:.3f} ms, concurrent {overlap_ms:.3f} ms")
    print(json.dumps(res), flush=True)
    return 0


def main(argv=None):
    args = parse_args(argv)
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the repack shards by request (each GPU owns "
              f"its requests and its block pool) with no cross-GPU traffic, so there is no "
              f"multi-GPU path to time; got --gpus {args.gpus}", file=sys.stderr)
        return 2
    import torch
    from paper_2608_13263_amd import binding as B
    B.load_library()
    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU (MI355X, gfx950)")
    if args.mode == "copy":
        return run_copy(args)
    if args.mode == "stream":
        return run_stream(args)
    if args.mode == "placement":
        return run_placement(args)
    if args.mode == "plan":
        return run_plan(args)
    if args.config == "llama3_8b_scissorhands":
        return run_partial_stream(args) if args.partial else run_scissorhands(args)
    if args.config == "llama3_8b_shared_prefix":
        return run_partial_pass(args)

    t_setup = time.perf_counter()
    inp = make_workload(args)
    from paper_2608_13263_amd import workloads as W
    sh = inp.shape
    log(f"{inp.name}: {inp.num_reqs} requests, {inp.num_tokens} tokens, pool "
        f"{inp.num_blocks} blocks = {inp.pool_bytes() / 2**30:.1f} GiB")
    kv = W.kv_device(sh, inp.num_blocks, 1)
    cache = B.KVCache(kv, sh.num_layers, sh.num_kv_heads, sh.head_dim, sh.block_size)
    batch = B.Batch.from_inputs(inp)
    plan = B.Plan.allocate(batch, sh.block_size, inplace=args.inplace)
    stream = torch.cuda.current_stream()
    if args.inplace:
        return run_inplace(args, inp, kv, cache, batch, plan, stream)
    if args.mode == "decode":
        return run_decode(args, inp, kv, cache, batch, plan, stream)
    if args.mode == "overlap":
        return run_overlap(args, inp, kv, cache, batch, plan, stream)
    if args.config == "llama3_70b_h2o":
        return run_waves(args, inp, kv, cache, stream)
    torch.cuda.synchronize()
    log(f"setup {time.perf_counter() - t_setup:.1f} s; warmup {args.warmup} steps")

    three = separate_free(args)

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        B.build_token_table(cache, batch, plan, stream)
        if ev is not None:
            ev[1].record(stream)
        if three:
            B.repack_ex(cache, batch, plan, args.variant, args.grid, args.order, stream)
        else:
            B.repack_free(cache, batch, plan, stream=stream)
        if ev is not None:
            ev[2].record(stream)
        if three:
            B.free_blocks(batch, plan, stream=stream)
        if ev is not None:
            ev[3].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(4))
           for _ in range(args.steps)]
    log(f"timing {args.steps} steps")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    # the per-call breakdown: as many steps again with events between the calls (outside the
    # timed region, so the events do not add to ms_per_step)
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    graph_ms = timed_graph(args, cache, batch, plan) if args.graph else None
    repack_ms = [e[1].elapsed_time(e[2]) for e in evs]
    repack_avg = sum(repack_ms) / len(repack_ms)
    build_ms = sum(e[0].elapsed_time(e[1]) for e in evs) / len(evs)
    free_ms = sum(e[2].elapsed_time(e[3]) for e in evs) / len(evs)

    counters = plan.counters.cpu().tolist()
    if counters[3] != 0:
        raise SystemExit(f"device status {B.STATUS.get(counters[3], counters[3])}")
    R = inp.num_reqs
    live = plan.live_count[:R].to(torch.int64)
    adm = plan.admitted[:R].to(torch.int64)
    moved_tokens = int((live * adm).sum().item())
    bytes_alg = 2 * moved_tokens * sh.token_bytes
    value = bytes_alg / (ms_per_step / 1e3) / 1e9
    achieved = bytes_alg / (repack_avg / 1e3) / 1e9
    traffic = recorded_traffic("repack_direct_kernel", inp.name, bytes_alg)
    log(f"step {ms_per_step:.3f} ms, repack {repack_avg:.3f} ms "
        f"(min {min(repack_ms):.3f}), {achieved:.0f} GB/s repack")

    ceiling = None
    if args.ceiling != "none":
        ceiling = streaming_ceiling(args, inp, kv, cache, bytes_alg, stream,
                                    block_copy=args.ceiling == "all")

    cpu = None
    if not args.no_cpu_baseline:
        log(f"CPU oracle on {args.cpu_planes} planes")
        cpu = cpu_baseline(inp, args.cpu_planes)

    out = {
        "metric": "repacked KV GB/s (read+write) as % of HBM peak; live tokens repacked/ms",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8",
        "data": "synthetic",
        "pct_of_hbm_peak": round(100 * value / HBM_PEAK_GBS, 2),
        "live_tokens_per_ms": round(moved_tokens / ms_per_step, 1),
        "repack_ms": round(repack_avg, 4),
        "repack_ms_median": round(statistics.median(repack_ms), 4),
        "repack_ms_min": round(min(repack_ms), 4),
        "graph_ms_per_step": round(graph_ms, 4) if graph_ms is not None else None,
        "build_token_table_ms": round(build_ms, 4),
        "free_blocks_ms": round(free_ms, 4) if three else None,
        "pass_calls": ("vtoken_build_token_table, vtoken_repack_ex, vtoken_free_blocks" if three
                       else "vtoken_build_token_table, vtoken_repack_free (copy and freed "
                            "list in one launch)"),
        "config": {
            "workload": inp.name,
            "recipe": inp.note,
            "layers": sh.num_layers, "kv_heads": sh.num_kv_heads, "head_dim": sh.head_dim,
            "block_size": sh.block_size, "kv_dtype": sh.dtype, "requests": inp.num_reqs,
            "tokens": inp.num_tokens, "live_tokens_repacked": moved_tokens,
            "pool_blocks": inp.num_blocks, "pool_gib": round(inp.pool_bytes() / 2 ** 30, 2),
            "used_blocks": counters[0], "admitted": counters[1], "freed_blocks": counters[2],
            "bytes_alg_per_step": bytes_alg, "variant": args.variant, "grid": args.grid,
            "order": args.order, "inputs_sha256": inputs_sha256(inp),
        },
        "roofline": {
            "bound": "hbm", "kernel": "repack_direct_kernel",
            "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": traffic,
            "practical_ceiling": (ceiling or {}).get("probe_copy_GBps"),
            "frac_of_practical_ceiling": round(achieved / ceiling["probe_copy_GBps"], 4)
            if ceiling and ceiling.get("probe_copy_GBps") else None,
        },
        "ceiling": ceiling,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
