"""The memory-system probes of `bench.py` (bench_probe.hip, built on demand) do the work
their rates are counted on: the copy reproduces its source in both work orders, the write
fills every chunk with its (thread, workgroup) pattern, and the read kernels leave their
sink untouched on zero-filled input. Small buffers (64 MiB), the same kernels and
arguments as the benchmark."""
import ctypes

import numpy as np
import pytest

from gpu_helpers import torch

pytestmark = pytest.mark.gpu

CHUNK = 32768


def _lib():
    import bench
    return bench.probe_library()


def _stream():
    t = torch()
    return ctypes.c_void_p(t.cuda.current_stream().cuda_stream)


@pytest.mark.parametrize("ways", [1, 64])
def test_copy_probe_copies(ways):
    t = torch()
    lib = _lib()
    n = 64 << 20
    print(f"[gpu] stream probe copy ways={ways}", flush=True)
    g = t.Generator(device="cuda").manual_seed(ways)
    src = t.randint(0, 256, (n,), dtype=t.uint8, device="cuda", generator=g)
    dst = t.zeros(n, dtype=t.uint8, device="cuda")
    assert lib.vtoken_probe_copy(src.data_ptr(), dst.data_ptr(), n, ways, _stream()) == 0
    t.cuda.synchronize()
    assert t.equal(src, dst)


@pytest.mark.parametrize("ways", [1, 64])
def test_write_probe_writes_every_chunk(ways):
    t = torch()
    lib = _lib()
    n = 64 << 20
    chunks = n // CHUNK
    print(f"[gpu] stream probe write ways={ways}", flush=True)
    buf = t.full((n,), 0xAB, dtype=t.uint8, device="cuda")
    assert lib.vtoken_probe_write(buf.data_ptr(), n, ways, _stream()) == 0
    t.cuda.synchronize()
    words = buf.view(t.int32).view(chunks, 8, 256, 4).cpu().numpy()
    # workgroup w writes chunk (w % ways) * (chunks / ways) + w / ways; every 16-byte unit
    # holds (thread, workgroup, 0, 0)
    w = np.arange(chunks)
    c = (w % ways) * (chunks // ways) + w // ways
    expect_wg = np.empty(chunks, np.int64)
    expect_wg[c] = w
    assert (words[:, :, :, 0] == np.arange(256)[None, None, :]).all()
    assert (words[:, :, :, 1] == expect_wg[:, None, None]).all()
    assert (words[:, :, :, 2:] == 0).all()


def test_read_probes_leave_the_sink_alone():
    t = torch()
    lib = _lib()
    n = 64 << 20
    print("[gpu] stream probe reads", flush=True)
    buf = t.zeros(n, dtype=t.uint8, device="cuda")
    sink = t.full((1,), 7, dtype=t.int32, device="cuda")
    for nt in (0, 1):
        assert lib.vtoken_probe_read(buf.data_ptr(), n, nt, sink.data_ptr(), _stream()) == 0
    plane = n // 2
    rows = plane // 2048
    slots = t.randperm(rows, device="cuda").to(t.int32)
    for nt in (0, 1):
        assert lib.vtoken_probe_head_read(buf.data_ptr(), plane, 2048, slots.data_ptr(),
                                          rows, nt, sink.data_ptr(), _stream()) == 0
    t.cuda.synchronize()
    assert int(sink.item()) == 7


def test_plane_copy_probe_copies_in_every_plane():
    """The ceiling probe of the bench line copies chunks [src0, src0 + n) to [dst0, dst0 + n) in
    every plane and touches nothing else."""
    t = torch()
    lib = _lib()
    planes, per_plane = 6, 64
    print("[gpu] stream probe plane copy", flush=True)
    g = t.Generator(device="cuda").manual_seed(9)
    buf = t.randint(0, 256, (planes, per_plane, CHUNK), dtype=t.uint8, device="cuda",
                    generator=g)
    before = buf.clone()
    assert lib.vtoken_probe_plane_copy(buf.data_ptr(), per_plane * CHUNK, planes, 3, 40, 20,
                                       _stream()) == 0
    t.cuda.synchronize()
    expect = before.clone()
    expect[:, 40:60] = before[:, 3:23]
    assert t.equal(buf, expect)
