"""The C-ABI library on a host without a GPU: it loads, exports every function that
include/vtoken.h declares, and its host-side argument checks return the documented status
codes before any device work (no compute call is made here)."""
import ctypes
import os
import re

import pytest

from paper_2608_13263_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "vtoken.h")

pytestmark = pytest.mark.skipif(not os.path.exists(B.LIB_PATH),
                                reason="libvtoken.so not built (run __graft_entry__.build())")


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(vtoken_[a-z_]+)\s*\(", text)))


def header_status_codes():
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    return {m.group(1): int(m.group(2)) for m in re.finditer(r"(VTOKEN_[A-Z_]+)\s*=\s*(-?\d+)", text)}


def test_exports_every_declared_function():
    lib = B.load_library()
    names = header_functions()
    assert {"vtoken_build_token_table", "vtoken_repack", "vtoken_free_blocks"} <= set(names)
    for name in names:
        assert hasattr(lib, name), f"{name} declared in vtoken.h but not exported"
    assert set(names) == set(B._SIGNATURES), "binding signatures out of sync with the header"


def test_status_codes_match_binding():
    codes = header_status_codes()
    assert codes == B.STATUS_CODE
    for name, code in codes.items():
        assert B.status_string(code).startswith(name)
    assert B.status_string(12345) == "unknown vtoken status"
    assert B.load_library().vtoken_version() == 200


def test_struct_layouts_match_header(tmp_path):
    """Field offsets and sizes of the ctypes structs equal what the C compiler lays out
    for include/vtoken.h."""
    import shutil
    import subprocess
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    structs = {"vtoken_cache": B.CCache, "vtoken_batch": B.CBatch, "vtoken_plan": B.CPlan,
               "vtoken_repack_options": B.CRepackOptions, "vtoken_decode": B.CDecode,
               "vtoken_planner_params": B.CPlannerParams,
               "vtoken_planner_state": B.CPlannerState}
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "vtoken.h"', "int main(void){"]
    for cname, cls in structs.items():
        lines.append(f'printf("{cname} sizeof %zu\\n", sizeof({cname}));')
        for fname, _ in cls._fields_:
            lines.append(f'printf("{cname} {fname} %zu\\n", offsetof({cname}, {fname}));')
    lines.append("return 0;}")
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
                    "-I", "/opt/rocm/include", str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout
    got = {}
    for line in out.splitlines():
        cname, field, val = line.split()
        got[(cname, field)] = int(val)
    for cname, cls in structs.items():
        assert got[(cname, "sizeof")] == ctypes.sizeof(cls), cname
        for fname, _ in cls._fields_:
            assert got[(cname, fname)] == getattr(cls, fname).offset, (cname, fname)


def _fake_ptr():
    # a non-NULL host address that host validation only compares against NULL
    return ctypes.cast(ctypes.create_string_buffer(64), ctypes.c_void_p).value


def _good():
    p = _fake_ptr()
    cache = B.CCache(p, 2, 8, 128, 16, 100, 2)
    batch = B.CBatch(2, 40, 4, p, p, p, p, p, p, 10)
    plan = B.CPlan(p, p, p, p, p, p, p, p, p, 4, 4 * 16)
    return cache, batch, plan


@pytest.mark.parametrize("mutate,code", [
    (lambda c, b, p: setattr(c, "kv", None), "VTOKEN_ERR_NULL"),
    (lambda c, b, p: setattr(c, "elem_bytes", 4), "VTOKEN_ERR_SHAPE"),
    (lambda c, b, p: setattr(c, "num_kv_heads", 1) or setattr(c, "head_dim", 4),
     "VTOKEN_ERR_SHAPE"),                                                 # 8-byte rows
    (lambda c, b, p: setattr(c, "num_kv_heads", 1) or setattr(c, "head_dim", 3),
     "VTOKEN_ERR_SHAPE"),                                                 # 6-byte rows
    (lambda c, b, p: setattr(c, "num_blocks", 2 ** 28), "VTOKEN_ERR_SHAPE"),  # slots >= 2^31
    (lambda c, b, p: setattr(c, "block_size", 0), "VTOKEN_ERR_SHAPE"),
    (lambda c, b, p: setattr(b, "num_reqs", -1), "VTOKEN_ERR_SHAPE"),
    (lambda c, b, p: setattr(b, "num_tokens", 2 ** 31), "VTOKEN_ERR_SHAPE"),
    (lambda c, b, p: setattr(b, "tok_indptr", None), "VTOKEN_ERR_NULL"),
    (lambda c, b, p: setattr(b, "live", None), "VTOKEN_ERR_NULL"),
    (lambda c, b, p: setattr(p, "counters", None), "VTOKEN_ERR_NULL"),
    (lambda c, b, p: setattr(p, "src_plan", None), "VTOKEN_ERR_NULL"),
    (lambda c, b, p: setattr(p, "new_bt_capacity", 3), "VTOKEN_ERR_CAPACITY"),
    (lambda c, b, p: setattr(p, "src_plan_capacity", 4 * 16 - 1), "VTOKEN_ERR_CAPACITY"),
])
def test_build_rejects_bad_arguments(mutate, code):
    lib = B.load_library()
    cache, batch, plan = _good()
    mutate(cache, batch, plan)
    st = lib.vtoken_build_token_table(ctypes.byref(cache), ctypes.byref(batch),
                                      ctypes.byref(plan), None)
    assert st == B.STATUS_CODE[code], (st, code)


def test_repack_and_free_reject_bad_arguments():
    lib = B.load_library()
    cache, batch, plan = _good()
    opts = B.CRepackOptions(7, 0, 0, 0)
    assert lib.vtoken_repack_ex(ctypes.byref(cache), ctypes.byref(batch), ctypes.byref(plan),
                                ctypes.byref(opts), None) == B.STATUS_CODE["VTOKEN_ERR_ARGUMENT"]
    opts = B.CRepackOptions(0, 0, 3, 0)
    assert lib.vtoken_repack_ex(ctypes.byref(cache), ctypes.byref(batch), ctypes.byref(plan),
                                ctypes.byref(opts), None) == B.STATUS_CODE["VTOKEN_ERR_ARGUMENT"]
    assert lib.vtoken_repack(None, ctypes.byref(batch), ctypes.byref(plan), None) == \
        B.STATUS_CODE["VTOKEN_ERR_NULL"]
    assert lib.vtoken_free_blocks(ctypes.byref(batch), ctypes.byref(plan), _fake_ptr(), 3,
                                  None) == B.STATUS_CODE["VTOKEN_ERR_CAPACITY"]
    assert lib.vtoken_free_blocks(ctypes.byref(batch), ctypes.byref(plan), None, 4, None) == \
        B.STATUS_CODE["VTOKEN_ERR_NULL"]
    # a batch that cannot have admitted anything returns before any launch
    batch.free_len = 0
    assert lib.vtoken_repack(ctypes.byref(cache), ctypes.byref(batch), ctypes.byref(plan),
                             None) == 0


def test_repack_free_rejects_bad_arguments():
    """The one-launch copy and freed list checks what vtoken_repack and vtoken_free_blocks
    check, before enqueueing anything."""
    lib = B.load_library()
    cache, batch, plan = _good()
    call = lambda c, b, p, freed, cap: lib.vtoken_repack_free(  # noqa: E731
        c, b, p, freed, cap, None)
    C, Bt, P = ctypes.byref(cache), ctypes.byref(batch), ctypes.byref(plan)
    assert call(C, Bt, P, _fake_ptr(), 3) == B.STATUS_CODE["VTOKEN_ERR_CAPACITY"]
    assert call(C, Bt, P, None, 4) == B.STATUS_CODE["VTOKEN_ERR_NULL"]
    assert call(None, Bt, P, _fake_ptr(), 4) == B.STATUS_CODE["VTOKEN_ERR_NULL"]
    assert call(C, None, P, _fake_ptr(), 4) == B.STATUS_CODE["VTOKEN_ERR_NULL"]
    assert call(C, Bt, None, _fake_ptr(), 4) == B.STATUS_CODE["VTOKEN_ERR_NULL"]
    plan.freed_indptr = None
    assert call(C, Bt, P, _fake_ptr(), 4) == B.STATUS_CODE["VTOKEN_ERR_NULL"]


def test_decode_workspace_bytes():
    lib = B.load_library()
    # R * Hq * ceil(max_tokens / (16384 / D)) * (D + 2) float32 partial records, at least one
    assert lib.vtoken_decode_workspace_bytes(3, 32, 128, 1000) == 3 * 32 * 8 * 130 * 4
    assert lib.vtoken_decode_workspace_bytes(3, 32, 128, 1024) == 3 * 32 * 8 * 130 * 4
    assert lib.vtoken_decode_workspace_bytes(3, 32, 128, 1025) == 3 * 32 * 9 * 130 * 4
    assert lib.vtoken_decode_workspace_bytes(2, 8, 64, 0) == 2 * 8 * 1 * 66 * 4
    assert lib.vtoken_decode_workspace_bytes(2, 8, 32, 513) == 2 * 8 * 2 * 34 * 4
    assert lib.vtoken_decode_workspace_bytes(2, 8, 256, 65) == 2 * 8 * 2 * 258 * 4
    assert lib.vtoken_decode_workspace_bytes(2, 0, 64, 10) == -1
    assert lib.vtoken_decode_workspace_bytes(-1, 8, 64, 10) == -1
    assert lib.vtoken_decode_workspace_bytes(2, 8, 96, 10) == -1


def _good_decode(cache, nreq=2, hq=32, max_tokens=700):
    ws = lib_ws = B.load_library().vtoken_decode_workspace_bytes(nreq, hq, cache.head_dim,
                                                                 max_tokens)
    p = _fake_ptr()
    return B.CDecode(p, p, hq, 1, B.KV_BF16, 0.088, max_tokens, p, ws, None), lib_ws


@pytest.mark.parametrize("mutate,code", [
    (lambda c, d: setattr(d, "num_q_heads", 24), "VTOKEN_ERR_SHAPE"),      # G = 3
    (lambda c, d: setattr(d, "num_q_heads", 12), "VTOKEN_ERR_SHAPE"),      # not a multiple
    (lambda c, d: setattr(d, "num_q_heads", 128), "VTOKEN_ERR_SHAPE"),     # G = 16
    (lambda c, d: setattr(d, "layer", 2), "VTOKEN_ERR_SHAPE"),
    (lambda c, d: setattr(d, "layer", -1), "VTOKEN_ERR_SHAPE"),
    (lambda c, d: setattr(d, "kv_dtype", B.KV_FP8_E4M3), "VTOKEN_ERR_SHAPE"),  # 2-byte cache
    (lambda c, d: setattr(d, "kv_dtype", 3), "VTOKEN_ERR_SHAPE"),
    (lambda c, d: setattr(c, "head_dim", 512) or setattr(c, "num_kv_heads", 2),
     "VTOKEN_ERR_SHAPE"),                                                  # head_dim 512
    (lambda c, d: setattr(c, "head_dim", 16) or setattr(c, "num_kv_heads", 64),
     "VTOKEN_ERR_SHAPE"),                                                  # head_dim 16
    (lambda c, d: setattr(d, "workspace_bytes", d.workspace_bytes - 4), "VTOKEN_ERR_CAPACITY"),
    (lambda c, d: setattr(d, "max_tokens", 1100), "VTOKEN_ERR_CAPACITY"),
    (lambda c, d: setattr(d, "q", None), "VTOKEN_ERR_NULL"),
    (lambda c, d: setattr(d, "workspace", None), "VTOKEN_ERR_NULL"),
])
def test_paged_decode_rejects_bad_arguments(mutate, code):
    lib = B.load_library()
    cache, _, _ = _good()
    d, _ = _good_decode(cache)
    mutate(cache, d)
    p = _fake_ptr()
    st = lib.vtoken_paged_decode(ctypes.byref(cache), ctypes.byref(d), 2, p, p, None)
    assert st == B.STATUS_CODE[code], (st, code)


def test_paged_decode_max_tokens_at_int32_limit():
    """A bound within one split of INT32_MAX: the split count is taken in 64 bits, so the
    200 x 8 x 8,388,608-workgroup grid is refused rather than wrapped to a negative size."""
    lib = B.load_library()
    cache, _, _ = _good()
    d, _ = _good_decode(cache, nreq=200)
    d.max_tokens, d.workspace_bytes = 2 ** 31 - 1, 2 ** 62
    assert lib.vtoken_decode_workspace_bytes(200, 32, 128, 2 ** 31 - 1) < 2 ** 62
    p = _fake_ptr()
    assert lib.vtoken_paged_decode(ctypes.byref(cache), ctypes.byref(d), 200, p, p, None) == \
        B.STATUS_CODE["VTOKEN_ERR_SHAPE"]


def test_paged_decode_fp8_kind_requires_one_byte_cache():
    lib = B.load_library()
    cache, _, _ = _good()
    cache.elem_bytes = 1
    d, _ = _good_decode(cache)      # bf16 kind on a 1-byte cache
    p = _fake_ptr()
    assert lib.vtoken_paged_decode(ctypes.byref(cache), ctypes.byref(d), 2, p, p, None) == \
        B.STATUS_CODE["VTOKEN_ERR_SHAPE"]
    # no requests: nothing to do, no launch
    assert lib.vtoken_paged_decode(ctypes.byref(cache), ctypes.byref(d), 0, p, None, None) == 0


def test_slot_mapping_rejects_bad_arguments():
    lib = B.load_library()
    _, batch, plan = _good()
    p = _fake_ptr()
    assert lib.vtoken_build_slot_mapping(ctypes.byref(batch), ctypes.byref(plan), p, p, 39,
                                         None) == B.STATUS_CODE["VTOKEN_ERR_CAPACITY"]
    assert lib.vtoken_build_slot_mapping(ctypes.byref(batch), ctypes.byref(plan), None, p, 40,
                                         None) == B.STATUS_CODE["VTOKEN_ERR_NULL"]
    assert lib.vtoken_build_slot_mapping(ctypes.byref(batch), ctypes.byref(plan), p, None, 40,
                                         None) == B.STATUS_CODE["VTOKEN_ERR_NULL"]
    plan.token_slot = None
    assert lib.vtoken_build_slot_mapping(ctypes.byref(batch), ctypes.byref(plan), p, p, 40,
                                         None) == B.STATUS_CODE["VTOKEN_ERR_NULL"]


def test_plan_partial_rejects_bad_arguments():
    lib = B.load_library()
    cache, batch, plan = _good()
    p = _fake_ptr()
    st = B.CPlannerState(p, p, p, p, p, p, p, p, None)
    good = B.PlannerParams().c()

    def call(c=cache, prm=good, s=st, pl=plan, slot=p):
        return lib.vtoken_plan_partial(ctypes.byref(c), ctypes.byref(batch), slot,
                                       ctypes.byref(prm), ctypes.byref(s), ctypes.byref(pl),
                                       None)
    bad = B.PlannerParams(theta=(1, 0)).c()
    assert call(prm=bad) == B.STATUS_CODE["VTOKEN_ERR_ARGUMENT"]
    bad = B.PlannerParams(max_sources=-1).c()
    assert call(prm=bad) == B.STATUS_CODE["VTOKEN_ERR_ARGUMENT"]
    bad = B.PlannerParams(min_eligible=-2).c()
    assert call(prm=bad) == B.STATUS_CODE["VTOKEN_ERR_ARGUMENT"]
    big = B.CCache(p, 2, 8, 128, 128, 100, 2)          # block_size 128 > 64
    assert call(c=big) == B.STATUS_CODE["VTOKEN_ERR_SHAPE"]
    assert call(slot=None) == B.STATUS_CODE["VTOKEN_ERR_NULL"]
    s2 = B.CPlannerState(p, p, p, p, None, p, p, p, None)
    assert call(s=s2) == B.STATUS_CODE["VTOKEN_ERR_NULL"]
    s3 = B.CPlannerState(p, p, p, p, p, p, p, None, None)
    assert call(s=s3) == B.STATUS_CODE["VTOKEN_ERR_NULL"]
    small = B.CPlan(p, p, p, p, p, p, p, p, p, 3, 4 * 16)
    assert call(pl=small) == B.STATUS_CODE["VTOKEN_ERR_CAPACITY"]
    small = B.CPlan(p, p, p, p, p, p, p, p, p, 4, 4 * 16 - 1)
    assert call(pl=small) == B.STATUS_CODE["VTOKEN_ERR_CAPACITY"]


def test_slot_table_and_append_reject_bad_arguments():
    lib = B.load_library()
    _, batch, plan = _good()
    p = _fake_ptr()
    # capacity must cover num_tokens + num_reqs * reserve (40 + 2 * 5)
    assert lib.vtoken_build_slot_table(ctypes.byref(batch), ctypes.byref(plan), 5, p, p, p, 49,
                                       None) == B.STATUS_CODE["VTOKEN_ERR_CAPACITY"]
    assert lib.vtoken_build_slot_table(ctypes.byref(batch), ctypes.byref(plan), -1, p, p, p,
                                       100, None) == B.STATUS_CODE["VTOKEN_ERR_ARGUMENT"]
    assert lib.vtoken_build_slot_table(ctypes.byref(batch), ctypes.byref(plan), 5, p, None, p,
                                       100, None) == B.STATUS_CODE["VTOKEN_ERR_NULL"]
    assert lib.vtoken_append_slots(-1, p, p, p, p, p, p, None) == \
        B.STATUS_CODE["VTOKEN_ERR_SHAPE"]
    assert lib.vtoken_append_slots(2, p, p, p, p, p, None, None) == \
        B.STATUS_CODE["VTOKEN_ERR_NULL"]
    assert lib.vtoken_append_slots(2, p, None, p, p, p, p, None) == \
        B.STATUS_CODE["VTOKEN_ERR_NULL"]


def test_binding_fails_loudly_without_library(tmp_path):
    with pytest.raises(RuntimeError, match="missing"):
        B.load_library(str(tmp_path / "libvtoken.so"))


def test_no_undefined_library_symbols():
    """Every kernel the library launches is defined in it (a template kernel the host pass
    silently drops would leave an undefined handle that only fails at load time)."""
    import shutil
    import subprocess
    if shutil.which("nm") is None:
        pytest.skip("nm not available")
    out = subprocess.run(["nm", "-D", "--undefined-only", B.LIB_PATH], check=True,
                         capture_output=True, text=True).stdout
    bad = [ln for ln in out.splitlines() if "vtoken" in ln]
    assert not bad, bad


def test_stream_probe_library_rejects_bad_sizes():
    """The memory-system probes of `bench.py` (bench_probe.hip, bench tooling): every entry
    point is exported and refuses null pointers and sizes its kernels do not cover before any
    launch (no device needed)."""
    import bench
    lib = bench.probe_library()
    fake = 1 << 40          # never dereferenced: every call below fails its host checks
    chunk = 32768
    assert lib.vtoken_probe_read(None, chunk, 1, fake, None) == -2
    assert lib.vtoken_probe_read(fake, chunk + 16, 1, fake, None) == -2
    assert lib.vtoken_probe_read(fake, chunk * (1 << 24) + chunk, 1, fake, None) == -2
    assert lib.vtoken_probe_write(fake, 3 * chunk, 2, None) == -2        # ways must divide
    assert lib.vtoken_probe_write(fake, 4 * chunk, 0, None) == -2
    assert lib.vtoken_probe_copy(fake, None, 4 * chunk, 1, None) == -2
    assert lib.vtoken_probe_head_read(fake, 1 << 20, 2000, fake, 64, 1, fake, None) == -2
    assert lib.vtoken_probe_head_read(fake, 1 << 20, 2048, fake, 100, 1, fake, None) == -2
    assert lib.vtoken_probe_head_read(fake, 1024, 2048, fake, 64, 1, fake, None) == -2
    # plane copy: ranges inside the plane, not overlapping, planes and chunks positive
    assert lib.vtoken_probe_plane_copy(None, 8 * chunk, 2, 0, 4, 4, None) == -2
    assert lib.vtoken_probe_plane_copy(fake, 8 * chunk + 16, 2, 0, 4, 4, None) == -2
    assert lib.vtoken_probe_plane_copy(fake, 8 * chunk, 2, 0, 5, 4, None) == -2    # past it
    assert lib.vtoken_probe_plane_copy(fake, 8 * chunk, 2, 0, 3, 4, None) == -2    # overlap
    assert lib.vtoken_probe_plane_copy(fake, 8 * chunk, 0, 0, 4, 4, None) == -2
    assert lib.vtoken_probe_plane_copy(fake, 8 * chunk, 2, 0, 4, 0, None) == -2


def test_check_layout_workspace_bytes_and_bad_arguments():
    lib = B.load_library()
    # a flag word and one bit per block, in 32-bit words
    assert [lib.vtoken_check_layout_workspace_bytes(n) for n in (1, 32, 33, 64, 100)] == \
        [8, 8, 12, 12, 20]
    assert lib.vtoken_check_layout_workspace_bytes(0) == -1
    assert lib.vtoken_check_layout_workspace_bytes(2 ** 31 - 1) == 4 * (1 + 2 ** 26)
    cache, batch, _ = _good()                      # 100 blocks: 20 bytes of workspace
    ws, st = _fake_ptr(), _fake_ptr()
    call = lambda c, w, nbytes, s: lib.vtoken_check_layout(  # noqa: E731
        ctypes.byref(c) if c is not None else None, ctypes.byref(batch), w, nbytes, s, None)
    assert call(cache, ws, 19, st) == B.STATUS_CODE["VTOKEN_ERR_CAPACITY"]
    assert call(cache, None, 20, st) == B.STATUS_CODE["VTOKEN_ERR_NULL"]
    assert call(cache, ws, 20, None) == B.STATUS_CODE["VTOKEN_ERR_NULL"]
    assert call(None, ws, 20, st) == B.STATUS_CODE["VTOKEN_ERR_NULL"]
    cache.block_size = 0
    assert call(cache, ws, 20, st) == B.STATUS_CODE["VTOKEN_ERR_SHAPE"]
    assert lib.vtoken_status_string(-14).decode().startswith("VTOKEN_ERR_LAYOUT")


@pytest.mark.parametrize("mutate,code", [
    (lambda c, d: setattr(d, "num_q_heads", 24), "VTOKEN_ERR_SHAPE"),      # G = 3
    (lambda c, d: setattr(d, "layer", 2), "VTOKEN_ERR_SHAPE"),
    (lambda c, d: setattr(d, "kv_dtype", B.KV_FP8_E4M3), "VTOKEN_ERR_SHAPE"),
    (lambda c, d: setattr(d, "q", None), "VTOKEN_ERR_NULL"),
    (lambda c, d: setattr(d, "out", None), "VTOKEN_ERR_NULL"),
    # partials beyond the library-held array: 2 requests x 32 heads x 2344 splits x 130 x 4 B
    (lambda c, d: setattr(d, "max_tokens", 300000), "VTOKEN_ERR_CAPACITY"),
])
def test_paged_decode_noalloc_rejects_bad_arguments(mutate, code):
    """The allocation-free decode checks its arguments like vtoken_paged_decode, ignores the
    caller workspace fields, and refuses a call whose partials exceed the library-held array
    (VTOKEN_DECODE_SCRATCH_BYTES) before touching the device."""
    lib = B.load_library()
    cache, _, _ = _good()
    d, _ = _good_decode(cache)
    d.workspace, d.workspace_bytes = None, 0       # ignored by this entry point
    mutate(cache, d)
    p = _fake_ptr()
    st = lib.vtoken_paged_decode_noalloc(ctypes.byref(cache), ctypes.byref(d), 2, p, p, None)
    assert st == B.STATUS_CODE[code], (st, code)
    limit = lib.vtoken_decode_workspace_bytes(2, 32, 128, 300000)
    assert limit > B.DECODE_SCRATCH_BYTES >= lib.vtoken_decode_workspace_bytes(2, 32, 128, 250000)


def test_header_scratch_size_matches_binding():
    text = open(HEADER).read()
    m = re.search(r"#define VTOKEN_DECODE_SCRATCH_BYTES \((\d+)LL << (\d+)\)", text)
    assert m and int(m.group(1)) << int(m.group(2)) == B.DECODE_SCRATCH_BYTES


def test_build_id_is_the_hash_of_the_sources():
    """The loaded library carries the SHA-256 of the tree's csrc/ and include/vtoken.h (paths
    relative to the repository root in sorted order, each hashed as path, NUL, contents,
    NUL), recomputed here without the build script."""
    import hashlib
    csrc = os.path.join(ROOT, "paper_2608_13263_amd", "csrc")
    paths = [os.path.join("paper_2608_13263_amd", "csrc", f) for f in os.listdir(csrc)
             if f.endswith((".hip", ".h"))] + [os.path.join("include", "vtoken.h")]
    h = hashlib.sha256()
    for rel in sorted(paths):
        h.update(rel.encode() + b"\0" + open(os.path.join(ROOT, rel), "rb").read() + b"\0")
    assert B.load_library().vtoken_build_id().decode() == h.hexdigest()


def test_binding_refuses_a_library_of_other_sources(tmp_path, monkeypatch):
    """A library whose build id is not the tree's hash is refused at load time."""
    from paper_2608_13263_amd import build as Bld
    monkeypatch.setattr(Bld, "source_sha256", lambda: "0" * 64)
    monkeypatch.setattr(B, "_lib", None)
    with pytest.raises(RuntimeError, match="other sources"):
        B.load_library()


def test_binding_reuses_structs_until_an_attribute_changes():
    """The binding builds each object's C struct once (host overhead of small passes) and
    rebuilds it after any attribute is assigned, so a replaced buffer is never passed stale."""
    import torch
    t = lambda n: torch.zeros(n, dtype=torch.int32)  # noqa: E731
    batch = B.Batch(t(2), t(3), t(3), t(4), torch.zeros(5, dtype=torch.uint8), t(6))
    first = batch.c()
    assert batch.c() is first
    batch.free_list = t(9)
    second = batch.c()
    assert second is not first and second.free_list == batch.free_list.data_ptr()
    assert second.free_len == 6      # sizes are the constructor's; replacing a buffer keeps them
    plan = B.Plan(**{k: t(4) for k in B.Plan.FIELDS + ("freed",)})
    p1 = plan.c()
    plan.counters = t(5)
    assert plan.c() is not p1 and plan.c().counters == plan.counters.data_ptr()
