"""ctypes binding of libvtoken.so (include/vtoken.h): argument marshalling only.

Every step of the repack runs in the library's HIP kernels; this module turns torch device
tensors into the C structs, passes the current HIP stream and raises on a negative status.
It never falls back to another implementation: without the built library, or without a
GPU, the calls raise.

    cache = KVCache(kv_tensor, num_layers, num_kv_heads, head_dim, block_size)
    batch = Batch.from_host(seq_lens, tok_indptr, bt_indptr, block_ids, live, free_list)
    plan  = Plan.allocate(batch, block_size)
    build_token_table(cache, batch, plan)
    repack(cache, batch, plan)
    free_blocks(batch, plan)             # plan.freed[:plan.counters[2]]
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libvtoken.so")

VTOKEN_OK = 0
STATUS = {
    0: "VTOKEN_OK", -1: "VTOKEN_ERR_NULL", -2: "VTOKEN_ERR_SHAPE", -3: "VTOKEN_ERR_CAPACITY",
    -4: "VTOKEN_ERR_HIP", -5: "VTOKEN_ERR_ARGUMENT", -10: "VTOKEN_ERR_BLOCK_RANGE",
    -11: "VTOKEN_ERR_BT_LEN", -12: "VTOKEN_ERR_TOK_LEN", -13: "VTOKEN_ERR_SLOT",
    -14: "VTOKEN_ERR_LAYOUT", -15: "VTOKEN_ERR_PLAN_MODE",
}
STATUS_CODE = {v: k for k, v in STATUS.items()}


class VTokenError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {STATUS.get(status, status)}")
        self.status = status


class CCache(ctypes.Structure):
    _fields_ = [("kv", ctypes.c_void_p), ("num_layers", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("block_size", ctypes.c_int32), ("num_blocks", ctypes.c_int32),
                ("elem_bytes", ctypes.c_int32)]


class CBatch(ctypes.Structure):
    _fields_ = [("num_reqs", ctypes.c_int32), ("num_tokens", ctypes.c_int64),
                ("num_bt_entries", ctypes.c_int64), ("seq_lens", ctypes.c_void_p),
                ("tok_indptr", ctypes.c_void_p), ("bt_indptr", ctypes.c_void_p),
                ("block_ids", ctypes.c_void_p), ("live", ctypes.c_void_p),
                ("free_list", ctypes.c_void_p), ("free_len", ctypes.c_int32)]


class CPlan(ctypes.Structure):
    _fields_ = [("token_slot", ctypes.c_void_p), ("live_count", ctypes.c_void_p),
                ("admitted", ctypes.c_void_p), ("dst_indptr", ctypes.c_void_p),
                ("new_bt_indptr", ctypes.c_void_p), ("new_block_ids", ctypes.c_void_p),
                ("src_plan", ctypes.c_void_p), ("freed_indptr", ctypes.c_void_p),
                ("counters", ctypes.c_void_p), ("new_bt_capacity", ctypes.c_int64),
                ("src_plan_capacity", ctypes.c_int64)]


class CRepackOptions(ctypes.Structure):
    _fields_ = [("variant", ctypes.c_int32), ("grid", ctypes.c_int32),
                ("order", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class CDecode(ctypes.Structure):
    _fields_ = [("q", ctypes.c_void_p), ("out", ctypes.c_void_p),
                ("num_q_heads", ctypes.c_int32), ("layer", ctypes.c_int32),
                ("kv_dtype", ctypes.c_int32), ("scale", ctypes.c_float),
                ("max_tokens", ctypes.c_int32), ("workspace", ctypes.c_void_p),
                ("workspace_bytes", ctypes.c_int64), ("slot_count", ctypes.c_void_p)]


KV_FP16, KV_BF16, KV_FP8_E4M3 = 0, 1, 2


class CPlannerParams(ctypes.Structure):
    _fields_ = [("theta_num", ctypes.c_int32), ("theta_den", ctypes.c_int32),
                ("max_live_per_source", ctypes.c_int32), ("min_eligible", ctypes.c_int32),
                ("free_watermark", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("max_sources", ctypes.c_int64)]


class CPlannerState(ctypes.Structure):
    _fields_ = [("live_bits", ctypes.c_void_p), ("refs", ctypes.c_void_p),
                ("n_b", ctypes.c_void_p), ("selected", ctypes.c_void_p),
                ("elig_cum", ctypes.c_void_p), ("src_count", ctypes.c_void_p),
                ("sources", ctypes.c_void_p), ("stats", ctypes.c_void_p),
                ("pinned", ctypes.c_void_p)]


# Every extern "C" symbol of include/vtoken.h with its ctypes signature.
_SIGNATURES = {
    "vtoken_build_token_table": (ctypes.c_int32, [ctypes.POINTER(CCache), ctypes.POINTER(CBatch),
                                                  ctypes.POINTER(CPlan), ctypes.c_void_p]),
    "vtoken_repack": (ctypes.c_int32, [ctypes.POINTER(CCache), ctypes.POINTER(CBatch),
                                       ctypes.POINTER(CPlan), ctypes.c_void_p]),
    "vtoken_build_token_table_inplace": (ctypes.c_int32, [ctypes.POINTER(CCache),
                                                          ctypes.POINTER(CBatch),
                                                          ctypes.POINTER(CPlan),
                                                          ctypes.c_void_p]),
    "vtoken_repack_inplace": (ctypes.c_int32, [ctypes.POINTER(CCache), ctypes.POINTER(CBatch),
                                               ctypes.POINTER(CPlan), ctypes.c_void_p]),
    "vtoken_repack_inplace_ex": (ctypes.c_int32, [ctypes.POINTER(CCache), ctypes.POINTER(CBatch),
                                                  ctypes.POINTER(CPlan),
                                                  ctypes.POINTER(CRepackOptions),
                                                  ctypes.c_void_p]),
    "vtoken_repack_ex": (ctypes.c_int32, [ctypes.POINTER(CCache), ctypes.POINTER(CBatch),
                                          ctypes.POINTER(CPlan), ctypes.POINTER(CRepackOptions),
                                          ctypes.c_void_p]),
    "vtoken_check_layout_workspace_bytes": (ctypes.c_int64, [ctypes.c_int32]),
    "vtoken_check_layout": (ctypes.c_int32, [ctypes.POINTER(CCache), ctypes.POINTER(CBatch),
                                             ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                             ctypes.c_void_p]),
    "vtoken_free_blocks": (ctypes.c_int32, [ctypes.POINTER(CBatch), ctypes.POINTER(CPlan),
                                            ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]),
    "vtoken_repack_free": (ctypes.c_int32, [ctypes.POINTER(CCache), ctypes.POINTER(CBatch),
                                            ctypes.POINTER(CPlan), ctypes.c_void_p,
                                            ctypes.c_int64, ctypes.c_void_p]),
    "vtoken_build_slot_mapping": (ctypes.c_int32, [ctypes.POINTER(CBatch),
                                                   ctypes.POINTER(CPlan), ctypes.c_void_p,
                                                   ctypes.c_void_p, ctypes.c_int64,
                                                   ctypes.c_void_p]),
    "vtoken_build_slot_table": (ctypes.c_int32, [ctypes.POINTER(CBatch), ctypes.POINTER(CPlan),
                                                 ctypes.c_int32, ctypes.c_void_p,
                                                 ctypes.c_void_p, ctypes.c_void_p,
                                                 ctypes.c_int64, ctypes.c_void_p]),
    "vtoken_append_slots": (ctypes.c_int32, [ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                             ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                             ctypes.c_void_p, ctypes.c_void_p]),
    "vtoken_decode_workspace_bytes": (ctypes.c_int64, [ctypes.c_int32, ctypes.c_int32,
                                                       ctypes.c_int32, ctypes.c_int32]),
    "vtoken_paged_decode": (ctypes.c_int32, [ctypes.POINTER(CCache), ctypes.POINTER(CDecode),
                                             ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                             ctypes.c_void_p]),
    "vtoken_paged_decode_noalloc": (ctypes.c_int32, [ctypes.POINTER(CCache),
                                                     ctypes.POINTER(CDecode), ctypes.c_int32,
                                                     ctypes.c_void_p, ctypes.c_void_p,
                                                     ctypes.c_void_p]),
    "vtoken_plan_partial": (ctypes.c_int32, [ctypes.POINTER(CCache), ctypes.POINTER(CBatch),
                                             ctypes.c_void_p, ctypes.POINTER(CPlannerParams),
                                             ctypes.POINTER(CPlannerState),
                                             ctypes.POINTER(CPlan), ctypes.c_void_p]),
    "vtoken_last_hip_error": (ctypes.c_int32, []),
    "vtoken_status_string": (ctypes.c_char_p, [ctypes.c_int32]),
    "vtoken_version": (ctypes.c_int32, []),
    "vtoken_build_id": (ctypes.c_char_p, []),
}

_lib = None


def load_library(path: str = LIB_PATH):
    """Load libvtoken.so (built by paper_2608_13263_amd.build) and set the signatures."""
    global _lib
    if _lib is not None and path == LIB_PATH:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with "
                           "`python -m paper_2608_13263_amd.build` (hipcc, gfx950)")
    # torch first: the library must bind to the HIP runtime torch has loaded, since the
    # streams and device pointers it is handed are torch's (loaded the other way round, the
    # library's calls found no device)
    import torch  # noqa: F401
    lib = ctypes.CDLL(path)
    for name, (res, args) in _SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    if path == LIB_PATH:
        # a library built from other sources than this tree's is refused, not run
        from paper_2608_13263_amd.build import source_sha256
        built, tree = lib.vtoken_build_id().decode(), source_sha256()
        if built != tree:
            raise RuntimeError(f"{path} was built from other sources (build id {built[:16]}, "
                               f"tree {tree[:16]}): rebuild with "
                               "`python -m paper_2608_13263_amd.build`")
        _lib = lib
    return lib


def status_string(status: int) -> str:
    return load_library().vtoken_status_string(int(status)).decode()


def _ptr(t) -> int:
    return 0 if t is None else int(t.data_ptr())


def _check(status: int, where: str):
    if status == STATUS_CODE["VTOKEN_ERR_HIP"]:
        raise VTokenError(status, f"{where} (hipError_t {load_library().vtoken_last_hip_error()})")
    if status != VTOKEN_OK:
        raise VTokenError(status, where)


def _stream(stream) -> int:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream) if hasattr(stream, "cuda_stream") else int(stream)


class _Cached:
    """The C struct of an object is built once and reused (it only holds the tensors' device
    addresses and sizes); assigning any attribute drops it. Building the structs costs a few
    microseconds of Python per call, which a small pass would otherwise spend in every call."""

    def __setattr__(self, name, value):
        object.__setattr__(self, name, value)
        if name != "_c_cache":
            object.__setattr__(self, "_c_cache", None)

    def c(self):
        cached = getattr(self, "_c_cache", None)
        if cached is None:
            cached = self._make_c()
            object.__setattr__(self, "_c_cache", cached)
        return cached


class KVCache(_Cached):
    """A paged KV cache tensor [2L][num_blocks][S][H][D] (any 1- or 2-byte dtype)."""

    def __init__(self, kv, num_layers: int, num_kv_heads: int, head_dim: int, block_size: int):
        if not kv.is_cuda or not kv.is_contiguous():
            raise ValueError("kv must be a contiguous device tensor")
        self.kv = kv
        self.num_layers, self.num_kv_heads = int(num_layers), int(num_kv_heads)
        self.head_dim, self.block_size = int(head_dim), int(block_size)
        self.elem_bytes = kv.element_size()
        per_block = 2 * self.num_layers * block_size * num_kv_heads * head_dim
        if kv.numel() % per_block:
            raise ValueError("kv size is not a whole number of blocks")
        self.num_blocks = kv.numel() // per_block

    def _make_c(self) -> CCache:
        return CCache(_ptr(self.kv), self.num_layers, self.num_kv_heads, self.head_dim,
                      self.block_size, self.num_blocks, self.elem_bytes)


class Batch(_Cached):
    """Device-resident request batch (CSR), matching vtoken_batch."""

    def __init__(self, seq_lens, tok_indptr, bt_indptr, block_ids, live, free_list):
        self.seq_lens, self.tok_indptr, self.bt_indptr = seq_lens, tok_indptr, bt_indptr
        self.block_ids, self.live, self.free_list = block_ids, live, free_list
        self.num_reqs = int(seq_lens.numel())
        self.num_tokens = int(live.numel())
        self.num_bt_entries = int(block_ids.numel())
        self.free_len = int(free_list.numel())

    @classmethod
    def from_host(cls, seq_lens, tok_indptr, bt_indptr, block_ids, live, free_list,
                  device="cuda"):
        import numpy as np
        import torch

        def i32(x):
            return torch.from_numpy(np.ascontiguousarray(x, dtype=np.int32)).to(device)
        return cls(i32(seq_lens), i32(tok_indptr), i32(bt_indptr), i32(block_ids),
                   torch.from_numpy(np.ascontiguousarray(live, dtype=np.uint8)).to(device),
                   i32(free_list))

    @classmethod
    def from_inputs(cls, inp, device="cuda"):
        return cls.from_host(inp.seq_lens, inp.tok_indptr, inp.bt_indptr, inp.block_ids,
                             inp.live, inp.free_list, device)

    def _make_c(self) -> CBatch:
        return CBatch(self.num_reqs, self.num_tokens, self.num_bt_entries, _ptr(self.seq_lens),
                      _ptr(self.tok_indptr), _ptr(self.bt_indptr), _ptr(self.block_ids),
                      _ptr(self.live), _ptr(self.free_list), self.free_len)


class Plan(_Cached):
    """Caller-allocated outputs (vtoken_plan) plus the freed-list buffer."""

    FIELDS = ("token_slot", "live_count", "admitted", "dst_indptr", "new_bt_indptr",
              "new_block_ids", "src_plan", "freed_indptr", "counters")

    def __init__(self, **tensors):
        for k in self.FIELDS + ("freed",):
            setattr(self, k, tensors[k])

    @classmethod
    def allocate(cls, batch: Batch, block_size: int, device="cuda", inplace: bool = False):
        """Outputs sized for out-of-place mode, or for in-place mode (src_plan holds up to
        M destination blocks)."""
        import torch
        R, T, M, f = batch.num_reqs, batch.num_tokens, batch.num_bt_entries, batch.free_len

        def e(n):
            return torch.empty(max(int(n), 1), dtype=torch.int32, device=device)
        rows = M if inplace else min(f, M)
        return cls(token_slot=e(T), live_count=e(R), admitted=e(R), dst_indptr=e(R + 1),
                   new_bt_indptr=e(R + 1), new_block_ids=e(M),
                   src_plan=e(rows * block_size), freed_indptr=e(R + 1), counters=e(5),
                   freed=e(M))

    def _make_c(self) -> CPlan:
        return CPlan(*(_ptr(getattr(self, k)) for k in self.FIELDS),
                     int(self.new_block_ids.numel()), int(self.src_plan.numel()))


def build_token_table(cache: KVCache, batch: Batch, plan: Plan, stream=None) -> None:
    lib = load_library()
    c, b, p = cache.c(), batch.c(), plan.c()
    _check(lib.vtoken_build_token_table(ctypes.byref(c), ctypes.byref(b), ctypes.byref(p),
                                        _stream(stream)), "vtoken_build_token_table")


def build_token_table_inplace(cache: KVCache, batch: Batch, plan: Plan, stream=None) -> None:
    lib = load_library()
    c, b, p = cache.c(), batch.c(), plan.c()
    _check(lib.vtoken_build_token_table_inplace(ctypes.byref(c), ctypes.byref(b),
                                                ctypes.byref(p), _stream(stream)),
           "vtoken_build_token_table_inplace")


def repack_inplace(cache: KVCache, batch: Batch, plan: Plan, stream=None) -> None:
    lib = load_library()
    c, b, p = cache.c(), batch.c(), plan.c()
    _check(lib.vtoken_repack_inplace(ctypes.byref(c), ctypes.byref(b), ctypes.byref(p),
                                     _stream(stream)), "vtoken_repack_inplace")


def repack_inplace_ex(cache: KVCache, batch: Batch, plan: Plan, variant: int = 0,
                      stream=None) -> None:
    lib = load_library()
    c, b, p = cache.c(), batch.c(), plan.c()
    o = CRepackOptions(variant, 0, 0, 0)
    _check(lib.vtoken_repack_inplace_ex(ctypes.byref(c), ctypes.byref(b), ctypes.byref(p),
                                        ctypes.byref(o), _stream(stream)),
           "vtoken_repack_inplace_ex")


def repack(cache: KVCache, batch: Batch, plan: Plan, stream=None) -> None:
    lib = load_library()
    c, b, p = cache.c(), batch.c(), plan.c()
    _check(lib.vtoken_repack(ctypes.byref(c), ctypes.byref(b), ctypes.byref(p),
                             _stream(stream)), "vtoken_repack")


def repack_ex(cache: KVCache, batch: Batch, plan: Plan, variant: int = 0, grid: int = 0,
              order: int = 0, stream=None) -> None:
    lib = load_library()
    c, b, p = cache.c(), batch.c(), plan.c()
    o = CRepackOptions(variant, grid, order, 0)
    _check(lib.vtoken_repack_ex(ctypes.byref(c), ctypes.byref(b), ctypes.byref(p),
                                ctypes.byref(o), _stream(stream)), "vtoken_repack_ex")


def free_blocks(batch: Batch, plan: Plan, freed=None, stream=None) -> None:
    lib = load_library()
    b, p = batch.c(), plan.c()
    out = plan.freed if freed is None else freed
    _check(lib.vtoken_free_blocks(ctypes.byref(b), ctypes.byref(p), _ptr(out),
                                  int(out.numel()), _stream(stream)), "vtoken_free_blocks")


def repack_free(cache: KVCache, batch: Batch, plan: Plan, freed=None, stream=None) -> None:
    """vtoken_repack and vtoken_free_blocks in one launch (vtoken_repack_free)."""
    lib = load_library()
    c, b, p = cache.c(), batch.c(), plan.c()
    out = plan.freed if freed is None else freed
    _check(lib.vtoken_repack_free(ctypes.byref(c), ctypes.byref(b), ctypes.byref(p), _ptr(out),
                                  int(out.numel()), _stream(stream)), "vtoken_repack_free")


def check_layout(cache: KVCache, batch: Batch, workspace=None, stream=None):
    """Device check of the full pass's layout precondition (each block id in the pool and
    held at most once over the block tables and the free list); returns a device int32 [1]
    status tensor (VTOKEN_OK, VTOKEN_ERR_BLOCK_RANGE or VTOKEN_ERR_LAYOUT)."""
    import torch
    lib = load_library()
    need = int(lib.vtoken_check_layout_workspace_bytes(cache.num_blocks))
    if workspace is None:
        workspace = torch.empty(max(need // 4, 1), dtype=torch.int32, device=cache.kv.device)
    status = torch.empty(1, dtype=torch.int32, device=cache.kv.device)
    c, b = cache.c(), batch.c()
    _check(lib.vtoken_check_layout(ctypes.byref(c), ctypes.byref(b), _ptr(workspace),
                                   int(workspace.numel() * workspace.element_size()),
                                   _ptr(status), _stream(stream)), "vtoken_check_layout")
    return status


def run_pass(cache: KVCache, batch: Batch, plan: Optional[Plan] = None, stream=None,
             inplace: bool = False) -> Plan:
    """One repack pass enqueued in order on one stream: the table build, then the copy and the
    freed list (out of place in one launch, vtoken_repack_free; in place as two calls)."""
    if plan is None:
        plan = Plan.allocate(batch, cache.block_size, device=cache.kv.device, inplace=inplace)
    if inplace:
        build_token_table_inplace(cache, batch, plan, stream)
        repack_inplace(cache, batch, plan, stream)
        free_blocks(batch, plan, stream=stream)
    else:
        build_token_table(cache, batch, plan, stream)
        repack_free(cache, batch, plan, stream=stream)
    return plan


def build_slot_mapping(batch: Batch, plan: Plan, slot_indptr=None, slots=None,
                       stream=None):
    """Slots of every request's live tokens in logical order (CSR); returns
    (slot_indptr [R+1], slots [T]) device tensors."""
    import torch
    lib = load_library()
    dev = plan.counters.device
    if slot_indptr is None:
        slot_indptr = torch.empty(batch.num_reqs + 1, dtype=torch.int32, device=dev)
    if slots is None:
        slots = torch.empty(max(batch.num_tokens, 1), dtype=torch.int32, device=dev)
    b, p = batch.c(), plan.c()
    _check(lib.vtoken_build_slot_mapping(ctypes.byref(b), ctypes.byref(p), _ptr(slot_indptr),
                                         _ptr(slots), int(slots.numel()), _stream(stream)),
           "vtoken_build_slot_mapping")
    return slot_indptr, slots


def build_slot_table(batch: Batch, plan: Plan, reserve: int, stream=None):
    """The slot mapping as an append-only translation cache: returns (slot_start [R+1],
    slot_count [R], slots) with room for `reserve` more slots per request."""
    import torch
    lib = load_library()
    dev = plan.counters.device
    R = batch.num_reqs
    start = torch.empty(R + 1, dtype=torch.int32, device=dev)
    count = torch.empty(max(R, 1), dtype=torch.int32, device=dev)
    slots = torch.empty(max(batch.num_tokens + R * int(reserve), 1), dtype=torch.int32,
                        device=dev)
    b, p = batch.c(), plan.c()
    _check(lib.vtoken_build_slot_table(ctypes.byref(b), ctypes.byref(p), int(reserve),
                                       _ptr(start), _ptr(count), _ptr(slots),
                                       int(slots.numel()), _stream(stream)),
           "vtoken_build_slot_table")
    return start, count, slots


def append_slots(slot_start, slot_count, slots, append_indptr, append_slots, status=None,
                 stream=None):
    """Append each request's new slots to its region of a slot table; returns the device
    status word (0, or VTOKEN_ERR_CAPACITY when a region is full and a rebuild is due)."""
    import torch
    lib = load_library()
    if status is None:
        status = torch.empty(1, dtype=torch.int32, device=slots.device)
    R = int(append_indptr.numel()) - 1
    _check(lib.vtoken_append_slots(R, _ptr(append_indptr), _ptr(append_slots),
                                   _ptr(slot_start), _ptr(slot_count), _ptr(slots),
                                   _ptr(status), _stream(stream)), "vtoken_append_slots")
    return status


def decode_workspace_bytes(num_reqs: int, num_q_heads: int, head_dim: int,
                           max_tokens: int) -> int:
    n = load_library().vtoken_decode_workspace_bytes(int(num_reqs), int(num_q_heads),
                                                     int(head_dim), int(max_tokens))
    if n < 0:
        raise VTokenError(STATUS_CODE["VTOKEN_ERR_SHAPE"], "vtoken_decode_workspace_bytes")
    return n


def kv_dtype_code(dtype) -> int:
    import torch
    codes = {torch.float16: KV_FP16, torch.bfloat16: KV_BF16}
    if hasattr(torch, "float8_e4m3fn"):
        codes[torch.float8_e4m3fn] = KV_FP8_E4M3
    if dtype not in codes:
        raise ValueError(f"paged decode reads fp16, bf16 or fp8 e4m3 KV, not {dtype}")
    return codes[dtype]


def paged_decode(cache: KVCache, q, slot_indptr, slots, layer: int, max_tokens: int,
                 scale: Optional[float] = None, out=None, workspace=None, kv_dtype=None,
                 stream=None, slot_count=None):
    """Decode attention of one layer through a slot mapping; q and out are float32
    [R][num_q_heads][head_dim] device tensors. kv_dtype defaults to the cache tensor's
    dtype (a uint8 view of fp8 data needs KV_FP8_E4M3). With slot_count, (slot_indptr,
    slot_count, slots) is a slot table (build_slot_table / append_slots)."""
    import torch
    lib = load_library()
    if q.dtype != torch.float32 or not q.is_contiguous() or q.dim() != 3:
        raise ValueError("q must be a contiguous float32 [R][Hq][D] tensor")
    R, Hq, D = (int(x) for x in q.shape)
    if D != cache.head_dim:
        raise ValueError("q head_dim differs from the cache's")
    if out is None:
        out = torch.empty_like(q)
    if out.shape != q.shape or out.dtype != torch.float32 or not out.is_contiguous():
        raise ValueError("out must match q")
    need = decode_workspace_bytes(R, Hq, D, max_tokens)
    if workspace is None:
        workspace = torch.empty(max(need // 4, 1), dtype=torch.float32, device=q.device)
    code = kv_dtype_code(cache.kv.dtype) if kv_dtype is None else int(kv_dtype)
    if scale is None:
        scale = D ** -0.5
    d = CDecode(_ptr(q), _ptr(out), Hq, int(layer), code, float(scale), int(max_tokens),
                _ptr(workspace), int(workspace.numel() * workspace.element_size()),
                _ptr(slot_count))
    c = cache.c()
    _check(lib.vtoken_paged_decode(ctypes.byref(c), ctypes.byref(d), R, _ptr(slot_indptr),
                                   _ptr(slots), _stream(stream)), "vtoken_paged_decode")
    return out


DECODE_SCRATCH_BYTES = 64 << 20   # VTOKEN_DECODE_SCRATCH_BYTES


def paged_decode_noalloc(cache: KVCache, q, slot_indptr, slots, layer: int, max_tokens: int,
                         out, scale: Optional[float] = None, kv_dtype=None, stream=None,
                         slot_count=None):
    """paged_decode with the split partials in the library-held array
    (vtoken_paged_decode_noalloc): `out` is the caller's, nothing is allocated. Calls on one
    GPU must be stream-ordered (they share the array)."""
    import torch
    lib = load_library()
    if q.dtype != torch.float32 or not q.is_contiguous() or q.dim() != 3:
        raise ValueError("q must be a contiguous float32 [R][Hq][D] tensor")
    R, Hq, D = (int(x) for x in q.shape)
    if out.shape != q.shape or out.dtype != torch.float32 or not out.is_contiguous():
        raise ValueError("out must match q")
    code = kv_dtype_code(cache.kv.dtype) if kv_dtype is None else int(kv_dtype)
    if scale is None:
        scale = D ** -0.5
    d = CDecode(_ptr(q), _ptr(out), Hq, int(layer), code, float(scale), int(max_tokens),
                0, 0, _ptr(slot_count))
    c = cache.c()
    _check(lib.vtoken_paged_decode_noalloc(ctypes.byref(c), ctypes.byref(d), R,
                                           _ptr(slot_indptr), _ptr(slots), _stream(stream)),
           "vtoken_paged_decode_noalloc")
    return out


class PlannerParams:
    """Parameters of the partial pass (vtoken_planner_params); theta_F = theta[0]/theta[1]
    (the paper's default 0.25), max_live_per_source < 0 derives the utilisation bound from
    theta_F, max_sources is B, free_watermark < 0 drops the watermark condition."""

    def __init__(self, theta=(1, 4), max_live_per_source: int = -1, max_sources: int = 1 << 40,
                 min_eligible: int = 1, free_watermark: int = -1):
        self.theta = (int(theta[0]), int(theta[1]))
        self.max_live_per_source = int(max_live_per_source)
        self.max_sources = int(max_sources)
        self.min_eligible = int(min_eligible)
        self.free_watermark = int(free_watermark)

    def c(self) -> CPlannerParams:
        return CPlannerParams(self.theta[0], self.theta[1], self.max_live_per_source,
                              self.min_eligible, self.free_watermark, 0, self.max_sources)


class PlannerState:
    """Caller-allocated buffers of the partial pass (vtoken_planner_state)."""

    FIELDS = ("live_bits", "refs", "n_b", "selected", "elig_cum", "src_count", "sources",
              "stats")

    def __init__(self, pinned=None, **tensors):
        for k in self.FIELDS:
            setattr(self, k, tensors[k])
        self.pinned = pinned

    @classmethod
    def allocate(cls, num_blocks: int, batch: Batch, device="cuda", pinned=None):
        import torch

        def e(n, dt=torch.int32):
            return torch.empty(max(int(n), 1), dtype=dt, device=device)
        M, R = batch.num_bt_entries, batch.num_reqs
        if pinned is not None and not isinstance(pinned, torch.Tensor):
            import numpy as np
            pinned = torch.from_numpy(np.ascontiguousarray(pinned, dtype=np.uint8)).to(device)
        return cls(live_bits=e(num_blocks, torch.int64), refs=e(num_blocks), n_b=e(num_blocks),
                   selected=e(num_blocks), elig_cum=e(M), src_count=e(R), sources=e(M),
                   stats=e(8, torch.int64), pinned=pinned)

    def c(self) -> CPlannerState:
        return CPlannerState(*(_ptr(getattr(self, k)) for k in self.FIELDS), _ptr(self.pinned))


def plan_partial(cache: KVCache, batch: Batch, slot_in, plan: Plan, state: PlannerState,
                 params: Optional[PlannerParams] = None, stream=None) -> None:
    """The partial pass's planning kernels; follow with repack() on the same plan."""
    lib = load_library()
    c, b, p = cache.c(), batch.c(), plan.c()
    prm = (params or PlannerParams()).c()
    st = state.c()
    _check(lib.vtoken_plan_partial(ctypes.byref(c), ctypes.byref(b), _ptr(slot_in),
                                   ctypes.byref(prm), ctypes.byref(st), ctypes.byref(p),
                                   _stream(stream)), "vtoken_plan_partial")


def run_partial_pass(cache: KVCache, batch: Batch, slot_in, plan: Optional[Plan] = None,
                     state: Optional[PlannerState] = None,
                     params: Optional[PlannerParams] = None, pinned=None, stream=None):
    """Plan and copy of one partial pass, enqueued in order on one stream; returns
    (plan, state). The released sources are state.sources[:plan.counters[2]]."""
    if plan is None:
        plan = Plan.allocate(batch, cache.block_size, device=cache.kv.device)
    if state is None:
        state = PlannerState.allocate(cache.num_blocks, batch, device=cache.kv.device,
                                      pinned=pinned)
    plan_partial(cache, batch, slot_in, plan, state, params, stream)
    repack(cache, batch, plan, stream)
    return plan, state
