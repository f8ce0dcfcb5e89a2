"""vToken KV repack for AMD Instinct MI355X (gfx950).

The hot path - live-mask scan, admission, token table, the gather-repack of every live K/V
row and the freed-block list - runs in hand-written HIP kernels behind the C ABI of
include/vtoken.h (libvtoken.so). This package holds the thin ctypes binding to that
library (`paper_2608_13263_amd.binding`) and the seeded workload generators
(`paper_2608_13263_amd.workloads`). The binding is imported lazily so that the generators
can be used on hosts without a GPU.
"""

__all__ = ["build_token_table", "repack", "repack_ex", "free_blocks",
           "build_token_table_inplace", "repack_inplace", "binding", "workloads"]


def __getattr__(name):
    if name in ("build_token_table", "repack", "repack_ex", "free_blocks",
                "build_token_table_inplace", "repack_inplace"):
        from . import binding
        return getattr(binding, name)
    if name in ("binding", "workloads"):
        import importlib
        return importlib.import_module(f".{name}", __name__)
    raise AttributeError(name)
