"""MemDecay's per-decode-step retention path on AMD Instinct MI355X (gfx950).

The path (attention mass of the decode query against a paged bf16 key cache,
EWMA importance, refresh clocks, region-decayed retention scores, page
scores, budgeted page eviction, page-table compaction) runs in the HIP
kernels of ``libmemdecay.so`` behind a C ABI (include/memdecay.h).
``binding`` exposes that ABI to Python under the same names; ``cache``
holds the caller-side buffers and a thin driver.
"""
from . import binding  # noqa: F401

__all__ = ["binding", "build_library", "PagedCache", "MemDecay"]


def build_library(verbose: bool = False) -> str:
    from .build import build
    return build(verbose=verbose)


def __getattr__(name):
    if name in ("PagedCache", "MemDecay"):
        from . import cache
        return getattr(cache, name)
    raise AttributeError(name)
