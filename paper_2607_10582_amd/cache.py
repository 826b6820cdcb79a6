"""Caller-side buffers and a thin driver for the MemDecay C ABI.

``PagedCache`` owns (through PyTorch) every device buffer of the library's
cache view: the paged bf16 key pool, the per-slot side arrays (region,
insertion step, refresh clock, importance), the page tables, the per-session
counters and the free list.  ``MemDecay`` binds a cache to a library handle
and calls the entry points in order.  PyTorch only allocates memory, places
the initial prompt into the pool (the decode engine's prefill, not part of
the retention step) and provides the stream; every step of the path runs in
the library's kernels.
"""
from __future__ import annotations

import math
from typing import Optional, Sequence

import numpy as np
import torch

from . import binding as B


class PagedCache:
    """Device buffers of one batch of sessions (layouts as in memdecay.h)."""

    def __init__(self, *, L: int, Hq: int, Hkv: int, d: int, P: int, S: int,
                 max_pages: int, n_phys: int, device="cuda", offload_pages: int = 0):
        self.L, self.Hq, self.Hkv, self.d, self.P = L, Hq, Hkv, d, P
        self.S, self.max_pages, self.n_phys = S, max_pages, n_phys
        self.device = torch.device(device)
        dev = self.device
        i32 = dict(dtype=torch.int32, device=dev)
        # Slots past a session's token count are never used, so the pool is
        # left uninitialised.
        self.k_pool = torch.empty((n_phys, L, Hkv, P // 16, d // 8, 16, 8), dtype=torch.bfloat16, device=dev)
        self.region = torch.zeros((n_phys, P), dtype=torch.uint8, device=dev)
        self.t_ins = torch.zeros((n_phys, P), **i32)
        self.t_ref = torch.zeros((n_phys, P), **i32)
        self.importance = torch.zeros((n_phys, P), dtype=torch.float32, device=dev)
        self.page_table = torch.full((S, max_pages), -1, **i32)
        self.page_serial = torch.full((S, max_pages), -1, **i32)
        self.n_pages = torch.zeros(S, **i32)
        self.n_tokens = torch.zeros(S, **i32)
        self.n_live = torch.zeros(S, **i32)   # tokens without holes (region-aligned pages)
        self.page_format = torch.zeros(n_phys, dtype=torch.uint8, device=dev)   # 1: quantised page
        self.clock = torch.zeros(S, **i32)
        self.next_serial = torch.zeros(S, **i32)
        self.budget = torch.zeros(S, **i32)
        self.free_list = torch.zeros(n_phys, **i32)
        self.free_count = torch.zeros(1, **i32)
        # offload tier: offload_pages host-memory pages per session, their
        # keys in pinned host memory (hipHostMalloc underneath), their
        # per-token state on the device
        self.offload_pages = H = int(offload_pages)
        if H > 0:
            self.host_keys = torch.zeros((S, H, L * Hkv * P * d), dtype=torch.bfloat16, pin_memory=True)
            self.off_count = torch.zeros(S, **i32)
            self.off_serial = torch.full((S, H), -1, **i32)
            self.off_slot = torch.full((S, H), -1, **i32)
            self.off_region = torch.zeros((S, H, P), dtype=torch.uint8, device=dev)
            self.off_t_ins = torch.zeros((S, H, P), **i32)
            self.off_t_ref = torch.zeros((S, H, P), **i32)
            self.off_importance = torch.zeros((S, H, P), dtype=torch.float32, device=dev)
            self.off_format = torch.zeros((S, H), dtype=torch.uint8, device=dev)
            self.off_score = torch.zeros((S, H), dtype=torch.float32, device=dev)
            self.off_abar = torch.zeros((S, H, P), dtype=torch.float32, device=dev)

    OFFLOAD_BUFFERS = ("host_keys", "off_count", "off_serial", "off_slot", "off_region", "off_t_ins",
                       "off_t_ref", "off_importance", "off_format", "off_score", "off_abar")

    def view(self) -> B.md_cache_view:
        v = B.md_cache_view()
        names = ["k_pool", "region", "t_ins", "t_ref", "importance", "page_table",
                 "page_serial", "n_pages", "n_tokens", "clock", "next_serial", "budget",
                 "free_list", "free_count", "n_live", "page_format"]
        if self.offload_pages > 0:
            names += list(self.OFFLOAD_BUFFERS)
        for name in names:
            setattr(v, name, getattr(self, name).data_ptr())
        return v

    @staticmethod
    def to_pool_layout(k: torch.Tensor) -> torch.Tensor:
        """Keys [m][P][L][Hkv][d] of m pages -> the pool's page layout
        [m][L][Hkv][P/16][d/8][16][8] (memdecay.h)."""
        m, P, L, Hkv, d = k.shape
        return k.view(m, P // 16, 16, L, Hkv, d // 8, 8).permute(0, 3, 4, 1, 5, 2, 6).contiguous()

    @staticmethod
    def from_pool_layout(pages: torch.Tensor) -> torch.Tensor:
        """The inverse: pool pages [m][L][Hkv][P/16][d/8][16][8] (or the pool
        itself) -> keys [m][P][L][Hkv][d]."""
        m, L, Hkv, nb, db = pages.shape[:5]
        return pages.permute(0, 3, 5, 1, 2, 4, 6).reshape(m, nb * 16, L, Hkv, db * 8)

    @staticmethod
    def positions(region, P: int, region_aligned: bool) -> np.ndarray:
        """Slot position (page * P + offset) of each prompt token in the
        session's page sequence: consecutive, or with region-aligned pages a
        fresh page at every region change (the positions skipped are holes)."""
        reg = np.asarray(region, dtype=np.int64)
        n = reg.size
        if not region_aligned or n == 0:
            return np.arange(n, dtype=np.int64)
        pos = np.empty(n, dtype=np.int64)
        p = 0
        for i in range(n):
            if i > 0 and reg[i] != reg[i - 1] and p % P:
                p += P - p % P          # close the page at the region boundary
            pos[i] = p
            p += 1
        return pos

    @classmethod
    def pages_for(cls, region, P: int, region_aligned: bool) -> int:
        """Pages a prompt with these region codes takes."""
        n = len(region)
        return 0 if n == 0 else (int(cls.positions(region, P, region_aligned)[-1]) + P) // P

    def load_session(self, s: int, keys: torch.Tensor, region, page_ids: Sequence[int],
                     budget: int, clock: int, t_ins=None, region_aligned: bool = False):
        """Place a session's prompt: keys bf16 [n][L][Hkv][d] (device), region
        codes [n], physical page ids in logical order (as many as the layout
        takes: ceil(n / P), or with region-aligned pages one more per region
        change inside a page; ``pages_for``).  Token i gets t_ins = t_ref =
        t_ins[i] (default i) and importance 0; holes get the hole code."""
        P = self.P
        n = int(keys.shape[0])
        pos = self.positions(region, P, region_aligned)
        n_pos = int(pos[-1]) + 1 if n else 0
        m = (n_pos + P - 1) // P
        if len(page_ids) != m or m > self.max_pages:
            raise ValueError("need one page id per page of the layout, within max_pages")
        ids = torch.as_tensor(np.asarray(page_ids, dtype=np.int64), device=self.device)
        posd = torch.as_tensor(pos, device=self.device)
        k = keys.to(self.device, torch.bfloat16)
        full = torch.zeros((m * P,) + tuple(k.shape[1:]), dtype=k.dtype, device=k.device)
        full[posd] = k
        # [m][P][L][Hkv][d] -> [m][L][Hkv][P][d]
        self.k_pool.index_copy_(0, ids, self.to_pool_layout(full.view(m, P, self.L, self.Hkv, self.d)))
        reg = torch.as_tensor(np.asarray(region, dtype=np.uint8), device=self.device)
        t0 = torch.arange(n, dtype=torch.int32, device=self.device) if t_ins is None else \
            torch.as_tensor(np.asarray(t_ins, dtype=np.int32), device=self.device)
        slots = (ids.view(-1, 1) * P + torch.arange(P, device=self.device).view(1, -1)).view(-1)
        used = slots[:n_pos]
        self.region.view(-1)[used] = B.MD_REGION_HOLE
        self.t_ins.view(-1)[used] = 0
        self.t_ref.view(-1)[used] = 0
        self.importance.view(-1)[used] = 0.0
        flat = slots[posd]
        self.region.view(-1)[flat] = reg
        self.t_ins.view(-1)[flat] = t0
        self.t_ref.view(-1)[flat] = t0
        self.importance.view(-1)[flat] = 0.0
        self.page_format[ids] = 0
        self.page_table[s, :m] = ids.to(torch.int32)
        self.page_table[s, m:] = -1
        self.page_serial[s, :m] = torch.arange(m, dtype=torch.int32, device=self.device)
        self.page_serial[s, m:] = -1
        self.n_pages[s] = m
        self.n_tokens[s] = n_pos
        self.n_live[s] = n
        self.clock[s] = clock
        self.next_serial[s] = m
        self.budget[s] = budget

    def set_free_pages(self, ids: Sequence[int]):
        """The free list: ids pop from the end."""
        ids = np.ascontiguousarray(ids, dtype=np.int32)
        self.free_list.zero_()
        if ids.size:
            self.free_list[: ids.size] = torch.as_tensor(ids, device=self.device)
        self.free_count[0] = int(ids.size)


class MemDecay:
    """A library handle bound to a PagedCache, with the step's output buffers."""

    def __init__(self, cache: PagedCache, base_priority: torch.Tensor, decay_rate: torch.Tensor, *,
                 rho: float, alpha: float, tau_scale: float, pinned_mask: int,
                 n_regions: int = 7, stream: Optional[torch.cuda.Stream] = None,
                 fused: Optional[bool] = None, attention_norm: bool = False, window: int = 1,
                 region_aligned: bool = False, quant_threshold: float = 0.0, static: bool = False,
                 drop_threshold: float = 0.0, cooperative: bool = False, row_groups: bool = True):
        # fused: True = always the fused kernel, False = always the
        # multi-kernel path, None = the library picks from the cache's sizes;
        # cooperative: the fused kernel as a cooperative launch (for a GPU
        # shared with other streams); row_groups: False keeps every fused
        # unit on all rows
        self.cache = cache
        dev = cache.device
        self.b = base_priority.to(dev, torch.float32).contiguous()
        self.lam = decay_rate.to(dev, torch.float32).contiguous()
        cfg = B.md_config(n_layers=cache.L, n_q_heads=cache.Hq, n_kv_heads=cache.Hkv,
                          head_dim=cache.d, page_size=cache.P, max_sessions=cache.S,
                          max_pages=cache.max_pages, n_phys_pages=cache.n_phys,
                          n_regions=n_regions, pinned_region_mask=pinned_mask, rho=rho,
                          alpha=alpha, tau_scale=tau_scale,
                          flags=(0 if fused is None else (B.MD_FLAG_FUSED if fused else B.MD_FLAG_NO_FUSED))
                          | (B.MD_FLAG_NORM_ATTENTION if attention_norm else 0)
                          | (B.MD_FLAG_REGION_ALIGNED if region_aligned else 0)
                          | (B.MD_FLAG_COOPERATIVE if cooperative else 0)
                          | (0 if row_groups else B.MD_FLAG_NO_ROW_GROUPS),
                          window=window, quant_threshold=quant_threshold,
                          offload_pages=cache.offload_pages, drop_threshold=drop_threshold)
        rp = B.md_region_params(base_priority=self.b.data_ptr(), decay_rate=self.lam.data_ptr())
        self.stream = stream if stream is not None else torch.cuda.current_stream(dev)
        self._cfg, self._rp, self._cv = cfg, rp, cache.view()
        # static: md_init_static (the library's static scratch, no allocation)
        init = B.md_init_static if static else B.md_init
        self.handle = init(cfg, rp, self._cv, self.stream.cuda_stream)
        S, MP = cache.S, cache.max_pages
        self.page_score = torch.zeros((S, MP), dtype=torch.float32, device=dev)
        self.evict_serial = torch.zeros((S, MP), dtype=torch.int32, device=dev)
        self.evict_count = torch.zeros(S, dtype=torch.int32, device=dev)
        self.infeasible = torch.zeros(S, dtype=torch.uint8, device=dev)

    # ---- the four calls of one step
    def observe(self, step: int, q: torch.Tensor, new_k: Optional[torch.Tensor] = None,
                new_region: Optional[torch.Tensor] = None, abar_out: Optional[torch.Tensor] = None):
        B.md_observe_step(self.handle, step, None if q is None else _ptr(q, torch.float32),
                          None if new_k is None else _ptr(new_k, torch.bfloat16),
                          None if new_region is None else _ptr(new_region, torch.uint8),
                          None if abar_out is None else _ptr(abar_out, torch.float32))

    def score(self, token_score: Optional[torch.Tensor] = None, page_score: bool = True):
        B.md_score_pages(self.handle, self.page_score.data_ptr() if page_score else None,
                         None if token_score is None else _ptr(token_score, torch.float32))

    def select(self):
        B.md_select_evict(self.handle, self.evict_serial.data_ptr(), self.evict_count.data_ptr(),
                          self.infeasible.data_ptr())

    def compact(self, evict_serial: Optional[torch.Tensor] = None,
                evict_count: Optional[torch.Tensor] = None):
        """Apply this step's selection (no arguments), or the given lists."""
        if evict_serial is None and evict_count is None:
            B.md_compact(self.handle, None, None)
        else:
            B.md_compact(self.handle, _ptr(evict_serial, torch.int32), _ptr(evict_count, torch.int32))

    def select_compact(self):
        """select() then compact() with this step's selection, as one call
        (one launch when no tier is configured)."""
        B.md_select_compact(self.handle, self.evict_serial.data_ptr(), self.evict_count.data_ptr(),
                            self.infeasible.data_ptr())

    def step(self, step: int, q, new_k=None, new_region=None, page_scores: bool = True):
        """One decode step; page_scores=False leaves self.page_score untouched
        (the library still scores every page for its own selection).  The
        step's selection is applied as it stands (select_compact)."""
        self.observe(step, q, new_k, new_region)
        if q is None:   # a decode step without an observation only appends
            return
        self.score(page_score=page_scores)
        self.select_compact()

    def calib_accumulate(self, abar: torch.Tensor, bucket_steps: int, stats) -> None:
        """Add this observation to stats = (mass_fx, count, age_sum), int64
        tensors [S][n_regions][n_buckets] viewed as uint64 by the library."""
        mass, count, age = stats
        B.md_calib_accumulate(self.handle, _ptr(abar, torch.float32), bucket_steps, mass.shape[-1],
                              mass.data_ptr(), count.data_ptr(), age.data_ptr())

    def device_status(self, with_warning: bool = False):
        return B.md_read_device_status(self.handle, with_warning)

    def profile(self, kernels=("logits",)):
        """Time the named kernels with events from now on (() turns it off)."""
        mask = 0
        for k in kernels:
            mask |= 1 << B.KERNELS.index(k)
        B.md_profile_enable(self.handle, mask)

    def profile_read(self, kernel: str):
        return B.md_profile_read(self.handle, B.KERNELS.index(kernel))

    def counters(self):
        return B.md_read_counters(self.handle)

    def kernel_config(self) -> dict:
        return B.md_kernel_config(self.handle)

    def close(self):
        if self.handle is not None:
            B.md_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _ptr(t: torch.Tensor, dtype) -> int:
    if t.dtype != dtype or not t.is_contiguous():
        raise ValueError(f"expected a contiguous {dtype} tensor, got {t.dtype}")
    return t.data_ptr()
