"""Synthetic workload definitions for MemDecay's observation step.

Each workload fixes the attention shape (layers, query heads, KV heads,
head dim), the batch of agent sessions, the region-span recipe, the region
priors, the budget and the number of decode steps.  The region vocabulary and
its code order follow the label list of the problem setup (Sec. III-A):
system, plan, user, tool_in, tool_out, retrieval, scratchpad.

The shapes stand in for the paper's Qwen2.5-1.5B / 3B episodes (Sec. IV-A):
1.5B = 28 layers, 12 query / 2 KV heads; 3B = 36 layers, 16 / 2; head dim 128;
page size 16 as in the study, and 64 as the second page size of the ragged
batch.  Nothing here computes any part of the method.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Optional, Tuple

REGIONS: Tuple[str, ...] = (
    "system", "plan", "user", "tool_in", "tool_out", "retrieval", "scratchpad",
)
N_REGIONS = len(REGIONS)
SYSTEM, PLAN, USER, TOOL_IN, TOOL_OUT, RETRIEVAL, SCRATCHPAD = range(N_REGIONS)
MOVABLE = (PLAN, USER, TOOL_IN, TOOL_OUT, RETRIEVAL, SCRATCHPAD)

# Half-lives in decode steps for the movable regions (the small workload's
# values; reused by every workload, jittered per session in the ragged batch).
HALF_LIVES = {
    PLAN: 120.0, USER: 80.0, TOOL_IN: 40.0, TOOL_OUT: 30.0,
    RETRIEVAL: 50.0, SCRATCHPAD: 15.0,
}
# The system region is pinned, so its prior is never used when pinning is on.
# When a test turns pinning off it takes Fig. 2's example curve: b = 1.0,
# lambda = 0.002.
SYSTEM_B = 1.0
SYSTEM_LAMBDA = 0.002

APPEND_CYCLE = (SCRATCHPAD, TOOL_IN, TOOL_OUT)


@dataclass(frozen=True)
class Workload:
    name: str
    index: int                 # seed component
    L: int
    Hq: int
    Hkv: int
    d: int
    P: int                     # page size in tokens
    S: int                     # sessions
    n0: Optional[int]          # prefix length (None => drawn per session)
    n0_range: Optional[Tuple[int, int]]   # inclusive range when drawn
    system_len: int            # pinned system span at the start of each session
    mean_span: float           # geometric mean length of the movable spans
    budget_frac: float         # B_s = floor(frac * n0_s)
    steps: int                 # decode steps
    append_cycle: Tuple[int, ...]
    alpha: float = 1.0
    rho: float = 0.9
    tau_scale: float = 2.0     # tau = tau_scale / |K_t|
    pinned_mask: int = 1 << SYSTEM
    halflife_jitter: Optional[Tuple[float, float]] = None
    attention_norm: bool = False   # score's attention term relative to the uniform level
    window: int = 1                # decode queries per observation (W)
    obs_interval: int = 1          # one observation every k decode steps (k >= W)
    region_aligned: bool = False   # pages hold one region each (allocator variant)
    append_run: int = 1            # decode tokens per region run of the append cycle
    quant_threshold: float = 0.0   # quantised tier: pages scoring below it (0: off)
    b_range: Tuple[float, float] = (0.2, 1.0)
    extra: dict = field(default_factory=dict)

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    @property
    def k_bytes_per_token(self) -> int:
        return self.L * self.Hkv * self.d * 2


QWEN15 = dict(L=28, Hq=12, Hkv=2, d=128)
QWEN3 = dict(L=36, Hq=16, Hkv=2, d=128)

WORKLOADS = {
    # single layer, one 450-token session, 32 steps appending scratchpad
    "small": Workload("small", 0, L=1, Hq=12, Hkv=2, d=128, P=16, S=1, n0=450,
                      n0_range=None, system_len=60, mean_span=40.0,
                      budget_frac=0.5, steps=32, append_cycle=(SCRATCHPAD,)),
    # Qwen2.5-1.5B-shaped, one 1,700-token session, 256 steps
    "qwen15_1700": Workload("qwen15_1700", 1, **QWEN15, P=16, S=1, n0=1700,
                            n0_range=None, system_len=200, mean_span=40.0,
                            budget_frac=0.4, steps=256, append_cycle=APPEND_CYCLE),
    # Qwen2.5-3B-shaped, 32 sessions x 1,700 tokens, 256 steps
    "qwen3_32x1700": Workload("qwen3_32x1700", 2, **QWEN3, P=16, S=32, n0=1700,
                              n0_range=None, system_len=200, mean_span=40.0,
                              budget_frac=0.3, steps=256, append_cycle=APPEND_CYCLE),
    # long horizon: 1.5B shapes, 16 sessions x 32,768 tokens, 128 steps
    "long32k": Workload("long32k", 3, **QWEN15, P=16, S=16, n0=32768,
                        n0_range=None, system_len=1024, mean_span=512.0,
                        budget_frac=0.25, steps=128, append_cycle=APPEND_CYCLE),
    # ragged batch: 3B shapes, 64 sessions x U[2048, 65536], pages of 16 / 64
    "ragged_p16": Workload("ragged_p16", 4, **QWEN3, P=16, S=64, n0=None,
                           n0_range=(2048, 65536), system_len=1024,
                           mean_span=512.0, budget_frac=0.2, steps=64,
                           append_cycle=APPEND_CYCLE,
                           halflife_jitter=(0.8, 1.2)),
    "ragged_p64": Workload("ragged_p64", 4, **QWEN3, P=64, S=64, n0=None,
                           n0_range=(2048, 65536), system_len=1024,
                           mean_span=512.0, budget_frac=0.2, steps=64,
                           append_cycle=APPEND_CYCLE,
                           halflife_jitter=(0.8, 1.2)),
    # region-aligned pages: the small workload with turns of 5 decode tokens
    # per region, and the 32k batch with turns of 24
    "small_aligned": Workload("small_aligned", 5, L=1, Hq=12, Hkv=2, d=128, P=16, S=1, n0=450,
                              n0_range=None, system_len=60, mean_span=40.0,
                              budget_frac=0.5, steps=32, append_cycle=APPEND_CYCLE,
                              region_aligned=True, append_run=5),
    # the 32k batch observed every other decode step with a window of the
    # two latest queries (the multi-kernel path)
    "long32k_w2k2": Workload("long32k_w2k2", 3, **QWEN15, P=16, S=16, n0=32768,
                             n0_range=None, system_len=1024, mean_span=512.0,
                             budget_frac=0.25, steps=128, append_cycle=APPEND_CYCLE,
                             window=2, obs_interval=2),
    "long32k_aligned": Workload("long32k_aligned", 3, **QWEN15, P=16, S=16, n0=32768,
                                n0_range=None, system_len=1024, mean_span=512.0,
                                budget_frac=0.25, steps=128, append_cycle=APPEND_CYCLE,
                                region_aligned=True, append_run=24),
}


def get(name: str) -> Workload:
    return WORKLOADS[name]


def with_overrides(w: Workload, **kw) -> Workload:
    """A copy of ``w`` with some fields replaced (tests shrink workloads)."""
    d = {f: getattr(w, f) for f in w.__dataclass_fields__}
    d.update(kw)
    return Workload(**d)


def decay_rate_from_half_life(half_life: float) -> float:
    """Decay rate whose exponential halves after ``half_life`` steps.

    Input preparation: the workloads state region lifetimes as half-lives
    (Eq. 7 defines the half-life as ln 2 / lambda), while the method takes
    the rate lambda_r as its per-region parameter (Sec. III-B).
    """
    return math.log(2.0) / half_life
