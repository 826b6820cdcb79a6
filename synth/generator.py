"""Seeded synthetic inputs shared by the oracle and the device path.

This module only draws numbers; it holds none of the method's arithmetic.
Every draw comes from its own stream,

    numpy.random.Generator(PCG64(SeedSequence([2607, 10582, workload, session,
                                               stream, step])))

so any session or step can be regenerated on its own.  Keys are drawn as
standard normals in float32 and rounded to bfloat16 (round to nearest even);
queries stay float32.  Region labels come in contiguous spans (Sec. III-A):
a pinned system span first, then the six movable regions in a fresh seeded
order per round, each span geometric with the workload's mean length; the
last span is cut at the prefix length.

For the largest workloads the numpy draw of tens of GB of keys is too slow,
so ``torch_keys`` / ``torch_queries`` draw the same shapes with torch's
counter-based generator on the device, seeded from the same SeedSequence.
Both backends are deterministic; they do not produce the same numbers as
each other, and a consumer always takes one workload's inputs from one
backend.
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np

from .configs import (HALF_LIVES, MOVABLE, N_REGIONS, SYSTEM, SYSTEM_B,
                      SYSTEM_LAMBDA, Workload, decay_rate_from_half_life)

STREAMS = {"spans": 0, "prio": 1, "jitter": 2, "len": 3, "kpre": 4,
           "kapp": 5, "q": 6, "perm": 7}


def seed_sequence(w: Workload, session: int, stream: str, step: int = 0):
    return np.random.SeedSequence(
        [2607, 10582, w.index, session, STREAMS[stream], step])


def rng(w: Workload, session: int, stream: str, step: int = 0):
    return np.random.Generator(np.random.PCG64(seed_sequence(w, session, stream, step)))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    bias = ((u >> 16) & 1) + 0x7FFF
    return ((u + bias) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bfloat16 bits to float32 (exact)."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# ---------------------------------------------------------------- structure

def prefix_lengths(w: Workload) -> np.ndarray:
    """Cached prefix length n0 of every session."""
    if w.n0 is not None:
        return np.full(w.S, w.n0, dtype=np.int64)
    lo, hi = w.n0_range
    return np.array([int(rng(w, s, "len").integers(lo, hi + 1)) for s in range(w.S)],
                    dtype=np.int64)


def region_spans(w: Workload, session: int, n0: int) -> np.ndarray:
    """Region label per prefix token: system span, then seeded movable spans."""
    g = rng(w, session, "spans")
    out = np.empty(n0, dtype=np.uint8)
    pos = min(w.system_len, n0)
    out[:pos] = SYSTEM
    p = 1.0 / w.mean_span
    while pos < n0:
        order = g.permutation(np.array(MOVABLE, dtype=np.uint8))
        for r in order:
            if pos >= n0:
                break
            ln = int(g.geometric(p))
            ln = min(ln, n0 - pos)
            out[pos:pos + ln] = r
            pos += ln
    return out


def region_priors(w: Workload):
    """Per-session region tables (b_r, lambda_r), float32 [S][7].

    Base priorities of the movable regions are drawn U(b_range) once per
    workload; decay rates come from the configured half-lives, jittered per
    (session, region) when the workload asks for it.
    """
    g = rng(w, 0, "prio")
    b_mov = g.uniform(w.b_range[0], w.b_range[1], size=len(MOVABLE))
    b = np.empty((w.S, N_REGIONS), dtype=np.float32)
    lam = np.empty((w.S, N_REGIONS), dtype=np.float32)
    for s in range(w.S):
        b[s, SYSTEM] = SYSTEM_B
        lam[s, SYSTEM] = SYSTEM_LAMBDA
        if w.halflife_jitter is not None:
            jit = rng(w, s, "jitter").uniform(*w.halflife_jitter, size=len(MOVABLE))
        else:
            jit = np.ones(len(MOVABLE))
        for j, r in enumerate(MOVABLE):
            b[s, r] = b_mov[j]
            lam[s, r] = decay_rate_from_half_life(HALF_LIVES[r] * jit[j])
    return b, lam


def budgets(w: Workload, n0s: np.ndarray) -> np.ndarray:
    """Token budget per session, B_s = floor(frac * n0_s) in exact arithmetic."""
    f = Fraction(str(w.budget_frac))
    return np.array([int(f * int(n)) for n in n0s], dtype=np.int64)


def append_region(w: Workload, step: int) -> int:
    """Region of the token appended at decode step ``step`` (1-based): the
    append cycle's regions in turn, each for ``append_run`` steps."""
    return int(w.append_cycle[((step - 1) // w.append_run) % len(w.append_cycle)])


def pages_needed(w: Workload, n0s: np.ndarray) -> int:
    """Physical pages for every prefix plus every appended token, plus one
    spare page per session for the page a step may open.  With region-aligned
    pages, an upper bound: every region span of a prefix, and every region
    run of the appended tokens, may start a page of its own."""
    if not w.region_aligned:
        pre = int(sum((int(n) + w.P - 1) // w.P for n in n0s))
        app = w.S * ((w.steps + w.P - 1) // w.P + 1)
        return pre + app
    pre = 0
    for s, n in enumerate(n0s):
        reg = region_spans(w, s, int(n))
        spans = int(np.count_nonzero(np.diff(reg.astype(np.int64)))) + 1 if n else 0
        pre += (int(n) + w.P - 1) // w.P + spans
    runs = (w.steps + w.append_run - 1) // w.append_run
    app = w.S * ((w.steps + w.P - 1) // w.P + runs + 1)
    return pre + app


def page_permutation(w: Workload, n_phys: int) -> np.ndarray:
    """Seeded permutation of physical page ids (makes the indirection real)."""
    return rng(w, 0, "perm").permutation(n_phys).astype(np.int32)


# ---------------------------------------------------------------- tensors

def k_prefix(w: Workload, session: int, n0: int) -> np.ndarray:
    """bf16 bits [n0][L][Hkv][d] of the session's prefix keys."""
    x = rng(w, session, "kpre").standard_normal((n0, w.L, w.Hkv, w.d), dtype=np.float32)
    return f32_to_bf16_bits(x)


def k_append(w: Workload, session: int, step: int) -> np.ndarray:
    """bf16 bits [L][Hkv][d] of the key appended at ``step``."""
    x = rng(w, session, "kapp", step).standard_normal((w.L, w.Hkv, w.d), dtype=np.float32)
    return f32_to_bf16_bits(x)


def q_step(w: Workload, session: int, step: int) -> np.ndarray:
    """float32 [L][Hq][d] decode query of ``session`` at ``step``."""
    return rng(w, session, "q", step).standard_normal((w.L, w.Hq, w.d), dtype=np.float32)


def observes(w: Workload, step: int) -> bool:
    """Whether decode step ``step`` (1-based) is an observation step: every
    k-th one, k = w.obs_interval."""
    return step % w.obs_interval == 0


def q_window(w: Workload, session: int, step: int) -> np.ndarray:
    """float32 [W][L][Hq][d]: the decode queries of steps step - W + 1 ..
    step, oldest first (W = w.window)."""
    return np.stack([q_step(w, session, step - w.window + 1 + j) for j in range(w.window)])


# ---------------------------------------------------------------- device draws

def _torch_seed(w: Workload, session: int, stream: str, step: int) -> int:
    st = seed_sequence(w, session, stream, step).generate_state(2, dtype=np.uint32)
    return int(st[0]) | (int(st[1] & 0x7FFFFFFF) << 32)


def torch_keys(w: Workload, session: int, n: int, device, stream: str = "kpre", step: int = 0):
    """bf16 tensor [n][L][Hkv][d] drawn on ``device`` (large workloads)."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(_torch_seed(w, session, stream, step))
    x = torch.randn((n, w.L, w.Hkv, w.d), generator=g, device=device, dtype=torch.float32)
    return x.to(torch.bfloat16)


def torch_queries(w: Workload, step: int, device):
    """float32 tensor [S][L][Hq][d] drawn on ``device`` for one step."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(_torch_seed(w, 0, "q", step))
    return torch.randn((w.S, w.L, w.Hq, w.d), generator=g, device=device, dtype=torch.float32)


def torch_window_queries(w: Workload, step: int, device):
    """The decode queries of an observation step, drawn on ``device``:
    [S][L][Hq][d] for W = 1, else [S][W][L][Hq][d] for steps step - W + 1 ..
    step, oldest first; None for a step without an observation."""
    import torch
    if not observes(w, step):
        return None
    if w.window == 1:
        return torch_queries(w, step, device)
    return torch.stack([torch_queries(w, step - w.window + 1 + j, device) for j in range(w.window)],
                       dim=1).contiguous()


def torch_append_keys(w: Workload, step: int, device):
    """bf16 tensor [S][L][Hkv][d] drawn on ``device`` for one step."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(_torch_seed(w, 0, "kapp", step))
    x = torch.randn((w.S, w.L, w.Hkv, w.d), generator=g, device=device, dtype=torch.float32)
    return x.to(torch.bfloat16)


# ---------------------------------------------------------------- planted structure

def planted_tokens(w: Workload, session: int, n0: int, count: int) -> np.ndarray:
    """Seeded subset of prefix positions (outside the system span) that get
    keys along a fixed direction, so that attention concentrates on them."""
    g = rng(w, session, "perm", 1)
    lo = min(w.system_len, n0 - 1)
    return np.sort(g.choice(np.arange(lo, n0), size=min(count, n0 - lo), replace=False))


def planted_direction(w: Workload, session: int) -> np.ndarray:
    """Unit float32 directions [L][Hkv][d], one per (layer, KV head)."""
    u = rng(w, session, "perm", 2).standard_normal((w.L, w.Hkv, w.d))
    u /= np.linalg.norm(u, axis=-1, keepdims=True)
    return u.astype(np.float32)


def planted_keys(w: Workload, session: int, keys_bits: np.ndarray, tokens: np.ndarray,
                 strength) -> np.ndarray:
    """Replace the keys of ``tokens`` by strength * direction (+ the token's
    own key as noise); ``strength`` is a scalar or one value per token."""
    u = planted_direction(w, session)
    k = bf16_bits_to_f32(keys_bits).copy()
    st = np.broadcast_to(np.asarray(strength, dtype=np.float32), (len(tokens),))
    k[tokens] = 0.25 * k[tokens] + st[:, None, None, None] * u[None]
    return f32_to_bf16_bits(k)


def planted_query(w: Workload, session: int, q: np.ndarray, gain: float) -> np.ndarray:
    """Add gain * sqrt(d) * direction of each head's KV group to a query."""
    u = planted_direction(w, session)
    G = w.Hq // w.Hkv
    qq = q.astype(np.float32).copy()
    for h in range(w.Hq):
        qq[:, h, :] += np.float32(gain * np.sqrt(w.d)) * u[:, h // G, :]
    return qq
