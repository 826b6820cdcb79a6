"""Plain CPU oracle of MemDecay's observation step (Sec. III, Alg. 1).

TEST INFRASTRUCTURE ONLY.  Only the test suite, the package entry's smoke
check and the benchmark's CPU-baseline leg may import this module.  The
device path never calls it and shares no code with it.

Arithmetic is float64 throughout.  Keys arrive as bfloat16 bits and are
widened exactly; queries arrive as float32 and are widened exactly; the
region tables arrive as float32 and are widened exactly.  Sessions are
independent, and each one is a list of pages in logical (insertion) order.
A page has a serial number (opening order, never reused) and its member
token slots.  The one decode step of ``Session.step`` takes the paper's
steps in the paper's order:

  append   the step's new token joins the tail page, or opens a page
  O2/O3    attention of the decode query against every cached key, per
           layer and query head, softmax over the cached tokens, averaged
           over heads and layers: the attention mass A_i   (Sec. III-C)
  O4       EWMA of the importance a_i                      (Eq. 2)
  O5       refresh clock: t_ref_i <- t when A_i >= tau     (Eq. 3)
  O6       retention score s_i                              (Eq. 4)
  O7       page score S_p, mean over live members           (Eq. 5)
  O8       when |K_t| > B: evict non-pinned pages in ascending S_p until
           the budget holds                                 (Sec. III-D, Alg. 1)
  O9       drop the evicted pages

Readings where the paper leaves a choice:
  * observation steps and window (Sec. III-C): the caller decides which
    decode steps observe (every k-th one in the workloads; k = 1 is the
    study's setting); a step without an observation only appends.  At an
    observation step the window is the decode queries of the W most recent
    steps, this one last; each attends to the tokens cached now whose
    insertion step is no later than its own, and A_i averages over layers,
    query heads and window queries alike (W = 1 is the study's setting);
    eviction runs at observation steps only (Alg. 1 runs per observation);
  * the mass averages over all L*Hq query heads; query head h reads KV head
    h // (Hq/Hkv); scale 1/sqrt(d); no mask over the cached tokens; the new
    token attends to itself;
  * a new token starts with a = 0 and its own observation applies at once;
  * refresh compares this step's raw A_i with tau = tau_scale / |K_t|, where
    |K_t| counts the cached tokens after the append and before eviction;
  * pinned tokens (region in the pin mask) still get EWMA and refresh but
    score +inf; a page with any pinned member is pinned (+inf);
  * |p| in the page mean is the number of live members;
  * ties in S_p go to the smaller serial (the older page first);
  * if the pinned tokens alone exceed B, every unpinned page is evicted and
    the session is flagged infeasible;
  * optional magnitude-normalised attention term (the change Sec. IV-D
    names, measured against the uniform attention level 1/|K_t|): the score
    uses alpha * |K_t| * a_i in place of alpha * a_i, |K_t| being the same
    count as in tau.  The slower usage memory named with it is the EWMA rate
    rho taken closer to 1; it needs no change here;
  * optional region-aligned pages (the allocator variant Sec. III-D leaves
    to future work): a page holds tokens of one region only.  An appended
    token opens a fresh page when the last page is full or its last token's
    region differs; a prompt is laid out the same way, token by token.  A
    page left at a region boundary is closed for good: it takes no later
    token, also when the pages after it are evicted and it becomes the last
    page again (its unused places were given up when it was closed).  The
    rest of the method is unchanged: page sizes simply vary more, and Eq. 5
    still averages over the live members;
  * optional quantised tier (the first tier of the tiered extension,
    Sec. III-E): after an observation step's eviction, every surviving page
    that is not pinned, is not the page the step's token went to (the last
    page before eviction), is still in full precision and scores
    S_p < quant_threshold is quantised, once and for good.  Each group of
    16 consecutive tokens of the page, per (layer, KV head), gets one scale
    s = max|k| / 448 (float32) and 8-bit codes c = the FP8 E4M3 value
    nearest to k / s (float32 quotient, ties to even, at most 448 in
    magnitude); s = 0 and c = 0 when max|k| = 0.  Attention then uses
    s * c.  (Sec. III-E names low precision without a format; E4M3 is the
    8-bit format the device widens to its MFMA operand type in one
    instruction.)
  * optional offload tier (the second tier of Sec. III-E: pages below a
    second threshold go to host memory and come back when later queries make
    them relevant; below a final threshold they are dropped).  The budget
    bounds the pages in the cache (|K_t| and B count them only); a session
    keeps at most ``offload_pages`` pages in host memory.  At an observation
    step, after the attention over the cached tokens, every offloaded token
    is observed with the same query: its mass is the mean over the (layer,
    query head) rows of the weight exp(x - M_r) / Lambda_r it would take
    next to the cached tokens, M_r and Lambda_r being row r's maximum and
    sum over the cached tokens (so the cached tokens' masses do not change;
    with no cached token the weight is 0).  The EWMA and the refresh test
    (same tau) apply to it as to a cached token, and it is scored by Eq. 4
    and Eq. 5.  An offloaded page with a token refreshed by this step is
    recalled: it rejoins the cache in serial order before the eviction, which
    then counts it.  Offloaded pages that stay and score below
    ``drop_threshold`` are dropped.  Of the pages the eviction removes, those
    that take no more tokens (full) and score at least ``drop_threshold`` go
    to host memory, highest page score first (then the older page), while
    the session's host tier has room; the rest are dropped.  An offloaded
    page keeps its keys as they were (quantised or not).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np


def widen_bf16(bits) -> np.ndarray:
    """bfloat16 bit patterns (uint16) -> float32 values, exactly."""
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def softmax(x: np.ndarray) -> np.ndarray:
    """Textbook softmax of a 1-D float64 vector (shifted by its maximum)."""
    e = np.exp(x - np.max(x))
    return e / np.sum(e)


@dataclass
class Page:
    serial: int
    slots: List[int]
    quant: bool = False     # keys held as E4M3 codes and a scale per 16 tokens
    closed: bool = False    # region-aligned pages: left at a region boundary


E4M3_MAX = 448.0


def e4m3_decode(bits) -> np.ndarray:
    """FP8 E4M3 (OCP, 'FN': bias 7, no infinities, S.1111.111 is NaN) bit
    patterns -> float64 values."""
    b = np.asarray(bits, dtype=np.int64)
    sign = np.where(b & 0x80, -1.0, 1.0)
    e = (b >> 3) & 15
    m = (b & 7).astype(np.float64)
    val = np.where(e == 0, m / 8.0 * 2.0 ** -6, (1.0 + m / 8.0) * np.exp2(e.astype(np.float64) - 7.0))
    val = np.where((e == 15) & ((b & 7) == 7), np.nan, val)
    return sign * val


def e4m3_encode(v) -> np.ndarray:
    """float32 values -> the nearest FP8 E4M3 bit patterns (ties to even),
    magnitudes above 448 saturating to 448; the sign bit is set for v < 0."""
    v = np.asarray(v, dtype=np.float32)
    a = np.abs(v).astype(np.float64)
    sign = np.where(v < 0, 0x80, 0)
    # subnormal range (below 2^-6): steps of 2^-9; code 8 is the smallest normal
    sub = np.rint(a * 512.0)
    mant, ex = np.frexp(a)                      # a = mant 2^ex, mant in [0.5, 1)
    q = np.rint((2.0 * mant - 1.0) * 8.0)       # 3 mantissa bits of a = (2 mant) 2^(ex - 1)
    e = ex - 1 + (q == 8)
    q = np.where(q == 8, 0, q)
    norm = ((e + 7) << 3) | q.astype(np.int64)
    bits = np.where(a < 2.0 ** -6, sub.astype(np.int64), np.minimum(norm, 0x7E))
    return (sign | bits).astype(np.uint8)


def quantise_block(x: np.ndarray):
    """Codes and scale of one group of keys (float32 values, any shape): the
    scale max|x| / 448 and the E4M3 codes of x / scale, both computed in
    float32; an all-zero group gets scale 0 and codes 0."""
    x = np.asarray(x, dtype=np.float32)
    m = np.float32(np.max(np.abs(x))) if x.size else np.float32(0)
    if m == 0:
        return np.zeros(x.shape, np.uint8), np.float32(0)
    s = np.float32(m / np.float32(E4M3_MAX))
    return e4m3_encode(x / s), s


@dataclass
class StepRecord:
    """What one observation step produced, in the session's logical order
    (tokens are listed page by page, as the pages stood after the append)."""
    t: int
    n: int                       # |K_t| after the append, before eviction
    tau: float
    page_serial: np.ndarray      # [m] serials of the pages scored
    page_size: np.ndarray        # [m] live members per page
    page_pinned: np.ndarray      # [m] bool
    page_score: np.ndarray       # [m] S_p (+inf for pinned pages)
    abar: np.ndarray             # [n] attention mass A_i
    a: np.ndarray                # [n] importance after the EWMA
    t_ref: np.ndarray            # [n] refresh clock after this step
    region: np.ndarray           # [n]
    score: np.ndarray            # [n] s_i (+inf for pinned tokens)
    evicted: np.ndarray          # serials evicted this step, ascending
    n_after: int
    infeasible: bool
    # offload tier (empty without it).  The page and token arrays above cover
    # the cached pages at the selection, recalled pages included; n_select
    # counts their tokens (n is still the |K_t| of tau, before the recall).
    n_select: int = -1
    off_serial: np.ndarray = field(default_factory=lambda: np.zeros(0, np.int64))   # observed, after recall
    off_abar: np.ndarray = field(default_factory=lambda: np.zeros(0))     # their tokens, page by page
    off_a: np.ndarray = field(default_factory=lambda: np.zeros(0))
    off_t_ref: np.ndarray = field(default_factory=lambda: np.zeros(0, np.int64))
    off_score: np.ndarray = field(default_factory=lambda: np.zeros(0))
    off_page_score: np.ndarray = field(default_factory=lambda: np.zeros(0))
    recalled: np.ndarray = field(default_factory=lambda: np.zeros(0, np.int64))
    dropped: np.ndarray = field(default_factory=lambda: np.zeros(0, np.int64))       # from host memory
    offloaded_now: np.ndarray = field(default_factory=lambda: np.zeros(0, np.int64))
    off_after: np.ndarray = field(default_factory=lambda: np.zeros(0, np.int64))     # in host memory after


class Session:
    """One agent session's cache and MemDecay state."""

    def __init__(self, *, L: int, Hq: int, Hkv: int, d: int, P: int,
                 b: Sequence[float], lam: Sequence[float], alpha: float,
                 rho: float, tau_scale: float, pinned_mask: int, budget: int,
                 clock: int, region, keys_bits, t_ins=None, t_ref=None, a=None,
                 page_sizes: Optional[Sequence[int]] = None,
                 page_serials: Optional[Sequence[int]] = None,
                 next_serial: Optional[int] = None, capacity: Optional[int] = None,
                 attention_norm: bool = False, region_aligned: bool = False,
                 quant_threshold: float = 0.0, offload_pages: int = 0, drop_threshold: float = 0.0):
        if Hq % Hkv:
            raise ValueError("query heads must be a multiple of KV heads")
        self.L, self.Hq, self.Hkv, self.d, self.P = L, Hq, Hkv, d, P
        self.G = Hq // Hkv
        self.b = np.asarray(b, dtype=np.float64)
        self.lam = np.asarray(lam, dtype=np.float64)
        self.alpha, self.rho, self.tau_scale = float(alpha), float(rho), float(tau_scale)
        self.pinned_mask = int(pinned_mask)
        self.attention_norm = bool(attention_norm)
        self.region_aligned = bool(region_aligned)
        self.quant_threshold = float(quant_threshold)
        self.offload_pages = int(offload_pages)
        self.drop_threshold = float(drop_threshold)
        self.offloaded: List[Page] = []     # pages in host memory, serial order
        self.budget = int(budget)
        self.t = int(clock)

        region = np.asarray(region, dtype=np.int64)
        n = region.shape[0]
        cap = n if capacity is None else max(int(capacity), n)
        # Slot store: slot j holds one token's state; keys layer-major
        # [L][Hkv][slot][d] as their bfloat16 bit patterns, widened exactly
        # wherever they are used.
        self.region = np.zeros(cap, dtype=np.int64)
        self.t_ins = np.zeros(cap, dtype=np.int64)
        self.t_ref = np.zeros(cap, dtype=np.int64)
        self.a = np.zeros(cap, dtype=np.float64)
        self.keys = np.zeros((L, Hkv, cap, d), dtype=np.uint16)
        # quantised tokens: codes [L][Hkv][slot][d] and their group's scale
        self.codes = np.zeros((L, Hkv, cap, d), dtype=np.uint8) if self.quant_threshold > 0 else None
        self.qscale = np.zeros((L, Hkv, cap), dtype=np.float32) if self.quant_threshold > 0 else None
        self.is_quant = np.zeros(cap, dtype=bool)
        self.n_slots = n
        self.region[:n] = region
        self.t_ins[:n] = np.arange(n) if t_ins is None else np.asarray(t_ins)
        self.t_ref[:n] = self.t_ins[:n] if t_ref is None else np.asarray(t_ref)
        if a is not None:
            self.a[:n] = np.asarray(a, dtype=np.float64)
        kb = np.asarray(keys_bits, dtype=np.uint16).reshape(n, L, Hkv, d)
        self.keys[:, :, :n, :] = kb.transpose(1, 2, 0, 3)

        if page_sizes is None:
            page_sizes = (aligned_page_sizes(region, P) if self.region_aligned
                          else [min(P, n - i) for i in range(0, n, P)])
        if sum(page_sizes) != n or any(not 1 <= s <= P for s in page_sizes):
            raise ValueError("page sizes must be in [1, P] and cover the tokens")
        if page_serials is None:
            page_serials = list(range(len(page_sizes)))
        self.pages: List[Page] = []
        pos = 0
        for ser, sz in zip(page_serials, page_sizes):
            self.pages.append(Page(int(ser), list(range(pos, pos + sz))))
            pos += sz
        # region-aligned prompt: every page but the last was left full or at
        # a region boundary
        if self.region_aligned:
            for p in self.pages[:-1]:
                p.closed = True
        self.next_serial = (max(page_serials) + 1 if page_serials else 0) \
            if next_serial is None else int(next_serial)

    # ------------------------------------------------------------ helpers
    def live(self) -> np.ndarray:
        """Slot ids of the cached tokens in logical order."""
        if not self.pages:
            return np.zeros(0, dtype=np.int64)
        return np.concatenate([np.asarray(p.slots, dtype=np.int64) for p in self.pages])

    def n_tokens(self) -> int:
        return sum(len(p.slots) for p in self.pages)

    def is_pinned_region(self, r) -> np.ndarray:
        return ((self.pinned_mask >> np.asarray(r, dtype=np.int64)) & 1).astype(bool)

    def _grow(self, need: int):
        cap = self.region.shape[0]
        if need <= cap:
            return
        new = max(need, 2 * cap)
        for name in ("region", "t_ins", "t_ref"):
            arr = getattr(self, name)
            setattr(self, name, np.concatenate([arr, np.zeros(new - cap, dtype=arr.dtype)]))
        self.a = np.concatenate([self.a, np.zeros(new - cap)])
        self.is_quant = np.concatenate([self.is_quant, np.zeros(new - cap, dtype=bool)])
        k = np.zeros((self.L, self.Hkv, new, self.d), dtype=np.uint16)
        k[:, :, :cap, :] = self.keys
        self.keys = k
        if self.codes is not None:
            c = np.zeros((self.L, self.Hkv, new, self.d), dtype=np.uint8)
            c[:, :, :cap, :] = self.codes
            self.codes = c
            sc = np.zeros((self.L, self.Hkv, new), dtype=np.float32)
            sc[:, :, :cap] = self.qscale
            self.qscale = sc

    # ------------------------------------------------------------ steps
    def append(self, key_bits, region: int):
        """The decode engine caches the step's token (Fig. 1 'append KV')."""
        j = self.n_slots
        self._grow(j + 1)
        self.n_slots += 1
        self.region[j] = int(region)
        self.t_ins[j] = self.t
        self.t_ref[j] = self.t
        self.a[j] = 0.0
        self.keys[:, :, j, :] = np.asarray(key_bits, dtype=np.uint16).reshape(self.L, self.Hkv, self.d)
        tail = self.pages[-1] if self.pages else None
        joins = tail is not None and len(tail.slots) < self.P and not tail.closed
        if joins and self.region_aligned and int(self.region[tail.slots[-1]]) != int(region):
            tail.closed = True      # a region boundary closes the page for good
            joins = False
        if joins:
            tail.slots.append(j)
        else:
            self.pages.append(Page(self.next_serial, [j]))
            self.next_serial += 1

    def key_rows(self, l: int, kv: int, slots: np.ndarray) -> np.ndarray:
        """float64 keys of the given slots at (layer l, KV head kv): the cached
        values, or scale * code for quantised tokens."""
        k = widen_bf16(self.keys[l, kv][slots]).astype(np.float64)
        if self.codes is not None:
            qz = self.is_quant[slots]
            if np.any(qz):
                qs = slots[qz]
                k[qz] = e4m3_decode(self.codes[l, kv][qs]) * \
                    self.qscale[l, kv][qs].astype(np.float64)[:, None]
        return k

    def quantise_page(self, page: Page):
        """The quantised tier for one page, per 16-token group and (l, kv)."""
        slots = np.asarray(page.slots, dtype=np.int64)
        for g0 in range(0, slots.size, 16):
            grp = slots[g0:g0 + 16]
            for l in range(self.L):
                for kv in range(self.Hkv):
                    c, s = quantise_block(widen_bf16(self.keys[l, kv][grp]))
                    self.codes[l, kv][grp] = c
                    self.qscale[l, kv][grp] = s
        self.is_quant[slots] = True
        page.quant = True

    def attention_mass(self, q, live: np.ndarray) -> np.ndarray:
        """A_i: softmax attention of the window's decode queries, averaged
        over the L*Hq query heads and the W window queries (Sec. III-C).
        q is [W][L][Hq][d] (or [L][Hq][d] for W = 1), oldest query first;
        window query w belongs to step t - (W - 1 - w) and sees only the
        tokens inserted at or before that step."""
        q = np.asarray(q, dtype=np.float32).astype(np.float64).reshape(-1, self.L, self.Hq, self.d)
        W = q.shape[0]
        n = live.shape[0]
        mass = np.zeros(n, dtype=np.float64)
        inv_sqrt_d = 1.0 / math.sqrt(self.d)
        for w in range(W):
            seen = self.t_ins[live] <= self.t - (W - 1 - w)
            if not np.any(seen):
                continue
            for l in range(self.L):
                for kv in range(self.Hkv):
                    k = self.key_rows(l, kv, live[seen])                      # [n_seen][d]
                    x = (k @ q[w, l, kv * self.G:(kv + 1) * self.G].T) * inv_sqrt_d   # [n_seen][G]
                    for j in range(self.G):
                        mass[seen] += softmax(x[:, j])
        return mass / (self.L * self.Hq * W)

    def offloaded_mass(self, q, live: np.ndarray, off: np.ndarray) -> np.ndarray:
        """Offload tier: the mass each offloaded token would take from the
        query q ([L][Hq][d], one query) next to the cached tokens ``live``:
        the mean over the (layer, query head) rows of exp(x - M) / Lambda,
        M and Lambda being the row's maximum and sum over the cached tokens;
        0 when no token is cached."""
        mass = np.zeros(off.shape[0], dtype=np.float64)
        if live.shape[0] == 0 or off.shape[0] == 0:
            return mass
        q = np.asarray(q, dtype=np.float32).astype(np.float64).reshape(self.L, self.Hq, self.d)
        inv_sqrt_d = 1.0 / math.sqrt(self.d)
        for l in range(self.L):
            for kv in range(self.Hkv):
                qg = q[l, kv * self.G:(kv + 1) * self.G].T
                x = (self.key_rows(l, kv, live) @ qg) * inv_sqrt_d          # [n][G]
                xo = (self.key_rows(l, kv, off) @ qg) * inv_sqrt_d          # [n_off][G]
                for j in range(self.G):
                    m = np.max(x[:, j])
                    lam = np.sum(np.exp(x[:, j] - m))
                    mass += np.exp(xo[:, j] - m) / lam
        return mass / (self.L * self.Hq)

    def token_scores(self, slots: np.ndarray, n: int) -> np.ndarray:
        """s_i of Eq. 4 at the current clock (+inf for pinned tokens)."""
        r = self.region[slots]
        dt = (self.t - self.t_ref[slots]).astype(np.float64)
        weight = self.alpha * n if self.attention_norm else self.alpha
        score = self.b[r] * np.exp(-self.lam[r] * dt) + weight * self.a[slots]
        return np.where(self.is_pinned_region(r), np.inf, score)

    def page_scores(self, pages: List[Page], score_of_slot: np.ndarray):
        """S_p of Eq. 5 per page: the mean over its members, +inf when any
        member is pinned.  Returns (sizes, pinned, scores)."""
        m = len(pages)
        sizes = np.array([len(p.slots) for p in pages], dtype=np.int64)
        pinned = np.zeros(m, dtype=bool)
        scores = np.zeros(m, dtype=np.float64)
        for i, p in enumerate(pages):
            sl = np.asarray(p.slots, dtype=np.int64)
            pinned[i] = bool(np.any(self.is_pinned_region(self.region[sl])))
            scores[i] = np.inf if pinned[i] else float(np.sum(score_of_slot[sl])) / sizes[i]
        return sizes, pinned, scores

    def step(self, q, new_key_bits=None, new_region: Optional[int] = None) -> StepRecord:
        """One decode step at the next clock value: the append, then, when q
        is given, the observation and eviction of Alg. 1.  Without q the step
        only appends (the record then holds the counts and empty arrays)."""
        self.t += 1
        t = self.t
        if new_key_bits is not None:
            self.append(new_key_bits, new_region)
        live = self.live()
        n = live.shape[0]
        empty = np.zeros(0)
        if q is None:
            return StepRecord(t, n, math.inf, np.zeros(0, np.int64), np.zeros(0, np.int64),
                              np.zeros(0, bool), empty, empty, empty, np.zeros(0, np.int64),
                              np.zeros(0, np.int64), empty, np.zeros(0, np.int64), n, n > self.budget,
                              n_select=n)
        if n == 0 and not self.offloaded:
            return StepRecord(t, 0, math.inf, np.zeros(0, np.int64), np.zeros(0, np.int64),
                              np.zeros(0, bool), empty, empty, empty, np.zeros(0, np.int64),
                              np.zeros(0, np.int64), empty, np.zeros(0, np.int64), 0, False, n_select=0)

        # O2-O3: attention mass of the cached tokens; offload tier: the
        # offloaded tokens' mass next to them.
        abar = self.attention_mass(q, live) if n else empty
        off_pages = list(self.offloaded)
        off = (np.concatenate([np.asarray(p.slots, dtype=np.int64) for p in off_pages])
               if off_pages else np.zeros(0, dtype=np.int64))
        abar_off = self.offloaded_mass(q, live, off)
        # O4: EWMA over every cached token, pinned included (Eq. 2), and over
        # the offloaded tokens observed.
        self.a[live] = self.rho * self.a[live] + (1.0 - self.rho) * abar
        self.a[off] = self.rho * self.a[off] + (1.0 - self.rho) * abar_off
        # O5: refresh clock (Eq. 3), threshold scaled to the uniform level.
        tau = self.tau_scale / n if n else math.inf
        self.t_ref[live[abar >= tau]] = t
        self.t_ref[off[abar_off >= tau]] = t
        # O6: retention score (Eq. 4); pinned tokens bypass scoring.  With the
        # normalised attention term, a_i is measured in units of the uniform
        # attention level 1/n (Sec. IV-D).
        score_of = np.zeros(self.region.shape[0], dtype=np.float64)
        score_of[live] = self.token_scores(live, n)
        score_of[off] = self.token_scores(off, n)
        abar_of = np.zeros(self.region.shape[0], dtype=np.float64)
        abar_of[live] = abar
        abar_of[off] = abar_off
        # Offload tier: pages with a token refreshed now come back, in serial
        # order, before the eviction.
        refreshed_now = set(off[abar_off >= tau].tolist())
        recalled = [p for p in off_pages if any(x in refreshed_now for x in p.slots)]
        if recalled:
            self.offloaded = [p for p in off_pages if p not in recalled]
            self.pages = sorted(self.pages + recalled, key=lambda p: p.serial)
        live_sel = self.live()
        n_sel = live_sel.shape[0]
        # O7: page score (Eq. 5), mean over the page's live members.
        sizes, page_pinned, page_score = self.page_scores(self.pages, score_of)
        serials = np.array([p.serial for p in self.pages], dtype=np.int64)
        o_sizes, o_pinned, o_scores = self.page_scores(self.offloaded, score_of)
        o_serials = np.array([p.serial for p in self.offloaded], dtype=np.int64)
        o_slots = (np.concatenate([np.asarray(p.slots, dtype=np.int64) for p in self.offloaded])
                   if self.offloaded else np.zeros(0, dtype=np.int64))
        # O8: budget-aware page eviction (Alg. 1, min-heap order).
        evicted, n_after, infeasible = select_pages(page_score, serials, sizes,
                                                    page_pinned, n_sel, self.budget)
        # O9: the evicted pages leave the cache (irreversible, Sec. III-E,
        # unless the offload tier keeps them).
        last_serial = self.pages[-1].serial if self.pages else -1
        score_of_page = {int(s_): float(v) for s_, v in zip(serials, page_score)}
        leaving = [p for p in self.pages if int(p.serial) in set(evicted.tolist())]
        if evicted.size:
            gone = set(int(x) for x in evicted)
            self.pages = [p for p in self.pages if p.serial not in gone]
        dropped, offloaded_now = [], []
        if self.offload_pages > 0:
            # offloaded pages below the final threshold are dropped
            keep = []
            for p, v in zip(self.offloaded, o_scores):
                (keep if v >= self.drop_threshold else dropped).append(p)
            self.offloaded = keep
            # full pages leaving the cache at or above it go to host memory,
            # the best first, while there is room
            cand = [p for p in leaving if len(p.slots) == self.P
                    and score_of_page[p.serial] >= self.drop_threshold]
            cand.sort(key=lambda p: (-score_of_page[p.serial], p.serial))
            room = self.offload_pages - len(self.offloaded)
            chosen = cand[:max(room, 0)]
            offloaded_now = sorted(p.serial for p in chosen)
            self.offloaded = sorted(self.offloaded + chosen, key=lambda p: p.serial)
        # Quantised tier (Sec. III-E): surviving pages below the threshold.
        if self.quant_threshold > 0:
            sc_of = {int(s_): (float(v), bool(pn)) for s_, v, pn in zip(serials, page_score, page_pinned)}
            for p in self.pages:
                v, pn = sc_of[p.serial]
                if not pn and not p.quant and p.serial != last_serial and v < self.quant_threshold:
                    self.quantise_page(p)
        return StepRecord(t, n, tau, serials, sizes, page_pinned, page_score, abar_of[live_sel].copy(),
                          self.a[live_sel].copy(), self.t_ref[live_sel].copy(), self.region[live_sel].copy(),
                          score_of[live_sel].copy(), evicted, n_after, infeasible, n_select=n_sel,
                          off_serial=o_serials, off_abar=abar_of[o_slots].copy(), off_a=self.a[o_slots].copy(),
                          off_t_ref=self.t_ref[o_slots].copy(), off_score=score_of[o_slots].copy(),
                          off_page_score=o_scores,
                          recalled=np.array(sorted(p.serial for p in recalled), dtype=np.int64),
                          dropped=np.array(sorted(p.serial for p in dropped), dtype=np.int64),
                          offloaded_now=np.array(offloaded_now, dtype=np.int64),
                          off_after=np.array([p.serial for p in self.offloaded], dtype=np.int64))

    # ------------------------------------------------------------ views
    def state(self):
        """Per-page view: list of (serial, region[], t_ins[], t_ref[], a[])."""
        out = []
        for p in self.pages:
            s = np.asarray(p.slots, dtype=np.int64)
            out.append((p.serial, self.region[s].copy(), self.t_ins[s].copy(),
                        self.t_ref[s].copy(), self.a[s].copy()))
        return out


def aligned_page_sizes(region, P: int) -> List[int]:
    """Page sizes of a token sequence laid out with region-aligned pages:
    tokens in order, each joining the open page unless it is full or holds
    another region."""
    sizes: List[int] = []
    last = None
    for r in np.asarray(region, dtype=np.int64).tolist():
        if sizes and sizes[-1] < P and r == last:
            sizes[-1] += 1
        else:
            sizes.append(1)
        last = r
    return sizes


def select_pages(page_score, serials, sizes, pinned, n: int, budget: int):
    """Greedy page eviction (Alg. 1): while |K| > B, evict the non-pinned page
    of smallest (S_p, serial).  Returns (evicted serials ascending, n after,
    infeasible flag)."""
    evicted = []
    if n > budget:
        cand = [i for i in range(len(serials)) if not pinned[i]]
        cand.sort(key=lambda i: (page_score[i], serials[i]))
        for i in cand:
            if n <= budget:
                break
            evicted.append(int(serials[i]))
            n -= int(sizes[i])
    infeasible = n > budget
    return np.array(sorted(evicted), dtype=np.int64), n, infeasible


def session_from_workload(w, session: int, *, region, keys_bits, b, lam, budget,
                          alpha=None, rho=None, tau_scale=None, capacity=None,
                          attention_norm=None, region_aligned=None, quant_threshold=None) -> Session:
    """A session at the start of decoding: prefix token i has t_ins = t_ref = i,
    importance 0, and the clock stands at n0 (so decode step k runs at
    t = n0 + k)."""
    n0 = int(np.asarray(region).shape[0])
    return Session(L=w.L, Hq=w.Hq, Hkv=w.Hkv, d=w.d, P=w.P, b=b, lam=lam,
                   alpha=w.alpha if alpha is None else alpha,
                   rho=w.rho if rho is None else rho,
                   tau_scale=w.tau_scale if tau_scale is None else tau_scale,
                   pinned_mask=w.pinned_mask, budget=budget, clock=n0,
                   region=region, keys_bits=keys_bits,
                   capacity=capacity if capacity is not None else n0 + w.steps,
                   attention_norm=w.attention_norm if attention_norm is None else attention_norm,
                   region_aligned=w.region_aligned if region_aligned is None else region_aligned,
                   quant_threshold=w.quant_threshold if quant_threshold is None else quant_threshold)
