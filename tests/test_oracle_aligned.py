"""Pins of the oracle's region-aligned pages (the allocator variant that
Sec. III-D leaves to future work: a fresh page at every region boundary).

What the variant fixes: no page mixes regions, so a page's score (Eq. 5)
averages one region's tokens only, and the pinned-page collateral of mixed
pages disappears.  What it costs: pages below P tokens at region ends.
"""
import math

import numpy as np
import pytest

from oracle import Session, aligned_page_sizes
from synth import configs as C
from synth import generator as g

NREG = 7
PLAN, USER, TOOL_OUT = 1, 2, 4


def bf16(x):
    return (np.asarray(x, dtype=np.float32).view(np.uint32) >> 16).astype(np.uint16)


def session(region, *, P=16, aligned=True, keys=None, b=None, lam=None, alpha=0.0,
            pinned_mask=0, budget=10**9, clock=None, d=8, seed=0):
    region = np.asarray(region)
    n = region.size
    if keys is None:
        keys = np.random.default_rng(seed).normal(size=(n, 1, 1, d))
    return Session(L=1, Hq=1, Hkv=1, d=d, P=P,
                   b=np.ones(NREG) if b is None else b,
                   lam=np.zeros(NREG) if lam is None else lam,
                   alpha=alpha, rho=0.9, tau_scale=2.0, pinned_mask=pinned_mask,
                   budget=budget, clock=n if clock is None else clock, region=region,
                   keys_bits=bf16(keys), region_aligned=aligned)


def runs(*spec):
    """region codes from (region, length) pairs"""
    return np.concatenate([np.full(ln, r) for r, ln in spec])


# ------------------------------------------------------------ layout

def test_page_sizes_closed_form():
    # runs of 5, 20 and 3 tokens at P = 16: the 20-run needs a full page
    # and a page of 4; each run starts a page
    assert aligned_page_sizes(runs((1, 5), (2, 20), (3, 3)), 16) == [5, 16, 4, 3]
    # one region: the plain layout
    assert aligned_page_sizes(np.full(40, 2), 16) == [16, 16, 8]
    # a region change at every token: one page per token
    assert aligned_page_sizes(np.arange(9) % 2, 16) == [1] * 9
    assert aligned_page_sizes(np.zeros(0), 16) == []


@pytest.mark.parametrize("P", [16, 64])
def test_page_count_is_sum_of_ceil_over_runs(P):
    reg = g.region_spans(C.get("qwen15_1700"), 0, 1700)
    change = np.flatnonzero(np.diff(reg.astype(np.int64))) + 1
    lens = np.diff(np.concatenate([[0], change, [reg.size]]))
    sizes = aligned_page_sizes(reg, P)
    assert len(sizes) == sum(math.ceil(ln / P) for ln in lens)
    assert sum(sizes) == reg.size and max(sizes) <= P


def test_no_page_mixes_regions_in_a_prefix():
    reg = g.region_spans(C.get("qwen15_1700"), 0, 1700)
    s = session(reg)
    for ser, r, *_ in s.state():
        assert np.all(r == r[0])


def test_append_opens_a_page_at_a_region_change():
    s = session(runs((PLAN, 10)))
    d = 8
    k = bf16(np.ones((1, 1, d)))
    for r in [PLAN, PLAN, USER, USER, USER, PLAN]:
        s.step(None, k, r)
    sizes = [len(p.slots) for p in s.pages]
    assert sizes == [12, 3, 1]
    assert [p.serial for p in s.pages] == [0, 1, 2]
    # the plain allocator keeps filling the first page
    s2 = session(runs((PLAN, 10)), aligned=False)
    for r in [PLAN, PLAN, USER, USER, USER, PLAN]:
        s2.step(None, k, r)
    assert [len(p.slots) for p in s2.pages] == [16]


def test_full_page_still_closes_within_a_region():
    s = session(runs((PLAN, 15)))
    k = bf16(np.ones((1, 1, 8)))
    for _ in range(3):
        s.step(None, k, PLAN)
    assert [len(p.slots) for p in s.pages] == [16, 2]


# ------------------------------------------------------------ special cases

def test_single_region_reduces_to_the_plain_layout():
    # one region in the prefix and in every append: both allocators give the
    # same pages, so every record is identical
    rng = np.random.default_rng(4)
    n, d = 70, 8
    keys = rng.normal(size=(n, 1, 1, d))
    lam = np.full(NREG, 0.05)
    a = session(np.full(n, USER), keys=keys, lam=lam, alpha=1.0, budget=40, d=d)
    b = session(np.full(n, USER), keys=keys, lam=lam, alpha=1.0, budget=40, d=d, aligned=False)
    for step in range(6):
        q = rng.normal(size=(1, 1, d)).astype(np.float32)
        kn = bf16(rng.normal(size=(1, 1, d)))
        ra = a.step(q, kn, USER)
        rb = b.step(q, kn, USER)
        assert ra.page_size.tolist() == rb.page_size.tolist()
        np.testing.assert_array_equal(ra.abar, rb.abar)
        np.testing.assert_array_equal(ra.page_score, rb.page_score)
        assert ra.evicted.tolist() == rb.evicted.tolist()


def test_aligned_page_score_is_its_regions_closed_form():
    # alpha = 0 and no refresh yet: every token of a region-aligned page has
    # the same age profile only through t_ref; with every token inserted at
    # t = 0 and t = 30, the page score is exactly b_r exp(-lambda_r 30)
    n = 20
    reg = runs((PLAN, 12), (TOOL_OUT, 8))
    lam = np.zeros(NREG)
    lam[PLAN], lam[TOOL_OUT] = 0.01, 0.2
    bb = np.ones(NREG)
    bb[PLAN], bb[TOOL_OUT] = 0.7, 0.4
    keys = np.zeros((n, 1, 1, 8))       # equal keys: mass 1/n each, below tau = 2/n
    s = Session(L=1, Hq=1, Hkv=1, d=8, P=16, b=bb, lam=lam, alpha=0.0, rho=0.9,
                tau_scale=2.0, pinned_mask=0, budget=10**9, clock=29, region=reg,
                keys_bits=bf16(keys), t_ins=np.zeros(n, np.int64), region_aligned=True)
    rec = s.step(np.ones((1, 1, 8), np.float32))
    assert rec.t == 30
    assert rec.page_size.tolist() == [12, 8]
    np.testing.assert_allclose(rec.page_score, [0.7 * math.exp(-0.01 * 30), 0.4 * math.exp(-0.2 * 30)],
                               rtol=1e-15)
    # the plain layout mixes 4 tool_out tokens into the first page
    s2 = Session(L=1, Hq=1, Hkv=1, d=8, P=16, b=bb, lam=lam, alpha=0.0, rho=0.9,
                 tau_scale=2.0, pinned_mask=0, budget=10**9, clock=29, region=reg,
                 keys_bits=bf16(keys), t_ins=np.zeros(n, np.int64))
    rec2 = s2.step(np.ones((1, 1, 8), np.float32))
    mixed = (12 * 0.7 * math.exp(-0.3) + 4 * 0.4 * math.exp(-6.0)) / 16
    np.testing.assert_allclose(rec2.page_score[0], mixed, rtol=1e-15)


def test_no_pinned_collateral():
    # 10 pinned system tokens and 6 plan tokens: the plain layout puts them in
    # one pinned page; aligned, the plan tokens form their own evictable page
    reg = runs((0, 10), (PLAN, 6))
    s = session(reg, pinned_mask=1, budget=12, alpha=1.0)
    rec = s.step(np.ones((1, 1, 8), np.float32))
    assert rec.page_pinned.tolist() == [True, False]
    assert rec.evicted.tolist() == [1] and rec.n_after == 10
    s2 = session(reg, pinned_mask=1, budget=12, alpha=1.0, aligned=False)
    rec2 = s2.step(np.ones((1, 1, 8), np.float32))
    assert rec2.page_pinned.tolist() == [True]
    assert rec2.evicted.size == 0 and rec2.infeasible


# ------------------------------------------------------------ whole runs

def test_whole_run_invariants():
    w = C.with_overrides(C.get("small_aligned"), steps=24)
    n0 = 450
    reg = g.region_spans(w, 0, n0)
    b, lam = g.region_priors(w)
    s = Session(L=w.L, Hq=w.Hq, Hkv=w.Hkv, d=w.d, P=w.P, b=b[0], lam=lam[0], alpha=w.alpha,
                rho=w.rho, tau_scale=w.tau_scale, pinned_mask=w.pinned_mask,
                budget=int(g.budgets(w, np.array([n0]))[0]), clock=n0, region=reg,
                keys_bits=g.k_prefix(w, 0, n0), region_aligned=True)
    B = s.budget
    for k in range(1, w.steps + 1):
        rec = s.step(g.q_step(w, 0, k), g.k_append(w, 0, k), g.append_region(w, k))
        # every page holds one region and at most P tokens
        for ser, r, *_ in s.state():
            assert np.all(r == r[0]) and 1 <= r.size <= w.P
        # sizes reported with the record cover the tokens
        assert int(rec.page_size.sum()) == rec.n
        if not rec.infeasible:
            assert rec.n_after <= B
            if rec.evicted.size:
                assert rec.n_after > B - w.P


def test_a_page_closed_at_a_region_boundary_stays_closed():
    # 16 system tokens and 5 plan tokens; a user token closes the plan page
    # and opens a page of its own, which the step then evicts (user scores
    # 0, plan 1, system pinned).  The plan page is the last page again, yet
    # a later plan token opens a fresh page: the places the plan page gave up
    # at the boundary are not handed out again.
    b = np.zeros(NREG)
    b[PLAN] = 1.0
    reg = runs((0, 16), (PLAN, 5))
    s = session(reg, b=b, pinned_mask=1, budget=21, alpha=0.0)
    assert [len(p.slots) for p in s.pages] == [16, 5]
    rec = s.step(np.ones((1, 1, 8), np.float32), bf16(np.ones((1, 1, 8))), USER)
    assert rec.page_serial.tolist() == [0, 1, 2] and rec.page_size.tolist() == [16, 5, 1]
    assert rec.evicted.tolist() == [2] and rec.n_after == 21
    assert s.pages[-1].closed
    s.step(None, bf16(np.ones((1, 1, 8))), PLAN)          # a step that only appends
    assert [p.serial for p in s.pages] == [0, 1, 3]
    assert [len(p.slots) for p in s.pages] == [16, 5, 1]
    # the plain layout has no closed pages: the same tokens fill the page
    s2 = session(reg, b=b, pinned_mask=1, budget=21, alpha=0.0, aligned=False)
    rec2 = s2.step(np.ones((1, 1, 8), np.float32), bf16(np.ones((1, 1, 8))), USER)
    assert rec2.page_size.tolist() == [16, 6] and not any(p.closed for p in s2.pages)


def test_prompt_pages_before_the_last_are_closed():
    s = session(runs((PLAN, 5), (USER, 20), (TOOL_OUT, 3)))
    assert [len(p.slots) for p in s.pages] == [5, 16, 4, 3]
    assert [p.closed for p in s.pages] == [True, True, True, False]
    # the open last page takes a token of its own region
    s.step(None, bf16(np.ones((1, 1, 8))), TOOL_OUT)
    assert [len(p.slots) for p in s.pages] == [5, 16, 4, 4]
