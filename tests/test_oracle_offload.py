"""Pins of the oracle's offload tier (the second tier of Sec. III-E: pages
leave the cache for host memory instead of being dropped, come back when
later queries make them relevant again, and are dropped below a final
threshold).

The readings pinned here: the budget counts only cached tokens; an
offloaded token's mass is the weight exp(x - M) / Lambda it would take next
to the cached tokens (M, Lambda over the cached tokens, so their masses do
not change); EWMA, refresh and scores apply to it as to a cached token; a
page with a token refreshed now is recalled before the eviction; full pages
leaving the cache at or above the drop threshold go to host memory, the best
first, while the session's tier has room.
"""
import math

import numpy as np
import pytest
import scipy.special

from oracle import Session

NREG = 7
PLAN, USER = 1, 2


def bf16(x):
    return (np.asarray(x, dtype=np.float32).view(np.uint32) >> 16).astype(np.uint16)


def widen(bits):
    return (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32)


def session(keys, region, *, P=4, budget, offload_pages, drop_threshold=0.0, b=None, lam=None, alpha=0.0,
            pinned_mask=0, clock=None, tau_scale=2.0):
    keys = np.asarray(keys, dtype=np.float32)
    n, d = keys.shape
    return Session(L=1, Hq=1, Hkv=1, d=d, P=P, b=np.ones(NREG) if b is None else b,
                   lam=np.zeros(NREG) if lam is None else lam, alpha=alpha, rho=0.9, tau_scale=tau_scale,
                   pinned_mask=pinned_mask, budget=budget, clock=n if clock is None else clock,
                   region=np.asarray(region), keys_bits=bf16(keys.reshape(n, 1, 1, d)), capacity=n + 8,
                   offload_pages=offload_pages, drop_threshold=drop_threshold)


def zero_query(d=8):
    return np.zeros((1, 1, d), np.float32)


def test_leaving_full_pages_go_to_host_memory_the_best_first():
    # 4 pages of 4 tokens; plan b = 0.3, user b = 0.6, lambda = 0, alpha = 0:
    # page scores (0.3, 0.6, 0.3, 0.6).  A budget of 4 tokens evicts three
    # pages: the two plan pages and the older user page (tie at 0.6: the
    # older goes first).  Room for two: the user page (0.6) and the older
    # plan page (0.3 ties 0.3: the older).
    b = np.ones(NREG)
    b[PLAN], b[USER] = 0.3, 0.6
    reg = [PLAN] * 4 + [USER] * 4 + [PLAN] * 4 + [USER] * 4
    s = session(np.zeros((16, 8)), reg, budget=4, offload_pages=2, b=b)
    rec = s.step(zero_query())
    assert rec.page_score.tolist() == pytest.approx([0.3, 0.6, 0.3, 0.6])
    assert rec.evicted.tolist() == [0, 1, 2] and rec.n_after == 4
    assert rec.offloaded_now.tolist() == [0, 1] and rec.off_after.tolist() == [0, 1]
    assert [p.serial for p in s.pages] == [3]
    # the budget counts the cached tokens only
    assert s.n_tokens() == 4


def test_the_drop_threshold_and_partial_pages_decide_what_is_kept():
    b = np.ones(NREG)
    b[PLAN], b[USER] = 0.3, 0.6
    # 3 full pages and a partial last page (2 tokens), all leaving
    reg = [PLAN] * 4 + [USER] * 4 + [USER] * 4 + [USER] * 2
    s = session(np.zeros((14, 8)), reg, budget=0, offload_pages=8, drop_threshold=0.5, b=b)
    rec = s.step(zero_query())
    assert rec.evicted.tolist() == [0, 1, 2, 3]
    # plan (0.3) is below the threshold; the partial page could still take tokens
    assert rec.offloaded_now.tolist() == [1, 2]
    # once in host memory a page is dropped at the first step its score
    # falls below the threshold: with lambda = 0.01 the user pages (ages
    # about 9.5 and 5.5) leave at 0.6 exp(-0.01 age) >= 0.5 and fall below it
    # as they age, the older page first
    lam = np.zeros(NREG)
    lam[USER] = 0.01
    s2 = session(np.zeros((14, 8)), reg, budget=0, offload_pages=8, drop_threshold=0.5, b=b, lam=lam)
    rec = s2.step(zero_query())
    assert rec.offloaded_now.tolist() == [1, 2]
    drops = {}
    for _ in range(40):
        rec = s2.step(zero_query())
        low = [int(x) for x, v in zip(rec.off_serial, rec.off_page_score) if v < 0.5]
        assert rec.dropped.tolist() == low
        for x in low:
            drops[x] = s2.t
    assert s2.offloaded == [] and drops[1] < drops[2]


def test_an_offloaded_tokens_mass_is_its_weight_next_to_the_cached_tokens():
    # 8 cached tokens with zero keys (logit 0: M = 0, Lambda = 8) and an
    # offloaded page whose keys give logits x_j = q . k_j / sqrt(d): its
    # tokens' mass is exp(x_j) / 8, and the cached tokens' masses stay 1/8.
    d = 8
    rng = np.random.default_rng(3)
    keys = np.zeros((12, d), np.float32)
    keys[:4] = rng.normal(size=(4, d))
    reg = [PLAN] * 4 + [USER] * 8
    b = np.ones(NREG)
    b[PLAN], b[USER] = 0.3, 0.6
    s = session(keys, reg, budget=8, offload_pages=4, b=b, tau_scale=1e9)   # no refresh, no recall
    rec = s.step(zero_query())
    assert rec.offloaded_now.tolist() == [0]
    q = rng.normal(size=(1, 1, d)).astype(np.float32)
    rec = s.step(q)
    k = widen(bf16(keys[:4])).astype(np.float64)
    x = k @ q[0, 0].astype(np.float64) / math.sqrt(d)
    np.testing.assert_allclose(rec.off_abar, np.exp(x) / 8.0, rtol=1e-12)
    np.testing.assert_allclose(rec.abar, np.full(8, 1 / 8), rtol=1e-12)
    # EWMA from a = 0 at the first observation of the page (it was cached,
    # a = 0.1 * (1/12) at the first step), then the offloaded observation
    a0 = 0.1 * (1.0 / 12)
    np.testing.assert_allclose(rec.off_a, 0.9 * a0 + 0.1 * np.exp(x) / 8.0, rtol=1e-12)
    # the general case: the weight next to the cached tokens' softmax
    cached = widen(bf16(keys[4:])).astype(np.float64) @ q[0, 0].astype(np.float64) / math.sqrt(d)
    lam_ = np.sum(np.exp(cached - cached.max()))
    np.testing.assert_allclose(rec.off_abar, np.exp(x - cached.max()) / lam_, rtol=1e-12)


def test_a_page_a_later_query_makes_relevant_is_recalled():
    # The offloaded plan page holds one key along e_3; a query along e_3
    # gives it most of the mass: it refreshes, comes back before the
    # eviction in serial order, and the budget counts it.
    d = 8
    keys = np.zeros((12, d), np.float32)
    keys[1, 3] = 1.0
    reg = [PLAN] * 4 + [USER] * 8
    b = np.ones(NREG)
    b[PLAN], b[USER] = 0.3, 0.6
    s = session(keys, reg, budget=8, offload_pages=4, b=b)
    s.step(zero_query())
    assert [p.serial for p in s.offloaded] == [0]
    q = np.zeros((1, 1, d), np.float32)
    q[0, 0, 3] = 10.0 * math.sqrt(d)
    rec = s.step(q)
    assert rec.recalled.tolist() == [0]
    assert rec.off_serial.tolist() == []                     # observed list after the recall
    assert rec.page_serial.tolist() == [0, 1, 2]             # back in serial order
    assert rec.n == 8 and rec.n_select == 12                 # tau's |K_t|; the selection's count
    assert rec.t_ref[1] == s.t                               # the relevant token refreshed
    # the recalled page now scores b = 0.3 (lambda = 0, alpha = 0), below the
    # user pages: the eviction takes it again, and it goes back to host memory
    assert rec.evicted.tolist() == [0] and rec.offloaded_now.tolist() == [0]


def test_with_no_room_or_no_tier_the_base_policy_is_unchanged():
    rng = np.random.default_rng(5)
    d, n = 8, 40
    keys = rng.normal(size=(n, d)).astype(np.float32)
    reg = rng.integers(1, 7, size=n)
    lam = np.full(NREG, 0.05)
    qs = rng.normal(size=(6, 1, 1, d)).astype(np.float32)
    outs = []
    for kw in (dict(offload_pages=0), dict(offload_pages=4, drop_threshold=math.inf)):
        s = session(keys, reg, budget=17, lam=lam, alpha=0.5, **kw)
        outs.append([s.step(q) for q in qs])
    for r1, r2 in zip(*outs):
        assert r1.evicted.tolist() == r2.evicted.tolist()
        np.testing.assert_array_equal(r1.abar, r2.abar)
        np.testing.assert_array_equal(r1.page_score, r2.page_score)
        assert r2.off_after.size == 0


def test_whole_run_invariants():
    # random keys, planted relevant keys now and then, a decaying prior: the
    # tier never exceeds its capacity, holds full pages only, shares no page
    # with the cache, and every token is cached, offloaded or dropped
    rng = np.random.default_rng(7)
    d, n, P, H = 16, 96, 4, 5
    keys = rng.normal(size=(n, d)).astype(np.float32)
    reg = rng.integers(0, 7, size=n)
    lam = np.array([0.0, 0.02, 0.05, 0.1, 0.2, 0.08, 0.3])
    s = session(keys, reg, P=P, budget=40, offload_pages=H, drop_threshold=0.4, lam=lam, alpha=1.0,
                pinned_mask=1)
    seen_recall = seen_drop = 0
    for k in range(30):
        q = rng.normal(size=(1, 1, d)).astype(np.float32) * (3.0 if k % 4 == 3 else 1.0)
        rec = s.step(q, bf16(rng.normal(size=(1, 1, d))), int(rng.integers(1, 7)))
        seen_recall += rec.recalled.size
        seen_drop += rec.dropped.size
        assert len(s.offloaded) <= H
        assert all(len(p.slots) == P for p in s.offloaded)
        cached = {p.serial for p in s.pages}
        off = {p.serial for p in s.offloaded}
        assert not cached & off
        if not rec.infeasible:
            assert rec.n_after <= s.budget
        # the offloaded pages' serials ascend, and their scores as recorded
        assert [p.serial for p in s.offloaded] == sorted(off)
        assert set(rec.recalled.tolist()) <= set(rec.page_serial.tolist())
    assert seen_recall > 0 and seen_drop > 0
