"""Pins of the oracle's eviction (Sec. III-D, Alg. 1, Eq. 1).

* Brute force over every subset of non-pinned pages: when every page holds
  the same number of tokens, evicting pages in ascending S_p order keeps a
  total page score no smaller than any other set of pages meeting the budget
  (Sec. III-D, Eq. 1 taken at page granularity), and
  with one-token pages it keeps the top-B tokens after forcing the pinned
  set (the token-level optimum of Eq. 1).
* Invariants on whole runs of the synthetic workloads: pinned pages are
  never evicted, the budget is met with retained n in (B - P, B], the
  evicted set is the ascending-(S_p, serial) prefix, compaction keeps the
  page order, and an infeasible budget leaves only pinned pages.
"""
import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import Session, select_pages, session_from_workload
from oracle.bruteforce import best_eviction, best_tokens
from synth import configs as C
from synth import generator as g


def _distinct_scores(rng, m):
    return rng.permutation(np.linspace(0.01, 1.0, m)) + rng.uniform(0, 1e-3, m)


@settings(max_examples=150, deadline=None)
@given(seed=st.integers(0, 2**31 - 1), m=st.integers(1, 11), P=st.sampled_from([1, 2, 4, 16]),
       n_pinned=st.integers(0, 3), frac=st.floats(0.0, 1.2))
def test_greedy_equals_bruteforce_on_full_pages(seed, m, P, n_pinned, frac):
    rng = np.random.default_rng(seed)
    scores = _distinct_scores(rng, m)
    pinned = np.zeros(m, bool)
    pinned[rng.choice(m, size=min(n_pinned, m), replace=False)] = True
    scores = np.where(pinned, np.inf, scores)
    sizes = np.full(m, P)
    n = int(sizes.sum())
    budget = int(frac * n)
    serials = np.arange(m) * 3 + 5
    ev, n_after, infeasible = select_pages(scores, serials, sizes, pinned, n, budget)
    best = best_eviction(list(scores), list(sizes), list(pinned), budget)
    if best is None:
        assert infeasible
        assert sorted(ev.tolist()) == sorted(serials[~pinned].tolist())
    else:
        assert not infeasible
        assert ev.tolist() == sorted(serials[list(best)].tolist())


@settings(max_examples=150, deadline=None)
@given(seed=st.integers(0, 2**31 - 1), n=st.integers(1, 12), n_pinned=st.integers(0, 4),
       budget=st.integers(0, 14))
def test_token_pages_give_the_token_level_optimum(seed, n, n_pinned, budget):
    # P = 1: page eviction is token eviction, and greedy = top-B after F (Eq. 1).
    rng = np.random.default_rng(seed)
    scores = _distinct_scores(rng, n)
    pinned = np.zeros(n, bool)
    pinned[rng.choice(n, size=min(n_pinned, n), replace=False)] = True
    sc = np.where(pinned, np.inf, scores)
    ev, n_after, infeasible = select_pages(sc, np.arange(n), np.ones(n, int), pinned, n, budget)
    kept = sorted(set(range(n)) - set(ev.tolist()))
    if pinned.sum() > budget:
        assert infeasible and kept == sorted(np.flatnonzero(pinned).tolist())
    else:
        assert kept == list(best_tokens(list(scores), list(pinned), budget))


def test_ties_go_to_the_older_page():
    sc = np.array([0.5, 0.2, 0.2, 0.2, 0.9])
    serials = np.array([10, 11, 12, 13, 14])
    ev, n_after, inf = select_pages(sc, serials, np.full(5, 16), np.zeros(5, bool), 80, 50)
    assert ev.tolist() == [11, 12]


def test_partial_tail_counts_its_live_tokens():
    # Need 10 tokens gone; the lowest page is a 4-token tail, so greedy takes
    # it and then the next lowest full page (20 tokens evicted).
    sc = np.array([0.3, 0.5, 0.1])
    ev, n_after, inf = select_pages(sc, np.array([0, 1, 2]), np.array([16, 16, 4]),
                                    np.zeros(3, bool), 36, 26)
    assert ev.tolist() == [0, 2] and n_after == 16 and not inf


def _run_workload_checks(w, steps, sessions=None):
    n0s = g.prefix_lengths(w)
    B = g.budgets(w, n0s)
    b, lam = g.region_priors(w)
    for s in (range(w.S) if sessions is None else sessions):
        reg = g.region_spans(w, s, int(n0s[s]))
        sess = session_from_workload(w, s, region=reg, keys_bits=g.k_prefix(w, s, int(n0s[s])),
                                     b=b[s], lam=lam[s], budget=int(B[s]))
        prev_serials = [p.serial for p in sess.pages]
        for k in range(1, steps + 1):
            rec = sess.step(g.q_step(w, s, k), g.k_append(w, s, k), g.append_region(w, k))
            assert rec.t == int(n0s[s]) + k
            assert abs(rec.abar.sum() - 1.0) < 1e-12
            # pinned never evicted
            pinned_serials = set(rec.page_serial[rec.page_pinned].tolist())
            assert not (set(rec.evicted.tolist()) & pinned_serials)
            # budget
            if rec.infeasible:
                assert rec.n_after > B[s]
                assert [p.serial for p in sess.pages] == sorted(pinned_serials)
            else:
                assert rec.n_after <= B[s]
                if rec.evicted.size:
                    assert rec.n_after > B[s] - w.P
            # evicted = prefix of the ascending (S_p, serial) candidate order
            cand = [i for i in range(len(rec.page_serial)) if not rec.page_pinned[i]]
            cand.sort(key=lambda i: (rec.page_score[i], rec.page_serial[i]))
            pref = sorted(int(rec.page_serial[i]) for i in cand[:rec.evicted.size])
            assert rec.evicted.tolist() == pref
            # compaction keeps order; serials ascend along the page list
            after = [p.serial for p in sess.pages]
            assert after == [x for x in rec.page_serial.tolist() if x not in set(rec.evicted.tolist())]
            assert after == sorted(after)
            # all pages but the last are full
            assert all(len(p.slots) == w.P for p in sess.pages[:-1])
            assert sess.n_tokens() == rec.n_after
            prev_serials = after
    return True


def test_invariants_small_workload():
    assert _run_workload_checks(C.get("small"), 32)


def test_invariants_qwen15_shape_shortened():
    w = C.with_overrides(C.get("qwen15_1700"), L=2, steps=24)
    assert _run_workload_checks(w, 24)


def test_infeasible_budget_evicts_every_unpinned_page():
    # 200 pinned system tokens, budget 0.1 * 450 = 45 < 200.
    w = C.with_overrides(C.get("small"), system_len=200, budget_frac=0.1, steps=4)
    n0s = g.prefix_lengths(w)
    B = g.budgets(w, n0s)
    b, lam = g.region_priors(w)
    reg = g.region_spans(w, 0, 450)
    s = session_from_workload(w, 0, region=reg, keys_bits=g.k_prefix(w, 0, 450),
                              b=b[0], lam=lam[0], budget=int(B[0]))
    rec = s.step(g.q_step(w, 0, 1), g.k_append(w, 0, 1), g.append_region(w, 1))
    assert rec.infeasible
    assert all(p.serial in set(rec.page_serial[rec.page_pinned].tolist()) for p in s.pages)
    # 200 system tokens: pages 0..11 full and page 12 holds 8 system tokens
    assert rec.n_after == 13 * 16
    _run_workload_checks(w, 4)


def test_empty_session_then_refill():
    # budget 0 and no pinned tokens: everything goes, the next step opens a
    # fresh page with the next serial.
    d = 128
    s = Session(L=1, Hq=1, Hkv=1, d=d, P=4, b=np.ones(7), lam=np.zeros(7), alpha=1.0,
                rho=0.9, tau_scale=2.0, pinned_mask=0, budget=0, clock=0,
                region=np.full(6, 2), keys_bits=np.zeros((6, 1, 1, d), np.uint16))
    rec = s.step(np.zeros((1, 1, d), np.float32))
    assert rec.evicted.tolist() == [0, 1] and rec.n_after == 0 and not rec.infeasible
    rec = s.step(np.zeros((1, 1, d), np.float32))
    assert rec.n == 0 and rec.evicted.size == 0
    rec = s.step(np.zeros((1, 1, d), np.float32), np.zeros(d, np.uint16), 3)
    assert rec.n == 1 and rec.page_serial.tolist() == [2] and rec.evicted.tolist() == [2]
