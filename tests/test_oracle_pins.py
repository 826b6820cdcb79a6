"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test names the passage it follows.  None of them re-types the oracle's
own formula: they check closed forms, invariants, special cases that reduce
to a textbook routine, and the paper's worked example (Fig. 2).
"""
import math
import os

import numpy as np
import pytest
import scipy.special

from oracle import Session, softmax
from oracle.memdecay import widen_bf16

HERE = os.path.dirname(os.path.abspath(__file__))
NREG = 7


def bf16(x):
    """float -> bf16 bits (test-side, truncation is fine for exact values)."""
    return (np.asarray(x, dtype=np.float32).view(np.uint32) >> 16).astype(np.uint16)


def make_session(keys, *, L=1, Hq=1, Hkv=1, P=16, region=None, b=None, lam=None,
                 alpha=0.0, rho=0.9, tau_scale=2.0, pinned_mask=0, budget=10**9,
                 clock=0, t_ins=None, page_sizes=None, attention_norm=False):
    keys = np.asarray(keys, dtype=np.float32)
    n = keys.shape[0]
    d = keys.shape[-1]
    if region is None:
        region = np.full(n, 1)
    return Session(L=L, Hq=Hq, Hkv=Hkv, d=d, P=P,
                   b=np.ones(NREG) if b is None else b,
                   lam=np.zeros(NREG) if lam is None else lam,
                   alpha=alpha, rho=rho, tau_scale=tau_scale, pinned_mask=pinned_mask,
                   budget=budget, clock=clock, region=region,
                   keys_bits=bf16(keys.reshape(n, L, Hkv, d)),
                   t_ins=np.zeros(n, np.int64) if t_ins is None else t_ins,
                   page_sizes=page_sizes, attention_norm=attention_norm)


# ----------------------------------------------------------- O2/O3 attention

def test_softmax_matches_scipy():
    rng = np.random.default_rng(1)
    for n in (1, 2, 7, 64):
        x = rng.normal(size=n) * 5
        np.testing.assert_allclose(softmax(x), scipy.special.softmax(x), rtol=1e-13, atol=0)


def test_mass_is_softmax_on_one_head():
    # L = Hq = Hkv = 1: the mass is exactly the textbook softmax of q.k/sqrt(d).
    rng = np.random.default_rng(2)
    d = 128
    keys = widen_bf16(bf16(rng.normal(size=(9, d))))
    q = rng.normal(size=(1, 1, d)).astype(np.float32)
    s = make_session(keys)
    rec = s.step(q)
    x = keys.astype(np.float64) @ q[0, 0].astype(np.float64) / math.sqrt(d)
    np.testing.assert_allclose(rec.abar, scipy.special.softmax(x), rtol=1e-12)


def test_two_token_scale_closed_form():
    # Two tokens, key e0 * 2 and key 0; q = e0 * c.  The logit gap is 2c/sqrt(d),
    # so the first token's weight is the logistic function of it (scale 1/sqrt d).
    d = 128
    keys = np.zeros((2, d), np.float32)
    keys[0, 0] = 2.0
    q = np.zeros((1, 1, d), np.float32)
    q[0, 0, 0] = 3.0
    rec = make_session(keys).step(q)
    gap = 2.0 * 3.0 / math.sqrt(d)
    assert rec.abar[0] == pytest.approx(1.0 / (1.0 + math.exp(-gap)), rel=1e-14)
    assert rec.abar[1] == pytest.approx(1.0 / (1.0 + math.exp(gap)), rel=1e-14)


def test_mass_sums_to_one_multi_layer_gqa():
    rng = np.random.default_rng(3)
    L, Hq, Hkv, d, n = 3, 6, 2, 128, 37
    keys = rng.normal(size=(n, L, Hkv, d))
    s = make_session(keys, L=L, Hq=Hq, Hkv=Hkv)
    for _ in range(3):
        rec = s.step(rng.normal(size=(L, Hq, d)).astype(np.float32))
        assert abs(rec.abar.sum() - 1.0) < 1e-12
        assert np.all(rec.abar > 0)


def test_equal_keys_give_uniform_mass_and_no_refresh():
    rng = np.random.default_rng(4)
    L, Hq, Hkv, d, n = 2, 4, 2, 128, 23
    one = rng.normal(size=(L, Hkv, d))
    keys = np.broadcast_to(one, (n, L, Hkv, d))
    s = make_session(keys, L=L, Hq=Hq, Hkv=Hkv, t_ins=np.zeros(n, np.int64))
    rec = s.step(rng.normal(size=(L, Hq, d)).astype(np.float32))
    np.testing.assert_allclose(rec.abar, 1.0 / n, rtol=1e-14)
    assert np.all(rec.t_ref == 0)          # 1/n < 2/n: no token refreshes


def test_planted_key_takes_the_mass_and_refreshes():
    d, n = 128, 50
    keys = np.zeros((n, d), np.float32)
    keys[17, 5] = 1.0
    q = np.zeros((1, 1, d), np.float32)
    for c, lo in ((10.0, 0.0), (100.0, 0.9), (400.0, 0.999)):
        q[0, 0, 5] = c * math.sqrt(d)
        s = make_session(keys, clock=7)
        rec = s.step(q)
        assert rec.abar[17] > lo
        x = float(q[0, 0, 5]) / math.sqrt(d)          # the float32 query's exact logit
        assert rec.abar[17] == pytest.approx(1.0 / (1.0 + (n - 1) * math.exp(-x)), rel=1e-12)
    assert rec.t_ref[17] == 8 and np.all(np.delete(rec.t_ref, 17) == 0)


def test_query_head_reads_its_group_kv_head():
    # Hq = 4, Hkv = 2: heads 0,1 read KV head 0 and heads 2,3 read KV head 1.
    # Token 3 is planted in KV head 0 along q[0] and q[1], token 8 in KV head 1
    # along q[2] and q[3]: each takes (almost) all the mass of two of the four
    # heads, so each ends near 1/2.  Reading KV head h % Hkv would give each
    # planted token only one of its heads.
    d, n = 128, 12
    keys = np.zeros((n, 1, 2, d), np.float32)
    keys[3, 0, 0, 0] = 1.0
    keys[8, 0, 1, 1] = 1.0
    q = np.zeros((1, 4, d), np.float32)
    big = 60.0 * math.sqrt(d)
    q[0, 0, 0] = q[0, 1, 0] = big
    q[0, 2, 1] = q[0, 3, 1] = big
    rec = make_session(keys, Hq=4, Hkv=2).step(q)
    assert rec.abar[3] == pytest.approx(0.5, abs=1e-12)
    assert rec.abar[8] == pytest.approx(0.5, abs=1e-12)


def test_new_token_attends_to_itself():
    # The appended token is part of the softmax: planting it takes the mass.
    d = 128
    keys = np.zeros((5, d), np.float32)
    s = make_session(keys)
    newk = np.zeros(d, np.float32)
    newk[9] = 1.0
    q = np.zeros((1, 1, d), np.float32)
    q[0, 0, 9] = 50.0 * math.sqrt(d)
    rec = s.step(q, bf16(newk), 2)
    assert rec.n == 6 and rec.abar[5] > 0.999999


# ----------------------------------------------------------- O4 EWMA (Eq. 2)

@pytest.mark.parametrize("m,factor", [(1, 0.1), (10, 0.6513215599)])
def test_ewma_closed_form_from_zero(m, factor):
    # Constant mass A from a = 0: a_m = (1 - rho^m) A; rho = 0.9.
    n, d = 20, 128
    keys = np.zeros((n, d), np.float32)
    s = make_session(keys, rho=0.9)
    q = np.zeros((1, 1, d), np.float32)
    for _ in range(m):
        rec = s.step(q)
    np.testing.assert_allclose(rec.a, factor / n, rtol=1e-9)


def test_new_token_importance_starts_at_zero():
    n, d = 9, 128
    s = make_session(np.zeros((n, d), np.float32), rho=0.75)
    q = np.zeros((1, 1, d), np.float32)
    s.step(q)                                  # old tokens: a = 0.25/9
    rec = s.step(q, bf16(np.zeros(d)), 3)      # new token joins: n = 10
    assert rec.a[-1] == pytest.approx(0.25 / 10, rel=1e-14)
    assert rec.a[0] == pytest.approx(0.75 * 0.25 / 9 + 0.25 / 10, rel=1e-14)


def test_pinned_tokens_still_get_ewma_and_refresh():
    d, n = 128, 8
    keys = np.zeros((n, d), np.float32)
    keys[0, 0] = 1.0
    reg = np.array([0] + [2] * (n - 1))
    q = np.zeros((1, 1, d), np.float32)
    q[0, 0, 0] = 30 * math.sqrt(d)
    s = make_session(keys, region=reg, pinned_mask=1, clock=4)
    rec = s.step(q)
    assert rec.a[0] == pytest.approx(0.1 * rec.abar[0], rel=1e-14) and rec.a[0] > 0.09
    assert rec.t_ref[0] == 5
    assert math.isinf(rec.score[0])


# ----------------------------------------------------------- O5 refresh (Eq. 3)

def _mass_target_session(n_prefix, target, d=128):
    """n_prefix zero keys plus an appended key e0; q = e0 * x sqrt(d) with x
    chosen so the appended token's mass is ``target`` among n_prefix + 1."""
    n = n_prefix + 1
    x = math.log(target * (n - 1) / (1.0 - target))
    s = make_session(np.zeros((n_prefix, d), np.float32), clock=10)
    k = np.zeros(d, np.float32)
    k[0] = 1.0
    q = np.zeros((1, 1, d), np.float32)
    q[0, 0, 0] = x * math.sqrt(d)
    return s, k, q


@pytest.mark.parametrize("rel,expect", [(1.001, True), (0.999, False)])
def test_refresh_threshold_counts_tokens_after_append(rel, expect):
    # tau = 2/|K_t| with |K_t| after the append (n = 41).  A mass just above
    # 2/41 refreshes; one just below does not, although it is above 2/42 and
    # below 2/40 (so a count before the append, or after a further token,
    # would decide differently in one of the two cases).
    n = 41
    s, k, q = _mass_target_session(n - 1, rel * 2.0 / n)
    rec = s.step(q, bf16(k), 1)
    assert rec.n == n and rec.tau == pytest.approx(2.0 / n)
    assert rec.abar[-1] == pytest.approx(rel * 2.0 / n, rel=1e-6)
    # The appended token's clock starts at t; refresh also sets it to t, so
    # test the decision on a prefix token instead: plant it the same way.
    kk = np.zeros((n - 1, 128), np.float32)
    kk[4, 0] = 1.0
    s2 = make_session(kk, clock=10)
    x = math.log(rel * 2.0 / n * (n - 1) / (1.0 - rel * 2.0 / n))
    q2 = np.zeros((1, 1, 128), np.float32)
    q2[0, 0, 0] = x * math.sqrt(128)
    rec2 = s2.step(q2, bf16(np.zeros(128)), 1)
    assert rec2.abar[4] == pytest.approx(rel * 2.0 / n, rel=1e-6)
    assert (rec2.t_ref[4] == 11) == expect


def test_refresh_uses_raw_mass_not_importance():
    # After one step a = 0.1 * A < tau even when A >= tau: refresh must follow A.
    n, d = 30, 128
    keys = np.zeros((n, d), np.float32)
    keys[2, 0] = 1.0
    q = np.zeros((1, 1, d), np.float32)
    q[0, 0, 0] = 3.0 * math.sqrt(d)      # A_2 = e^3/(e^3 + 29) ~ 0.41 >> 2/30
    s = make_session(keys, clock=0)
    rec = s.step(q)
    assert rec.a[2] < rec.tau < rec.abar[2]
    assert rec.t_ref[2] == 1


# ----------------------------------------------------------- O6 score (Eq. 4)

def test_half_life_halves_the_structural_term():
    # Eq. 7: lambda = ln 2 / t_half.  Zero queries give A = 1/n < tau, so no
    # refresh: the decay factor at age t_half is 1/2 and at 2 t_half is 1/4.
    t_half = 30
    lam = np.zeros(NREG)
    lam[4] = math.log(2.0) / t_half
    b = np.ones(NREG)
    b[4] = 0.8
    s = make_session(np.zeros((6, 128), np.float32), region=np.full(6, 4), b=b, lam=lam)
    q = np.zeros((1, 1, 128), np.float32)
    got = {}
    for t in range(1, 2 * t_half + 1):
        rec = s.step(q)
        got[t] = rec.score[0]
    assert got[t_half] == pytest.approx(0.4, rel=1e-12)
    assert got[2 * t_half] == pytest.approx(0.2, rel=1e-12)


def test_zero_decay_rate_gives_base_plus_attention():
    n, d = 12, 128
    b = np.linspace(0.1, 0.7, NREG)
    s = make_session(np.zeros((n, d), np.float32), region=np.arange(n) % NREG,
                     b=b, lam=np.zeros(NREG), alpha=3.0)
    rec = s.step(np.zeros((1, 1, d), np.float32))
    expect = b[np.arange(n) % NREG] + 3.0 * 0.1 / n
    np.testing.assert_allclose(rec.score, expect, rtol=1e-14)


def test_score_uses_importance_after_this_steps_update():
    n, d = 10, 128
    s = make_session(np.zeros((n, d), np.float32), region=np.full(n, 5),
                     b=np.full(NREG, 0.5), lam=np.full(NREG, 0.1), alpha=2.0, rho=0.5)
    rec = s.step(np.zeros((1, 1, d), np.float32))
    # Age 1 (inserted at 0, now t = 1), a = 0.5 * (1/n).
    assert rec.score[0] == pytest.approx(0.5 * math.exp(-0.1) + 2.0 * 0.5 / n, rel=1e-14)


def _read_fig2():
    rows = []
    with open(os.path.join(HERE, "golden", "fig2_decay_curves.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            reg, b, lam, refr, age, val = line.split()
            rows.append((reg, float(b), float(lam), None if refr == "-" else int(refr),
                         int(age), float(val)))
    return rows


def test_fig2_worked_example():
    # Drive full observation steps: five tokens (system, plan, user, tool_out,
    # retrieval) inserted at t = 0, alpha = 0, no pinning.  Zero queries keep
    # every mass at 1/n (no refresh).  A second session plants the tool_out
    # key at t = 40 so that its mass crosses tau there (the figure's refresh).
    names = ["system", "plan", "user", "tool_in", "tool_out", "retrieval", "scratchpad"]
    rows = _read_fig2()
    b = np.zeros(NREG)
    lam = np.zeros(NREG)
    for reg, bb, ll, _, _, _ in rows:
        b[names.index(reg)], lam[names.index(reg)] = bb, ll
    order = [0, 1, 2, 4, 5]
    d = 128
    keys = np.zeros((len(order), d), np.float32)
    keys[3, 7] = 1.0                       # tool_out's key
    zero_q = np.zeros((1, 1, d), np.float32)
    plant_q = np.zeros((1, 1, d), np.float32)
    plant_q[0, 0, 7] = 20.0 * math.sqrt(d)
    runs = {}
    for refresh in (False, True):
        s = make_session(keys, region=np.array(order), b=b, lam=lam, alpha=0.0)
        scores = {}
        for t in range(1, 101):
            rec = s.step(plant_q if (refresh and t == 40) else zero_q)
            scores[t] = rec.score
        runs[refresh] = scores
    for reg, _, _, refr, age, val in rows:
        idx = order.index(names.index(reg))
        sc = runs[refr is not None]
        assert sc[age][idx] == pytest.approx(val, rel=1e-9), (reg, refr, age)


# ----------------------------------------------------------- O7 page score (Eq. 5)

def test_page_mean_counts_live_members_of_partial_tail():
    n, d = 20, 128                         # pages of 16 and 4 tokens
    reg = np.array([1] * 16 + [2] * 4)
    b = np.zeros(NREG)
    b[1], b[2] = 0.4, 0.8
    s = make_session(np.zeros((n, d), np.float32), region=reg, b=b, lam=np.zeros(NREG))
    rec = s.step(np.zeros((1, 1, d), np.float32))
    np.testing.assert_array_equal(rec.page_size, [16, 4])
    assert rec.page_score[0] == pytest.approx(0.4, rel=1e-15)
    assert rec.page_score[1] == pytest.approx(0.8, rel=1e-15)   # not 0.8 * 4/16


def test_page_with_one_pinned_member_is_pinned():
    n, d = 32, 128
    reg = np.array([0] + [3] * 31)         # page 0 holds one system token
    s = make_session(np.zeros((n, d), np.float32), region=reg, pinned_mask=1, budget=1)
    rec = s.step(np.zeros((1, 1, d), np.float32))
    assert rec.page_pinned.tolist() == [True, False]
    assert math.isinf(rec.page_score[0]) and np.isfinite(rec.page_score[1])
    assert rec.evicted.tolist() == [1] and rec.infeasible   # 16 pinned > B = 1


# ----------------------------------------------------------- appended token clocks

def test_appended_token_clocks_and_score_at_insertion():
    # The new token is inserted at the step's clock: t_ins = t_ref = t, so
    # its age at its own step is 0 and its score is b (alpha = 0); one step
    # later it is b * exp(-lambda).  Zero queries keep every mass below tau.
    d = 128
    b = np.full(NREG, 0.5)
    lam = np.full(NREG, 0.25)
    s = make_session(np.zeros((3, d), np.float32), b=b, lam=lam, clock=20)
    q = np.zeros((1, 1, d), np.float32)
    rec = s.step(q, bf16(np.zeros(d)), 6)
    assert rec.t == 21 and rec.t_ref[-1] == 21
    assert rec.score[-1] == pytest.approx(0.5, rel=1e-15)
    assert s.state()[-1][2][-1] == 21            # t_ins of the new slot
    rec = s.step(q)
    assert rec.score[-1] == pytest.approx(0.5 * math.exp(-0.25), rel=1e-14)


@pytest.mark.parametrize("n_planted,n", [(1, 2), (2, 4)])
def test_refresh_at_exactly_tau(n_planted, n):
    # Planted tokens share the mass equally while the others' weights
    # underflow to exactly 0 in float64 (logit gap 800), so the planted
    # tokens' mass is exactly 1/n_planted = 2/n = tau: refresh is '>='.
    d = 128
    keys = np.zeros((n, d), np.float32)
    keys[:n_planted, 0] = 1.0
    q = np.zeros((1, 1, d), np.float32)
    q[0, 0, 0] = 800.0 * math.sqrt(d)
    s = make_session(keys, clock=3)
    rec = s.step(q)
    assert rec.abar[0] == rec.tau == 2.0 / n
    assert np.all(rec.t_ref[:n_planted] == 4) and np.all(rec.t_ref[n_planted:] == 0)


# ------------------------------------- normalised attention term (Sec. IV-D)

@pytest.mark.parametrize("n", [12, 300])
@pytest.mark.parametrize("m,factor", [(1, 0.1), (10, 0.6513215599)])
def test_normalised_term_at_uniform_attention_is_independent_of_cache_size(n, m, factor):
    # Sec. IV-D proposes measuring the attention term against the uniform
    # attention level.  Equal keys give every token the uniform mass 1/n, so
    # from a = 0 the EWMA gives (1 - rho^m)/n (Eq. 2) and the normalised term
    # is alpha (1 - rho^m) whatever the cache size; the plain term shrinks
    # as 1/n.
    d = 128
    b = np.full(NREG, 0.25)
    for norm, expect in ((True, 0.25 + 1.5 * factor), (False, 0.25 + 1.5 * factor / n)):
        s = make_session(np.zeros((n, d), np.float32), b=b, lam=np.zeros(NREG), alpha=1.5,
                         rho=0.9, attention_norm=norm)
        q = np.zeros((1, 1, d), np.float32)
        for _ in range(m):
            rec = s.step(q)
        np.testing.assert_allclose(rec.score, expect, rtol=1e-9)


def test_normalised_term_of_a_new_token_follows_the_cache_size_at_its_step():
    # A token appended when the cache holds n tokens gets a = (1 - rho)/n at
    # once (its own observation, Eq. 2); the normalised term is then
    # alpha (1 - rho), for n = 10 and again for n = 11 one step later.
    d = 128
    s = make_session(np.zeros((9, d), np.float32), b=np.zeros(NREG), lam=np.zeros(NREG),
                     alpha=2.0, rho=0.75, attention_norm=True)
    q = np.zeros((1, 1, d), np.float32)
    rec = s.step(q, bf16(np.zeros(d)), 3)
    assert rec.n == 10 and rec.score[-1] == pytest.approx(2.0 * 0.25, rel=1e-14)
    rec = s.step(q, bf16(np.zeros(d)), 3)
    assert rec.n == 11 and rec.score[-1] == pytest.approx(2.0 * 0.25, rel=1e-14)
    # the token added a step earlier: a = 0.75 * 0.25/10 + 0.25/11, measured in 1/11
    assert rec.score[-2] == pytest.approx(2.0 * 11 * (0.75 * 0.25 / 10 + 0.25 / 11), rel=1e-13)


# ------------------------------ observation interval and window (Sec. III-C)

def test_window_mass_is_the_mean_of_its_queries_softmaxes():
    # Sec. III-C averages the attention mass over the window as well.  With
    # one layer and one head, and every token inserted before the window,
    # A is the mean of the window queries' textbook softmaxes.
    rng = np.random.default_rng(11)
    d, n, W = 128, 13, 3
    keys = widen_bf16(bf16(rng.normal(size=(n, d))))
    q = rng.normal(size=(W, 1, 1, d)).astype(np.float32)
    s = make_session(keys, clock=5)              # t_ins = 0, steps 4..6 see them all
    rec = s.step(q)
    x = keys.astype(np.float64) @ q[:, 0, 0].astype(np.float64).T / math.sqrt(d)   # [n][W]
    expect = np.mean([scipy.special.softmax(x[:, w]) for w in range(W)], axis=0)
    np.testing.assert_allclose(rec.abar, expect, rtol=1e-12)


def test_window_query_sees_only_tokens_of_its_step():
    # The older window query belongs to the previous step, before this
    # step's token was cached: it cannot attend to it, however well it
    # matches.  Here it matches nothing else (zero keys), the newer query is
    # zero: the new token gets (0 + 1/n) / 2, the others (1/(n-1) + 1/n) / 2.
    d, n0 = 128, 7
    s = make_session(np.zeros((n0, d), np.float32))
    newk = np.zeros(d, np.float32)
    newk[3] = 1.0
    q = np.zeros((2, 1, 1, d), np.float32)
    q[0, 0, 0, 3] = 40.0 * math.sqrt(d)            # older query: aimed at the new key
    rec = s.step(q, bf16(newk), 2)
    n = n0 + 1
    assert rec.abar[-1] == pytest.approx(0.5 / n, rel=1e-12)
    np.testing.assert_allclose(rec.abar[:-1], 0.5 * (1.0 / (n - 1) + 1.0 / n), rtol=1e-12)


def test_steps_without_observation_only_append_and_eviction_waits():
    # Attention is sampled only at observation steps (Sec. III-C); Alg. 1
    # runs per observation.  Steps in between append, advance the clock and
    # leave importance, refresh clocks and pages alone, even over budget.
    d, n0, P = 128, 32, 16
    s = make_session(np.zeros((n0, d), np.float32), P=P, budget=32, b=np.full(NREG, 0.5),
                     lam=np.full(NREG, 0.01))
    q = np.zeros((1, 1, d), np.float32)
    s.step(q)
    a0 = s.a[:n0].copy()
    tr0 = s.t_ref[:n0].copy()
    for k in range(3):
        rec = s.step(None, bf16(np.zeros(d)), 6)
        assert rec.evicted.size == 0 and rec.n == n0 + k + 1
    assert s.t == 4 and s.n_tokens() == n0 + 3
    np.testing.assert_array_equal(s.a[:n0], a0)
    np.testing.assert_array_equal(s.t_ref[:n0], tr0)
    rec = s.step(q, bf16(np.zeros(d)), 6)          # observation: 36 tokens > 32
    assert rec.n == 36 and rec.n_after <= 32 and rec.evicted.size >= 1
