"""Pins of the oracle's quantised tier (the first tier of the tiered
extension, Sec. III-E): pages scoring below a threshold keep their keys as
8-bit codes with one scale per 16 tokens and (layer, KV head).

The pins check the encoding against its defining properties (range, the
extreme element, the rounding error bound, exact cases), the tier's rules
(which pages, once only) and the attention over decoded keys against a
textbook softmax.
"""
import math

import numpy as np
import pytest
import scipy.special

from oracle import Session, quantise_block

NREG = 7
PLAN, USER = 1, 2


def bf16(x):
    return (np.asarray(x, dtype=np.float32).view(np.uint32) >> 16).astype(np.uint16)


def widen(bits):
    return (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32)


# ------------------------------------------------------------ the encoding

@pytest.mark.parametrize("seed", [0, 1, 2])
def test_codes_range_extreme_and_error_bound(seed):
    rng = np.random.default_rng(seed)
    x = widen(bf16(rng.normal(size=(16, 128)) * rng.uniform(0.1, 10)))
    c, s = quantise_block(x)
    assert c.dtype == np.int8 and c.min() >= -127 and c.max() <= 127
    i = np.unravel_index(np.argmax(np.abs(x)), x.shape)
    assert abs(int(c[i])) == 127 and np.sign(c[i]) == np.sign(x[i])
    # s is max|x| / 127 within one float32 rounding
    assert abs(float(s) - float(np.max(np.abs(x))) / 127) <= 2 ** -23 * float(s)
    # rounding to the nearest code: every decoded value within s/2, plus the
    # float32 rounding of the quotient x / s (|x / s| <= 127, so at most
    # 127 * 2^-24 steps)
    err = np.abs(c.astype(np.float64) * float(s) - x.astype(np.float64))
    assert np.all(err <= float(s) * (0.5 + 128 * 2.0 ** -24))


def test_exact_case_is_lossless():
    # integer multiples of 1/8 with largest magnitude 127/8: the scale is
    # exactly 1/8 and the codes are the integers themselves
    rng = np.random.default_rng(5)
    ints = rng.integers(-127, 128, size=(16, 128))
    ints[3, 7] = -127
    x = (ints / 8.0).astype(np.float32)
    c, s = quantise_block(x)
    assert s == np.float32(0.125)
    assert np.array_equal(c.astype(np.int64), ints)


def test_zero_group():
    c, s = quantise_block(np.zeros((16, 128), np.float32))
    assert s == 0 and not c.any()


def test_rounding_is_half_to_even():
    # codes at exact halves: 0.5 / s and 1.5 / s with s = 1 round to 0 and 2
    x = np.zeros((1, 128), np.float32)
    x[0, 0], x[0, 1], x[0, 2] = 127.0, 0.5, 1.5
    c, s = quantise_block(x)
    assert s == 1.0 and c[0, 1] == 0 and c[0, 2] == 2


# ------------------------------------------------------------ the tier's rules

def session(keys, region, *, thr, P=16, pinned_mask=0, budget=10**9, lam=None, alpha=0.0):
    keys = np.asarray(keys, dtype=np.float32)
    n, d = keys.shape[0], keys.shape[-1]
    return Session(L=1, Hq=1, Hkv=1, d=d, P=P, b=np.ones(NREG),
                   lam=np.zeros(NREG) if lam is None else lam, alpha=alpha, rho=0.9,
                   tau_scale=2.0, pinned_mask=pinned_mask, budget=budget, clock=n, region=region,
                   keys_bits=bf16(keys.reshape(n, 1, 1, d)), quant_threshold=thr)


def test_threshold_zero_changes_nothing():
    rng = np.random.default_rng(7)
    keys = rng.normal(size=(70, 32))
    reg = np.full(70, USER)
    lam = np.full(NREG, 0.05)
    a = session(keys, reg, thr=0.0, lam=lam, alpha=1.0, budget=40)
    b = session(keys, reg, thr=0.0, lam=lam, alpha=1.0, budget=40)
    b.quant_threshold = 0.0
    for _ in range(4):
        q = rng.normal(size=(1, 1, 32)).astype(np.float32)
        kn = bf16(rng.normal(size=(1, 1, 32)))
        ra, rb = a.step(q, kn, USER), b.step(q, kn, USER)
        np.testing.assert_array_equal(ra.abar, rb.abar)
    assert not any(p.quant for p in a.pages)


def test_which_pages_and_once_only():
    # 4 pages: a pinned one, two plain ones, and the open last page.  With an
    # infinite threshold every eligible page is quantised after the first
    # observation: not the pinned page, not the page the token went to.
    n = 60
    reg = np.concatenate([np.full(16, 0), np.full(n - 16, PLAN)])
    rng = np.random.default_rng(8)
    keys = rng.normal(size=(n, 32))
    s = session(keys, reg, thr=math.inf, pinned_mask=1)
    q = rng.normal(size=(1, 1, 32)).astype(np.float32)
    kn = bf16(rng.normal(size=(1, 1, 32)))
    s.step(q, kn, PLAN)                      # 61 tokens: pages of 16, 16, 16, 13
    assert [p.quant for p in s.pages] == [False, True, True, False]
    codes_before = s.codes.copy()
    for _ in range(3):                       # the open page fills to 16 ...
        s.step(q, kn, PLAN)
    assert [p.quant for p in s.pages] == [False, True, True, False]
    s.step(q, kn, PLAN)                      # ... and a new page opens: now it goes
    assert [p.quant for p in s.pages] == [False, True, True, True, False]
    # quantised once: the earlier pages' codes are untouched
    old = np.concatenate([s.pages[1].slots, s.pages[2].slots])
    assert np.array_equal(s.codes[0, 0][old], codes_before[0, 0][old])


def test_lossless_keys_give_unchanged_masses():
    # keys that quantise exactly: the masses with and without the tier agree
    rng = np.random.default_rng(9)
    n, d = 48, 32
    ints = rng.integers(-127, 128, size=(n, d))
    for g0 in range(0, n, 16):
        ints[g0, 0] = 127                    # every group reaches 127
    keys = ints / 8.0
    reg = np.full(n, USER)
    a = session(keys, reg, thr=math.inf)
    b = session(keys, reg, thr=0.0)
    q = rng.normal(size=(1, 1, d)).astype(np.float32)
    kn = bf16(np.full((1, 1, d), 0.25))
    for _ in range(3):
        ra, rb = a.step(q, kn, USER), b.step(q, kn, USER)
        np.testing.assert_array_equal(ra.abar, rb.abar)
    assert [p.quant for p in a.pages] == [True, True, True, False]


def test_mass_over_decoded_keys_is_the_textbook_softmax():
    # after quantisation, one head and one layer: A_i is scipy's softmax of
    # q . (s c_i) / sqrt(d), with the codes and scales the tier stored
    rng = np.random.default_rng(10)
    n, d = 40, 64
    keys = rng.normal(size=(n, d)) * 3
    s = session(keys, np.full(n, USER), thr=math.inf)
    q0 = rng.normal(size=(1, 1, d)).astype(np.float32)
    kn = bf16(rng.normal(size=(1, 1, d)))
    s.step(q0, kn, USER)                     # quantises the first two pages
    assert [p.quant for p in s.pages] == [True, True, False]
    q = rng.normal(size=(1, 1, d)).astype(np.float32)
    rec = s.step(q, None, None)
    live = s.live()
    dec = np.where(s.is_quant[live][:, None],
                   s.codes[0, 0][live].astype(np.float64) * s.qscale[0, 0][live][:, None].astype(np.float64),
                   s.keys[0, 0][live].astype(np.float64))
    want = scipy.special.softmax(dec @ q[0, 0].astype(np.float64) / math.sqrt(d))
    np.testing.assert_allclose(rec.abar, want, rtol=1e-12, atol=0)
    # and the decoded keys are within half a step of the cached ones
    err = np.abs(dec - s.keys[0, 0][live])
    assert np.all(err <= s.qscale[0, 0][live][:, None] * (0.5 + 128 * 2.0 ** -24))


def test_groups_of_sixteen_within_a_page_of_64():
    # P = 64: a page holds four groups, each with its own scale
    rng = np.random.default_rng(11)
    n = 130
    keys = rng.normal(size=(n, 16))
    keys[16:32] *= 100.0                     # the second group is much larger
    s = session(keys, np.full(n, USER), thr=math.inf, P=64)
    s.step(rng.normal(size=(1, 1, 16)).astype(np.float32), bf16(np.ones((1, 1, 16))), USER)
    assert [p.quant for p in s.pages] == [True, True, False]
    sc = s.qscale[0, 0][s.pages[0].slots]
    assert len(set(sc[:16].tolist())) == 1 and len(set(sc[16:32].tolist())) == 1
    assert sc[16] > 50 * sc[0]
