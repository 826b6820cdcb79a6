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

from oracle import Session, e4m3_decode, e4m3_encode, quantise_block
from oracle.memdecay import widen_bf16

NREG = 7
PLAN, USER = 1, 2


def bf16(x):
    return (np.asarray(x, dtype=np.float32).view(np.uint32) >> 16).astype(np.uint16)


def widen(bits):
    return (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32)


# ------------------------------------------------------------ the encoding

def test_e4m3_table_follows_the_format():
    # OCP FP8 E4M3 ("FN"): bias 7, three mantissa bits, no infinities
    d = e4m3_decode(np.arange(256))
    assert d[0x38] == 1.0 and d[0x7E] == 448.0 and d[0xFE] == -448.0
    assert d[0x08] == 2.0 ** -6 and d[0x01] == 2.0 ** -9 and d[0x07] == 7 * 2.0 ** -9
    assert d[0x40] == 2.0 and d[0x3C] == 1.5 and d[0x80] == 0.0
    assert np.isnan(d[0x7F]) and np.isnan(d[0xFF])
    fin = d[np.isfinite(d)]
    assert fin.size == 254 and np.all(np.diff(np.sort(np.unique(fin))) > 0)


def test_encode_round_trips_every_code():
    codes = np.array([c for c in range(256) if c not in (0x7F, 0xFF, 0x80)], np.uint8)
    assert np.array_equal(e4m3_encode(e4m3_decode(codes).astype(np.float32)), codes)


def test_encode_rounds_to_nearest_even():
    # midpoints: 1.0625 between 1 and 1.125 (goes to the even mantissa, 1);
    # 1.1875 between 1.125 and 1.25 (to 1.25); subnormal 2^-10 between 0 and
    # 2^-9 (to 0) and 3 * 2^-10 (to 2 * 2^-9); just above a midpoint goes up
    v = np.array([1.0625, 1.1875, 2.0 ** -10, 3 * 2.0 ** -10, 1.0625 + 2.0 ** -20, 500.0, -1.0625], np.float32)
    assert e4m3_decode(e4m3_encode(v)).tolist() == [1.0, 1.25, 0.0, 2.0 ** -8, 1.125, 448.0, -1.0]


def brute_nearest(v):
    grid = e4m3_decode(np.arange(0x7F))                      # the non-negative finite values
    a = abs(float(v))
    return np.sign(v) * grid[np.argmin(np.abs(grid - a))]


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_codes_are_the_nearest_e4m3_values(seed):
    rng = np.random.default_rng(seed)
    x = widen(bf16(rng.normal(size=(16, 128)) * rng.uniform(0.1, 10)))
    c, s = quantise_block(x)
    dec = e4m3_decode(c)
    assert np.all(np.abs(dec) <= 448)
    i = np.unravel_index(np.argmax(np.abs(x)), x.shape)
    assert abs(dec[i]) == 448 and np.sign(dec[i]) == np.sign(x[i])
    assert abs(float(s) - float(np.max(np.abs(x))) / 448) <= 2 ** -23 * float(s)
    # each code is the grid value nearest to the float32 quotient (brute force)
    qt = (x / s).astype(np.float32)
    for idx in zip(*np.unravel_index(rng.choice(x.size, 300, replace=False), x.shape)):
        assert abs(dec[idx] - brute_nearest(qt[idx])) == 0 or \
            abs(abs(dec[idx]) - abs(float(qt[idx]))) == abs(abs(brute_nearest(qt[idx])) - abs(float(qt[idx])))


def test_exact_case_is_lossless():
    # E4M3 values times 1/8 whose largest magnitude is 448 / 8: the scale is
    # exactly 1/8 and the codes are those values
    rng = np.random.default_rng(5)
    vals = e4m3_decode(rng.integers(0, 0x7F, size=(16, 128)))
    vals *= np.where(rng.random((16, 128)) < 0.5, -1.0, 1.0)
    vals[3, 7] = -448.0
    x = (vals / 8.0).astype(np.float32)
    c, s = quantise_block(x)
    assert s == np.float32(0.125)
    assert np.array_equal(e4m3_decode(c), vals)


def test_zero_group():
    c, s = quantise_block(np.zeros((16, 128), np.float32))
    assert s == 0 and not c.any()


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
    vals = e4m3_decode(rng.integers(0, 0x7F, size=(n, d))) * np.where(rng.random((n, d)) < 0.5, -1.0, 1.0)
    for g0 in range(0, n, 16):
        vals[g0, 0] = 448.0                  # every group reaches 448
    keys = vals / 8.0
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
                   e4m3_decode(s.codes[0, 0][live]) * s.qscale[0, 0][live][:, None].astype(np.float64),
                   widen_bf16(s.keys[0, 0][live]).astype(np.float64))
    want = scipy.special.softmax(dec @ q[0, 0].astype(np.float64) / math.sqrt(d))
    np.testing.assert_allclose(rec.abar, want, rtol=1e-12, atol=0)
    # and the decoded keys are within half a grid step of the cached ones:
    # 2^-4 of the value for normal codes, 2^-10 s below them
    k = widen_bf16(s.keys[0, 0][live]).astype(np.float64)
    sc = s.qscale[0, 0][live][:, None].astype(np.float64)
    err = np.abs(dec - k)
    assert np.all(err <= np.abs(k) * (2.0 ** -4 + 2.0 ** -20) + sc * 2.0 ** -10)


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
