"""The seeded workload generator: reproducible, and shaped like the recipe."""
import math

import numpy as np
import pytest

from synth import configs as C
from synth import generator as g


def test_streams_are_reproducible_and_independent():
    w = C.get("qwen15_1700")
    a = g.q_step(w, 0, 3)
    assert np.array_equal(a, g.q_step(w, 0, 3))
    assert not np.array_equal(a, g.q_step(w, 0, 4))
    assert np.array_equal(g.region_spans(w, 0, 1700), g.region_spans(w, 0, 1700))
    assert np.array_equal(g.k_append(w, 0, 9), g.k_append(w, 0, 9))


def test_bf16_rounding_ties_to_even_and_widening_is_exact():
    x = np.array([1.0, 1 + 2**-8, 1 + 3 * 2**-8, 1 + 2**-7, -2.5, 3.0e38], np.float32)
    bits = g.f32_to_bf16_bits(x)
    assert bits.tolist() == [0x3F80, 0x3F80, 0x3F82, 0x3F81, 0xC020, 0x7F62]
    back = g.bf16_bits_to_f32(bits)
    assert np.array_equal(g.f32_to_bf16_bits(back), bits)
    r = np.random.default_rng(0).standard_normal(10000).astype(np.float32)
    err = np.abs(g.bf16_bits_to_f32(g.f32_to_bf16_bits(r)) - r) / np.abs(r)
    assert err.max() <= 2.0**-8           # unit roundoff of an 8-bit significand


@pytest.mark.parametrize("name", ["small", "qwen15_1700", "long32k"])
def test_region_spans(name):
    w = C.get(name)
    n0 = int(g.prefix_lengths(w)[0])
    r = g.region_spans(w, 0, n0)
    assert r.shape == (n0,) and r.dtype == np.uint8
    assert np.all(r[:w.system_len] == C.SYSTEM)
    assert np.all(r[w.system_len:] != C.SYSTEM)
    assert r.max() < C.N_REGIONS


def test_span_lengths_are_geometric_with_the_mean():
    w = C.with_overrides(C.get("small"), system_len=0)
    lens = []
    for s in range(40):
        r = g.region_spans(w, s, 20000)
        cuts = np.flatnonzero(np.diff(r.astype(int)) != 0)
        lens += np.diff(cuts).tolist()
    lens = np.array(lens)
    # consecutive spans of the same region (across a reshuffle) merge, which
    # lengthens the mean by 1/(6*6 - 1); allow 3 %.
    assert abs(lens.mean() / (w.mean_span * 36 / 35) - 1) < 0.03
    assert lens.min() >= 1


@pytest.mark.parametrize("m,P,expect", [(40, 16, 0.316), (512, 16, 0.029), (512, 64, 0.116)])
def test_straddle_fraction(m, P, expect):
    # A page straddles when one of its P-1 inner gaps is a region boundary:
    # 1 - (1 - 1/m)^(P-1) for geometric spans of mean m (Sec. III-D's bound).
    w = C.with_overrides(C.get("small"), system_len=0, mean_span=float(m))
    n = 400000 if m > 100 else 100000
    r = g.region_spans(w, 3, n)
    pages = r[: n // P * P].reshape(-1, P)
    frac = np.mean(np.any(pages != pages[:, :1], axis=1))
    assert expect == pytest.approx(1 - (1 - 1 / m) ** (P - 1), abs=2e-3)
    assert frac == pytest.approx(expect, rel=0.08)


def test_budgets_and_lengths():
    assert g.budgets(C.get("small"), np.array([450])).tolist() == [225]
    assert g.budgets(C.get("qwen15_1700"), np.array([1700])).tolist() == [680]
    assert g.budgets(C.get("qwen3_32x1700"), np.array([1700])).tolist() == [510]
    assert g.budgets(C.get("long32k"), np.array([32768])).tolist() == [8192]
    w = C.get("ragged_p16")
    n0 = g.prefix_lengths(w)
    assert n0.shape == (64,) and n0.min() >= 2048 and n0.max() <= 65536
    assert np.array_equal(n0, g.prefix_lengths(C.get("ragged_p64")))
    B = g.budgets(w, n0)
    assert np.array_equal(B, (n0 * 2) // 10)
    # sessions whose pinned system span exceeds the budget exist by design
    assert 0 < np.sum(B < 1024) < 10


def test_region_priors_follow_the_half_lives():
    w = C.get("small")
    b, lam = g.region_priors(w)
    assert b.shape == (1, 7) and lam.dtype == np.float32
    for r, th in C.HALF_LIVES.items():
        assert math.exp(-float(lam[0, r]) * th) == pytest.approx(0.5, rel=1e-6)
        assert 0.2 <= b[0, r] <= 1.0
    w4 = C.get("ragged_p16")
    b4, lam4 = g.region_priors(w4)
    for r, th in C.HALF_LIVES.items():
        th_s = math.log(2) / lam4[:, r].astype(np.float64)
        assert np.all(th_s >= 0.8 * th * (1 - 1e-6)) and np.all(th_s <= 1.2 * th * (1 + 1e-6))
        assert np.unique(th_s).size > 50
    assert np.all(b4 == b4[0])             # base priorities: once per workload


def test_append_cycle():
    w = C.get("qwen15_1700")
    assert [g.append_region(w, k) for k in range(1, 7)] == [6, 3, 4, 6, 3, 4]
    assert g.append_region(C.get("small"), 5) == C.SCRATCHPAD


def test_page_permutation_is_a_permutation():
    w = C.get("small")
    p = g.page_permutation(w, 100)
    assert sorted(p.tolist()) == list(range(100))
