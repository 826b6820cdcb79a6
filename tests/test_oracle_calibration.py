"""Pins of the calibration oracle (Sec. IV-B, Eq. 6-7) against closed forms
and a library least-squares routine."""
import math

import numpy as np
import pytest

from oracle.calibration import LifetimeStats, fit_decay, half_life


def exact_buckets(lam, c, ages, counts):
    """Sums for buckets whose observations all sit at one age with mass
    c exp(-lam age): the data of an exact Eq. 6 law."""
    counts = np.asarray(counts, np.int64)
    ages = np.asarray(ages, np.float64)
    mass = counts * c * np.exp(-lam * ages)
    return mass[None, :], counts[None, :], (counts * ages).astype(np.int64)[None, :]


@pytest.mark.parametrize("lam,c", [(math.log(2) / 15, 0.02), (math.log(2) / 120, 3e-4), (0.0, 1e-3)])
def test_exact_exponential_law_is_recovered(lam, c):
    m, n, a = exact_buckets(lam, c, [2, 6, 10, 30, 70], [50, 40, 30, 5, 1])
    got, logc = fit_decay(m, n, a)
    assert got[0] == pytest.approx(lam, abs=1e-12)
    assert logc[0] == pytest.approx(math.log(c), rel=1e-12)


def test_half_life_is_ln2_over_rate():
    # Eq. 7: a mass that halves every 40 steps fits to a 40-step half-life.
    ages = np.arange(0, 200, 8)
    m, n, a = exact_buckets(math.log(2) / 40, 0.01, ages, np.full(ages.size, 7))
    lam, _ = fit_decay(m, n, a)
    assert half_life(lam)[0] == pytest.approx(40.0, rel=1e-12)


def test_weighted_fit_matches_library_polyfit():
    # Count-weighted least squares of log mean mass on mean age: numpy's
    # polyfit minimises sum (w_i (y_i - p(x_i)))^2, so weights sqrt(count).
    rng = np.random.default_rng(3)
    nb = 12
    count = rng.integers(1, 500, nb)
    ages = np.arange(nb) * 4 + 1.5
    mass = count * 0.01 * np.exp(-0.05 * ages) * np.exp(rng.normal(0, 0.3, nb))
    age_sum = (count * ages).astype(np.int64)
    lam, logc = fit_decay(mass[None], count[None], age_sum[None])
    x = age_sum / count
    slope, icpt = np.polyfit(x, np.log(mass / count), 1, w=np.sqrt(count))
    assert lam[0] == pytest.approx(-slope, rel=1e-10)
    assert logc[0] == pytest.approx(icpt, rel=1e-10)


def test_heavy_bucket_anchors_the_fit():
    # Sec. IV-A: the count-weighted fit anchors toward observation-dense
    # buckets.  Two light buckets on one line, one dense bucket off it: the
    # fit passes within 1e-4 of the dense bucket's point.
    mass = np.array([[1.0 * 1, math.exp(-1.0) * 1, 0.5 * 10**6]])
    count = np.array([[1, 1, 10**6]])
    age_sum = np.array([[0, 10, 5 * 10**6]])
    lam, logc = fit_decay(mass, count, age_sum)
    assert logc[0] - lam[0] * 5 == pytest.approx(math.log(0.5), abs=1e-4)


def test_regions_without_two_buckets_have_no_fit():
    mass = np.array([[0.1, 0, 0], [0.1, 0.05, 0], [0, 0, 0]])
    count = np.array([[3, 0, 0], [3, 2, 0], [0, 0, 0]])
    age_sum = np.array([[3, 0, 0], [3, 14, 0], [0, 0, 0]])
    lam, _ = fit_decay(mass, count, age_sum)
    assert math.isnan(lam[0]) and not math.isnan(lam[1]) and math.isnan(lam[2])


def test_accumulation_buckets_by_age_since_insertion():
    st = LifetimeStats(n_regions=3, bucket_steps=4, n_buckets=3)
    # clock 20: ages 20-17=3 (bucket 0), 20-12=8 (bucket 2), 20-4=16 (dropped), 20-20=0
    st.add(20, t_ins=[17, 12, 4, 20], region=[1, 2, 1, 1], abar=[0.25, 0.5, 0.125, 0.0625])
    assert st.count[1].tolist() == [2, 0, 0] and st.count[2].tolist() == [0, 0, 1]
    assert st.mass[1, 0] == 0.25 + 0.0625 and st.mass[2, 2] == 0.5
    assert st.age_sum[1, 0] == 3 and st.age_sum[2, 2] == 8
    assert st.count.sum() == 3
