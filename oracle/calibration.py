"""Plain CPU oracle of the region-lifetime calibration (Sec. IV-B, Eq. 6-7).

TEST INFRASTRUCTURE ONLY, like the rest of this package: only the tests may
import it; the device path shares no code with it.

The calibration aggregates, over observation steps and sessions, the
attention mass received by the tokens of each region at each age, and fits
the log-linear decay of Eq. 6 by count-weighted least squares:

    log A_r(dt) ~= log c_r - lambda_r dt,        half-life ln 2 / lambda_r (Eq. 7)

Readings where the paper leaves a choice: a token's age is the decode steps
since its insertion, t - t_ins; ages are grouped into buckets of
``bucket_steps`` steps and ages past the last bucket are left out; a
bucket's abscissa is the mean age of its observations and its ordinate the
log of their mean mass; the weight of a bucket is its observation count (the
count-weighted fit of Sec. IV-A); buckets without observations, or whose
mean mass is zero, are left out; a region with fewer than two distinct
abscissae has no fit (NaN).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np


@dataclass
class LifetimeStats:
    """Float64 sums per (region, age bucket), over sessions and observations."""
    n_regions: int
    bucket_steps: int
    n_buckets: int
    mass: np.ndarray = field(init=False)
    count: np.ndarray = field(init=False)
    age_sum: np.ndarray = field(init=False)

    def __post_init__(self):
        shape = (self.n_regions, self.n_buckets)
        self.mass = np.zeros(shape, np.float64)
        self.count = np.zeros(shape, np.int64)
        self.age_sum = np.zeros(shape, np.int64)

    def add(self, t: int, t_ins, region, abar):
        """One observation of one session: the live tokens' insertion steps,
        regions and attention masses A_i at clock t."""
        age = t - np.asarray(t_ins, np.int64)
        b = age // self.bucket_steps
        keep = (age >= 0) & (b < self.n_buckets)
        r = np.asarray(region, np.int64)[keep]
        b = b[keep]
        np.add.at(self.mass, (r, b), np.asarray(abar, np.float64)[keep])
        np.add.at(self.count, (r, b), 1)
        np.add.at(self.age_sum, (r, b), age[keep])


def fit_decay(mass, count, age_sum):
    """Eq. 6 per region by count-weighted least squares.

    mass, count, age_sum: [n_regions][n_buckets] sums.  Returns
    (lambda_hat[n_regions], log_c[n_regions]), NaN where a region has fewer
    than two distinct bucket abscissae with positive mean mass."""
    mass = np.asarray(mass, np.float64)
    count = np.asarray(count, np.float64)
    age_sum = np.asarray(age_sum, np.float64)
    n_regions = mass.shape[0]
    lam = np.full(n_regions, np.nan)
    logc = np.full(n_regions, np.nan)
    for r in range(n_regions):
        ok = (count[r] > 0) & (mass[r] > 0)
        if np.count_nonzero(ok) < 2:
            continue
        w = count[r][ok]
        x = age_sum[r][ok] / w            # mean age of the bucket's observations
        y = np.log(mass[r][ok] / w)       # log of their mean mass
        xm = np.sum(w * x) / np.sum(w)
        ym = np.sum(w * y) / np.sum(w)
        sxx = np.sum(w * (x - xm) ** 2)
        if sxx == 0.0:
            continue
        slope = np.sum(w * (x - xm) * (y - ym)) / sxx
        lam[r] = -slope
        logc[r] = ym - slope * xm
    return lam, logc


def half_life(lam):
    """Eq. 7: the age at which the fitted mass halves."""
    return math.log(2.0) / np.asarray(lam, np.float64)
