"""Arrival generators of the co-run workloads (§8.1 clients: uniform and Poisson
arrivals; closed-loop clients need no generator): exact periodic release times, and
Poisson releases whose inter-arrival gaps are exponential with the requested mean."""
import numpy as np
import pytest
from scipy import stats

from paper_2307_04339_amd import synth


def test_periodic_releases_exact():
    r = synth.periodic_releases(5, 20_000_000)
    assert r.dtype == np.int64
    assert r.tolist() == [0, 20_000_000, 40_000_000, 60_000_000, 80_000_000]
    r = synth.periodic_releases(3, 7, start_ns=100)
    assert r.tolist() == [100, 107, 114]
    assert synth.periodic_releases(0, 10).size == 0


def test_poisson_releases_seeded_and_ordered():
    a = synth.poisson_releases(1000, 15e6, seed=11)
    b = synth.poisson_releases(1000, 15e6, seed=11)
    c = synth.poisson_releases(1000, 15e6, seed=12)
    assert a.dtype == np.int64 and a.size == 1000
    assert np.array_equal(a, b)
    assert not np.array_equal(a, c)
    assert a[0] == 0                      # the first request arrives at the start
    assert np.all(np.diff(a) >= 0)
    s = synth.poisson_releases(4, 1e6, seed=3, start_ns=500)
    assert s[0] == 500


@pytest.mark.parametrize("mean_ns", [15e6, 1e6])
def test_poisson_gaps_are_exponential(mean_ns):
    n = 100_000
    r = synth.poisson_releases(n + 1, mean_ns, seed=7)
    gaps = np.diff(r).astype(np.float64)
    # sample mean within 4 standard errors (the exponential's sd equals its mean); truncation of
    # the cumulative times to whole ns moves a gap by less than 1 ns
    se = mean_ns / np.sqrt(n)
    assert abs(gaps.mean() - mean_ns) < 4 * se + 1.0
    # coefficient of variation of an exponential is 1
    assert abs(gaps.std() / gaps.mean() - 1.0) < 0.02
    # memorylessness shows in the distribution: Kolmogorov-Smirnov against Exp(mean)
    ks = stats.kstest(gaps, "expon", args=(0.0, mean_ns))
    assert ks.pvalue > 1e-3, ks
    # a uniform (periodic) sequence with the same mean is rejected by the same test
    ks_u = stats.kstest(np.full(1000, mean_ns), "expon", args=(0.0, mean_ns))
    assert ks_u.pvalue < 1e-6
