"""Pins of the privacy-accounting oracle (appendix: envelope CDF, x_+, accountant).

* Two-term chi-squared mixture CDF: the values the paper prints for the
  counter-example to Szekely and Bakirov's supremum claim, an independent
  characteristic-function inversion (Imhof's formula, written here), Monte
  Carlo, and exact special cases (equal scales add degrees of freedom).
* Envelope: below 1 the single-coordinate law attains MiddleRegionCDF (x_- = 1);
  from x_+ on the uniform law dominates; x_+ = 1 + 2/(dk) + O(1/k^2) for d = 2.
* Accountant: the Gaussian mechanism's closed-form delta(eps) for one step and
  for composed steps without subsampling, one subsampled step against direct
  integration of E[(1 - e^(eps - L))_+], and an envelope concentrated at c
  equal to plain accounting with sigma sqrt(c).
"""

import math

import numpy as np
import pytest
from scipy import integrate, optimize, stats

from oracle import accountant as ac


def imhof(x, lams, dofs, upper=1e4):
    """P(sum_i lam_i chi^2(dof_i) <= x) by Imhof's inversion of the characteristic function:
    1/2 - (1/pi) int_0^inf sin(theta(u)) / (u rho(u)) du, integrated period by period up to
    `upper` (the remainder decays like upper^(-sum(dof)/2))."""
    lams, dofs = np.asarray(lams, float), np.asarray(dofs, float)

    def f(u):
        th = 0.5 * np.sum(dofs * np.arctan(lams * u)) - 0.5 * x * u
        rho = np.prod((1.0 + lams ** 2 * u ** 2) ** (dofs / 4.0))
        return math.sin(th) / (u * rho)
    edges = np.arange(0.0, upper, 4.0 * math.pi / x)
    tot = sum(integrate.quad(f, a, b, epsabs=1e-15, epsrel=1e-13, limit=200)[0] for a, b in zip(edges[:-1], edges[1:]))
    return 0.5 - tot / math.pi


def test_szekely_counterexample_values():
    # printed: P(chi^2_3/3 <= 1.5) ~ 0.7877; sup_lam P(lam Z1^2 + (1-lam) Z2^2 <= 1.5) ~ 0.7872
    assert abs(ac.chi2_cdf(4.5, 3) - 0.7877) < 5e-5
    lam = np.linspace(0.0, 1.0, 2001)
    rank2 = max(ac.mix2_cdf(1.5, l, 1, 1.0 - l, 1) for l in lam)
    assert abs(rank2 - 0.7872) < 5e-5
    # the mixed form 0.71 Z1^2 + 0.145 (Z2^2 + Z3^2): the paper prints ~0.7961; its exact value
    # (convolution and Imhof agree) is 0.79518, still above both forms above, which is the claim
    mixed = ac.mix2_cdf(1.5, 0.71, 1, 0.145, 2)
    assert abs(mixed - imhof(1.5, [0.71, 0.145], [1, 2])) < 1e-9
    assert abs(mixed - 0.79518) < 1e-5
    assert mixed > ac.chi2_cdf(4.5, 3) > rank2


@pytest.mark.parametrize("x,a,n1,b,n2", [(1.0, 0.3, 1, 0.35, 4), (2.2, 0.05, 20, 0.02, 48),
                                         (0.9, 0.5 / 32, 32, 0.5 / 96, 96), (1.3, 0.9, 2, 0.1 / 3, 3)])
def test_mix2_matches_imhof(x, a, n1, b, n2):
    assert abs(ac.mix2_cdf(x, a, n1, b, n2) - imhof(x, [a, b], [n1, n2])) < 1e-8


def test_mix2_special_cases_and_monte_carlo():
    for (x, s, n1, n2) in [(3.0, 0.5, 4, 6), (10.0, 1.0, 3, 5), (0.2, 0.1, 1, 1)]:
        assert abs(ac.mix2_cdf(x, s, n1, s, n2) - ac.chi2_cdf(x / s, n1 + n2)) < 1e-11
    assert ac.mix2_cdf(2.0, 0.7, 3, 0.0, 5) == ac.chi2_cdf(2.0 / 0.7, 3)
    r = np.random.default_rng(3)
    n = 2_000_000
    v = 0.2 * r.chisquare(6, n) + 0.05 * r.chisquare(10, n)
    p = ac.mix2_cdf(1.6, 0.2, 6, 0.05, 10)
    assert abs(np.mean(v <= 1.6) - p) < 5 * math.sqrt(p * (1 - p) / n)


def test_envelope_regions():
    k, d = 4, 3
    for x in (0.5, 0.9, 0.999):                      # x_- = 1: the single coordinate attains the sup
        mr, arg = ac.middle_region(x, k, d, 11)
        assert abs(mr - ac.vertex_cdf(x, k)) < 1e-10 and arg[2] == 0.0 and arg[1] == 1
    xp = ac.x_plus(k, d, tol=1e-6, n_lambda=11)
    assert 1.0 < xp < 2.0
    for x in (xp + 1e-3, 1.5, 1.9):                  # from x_+ on the uniform law dominates
        assert ac.uniform_cdf(x, k, d) >= ac.middle_region(x, k, d, 11)[0] - 1e-10
    mid = 0.5 * (1.0 + xp)                           # in between a two-level form does better
    assert ac.middle_region(mid, k, d, 11)[0] > max(ac.uniform_cdf(mid, k, d), ac.vertex_cdf(mid, k))
    env = ac.envelope_cdf(np.linspace(0.2, 2.0, 40), k, d, xp, 11)
    assert np.all(np.diff(env) >= -1e-12)


@pytest.mark.parametrize("k", [64, 256])
def test_x_plus_asymptotic_d2(k):
    xp = ac.x_plus(k, 2, tol=1e-8, n_lambda=51)
    assert abs((xp - 1.0) / (2.0 / (2 * k)) - 1.0) < 2e-3


@pytest.mark.parametrize("k,d", [(16, 3), (64, 3), (16, 4)])
def test_x_plus_remainder_is_order_inverse_k_squared(k, d):
    # x_+ = 1 + 2/(dk) + O(1/k^2); the remainder times k^2 stays bounded (about 1 to 2.5 here)
    xp = ac.x_plus(k, d, tol=1e-8, n_lambda=51)
    assert 0.0 < (xp - 1.0 - 2.0 / (d * k)) * k * k < 4.0


def _gauss_eps(mu, delta):
    return optimize.brentq(lambda e: ac.gaussian_delta(e, mu) - delta, 0.0, 100.0)


def test_accountant_gaussian_closed_forms():
    # p = 1 (every sample every step): one step is the Gaussian mechanism with mu = 1/sigma,
    # T steps compose to mu sqrt(T)
    assert abs(ac.epsilon(1.0, 10, 10, 1, 1e-5) / _gauss_eps(1.0, 1e-5) - 1.0) < 1e-6
    assert abs(ac.epsilon(2.0, 40, 40, 9, 1e-5) / _gauss_eps(1.5, 1e-5) - 1.0) < 1e-6
    assert abs(ac.epsilon(3.0, 7, 7, 16, 1e-6) / _gauss_eps(4.0 / 3.0, 1e-6) - 1.0) < 1e-6


def test_accountant_subsampled_step_against_direct_integration():
    sigma, p = 0.8, 0.25
    mu = 1.0 / sigma
    grid, q, qinf = ac.single_step_pld(sigma, p, 1e-4, 20.0)

    def loss(x):   # privacy loss of the Poisson-subsampled Gaussian at output x
        return math.log((1 - p) + p * math.exp(mu * x - mu * mu / 2))

    for eps in (0.5, 1.0, 2.0):
        f = lambda x: max(0.0, 1.0 - math.exp(eps - loss(x))) * ((1 - p) * stats.norm.pdf(x) + p * stats.norm.pdf(x - mu))
        ref, _ = integrate.quad(f, -10, 15, limit=400, epsabs=1e-14)
        assert abs(ac.delta_of_eps(grid, q, qinf, eps) - ref) < 2e-5 * max(ref, 1e-3)


def test_accountant_envelope_point_mass_is_a_rescaled_sigma():
    # Y == c everywhere: a = 1/sqrt(c), the same as plain accounting with sigma sqrt(c)
    e1 = ac.epsilon(1.1, 1000, 100, 2, 1e-5, y=np.array([0.81]), w=np.array([1.0]))
    e2 = ac.epsilon(1.1 * 0.9, 1000, 100, 2, 1e-5)
    assert abs(e1 - e2) < 1e-9
    e3 = ac.epsilon(1.1, 1000, 100, 2, 1e-5, y=np.array([1.0]), w=np.array([1.0]))
    assert abs(e3 - ac.epsilon(1.1, 1000, 100, 2, 1e-5)) < 1e-12
    # more noise, less privacy loss; more sampling, more loss
    assert ac.epsilon(1.5, 1000, 100, 2, 1e-5) < ac.epsilon(1.1, 1000, 100, 2, 1e-5)
    assert ac.epsilon(1.1, 1000, 50, 2, 1e-5) < ac.epsilon(1.1, 1000, 100, 2, 1e-5)


# ---- envelope binning (Algorithm accounting: bins of the envelope law) -----------------------

@pytest.mark.parametrize("c", [0.3141, 1.0 + 1e-9, 2.99])
def test_envelope_bins_step_cdf_puts_one_unit_at_the_midpoint_of_its_bin(c):
    # Y == c: the CDF jumps from 0 to 1 inside the bin (y_{j-1}, y_j] that holds c, so all of
    # the weight sits there and its representative is that bin's midpoint
    y0, y1, n = 0.0, 3.0, 300
    ybar, w = ac.envelope_bins(lambda y: 1.0 if y >= c else 0.0, y0, y1, n)
    edges = np.linspace(y0, y1, n + 1)
    j = int(np.searchsorted(edges, c))               # edges[j - 1] < c <= edges[j]
    assert edges[j - 1] < c <= edges[j]
    assert w[j - 1] == 1.0 and np.count_nonzero(w) == 1
    assert abs(ybar[j - 1] - 0.5 * (edges[j - 1] + edges[j])) < 1e-15
    assert abs(ybar[j - 1] - c) <= 0.5 * (y1 - y0) / n


def test_envelope_bins_linear_cdf_gives_equal_weights_and_midpoints():
    y0, y1, n = 0.5, 2.5, 64
    ybar, w = ac.envelope_bins(lambda y: (y - y0) / (y1 - y0), y0, y1, n)
    assert np.allclose(w, 1.0 / n, rtol=0, atol=1e-15)
    assert np.allclose(ybar, y0 + (np.arange(n) + 0.5) * (y1 - y0) / n, rtol=0, atol=1e-15)


def test_envelope_bins_normalise_a_cdf_that_stops_short_of_one():
    # a law with mass outside [y_min, y_max]: only the increments inside count, rescaled to sum
    # to one (here half the mass, uniform over the range, so still 1/n per bin)
    y0, y1, n = 0.0, 1.0, 50
    ybar, w = ac.envelope_bins(lambda y: 0.25 + 0.5 * y, y0, y1, n)
    assert abs(w.sum() - 1.0) < 1e-14
    assert np.allclose(w, 1.0 / n, rtol=0, atol=1e-15)


def test_envelope_bins_clip_a_cdf_that_dips():
    # a CDF evaluated with a small dip (rounding) never yields negative weights: the running
    # maximum makes it monotone, so the dip's bin and the recovery bin get zero weight
    vals = {0: 0.0, 1: 0.4, 2: 0.39, 3: 0.4, 4: 1.0}
    ybar, w = ac.envelope_bins(lambda y: vals[int(round(y))], 0.0, 4.0, 4)
    assert np.all(w >= 0.0)
    assert np.allclose(w, [0.4, 0.0, 0.0, 0.6], atol=1e-15)


def test_envelope_bins_reproduce_the_chi_square_moments():
    # Y = chi^2(k)/k: mean 1, variance 2/k.  The binned law puts each bin's mass at the bin
    # midpoint.  Its mean is a midpoint Riemann-Stieltjes sum whose h^2 term is
    # (h^2/12) (f(y_max) - f(y_min)) = 0 for a density vanishing at both ends, so it is exact
    # to rounding (a representative at the bin's right edge would be off by h/2); its variance
    # exceeds 2/k by h^2/12, Sheppard's correction for grouping into bins of width h.
    k = 32
    y_max = 1.0 + 12.0 * math.sqrt(2.0 / k)
    for n in (100, 400, 1600):
        h = y_max / n
        ybar, w = ac.envelope_bins(lambda y: ac.vertex_cdf(y, k), 0.0, y_max, n)
        mean = float(np.sum(w * ybar))
        var = float(np.sum(w * ybar ** 2)) - mean * mean
        assert abs(mean - 1.0) < 1e-9, n
        assert abs((var - 2.0 / k) / (h * h / 12.0) - 1.0) < 1e-3, n
