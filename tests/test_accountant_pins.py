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
