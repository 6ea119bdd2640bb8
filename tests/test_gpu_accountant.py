"""GPU privacy accounting against the oracle.

The chi-squared CDF and MiddleRegionCDF kernels (fp64) against the oracle's
scipy-based CDF and brute-force supremum, the paper's d = 3 counter-example
evaluated by the kernel, x_+ from the GPU binary search, and eps / noise
multipliers from the GPU accountant (torch fp64 PLD) against the oracle's
numpy accountant, without and with the Hutchinson envelope.
"""

import math

import numpy as np
import pytest
import torch

from oracle import accountant as ac

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def mods():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2605_24879_amd import accountant, dprc
    dprc.lib()
    return dprc, accountant


def _t(x):
    return torch.tensor(np.asarray(x, dtype=np.float64), device="cuda")


@pytest.mark.parametrize("dof", [1, 3, 16, 100, 1000, 32768])
def test_chi2_cdf(mods, dof):
    D, _ = mods
    xs = np.concatenate([np.linspace(0.0, 3.0, 31) * dof, [1e-6 * dof, dof - math.sqrt(dof), dof + 0.5]])
    got = D.dprc_chi2_cdf(_t(xs), dof).cpu().numpy()
    ref = np.array([ac.chi2_cdf(x, dof) for x in xs])
    assert np.all(np.abs(got - ref) <= 1e-12 + 1e-9 * ref)


@pytest.mark.parametrize("k,d,nl,xs", [
    (4, 3, 11, [0.7, 1.0, 1.1, 1.3, 1.9]),
    (2, 5, 6, [0.95, 1.05, 1.2, 1.5]),
    (8, 4, 7, [1.02, 1.06]),
    (1, 2, 21, [0.4, 1.5, 3.0]),
])
def test_middle_region_matches_brute_force(mods, k, d, nl, xs):
    D, _ = mods
    best, arg = D.dprc_envelope_middle(_t(xs), k, d, nl)
    best, arg = best.cpu().numpy(), arg.cpu().numpy()
    lam = ac.lambda_grid(nl)
    for e, x in enumerate(xs):
        ref, rarg = ac.middle_region(x, k, d, nl)
        assert abs(best[e] - ref) < 1e-10, (x, best[e], ref)
        i, j, l = arg[e]
        assert 1 <= i and 1 <= j and i + j <= d and 0 <= l < nl
        assert abs(ac.two_level_cdf(x, int(i), int(j), float(lam[l]), k) - ref) < 1e-10


def test_szekely_counterexample_on_gpu(mods):
    # d = 3, k = 1 at x = 1.5: the best two-level form puts 0.7 on one coordinate and 0.15 on each
    # of the others, above the uniform form 0.7877 and every rank-2 form (0.7872)
    D, _ = mods
    best, arg = D.dprc_envelope_middle(_t([1.5]), 1, 3, 51)
    assert abs(best.item() - 0.79519) < 1e-5
    assert best.item() > ac.chi2_cdf(4.5, 3) > 0.7872
    i, j, l = arg[0].tolist()
    assert (i, j, l) == (2, 1, 30)          # lam = 0.3 on the pair: 0.15 + 0.15, 0.7 on the single one


def test_x_plus(mods):
    _, A = mods
    for k, d in [(4, 3), (16, 2)]:
        assert abs(A.x_plus(k, d, tol=1e-7, n_lambda=11) - ac.x_plus(k, d, tol=1e-7, n_lambda=11)) < 3e-7


def test_epsilon_plain_matches_oracle(mods):
    _, A = mods
    for (sigma, N, B, E, delta) in [(1.1, 1000, 50, 2, 1e-5), (0.9, 600, 64, 3, 1e-6), (2.0, 40, 40, 9, 1e-5)]:
        got = A.epsilon(sigma, N, B, E, delta)
        ref = ac.epsilon(sigma, N, B, E, delta)
        assert abs(got - ref) <= 1e-6 * ref, (got, ref)


def test_epsilon_with_envelope_matches_oracle(mods):
    _, A = mods
    k, d, nl, nb = 8, 4, 7, 600
    y, w = A.envelope_law(k, d, n_bins=nb, n_lambda=nl)
    xp = ac.x_plus(k, d, tol=1e-6, n_lambda=nl)
    y_max = 1.0 + 12.0 * math.sqrt(2.0 / k)
    yr, wr = ac.envelope_bins(lambda v: ac.envelope_cdf([v], k, d, xp, nl)[0], 0.0, y_max, nb)
    assert np.allclose(y.cpu().numpy(), yr, rtol=0, atol=1e-12)
    assert np.max(np.abs(w.cpu().numpy() - wr)) < 1e-8
    got = A.epsilon(1.0, 1000, 50, 2, 1e-5, envelope=(y, w))
    ref = ac.epsilon(1.0, 1000, 50, 2, 1e-5, y=yr, w=wr)
    assert abs(got - ref) <= 1e-5 * ref
    # randomized clipping costs privacy: more eps than deterministic clipping at the same sigma
    assert got > A.epsilon(1.0, 1000, 50, 2, 1e-5)


def test_noise_multiplier_brackets_the_target(mods):
    _, A = mods
    s = A.noise_multiplier(2.0, 1000, 50, 2, 1e-5, tol=1e-3)
    assert A.epsilon(s, 1000, 50, 2, 1e-5) <= 2.0 < A.epsilon(s - 2e-3, 1000, 50, 2, 1e-5)


def test_envelope_bins_kernel_matches_oracle(mods):
    # the binning kernel on a smooth CDF (chi^2(k)/k), a step CDF and a CDF with a dip
    D, _ = mods
    k, y_max = 32, 1.0 + 12.0 * math.sqrt(2.0 / 32)
    for n in (7, 1000, 4000, 70000):
        ys = np.linspace(0.0, y_max, n + 1)
        F = np.array([ac.vertex_cdf(y, k) for y in ys])
        ybar, w = D.dprc_envelope_bins(_t(F), 0.0, y_max)
        yr, wr = ac.envelope_bins(lambda v: ac.vertex_cdf(v, k), 0.0, y_max, n)
        assert np.allclose(ybar.cpu().numpy(), yr, rtol=0, atol=1e-13), n
        assert np.max(np.abs(w.cpu().numpy() - wr)) < 1e-14, n
    vals = np.array([0.0, 0.4, 0.39, 0.4, 1.0])
    ybar, w = D.dprc_envelope_bins(_t(vals), 0.0, 4.0)
    assert np.allclose(w.cpu().numpy(), [0.4, 0.0, 0.0, 0.6], atol=1e-15)
    step = (np.linspace(0.0, 3.0, 301) >= 0.3141).astype(np.float64)
    _, w = D.dprc_envelope_bins(_t(step), 0.0, 3.0)
    w = w.cpu().numpy()
    assert w[31] == 1.0 and np.count_nonzero(w) == 1


@pytest.mark.parametrize("sigma,p,envelope", [(0.8, 0.25, False), (1.1, 0.05, True), (2.0, 1.0, False),
                                              (0.9, 1.0, True)])
def test_step_pld_kernel_matches_oracle(mods, sigma, p, envelope):
    D, A = mods
    h, t_max = 1e-3, 20.0
    y = w = None
    if envelope:
        y, w = A.envelope_law(8, 4, n_bins=300, n_lambda=7)
    q, qi = D.dprc_pld_step(sigma, p, h, int(round(t_max / h)), y, w)
    grid, qr, qir = ac.single_step_pld(sigma, p, h, t_max, None if y is None else y.cpu().numpy(),
                                       None if w is None else w.cpu().numpy())
    got = q.cpu().numpy()
    assert got.shape == qr.shape
    assert np.max(np.abs(got - qr)) < 1e-13
    assert abs(qi.item() - qir) < 1e-13
    assert abs(got.sum() + qi.item() - 1.0) < 1e-12


def test_pld_fold_and_delta_kernels_match_oracle(mods):
    # one composition and delta(eps) at a batch of eps values against the oracle's numpy steps
    D, A = mods
    h, t_max = 1e-3, 8.0
    q, qi = D.dprc_pld_step(0.7, 0.3, h, int(round(t_max / h)))
    grid, qr, qir = ac.single_step_pld(0.7, 0.3, h, t_max)
    q2, qi2 = A._compose2(q, qi, q, qi)
    r2, ri2 = ac._conv_truncated(qr, qir, qr, qir)
    assert np.max(np.abs(q2.cpu().numpy() - r2)) < 1e-12
    assert abs(qi2.item() - ri2) < 1e-12
    eps = np.array([0.0, 0.1, 0.5, 1.0, 2.5, 7.9995, 8.5])
    got = D.dprc_pld_delta(q2, h, qi2, _t(eps)).cpu().numpy()
    ref = np.array([ac.delta_of_eps(grid, r2, ri2, e) for e in eps])
    assert np.max(np.abs(got - ref)) < 1e-12
