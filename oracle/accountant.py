"""fp64 reference of the DP-SGD-RC privacy accounting (appendix "Additional
details to Privacy Accounting": envelope CDF, binary search for x_+, and the
accountant with an envelope CDF).

TEST INFRASTRUCTURE: see the package docstring.

Notation.  chi^2(n) is a chi-squared variable with n degrees of freedom.  For
the Hutchinson estimator with k probes on a layer whose non-projected
dimension is d, the normalised estimate is X(lam) = sum_i lam_i chi^2_i(k)/k
over the simplex lam; its envelope CDF is f(x) = sup_lam P(X(lam) <= x)
(Theorem 1 and the proposition on the extremal envelope):

* below 1 the vertex (one coordinate) dominates: F(x; chi^2(k)/k);
* above x_+ the uniform weights dominate: F(x; chi^2(kd)/(kd));
* in between, the supremum over the two-level forms
  S(i, j, lam) = lam/(ik) chi^2(ik) + (1-lam)/(jk) chi^2(jk), i, j >= 1,
  i + j <= d, lam in [0, 1/2] (MiddleRegionCDF).

Readings (listed in the design notes): Theorem 1 as printed swaps the two
tails relative to the proof and to Algorithm cdf-grid; the proof's version is
used.  The binary search for x_+ tests the single-crossing property directly
(x >= x_+ exactly when the uniform form dominates every two-level form at x);
the printed test "F_unif > 0.5" would send the search to 1 for every d, k.

Library routines used as steps: scipy.special.gammainc (chi-squared CDF),
scipy.integrate.quad (one-dimensional convolution integrals), numpy FFT
(composition of privacy-loss distributions), scipy.optimize.brentq.
"""

import math

import numpy as np
from scipy import integrate, optimize, special, stats


# ---- chi-squared mixtures -------------------------------------------------------------

def chi2_cdf(x, n):
    """P(chi^2(n) <= x)."""
    if x <= 0:
        return 0.0
    return float(special.gammainc(n / 2.0, x / 2.0))


def mix2_cdf(x, a, n1, b, n2):
    """P(a chi^2(n1) + b chi^2(n2) <= x) for independent chi-squares, a, b >= 0.

    The convolution integral over the first term, with u = s^2 so that the
    integrand is smooth at 0 for every n1 >= 1:
      F(x) = int_0^{sqrt(x/a)} 2 s f_{n1}(s^2) P(chi^2(n2) <= (x - a s^2)/b) ds.
    """
    if x <= 0:
        return 0.0
    if a == 0 and b == 0:
        return 1.0
    if a == 0:
        return chi2_cdf(x / b, n2)
    if b == 0:
        return chi2_cdf(x / a, n1)
    smax = math.sqrt(x / a)
    logc = -(n1 / 2.0) * math.log(2.0) - special.gammaln(n1 / 2.0)

    def integrand(s):
        u = s * s
        if u <= 0:
            dens = 2.0 * math.exp(logc) if n1 == 1 else 0.0
        else:
            dens = 2.0 * s * math.exp(logc + (n1 / 2.0 - 1.0) * math.log(u) - u / 2.0)
        return dens * special.gammainc(n2 / 2.0, max(x - a * u, 0.0) / (2.0 * b))

    # break points around the bulk of the first term (concentrated for large n1)
    pts = []
    sd = math.sqrt(2.0 * n1)
    for z in (-6, -3, 0, 3, 6):
        u = n1 + z * sd
        if 0 < u < smax * smax:
            pts.append(math.sqrt(u))
    val, _ = integrate.quad(integrand, 0.0, smax, points=sorted(pts) or None, limit=400,
                            epsabs=1e-14, epsrel=1e-12)
    return min(max(val, 0.0), 1.0)


def two_level_cdf(x, i, j, lam, k):
    """F(x; S(i, j, lam)) with S = lam/(ik) chi^2(ik) + (1-lam)/(jk) chi^2(jk)."""
    return mix2_cdf(x, lam / (i * k), i * k, (1.0 - lam) / (j * k), j * k)


def lambda_grid(n_lambda):
    """The discretised lam in [0, 1/2] of MiddleRegionCDF: n_lambda equally spaced points."""
    return np.linspace(0.0, 0.5, n_lambda)


def middle_region(x, k, d, n_lambda=51):
    """MiddleRegionCDF: max over i, j >= 1, i + j <= d, lam on the grid of F(x; S(i, j, lam)).
    Returns (value, (i, j, lam)); ties keep the first in (i, j, lam) order."""
    best, arg = -1.0, None
    for i in range(1, d):
        for j in range(1, d - i + 1):
            for lam in lambda_grid(n_lambda):
                v = two_level_cdf(x, i, j, float(lam), k)
                if v > best:
                    best, arg = v, (i, j, float(lam))
    return best, arg


def uniform_cdf(x, k, d):
    """F(x; chi^2(kd)/(kd)), the uniform-weights form."""
    return chi2_cdf(x * k * d, k * d)


def vertex_cdf(x, k):
    """F(x; chi^2(k)/k), a single coordinate."""
    return chi2_cdf(x * k, k)


TIE = 1e-10    # the uniform law is itself a two-level form (i = j = d/2, lam = 1/2): equal up to rounding


def x_plus(k, d, tol=1e-6, n_lambda=51):
    """Binary search on [1, 2] for x_+ (Algorithm binary-search-xplus), testing dominance of the
    uniform form over the middle region at the midpoint (to within TIE)."""
    lo, hi = 1.0, 2.0
    while hi - lo > tol:
        mid = 0.5 * (lo + hi)
        mr, _ = middle_region(mid, k, d, n_lambda)
        if uniform_cdf(mid, k, d) >= mr - TIE:
            hi = mid
        else:
            lo = mid
    return 0.5 * (lo + hi)


def envelope_cdf(xs, k, d, xp, n_lambda=51):
    """Envelope CDF on the points xs (Algorithm cdf-grid): vertex below 1, uniform at and above
    x_+, the middle region in between."""
    out = []
    for x in xs:
        if x <= 1.0:
            out.append(vertex_cdf(x, k))
        elif x >= xp:
            out.append(uniform_cdf(x, k, d))
        else:
            out.append(middle_region(x, k, d, n_lambda)[0])
    return np.array(out)


# ---- privacy accountant (Algorithm accounting) -----------------------------------------

def _phi(z):
    return special.ndtr(z)


def _phibar(z):
    return special.ndtr(-z)


def mechanism_kernels(t, sigma, y=None, w=None):
    """alpha, beta, alpha-bar, beta-bar of one step at privacy-loss points t: a Gaussian of scale
    a / sigma with a = 1, or averaged over a = 1/sqrt(y_i) with weights w_i."""
    t = np.asarray(t, dtype=np.float64)
    if y is None:
        mu = np.array([1.0 / sigma])
        w = np.array([1.0])
    else:
        mu = (1.0 / np.sqrt(np.asarray(y, dtype=np.float64))) / sigma
        w = np.asarray(w, dtype=np.float64)
    al = np.zeros_like(t); be = np.zeros_like(t); alb = np.zeros_like(t); beb = np.zeros_like(t)
    for m, wi in zip(mu, w):
        za = -t / m - m / 2.0
        zb = t / m - m / 2.0
        al += wi * _phi(za); alb += wi * _phibar(za)
        be += wi * _phi(zb); beb += wi * _phibar(zb)
    return al, be, alb, beb


def envelope_bins(cdf_fn, y_min, y_max, n_bins):
    """Weights and representative points of Y from its CDF on [y_min, y_max] (bin increments,
    negatives clipped, normalised; midpoints as representatives)."""
    ys = np.linspace(y_min, y_max, n_bins + 1)
    F = np.clip(np.maximum.accumulate(np.array([cdf_fn(y) for y in ys])), 0.0, 1.0)
    w = np.maximum(np.diff(F), 0.0)
    w = w / w.sum()
    ybar = 0.5 * (ys[:-1] + ys[1:])
    return ybar, w


def single_step_pld(sigma, p, h, t_max, y=None, w=None):
    """One subsampled step's privacy-loss distribution on the cell-centred grid t = m h,
    |m| <= n - 1 (n = t_max / h), from the survival function S(t) = P(L > t) at the cut points
    +-(m - 1/2) h: S(t) = p betabar(t + s(t)) + (1 - p) alpha(t + s(t)) with
    s(t) = log(1/p - (1-p)/p e^-t) above the support bound log(1 - p), and S = 1 below it.
    Returns (grid, masses, mass at +infinity)."""
    n = int(round(t_max / h))
    m = np.arange(1, n + 1) - 0.5
    cuts = np.concatenate([-m[::-1] * h, m * h])
    t_min = math.log1p(-p) if p < 1 else -np.inf
    S = np.ones_like(cuts)
    ok = cuts > t_min
    tt = cuts[ok]
    s = np.log(1.0 / p - (1.0 - p) / p * np.exp(-tt)) if p < 1 else np.zeros_like(tt)
    al, be, alb, beb = mechanism_kernels(tt + s, sigma, y, w)
    S[ok] = p * beb + (1.0 - p) * al
    grid = np.arange(-(n - 1), n) * h
    q = np.maximum(S[:-1] - S[1:], 0.0)
    q[0] += max(1.0 - S[0], 0.0)                 # below the first cut
    q_inf = max(float(S[-1]), 0.0)               # above the last cut
    tot = q.sum() + q_inf
    return grid, q / tot, q_inf / tot


def _conv_truncated(a, ainf, b, binf):
    """Composition of two distributions on the same centred grid: linear convolution (FFT),
    negatives clipped; mass past the top of the grid joins the +infinity atom, mass below the
    bottom is folded into the lowest cell."""
    L = len(a)
    n = 2 * L - 1
    size = 1 << (n - 1).bit_length()
    r = np.fft.irfft(np.fft.rfft(a, size) * np.fft.rfft(b, size), size)[:n]
    r = np.maximum(r, 0.0)
    half = (L - 1) // 2                          # r[j] sits at grid index j - half of a centred grid of n
    out = r[half:half + L].copy()
    out[0] += r[:half].sum()
    inf = 1.0 - (1.0 - ainf) * (1.0 - binf)
    top = r[half + L:].sum()
    fin = out.sum() + top
    out *= (1.0 - inf) / fin if fin > 0 else 0.0
    inf += top * (1.0 - inf) / fin if fin > 0 else 0.0
    return out, inf


def compose(grid, q, qinf, steps):
    """Privacy-loss distribution of `steps` independent steps (exponentiation by squaring)."""
    res, rinf = None, 0.0
    base, binf, e = q, qinf, steps
    while e:
        if e & 1:
            if res is None:
                res, rinf = base.copy(), binf
            else:
                res, rinf = _conv_truncated(res, rinf, base, binf)
        e >>= 1
        if e:
            base, binf = _conv_truncated(base, binf, base, binf)
    return grid, res, rinf


def delta_of_eps(grid, q, qinf, eps):
    """delta(eps) = sum over t_j >= eps of q_j (1 - exp(eps - t_j)) + the mass at +infinity."""
    m = grid >= eps
    return float(np.clip(np.sum(q[m] * (1.0 - np.exp(eps - grid[m]))) + qinf, 0.0, 1.0))


def epsilon(sigma, N, B, epochs, delta, h=1e-3, t_max=20.0, y=None, w=None):
    """eps with delta(eps) = delta after ceil(N/B) steps per epoch for `epochs` epochs, each step
    sampling with rate B/N (Algorithm accounting)."""
    T = math.ceil(N / B)
    p = B / N
    grid, q, qinf = single_step_pld(sigma, p, h, t_max, y, w)
    _, q1, i1 = compose(grid, q, qinf, T)
    _, q2, i2 = compose(grid, q1, i1, epochs)
    if delta_of_eps(grid, q2, i2, 0.0) <= delta:
        return 0.0
    hi = float(grid[-1])
    if delta_of_eps(grid, q2, i2, hi) > delta:
        return math.inf
    return optimize.brentq(lambda e: delta_of_eps(grid, q2, i2, e) - delta, 0.0, hi, xtol=1e-10)


def gaussian_delta(eps, mu):
    """delta(eps) of the Gaussian mechanism with sensitivity / noise = mu (closed form)."""
    return float(stats.norm.cdf(-eps / mu + mu / 2.0) - math.exp(eps) * stats.norm.cdf(-eps / mu - mu / 2.0))
