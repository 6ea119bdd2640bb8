"""Privacy accounting for DP-SGD-RC with the Hutchinson estimator.

Appendix "Additional details to Privacy Accounting":

* ``envelope_cdf`` -- Algorithm cdf-grid: the envelope CDF of the normalised
  estimate Y = n_hat / n, the single-coordinate law chi^2(k)/k below 1, the
  uniform law chi^2(kd)/(kd) from x_+ on, and MiddleRegionCDF in between
  (``dprc_envelope_middle`` on the GPU, all two-level forms in parallel);
* ``x_plus`` -- Algorithm binary-search-xplus on [1, 2], deciding at each
  midpoint whether the uniform law dominates every two-level form there
  (single crossing puts x_+ at the first point where it does);
* ``envelope_law`` -- the bins of Algorithm accounting (``dprc_envelope_bins``);
* ``epsilon`` / ``noise_multiplier`` -- Algorithm accounting: one
  Poisson-subsampled Gaussian step whose scale a = 1/sqrt(Y) is averaged over
  the envelope (``dprc_pld_step``: survival function, then cell masses),
  composed over the steps of all epochs by repeated squaring, each product a
  linear convolution (an FFT product, rocFFT through torch.fft) that
  ``dprc_pld_fold`` truncates back to the grid, and delta(eps) evaluated for a
  batch of eps values per round (``dprc_pld_delta``) to narrow a bracket around
  the target.  Without an envelope this is plain DP-SGD accounting.

The PLD lives on the cell-centred grid t = m h, |t| < t_max; mass that
composition pushes past t_max is kept as an atom at +infinity (it counts
fully towards delta) and mass below -t_max is folded into the lowest cell.
Every arithmetic step runs in HIP kernels of libdprc except the FFTs; this
module holds the control flow (searches, the squaring schedule).
"""

import math

import torch

from . import dprc as D


def _dev(device):
    return torch.device(device if device is not None else "cuda")


def chi2_cdf(x, dof, scale=1.0):
    """P(chi^2(dof) <= x * scale) for an fp64 device tensor x (libdprc)."""
    return D.dprc_chi2_cdf(x.to(torch.float64), dof, scale)


def x_plus(k, d, tol=1e-6, n_lambda=51, device=None):
    """x_+ of the Hutchinson envelope for k probes and non-projected dimension d."""
    dev = _dev(device)
    lo, hi = 1.0, 2.0
    while hi - lo > tol:
        mid = 0.5 * (lo + hi)
        xm = torch.tensor([mid], dtype=torch.float64, device=dev)
        mr, _ = D.dprc_envelope_middle(xm, k, d, n_lambda)
        uni = chi2_cdf(xm, k * d, k * d)
        if uni.item() >= mr.item() - 1e-10:        # the uniform law is itself a two-level form
            hi = mid
        else:
            lo = mid
    return 0.5 * (lo + hi)


def envelope_cdf(x, k, d, xp=None, n_lambda=51):
    """Envelope CDF at the points x (fp64 device tensor).  xp: x_+ (searched when None)."""
    x = x.to(torch.float64)
    if xp is None:
        xp = x_plus(k, d, n_lambda=n_lambda, device=x.device)
    out = torch.empty_like(x)
    lowm, highm = x <= 1.0, x >= xp
    midm = ~(lowm | highm)
    if lowm.any():
        out[lowm] = chi2_cdf(x[lowm], k, k)
    if highm.any():
        out[highm] = chi2_cdf(x[highm], k * d, k * d)
    if midm.any():
        out[midm] = D.dprc_envelope_middle(x[midm], k, d, n_lambda)[0]
    return out


def envelope_law(k, d, y_max=None, n_bins=4000, n_lambda=51, device=None):
    """Bins of the envelope law of Y on [0, y_max]: representative points (bin midpoints) and
    weights (CDF increments, made monotone, clipped and normalised) from dprc_envelope_bins."""
    dev = _dev(device)
    if y_max is None:
        y_max = 1.0 + 12.0 * math.sqrt(2.0 / k)            # far into the single-coordinate tail
    ys = torch.linspace(0.0, y_max, n_bins + 1, dtype=torch.float64, device=dev)
    F = envelope_cdf(ys, k, d, n_lambda=n_lambda).contiguous()
    return D.dprc_envelope_bins(F, 0.0, y_max)


def step_pld(sigma, p, h, t_max, y=None, w=None, device=None):
    """(masses on the grid, mass at +infinity [1]) of one subsampled step, on the device."""
    dev = _dev(device if y is None else y.device)
    return D.dprc_pld_step(sigma, p, h, int(round(t_max / h)), y, w, device=dev)


def _compose2(a, ainf, b, binf):
    """Composition of two PLDs on one grid: the FFT product gives their linear convolution,
    dprc_pld_fold truncates it back to the grid and updates the atom."""
    L = a.numel()
    size = 1 << (2 * L - 2).bit_length()
    r = torch.fft.irfft(torch.fft.rfft(a, size) * torch.fft.rfft(b, size), size)
    return D.dprc_pld_fold(r, L, ainf, binf)


def compose(q, qinf, steps):
    """PLD of `steps` independent steps (repeated squaring)."""
    res, rinf = None, None
    base, binf = q, qinf
    while steps:
        if steps & 1:
            res, rinf = (base.clone(), binf.clone()) if res is None else _compose2(res, rinf, base, binf)
        steps >>= 1
        if steps:
            base, binf = _compose2(base, binf, base, binf)
    return res, rinf


EPS_POINTS = 64          # delta evaluations per round of the eps search
EPS_TOL = 1e-10


def _solve_eps(q, qinf, h, delta):
    """eps with delta(eps) = delta: delta is continuous and non-increasing in eps, so each round
    evaluates it at EPS_POINTS points across the bracket and keeps the cell where it crosses."""
    L = q.numel()
    t_top = (L - 1) // 2 * h
    ends = D.dprc_pld_delta(q, h, qinf, torch.tensor([0.0, t_top], dtype=torch.float64, device=q.device)).tolist()
    if ends[0] <= delta:
        return 0.0
    if ends[1] > delta:
        return math.inf
    lo, hi = 0.0, t_top
    while hi - lo > EPS_TOL:
        xs = torch.linspace(lo, hi, EPS_POINTS + 2, dtype=torch.float64, device=q.device)[1:-1].contiguous()
        vals = D.dprc_pld_delta(q, h, qinf, xs).tolist()
        xl = xs.tolist()
        j = next((i for i, v in enumerate(vals) if v <= delta), EPS_POINTS)
        lo, hi = (xl[j - 1] if j > 0 else lo), (xl[j] if j < EPS_POINTS else hi)
    return 0.5 * (lo + hi)


def epsilon(sigma, N, B, epochs, delta, h=1e-3, t_max=20.0, envelope=None, device=None):
    """eps after ceil(N/B) steps per epoch over `epochs` epochs at sampling rate B/N with noise
    multiplier sigma; envelope = (y, w) from ``envelope_law`` for randomized clipping."""
    y, w = envelope if envelope is not None else (None, None)
    dev = y.device if y is not None else _dev(device)
    T, p = math.ceil(N / B), B / N
    q, qi = step_pld(sigma, p, h, t_max, y, w, dev)
    q, qi = compose(q, qi, T)
    q, qi = compose(q, qi, epochs)
    return _solve_eps(q, qi, h, delta)


def noise_multiplier(eps, N, B, epochs, delta, envelope=None, lo=0.3, hi=50.0, tol=1e-3, **kw):
    """Smallest sigma (to tol) whose accounted eps is at most the target."""
    if epsilon(hi, N, B, epochs, delta, envelope=envelope, **kw) > eps:
        return math.inf
    while hi - lo > tol:
        mid = 0.5 * (lo + hi)
        if epsilon(mid, N, B, epochs, delta, envelope=envelope, **kw) > eps:
            lo = mid
        else:
            hi = mid
    return hi
