"""Privacy accounting for DP-SGD-RC with the Hutchinson estimator.

Appendix "Additional details to Privacy Accounting":

* ``envelope_cdf`` -- Algorithm cdf-grid: the envelope CDF of the normalised
  estimate Y = n_hat / n, the single-coordinate law chi^2(k)/k below 1, the
  uniform law chi^2(kd)/(kd) from x_+ on, and MiddleRegionCDF in between
  (``dprc_envelope_middle`` on the GPU, all two-level forms in parallel);
* ``x_plus`` -- Algorithm binary-search-xplus on [1, 2], deciding at each
  midpoint whether the uniform law dominates every two-level form there
  (single crossing puts x_+ at the first point where it does);
* ``epsilon`` / ``noise_multiplier`` -- Algorithm accounting: the privacy-loss
  distribution (PLD) of one Poisson-subsampled Gaussian step whose scale
  a = 1/sqrt(Y) is averaged over the envelope, composed over the steps of
  all epochs by FFT, and delta(eps) = E[(1 - e^(eps - L))_+] solved for eps.
  Without an envelope this is plain DP-SGD accounting.

The PLD lives on the cell-centred grid t = m h, |t| < t_max; mass that
composition pushes past t_max is kept as an atom at +infinity (it counts
fully towards delta) and mass below -t_max is folded into the lowest cell.
PLD arithmetic runs in fp64 torch on the envelope's device.
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
    weights (CDF increments, negatives clipped, normalised)."""
    dev = _dev(device)
    if y_max is None:
        y_max = 1.0 + 12.0 * math.sqrt(2.0 / k)            # far into the single-coordinate tail
    ys = torch.linspace(0.0, y_max, n_bins + 1, dtype=torch.float64, device=dev)
    F = torch.cummax(envelope_cdf(ys, k, d, n_lambda=n_lambda), dim=0).values.clamp(0.0, 1.0)
    w = torch.clamp(F[1:] - F[:-1], min=0.0)
    w = w / w.sum()
    return 0.5 * (ys[1:] + ys[:-1]), w


def _kernels(t, sigma, y, w):
    """alpha(t), betabar(t) of one step averaged over a = 1/sqrt(y) with weights w
    (a = 1 when y is None)."""
    if y is None:
        mu = torch.tensor([1.0 / sigma], dtype=torch.float64, device=t.device)
        w = torch.ones(1, dtype=torch.float64, device=t.device)
    else:
        keep = w > 0
        mu = (1.0 / torch.sqrt(y[keep])) / sigma
        w = w[keep]
    al = torch.zeros_like(t)
    beb = torch.zeros_like(t)
    chunk = max(1, (1 << 24) // max(1, t.numel()))
    for s in range(0, mu.numel(), chunk):
        m = mu[s:s + chunk, None]
        ww = w[s:s + chunk, None]
        al += (ww * torch.special.ndtr(-t[None, :] / m - m / 2.0)).sum(0)
        beb += (ww * torch.special.ndtr(-(t[None, :] / m - m / 2.0))).sum(0)
    return al, beb


def step_pld(sigma, p, h, t_max, y=None, w=None, device=None):
    """(masses on the grid, mass at +infinity) of one subsampled step."""
    dev = _dev(device if y is None else y.device)
    n = int(round(t_max / h))
    half = (torch.arange(1, n + 1, dtype=torch.float64, device=dev) - 0.5) * h
    cuts = torch.cat([-half.flip(0), half])
    S = torch.ones_like(cuts)                              # survival P(L > t); 1 below the support
    t_min = math.log1p(-p) if p < 1 else -math.inf
    ok = cuts > t_min
    tt = cuts[ok]
    s = torch.log(1.0 / p - (1.0 - p) / p * torch.exp(-tt)) if p < 1 else torch.zeros_like(tt)
    al, beb = _kernels(tt + s, sigma, y, w)
    S[ok] = p * beb + (1.0 - p) * al
    q = torch.clamp(S[:-1] - S[1:], min=0.0)
    q[0] += torch.clamp(1.0 - S[0], min=0.0)
    inf = float(torch.clamp(S[-1], min=0.0))
    tot = float(q.sum()) + inf
    return q / tot, inf / tot


def _compose2(a, ainf, b, binf):
    L = a.numel()
    n = 2 * L - 1
    size = 1 << (n - 1).bit_length()
    r = torch.fft.irfft(torch.fft.rfft(a, size) * torch.fft.rfft(b, size), size)[:n].clamp(min=0.0)
    c = (L - 1) // 2
    out = r[c:c + L].clone()
    out[0] += r[:c].sum()
    top = float(r[c + L:].sum())
    inf = 1.0 - (1.0 - ainf) * (1.0 - binf)
    fin = float(out.sum()) + top
    if fin > 0:
        out *= (1.0 - inf) / fin
        inf += top * (1.0 - inf) / fin
    return out, inf


def compose(q, qinf, steps):
    """PLD of `steps` independent steps (repeated squaring)."""
    res, rinf = None, 0.0
    base, binf = q, qinf
    while steps:
        if steps & 1:
            res, rinf = (base.clone(), binf) if res is None else _compose2(res, rinf, base, binf)
        steps >>= 1
        if steps:
            base, binf = _compose2(base, binf, base, binf)
    return res, rinf


def _delta(grid, q, qinf, eps):
    m = grid >= eps
    return min(1.0, max(0.0, float((q[m] * (1.0 - torch.exp(eps - grid[m]))).sum()) + qinf))


def epsilon(sigma, N, B, epochs, delta, h=1e-3, t_max=20.0, envelope=None, device=None):
    """eps after ceil(N/B) steps per epoch over `epochs` epochs at sampling rate B/N with noise
    multiplier sigma; envelope = (y, w) from ``envelope_law`` for randomized clipping."""
    y, w = envelope if envelope is not None else (None, None)
    dev = y.device if y is not None else _dev(device)
    T, p = math.ceil(N / B), B / N
    q, qi = step_pld(sigma, p, h, t_max, y, w, dev)
    q, qi = compose(q, qi, T)
    q, qi = compose(q, qi, epochs)
    n = (q.numel() + 1) // 2
    grid = torch.arange(-(n - 1), n, dtype=torch.float64, device=dev) * h
    f = lambda e: _delta(grid, q, qi, e) - delta
    if f(0.0) <= 0:
        return 0.0
    hi = float(grid[-1])
    if f(hi) > 0:
        return math.inf
    lo = 0.0
    for _ in range(200):                                   # bisection to 1e-10
        mid = 0.5 * (lo + hi)
        if f(mid) > 0:
            lo = mid
        else:
            hi = mid
        if hi - lo < 1e-10:
            break
    return 0.5 * (lo + hi)


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
