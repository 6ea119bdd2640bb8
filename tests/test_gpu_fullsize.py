"""Parity at the full sizes of the five workloads, in the launch configuration
bench.py times (all layers of a workload in one norm call).

The oracle checks outputs it can compute one by one: every per-layer,
per-sample estimate (Algorithm 2's projected association order, pinned to the
explicit-gradient form in the oracle tests; for the 113-layer stack all 904 of
them, one layer at a time on the host), and rows of the clipped gradients --
on the stack and decoder workloads one row in every 256-row tile row of every
layer, over all columns.  Properties that hold at any size are checked on the
rest: the layer sum equals n2, and clip factors follow from n2.
"""

import gc

import numpy as np
import pytest
import torch

from oracle import estimators as est
from oracle import philox
import workloads

pytestmark = pytest.mark.gpu

NORM_RTOL = 1e-3
GRAD_RTOL = 2e-3


@pytest.fixture(scope="module")
def D():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2605_24879_amd import dprc
    dprc.lib()
    return dprc


def _free():
    gc.collect()
    torch.cuda.empty_cache()


def _rel(a, b):
    return abs(float(a) - float(b)) / abs(float(b))


def _np(x):
    return est.as_f64(x)


def _check_grad_block(A, E, c, g, rows, cols):
    """grad[rows][:, cols] against the oracle on the sliced operands."""
    As = A[:, :, rows]
    Es = E[:, :, cols]
    ref = est.clip_accumulate(_np(As), _np(Es), c.cpu().numpy().astype(np.float64))
    got = g[rows][:, cols].cpu().numpy().astype(np.float64)
    err = np.linalg.norm(got - ref) / np.linalg.norm(ref)
    assert err < GRAD_RTOL, err


def _host_f64(x):
    """fp64 host copy of a device tensor (bf16 -> fp64 is exact; torch converts on the host's
    cores, which the oracle's single-threaded widening would not)."""
    return x.to("cpu").to(torch.float64).numpy()


def _tile_rows(d, li):
    """One row in every 256-row tile row of a d-row gradient (the accumulation kernel's tiles)."""
    return [t * 256 + (37 * t + 11 * li) % min(256, d - t * 256) for t in range((d + 255) // 256)]


def _check_rows(D, A, E, c, li, cn, samples_f64=None, g=None):
    """grad rows (one per tile row, all columns) against the oracle; samples_f64 may hold
    the fp64 host copies of (A_i, E_i) already made; g, the layer's gradient from a call
    for several layers (else a call of its own computes it)."""
    d = A.shape[2]
    rows = _tile_rows(d, li)
    if g is None:
        g = D.dprc_clip_accumulate(A, E, c)
    got = g[rows].cpu().numpy().astype(np.float64)
    del g
    ref = np.zeros_like(got)
    for i in range(A.shape[0]):
        if cn[i] == 0.0:
            continue
        Ai, Ei = samples_f64[i] if samples_f64 is not None else (_host_f64(A[i]), _host_f64(E[i]))
        ref += est.clip_accumulate_rows(Ai[None], Ei[None], cn[i:i + 1], rows)
    err = np.linalg.norm(got - ref) / np.linalg.norm(ref)
    assert err < GRAD_RTOL, (li, err)
    return err


def _hutch_pair(A, E, i, li, k):
    p = E.shape[2]
    Z = philox.rademacher_matrix(0, li, 0, p, k)
    return est.hutch_sample_projected(_np(A[i]), _np(E[i]), Z)


def _run_norm(D, cfg, pairs):
    B, L = cfg["B"], len(pairs)
    n2l = torch.zeros(L, B, device="cuda")
    if cfg["estimator"] == "hutch":
        n2 = D.dprc_norm_hutch(pairs, cfg["k"], 0, n2_layers=n2l)
    else:
        n2 = D.dprc_norm_hutchpp(pairs, cfg["s"], cfg["r"], 0, n2_layers=n2l)
    torch.cuda.synchronize()
    return n2, n2l


def _inputs(cfg, layers=None):
    idx = range(len(cfg["layers"])) if layers is None else layers
    out = [(*workloads.layer_inputs(cfg, li, device="cuda"), li) for li in idx]
    for (A, E, li) in out:                      # full workload sizes, nothing shrunk
        _, d, p = cfg["layers"][li]
        assert tuple(A.shape) == (cfg["B"], cfg["T"], d) and tuple(E.shape) == (cfg["B"], cfg["T"], p)
    return out


def test_tiny_full(D):
    cfg = workloads.BY_NAME["tiny"]
    pairs = _inputs(cfg)
    n2, n2l = _run_norm(D, cfg, pairs)
    A, E, _ = pairs[0]
    ref = est.hutch_layer(_np(A), _np(E), cfg["k"], 0, 0)
    assert np.all(np.abs(n2.cpu().numpy() - ref) <= NORM_RTOL * ref)
    c = D.dprc_clip_scale(n2, cfg["C"])
    assert np.allclose(c.cpu().numpy(), est.clip_scale(n2.cpu().numpy().astype(np.float64), cfg["C"]), rtol=1e-6)
    g = D.dprc_clip_accumulate(A, E, c)
    ref_g = est.clip_accumulate(_np(A), _np(E), c.cpu().numpy().astype(np.float64))
    assert np.linalg.norm(g.cpu().numpy() - ref_g) / np.linalg.norm(ref_g) < GRAD_RTOL
    D.dprc_add_noise(g, 0.8, cfg["C"], 0, 0)
    ref_n = est.add_noise(ref_g, 0.8, cfg["C"], 0, 0)
    assert np.linalg.norm(g.cpu().numpy() - ref_n) / np.linalg.norm(ref_n) < GRAD_RTOL


def test_q_proj_full(D):
    cfg = workloads.BY_NAME["q_proj"]
    pairs = _inputs(cfg)
    n2, n2l = _run_norm(D, cfg, pairs)
    A, E, _ = pairs[0]
    ref = est.hutch_layer(_np(A), _np(E), cfg["k"], 0, 0)       # explicit per-sample gradients
    got = n2.cpu().numpy()
    assert all(_rel(got[i], ref[i]) < NORM_RTOL for i in range(cfg["B"]))
    c = D.dprc_clip_scale(n2, cfg["C"])
    assert np.allclose(c.cpu().numpy(), est.clip_scale(got.astype(np.float64), cfg["C"]), rtol=1e-6)
    g = D.dprc_clip_accumulate(A, E, c)
    _check_grad_block(A, E, c, g, [0, 1, 777, 2047], list(range(0, 2048, 7)))
    del pairs, A, E, g
    _free()


def test_q_proj_full_gaussian_probes(D):
    # the q_proj workload with Gaussian probes (k = 16 dense columns), sampled samples
    cfg = workloads.BY_NAME["q_proj"]
    pairs = _inputs(cfg)
    n2 = D.dprc_norm_hutch(pairs, cfg["k"], 5, probe=D.PROBE_GAUSSIAN)
    torch.cuda.synchronize()
    A, E, li = pairs[0]
    Z = philox.gaussian_probe_matrix(5, li, E.shape[2], cfg["k"])
    got = n2.cpu().numpy()
    for i in (0, cfg["B"] // 2, cfg["B"] - 1):
        ref = est.hutch_sample_projected(_np(A[i]), _np(E[i]), Z)
        assert _rel(got[i], ref) < NORM_RTOL
    del pairs, A, E
    _free()


def test_mlp_full(D):
    cfg = workloads.BY_NAME["mlp"]
    pairs = _inputs(cfg)
    n2, n2l = _run_norm(D, cfg, pairs)
    got = n2l.cpu().numpy()
    for (A, E, li) in pairs:
        for i in range(cfg["B"]):
            assert _rel(got[li, i], _hutch_pair(A, E, i, li, cfg["k"])) < NORM_RTOL, (li, i)
    assert np.allclose(got.sum(axis=0), n2.cpu().numpy(), rtol=1e-6)
    c = D.dprc_clip_scale(n2, cfg["C"])
    for (A, E, li) in pairs:
        g = D.dprc_clip_accumulate(A, E, c)
        d, p = A.shape[2], E.shape[2]
        _check_grad_block(A, E, c, g, [0, 5, d // 2, d - 1], list(range(3, p, 61)))
        del g
    del pairs
    _free()


def test_decoder_hutchpp_full(D):
    cfg = workloads.BY_NAME["decoder"]
    pairs = _inputs(cfg)
    n2, n2l = _run_norm(D, cfg, pairs)
    got = n2l.cpu().numpy()
    for (A, E, li) in pairs:
        p = E.shape[2]
        ZS = philox.rademacher_matrix(0, li, 1, p, cfg["s"])
        ZP = philox.rademacher_matrix(0, li, 0, p, cfg["r"])
        ref = est.hutchpp_sample_projected(_np(A[0]), _np(E[0]), ZS, ZP)
        assert _rel(got[li, 0], ref) < NORM_RTOL, (li, got[li, 0], ref)
    c = D.dprc_clip_scale(n2, cfg["C"])
    cn = c.cpu().numpy().astype(np.float64)
    assert np.allclose(cn, est.clip_scale(n2.cpu().numpy().astype(np.float64), cfg["C"]), rtol=1e-6)
    for (A, E, li) in pairs:                                      # every layer's gradient
        _check_rows(D, A, E, c, li, cn)
    del pairs
    _free()


@pytest.mark.timeout(900)
def test_stack_full(D):
    cfg = workloads.BY_NAME["stack"]
    pairs = _inputs(cfg)
    n2, n2l = _run_norm(D, cfg, pairs)
    got = n2l.cpu().numpy()
    B, L, k = cfg["B"], len(pairs), cfg["k"]
    assert np.allclose(got.sum(axis=0), n2.cpu().numpy(), rtol=1e-5)
    c = D.dprc_clip_scale(n2, cfg["C"])
    cn = c.cpu().numpy().astype(np.float64)
    assert np.allclose(cn, est.clip_scale(n2.cpu().numpy().astype(np.float64), cfg["C"]), rtol=1e-6)
    # the gradients as the bench's step computes them: one call for every layer
    grads = D.dprc_clip_accumulate_layers(pairs, c)
    for li in (0, 1):                                              # q and k, split when alone
        A, E, _ = pairs[li]
        solo = D.dprc_clip_accumulate(A, E, c)
        assert ((grads[li] - solo).norm() / solo.norm()).item() < 1e-5
        del solo
    worst_n = worst_g = 0.0
    for (A, E, li) in pairs:
        # every sample's estimate of this layer, then its gradient rows, from one host copy
        p = E.shape[2]
        Z = philox.rademacher_matrix(0, li, 0, p, k)
        host = [(_host_f64(A[i]), _host_f64(E[i])) for i in range(B)] if p <= 8192 else None
        for i in range(B):
            Ai, Ei = host[i] if host is not None else (_host_f64(A[i]), _host_f64(E[i]))
            r = _rel(got[li, i], est.hutch_sample_projected(Ai, Ei, Z))
            assert r < NORM_RTOL, (li, i, r)
            worst_n = max(worst_n, r)
            del Ai, Ei
        worst_g = max(worst_g, _check_rows(D, A, E, c, li, cn, host, g=grads[li]))
        grads[li] = None
        del host
        if li % 16 == 15 or li == L - 1:
            print(f"[stack parity] layers 0..{li}: worst norm rel {worst_n:.2e}, worst grad rel {worst_g:.2e}",
                  flush=True)
    for li in (1, L - 1):                                          # noise on k (2048 x 512) and lm_head
        A, E, _ = pairs[li]
        g = D.dprc_clip_accumulate(A, E, c)
        g0 = g.clone()
        D.dprc_add_noise(g, cfg["noise_sigma"], cfg["C"], 0, li)
        noise = (g - g0)[:4].flatten()[:100_000].cpu().numpy().astype(np.float64)
        ref = cfg["noise_sigma"] * cfg["C"] * philox.gaussian(0, li, 0, noise.size)
        assert np.max(np.abs(noise - ref)) < 1e-5 + 1e-6 * np.max(np.abs(g0[:4].cpu().numpy()))
        del g, g0
    del pairs
    _free()
