"""Parity at the full sizes of the five workloads, in the launch configuration
bench.py times (all layers of a workload in one norm call).

The oracle checks sampled outputs it can compute one by one: every per-layer,
per-sample estimate where that is cheap (Algorithm 2's projected association
order, pinned to the explicit-gradient form in the oracle tests), a few
(layer, sample) pairs of the 113-layer stack, and rows x columns blocks of the
clipped gradients.  Properties that hold at any size are checked on the rest:
the layer sum equals n2, and clip factors follow from n2.
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
    A, E, _ = pairs[6]                                            # down: 8192 -> 2048
    g = D.dprc_clip_accumulate(A, E, c)
    _check_grad_block(A, E, c, g, [0, 4095, 8191], list(range(0, 2048, 13)))
    del pairs, A, E, g
    _free()


def test_stack_full(D):
    cfg = workloads.BY_NAME["stack"]
    pairs = _inputs(cfg)
    n2, n2l = _run_norm(D, cfg, pairs)
    got = n2l.cpu().numpy()
    L = len(pairs)
    assert np.allclose(got.sum(axis=0), n2.cpu().numpy(), rtol=1e-5)
    assert np.all(got > 0)
    for (li, i) in [(0, 0), (1, 3), (6, 7), (57, 2), (L - 2, 5), (L - 1, 1)]:   # q, k, down, ..., lm_head
        A, E, _ = pairs[li]
        assert _rel(got[li, i], _hutch_pair(A, E, i, li, cfg["k"])) < NORM_RTOL, (li, i)
    c = D.dprc_clip_scale(n2, cfg["C"])
    assert np.allclose(c.cpu().numpy(), est.clip_scale(n2.cpu().numpy().astype(np.float64), cfg["C"]), rtol=1e-6)
    for li in (1, L - 1):                                          # k (2048 x 512) and lm_head (2048 x 128256)
        A, E, _ = pairs[li]
        g = D.dprc_clip_accumulate(A, E, c)
        _check_grad_block(A, E, c, g, [0, 1000, 2047], list(range(11, E.shape[2], max(1, E.shape[2] // 97))))
        g0 = g.clone()
        D.dprc_add_noise(g, cfg["noise_sigma"], cfg["C"], 0, li)
        noise = (g - g0)[:4].flatten()[:100_000].cpu().numpy().astype(np.float64)
        ref = cfg["noise_sigma"] * cfg["C"] * philox.gaussian(0, li, 0, noise.size)
        assert np.max(np.abs(noise - ref)) < 1e-5 + 1e-6 * np.max(np.abs(g0[:4].cpu().numpy()))
        del g, g0
    del pairs
    _free()
