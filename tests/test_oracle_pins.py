"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each test fixes part of the oracle to something independent: published
known-answer vectors, a library routine (scipy's Hadamard, torch autograd,
LAPACK through a second formulation), a closed form, or an exact identity from
the paper (the ghost-clipping Gram identity; Hutch++ exactness on low-rank
inputs).  A plausible slip in the oracle (a dropped term, a wrong sign or
index, a transposed operand, a missing 1/k) fails at least one of them.
"""

import json
import math
import os

import numpy as np
import pytest
import scipy.linalg
import scipy.stats
import torch

from oracle import philox
from oracle import estimators as est
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rng_inputs(B, T, d, p, seed=0, scale=None):
    r = np.random.default_rng(seed)
    A = r.standard_normal((B, T, d))
    E = r.standard_normal((B, T, p))
    if scale is not None:
        E *= np.asarray(scale).reshape(B, 1, 1)
    return A, E


# ---- generator -------------------------------------------------------------

def test_philox_known_answer_vectors():
    kat = json.load(open(os.path.join(GOLDEN, "philox4x32_10_kat.json")))
    for v in kat["vectors"]:
        ctr = np.array([int(x, 16) for x in v["ctr"]], dtype=np.uint64)
        key = np.array([int(x, 16) for x in v["key"]], dtype=np.uint64)
        out = philox.philox4x32_10(ctr, key)
        assert [f"{int(x):08x}" for x in out] == v["out"]


def test_philox_vectorised_matches_scalar():
    ctr = np.array([[i, 7 * i, 3, 11] for i in range(50)], dtype=np.uint64)
    batch = philox.philox4x32_10(ctr, np.array([5, 9], dtype=np.uint64))
    for i in range(50):
        one = philox.philox4x32_10(ctr[i], np.array([5, 9], dtype=np.uint64))
        assert np.array_equal(batch[i], one)


def test_rademacher_statistics():
    m, k = 4096, 64
    Z = philox.rademacher_matrix(0, 3, philox.STREAM_PROBE, m, k)
    assert set(np.unique(Z)) == {-1.0, 1.0}
    col_mean = Z.mean(axis=0)
    assert np.all(np.abs(col_mean) < 5.0 / math.sqrt(m))
    corr = (Z.T @ Z) / m
    off = corr[~np.eye(k, dtype=bool)]
    assert np.max(np.abs(off)) < 5.0 / math.sqrt(m)
    # streams, layers and seeds are distinct
    Z2 = philox.rademacher_matrix(0, 4, philox.STREAM_PROBE, m, k)
    Z3 = philox.rademacher_matrix(0, 3, philox.STREAM_SKETCH, m, k)
    Z4 = philox.rademacher_matrix(1, 3, philox.STREAM_PROBE, m, k)
    for other in (Z2, Z3, Z4):
        assert abs((Z * other).mean()) < 5.0 / math.sqrt(m * k)


def test_rademacher_tail_bits_cleared_and_prefix_stable():
    w = philox.rademacher_words(7, 1, 0, 45, 3)          # 2 words per column, 13 valid bits in the last
    assert w.shape == (3, 2)
    assert np.all(w[:, 1] >> np.uint32(13) == 0)
    w_long = philox.rademacher_words(7, 1, 0, 64, 3)
    assert np.array_equal(w[:, 0], w_long[:, 0])
    assert np.array_equal(w[:, 1], w_long[:, 1] & np.uint32((1 << 13) - 1))
    Z = philox.rademacher_matrix(7, 1, 0, 45, 3)
    Zl = philox.rademacher_matrix(7, 1, 0, 64, 3)
    assert np.array_equal(Z, Zl[:45])


def test_hadamard_mode_is_sylvester():
    for n in (1, 2, 16, 64):
        assert np.array_equal(philox.hadamard_matrix(n, n), scipy.linalg.hadamard(n).astype(float))
    H = philox.hadamard_matrix(48, 64)
    assert np.allclose(H @ H.T, 64 * np.eye(48))


def test_gaussian_moments_and_ks():
    x = philox.gaussian(11, 5, 0, 400_000)
    assert abs(x.mean()) < 5 / math.sqrt(x.size)
    assert abs(x.var() - 1.0) < 5 * math.sqrt(2.0 / x.size)
    assert scipy.stats.kstest(x, "norm").pvalue > 1e-4
    # window consistency and distinct tensors
    assert np.array_equal(philox.gaussian(11, 5, 5, 10), x[5:15])
    y = philox.gaussian(11, 6, 0, 10_000)
    assert abs(np.corrcoef(x[:10_000], y)[0, 1]) < 0.05


def test_gaussian_probes_are_standard_normal_and_independent():
    """The Gaussian probe option (Algorithm 2 draws P from a normal law): moments, a KS test,
    kurtosis 3 (+-1 probes have 1), and uncorrelated columns and layers."""
    Z = philox.gaussian_probe_matrix(3, 7, 4099, 64)          # ragged m: the last block is cut
    x = Z.reshape(-1)
    assert Z.shape == (4099, 64)
    assert abs(x.mean()) < 5 / math.sqrt(x.size)
    assert abs(x.var() - 1.0) < 5 * math.sqrt(2.0 / x.size)
    assert abs(scipy.stats.kurtosis(x, fisher=False) - 3.0) < 0.1
    assert scipy.stats.kstest(x, "norm").pvalue > 1e-4
    C = np.corrcoef(Z.T)
    assert np.max(np.abs(C - np.eye(64))) < 5.5 / math.sqrt(4099)
    Z2 = philox.gaussian_probe_matrix(3, 8, 4099, 4)
    assert abs(np.corrcoef(Z[:, 0], Z2[:, 0])[0, 1]) < 5 / math.sqrt(4099)
    # a prefix of rows does not depend on m
    assert np.array_equal(philox.gaussian_probe_matrix(3, 7, 10, 2), Z[:10, :2])


def test_hutch_gaussian_moments_match_closed_form():
    """Gaussian probes: mean -> ||G||_F^2 and variance -> (2/k) ||O||_F^2, O = G^T G, which
    differs from the +-1 value (2/k)(||O||_F^2 - sum_u O_uu^2) by the diagonal term."""
    A, E = _rng_inputs(1, 4, 3, 6, seed=5)
    G = est.per_sample_grad(A[0], E[0])
    O = G.T @ G
    k, n = 2, 6000
    vals = np.array([est.hutch_layer(A, E, k, seed, 0, probe="gaussian")[0] for seed in range(n)])
    var_th = 2.0 / k * np.sum(O * O)
    var_rad = 2.0 / k * (np.sum(O * O) - np.sum(np.diag(O) ** 2))
    assert var_th > 1.5 * var_rad                      # the two laws are told apart below
    assert abs(vals.mean() - np.sum(G * G)) < 5 * math.sqrt(var_th / n)
    assert 0.85 < vals.var(ddof=1) / var_th < 1.18


# ---- exact norms -------------------------------------------------------------

@pytest.mark.parametrize("T,d,p", [(64, 64, 48), (7, 3, 5), (33, 17, 70)])
def test_gc_identity_equals_fgc(T, d, p):
    A, E = _rng_inputs(1, T, d, p, seed=T)
    a = est.norm_fgc(A[0], E[0])
    b = est.norm_gc(A[0], E[0])
    assert abs(a - b) <= 1e-12 * abs(a)


def test_per_sample_grad_matches_autograd():
    """G_i = A_i^T E_i is the gradient of sample i's loss for S = A W, E = dL/dS."""
    A, E = _rng_inputs(3, 9, 6, 4, seed=1)
    for i in range(3):
        W = torch.zeros(6, 4, dtype=torch.float64, requires_grad=True)
        S = torch.from_numpy(A[i]) @ W
        (S * torch.from_numpy(E[i])).sum().backward()
        assert np.allclose(W.grad.numpy(), est.per_sample_grad(A[i], E[i]), rtol=1e-13, atol=1e-13)


def test_clipped_sum_matches_second_backward():
    """Back-propagating sum_i c_i L_i (c_i constant) gives the clipped sum of Algorithm 1."""
    A, E = _rng_inputs(4, 11, 5, 7, seed=2)
    c = np.array([0.3, 1.0, 0.0, 0.75])
    W = torch.zeros(5, 7, dtype=torch.float64, requires_grad=True)
    loss = 0
    for i in range(4):
        S = torch.from_numpy(A[i]) @ W
        loss = loss + float(c[i]) * (S * torch.from_numpy(E[i])).sum()
    loss.backward()
    assert np.allclose(W.grad.numpy(), est.clip_accumulate(A, E, c), rtol=1e-12, atol=1e-12)


# ---- Hutchinson ----------------------------------------------------------------

@pytest.mark.parametrize("side", [est.SIDE_OUT, est.SIDE_IN])
def test_hutch_with_hadamard_probes_is_exact(side):
    # cfg-1 shape: d=64, p=48; 64 Hadamard columns make Z Z^T = 64 I on either side
    A, E = _rng_inputs(2, 64, 64, 48, seed=3, scale=[0.1, 10.0])
    h = est.hutch_layer(A, E, 64, 0, 0, side=side, probe="hadamard")
    ex = est.exact_layer(A, E)
    assert np.all(np.abs(h - ex) <= 1e-12 * ex)


def test_hutch_sides_agree_with_transposed_problem():
    A, E = _rng_inputs(2, 10, 6, 9, seed=4)
    out_in = est.hutch_layer(A, E, 5, 3, 2, side=est.SIDE_IN)
    swapped = est.hutch_layer(E, A, 5, 3, 2, side=est.SIDE_OUT)
    assert np.allclose(out_in, swapped, rtol=1e-14)
    assert est.resolve_side(8, 4, est.SIDE_AUTO) == est.SIDE_IN
    assert est.resolve_side(4, 8, est.SIDE_AUTO) == est.SIDE_OUT
    assert est.resolve_side(4, 4, est.SIDE_AUTO) == est.SIDE_OUT


def test_hutch_moments_match_closed_form():
    """Mean -> ||G||_F^2; variance -> (2/k)(||O||_F^2 - sum_u O_uu^2), O = G^T G (Rademacher)."""
    A, E = _rng_inputs(1, 4, 3, 6, seed=5)
    G = est.per_sample_grad(A[0], E[0])
    O = G.T @ G
    k = 2
    n = 6000
    vals = np.array([est.hutch_layer(A, E, k, seed, 0)[0] for seed in range(n)])
    true = np.sum(G * G)
    var_th = 2.0 / k * (np.sum(O * O) - np.sum(np.diag(O) ** 2))
    se = math.sqrt(var_th / n)
    assert abs(vals.mean() - true) < 5 * se
    # sample variance of n draws: relative sd about sqrt(2/(n-1)) for light tails; allow a wide band
    assert 0.8 < vals.var(ddof=1) / var_th < 1.25


def test_hutch_d1_is_jl_sketch_of_gradient_vector():
    """With d = 1 the per-sample gradient is a vector g and Hutch is a Rademacher JL sketch of it:
    each probe column contributes (g.z)^2, whose mean is ||g||^2 and whose variance is
    2(||g||^4 - sum g_u^4)."""
    A, E = _rng_inputs(1, 5, 1, 8, seed=6)
    g = est.per_sample_grad(A[0], E[0])[0]
    k, n = 1, 8000
    vals = np.array([est.hutch_layer(A, E, k, seed, 1)[0] for seed in range(n)])
    var_th = 2.0 * (np.sum(g * g) ** 2 - np.sum(g ** 4))
    assert abs(vals.mean() - np.sum(g * g)) < 5 * math.sqrt(var_th / n)


# ---- Hutch++ ---------------------------------------------------------------------

def test_hutchpp_exact_when_rank_at_most_sketch():
    # T = 12 tokens < s = 16 -> rank(G_i) <= 12
    A, E = _rng_inputs(2, 12, 40, 64, seed=7)
    h = est.hutchpp_layer(A, E, 16, 8, 0, 0)
    ex = est.exact_layer(A, E)
    assert np.all(np.abs(h - ex) <= 1e-10 * ex)


def test_hutchpp_exact_when_sketch_covers_dimension():
    A, E = _rng_inputs(1, 30, 20, 10, seed=8)
    h = est.hutchpp_layer(A, E, 10, 4, 1, 0)
    assert abs(h[0] - est.exact_layer(A, E)[0]) <= 1e-10 * h[0]


def test_hutchpp_without_sketch_is_hutch():
    A, E = _rng_inputs(2, 20, 8, 12, seed=9)
    assert np.array_equal(est.hutchpp_layer(A, E, 0, 6, 5, 2), est.hutch_layer(A, E, 6, 5, 2))


def test_hutchpp_unbiased():
    A, E = _rng_inputs(1, 6, 5, 9, seed=10)
    true = est.exact_layer(A, E)[0]
    vals = np.array([est.hutchpp_layer(A, E, 2, 2, seed, 0)[0] for seed in range(3000)])
    assert abs(vals.mean() - true) < 5 * vals.std(ddof=1) / math.sqrt(vals.size)


def test_hutchpp_beats_hutch_on_decaying_spectrum():
    """On a gradient with a few dominant directions the head is captured exactly."""
    r = np.random.default_rng(11)
    T, d, p = 40, 30, 50
    A = r.standard_normal((1, T, 3)) @ r.standard_normal((3, d)) + 1e-3 * r.standard_normal((1, T, d))
    E = r.standard_normal((1, T, p))
    true = est.exact_layer(A, E)[0]
    e_pp = np.mean([abs(est.hutchpp_layer(A, E, 4, 4, s, 0)[0] - true) for s in range(40)]) / true
    e_h = np.mean([abs(est.hutch_layer(A, E, 8, s, 0)[0] - true) for s in range(40)]) / true
    assert e_pp < 1e-3 < e_h


# ---- clip, accumulate, noise -------------------------------------------------------

def test_clip_scale_closed_forms():
    C = 2.0
    c = est.clip_scale([0.0, 4.0, 16.0, 1.0, math.inf, math.nan, -1.0, 1e300], C)
    assert c[0] == 1.0 and c[1] == 1.0 and c[3] == 1.0
    assert c[2] == 0.5
    assert c[4] == 0.0 and c[5] == 0.0 and c[6] == 0.0
    assert abs(c[7] - 2e-150) < 1e-160


def test_clip_accumulate_unit_scale_is_plain_weight_gradient():
    A, E = _rng_inputs(3, 13, 6, 5, seed=12)
    flat = torch.from_numpy(A.reshape(-1, 6)).T @ torch.from_numpy(E.reshape(-1, 5))
    assert np.allclose(est.clip_accumulate(A, E, np.ones(3)), flat.numpy(), rtol=1e-12, atol=1e-12)


def test_clip_accumulate_linear_and_excludes_zero_scale():
    A, E = _rng_inputs(3, 8, 4, 6, seed=13)
    c = np.array([0.2, 0.5, 0.9])
    g = est.clip_accumulate(A, E, c)
    assert np.allclose(est.clip_accumulate(A, E, 3 * c), 3 * g, rtol=1e-12)
    A2, E2 = A.copy(), E.copy()
    A2[1, 0, 0] = np.nan
    E2[1, 2, 3] = np.inf
    c2 = c.copy()
    c2[1] = 0.0
    g2 = est.clip_accumulate(A2, E2, c2)
    assert np.all(np.isfinite(g2))
    assert np.allclose(g2, est.clip_accumulate(A, E, c2), rtol=1e-12)


def test_noise_zero_sigma_and_scale():
    g = np.arange(12.0).reshape(3, 4)
    assert np.array_equal(est.add_noise(g, 0.0, 1.0, 0, 0), g)
    a = est.add_noise(g, 0.8, 1.0, 3, 2) - g
    b = est.add_noise(g, 0.4, 2.0, 3, 2) - g
    assert np.allclose(a, b)
    assert np.allclose(a.ravel() / 0.8, philox.gaussian(3, 2, 0, 12))


# ---- FLOP model (appendix table) ---------------------------------------------------

def test_flop_model_reproduces_printed_reductions():
    gold = json.load(open(os.path.join(GOLDEN, "flops_reduction.json")))
    for row in gold["hutch_reduction_percent"]:
        B = 2
        rc = est.flops_rc(B, row["T"], row["d"], row["p"], row["k"])
        fgc = est.flops_fgc(B, row["T"], row["d"], row["p"])
        assert round(100.0 * (1.0 - rc / fgc), 2) == row["percent"]
    ex = gold["ratio_example"]
    rc = est.flops_rc(1, ex["T"], ex["d"], ex["p"], ex["k"])
    assert round(est.flops_gc(1, ex["T"], ex["d"], ex["p"]) / rc) == ex["vs_gc"]
    assert round(est.flops_fgc(1, ex["T"], ex["d"], ex["p"]) / rc) == ex["vs_fgc"]


# ---- input generators ----------------------------------------------------------------

def test_workload_generators_are_seeded_and_shaped():
    A, E = workloads.draw(2, 16, 8, 12, dtype="bf16", law="lognormal", seed=0, layer=3)
    A2, E2 = workloads.draw(2, 16, 8, 12, dtype="bf16", law="lognormal", seed=0, layer=3)
    assert A.dtype == torch.bfloat16 and A.shape == (2, 16, 8) and E.shape == (2, 16, 12)
    assert torch.equal(A, A2) and torch.equal(E, E2)
    Ap, Ep = workloads.draw(2, 16, 8, 12, dtype="f32", law="student_t", seed=0, layer=1, row_pad_a=8)
    assert Ap.stride(1) == 16 and Ap.shape == (2, 16, 8)
    assert len(workloads.CONFIGS) == 5
    assert workloads.algorithmic_norm_bytes(workloads.BY_NAME["q_proj"]) == 67_108_864
    assert workloads.algorithmic_norm_bytes(workloads.BY_NAME["stack"]) == 54_710_501_376


# ---- projected-order variants used for sampled full-size checks ----------------------

@pytest.mark.parametrize("side", [est.SIDE_OUT, est.SIDE_IN])
def test_projected_order_matches_explicit(side):
    A, E = _rng_inputs(2, 30, 11, 17, seed=14)
    m = 17 if side == est.SIDE_OUT else 11
    Z = philox.rademacher_matrix(2, 5, 0, m, 6)
    ref = est.hutch_layer(A, E, 6, 2, 5, side=side)
    for i in range(2):
        assert abs(est.hutch_sample_projected(A[i], E[i], Z, side) - ref[i]) <= 1e-12 * ref[i]
    ZS = philox.rademacher_matrix(2, 5, 1, m, 4)
    ZP = philox.rademacher_matrix(2, 5, 0, m, 5)
    refpp = est.hutchpp_layer(A, E, 4, 5, 2, 5, side=side)
    for i in range(2):
        assert abs(est.hutchpp_sample_projected(A[i], E[i], ZS, ZP, side) - refpp[i]) <= 1e-10 * refpp[i]
    c = np.array([0.5, 0.25])
    assert np.allclose(est.clip_accumulate_rows(A, E, c, [1, 4]), est.clip_accumulate(A, E, c)[[1, 4]])


def test_adamw_matches_torch_and_first_step_closed_form():
    # torch's AdamW (decoupled weight decay) on fp64 CPU tensors, three steps
    r = np.random.default_rng(5)
    theta0 = r.standard_normal((7, 5))
    grads = [r.standard_normal((7, 5)) * s for s in (1.0, 0.1, 3.0)]
    lr, b1, b2, eps, wd = 1e-2, 0.9, 0.99, 1e-8, 0.1
    p = torch.tensor(theta0, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.AdamW([p], lr=lr, betas=(b1, b2), eps=eps, weight_decay=wd)
    th, m, v = theta0, np.zeros_like(theta0), np.zeros_like(theta0)
    for t, g in enumerate(grads, start=1):
        p.grad = torch.tensor(g)
        opt.step()
        th, m, v = est.adamw(th, g, m, v, t, lr, b1, b2, eps, wd)
        assert np.allclose(th, p.detach().numpy(), rtol=1e-12, atol=1e-14)
    # first step without decay: theta - lr g / (|g| + eps)
    g = grads[0]
    th1, _, _ = est.adamw(theta0, g, 0.0, 0.0, 1, lr, b1, b2, eps, 0.0)
    assert np.allclose(th1, theta0 - lr * g / (np.abs(g) + eps), rtol=1e-13, atol=1e-15)


def test_private_gradient_composition():
    A, E = _rng_inputs(3, 6, 4, 5, seed=8)
    c = np.array([1.0, 0.5, 0.0])
    g = est.private_gradient(A, E, c, 0.0, 1.0, 0, 0, 3)
    assert np.allclose(g, est.clip_accumulate(A, E, c) / 3, rtol=1e-15)
    g = est.private_gradient(A, E, c, 0.7, 2.0, 9, 4, 3)
    assert np.allclose(g, est.add_noise(est.clip_accumulate(A, E, c), 0.7, 2.0, 9, 4) / 3, rtol=1e-15)
