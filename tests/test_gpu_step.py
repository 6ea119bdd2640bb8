"""End-to-end DP-SGD-RC step (Alg. DP-SGD-RC) on the GPU against the oracle.

A Llama-shaped stack at small sizes (bf16) runs forward, the driver captures
every linear layer's (A, E), and the library computes the norm estimates, clip
factors, clipped gradients and noise.  The oracle takes the identical captured
bf16 tensors and the same keys.  Tolerances as in the kernel parity tests;
the AdamW update is compared with the oracle's AdamW on the oracle's private
gradient.  The clipped gradient is also compared with Algorithm 1's second
backward pass (torch autograd of sum_i c_i L_i in bf16, 2e-2 relative).
"""

import numpy as np
import pytest
import torch

from oracle import estimators as est
from workloads import llama

pytestmark = pytest.mark.gpu

NORM_RTOL = 1e-3
GRAD_RTOL = 2e-3
SIZES = dict(layers=2, hidden=128, mlp=256, heads=4, kv_heads=2, vocab=200)


@pytest.fixture(scope="module")
def mods():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2605_24879_amd import dprc, dpsgd
    dprc.lib()
    return dprc, dpsgd


def _setup(dpsgd, seed=1, **kw):
    model = llama.build(seed=seed, device="cuda", dtype=torch.bfloat16, **SIZES)
    tok = llama.tokens(3, 40, SIZES["vocab"], seed=seed, device="cuda")
    drv = dpsgd.DPSGDRC(model.linears(), **kw)
    loss_fn = lambda: llama.per_sample_loss(model(tok[:, :-1]), tok[:, 1:])
    return model, drv, loss_fn


def _rel_fro(a, b):
    return np.linalg.norm(a - b) / np.linalg.norm(b)


def test_step_stages_match_oracle(mods):
    D, dpsgd = mods
    C, sigma, k = 0.05, 0.6, 16
    model, drv, loss_fn = _setup(dpsgd, C=C, sigma=sigma, k=k, seed=11, lr=1e-3, weight_decay=0.01,
                                 fused_adamw=False)
    losses, pairs = drv.capture(loss_fn)
    assert pairs[0][0].data_ptr() == pairs[1][0].data_ptr() == pairs[2][0].data_ptr()   # q, k, v
    key = dpsgd.step_seed(11, 0)
    n2, c, grads = drv.private_grads(pairs, key)
    torch.cuda.synchronize()
    A64 = [est.as_f64(A) for (A, _, _) in pairs]
    E64 = [est.as_f64(E) for (_, E, _) in pairs]
    n2_ref = sum(est.hutch_layer(A64[j], E64[j], k, key, j) for j in range(len(pairs)))
    assert np.all(np.abs(n2.cpu().numpy() - n2_ref) <= NORM_RTOL * n2_ref)
    c_ref = est.clip_scale(n2.cpu().numpy().astype(np.float64), C)     # same decision input
    assert np.allclose(c.cpu().numpy(), c_ref, rtol=1e-6)
    B = losses.numel()
    masters0 = [m.detach().cpu().double().numpy() for m in drv.master]
    g_ref = []
    for j in range(len(pairs)):
        clip = est.clip_accumulate(A64[j], E64[j], c_ref)
        ref = est.add_noise(clip, sigma, C, key, j)
        got = grads[j].cpu().double().numpy()
        assert np.linalg.norm(got - ref) <= GRAD_RTOL * np.linalg.norm(clip), j
        g_ref.append(ref / B)
    # AdamW (step 1) on the fp32 masters
    drv.apply(grads, B)
    torch.cuda.synchronize()
    for j, lin in enumerate(drv.linears):
        th, _, _ = est.adamw(masters0[j], g_ref[j], 0.0, 0.0, 1, 1e-3, 0.9, 0.999, 1e-8, 0.01)
        got = drv.master[j].detach().cpu().double().numpy()
        # the first update is lr g / (|g| + eps): flat except where |g| nears eps, so
        # entries with |g| below 1e-5 (a handful) may differ by up to the step size
        firm = np.abs(g_ref[j]) > 1e-5
        assert firm.mean() > 0.99
        assert np.max(np.abs(got - th)[firm]) <= 1e-6, j
        assert np.max(np.abs(got - th)) <= 2.1e-3, j
        assert torch.equal(lin.weight.detach(), drv.master[j].t().to(torch.bfloat16))
    drv.remove_hooks()


def test_fused_update_matches_oracle(mods):
    # steps 6-7 in one kernel per layer: noise + 1/B + AdamW + transposed bf16 weights
    D, dpsgd = mods
    C, sigma, k, lr, wd = 0.05, 0.6, 16, 1e-3, 0.01
    model, drv, loss_fn = _setup(dpsgd, C=C, sigma=sigma, k=k, seed=12, lr=lr, weight_decay=wd)
    assert drv.fused
    losses, pairs = drv.capture(loss_fn)
    key = dpsgd.step_seed(12, 0)
    n2, c, clipped = drv.private_grads(pairs, key, noise=False)
    torch.cuda.synchronize()
    B = losses.numel()
    masters0 = [m.detach().cpu().double().numpy() for m in drv.master]
    c_ref = est.clip_scale(n2.cpu().numpy().astype(np.float64), C)
    refs = []
    for (A, E, j) in pairs:
        A64, E64 = est.as_f64(A), est.as_f64(E)
        clip = est.clip_accumulate(A64, E64, c_ref)
        assert np.linalg.norm(clipped[j].cpu().double().numpy() - clip) <= GRAD_RTOL * np.linalg.norm(clip), j
        refs.append(est.private_gradient(A64, E64, c_ref, sigma, C, key, j, B))
    drv.update(clipped, B, key)
    torch.cuda.synchronize()
    for j, lin in enumerate(drv.linears):
        th, m, v = est.adamw(masters0[j], refs[j], 0.0, 0.0, 1, lr, 0.9, 0.999, 1e-8, wd)
        got = drv.master[j].detach().cpu().double().numpy()
        firm = np.abs(refs[j]) > 1e-5
        assert firm.mean() > 0.99
        assert np.max(np.abs(got - th)[firm]) <= 1e-6, j
        assert np.max(np.abs(got - th)) <= 2.1e-3, j
        assert np.allclose(drv.m[j].cpu().double().numpy(), m, rtol=1e-3, atol=1e-7)
        assert torch.equal(lin.weight.detach(), drv.master[j].t().to(torch.bfloat16))
    drv.remove_hooks()


def test_clipped_gradient_is_the_second_backward_pass(mods):
    # sum_i c_i A_i^T E_i equals the weight gradient of the scaled loss sum_i c_i L_i
    D, dpsgd = mods
    model, drv, loss_fn = _setup(dpsgd, C=0.05, sigma=0.0, k=16, seed=5)
    losses, pairs = drv.capture(loss_fn)
    _, c, grads = drv.private_grads(pairs, dpsgd.step_seed(0, 0))
    drv.remove_hooks()
    scaled = (loss_fn() * c).sum()
    gw = torch.autograd.grad(scaled, [lin.weight for lin in model.linears()])
    for j, g in enumerate(grads):
        ref = gw[j].float().t().cpu().double().numpy()
        assert _rel_fro(g.cpu().double().numpy(), ref) < 2e-2, j


@pytest.mark.parametrize("estimator,probe", [("hutchpp", "rademacher"), ("hutch", "gaussian")])
def test_step_estimator_options(mods, estimator, probe):
    D, dpsgd = mods
    model, drv, loss_fn = _setup(dpsgd, C=0.05, sigma=0.0, estimator=estimator, probe=probe, k=8, s=4, r=8,
                                 seed=7)
    losses, pairs = drv.capture(loss_fn)
    key = dpsgd.step_seed(7, 0)
    n2, c, grads = drv.private_grads(pairs, key)
    torch.cuda.synchronize()
    ref = 0.0
    for (A, E, j) in pairs:
        if estimator == "hutchpp":
            ref = ref + est.hutchpp_layer(est.as_f64(A), est.as_f64(E), 4, 8, key, j)
        else:
            ref = ref + est.hutch_layer(est.as_f64(A), est.as_f64(E), 8, key, j, probe=probe)
    assert np.all(np.abs(n2.cpu().numpy() - ref) <= NORM_RTOL * ref)
    drv.remove_hooks()


def test_training_steps_run_and_stay_finite(mods):
    D, dpsgd = mods
    model, drv, loss_fn = _setup(dpsgd, C=1.0, sigma=0.5, k=16, seed=2, lr=1e-3)
    w0 = model.lm_head.weight.detach().clone()
    for _ in range(3):
        losses = drv.step(loss_fn)
        assert torch.isfinite(losses).all()
        assert torch.isfinite(drv.last["n2"]).all() and (drv.last["c"] > 0).all()
    assert drv.steps == 3
    assert not torch.equal(model.lm_head.weight, w0)
    drv.remove_hooks()
