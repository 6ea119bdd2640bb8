"""Host logic of the end-to-end DP-SGD-RC step (no GPU): the activations and
output gradients that the step driver captures are the ones per-sample
gradients are made of.

The model is the Llama-shaped stack at toy sizes in fp32 on the CPU.  The
captured (A, E) of every trained layer must give A_i^T E_i equal to the
gradient of sample i's own loss obtained by running that sample alone through
torch autograd, and layers fed the same activations must see one tensor.
"""

import numpy as np
import torch

from paper_2605_24879_amd import dpsgd
from workloads import llama

SIZES = dict(layers=2, hidden=32, mlp=48, heads=4, kv_heads=2, vocab=37)


def _model():
    torch.manual_seed(0)
    return llama.build(seed=3, device="cpu", dtype=torch.float32, **SIZES)


def test_capture_gives_per_sample_gradients():
    model = _model()
    tok = llama.tokens(3, 9, SIZES["vocab"], seed=4, device="cpu")
    drv = dpsgd.DPSGDRC(model.linears(), C=1.0, sigma=0.0)
    losses, pairs = drv.capture(lambda: llama.per_sample_loss(model(tok[:, :-1]), tok[:, 1:]))
    assert losses.shape == (3,)
    lins = model.linears()
    for i in range(3):
        model.zero_grad(set_to_none=True)
        li = llama.per_sample_loss(model(tok[i:i + 1, :-1]), tok[i:i + 1, 1:])[0]
        gw = torch.autograd.grad(li, [m.weight for m in lins])
        for (A, E, j) in pairs:
            got = A[i].double().T @ E[i].double()                 # [d, p] = weight gradient^T
            ref = gw[j].double().T
            assert torch.allclose(got, ref, rtol=1e-4, atol=1e-7 * ref.abs().max().item()), (i, j)
    drv.remove_hooks()


def test_shared_inputs_are_one_tensor():
    model = _model()
    tok = llama.tokens(2, 5, SIZES["vocab"], device="cpu")
    drv = dpsgd.DPSGDRC(model.linears(), C=1.0, sigma=0.0)
    _, pairs = drv.capture(lambda: llama.per_sample_loss(model(tok[:, :-1]), tok[:, 1:]))
    ptr = [A.data_ptr() for (A, _, _) in pairs]
    for blk in range(SIZES["layers"]):
        q, k, v, o, gate, up, down = ptr[7 * blk:7 * blk + 7]
        assert q == k == v and gate == up
        assert len({q, o, gate, down}) == 4
    drv.remove_hooks()


def test_step_seed_changes_every_step():
    keys = {dpsgd.step_seed(7, t) for t in range(100)}
    assert len(keys) == 100 and all(0 <= x < 2 ** 64 for x in keys)
    assert dpsgd.step_seed(7, 0) == 7
