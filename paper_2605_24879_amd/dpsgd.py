"""One DP-SGD-RC training step (Alg. DP-SGD-RC) around libdprc.

Per step:

1. forward with hooks: each trained bias-free linear layer keeps its input A
   ([B, T, d]) and its output S ([B, T, p]);
2. one autograd pass from the summed per-sample losses to the layer outputs
   gives E = dL/dS for every layer (the backward-hook step of the algorithm;
   sample i's rows of E are dL_i/dS_i because samples do not interact, and
   no weight gradient is formed);
3. ``dprc_norm_hutch`` (or ``dprc_norm_hutchpp``) estimates every sample's
   squared gradient norm summed over the layers; adjacent layers that read
   the same activations (q, k, v; gate, up) share one pass over A;
4. ``dprc_clip_scale``: c_i = min(1, C / sqrt(n_i));
5. ``dprc_clip_accumulate_layers``: each layer's clipped gradient sum_i c_i A_i^T E_i
   is formed directly on the matrix cores.  For a linear layer it equals the
   weight gradient of the scaled loss sum_i c_i L_i, i.e. the algorithm's
   second backward pass, without running it;
6. ``dprc_add_noise``: + sigma C N(0, I) per element of the summed gradient;
7. AdamW on fp32 master weights (kept in the [d, p] layout of the clipped
   gradient) with the private gradient divided by the batch size, then the
   bf16 weights are refreshed from the masters.  By default steps 6 and 7
   run as one ``dprc_private_adamw`` pass per layer (noise, division, AdamW
   and the transposed bf16 weight write); ``fused_adamw=False`` runs
   ``dprc_add_noise`` and ``torch.optim.AdamW`` instead.

Only the listed linear layers are trained; every other parameter (embedding,
norms) is held fixed.  Probes and noise are keyed by a per-step seed derived
from (seed, step), so they are fresh every step.
"""

import torch

from . import dprc as D

_GOLDEN = 0x9E3779B97F4A7C15


def _rows(x):
    B, T, n = x.shape
    return x if x.stride(2) == 1 and x.stride(0) == T * x.stride(1) else x.contiguous()


def step_seed(seed, step):
    """The key of step ``step``: seed + step * 0x9E3779B97F4A7C15 mod 2^64."""
    return (int(seed) + int(step) * _GOLDEN) & 0xFFFFFFFFFFFFFFFF


class DPSGDRC:
    """DP-SGD with randomized clipping for a model's bias-free linear layers.

    ``linears``: the trained ``nn.Linear`` modules (bias-free), in model order
    so that layers reading the same input are adjacent.  ``estimator``:
    "hutch" (k probes, ``probe`` "rademacher" or "gaussian") or "hutchpp"
    (sketch s, residual probes r).  ``C``: clipping threshold; ``sigma``:
    noise multiplier.  AdamW hyper-parameters as in ``torch.optim.AdamW``.
    """

    def __init__(self, linears, C, sigma, estimator="hutch", k=16, probe="rademacher", s=16, r=32,
                 side=D.SIDE_OUT, seed=0, lr=1e-4, betas=(0.9, 0.999), eps=1e-8, weight_decay=0.0,
                 fused_adamw=True):
        self.linears = list(linears)
        for lin in self.linears:
            if lin.bias is not None:
                raise ValueError("DP-SGD-RC here covers bias-free linear layers")
        if estimator not in ("hutch", "hutchpp"):
            raise ValueError(estimator)
        self.C, self.sigma = float(C), float(sigma)
        self.estimator, self.k, self.s, self.r, self.side, self.seed = estimator, k, s, r, side, seed
        self.probe = {"rademacher": D.PROBE_RADEMACHER, "gaussian": D.PROBE_GAUSSIAN}[probe]
        self.master = [lin.weight.detach().t().float().contiguous() for lin in self.linears]
        for lin in self.linears:
            lin.weight.requires_grad_(True)
        self.hp = dict(lr=lr, beta1=betas[0], beta2=betas[1], eps=eps, weight_decay=weight_decay)
        self.fused = bool(fused_adamw)
        if self.fused:
            self.m = [torch.zeros_like(x) for x in self.master]
            self.v = [torch.zeros_like(x) for x in self.master]
        else:
            self.opt = torch.optim.AdamW(self.master, lr=lr, betas=betas, eps=eps, weight_decay=weight_decay)
        self.steps = 0
        self._A = [None] * len(self.linears)
        self._S = [None] * len(self.linears)
        self._hooks = [lin.register_forward_hook(self._tap(j)) for j, lin in enumerate(self.linears)]
        self._ws_acc = None
        self.last = {}

    def _tap(self, j):
        def hook(mod, inputs, output):
            self._A[j] = inputs[0]
            self._S[j] = output
        return hook

    def remove_hooks(self):
        for h in self._hooks:
            h.remove()

    def capture(self, loss_fn):
        """Steps 1-2: per-sample losses [B] and the layers' (A, E) pairs."""
        losses = loss_fn()
        if losses.dim() != 1:
            raise ValueError("loss_fn must return per-sample losses [B]")
        E = torch.autograd.grad(losses.sum(), self._S)
        # token-row layouts for the library (no copy when already so; layers fed the
        # same activations keep one pointer, so they share a pass over A)
        pairs = [(_rows(self._A[j].detach()), _rows(E[j]), j) for j in range(len(self.linears))]
        self._A = [None] * len(self.linears)
        self._S = [None] * len(self.linears)
        return losses.detach(), pairs

    def private_grads(self, pairs, key, noise=True):
        """Steps 3-6: n2 [B], c [B] and the clipped gradients ([d, p] fp32 per layer), with
        the noise added unless ``noise`` is false."""
        if self.estimator == "hutch":
            n2, c = D.dprc_norm_hutch_clip(pairs, self.k, key, self.C, side=self.side, probe=self.probe)
        else:
            n2 = D.dprc_norm_hutchpp(pairs, self.s, self.r, key, side=self.side)
            c = D.dprc_clip_scale(n2, self.C)
        grads = self.clipped_sums(pairs, c)
        if noise and self.sigma > 0:
            for (A, E, j), g in zip(pairs, grads):
                D.dprc_add_noise(g, self.sigma, self.C, key, j)
        return n2, c, grads

    def clipped_sums(self, pairs, c):
        """Step 5 for every layer: one call when all are bf16 (the small layers share
        launches), else one call per layer."""
        if all(A.dtype == torch.bfloat16 and E.dtype == torch.bfloat16 for (A, E, _) in pairs):
            return D.dprc_clip_accumulate_layers(pairs, c)
        need = max(D.dprc_clip_accumulate_workspace(A, E) for (A, E, _) in pairs)
        if self._ws_acc is None or self._ws_acc.numel() < need:
            self._ws_acc = torch.empty(max(need, 1), dtype=torch.uint8, device=c.device)
        return [D.dprc_clip_accumulate(A, E, c, ws=self._ws_acc) for (A, E, _) in pairs]

    def update(self, clipped, batch, key):
        """Steps 6-7 fused: per layer, noise + 1/batch + AdamW + bf16 weight write in one pass."""
        t = self.steps + 1
        for j, (lin, th, G) in enumerate(zip(self.linears, self.master, clipped)):
            D.dprc_private_adamw(th, self.m[j], self.v[j], G, self.sigma, self.C, key, j, 1.0 / batch,
                                 step=t, w=lin.weight.detach(), **self.hp)
            lin.weight.grad = None
        self.steps = t

    def apply(self, grads, batch):
        """Step 7 with torch's AdamW (noisy grads / batch), then refresh the model weights."""
        for m, g in zip(self.master, grads):
            m.grad = g.div_(batch)
        self.opt.step()
        with torch.no_grad():
            for lin, m in zip(self.linears, self.master):
                lin.weight.copy_(m.t())
                lin.weight.grad = None
        self.opt.zero_grad(set_to_none=True)
        self.steps += 1

    def step(self, loss_fn):
        """One full step; returns the per-sample losses (before the update)."""
        losses, pairs = self.capture(loss_fn)
        key = step_seed(self.seed, self.steps)
        n2, c, grads = self.private_grads(pairs, key, noise=not self.fused)
        del pairs
        if self.fused:
            self.update(grads, losses.numel(), key)
        else:
            self.apply(grads, losses.numel())
        self.last = {"n2": n2, "c": c}
        return losses
