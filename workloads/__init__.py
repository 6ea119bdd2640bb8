"""Seeded synthetic inputs for the DP-SGD-RC norm-estimation path.

This module only draws inputs; it holds none of the method's arithmetic, and
both the CPU oracle's tests and the GPU path consume the same tensors from it.

The five workloads stand in for the paper's Llama-3.2-1B fine-tuning runs
(datasets and trained weights are not available): they take the layer shapes
of that model (hidden 2048, MLP 8192, key/value width 512, vocabulary 128256)
and synthetic activations / output gradients with the value laws below.

* ``tiny``    : one 64 -> 48 layer, B=2, T=64, fp32; A ~ N(0,1); sample i's
                output gradient ~ N(0, sigma_i^2), sigma_i = 10^U(-1,1).
* ``q_proj``  : one 2048 -> 2048 layer, B=4, T=2048, bf16; A ~ N(0,1);
                E_i ~ N(0, 1e-4 s_i^2), s_i = exp(N(0,1)) per sample.
* ``mlp``     : gate, up (2048 -> 8192) and down (8192 -> 2048), B=2, T=8192,
                bf16, laws as ``q_proj``.
* ``decoder`` : q, k, v, o, gate, up, down of one decoder layer, B=1,
                T=32768, bf16; A ~ N(0,1); E = 0.01 * Student-t(3).
* ``stack``   : 16 decoder layers x 7 projections + a 2048 -> 128256 lm_head,
                B=8, T=4096, bf16, laws as ``q_proj``.

bf16 inputs are drawn in fp32 and rounded to nearest-even; the oracle reads the
identical bf16 values.  Every layer has its own generator stream, so a layer's
inputs do not depend on which other layers were drawn.
"""

import math

import torch

HIDDEN, MLP, KV, VOCAB = 2048, 8192, 512, 128256

DECODER_LAYERS = [("q", HIDDEN, HIDDEN), ("k", HIDDEN, KV), ("v", HIDDEN, KV), ("o", HIDDEN, HIDDEN),
                  ("gate", HIDDEN, MLP), ("up", HIDDEN, MLP), ("down", MLP, HIDDEN)]

CONFIGS = [
    dict(name="tiny", layers=[("fc", 64, 48)], B=2, T=64, dtype="f32", law="loguniform",
         estimator="hutch", k=4, C=1.0, accumulate=True, noise_sigma=None),
    dict(name="q_proj", layers=[("q", HIDDEN, HIDDEN)], B=4, T=2048, dtype="bf16", law="lognormal",
         estimator="hutch", k=16, C=1.0, accumulate=False, noise_sigma=None),
    dict(name="mlp", layers=[("gate", HIDDEN, MLP), ("up", HIDDEN, MLP), ("down", MLP, HIDDEN)],
         B=2, T=8192, dtype="bf16", law="lognormal", estimator="hutch", k=16, C=1.0,
         accumulate=True, noise_sigma=None),
    dict(name="decoder", layers=list(DECODER_LAYERS), B=1, T=32768, dtype="bf16", law="student_t",
         estimator="hutchpp", s=16, r=32, C=1.0, accumulate=False, noise_sigma=None),
    dict(name="stack",
         layers=[(f"L{l}.{n}", d, p) for l in range(16) for (n, d, p) in DECODER_LAYERS]
         + [("lm_head", HIDDEN, VOCAB)],
         B=8, T=4096, dtype="bf16", law="lognormal", estimator="hutch", k=32, C=1.0,
         accumulate=True, noise_sigma=0.8),
]
BY_NAME = {c["name"]: c for c in CONFIGS}


def torch_dtype(name):
    return {"f32": torch.float32, "bf16": torch.bfloat16}[name]


def _gen(device, seed, stream):
    g = torch.Generator(device=device)
    g.manual_seed((int(seed) * 1_000_003 + int(stream)) % (2 ** 63))
    return g


def sample_scales(law, B, seed=0, device="cpu"):
    """Per-sample output-gradient scale (std) used by ``law``; shared by all layers."""
    g = _gen("cpu", seed, 999_983)
    if law == "loguniform":
        u = torch.rand(B, generator=g, dtype=torch.float64) * 2.0 - 1.0
        s = 10.0 ** u
    elif law == "lognormal":
        s = 0.01 * torch.exp(torch.randn(B, generator=g, dtype=torch.float64))
    elif law == "student_t":
        s = torch.full((B,), 0.01, dtype=torch.float64)
    elif law == "unit":
        s = torch.ones(B, dtype=torch.float64)
    else:
        raise ValueError(law)
    return s.to(device=device, dtype=torch.float32)


def draw(B, T, d, p, dtype="bf16", law="lognormal", seed=0, layer=0, device="cpu",
         row_pad_a=0, row_pad_e=0):
    """Activations A [B,T,d] and output gradients E [B,T,p] for one layer.

    ``row_pad_*`` > 0 returns strided views whose token rows are longer than
    the logical width (to exercise row strides).
    """
    g = _gen(device, seed, 2 * layer + 1)
    dt = torch_dtype(dtype)
    A = torch.randn(B, T, d + row_pad_a, generator=g, device=device, dtype=torch.float32)
    if law == "student_t":
        z = torch.randn(B, T, p + row_pad_e, generator=g, device=device, dtype=torch.float32)
        chi = torch.zeros_like(z)
        for _ in range(3):
            chi += torch.randn(B, T, p + row_pad_e, generator=g, device=device, dtype=torch.float32) ** 2
        E = 0.01 * z / torch.sqrt(chi / 3.0)
        del chi, z
    else:
        E = torch.randn(B, T, p + row_pad_e, generator=g, device=device, dtype=torch.float32)
        s = sample_scales(law, B, seed, device)
        E *= s.view(B, 1, 1)
    A = A.to(dt)
    E = E.to(dt)
    if row_pad_a:
        A = A[:, :, :d]
    if row_pad_e:
        E = E[:, :, :p]
    return A, E


def layer_inputs(cfg, li, device="cpu", seed=0):
    """(A, E) of layer ``li`` of a named workload."""
    _, d, p = cfg["layers"][li]
    return draw(cfg["B"], cfg["T"], d, p, cfg["dtype"], cfg["law"], seed=seed, layer=li, device=device)


def algorithmic_norm_bytes(cfg):
    """Bytes the norm stage must read: sum over layers of B*T*(d+p)*elem (x3 for Hutch++ passes)."""
    elem = 4 if cfg["dtype"] == "f32" else 2
    per = sum(cfg["B"] * cfg["T"] * (d + p) * elem for (_, d, p) in cfg["layers"])
    return per * (3 if cfg["estimator"] == "hutchpp" else 1)


def accumulate_flops(cfg):
    return sum(2 * cfg["B"] * cfg["T"] * d * p for (_, d, p) in cfg["layers"])


def describe(cfg):
    return {"workload": cfg["name"], "B": cfg["B"], "T": cfg["T"],
            "layers": [f"{n}:{d}x{p}" for (n, d, p) in cfg["layers"]][:8]
            + ([f"... {len(cfg['layers'])} layers"] if len(cfg["layers"]) > 8 else []),
            "dtype": cfg["dtype"], "estimator": cfg["estimator"],
            "probes": cfg.get("k", None) if cfg["estimator"] == "hutch" else f"s={cfg['s']},r={cfg['r']}"} \
        | ({"probe_family": cfg.get("probe", "rademacher")} if cfg["estimator"] == "hutch" else {})


def ceil_div(a, b):
    return -(-a // b)


__all__ = ["CONFIGS", "BY_NAME", "draw", "layer_inputs", "sample_scales", "algorithmic_norm_bytes",
           "accumulate_flops", "describe", "ceil_div", "math"]
