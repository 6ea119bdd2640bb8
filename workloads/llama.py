"""A Llama-3.2-1B-shaped decoder stack with seeded random weights.

It is the synthetic model of the end-to-end DP-SGD-RC step (no trained weights
or datasets are available): token embedding, ``layers`` blocks of RMSNorm ->
grouped-query attention with rotary positions -> residual, RMSNorm -> SwiGLU
MLP -> residual, a final RMSNorm and an untied lm_head.  Every projection is a
bias-free ``nn.Linear``.  Default sizes are Llama-3.2-1B's: hidden 2048, MLP
8192, 32 query heads and 8 key/value heads of width 64, vocabulary 128256, 16
blocks, rotary base 500000.

Attention scores, softmax and the value product run in fp32 on contiguous
operands; the projections run in the weights' dtype (bf16 by default).  q, k
and v read the same normed activations, as do gate and up.

``linears()`` lists the projections in model order (per block q, k, v, o,
gate, up, down; then lm_head), which keeps the shared-input layers adjacent.
"""

import math

import torch
import torch.nn as nn
import torch.nn.functional as F

LLAMA_3_2_1B = dict(layers=16, hidden=2048, mlp=8192, heads=32, kv_heads=8, vocab=128256, rope_base=500000.0)


class RMSNorm(nn.Module):
    def __init__(self, n, eps=1e-5):
        super().__init__()
        self.weight = nn.Parameter(torch.ones(n))
        self.eps = eps

    def forward(self, x):
        xf = x.float()
        y = xf * torch.rsqrt(xf.pow(2).mean(-1, keepdim=True) + self.eps)
        return (y * self.weight.float()).to(x.dtype)


def _rope_tables(T, hd, base, device):
    inv = 1.0 / (base ** (torch.arange(0, hd, 2, device=device, dtype=torch.float32) / hd))
    ang = torch.arange(T, device=device, dtype=torch.float32)[:, None] * inv[None, :]
    return torch.cos(ang), torch.sin(ang)


def _rope(x, cos, sin):
    # x: [B, H, T, hd] fp32; rotate the (first half, second half) pairs
    h = x.shape[-1] // 2
    x1, x2 = x[..., :h], x[..., h:]
    return torch.cat([x1 * cos - x2 * sin, x2 * cos + x1 * sin], dim=-1)


class Block(nn.Module):
    def __init__(self, hidden, mlp, heads, kv_heads):
        super().__init__()
        hd = hidden // heads
        self.heads, self.kv_heads, self.hd = heads, kv_heads, hd
        self.norm1 = RMSNorm(hidden)
        self.q = nn.Linear(hidden, heads * hd, bias=False)
        self.k = nn.Linear(hidden, kv_heads * hd, bias=False)
        self.v = nn.Linear(hidden, kv_heads * hd, bias=False)
        self.o = nn.Linear(heads * hd, hidden, bias=False)
        self.norm2 = RMSNorm(hidden)
        self.gate = nn.Linear(hidden, mlp, bias=False)
        self.up = nn.Linear(hidden, mlp, bias=False)
        self.down = nn.Linear(mlp, hidden, bias=False)

    def forward(self, x, cos, sin, mask):
        B, T, _ = x.shape
        h = self.norm1(x)
        q = self.q(h).view(B, T, self.heads, self.hd).transpose(1, 2).float()
        k = self.k(h).view(B, T, self.kv_heads, self.hd).transpose(1, 2).float()
        v = self.v(h).view(B, T, self.kv_heads, self.hd).transpose(1, 2).float()
        q, k = _rope(q, cos, sin), _rope(k, cos, sin)
        rep = self.heads // self.kv_heads
        k = k.repeat_interleave(rep, dim=1)
        v = v.repeat_interleave(rep, dim=1).contiguous()
        s = torch.matmul(q.contiguous(), k.transpose(-1, -2).contiguous()) * (1.0 / math.sqrt(self.hd))
        p = torch.softmax(s + mask, dim=-1)
        a = torch.matmul(p, v).transpose(1, 2).reshape(B, T, self.heads * self.hd).to(x.dtype)
        x = x + self.o(a)
        h = self.norm2(x)
        return x + self.down(F.silu(self.gate(h)) * self.up(h))


class LlamaShaped(nn.Module):
    def __init__(self, layers=16, hidden=2048, mlp=8192, heads=32, kv_heads=8, vocab=128256,
                 rope_base=500000.0):
        super().__init__()
        self.embed = nn.Embedding(vocab, hidden)
        self.blocks = nn.ModuleList([Block(hidden, mlp, heads, kv_heads) for _ in range(layers)])
        self.norm = RMSNorm(hidden)
        self.lm_head = nn.Linear(hidden, vocab, bias=False)
        self.rope_base = rope_base
        self.hd = hidden // heads

    def linears(self):
        out = []
        for b in self.blocks:
            out += [b.q, b.k, b.v, b.o, b.gate, b.up, b.down]
        return out + [self.lm_head]

    def forward(self, tokens):
        B, T = tokens.shape
        cos, sin = _rope_tables(T, self.hd, self.rope_base, tokens.device)
        mask = torch.full((T, T), float("-inf"), device=tokens.device).triu(1)
        x = self.embed(tokens)
        for b in self.blocks:
            x = b(x, cos, sin, mask)
        return self.lm_head(self.norm(x))


def build(seed=0, device="cuda", dtype=torch.bfloat16, **sizes):
    """A seeded LlamaShaped model (weights ~ N(0, 0.02^2), norms 1) in ``dtype``."""
    cfg = dict(LLAMA_3_2_1B)
    cfg.update(sizes)
    g = torch.Generator(device=device).manual_seed(seed)
    with torch.device("meta"):
        model = LlamaShaped(**cfg)
    model = model.to_empty(device=device)
    with torch.no_grad():
        for name, prm in model.named_parameters():
            if prm.dim() == 2:
                prm.normal_(0.0, 0.02, generator=g)
            else:
                prm.fill_(1.0)
    return model.to(dtype)


def tokens(B, T, vocab, seed=0, device="cuda"):
    """Seeded token ids [B, T + 1] (inputs are [:, :-1], next-token targets [:, 1:])."""
    g = torch.Generator(device=device).manual_seed(seed + 1)
    return torch.randint(0, vocab, (B, T + 1), generator=g, device=device)


def per_sample_loss(logits, targets):
    """Mean next-token cross-entropy of each sample (fp32): [B]."""
    B, T, V = logits.shape
    ce = F.cross_entropy(logits.float().reshape(B * T, V), targets.reshape(B * T), reduction="none")
    return ce.view(B, T).mean(dim=1)
