"""GPU parity of libdprc against the CPU oracle on identical seeded inputs.

Sizes span several tiles with ragged tails (token counts, widths and probe
counts that are not multiples of the kernels' tiles).  Tolerances: probe bits
bit-exact; squared-norm estimates 1e-3 relative; clipped gradients 2e-3
relative Frobenius; noise 1e-5 * sigma * C absolute on the added term.
"""

import math

import numpy as np
import pytest
import torch

from oracle import philox
from oracle import estimators as est
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


def _draw(B, T, d, p, dtype="bf16", law="lognormal", layer=0, seed=0, **kw):
    return workloads.draw(B, T, d, p, dtype=dtype, law=law, seed=seed, layer=layer, device="cuda", **kw)


def _np(x):
    return est.as_f64(x)


def _rel(a, b):
    a, b = np.asarray(a, dtype=np.float64), np.asarray(b, dtype=np.float64)
    return np.abs(a - b) / np.maximum(np.abs(b), 1e-300)


def _hadamard_words(m, k):
    H = philox.hadamard_matrix(m, k)           # +-1
    bits = (H < 0).astype(np.uint64).T         # [k, m]
    nw = (m + 31) // 32
    out = np.zeros((k, nw), dtype=np.uint64)
    for u in range(m):
        out[:, u // 32] |= bits[:, u] << np.uint64(u % 32)
    return out.astype(np.uint32)


# ---- probe bits --------------------------------------------------------------------------

@pytest.mark.parametrize("seed,layer,stream,m,k", [
    (0, 0, 0, 48, 4), (0, 3, 1, 2048, 16), (12345678901234, 7, 0, 45, 3), (5, 112, 0, 128256, 2),
    (2**64 - 1, 2**32 - 1, 2, 100, 33), (9, 1, 0, 1, 1), (9, 1, 0, 130, 1)])
def test_probe_bits_bitexact(D, seed, layer, stream, m, k):
    got = D.dprc_probe_bits(D.PROBE_RADEMACHER, seed, layer, stream, m, k).cpu().numpy().view(np.uint32)
    ref = philox.rademacher_words(seed, layer, stream, m, k)
    assert np.array_equal(got, ref)


@pytest.mark.parametrize("m,k", [(64, 64), (48, 64), (100, 7)])
def test_hadamard_bits_bitexact(D, m, k):
    got = D.dprc_probe_bits(D.PROBE_HADAMARD, 0, 0, 0, m, k).cpu().numpy().view(np.uint32)
    assert np.array_equal(got, _hadamard_words(m, k))


@pytest.mark.parametrize("seed,layer,m,k", [
    (0, 0, 48, 4), (7, 3, 130, 33), (2**64 - 1, 2**32 - 1, 1, 1), (11, 5, 4097, 2)])
def test_gaussian_probe_values(D, seed, layer, m, k):
    # fp32 Box-Muller on the GPU against the fp64 transform of the same Philox words
    got = D.dprc_probe_gaussian(seed, layer, m, k).cpu().numpy().astype(np.float64).T
    ref = philox.gaussian_probe_matrix(seed, layer, m, k)
    assert got.shape == ref.shape
    assert np.all(np.abs(got - ref) <= 2e-6 * np.maximum(1.0, np.abs(ref)))


# ---- Hutchinson ---------------------------------------------------------------------------

@pytest.mark.parametrize("B,T,d,p,k,side", [
    (3, 200, 300, 260, 16, 0),     # ragged tokens / widths, 3 x 3 tiles
    (2, 130, 72, 520, 5, 1),       # side IN, odd k
    (2, 96, 520, 72, 33, 2),       # AUTO -> IN (d > p), 3 column blocks
    (1, 1, 8, 8, 1, 0),            # a single token
    (2, 64, 64, 48, 4, 0),         # the tiny workload's shape in bf16
])
def test_hutch_parity_bf16(D, B, T, d, p, k, side):
    A, E = _draw(B, T, d, p, layer=1)
    n2l = torch.zeros(1, B, device="cuda")
    n2 = D.dprc_norm_hutch([(A, E, 1)], k, 42, side=side, n2_layers=n2l)
    ref = est.hutch_layer(_np(A), _np(E), k, 42, 1, side=side)
    assert np.all(_rel(n2.cpu().numpy(), ref) < NORM_RTOL)
    assert torch.equal(n2, n2l[0])


@pytest.mark.parametrize("B,T,d,p,k,side,dtype", [
    (3, 200, 300, 260, 16, 0, "bf16"),    # ragged tokens / widths
    (2, 130, 72, 1100, 5, 1, "bf16"),     # side IN, odd k, wide reduced operand
    (2, 96, 1100, 72, 32, 2, "bf16"),     # AUTO -> IN, 1100 sketched columns (3 stages), k at its maximum
    (1, 1, 8, 8, 1, 0, "bf16"),           # a single token
    (2, 64, 64, 48, 4, 0, "f32"),
    (2, 100, 130, 70, 32, 1, "f32"),
])
def test_hutch_gaussian_parity(D, B, T, d, p, k, side, dtype):
    A, E = _draw(B, T, d, p, dtype=dtype, layer=6)
    n2 = D.dprc_norm_hutch([(A, E, 4)], k, 77, side=side, probe=D.PROBE_GAUSSIAN)
    ref = est.hutch_layer(_np(A), _np(E), k, 77, 4, side=side, probe="gaussian")
    assert np.all(_rel(n2.cpu().numpy(), ref) < NORM_RTOL)


def test_hutch_gaussian_multilayer_accumulate(D):
    # per-layer probes differ (layer id in the counter); the workspace is reused across layers
    A1, E1 = _draw(2, 300, 256, 200, layer=0)
    A2, E2 = _draw(2, 150, 136, 700, layer=1)
    n2 = torch.tensor([0.5, 1.0], device="cuda")
    n2l = torch.zeros(2, 2, device="cuda")
    D.dprc_norm_hutch([(A1, E1, 20), (A2, E2, 21)], 8, 3, probe=D.PROBE_GAUSSIAN, n2=n2, n2_layers=n2l,
                      accumulate=True)
    r1 = est.hutch_layer(_np(A1), _np(E1), 8, 3, 20, probe="gaussian")
    r2 = est.hutch_layer(_np(A2), _np(E2), 8, 3, 21, probe="gaussian")
    got = n2l.cpu().numpy()
    assert np.all(_rel(got[0], r1) < NORM_RTOL) and np.all(_rel(got[1], r2) < NORM_RTOL)
    assert np.all(_rel(n2.cpu().numpy(), np.array([0.5, 1.0]) + r1 + r2) < NORM_RTOL)


# ---- layers sharing their activations (one token reduction over A) -------------------------

def _shared_a(B, T, d, ps, layer0=0):
    """Layers that read the same A (as q, k, v do), each with its own E."""
    A, _ = _draw(B, T, d, 8, layer=layer0)
    Es = [_draw(B, T, 8, p, layer=layer0 + 1 + j)[1] for j, p in enumerate(ps)]
    return A, Es


@pytest.mark.parametrize("B,T,d,ps,k,probe", [
    (2, 200, 300, (260, 72, 72), 16, "rademacher"),     # q, k, v-like widths (ragged)
    (3, 130, 136, (520, 520), 5, "rademacher"),         # gate/up-like pair, k not a multiple of 16
    (2, 700, 256, (200, 100, 64, 48, 30), 16, "rademacher"),   # five sharing layers -> groups of 4 and 1
    (2, 96, 64, (128, 40, 72), 100, "rademacher"),      # 3k > 256 columns -> groups of 2 and 1
    (2, 100, 64, (1100, 600), 16, "rademacher"),        # wide, unequal sketched sides in one group
    (2, 150, 520, (96, 260), 7, "gaussian"),
])
def test_hutch_shared_activations(D, B, T, d, ps, k, probe):
    A, Es = _shared_a(B, T, d, ps)
    pairs = [(A, E, 30 + j) for j, E in enumerate(Es)]
    pid = D.PROBE_GAUSSIAN if probe == "gaussian" else D.PROBE_RADEMACHER
    n2l = torch.zeros(len(Es), B, device="cuda")
    n2 = D.dprc_norm_hutch(pairs, k, 8, probe=pid, n2_layers=n2l)
    refs = [est.hutch_layer(_np(A), _np(E), k, 8, 30 + j, probe=probe) for j, E in enumerate(Es)]
    got = n2l.cpu().numpy()
    for j in range(len(Es)):
        assert np.all(_rel(got[j], refs[j]) < NORM_RTOL), j
    assert np.all(_rel(n2.cpu().numpy(), np.sum(refs, axis=0)) < NORM_RTOL)
    # same estimates as with a private copy of A per layer (no shared reduction)
    n2l_sep = torch.zeros_like(n2l)
    n2_sep = D.dprc_norm_hutch([(A.clone(), E, 30 + j) for j, E in enumerate(Es)], k, 8, probe=pid,
                               n2_layers=n2l_sep)
    assert np.all(_rel(got, n2l_sep.cpu().numpy()) < 1e-6)
    assert np.all(_rel(n2.cpu().numpy(), n2_sep.cpu().numpy()) < 1e-6)
    if k % 16 == 0:
        assert torch.equal(n2l, n2l_sep)


def test_hutch_shared_activations_mixed_sides(D):
    # AUTO: q (d == p) sketches OUT, k/v (d > p) sketch IN; only OUT layers share a reduction
    A, Es = _shared_a(2, 160, 256, (256, 64, 64))
    pairs = [(A, E, 40 + j) for j, E in enumerate(Es)]
    n2l = torch.zeros(3, 2, device="cuda")
    D.dprc_norm_hutch(pairs, 16, 2, side=2, n2_layers=n2l)
    for j, E in enumerate(Es):
        ref = est.hutch_layer(_np(A), _np(E), 16, 2, 40 + j, side=2)
        assert np.all(_rel(n2l[j].cpu().numpy(), ref) < NORM_RTOL), j


@pytest.mark.parametrize("k,probe", [(16, "rademacher"), (12, "hadamard"), (40, "rademacher"),
                                     (100, "rademacher")])
def test_hutch_many_groups_batched(D, k, probe):
    # 15 bf16 layers in 11 activation groups (one batch of up to 32): shared groups of
    # three and two layers between single layers, so one batch holds more than eight
    # projections and token reductions of several column counts (k = 40: groups over 64
    # columns; k = 100: projections over 64 columns, one launch each)
    B, T = 2, 150
    groups = [(96, (130, 72, 72)), (64, (300,)), (136, (520, 260)), (48, (90,)), (80, (200,)),
              (72, (64,)), (40, (150,)), (88, (110, 96)), (56, (70,)), (64, (260,)), (120, (100,))]
    pairs, lid = [], 0
    for g, (d, ps) in enumerate(groups):
        A, Es = _shared_a(B, T, d, ps, layer0=60 + 10 * g)
        for E in Es:
            pairs.append((A, E, lid))
            lid += 1
    pid = D.PROBE_HADAMARD if probe == "hadamard" else D.PROBE_RADEMACHER
    n2l = torch.zeros(len(pairs), B, device="cuda")
    n2 = D.dprc_norm_hutch(pairs, k, 3, probe=pid, n2_layers=n2l)
    refs = [est.hutch_layer(_np(A), _np(E), k, 3, j, probe=probe) for (A, E, j) in pairs]
    got = n2l.cpu().numpy()
    for j in range(len(pairs)):
        assert np.all(_rel(got[j], refs[j]) < NORM_RTOL), j
    assert np.all(_rel(n2.cpu().numpy(), np.sum(refs, axis=0)) < NORM_RTOL)
    # each layer's estimate as from a call of its own (no batching, no shared reduction)
    solo = torch.stack([D.dprc_norm_hutch([(A.clone(), E, j)], k, 3, probe=pid) for (A, E, j) in pairs])
    assert np.all(_rel(got, solo.cpu().numpy()) < 1e-6)
    if k % 16 == 0:
        assert torch.equal(n2l, solo)


@pytest.mark.parametrize("accumulate", [False, True])
def test_hutch_more_groups_than_one_sample_sum(D, accumulate):
    # 131 single-layer groups (the per-sample sums of a call take 128 groups per launch, so
    # a second launch continues n2), ragged widths; each layer's estimate equals that of a
    # call of its own bit for bit, n2 their sum in layer order, the clip factors follow n2
    B, T, k, C = 3, 70, 16, 0.5
    pairs = []
    for j in range(131):
        d, p = 40 + 8 * (j % 5), 24 + 16 * (j % 7)
        A, E = _draw(B, T, d, p, layer=300 + j)
        pairs.append((A, E, j))
    n2l = torch.zeros(len(pairs), B, device="cuda")
    n2 = torch.full((B,), 0.25, device="cuda")
    c = torch.zeros(B, device="cuda")
    D.dprc_norm_hutch_clip(pairs, k, 9, C, n2=n2, c=c, n2_layers=n2l, accumulate=accumulate)
    solo = torch.stack([D.dprc_norm_hutch([(A, E, j)], k, 9) for (A, E, j) in pairs])
    assert torch.equal(n2l, solo)
    ref = np.full(B, 0.25 if accumulate else 0.0, dtype=np.float32)
    for j in range(len(pairs)):                       # float adds in layer order
        ref = (ref + solo[j].cpu().numpy()).astype(np.float32)
    assert np.array_equal(n2.cpu().numpy(), ref)
    assert np.allclose(c.cpu().numpy(), est.clip_scale(ref.astype(np.float64), C), rtol=1e-6)
    for j in (0, 64, 127, 128, 130):                  # against the oracle
        A, E, _ = pairs[j]
        assert np.all(_rel(n2l[j].cpu().numpy(), est.hutch_layer(_np(A), _np(E), k, 9, j)) < NORM_RTOL), j


@pytest.mark.parametrize("k", [32, 20])
def test_hutch_large_batch_unsplit(D, k):
    # a batch of eight layers with 1028 (sample, 128-column tile) pairs: its token reductions
    # run without token splits (one workgroup per pair of tiles over all 200 tokens, a ragged
    # last stage; the last layer has an odd number of tiles, its last one 8 columns wide), the
    # layers ragged in both widths; a second call of one layer runs split
    B, T = 4, 200
    shapes = [(4000, 300), (4096, 130), (4000, 520), (4096, 96), (4000, 72), (4096, 260), (4000, 1000), (4104, 40)]
    pairs = []
    for j, (d, p) in enumerate(shapes):
        A, E = _draw(B, T, d, p, layer=200 + j)
        pairs.append((A, E, j))
    n2l = torch.zeros(len(pairs), B, device="cuda")
    n2 = D.dprc_norm_hutch(pairs, k, 11, n2_layers=n2l)
    refs = [est.hutch_layer(_np(A), _np(E), k, 11, j) for (A, E, j) in pairs]
    got = n2l.cpu().numpy()
    for j in range(len(pairs)):
        assert np.all(_rel(got[j], refs[j]) < NORM_RTOL), j
    assert np.all(_rel(n2.cpu().numpy(), np.sum(refs, axis=0)) < NORM_RTOL)
    A, E, j = pairs[0]
    solo = D.dprc_norm_hutch([(A, E, j)], k, 11).cpu().numpy()     # 128 pairs: four token splits
    assert np.all(_rel(got[0], solo) < 1e-5)


@pytest.mark.parametrize("case,probe", [("narrow", "rademacher"), ("chunked", "rademacher"), ("narrow", "hadamard")])
def test_hutch_row_blocks_per_workgroup(D, case, probe):
    # a batch of 32 layers with enough row blocks that each projection workgroup streams
    # several of them (narrow: 512-wide E, four 32-row blocks per workgroup, one probe chunk
    # per row; chunked: 8200-wide E, four 16-row blocks per workgroup, three probe chunks per
    # row and a ragged last stage); a call of one layer gives each workgroup one block
    k = 32
    if case == "narrow":
        B, T, d, p, check = 8, 1024, 64, 512, range(32)
    else:
        B, T, d, p, check = 4, 1024, 48, 8200, (0, 17, 31)
    pairs = []
    for j in range(32):
        A, E = _draw(B, T, d, p, layer=400 + j)
        pairs.append((A, E, j))
    pid = D.PROBE_HADAMARD if probe == "hadamard" else D.PROBE_RADEMACHER
    n2l = torch.zeros(len(pairs), B, device="cuda")
    n2 = D.dprc_norm_hutch(pairs, k, 21, n2_layers=n2l, probe=pid)
    torch.cuda.synchronize()
    got = n2l.cpu().numpy()
    solo = torch.stack([D.dprc_norm_hutch([(A, E, j)], k, 21, probe=pid) for (A, E, j) in pairs]).cpu().numpy()
    assert np.all(_rel(got, solo) < 1e-5)
    assert np.all(_rel(n2.cpu().numpy(), got.astype(np.float64).sum(axis=0)) < 1e-5)
    for j in check:
        A, E, _ = pairs[j]
        assert np.all(_rel(got[j], est.hutch_layer(_np(A), _np(E), k, 21, j, probe=probe)) < NORM_RTOL), j


@pytest.mark.parametrize("B,T,p,k", [(1, 64, 4100, 16), (2, 40, 2600, 5), (1, 200, 4096, 32)])
def test_hutch_few_rows_wide_sketch(D, B, T, p, k):
    # few token rows and a wide sketched side (many 512-column stages per workgroup, ragged end)
    A, E = _draw(B, T, 72, p, layer=9)
    n2 = D.dprc_norm_hutch([(A, E, 3)], k, 5)
    ref = est.hutch_layer(_np(A), _np(E), k, 5, 3)
    assert np.all(_rel(n2.cpu().numpy(), ref) < NORM_RTOL)


@pytest.mark.parametrize("case", ["bf16", "shared", "gaussian", "fp32", "accumulate"])
def test_hutch_clip_fused_matches_separate_calls(D, case):
    C = 0.3
    if case == "shared":
        A, Es = _shared_a(3, 150, 200, (200, 64, 64))
        pairs = [(A, E, j) for j, E in enumerate(Es)]
    elif case == "fp32":
        A, E = _draw(2, 64, 64, 48, dtype="f32", layer=2)
        pairs = [(A, E, 0)]
    else:
        A, E = _draw(3, 130, 96, 300, layer=2)
        pairs = [(A, E, 0)]
    probe = D.PROBE_GAUSSIAN if case == "gaussian" else D.PROBE_RADEMACHER
    prior = torch.tensor([0.5, 0.01, 2.0][:pairs[0][0].shape[0]], device="cuda")
    acc = case == "accumulate"
    n2f, cf = D.dprc_norm_hutch_clip(pairs, 16, 4, C, probe=probe, n2=prior.clone() if acc else None, accumulate=acc)
    n2 = D.dprc_norm_hutch(pairs, 16, 4, probe=probe, n2=prior.clone() if acc else None, accumulate=acc)
    c = D.dprc_clip_scale(n2, C)
    assert torch.equal(n2f, n2) and torch.equal(cf, c)
    assert np.allclose(cf.cpu().numpy(), est.clip_scale(n2.cpu().numpy().astype(np.float64), C), rtol=1e-6)


def test_hutch_tiny_workload_fp32(D):
    cfg = workloads.BY_NAME["tiny"]
    A, E = workloads.layer_inputs(cfg, 0, device="cuda")
    n2 = D.dprc_norm_hutch([(A, E, 0)], cfg["k"], 0)
    ref = est.hutch_layer(_np(A), _np(E), cfg["k"], 0, 0)
    assert np.all(_rel(n2.cpu().numpy(), ref) < NORM_RTOL)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("side", [0, 1])
def test_hutch_hadamard_probes_give_exact_norm(D, dtype, side):
    # 64 Sylvester-Hadamard columns span the sketched dimension (<= 64): estimate == ||A_i^T E_i||^2
    A, E = _draw(2, 150, 64, 48, dtype=dtype, layer=3)
    n2 = D.dprc_norm_hutch([(A, E, 0)], 64, 0, side=side, probe=D.PROBE_HADAMARD)
    exact = est.exact_layer(_np(A), _np(E))
    assert np.all(_rel(n2.cpu().numpy(), exact) < NORM_RTOL)


def test_hutch_token_splits_and_multilayer(D):
    # long token range -> several token splits per tile; two layers summed on top of a prior n2
    A1, E1 = _draw(2, 3000, 256, 200, layer=0)
    A2, E2 = _draw(2, 700, 136, 1100, layer=1)
    n2 = torch.tensor([1.5, 2.5], device="cuda")
    n2l = torch.zeros(2, 2, device="cuda")
    D.dprc_norm_hutch([(A1, E1, 10), (A2, E2, 11)], 16, 7, n2=n2, n2_layers=n2l, accumulate=True)
    r1 = est.hutch_layer(_np(A1), _np(E1), 16, 7, 10)
    r2 = est.hutch_layer(_np(A2), _np(E2), 16, 7, 11)
    got = n2l.cpu().numpy()
    assert np.all(_rel(got[0], r1) < NORM_RTOL) and np.all(_rel(got[1], r2) < NORM_RTOL)
    assert np.all(_rel(n2.cpu().numpy(), np.array([1.5, 2.5]) + r1 + r2) < NORM_RTOL)


def test_hutch_strided_rows(D):
    A, E = _draw(2, 100, 120, 90, layer=5, row_pad_a=8, row_pad_e=38)
    assert A.stride(1) == 128 and E.stride(1) == 128
    n2 = D.dprc_norm_hutch([(A, E, 2)], 8, 1)
    ref = est.hutch_layer(_np(A), _np(E), 8, 1, 2)
    assert np.all(_rel(n2.cpu().numpy(), ref) < NORM_RTOL)


def test_hutch_deterministic(D):
    A, E = _draw(2, 2048, 512, 384, layer=4)
    a = D.dprc_norm_hutch([(A, E, 3)], 16, 9)
    b = D.dprc_norm_hutch([(A, E, 3)], 16, 9)
    assert torch.equal(a, b)


# ---- Hutch++ ------------------------------------------------------------------------------

# The QR tree factors 128-row blocks and stacks their s x s R factors: the cases
# below take 2 and 3 levels, odd s (s = 5, padded to 8 register columns), s = 1
# and s = 32 (the largest), with ragged last blocks.
@pytest.mark.parametrize("B,T,d,p,s,r,side,dtype", [
    (2, 300, 200, 150, 8, 12, 0, "bf16"),
    (1, 520, 136, 300, 16, 32, 1, "bf16"),
    (2, 64, 64, 48, 4, 4, 0, "f32"),
    (1, 200, 600, 96, 32, 16, 1, "bf16"),      # m = 600: 5 blocks -> 160 rows -> 2 -> 1 (3 levels)
    (2, 150, 64, 1100, 5, 7, 0, "bf16"),       # m = 1100: 9 blocks -> 45 rows -> 1
    (2, 100, 50, 260, 1, 3, 0, "bf16"),        # s = 1
    (1, 180, 72, 130, 6, 40, 0, "bf16"),       # r = 40: the finalize's residual columns take two passes
])
def test_hutchpp_parity(D, B, T, d, p, s, r, side, dtype):
    A, E = _draw(B, T, d, p, dtype=dtype, law="student_t", layer=2)
    n2 = D.dprc_norm_hutchpp([(A, E, 6)], s, r, 3, side=side)
    ref = est.hutchpp_layer(_np(A), _np(E), s, r, 3, 6, side=side)
    assert np.all(_rel(n2.cpu().numpy(), ref) < NORM_RTOL)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_hutchpp_low_rank_is_exact(D, dtype):
    A, E = _draw(2, 12, 80, 96, dtype=dtype, layer=7)      # rank(A_i^T E_i) <= 12 <= s
    n2 = D.dprc_norm_hutchpp([(A, E, 0)], 16, 8, 11)
    exact = est.exact_layer(_np(A), _np(E))
    assert np.all(_rel(n2.cpu().numpy(), exact) < NORM_RTOL)


@pytest.mark.parametrize("side", [0, 1])
def test_hutchpp_low_rank_is_exact_deep_tree(D, side):
    # rank(A_i^T E_i) <= 12 <= s; the sketched width 1500 takes a 3-level QR tree
    A, E = _draw(2, 12, 1500 if side == 1 else 80, 80 if side == 1 else 1500, layer=9)
    n2 = D.dprc_norm_hutchpp([(A, E, 0)], 16, 8, 13, side=side)
    exact = est.exact_layer(_np(A), _np(E))
    assert np.all(_rel(n2.cpu().numpy(), exact) < NORM_RTOL)


@pytest.mark.parametrize("estimator", ["hutchpp", "gaussian"])
def test_dense_columns_many_rows(D, estimator):
    # B*T >= 16384 token rows: the passes with dense columns (Hutch++ W_S and Q, Gaussian
    # probes) take 64-row projection workgroups; T is ragged
    B, T, d, p = 2, 8200, 72, 200
    A, E = _draw(B, T, d, p, law="student_t", layer=12)
    if estimator == "hutchpp":
        n2 = D.dprc_norm_hutchpp([(A, E, 5)], 8, 12, 6)
        ref = est.hutchpp_layer(_np(A), _np(E), 8, 12, 6, 5)
    else:
        n2 = D.dprc_norm_hutch([(A, E, 5)], 16, 6, probe=D.PROBE_GAUSSIAN)
        ref = est.hutch_layer(_np(A), _np(E), 16, 6, 5, probe="gaussian")
    assert np.all(_rel(n2.cpu().numpy(), ref) < NORM_RTOL)


def test_hutchpp_many_layers_grouped(D):
    # 10 layers: two groups of the batched QR, sketched widths that take 1, 2 and 3 tree levels
    B, T = 2, 160
    shapes = [(64, 100), (96, 300), (48, 1500), (80, 130), (72, 640), (64, 90), (56, 2100), (40, 200),
              (88, 120), (64, 700)]
    pairs = []
    for li, (d, p) in enumerate(shapes):
        A, E = _draw(B, T, d, p, law="student_t", layer=20 + li)
        pairs.append((A, E, li))
    n2l = torch.zeros(len(pairs), B, device="cuda")
    n2 = D.dprc_norm_hutchpp(pairs, 8, 12, 4, n2_layers=n2l)
    ref_l = [est.hutchpp_layer(_np(A), _np(E), 8, 12, 4, li) for (A, E, li) in pairs]
    got_l = n2l.cpu().numpy()
    for li in range(len(pairs)):
        assert np.all(_rel(got_l[li], ref_l[li]) < NORM_RTOL), li
    assert np.all(_rel(n2.cpu().numpy(), sum(ref_l)) < NORM_RTOL)


def test_hutchpp_grouped_wide_passes(D):
    # three bf16 layers with s + r = 80 > 64 columns: the grouped passes take one launch pair
    # per layer (wider than the batched kernels), all sharing the group's pass scratch
    B, T, s, r = 2, 300, 16, 64
    shapes = [(120, 260), (72, 500), (200, 136)]
    pairs = []
    for li, (d, p) in enumerate(shapes):
        A, E = _draw(B, T, d, p, law="student_t", layer=40 + li)
        pairs.append((A, E, li))
    n2l = torch.zeros(len(pairs), B, device="cuda")
    n2 = D.dprc_norm_hutchpp(pairs, s, r, 8, n2_layers=n2l)
    ref_l = [est.hutchpp_layer(_np(A), _np(E), s, r, 8, li) for (A, E, li) in pairs]
    got_l = n2l.cpu().numpy()
    for li in range(len(pairs)):
        assert np.all(_rel(got_l[li], ref_l[li]) < NORM_RTOL), li
    assert np.all(_rel(n2.cpu().numpy(), sum(ref_l)) < NORM_RTOL)


def test_hutchpp_without_sketch_equals_hutch(D):
    A, E = _draw(2, 300, 100, 180, layer=8)
    a = D.dprc_norm_hutchpp([(A, E, 4)], 0, 16, 5)
    b = D.dprc_norm_hutch([(A, E, 4)], 16, 5)
    assert torch.equal(a, b)


# ---- clip factors, accumulation, noise --------------------------------------------------------

def test_clip_scale_edges(D):
    C = 2.0
    vals = [0.0, 4.0, 16.0, 1.0, math.inf, math.nan, -1.0, 1e30, 3.9999998]
    n2 = torch.tensor(vals, dtype=torch.float32, device="cuda")
    c = D.dprc_clip_scale(n2, C).cpu().numpy()
    ref = est.clip_scale(np.array(vals, dtype=np.float32).astype(np.float64), C)
    assert np.all(np.abs(c - ref) <= 1e-6 * np.maximum(ref, 1e-30))


@pytest.mark.parametrize("B,T,d,p,dtype", [
    (3, 150, 200, 260, "bf16"),     # ragged tiles; per-sample scaling inside a tile
    (2, 2000, 96, 72, "bf16"),      # few tiles -> split over samples and tokens
    (2, 64, 64, 48, "f32"),         # the tiny workload
    (2, 300, 500, 1000, "bf16"),    # 2 x 4 = 8 tiles: the XCD tile order (a multiple of 8 tiles), ragged
    (1, 260, 2000, 700, "bf16"),    # 8 x 3 = 24 tiles with d > p (the other walking order), ragged
])
def test_clip_accumulate_parity(D, B, T, d, p, dtype):
    A, E = _draw(B, T, d, p, dtype=dtype, layer=9)
    cvals = [0.25, 0.0, 0.8] if B == 3 else [0.37, 1.0][:B]
    c = torch.tensor(cvals, dtype=torch.float32, device="cuda")
    g = D.dprc_clip_accumulate(A, E, c)
    ref = est.clip_accumulate(_np(A), _np(E), np.array(cvals, dtype=np.float32).astype(np.float64))
    err = np.linalg.norm(g.cpu().numpy() - ref) / np.linalg.norm(ref)
    assert err < GRAD_RTOL
    # accumulate onto an existing gradient
    g0 = torch.full_like(g, 0.5)
    D.dprc_clip_accumulate(A, E, c, grad=g0, accumulate=True)
    err2 = np.linalg.norm(g0.cpu().numpy() - (ref + 0.5)) / np.linalg.norm(ref + 0.5)
    assert err2 < GRAD_RTOL


@pytest.mark.parametrize("aligned", [True, False])
def test_clip_accumulate_layers_parity(D, aligned):
    # several layers of one batch in one launch, no token splits: each layer's gradient against
    # the oracle and against a call of its own (which splits the small ones over tokens); 8 and
    # 15 tiles (the XCD ordering, ragged edges), T free per layer; with a 1001-wide layer the
    # launch takes element loads; then accumulation onto existing gradients
    B = 3
    shapes = [(150, 1024, 512), (100, 520, 1032), (64, 64, 48), (77, 256, 256), (150, 2048, 512)]
    if not aligned:
        shapes.append((90, 1001, 96))
    pairs = [(*_draw(B, T, d, p, layer=500 + j), j) for j, (T, d, p) in enumerate(shapes)]
    cvals = [0.25, 0.0, 0.8]
    c = torch.tensor(cvals, dtype=torch.float32, device="cuda")
    grads = D.dprc_clip_accumulate_layers(pairs, c)
    for (A, E, j), g in zip(pairs, grads):
        ref = est.clip_accumulate(_np(A), _np(E), np.array(cvals, dtype=np.float32).astype(np.float64))
        got = g.cpu().numpy()
        assert np.linalg.norm(got - ref) / np.linalg.norm(ref) < GRAD_RTOL, j
        solo = D.dprc_clip_accumulate(A, E, c).cpu().numpy()
        assert np.linalg.norm(got - solo) / np.linalg.norm(solo) < 1e-5, j
    g0 = [torch.full_like(g, 0.5) for g in grads]
    D.dprc_clip_accumulate_layers(pairs, c, grads=g0, accumulate=True)
    for g, gacc in zip(grads, g0):
        assert torch.allclose(gacc, g + 0.5, rtol=1e-6, atol=1e-6)


def test_clip_accumulate_layers_two_launches(D):
    # 70 layers (64 per launch), gradients with row strides wider than p
    B, pairs, grads = 2, [], []
    for j in range(70):
        d, p = 40 + 8 * (j % 4), 24 + 8 * (j % 5)
        A, E = _draw(B, 30 + j, d, p, layer=600 + j)
        pairs.append((A, E, j))
        grads.append(torch.zeros(d, p + 8, device="cuda")[:, :p])
    c = torch.tensor([0.6, 1.0], device="cuda")
    D.dprc_clip_accumulate_layers(pairs, c, grads=grads)
    for (A, E, j), g in zip(pairs, grads):
        solo = D.dprc_clip_accumulate(A, E, c).cpu().numpy()
        assert np.linalg.norm(g.cpu().numpy() - solo) / np.linalg.norm(solo) < 1e-5, j


def test_clip_accumulate_layers_edges(D):
    # a layer with a whole round of tiles (a launch of its own) between small ones, a
    # one-token layer, and all-zero factors (nothing added, accumulation leaves the
    # gradients as they were)
    B = 2
    shapes = [(64, 40, 24), (64, 4096, 4096), (1, 8, 8), (33, 300, 72)]
    pairs = [(*_draw(B, T, d, p, layer=700 + j), j) for j, (T, d, p) in enumerate(shapes)]
    c = torch.tensor([0.3, 0.9], device="cuda")
    grads = D.dprc_clip_accumulate_layers(pairs, c)
    for (A, E, j), g in zip(pairs, grads):
        solo = D.dprc_clip_accumulate(A, E, c)
        assert ((g - solo).norm() / solo.norm()).item() < 1e-5, j
        rows = [0, A.shape[2] // 2, A.shape[2] - 1]
        ref = est.clip_accumulate_rows(_np(A), _np(E), np.array([0.3, 0.9], dtype=np.float32).astype(np.float64), rows)
        got = g[rows].cpu().numpy().astype(np.float64)
        assert np.linalg.norm(got - ref) / np.linalg.norm(ref) < GRAD_RTOL, j
    zero = torch.zeros(B, device="cuda")
    fresh = D.dprc_clip_accumulate_layers(pairs, zero)
    assert all(torch.count_nonzero(g) == 0 for g in fresh)
    before = [g.clone() for g in grads]
    D.dprc_clip_accumulate_layers(pairs, zero, grads=grads, accumulate=True)
    assert all(torch.equal(g, b) for g, b in zip(grads, before))


def test_clip_accumulate_zero_factor_drops_nonfinite_sample(D):
    A, E = _draw(2, 100, 64, 64, layer=10)
    A[1, 3, 5] = float("nan")
    E[1, 7, 9] = float("inf")
    c = torch.tensor([0.5, 0.0], device="cuda")
    g = D.dprc_clip_accumulate(A, E, c).cpu().numpy()
    assert np.all(np.isfinite(g))
    ref = est.clip_accumulate(_np(A)[:1], _np(E)[:1], [0.5])
    assert np.linalg.norm(g - ref) / np.linalg.norm(ref) < GRAD_RTOL


def test_clip_accumulate_all_zero_factors(D):
    A, E = _draw(2, 70, 40, 30, layer=11)
    g = D.dprc_clip_accumulate(A, E, torch.zeros(2, device="cuda"))
    assert torch.count_nonzero(g) == 0


@pytest.mark.parametrize("numel,offset", [(1000, 0), (1023, 0), (7, 1)])
def test_add_noise_parity(D, numel, offset):
    sigma, C = 0.8, 1.0
    base = torch.randn(numel + offset, device="cuda", generator=torch.Generator("cuda").manual_seed(1))
    g = base[offset:].clone() if offset == 0 else base[offset:]
    g0 = g.clone().cpu().numpy().astype(np.float64)
    D.dprc_add_noise(g, sigma, C, 77, 5)
    ref = est.add_noise(g0, sigma, C, 77, 5)
    assert np.max(np.abs(g.cpu().numpy() - ref)) <= 1e-5 * sigma * C + 4e-7 * np.max(np.abs(ref))


def test_add_noise_moments(D):
    g = torch.zeros(1 << 22, device="cuda")
    D.dprc_add_noise(g, 1.0, 1.0, 3, 9)
    x = g.double()
    n = x.numel()
    assert abs(x.mean().item()) < 5 / math.sqrt(n)
    assert abs(x.var().item() - 1.0) < 5 * math.sqrt(2.0 / n)


# ---- private AdamW step (noise + 1/B + AdamW + transposed bf16 weights) ---------------------

@pytest.mark.parametrize("d,p,ld_pad,sigma,steps,wout", [
    (128, 256, 0, 0.7, 3, True),      # vector path, three steps
    (67, 130, 3, 0.5, 2, True),       # p not a multiple of 4, padded rows: element path, ragged tiles
    (64, 64, 4, 0.0, 1, False),       # no noise, no weight copy, padded rows
    (1, 5, 0, 1.0, 1, True),
])
def test_private_adamw_parity(D, d, p, ld_pad, sigma, steps, wout):
    r = np.random.default_rng(1000 * d + p)
    ld = p + ld_pad
    C, Bsz, lr, b1, b2, eps, wd, seed, tid = 1.5, 4, 1e-2, 0.9, 0.99, 1e-8, 0.05, 21, 5

    def dev(x):
        buf = torch.zeros(d, ld, dtype=torch.float32, device="cuda")
        buf[:, :p] = torch.tensor(x, dtype=torch.float32)
        return buf[:, :p]
    th0 = (r.standard_normal((d, p)) * 0.02).astype(np.float32)
    theta, m, v = dev(th0), dev(np.zeros((d, p))), dev(np.zeros((d, p)))
    w = torch.empty(p, d, dtype=torch.bfloat16, device="cuda") if wout else None
    th, mr, vr = th0.astype(np.float64), 0.0, 0.0
    firm = None
    for t in range(1, steps + 1):
        G = dev((r.standard_normal((d, p)) * 0.3).astype(np.float32))
        D.dprc_private_adamw(theta, m, v, G, sigma, C, seed, tid, 1.0 / Bsz, lr, b1, b2, eps, wd, t, w=w)
        G64 = est.as_f64(G.cpu())
        g = (est.add_noise(G64, sigma, C, seed, tid) if sigma > 0 else G64) / Bsz
        if firm is None:
            firm = np.abs(g) > 1e-4               # first update lr g/(|g|+eps) is steep near g = 0
        th, mr, vr = est.adamw(th, g, mr, vr, t, lr, b1, b2, eps, wd)
    torch.cuda.synchronize()
    got = theta.cpu().double().numpy()
    assert firm.mean() > 0.99
    assert np.max(np.abs(got - th)[firm]) <= 2e-6
    assert np.max(np.abs(got - th)) <= 2 * lr * steps
    assert np.allclose(m.cpu().double().numpy(), mr, rtol=1e-5, atol=1e-8)
    assert np.allclose(v.cpu().double().numpy(), vr, rtol=1e-5, atol=1e-10)
    if wout:
        assert torch.equal(w, theta.t().to(torch.bfloat16))
