"""The library's calls can be captured into a HIP graph: they allocate nothing,
never synchronise and clear their scratch with kernels.  A captured step
(norms, clip factors, clipped accumulation with split-K, noise) is replayed
several times, with eager library work and synchronisations in between, and
every replay must reproduce the eager result bit for bit."""

import pytest
import torch

import workloads

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def D():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2605_24879_amd import dprc
    dprc.lib()
    return dprc


@pytest.mark.parametrize("estimator", ["hutch", "hutchpp"])
def test_graph_replays_match_eager(D, estimator):
    B, T = 2, 1000
    shapes = [(256, 384), (520, 96)]         # the second layer takes the split-K accumulation path
    pairs = []
    for li, (d, p) in enumerate(shapes):
        A, E = workloads.draw(B, T, d, p, dtype="bf16", law="lognormal", seed=3, layer=li, device="cuda")
        pairs.append((A, E, li))
    if estimator == "hutch":
        need = D.dprc_norm_hutch_workspace(pairs, 16)
    else:
        need = D.dprc_norm_hutchpp_workspace(pairs, 8, 16)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    acc_need = max(D.dprc_clip_accumulate_workspace(A, E) for (A, E, _) in pairs)
    assert acc_need > 0
    ws_acc = torch.empty(acc_need, dtype=torch.uint8, device="cuda")
    n2 = torch.zeros(B, device="cuda")
    c = torch.zeros(B, device="cuda")
    grads = [torch.zeros(d, p, device="cuda") for (d, p) in shapes]

    def step():
        if estimator == "hutch":
            D.dprc_norm_hutch(pairs, 16, 5, n2=n2, ws=ws)
        else:
            D.dprc_norm_hutchpp(pairs, 8, 16, 5, n2=n2, ws=ws)
        D.dprc_clip_scale(n2, 1.0, c=c)
        for (A, E, li), g in zip(pairs, grads):
            D.dprc_clip_accumulate(A, E, c, grad=g, ws=ws_acc)
            D.dprc_add_noise(g, 0.8, 1.0, 9, li)

    step()
    torch.cuda.synchronize()
    ref_n2, ref_c = n2.clone(), c.clone()
    ref_g = [g.clone() for g in grads]

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for rep in range(4):
        # eager work on the same buffers between replays, then clear the outputs
        step()
        n2.fill_(-1.0)
        c.fill_(-1.0)
        for g in grads:
            g.fill_(123.0)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(n2, ref_n2), rep
        assert torch.equal(c, ref_c), rep
        for g, r in zip(grads, ref_g):
            assert torch.equal(g, r), rep


def test_capture_before_any_eager_call(D):
    # a grouped Hutch++ call (three bf16 layers, one QR launch per tree level for all of them)
    # captured before the same buffers ever ran eagerly: the call keeps no lazily created
    # state, so the replays must equal the eager result computed afterwards
    B, T = 1, 700
    shapes = [(256, 384), (96, 520), (200, 136)]
    pairs = []
    for li, (d, p) in enumerate(shapes):
        A, E = workloads.draw(B, T, d, p, dtype="bf16", law="student_t", seed=11, layer=li, device="cuda")
        pairs.append((A, E, li))
    ws = torch.empty(D.dprc_norm_hutchpp_workspace(pairs, 8, 24), dtype=torch.uint8, device="cuda")
    n2 = torch.zeros(B, device="cuda")
    n2l = torch.zeros(len(shapes), B, device="cuda")
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        D.dprc_norm_hutchpp(pairs, 8, 24, 21, n2=n2, n2_layers=n2l, ws=ws)
    outs = []
    for _ in range(3):
        n2.fill_(-1.0)
        n2l.fill_(-1.0)
        graph.replay()
        torch.cuda.synchronize()
        outs.append((n2.clone(), n2l.clone()))
    ref_n2 = torch.zeros(B, device="cuda")
    ref_l = torch.zeros(len(shapes), B, device="cuda")
    D.dprc_norm_hutchpp(pairs, 8, 24, 21, n2=ref_n2, n2_layers=ref_l, ws=ws)
    torch.cuda.synchronize()
    assert torch.all(ref_n2 > 0)
    for rep, (a, b) in enumerate(outs):
        assert torch.equal(a, ref_n2), rep
        assert torch.equal(b, ref_l), rep
