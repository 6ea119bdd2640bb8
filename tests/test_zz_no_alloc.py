"""dprc_norm_hutch_clip_static (the entry point for callers that cannot allocate)
against dprc_norm_hutch_clip with a caller workspace: bit-identical estimates,
per-layer estimates and clip factors, on two calls in a row, the second smaller
than the first (the static scratch keeps the first call's contents)."""

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


def _pairs(specs, B, T, seed):
    out = []
    for li, (d, p, share) in enumerate(specs):
        if share and out:
            A = out[-1][0]                                   # same activations as the previous layer
            _, E = workloads.draw(B, T, d, p, dtype="bf16", law="lognormal", seed=seed, layer=li, device="cuda")
        else:
            A, E = workloads.draw(B, T, d, p, dtype="bf16", law="lognormal", seed=seed, layer=li, device="cuda")
        out.append((A, E, li))
    return out


def _both(D, pairs, k, seed, C):
    B = pairs[0][0].shape[0]
    L = len(pairs)
    arr, nl, _, dev = D._layers(pairs)
    stream = D._stream(dev)
    outs = []
    for static in (True, False):
        n2 = torch.full((B,), -7.0, device="cuda")
        c = torch.full((B,), -7.0, device="cuda")
        n2l = torch.full((L, B), -7.0, device="cuda")
        if static:
            st = D.lib().dprc_norm_hutch_clip_static(arr, nl, k, D.PROBE_RADEMACHER, seed, D.SIDE_OUT, C,
                                                    n2.data_ptr(), c.data_ptr(), n2l.data_ptr(), 0, stream)
        else:
            need = D.lib().dprc_norm_hutch_workspace(arr, nl, k, D.PROBE_RADEMACHER, D.SIDE_OUT)
            ws = torch.empty(need, dtype=torch.uint8, device="cuda")
            st = D.lib().dprc_norm_hutch_clip(arr, nl, k, D.PROBE_RADEMACHER, seed, D.SIDE_OUT, C,
                                             n2.data_ptr(), c.data_ptr(), n2l.data_ptr(), 0, ws.data_ptr(),
                                             need, stream)
        assert st == D.SUCCESS, D.lib().dprc_status_string(st)
        torch.cuda.synchronize()
        outs.append((n2, c, n2l))
    return outs


def test_static_scratch_matches_workspace_call_twice(D):
    # first call: seven bf16 layers in three activation groups (q, k, v share A; gate, up share
    # A), ragged T; second call: one smaller layer, run on the scratch the first one left
    big = _pairs([(256, 384, False), (256, 96, True), (256, 96, True), (384, 256, False),
                  (256, 520, False), (256, 520, True), (520, 256, False)], B=3, T=700, seed=4)
    small = _pairs([(136, 200, False)], B=2, T=130, seed=5)
    for pairs, k, seed in ((big, 32, 17), (small, 16, 18)):
        (n2s, cs, ls), (n2w, cw, lw) = _both(D, pairs, k, seed, 1.0)
        assert torch.all(n2s > 0)
        assert torch.equal(n2s, n2w)
        assert torch.equal(cs, cw)
        assert torch.equal(ls, lw)
