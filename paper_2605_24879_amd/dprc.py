"""Python binding of libdprc (include/dprc.h): argument marshalling only.

Each function has the name of the C entry point it calls and takes torch
tensors on the GPU; every step of the computation runs in the HIP kernels of
libdprc.so.  Outputs and workspaces that the caller does not pass are
allocated with torch on the tensors' device, and calls are enqueued on torch's
current stream.  A missing library or a non-zero dprc_status raises
RuntimeError; there is no fallback.
"""

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdprc.so")

SUCCESS = 0
F32, BF16 = 0, 1
SIDE_OUT, SIDE_IN, SIDE_AUTO = 0, 1, 2
PROBE_RADEMACHER, PROBE_HADAMARD, PROBE_GAUSSIAN = 0, 1, 2
STREAM_PROBE, STREAM_SKETCH, STREAM_NOISE = 0, 1, 2

EXPORTS = ["dprc_norm_hutch_workspace", "dprc_norm_hutch", "dprc_norm_hutch_clip", "dprc_norm_hutch_clip_static", "dprc_norm_hutchpp_workspace",
           "dprc_norm_hutchpp", "dprc_clip_scale", "dprc_clip_accumulate_workspace",
           "dprc_clip_accumulate", "dprc_clip_accumulate_layers", "dprc_add_noise", "dprc_probe_bits", "dprc_probe_gaussian", "dprc_private_adamw", "dprc_envelope_middle_workspace",
           "dprc_envelope_middle", "dprc_chi2_cdf", "dprc_envelope_bins", "dprc_pld_step_workspace",
           "dprc_pld_step", "dprc_pld_fold", "dprc_pld_delta", "dprc_status_string",
           "dprc_version", "dprc_trace_launches"]


class Layer(ctypes.Structure):
    """Mirror of dprc_layer."""
    _fields_ = [("A", ctypes.c_void_p), ("E", ctypes.c_void_p),
                ("B", ctypes.c_int64), ("T", ctypes.c_int64), ("d", ctypes.c_int64), ("p", ctypes.c_int64),
                ("lda", ctypes.c_int64), ("lde", ctypes.c_int64),
                ("dtype", ctypes.c_int), ("layer_id", ctypes.c_uint32)]


class AdamWParams(ctypes.Structure):
    """Mirror of dprc_adamw_params."""
    _fields_ = [("lr", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
                ("eps", ctypes.c_float), ("weight_decay", ctypes.c_float), ("step", ctypes.c_int32)]


_lib = None


def lib():
    """Load libdprc.so (built in-tree by paper_2605_24879_amd.build)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2605_24879_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P, I32, I64, U32, U64, F, SZ = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32,
                                         ctypes.c_uint64, ctypes.c_float, ctypes.c_size_t)
        LP = ctypes.POINTER(Layer)
        sig = {
            "dprc_norm_hutch_workspace": (SZ, [LP, I32, I32, ctypes.c_int, ctypes.c_int]),
            "dprc_norm_hutch": (ctypes.c_int, [LP, I32, I32, ctypes.c_int, U64, ctypes.c_int, P, P, I32, P, SZ, P]),
            "dprc_norm_hutch_clip": (ctypes.c_int, [LP, I32, I32, ctypes.c_int, U64, ctypes.c_int, F, P, P, P, I32, P, SZ,
                                                    P]),
            "dprc_norm_hutch_clip_static": (ctypes.c_int, [LP, I32, I32, ctypes.c_int, U64, ctypes.c_int, F, P, P, P,
                                                           I32, P]),
            "dprc_norm_hutchpp_workspace": (SZ, [LP, I32, I32, I32, ctypes.c_int]),
            "dprc_norm_hutchpp": (ctypes.c_int, [LP, I32, I32, I32, U64, ctypes.c_int, P, P, I32, P, SZ, P]),
            "dprc_clip_scale": (ctypes.c_int, [P, I64, F, P, P]),
            "dprc_clip_accumulate_workspace": (SZ, [LP]),
            "dprc_clip_accumulate": (ctypes.c_int, [LP, P, P, I64, I32, P, SZ, P]),
            "dprc_clip_accumulate_layers": (ctypes.c_int, [LP, I32, P, P, P, I32, P]),
            "dprc_add_noise": (ctypes.c_int, [P, I64, F, F, U64, U32, P]),
            "dprc_probe_bits": (ctypes.c_int, [ctypes.c_int, U64, U32, U32, I64, I32, P, P]),
            "dprc_probe_gaussian": (ctypes.c_int, [U64, U32, I64, I32, P, P]),
            "dprc_envelope_middle_workspace": (SZ, [I32, I32, I32]),
            "dprc_envelope_middle": (ctypes.c_int, [P, I32, I32, I32, I32, P, P, P, SZ, P]),
            "dprc_chi2_cdf": (ctypes.c_int, [P, I64, ctypes.c_double, ctypes.c_double, P, P]),
            "dprc_envelope_bins": (ctypes.c_int, [P, I32, ctypes.c_double, ctypes.c_double, P, P, P]),
            "dprc_pld_step_workspace": (SZ, [I64]),
            "dprc_pld_step": (ctypes.c_int, [ctypes.c_double, ctypes.c_double, ctypes.c_double, I64, P, P, I32, P, P,
                                             P, SZ, P]),
            "dprc_pld_fold": (ctypes.c_int, [P, I64, P, P, P, P, P]),
            "dprc_pld_delta": (ctypes.c_int, [P, I64, ctypes.c_double, P, P, I32, P, P]),
            "dprc_private_adamw": (ctypes.c_int, [P, P, P, I64, P, I64, I64, I64, F, F, U64, U32, F,
                                                  ctypes.POINTER(AdamWParams), P, I64, P]),
            "dprc_status_string": (ctypes.c_char_p, [ctypes.c_int]),
            "dprc_version": (ctypes.c_char_p, []),
            "dprc_trace_launches": (ctypes.c_int, [P, P, I32, P]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _check(status):
    if status != SUCCESS:
        raise RuntimeError(lib().dprc_status_string(status).decode())


def _stream(dev):
    return ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)


def _dtype_code(t):
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise TypeError(f"unsupported dtype {t.dtype}; use bfloat16 or float32")


def make_layer(A, E, layer_id):
    """dprc_layer for activations A [B,T,d] and output gradients E [B,T,p] (token rows)."""
    if A.dim() != 3 or E.dim() != 3:
        raise ValueError("A and E must be [B, T, features]")
    if not (A.is_cuda and E.is_cuda):
        raise ValueError("A and E must be GPU tensors")
    if A.dtype != E.dtype:
        raise TypeError("A and E must share a dtype")
    B, T, d = A.shape
    if E.shape[0] != B or E.shape[1] != T:
        raise ValueError("A and E must agree on B and T")
    p = E.shape[2]
    for X in (A, E):
        if X.stride(2) != 1 or X.stride(0) != T * X.stride(1):
            raise ValueError("tensors must have contiguous features, token rows of stride ld, samples of stride T*ld")
    return Layer(A.data_ptr(), E.data_ptr(), B, T, d, p, A.stride(1), E.stride(1), _dtype_code(A), layer_id)


def _layers(pairs):
    """pairs: list of (A, E, layer_id); returns (ctypes array, count, B, device)."""
    arr = (Layer * len(pairs))(*[make_layer(A, E, lid) for (A, E, lid) in pairs])
    return arr, len(pairs), pairs[0][0].shape[0], pairs[0][0].device


def _workspace(nbytes, dev, ws):
    if ws is not None:
        if ws.numel() * ws.element_size() < nbytes:
            raise ValueError("workspace too small")
        return ws
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=dev)


def dprc_norm_hutch_workspace(pairs, k, side=SIDE_OUT, probe=PROBE_RADEMACHER):
    arr, nl, _, _ = _layers(pairs)
    return lib().dprc_norm_hutch_workspace(arr, nl, k, probe, side)


def dprc_norm_hutch(pairs, k, seed, side=SIDE_OUT, probe=PROBE_RADEMACHER, n2=None, n2_layers=None,
                    accumulate=False, ws=None):
    """Hutchinson estimates summed over layers: returns n2 [B] (fp32).  pairs = [(A, E, layer_id), ...]."""
    arr, nl, B, dev = _layers(pairs)
    if n2 is None:
        n2 = torch.zeros(B, dtype=torch.float32, device=dev)
    need = lib().dprc_norm_hutch_workspace(arr, nl, k, probe, side)
    ws = _workspace(need, dev, ws)
    _check(lib().dprc_norm_hutch(arr, nl, k, probe, seed, side, n2.data_ptr(),
                                 n2_layers.data_ptr() if n2_layers is not None else None,
                                 int(bool(accumulate)), ws.data_ptr(), need, _stream(dev)))
    return n2


def dprc_norm_hutch_clip(pairs, k, seed, C, side=SIDE_OUT, probe=PROBE_RADEMACHER, n2=None, c=None,
                         n2_layers=None, accumulate=False, ws=None):
    """Hutchinson estimates and their clip factors in one call: returns (n2 [B], c [B])."""
    arr, nl, B, dev = _layers(pairs)
    if n2 is None:
        n2 = torch.zeros(B, dtype=torch.float32, device=dev)
    if c is None:
        c = torch.empty(B, dtype=torch.float32, device=dev)
    need = lib().dprc_norm_hutch_workspace(arr, nl, k, probe, side)
    ws = _workspace(need, dev, ws)
    _check(lib().dprc_norm_hutch_clip(arr, nl, k, probe, seed, side, C, n2.data_ptr(), c.data_ptr(),
                                      n2_layers.data_ptr() if n2_layers is not None else None,
                                      int(bool(accumulate)), ws.data_ptr(), need, _stream(dev)))
    return n2, c


def dprc_norm_hutchpp_workspace(pairs, s, r, side=SIDE_OUT):
    arr, nl, _, _ = _layers(pairs)
    return lib().dprc_norm_hutchpp_workspace(arr, nl, s, r, side)


def dprc_norm_hutch_clip_static(pairs, k, seed, C, side=SIDE_OUT, probe=PROBE_RADEMACHER, n2=None, c=None,
                                n2_layers=None, accumulate=False):
    """dprc_norm_hutch_clip on the library's static scratch (no workspace): returns (n2, c).
    Outputs the caller does not pass are allocated here, by torch; pass them to allocate
    nothing."""
    arr, nl, B, dev = _layers(pairs)
    if n2 is None:
        n2 = torch.zeros(B, dtype=torch.float32, device=dev)
    if c is None:
        c = torch.empty(B, dtype=torch.float32, device=dev)
    _check(lib().dprc_norm_hutch_clip_static(arr, nl, k, probe, seed, side, C, n2.data_ptr(), c.data_ptr(),
                                             n2_layers.data_ptr() if n2_layers is not None else None,
                                             int(bool(accumulate)), _stream(dev)))
    return n2, c


def dprc_norm_hutchpp(pairs, s, r, seed, side=SIDE_OUT, n2=None, n2_layers=None, accumulate=False, ws=None):
    """Hutch++ estimates summed over layers: returns n2 [B] (fp32)."""
    arr, nl, B, dev = _layers(pairs)
    if n2 is None:
        n2 = torch.zeros(B, dtype=torch.float32, device=dev)
    need = lib().dprc_norm_hutchpp_workspace(arr, nl, s, r, side)
    ws = _workspace(need, dev, ws)
    _check(lib().dprc_norm_hutchpp(arr, nl, s, r, seed, side, n2.data_ptr(),
                                   n2_layers.data_ptr() if n2_layers is not None else None,
                                   int(bool(accumulate)), ws.data_ptr(), need, _stream(dev)))
    return n2


def dprc_clip_scale(n2, C, c=None):
    if c is None:
        c = torch.empty_like(n2)
    _check(lib().dprc_clip_scale(n2.data_ptr(), n2.numel(), float(C), c.data_ptr(), _stream(n2.device)))
    return c


def dprc_clip_accumulate_workspace(A, E):
    return lib().dprc_clip_accumulate_workspace(ctypes.byref(make_layer(A, E, 0)))


def dprc_clip_accumulate(A, E, c, grad=None, accumulate=False, ws=None):
    """grad [d, p] (fp32) (=|+=) sum_i c_i A_i^T E_i."""
    L = make_layer(A, E, 0)
    if grad is None:
        grad = torch.empty(A.shape[2], E.shape[2], dtype=torch.float32, device=A.device)
    if grad.stride(1) != 1:
        raise ValueError("grad must have contiguous rows")
    need = lib().dprc_clip_accumulate_workspace(ctypes.byref(L))
    ws = _workspace(need, A.device, ws) if need else None
    _check(lib().dprc_clip_accumulate(ctypes.byref(L), c.data_ptr(), grad.data_ptr(), grad.stride(0),
                                      int(bool(accumulate)), ws.data_ptr() if ws is not None else None,
                                      need, _stream(A.device)))
    return grad


def dprc_clip_accumulate_layers(pairs, c, grads=None, accumulate=False):
    """grads[l] [d_l, p_l] (fp32) (=|+=) sum_i c_i A_i^T E_i for every (A, E) of pairs (bf16), in
    one launch per 64 layers.  Returns the list of gradients."""
    pairs = [(A, E) for (A, E, *_) in pairs]
    n = len(pairs)
    if grads is None:
        grads = [torch.empty(A.shape[2], E.shape[2], dtype=torch.float32, device=A.device) for (A, E) in pairs]
    if len(grads) != n:
        raise ValueError("one gradient per layer")
    for g in grads:
        if g.stride(1) != 1:
            raise ValueError("grad must have contiguous rows")
    arr = (Layer * n)(*[make_layer(A, E, 0) for (A, E) in pairs])
    ptrs = (ctypes.c_void_p * n)(*[g.data_ptr() for g in grads])
    lds = (ctypes.c_int64 * n)(*[g.stride(0) for g in grads])
    dev = pairs[0][0].device if n else c.device
    _check(lib().dprc_clip_accumulate_layers(arr, n, c.data_ptr(), ptrs, lds, int(bool(accumulate)), _stream(dev)))
    return grads


def dprc_add_noise(grad, sigma, C, seed, tensor_id):
    """grad += sigma * C * N(0, I) in place (grad contiguous fp32)."""
    if not grad.is_contiguous() or grad.dtype != torch.float32:
        raise ValueError("grad must be contiguous fp32")
    _check(lib().dprc_add_noise(grad.data_ptr(), grad.numel(), float(sigma), float(C), seed, tensor_id,
                                _stream(grad.device)))
    return grad


def dprc_private_adamw(theta, m, v, G, sigma, C, seed, tensor_id, inv_batch, lr, beta1, beta2, eps,
                       weight_decay, step, w=None):
    """One private AdamW step: theta, m, v ([d, p] fp32, updated in place) from the clipped
    gradient G [d, p]; w (optional, [p, d] bf16) receives bf16(theta) transposed."""
    d, p = G.shape
    for X in (theta, m, v):
        if X.shape != (d, p) or X.dtype != torch.float32 or X.stride(1) != 1 or X.stride(0) != theta.stride(0):
            raise ValueError("theta, m, v must be fp32 [d, p] with one row stride")
    if G.dtype != torch.float32 or G.stride(1) != 1:
        raise ValueError("G must be fp32 [d, p] with contiguous rows")
    if w is not None and (w.shape != (p, d) or w.dtype != torch.bfloat16 or w.stride(1) != 1):
        raise ValueError("w must be bf16 [p, d] with contiguous rows")
    hp = AdamWParams(lr, beta1, beta2, eps, weight_decay, int(step))
    _check(lib().dprc_private_adamw(theta.data_ptr(), m.data_ptr(), v.data_ptr(), theta.stride(0), G.data_ptr(),
                                    G.stride(0), d, p, sigma, C, seed, tensor_id, inv_batch, ctypes.byref(hp),
                                    w.data_ptr() if w is not None else None, w.stride(0) if w is not None else 0,
                                    _stream(G.device)))
    return theta


def dprc_envelope_middle(x, k, d, n_lambda):
    """MiddleRegionCDF at the points x (fp64 device tensor): (best [nx], arg [nx, 3] = i, j, l)."""
    x = x.contiguous()
    nx = x.numel()
    best = torch.empty(nx, dtype=torch.float64, device=x.device)
    arg = torch.empty(nx, 3, dtype=torch.int32, device=x.device)
    need = lib().dprc_envelope_middle_workspace(nx, d, n_lambda)
    ws = _workspace(need, x.device, None)
    _check(lib().dprc_envelope_middle(x.data_ptr(), nx, k, d, n_lambda, best.data_ptr(), arg.data_ptr(),
                                      ws.data_ptr(), need, _stream(x.device)))
    return best, arg


def dprc_chi2_cdf(x, dof, scale=1.0):
    """P(chi^2(dof) <= x * scale) elementwise (fp64 device tensor)."""
    x = x.contiguous()
    out = torch.empty_like(x)
    _check(lib().dprc_chi2_cdf(x.data_ptr(), x.numel(), float(dof), float(scale), out.data_ptr(),
                               _stream(x.device)))
    return out


def dprc_probe_bits(probe, seed, layer_id, stream_id, m, k, device="cuda", out=None):
    """Packed probe words [k, ceil(m/32)] (int32 view of the uint32 words)."""
    nw = (m + 31) // 32
    if out is None:
        out = torch.empty(k, nw, dtype=torch.int32, device=device)
    _check(lib().dprc_probe_bits(probe, seed, layer_id, stream_id, m, k, out.data_ptr(), _stream(out.device)))
    return out


def _f64_dev(x, name):
    if not (x.is_cuda and x.dtype == torch.float64 and x.is_contiguous()):
        raise ValueError(f"{name} must be a contiguous fp64 GPU tensor")
    return x


def dprc_envelope_bins(F, y_min, y_max):
    """Envelope-law bins from the CDF at n_bins + 1 even grid points: returns (ybar, w) [n_bins]."""
    _f64_dev(F, "F")
    n = F.numel() - 1
    ybar = torch.empty(n, dtype=torch.float64, device=F.device)
    w = torch.empty(n, dtype=torch.float64, device=F.device)
    _check(lib().dprc_envelope_bins(F.data_ptr(), n, float(y_min), float(y_max), ybar.data_ptr(), w.data_ptr(),
                                    _stream(F.device)))
    return ybar, w


def dprc_pld_step(sigma, p, h, n_half, ybar=None, w=None, device=None):
    """One subsampled step's PLD: returns (q [2 n_half - 1], q_inf [1]) as fp64 GPU tensors."""
    dev = ybar.device if ybar is not None else torch.device(device if device is not None else "cuda")
    if ybar is not None:
        _f64_dev(ybar, "ybar")
        _f64_dev(w, "w")
    q = torch.empty(2 * n_half - 1, dtype=torch.float64, device=dev)
    q_inf = torch.empty(1, dtype=torch.float64, device=dev)
    need = lib().dprc_pld_step_workspace(n_half)
    ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    _check(lib().dprc_pld_step(float(sigma), float(p), float(h), n_half,
                               ybar.data_ptr() if ybar is not None else None,
                               w.data_ptr() if w is not None else None, ybar.numel() if ybar is not None else 0,
                               q.data_ptr(), q_inf.data_ptr(), ws.data_ptr(), need, _stream(dev)))
    return q, q_inf


def dprc_pld_fold(r, L, ainf, binf):
    """Kept cells and atom of the composition whose linear convolution is r[:2L-1]."""
    for x, nm in ((r, "r"), (ainf, "ainf"), (binf, "binf")):
        _f64_dev(x, nm)
    if r.numel() < 2 * L - 1:
        raise ValueError("r must hold the 2L - 1 values of the linear convolution")
    q = torch.empty(L, dtype=torch.float64, device=r.device)
    q_inf = torch.empty(1, dtype=torch.float64, device=r.device)
    _check(lib().dprc_pld_fold(r.data_ptr(), L, ainf.data_ptr(), binf.data_ptr(), q.data_ptr(), q_inf.data_ptr(),
                               _stream(r.device)))
    return q, q_inf


def dprc_pld_delta(q, h, q_inf, eps):
    """delta(eps) for a batch of eps values (fp64 GPU tensor): returns delta [len(eps)]."""
    for x, nm in ((q, "q"), (q_inf, "q_inf"), (eps, "eps")):
        _f64_dev(x, nm)
    out = torch.empty(eps.numel(), dtype=torch.float64, device=q.device)
    _check(lib().dprc_pld_delta(q.data_ptr(), q.numel(), float(h), q_inf.data_ptr(), eps.data_ptr(), eps.numel(),
                                out.data_ptr(), _stream(q.device)))
    return out


def dprc_probe_gaussian(seed, layer_id, m, k, device="cuda", out=None):
    """Gaussian probe values [k, m] (fp32): out[j, u] = probe entry (u, j)."""
    if out is None:
        out = torch.empty(k, m, dtype=torch.float32, device=device)
    _check(lib().dprc_probe_gaussian(seed, layer_id, m, k, out.data_ptr(), _stream(out.device)))
    return out


def dprc_version():
    return lib().dprc_version().decode()


KERNEL_NAMES = {1: "project", 2: "token_reduce", 3: "qr", 4: "hutchpp_final", 5: "clip_scale",
                6: "accumulate", 7: "splitk_reduce", 8: "noise", 9: "probe_bits", 10: "project_f32",
                11: "token_reduce_f32", 12: "sample_sq", 13: "accumulate_f32",
                14: "token_splits", 15: "sample_sum", 16: "qr_combine", 17: "qr_expand", 18: "hutchpp_sum",
                19: "probe_gauss", 20: "adamw", 21: "envelope", 22: "chi2_cdf", 23: "pld"}


def dprc_trace_launches(events_ptr, kinds_ptr, capacity, count_ptr):
    """Switch the per-launch event hook on (events_ptr = hipEvent_t array) or off (None)."""
    _check(lib().dprc_trace_launches(events_ptr, kinds_ptr, capacity, count_ptr))
