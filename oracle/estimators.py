"""fp64 reference of the DP-SGD-RC hot path for bias-free linear layers.

TEST INFRASTRUCTURE: see the package docstring.

Notation (Section "Proposed Method"): a linear layer S = A W with activations
A in R^{B x T x d}, output gradients G = dL/dS in R^{B x T x p} (called E here)
and per-sample gradient G_i = A_i^T E_i in R^{d x p}.  Everything below works
sample by sample, in float64, materialising G_i explicitly.  That is the plain
definition the estimators approximate; it is slow on purpose.

Readings taken where the paper is silent or inconsistent (each is listed in the
design notes of the repository):

* probes are +-1 (the {+1,-1} variant named as future work in the conclusion),
  shared by all samples of a layer, and the estimate is divided by k so that it
  is unbiased (the Gaussian probes of Algorithm 2 have variance 1/k instead);
* the projected side is a choice: "out" sketches the p side (Algorithm 2 as
  printed), "in" sketches the d side (the text notes both are equivalent), and
  "auto" takes the larger of the two dimensions, ties going to "out";
* the Hutch++ basis Q spans the columns of O S with O = G_i^T G_i (p x p);
  Algorithm 2 prints Q as d x k, the estimator section gives p x k, and only
  the latter type-checks;
* Hutch++ takes the sketch width s and the residual probe count r separately;
  the head term is not normalised, the residual term is divided by r;
* clip factor c_i = min(1, C / sqrt(n_i)) with n_i the summed squared estimate
  (Algorithm 1); n_i = 0 gives 1; a non-finite or negative n_i gives 0, and a
  sample with c_i = 0 is left out of the clipped sum altogether;
* the noise sigma*C*N(0, I) is added to the summed clipped gradient, with no
  division by the batch size (that belongs to the optimizer step).
"""

import numpy as np

from . import philox

SIDE_OUT, SIDE_IN, SIDE_AUTO = 0, 1, 2


def as_f64(x):
    """Widen an input array (float32, float64, or a torch tensor of bf16/fp32) exactly."""
    if hasattr(x, "detach"):                      # torch tensor: bf16 -> fp32 is exact
        x = x.detach().to("cpu").float().numpy()
    return np.asarray(x, dtype=np.float64)


def resolve_side(d, p, side):
    """Which dimension is projected: returns SIDE_OUT (p) or SIDE_IN (d)."""
    if side == SIDE_AUTO:
        return SIDE_IN if d > p else SIDE_OUT
    if side not in (SIDE_OUT, SIDE_IN):
        raise ValueError("side must be 0 (out), 1 (in) or 2 (auto)")
    return side


def per_sample_grad(A_i, E_i):
    """G_i = A_i^T E_i (d x p): the gradient of sample i's loss w.r.t. W for S = A W."""
    return as_f64(A_i).T @ as_f64(E_i)


def norm_fgc(A_i, E_i):
    """Exact squared norm by materialising the per-sample gradient (FGC form)."""
    G = per_sample_grad(A_i, E_i)
    return float(np.sum(G * G))


def norm_gc(A_i, E_i):
    """Exact squared norm by the ghost-clipping Gram identity vec(A A^T)^T vec(E E^T)."""
    A_i, E_i = as_f64(A_i), as_f64(E_i)
    return float(np.sum((A_i @ A_i.T) * (E_i @ E_i.T)))


def _oriented(G, side):
    """The matrix whose columns are probed: G (d x p) for "out", G^T (p x d) for "in"."""
    return G if side == SIDE_OUT else G.T


def probe_matrix(kind, seed, layer_id, stream_id, m, k):
    """m x k probes: +-1 from stream `stream_id`, Sylvester-Hadamard signs, or
    standard normals (the Gaussian probes of Algorithm 2 scaled by sqrt(k); they
    have their own stream, 3, whatever `stream_id` says)."""
    if kind == "rademacher":
        return philox.rademacher_matrix(seed, layer_id, stream_id, m, k)
    if kind == "hadamard":
        return philox.hadamard_matrix(m, k)
    if kind == "gaussian":
        return philox.gaussian_probe_matrix(seed, layer_id, m, k)
    raise ValueError(kind)


def hutch_layer(A, E, k, seed, layer_id, side=SIDE_OUT, probe="rademacher", Z=None):
    """Hutchinson estimate per sample for one layer (Algorithm 2, Hutch branch).

    A: [B, T, d], E: [B, T, p].  For each sample, W = G_i Z with Z the m x k
    probe matrix (m = p for "out"), and the estimate is ||W||_F^2 / k, an
    unbiased estimate of ||G_i||_F^2 = tr(G_i^T G_i).
    Returns float64 [B].
    """
    A, E = as_f64(A), as_f64(E)
    B, _, d = A.shape
    p = E.shape[2]
    side = resolve_side(d, p, side)
    m = p if side == SIDE_OUT else d
    if Z is None:
        Z = probe_matrix(probe, seed, layer_id, philox.STREAM_PROBE, m, k)
    out = np.empty(B)
    for i in range(B):
        M = _oriented(per_sample_grad(A[i], E[i]), side)    # (other) x m
        W = M @ Z
        out[i] = np.sum(W * W) / k
    return out


def hutchpp_layer(A, E, s, r, seed, layer_id, side=SIDE_OUT, ZS=None, ZP=None):
    """Hutch++ estimate per sample for one layer (Algorithm 2, Hutch++ branch).

    With M = G_i (oriented so that its columns are probed, m columns):
      1. sketch: O S = M^T (M S) with S the m x s sketch probes (stream 1);
      2. Q = orthonormal basis of the columns of O S (Householder QR);
      3. U = M Q (head, exact part);
      4. V = M P - U (Q^T P) with P the m x r residual probes (stream 0);
      5. estimate = ||U||_F^2 + ||V||_F^2 / r.
    s = 0 reduces to Hutchinson with r probes.  Returns float64 [B].
    """
    A, E = as_f64(A), as_f64(E)
    B, _, d = A.shape
    p = E.shape[2]
    side = resolve_side(d, p, side)
    m = p if side == SIDE_OUT else d
    if ZS is None:
        ZS = philox.rademacher_matrix(seed, layer_id, philox.STREAM_SKETCH, m, s)
    if ZP is None:
        ZP = philox.rademacher_matrix(seed, layer_id, philox.STREAM_PROBE, m, r)
    out = np.empty(B)
    for i in range(B):
        M = _oriented(per_sample_grad(A[i], E[i]), side)
        if s > 0:
            OS = M.T @ (M @ ZS)                              # m x s
            Q, _ = np.linalg.qr(OS, mode="reduced")          # LAPACK Householder
            U = M @ Q
            V = M @ ZP - U @ (Q.T @ ZP)
            head = np.sum(U * U)
        else:
            V = M @ ZP
            head = 0.0
        out[i] = head + (np.sum(V * V) / r if r > 0 else 0.0)
    return out


def hutch_sample_projected(A_i, E_i, Z, side=SIDE_OUT):
    """One sample's Hutchinson estimate in the association order of Algorithm 2,
    Y = A_i^T (E_i Z), without forming G_i (O(T k (d+p)) work).  Used for
    sampled checks at full workload sizes; pinned to ``hutch_layer``."""
    A_i, E_i = as_f64(A_i), as_f64(E_i)
    X, Xo = (E_i, A_i) if side == SIDE_OUT else (A_i, E_i)
    W = Xo.T @ (X @ Z)
    return float(np.sum(W * W)) / Z.shape[1]


def hutchpp_sample_projected(A_i, E_i, ZS, ZP, side=SIDE_OUT):
    """One sample's Hutch++ estimate in the association order of Algorithm 2:
    Q = orth(G^T (A (A^T (G S)))) with the roles of A and E set by ``side``,
    U = A^T (G Q), V = A^T (G P) - U (Q^T P).  Pinned to ``hutchpp_layer``."""
    A_i, E_i = as_f64(A_i), as_f64(E_i)
    X, Xo = (E_i, A_i) if side == SIDE_OUT else (A_i, E_i)
    r = ZP.shape[1]
    if ZS.shape[1] == 0:
        V = Xo.T @ (X @ ZP)
        return float(np.sum(V * V)) / r
    OS = X.T @ (Xo @ (Xo.T @ (X @ ZS)))
    Q, _ = np.linalg.qr(OS, mode="reduced")
    U = Xo.T @ (X @ Q)
    V = Xo.T @ (X @ ZP) - U @ (Q.T @ ZP)
    return float(np.sum(U * U) + np.sum(V * V) / r)


def clip_accumulate_rows(A, E, c, rows):
    """Rows ``rows`` of the clipped gradient sum_i c_i A_i^T E_i (for sampled checks)."""
    out = np.zeros((len(rows), E.shape[2]))
    for i in range(A.shape[0]):
        if c[i] != 0.0:
            out += c[i] * (as_f64(A[i][:, rows]).T @ as_f64(E[i]))
    return out


def exact_layer(A, E):
    """Exact squared per-sample norms of one layer, [B]."""
    A, E = as_f64(A), as_f64(E)
    return np.array([norm_fgc(A[i], E[i]) for i in range(A.shape[0])])


def clip_scale(n2, C):
    """c_i = min(1, C / sqrt(n_i)) (Algorithm 1, scaled loss), with the edge rules above."""
    n2 = np.asarray(n2, dtype=np.float64)
    c = np.zeros_like(n2)
    for i, v in enumerate(n2):
        if not np.isfinite(v) or v < 0:
            c[i] = 0.0
        elif v <= C * C:
            c[i] = 1.0
        else:
            c[i] = C / np.sqrt(v)
    return c


def clip_accumulate(A, E, c):
    """Clipped gradient of one layer: sum_i c_i G_i (d x p), samples with c_i = 0 left out.

    This is what the second backward pass of Algorithm 1 produces for a
    bias-free linear layer: back-propagating sum_i c_i L_i with the c_i held
    constant gives sum_i c_i A_i^T E_i.
    """
    A, E = as_f64(A), as_f64(E)
    grad = np.zeros((A.shape[2], E.shape[2]))
    for i in range(A.shape[0]):
        if c[i] != 0.0:
            grad += c[i] * per_sample_grad(A[i], E[i])
    return grad


def add_noise(grad, sigma, C, seed, tensor_id, start=0):
    """grad + sigma * C * xi with xi ~ N(0, I) from the noise stream (Algorithm 1)."""
    g = np.asarray(grad, dtype=np.float64)
    xi = philox.gaussian(seed, tensor_id, start, g.size).reshape(g.shape)
    return g + sigma * C * xi


def private_gradient(A, E, c, sigma, C, seed, tensor_id, batch):
    """The private gradient of one layer as the optimizer sees it (Algorithm 1):
    (sum_i c_i G_i + sigma C xi) / batch, the division by the batch size being
    the optimizer's normalisation."""
    g = clip_accumulate(A, E, c)
    if sigma > 0:
        g = add_noise(g, sigma, C, seed, tensor_id)
    return g / batch


def adamw(theta, grad, m, v, t, lr, beta1, beta2, eps, weight_decay):
    """One AdamW update (Algorithm 1's optimizer step; AdamW = Adam with decoupled
    weight decay, Loshchilov and Hutter, which the paper's experiments use).

    theta <- theta (1 - lr wd); m <- beta1 m + (1 - beta1) g;
    v <- beta2 v + (1 - beta2) g^2; theta <- theta - lr m_hat / (sqrt(v_hat) + eps)
    with m_hat = m / (1 - beta1^t), v_hat = v / (1 - beta2^t), t the 1-based step.
    Returns (theta, m, v) in fp64.
    """
    theta, g = np.asarray(theta, dtype=np.float64), np.asarray(grad, dtype=np.float64)
    theta = theta * (1.0 - lr * weight_decay)
    m = beta1 * m + (1.0 - beta1) * g
    v = beta2 * v + (1.0 - beta2) * g * g
    m_hat = m / (1.0 - beta1 ** t)
    v_hat = v / (1.0 - beta2 ** t)
    return theta - lr * m_hat / (np.sqrt(v_hat) + eps), m, v


# ---- FLOP model of the appendix table (tab:flops_analysis) -----------------

def flops_fgc(B, T, d, p):
    """Exact FLOPs of the FGC norm: B p d (2T - 1)."""
    return B * p * d * (2 * T - 1)


def flops_gc(B, T, d, p):
    """Exact FLOPs of the GC norm: 2 B T^2 (p + d) - B."""
    return 2 * B * T * T * (p + d) - B


def flops_rc(B, T, d, p, k):
    """Exact FLOPs of the randomized (Hutchinson) norm: 2 B T k (p + d) + B k (d - T) - B."""
    return 2 * B * T * k * (p + d) + B * k * (d - T) - B
