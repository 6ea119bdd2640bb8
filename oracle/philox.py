"""Philox4x32-10 and the probe / noise streams built on it (oracle side).

TEST INFRASTRUCTURE: see the package docstring.

The generator follows the published definition of Philox-4x32 with 10 rounds
(J. Salmon, M. Moraes, R. Dror, D. Shaw, "Parallel random numbers: as easy as
1, 2, 3", SC'11): a 4x32-bit counter and a 2x32-bit key; each round takes two
32x32->64-bit products of counter words 0 and 2 with the round multipliers,
xors their high halves with the other counter words and the key, and the key
is advanced by the Weyl constants between rounds.

Why a counter generator: Algorithm 2 draws a projection per layer (the proof
sketch of the privacy theorem states a fresh projection for every layer) and
the conclusion names {+1,-1} probes as the cheaper variant.  A counter
generator keyed by (seed, layer, stream) lets the CPU and the GPU produce the
identical probe matrix without storing it.

Stream layout (implementation-defined; the GPU side implements the same
definition independently):

* key   = (seed mod 2^32, seed div 2^32)
* probe word ``w`` (rows 32w .. 32w+31) of column ``j`` of a layer's probe
  matrix in stream ``s``: word ``w mod 4`` of Philox(counter = (w div 4, j,
  layer_id, s)).  Bit ``b`` of the word is row ``32w+b``; bit 0 means +1 and
  bit 1 means -1.
* streams: 0 = Hutchinson probes P (also the Hutch++ residual probes),
  1 = Hutch++ sketch S, 2 = Gaussian noise, 3 = Gaussian Hutchinson probes.
* Gaussian probe entry of row ``u`` and column ``j`` (the Gaussian probes of
  Algorithm 2, standard normal here and divided by k in the estimate): block
  q = u div 4, counter = (q, j, layer_id, 3); words (x0,x1) give rows 4q, 4q+1
  and (x2,x3) give 4q+2, 4q+3 by the same Box-Muller transform as the noise.
* noise element ``e`` of tensor ``t``: block q = e div 4, counter =
  (q mod 2^32, q div 2^32, t, 2); words (x0,x1) give elements 4q, 4q+1 and
  (x2,x3) give 4q+2, 4q+3 by the Box-Muller transform with
  u = (floor(x / 2^9) + 1/2) * 2^-23 (exact in binary32 and in binary64).
"""

import numpy as np

_M0 = np.uint64(0xD2511F53)
_M1 = np.uint64(0xCD9E8D57)
_W0 = np.uint64(0x9E3779B9)
_W1 = np.uint64(0xBB67AE85)
_MASK = np.uint64(0xFFFFFFFF)
_SH = np.uint64(32)

STREAM_PROBE = 0
STREAM_SKETCH = 1
STREAM_NOISE = 2
STREAM_GAUSS_PROBE = 3


def philox4x32_10(ctr, key):
    """Philox4x32-10 on arrays of counters.

    ctr: uint array [..., 4] (values < 2^32); key: uint array [..., 2] or a
    pair broadcastable to it.  Returns uint32 array [..., 4].
    """
    c = np.asarray(ctr, dtype=np.uint64) & _MASK
    k = np.asarray(key, dtype=np.uint64) & _MASK
    c0, c1, c2, c3 = c[..., 0], c[..., 1], c[..., 2], c[..., 3]
    k0 = np.broadcast_to(k[..., 0], c0.shape).copy()
    k1 = np.broadcast_to(k[..., 1], c0.shape).copy()
    for rnd in range(10):
        if rnd > 0:
            k0 = (k0 + _W0) & _MASK
            k1 = (k1 + _W1) & _MASK
        p0 = _M0 * c0          # < 2^64: exact in uint64
        p1 = _M1 * c2
        hi0, lo0 = p0 >> _SH, p0 & _MASK
        hi1, lo1 = p1 >> _SH, p1 & _MASK
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return np.stack([c0, c1, c2, c3], axis=-1).astype(np.uint32)


def _key(seed):
    seed = int(seed) & 0xFFFFFFFFFFFFFFFF
    return np.array([seed & 0xFFFFFFFF, seed >> 32], dtype=np.uint64)


def rademacher_words(seed, layer_id, stream_id, m, k):
    """Packed probe bits: uint32 [k, ceil(m/32)], bits of rows >= m cleared."""
    nw = (m + 31) // 32
    w = np.arange(nw, dtype=np.uint64)
    j = np.arange(k, dtype=np.uint64)
    ctr = np.zeros((k, nw, 4), dtype=np.uint64)
    ctr[..., 0] = (w // 4)[None, :]
    ctr[..., 1] = j[:, None]
    ctr[..., 2] = np.uint64(layer_id & 0xFFFFFFFF)
    ctr[..., 3] = np.uint64(stream_id & 0xFFFFFFFF)
    out = philox4x32_10(ctr, _key(seed))                  # [k, nw, 4]
    words = np.take_along_axis(out, (w % 4).astype(np.int64)[None, :, None], axis=2)[..., 0]
    tail = m - 32 * (nw - 1)
    if nw and tail < 32:
        words[:, -1] &= np.uint32((1 << tail) - 1)
    return words.astype(np.uint32)


def rademacher_matrix(seed, layer_id, stream_id, m, k):
    """The probe matrix Z in {+1,-1}^{m x k} as float64."""
    words = rademacher_words(seed, layer_id, stream_id, m, k)   # [k, nw]
    u = np.arange(m)
    bits = (words[:, u // 32] >> (u % 32).astype(np.uint32)) & np.uint32(1)   # [k, m]
    return (1.0 - 2.0 * bits.astype(np.float64)).T


def hadamard_matrix(m, k):
    """Columns 0..k-1 of the Sylvester-Hadamard sign pattern restricted to rows 0..m-1.

    z(u, j) = (-1)^popcount(u & j).  For m = k = 2^q this is the Sylvester
    matrix H with H H^T = m I.
    """
    u = np.arange(m, dtype=np.uint64)[:, None]
    j = np.arange(k, dtype=np.uint64)[None, :]
    x = u & j
    par = np.zeros(x.shape, dtype=np.uint64)
    while np.any(x):
        par ^= x & np.uint64(1)
        x = x >> np.uint64(1)
    return 1.0 - 2.0 * par.astype(np.float64)


def _uniform_open(x):
    """u = (floor(x/2^9) + 1/2) * 2^-23 in (0, 1), exactly representable."""
    return ((x.astype(np.uint64) >> np.uint64(9)).astype(np.float64) + 0.5) * 2.0 ** -23


def gaussian(seed, tensor_id, start, count):
    """Standard normals for elements start .. start+count-1 of a tensor (fp64)."""
    if count <= 0:
        return np.zeros(0, dtype=np.float64)
    q0 = start // 4
    q1 = (start + count - 1) // 4
    q = np.arange(q0, q1 + 1, dtype=np.uint64)
    ctr = np.zeros((q.size, 4), dtype=np.uint64)
    ctr[:, 0] = q & _MASK
    ctr[:, 1] = q >> _SH
    ctr[:, 2] = np.uint64(tensor_id & 0xFFFFFFFF)
    ctr[:, 3] = np.uint64(STREAM_NOISE)
    x = philox4x32_10(ctr, _key(seed))                     # [nq, 4]
    out = np.empty((q.size, 4), dtype=np.float64)
    for pair in range(2):
        u1 = _uniform_open(x[:, 2 * pair])
        u2 = _uniform_open(x[:, 2 * pair + 1])
        r = np.sqrt(-2.0 * np.log(u1))
        out[:, 2 * pair] = r * np.cos(2.0 * np.pi * u2)
        out[:, 2 * pair + 1] = r * np.sin(2.0 * np.pi * u2)
    flat = out.reshape(-1)
    off = start - 4 * q0
    return flat[off:off + count]


def _box_muller_blocks(x):
    """Four standard normals per Philox block: (x0,x1) and (x2,x3) through Box-Muller."""
    out = np.empty(x.shape[:-1] + (4,), dtype=np.float64)
    for pair in range(2):
        u1 = _uniform_open(x[..., 2 * pair])
        u2 = _uniform_open(x[..., 2 * pair + 1])
        r = np.sqrt(-2.0 * np.log(u1))
        out[..., 2 * pair] = r * np.cos(2.0 * np.pi * u2)
        out[..., 2 * pair + 1] = r * np.sin(2.0 * np.pi * u2)
    return out


def gaussian_probe_matrix(seed, layer_id, m, k):
    """m x k standard-normal probes (fp64) of the Gaussian Hutchinson option."""
    if m <= 0 or k <= 0:
        return np.zeros((max(m, 0), max(k, 0)))
    nq = (m + 3) // 4
    q = np.arange(nq, dtype=np.uint64)
    j = np.arange(k, dtype=np.uint64)
    ctr = np.zeros((k, nq, 4), dtype=np.uint64)
    ctr[:, :, 0] = q[None, :]
    ctr[:, :, 1] = j[:, None]
    ctr[:, :, 2] = np.uint64(layer_id & 0xFFFFFFFF)
    ctr[:, :, 3] = np.uint64(STREAM_GAUSS_PROBE)
    x = philox4x32_10(ctr, _key(seed))                     # [k, nq, 4]
    z = _box_muller_blocks(x).reshape(k, 4 * nq)[:, :m]    # [k, m]
    return z.T.copy()
