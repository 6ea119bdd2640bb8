"""CPU oracle for DP-SGD with randomized clipping (DP-SGD-RC).

This package is TEST INFRASTRUCTURE. It is a plain, slow, fp64 implementation
of what the GPU hot path computes, written from the paper "Efficient DP-SGD for
LLMs with Randomized Clipping" (Ullah, Aketi, Gupta, Zhang, Razaviyayn):

* ``philox``     -- the counter-based generator (Philox4x32-10, Salmon et al.,
                    SC'11) and the probe / noise streams derived from it.
* ``estimators`` -- per-sample gradients of a bias-free linear layer, the exact
                    FGC and GC norms, the Hutchinson and Hutch++ estimators of
                    Algorithm 2, the clip factors, the clipped accumulation and
                    the Gaussian noise of Algorithm 1, and the FLOP model of the
                    appendix table on FLOPs.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import anything from here.  The library under
``paper_2605_24879_amd`` never imports it, and this package imports nothing
from the library: the two share no code.  The seeded input generators live in
``workloads/``, which holds none of the method's arithmetic.
"""

from . import philox, estimators  # noqa: F401
