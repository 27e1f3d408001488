"""Plain fp64 CPU oracle for the A-PACK hot path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this package: only the tests, the smoke check and the benchmark's CPU
baseline leg use it.  It shares no code with the HIP library or its Python
binding, and it never receives a value computed by them.

Two modules, one per half of the method:

* ``oracle.prune``    -- the in-LLM query-conditioned prune (Section 3.2,
  Eq. 5 and Eq. 6; the inner loop of Algorithm 1): attention mass of the
  query rows over the cached audio/visual keys, per-modality top-k, and the
  gather of the kept rows.
* ``oracle.dynamics`` -- the pre-LLM local audio-visual dynamics scorer
  (Section 3.1, Eq. 1-4; the first loop of Algorithm 1; the pre-LLM
  compression details of the supplement): frame pooling, windowed CKA, the
  gate, segmentation, budgets and anchor / non-anchor token selection.

Every floating-point step is binary64.  Inputs are the exact values of the
bf16 or fp32 bit patterns, widened to fp64 by :func:`widen`.
"""

import numpy as np

from . import prune, dynamics  # noqa: F401

AUDIO = 1
VISUAL = 2
OTHER = 0


def widen(x, dtype):
    """Exact fp64 values of a raw input array.

    ``dtype`` is ``"bf16"`` (``x`` holds uint16 bit patterns) or ``"f32"``
    (``x`` holds float32 values or their uint32 bit patterns).
    """
    x = np.asarray(x)
    if dtype == "bf16":
        if x.dtype != np.uint16:
            raise TypeError("bf16 input must be given as uint16 bit patterns")
        return (x.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    if dtype == "f32":
        if x.dtype == np.uint32:
            x = x.view(np.float32)
        if x.dtype != np.float32:
            raise TypeError("f32 input must be float32 values or uint32 bits")
        return x.astype(np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")
