"""CPU oracle for the Fathom hot path -- TEST INFRASTRUCTURE ONLY.

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product library never does, and
this package never imports the product.  See ``oracle/fathom_oracle.c`` for
the arithmetic and the paper passages each function follows.

Parity status per function (what pins it to the paper, in ``tests/``):
  f32_to_f16_*    numpy binary16 conversion on every half, midpoint and neighbour
  pack            App. A codes, Sec. 3.2 prefix-quantiser invariant, MSB = sign,
                  fp16-subnormal and near-65504 block scales
  alloc_waterfill App. A g, theta, depths at B = 8 and 6; brute force; Eq. (wf)
  bisect          App. A bisection trace, row by row
  alloc_topr      App. A SparQ tie rule and sum |q|
  scores_f64      App. A approximate and exact scores; Sec. 3.2 full 4-bit case;
                  Sec. 3.3 error-variance law (Monte Carlo)
  scores_f32      within its fp32 error bound of scores_f64 (order is a reading)
  topk            brute-force sort on tiny inputs; App. A top-2 sets
  sparse_attn     k = n equals dense softmax attention; one-row set = V row
  klt_calibrate   Hadamard-design keys with known mean and covariance give the
                  known eigenvalues and eigenvectors (``klt.py``, Sec. 3.5)
  klt_rotate_*    identity / permutation bases exact; fp32 error bound; q'.k'
                  equals q.(k - mu)
"""
from .oracle import *  # noqa: F401,F403
from .oracle import build, lib_path  # noqa: F401
from .klt import *  # noqa: F401,F403
