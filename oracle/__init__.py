"""fp64 CPU oracle for the fused attention forward -- TEST INFRASTRUCTURE, not part of the product.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may import
this package. The GPU library never calls it, shares no code with it, and does not fall back to it.

Contents (all NumPy float64 or plain Python, no GPU):

* :mod:`oracle.naive` -- the plain definition of scaled dot-product attention (Eq. 1): materialise
  the score matrix, mask, softmax, multiply by V. This is what the GPU path is checked against.
* :mod:`oracle.tiled` -- a separately written online-softmax version following the per-tile
  algorithm (Alg. 1) and the tile-to-tile split/merge (Alg. 2, with the merge read as the standard
  log-sum-exp combination). Used to cross-check the naive oracle.
* :mod:`oracle.brute` -- scalar double loops over Python floats with ``math.exp``, for tiny inputs.
* :func:`bf16_bits_to_f64` -- exact decoding of bfloat16 bit patterns.

Every function is pinned by ``tests/test_oracle_*.py`` against facts that do not come from the
oracle itself: torch's float64 CPU attention routine, closed forms, invariances, the brute force.
"""

from .naive import attention_head, bf16_bits_to_f64, naive_attention, naive_attention_rows  # noqa: F401
from .tiled import flash_tile, spatial_flash_attention  # noqa: F401
from .brute import brute_attention  # noqa: F401
