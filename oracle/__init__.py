"""fp64 CPU oracle for the fused attention forward -- TEST INFRASTRUCTURE, not part of the product.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may import
this package. The GPU library never calls it, shares no code with it, and does not fall back to it.

Contents (all NumPy float64 or plain Python, no GPU):

* :mod:`oracle.naive` -- the plain definition of scaled dot-product attention (Eq. 1): materialise
  the score matrix, mask, softmax, multiply by V. This is what the GPU path is checked against.
* :mod:`oracle.tiled` -- a separately written streaming version built on the decomposition the
  paper's per-tile (Alg. 1) and tile-to-tile (Alg. 2) algorithms rest on: per query row, the
  attention over a key set and that set's log-sum-exp, folded over key chunks and key-range parts
  (the log-sum-exp merge). Used to cross-check the naive oracle.
* :mod:`oracle.brute` -- scalar double loops over Python floats with ``math.exp``, for tiny inputs.
* :mod:`oracle.layer_by_layer` -- the paper's unfused layer-by-layer mapping as three operators with
  bfloat16 intermediates (score matrix, probabilities), the oracle of the unfused GPU baseline, with
  a direct float64 -> bfloat16 rounding and the error bound of the three roundings.
* :func:`bf16_bits_to_f64` -- exact decoding of bfloat16 bit patterns.

Every function is pinned by ``tests/test_oracle_*.py`` against facts that do not come from the
oracle itself: torch's float64 CPU attention routine, closed forms, invariances, the brute force.
"""

from .naive import attention_head, bf16_bits_to_f64, naive_attention, naive_attention_rows  # noqa: F401
from .tiled import flash_tile, spatial_flash_attention  # noqa: F401
from .brute import brute_attention  # noqa: F401
from .layer_by_layer import (lbl_error_bound, lbl_pv_head, lbl_scores_head, lbl_softmax_head,  # noqa: F401
                             layer_by_layer_attention, round_bf16)
