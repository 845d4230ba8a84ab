"""Oracle for the single-GPU tile compute of Mesh-Attention (arXiv 2512.20968).

TEST INFRASTRUCTURE ONLY.  The test suite, the smoke check and the CPU-baseline
leg of the benchmark are the only callers allowed to import this package.  The
HIP library and its Python binding never import it, and it imports neither of
them: the two implementations share no code, no headers, no tables and no
helpers.  The seeded input generators live in their own package
(``mesh_inputs``) and hold none of the method's arithmetic.

Everything here is plain float64 NumPy, written for a reader who checks it
against the paper by eye, not for speed:

* ``attention``  -- the attention definition (Section 2.1), the partial
  ``(O, lse)`` of a Q partition over a KV partition set (Section 2.2), the
  online-softmax reducer used to merge partials (Section 2.2, Algorithm 2), the
  causal rule on global token positions under the contiguous and the striped
  sequence layouts (Section 3.7), GQA head sharing
  (Section 4.8), and the attention gradients the backward pass of Algorithm 3
  needs.
* ``worklist``   -- classification of the tile's (Q block, KV block) pairs into
  empty / partially masked / fully visible (causal rule of Section 3.7) and the
  canonical run list built from it.
* ``tiling``     -- the Q/KV partition index lists of a GPU's tile under basic
  2-D tiling (Section 3.2) and under KV Partition Rotation (Section 3.3).

Pins (the tests in ``tests/test_oracle_*.py``) tie every function to something
other than itself: closed forms, a library routine
(``torch.nn.functional.scaled_dot_product_attention`` in float64), brute force
on tiny inputs, finite differences, invariants of the merge, and the worked
examples the paper prints (``tests/golden``).
"""

from .attention import (  # noqa: F401
    CONTIGUOUS,
    STRIPED,
    token_positions,
    problem_positions,
    attention_rows,
    lse_merge,
    attention_rows_bwd,
    tile_forward,
    tile_backward,
    q_head_to_kv_head,
)
from .worklist import (  # noqa: F401
    EMPTY,
    PARTIAL,
    FULL,
    classify_blocks,
    classify_blocks_bruteforce,
    run_list,
    kv_major_run_list,
)
from .tiling import basic_tile, kvr_tile  # noqa: F401
