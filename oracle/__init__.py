"""Oracle: a plain, slow, float64 CPU statement of what the hot path computes.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the bench's
CPU-baseline leg may import or call anything in this package; the product
(the HIP library and its Python binding) never does, and this package never
imports the product.  The two share no code: inputs come from ``fixtures``.

Contents (each function cites the passage of the paper it follows):

* ``state``  - blocked attention state (OUT, LSE) of one key/value partition
  (Sec. 2.2.4, Eq. attention_state), the state composition (Eq. composition)
  in binary and n-ary form, full softmax attention, the selective step that
  composes fresh and reused states (Sec. 2.2.4, Fig. 4), the contribution
  weights w_i = exp(LSE_i)/sum exp(LSE) (Sec. 4.1.1 and Eq. lse_weight),
  and the ranking / threshold selection used by the planner-driven workload.
* ``brute``  - the same quantities by pure-Python loops with ``math.exp``,
  for tiny shapes only.
* ``multistep`` - the planner-driven multi-step workload: per-block state
  caches across denoising steps, anchor steps and threshold selection.

All pins (what the oracle is checked against besides itself) are in
``tests/test_oracle_pins.py``.  The paper's own error-model planner (Alg. 1)
is not part of the hot path and is not represented here.
"""
from .state import (  # noqa: F401
    partition_state,
    partition_states,
    compose2,
    merge,
    full_attention,
    selective_step,
    contrib,
    rank_partitions,
    plan_threshold,
)
