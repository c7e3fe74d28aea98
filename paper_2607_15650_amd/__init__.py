"""MI355X (gfx950) hot path of selective attention-state reuse for
context-parallel DiT inference: fresh partition states, state composition and
contribution weights, as HIP kernels behind a C ABI (include/ditango.h)."""
from .api import (attn_partition_states, merge_states, contrib, contrib_workspace_bytes,  # noqa: F401
                  state_norms, norms_workspace_bytes)
from .planner import AnchorPlanner, plan_threshold, rank_partitions  # noqa: F401,E402
