"""Device workspace of the attention launch, kept across calls.

ditango_attn_partition_states_ws balances a launch over the XCDs with queue
counters in the workspace, and splits its last, partly filled round when
given room for the partial states; the bytes depend on the shape, the
selection and the device.  This holder asks the library for them once per
(shape, selection) and keeps one device buffer that only grows.
"""
from __future__ import annotations

from typing import Dict, Optional, Sequence, Tuple

import torch

from . import api


class AttnWorkspace:
    def __init__(self, device="cuda"):
        self.device = device
        self.buf: Optional[torch.Tensor] = None
        self._bytes: Dict[Tuple, int] = {}

    def get(self, dtype: torch.dtype, B: int, H: int, D: int, q_len: int,
            offsets: Sequence[int], select: Sequence[int]) -> Optional[torch.Tensor]:
        """The buffer for this launch, or None for float32 inputs."""
        key = (dtype, B, H, D, q_len, tuple(int(o) for o in offsets), tuple(1 if s else 0 for s in select))
        n = self._bytes.get(key)
        if n is None:
            n = self._bytes[key] = api.attn_workspace_bytes(dtype, B, H, D, q_len, offsets, select)
        if n == 0:
            return None
        if self.buf is None or self.buf.numel() < n:
            self.buf = torch.empty(n, dtype=torch.uint8, device=self.device)
        return self.buf
