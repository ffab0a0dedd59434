"""Opaque keys on the device path: a directory from 32-bit opaque ids to dense indices
(cr_keymap_*), built from the request stream, so that counting, planning, dispatch and
replay run unchanged on dense keys (Appendix A.2 "Data handling": b may be salted or
ephemeral). Marshalling only; the library does the work.
"""
from __future__ import annotations

import numpy as np
import torch

from . import binding as B


class KeyMap:
    """Device directory for up to ``capacity`` distinct opaque ids."""

    def __init__(self, capacity: int, device="cuda"):
        self.capacity = capacity
        self.device = device
        self.table = torch.empty(B.cr_keymap_bytes(capacity), dtype=torch.uint8, device=device)
        self.num_keys = torch.zeros(1, dtype=torch.int32, device=device)
        self.ws = None

    def build(self, ids: torch.Tensor, err: torch.Tensor, stream=None):
        need = B.cr_keymap_workspace_bytes(ids.numel())
        if self.ws is None or self.ws.numel() < need:
            self.ws = torch.empty(need, dtype=torch.uint8, device=self.device)
        B.cr_keymap_build(ids, self.capacity, self.table, self.ws, self.num_keys, err, stream)

    def lookup(self, ids: torch.Tensor, out: torch.Tensor, stream=None):
        B.cr_keymap_lookup(self.table, self.capacity, ids, out, stream)

    def scatter(self, ids: torch.Tensor, values: torch.Tensor, out: torch.Tensor, stream=None):
        B.cr_keymap_scatter(self.table, self.capacity, ids, values, out, stream)


def to_device(a, device="cuda") -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint32).view(np.int32)).to(device)
