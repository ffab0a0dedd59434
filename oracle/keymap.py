"""Opaque-key remap -- TEST INFRASTRUCTURE.

The planner needs only {(b, lambda_b)}, and b may be a salted or ephemeral identifier
(Appendix A.2 "Data handling"); the paper's summaries carry opaque business keys
(Section 2.1). Counting into dense per-key rows needs each opaque id mapped to a dense
index first. The mapping fixed here: an id's dense index is the rank of its first
occurrence among the distinct ids of the stream (order of first appearance), so it does
not depend on how the work is scheduled. 0xFFFFFFFF is not an id; it, and any id not in
the directory, maps to 0xFFFFFFFF.
"""
from __future__ import annotations

from typing import Dict, Tuple

import numpy as np

NO_KEY = 0xFFFFFFFF


def build(ids) -> Dict[int, int]:
    """Directory {opaque id: dense index} in order of first appearance."""
    d: Dict[int, int] = {}
    for x in np.asarray(ids, dtype=np.uint32).tolist():
        if x != NO_KEY and x not in d:
            d[x] = len(d)
    return d


def lookup(directory: Dict[int, int], ids) -> np.ndarray:
    return np.array([directory.get(x, NO_KEY) for x in np.asarray(ids, dtype=np.uint32).tolist()], dtype=np.uint32)


def scatter(directory: Dict[int, int], attr_ids, values, num_keys: int, fill: int = 0) -> np.ndarray:
    """Per-key attribute given by opaque id -> array indexed by dense index (ids absent
    from the directory are dropped; dense indices without an attribute keep ``fill``)."""
    out = np.full(num_keys, fill, dtype=np.uint32)
    for x, v in zip(np.asarray(attr_ids, dtype=np.uint32).tolist(), np.asarray(values).tolist()):
        k = directory.get(x)
        if k is not None and k < num_keys:
            out[k] = v
    return out


def remap(ids) -> Tuple[np.ndarray, Dict[int, int]]:
    d = build(ids)
    return lookup(d, ids), d
