"""Reporting from the library's outputs (hit rates, imbalance) for the component ablation
(Section 5.2, 8B component ablation table): ratios of the integers and loads the device
produced, computed on the host after the step.

* KV hit: token weighted (hit prefix tokens over all prompt tokens) and request weighted.
* Planned imbalance: max L / mean L of the plan in force, averaged over the intervals.
* Realised imbalance: max / mean over destinations of the requests (and of the prefill
  tokens) each destination received, over the whole stream and per interval (averaged
  over the intervals that carry requests).
"""
from __future__ import annotations

from typing import Dict, List

import numpy as np


def hit_rates(stats: np.ndarray):
    """(token-weighted, request-weighted) hit rate of u64 stats [..., 4] summed over all
    leading axes; columns are requests, hits, prefill tokens, hit prefix tokens."""
    s = np.asarray(stats).reshape(-1, 4).sum(axis=0, dtype=np.uint64).astype(np.float64)
    tok = s[3] / (s[2] + s[3]) if s[2] + s[3] else 0.0
    req = s[1] / s[0] if s[0] else 0.0
    return float(tok), float(req)


def _max_over_mean(x: np.ndarray) -> float:
    m = float(np.mean(x))
    return float(np.max(x)) / m if m > 0 else 0.0


def ablation_summary(wl, stats: np.ndarray, loads: np.ndarray, gmap: List[int]) -> Dict:
    """One row per candidate. stats u64 [J][P][R][4]; loads f64 [NP][R] with plan
    p = gmap[j] * P + c in force for candidate c during interval j."""
    P = wl.P
    J = stats.shape[0]
    rows = []
    for c, cand in enumerate(wl.candidates):
        st = stats[:, c].astype(np.float64)            # [J][R][4]
        tok, req = hit_rates(stats[:, c])
        per_dest = st.sum(axis=0)                      # [R][4]
        live = [j for j in range(J) if st[j, :, 0].sum() > 0]
        rows.append(dict(
            variant=getattr(cand, "variant", "full"), W=cand.W,
            kv_hit=tok, request_hit=req,
            planned_imbalance=float(np.mean([_max_over_mean(loads[gmap[j] * P + c]) for j in live])) if live else 0.0,
            realised_imbalance=_max_over_mean(per_dest[:, 0]),
            realised_prefill_imbalance=_max_over_mean(per_dest[:, 2]),
            realised_imbalance_per_interval=float(np.mean([_max_over_mean(st[j, :, 0]) for j in live])) if live else 0.0,
        ))
    return dict(candidates=rows)
