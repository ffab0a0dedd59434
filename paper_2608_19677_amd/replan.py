"""Replanning under rate drift on the device path (Section 5.4 "Rate drift and
remapping"; Appendix E, table of replan measurements).

The study stream (``workload.drift``) has one control interval per drift step and
candidates that differ only in which window each interval's plan comes from:
candidate 0 installs a fresh plan at every boundary; candidate t keeps the plan of
interval t-1 through interval t. Both therefore route the same requests the same way
up to boundary t, so their replay statistics agree until then, and over interval t
they measure the two sides of the install decision:

* stale loss: hit of the fresh plan minus hit of the held plan over interval t (and
  over its second half, once the fresh plan's caches have rewarmed);
* warm-up dip: hit of the held plan minus hit of the fresh plan in the first
  statistics bin after the boundary;
* cache churn and count churn between the consecutive fresh plans, from
  cr_plan_churn.

Hit rates are token weighted (hit prefix tokens over all prompt tokens, the served
KV-hit of Section 4) and request weighted. Every number here is a ratio of integers
the library produced; nothing of the path itself is computed on the host.
"""
from __future__ import annotations

from typing import Dict, List

import numpy as np

from .pipeline import Pipeline


class DriftStudy:
    """Count -> plan -> route -> replay -> churn for a drift stream on the GPU."""

    STAGES = Pipeline.STAGES + ("churn",)

    def __init__(self, wl, device="cuda"):
        if wl.plan_windows is None or wl.J < 2:
            raise ValueError("the drift study needs a stream with plan windows and at least two intervals")
        self.wl = wl
        self.pipe = Pipeline(wl, device)
        P = wl.P
        self.transitions = list(range(1, wl.J))
        self.pipe.set_churn_pairs([((t - 1) * P, t * P) for t in self.transitions])

    def step(self, stream=None):
        self.pipe.step(stream)
        self.pipe.churn(stream)

    def summary(self) -> Dict:
        p = self.pipe
        h = p.host()
        A = h["num_admitted"].astype(np.int64)
        S = np.array([int(h["member_off"][i, A[i]]) for i in range(A.shape[0])], dtype=np.int64)
        return summarize(self.wl, h["stats"], h["churn"], S, A, self.transitions) | dict(err=h["err"])


def _hits(st: np.ndarray):
    """(token-weighted, request-weighted) hit rate of stats summed over leading axes."""
    s = st.reshape(-1, 4).sum(axis=0, dtype=np.uint64).astype(np.float64)
    tok = s[3] / (s[2] + s[3]) if s[2] + s[3] else 0.0
    req = s[1] / s[0] if s[0] else 0.0
    return tok, req


def churn_rates(out4, s_p: int, s_q: int, a_p: int, a_q: int) -> Dict[str, float]:
    """Ratios from one cr_plan_churn row and the two plans' |S| and admitted counts."""
    common, both, k_changed, same = (int(x) for x in out4)
    union = s_p + s_q - common
    kunion = a_p + a_q - both
    return dict(cache_churn=1.0 - common / union if union else 0.0,
                count_churn=k_changed / both if both else 0.0,
                warm_set_churn=1.0 - both / kunion if kunion else 0.0,
                moved=1.0 - same / both if both else 0.0)


def summarize(wl, stats: np.ndarray, churn: np.ndarray, S: np.ndarray, A: np.ndarray,
              transitions: List[int]) -> Dict:
    """Per-transition churn, stale loss and warm-up dip (percentage points) and their means.

    stats u64 [bins][P][R][4]; churn u64 [transitions][4]; S, A per plan p = g * P + c."""
    P = wl.P
    soff = np.asarray(wl.stat_offsets, dtype=np.int64)
    off = np.asarray(wl.offsets, dtype=np.int64)
    rows = []
    for i, t in enumerate(transitions):
        b0 = int(np.searchsorted(soff, off[t]))
        b1 = int(np.searchsorted(soff, off[t + 1]))
        if soff[b0] != off[t] or soff[b1] != off[t + 1]:
            raise ValueError("statistics bins must nest in the control intervals")
        half = b0 + (b1 - b0) // 2
        fresh, held = stats[b0:b1, 0], stats[b0:b1, t]
        f_tok, f_req = _hits(fresh)
        h_tok, h_req = _hits(held)
        fs_tok, _ = _hits(stats[half:b1, 0])
        hs_tok, _ = _hits(stats[half:b1, t])
        f1_tok, f1_req = _hits(stats[b0:b0 + 1, 0])
        h1_tok, h1_req = _hits(stats[b0:b0 + 1, t])
        pa, pb = (t - 1) * P, t * P
        row = dict(transition=f"{t - 1}->{t}",
                   **churn_rates(churn[i], int(S[pa]), int(S[pb]), int(A[pa]), int(A[pb])),
                   stale_loss_pts=100.0 * (f_tok - h_tok), stale_loss_steady_pts=100.0 * (fs_tok - hs_tok),
                   stale_loss_req_pts=100.0 * (f_req - h_req),
                   warmup_dip_pts=100.0 * (h1_tok - f1_tok), warmup_dip_req_pts=100.0 * (h1_req - f1_req),
                   fresh_hit=f_tok, held_hit=h_tok)
        rows.append(row)
    keys = [k for k in rows[0] if k != "transition"] if rows else []
    mean = {k: float(np.mean([r[k] for r in rows])) for k in keys}
    return dict(transitions=rows, mean=mean)
