"""The oracle's own driver: one pass of the whole path over a workload.

Semantics it fixes (each restated from the paper or from the reading noted):

* Counting windows are the control intervals; the plan used during interval j
  is built from the counts of interval j-1 (the table stays fixed for an
  interval and is rebuilt from the latest telemetry, Section 3.2); interval 0
  has no earlier window and uses its own.
* A workload may name the window of every (interval, candidate) plan itself
  (``plan_windows``), as the replanning study does to compare fresh and stale
  plans (Section 5.4, Appendix E).
* A candidate may be a stage of the component ablation (Section 5.2): "flat"
  admits nothing, "affinity" admits the top C keys with one copy each and
  places them by hash, "replicated" keeps Eq. 1 and places by hash, "full" is
  the method.
* Candidate (W, a, b) has C = R W warm slots and q_cap = (a/b) x N_w / R,
  i.e. q_num = a N_w and q_den = b R with N_w the window's request count.
* Dispatch is static by default (planned interval-start loads, order
  independent) or live: least-loaded member and power of two choices on the
  running per-destination counts of the interval (Section 3.1 "Placement and
  dispatch").
* The replay's LRU state per (candidate, destination) starts empty and is
  carried across intervals and plan changes (Section 3.2, Appendix E).

TEST INFRASTRUCTURE: see the package docstring.
"""
from __future__ import annotations

import time
from typing import Dict, List, Optional, Tuple

import numpy as np

from . import admit, admit_affinity, count_rates, place_hash, place_lpt, replay, route, route_live


def plan_window(j: int) -> int:
    return max(j - 1, 0)


def build_plans(counts: np.ndarray, R: int, candidates, pairs: List[Tuple[int, int]]) -> Dict:
    """The plan of every (window, candidate) pair in ``pairs``: dict[(w, c)] -> plan dict."""
    plans = {}
    for w, c in pairs:
        row = counts[w]
        n_w = int(row.sum(dtype=np.uint64))
        cand = candidates[c]
        variant = getattr(cand, "variant", "full")
        q_num, q_den = cand.a * n_w, cand.b * R
        if n_w == 0 or variant == "flat":
            adm_keys = np.zeros(0, np.uint32)
            adm_k = np.zeros(0, np.uint32)
            cold, clamped = n_w, 0
        elif variant == "affinity":
            adm_keys, adm_k, cold = admit_affinity(row, R, cand.W, n_w)
            clamped = 0
        elif variant in ("full", "replicated"):
            adm_keys, adm_k, cold, clamped = admit(row, R, cand.W, n_w, q_num, q_den)
        else:
            raise ValueError(f"unknown plan variant {variant!r}")
        if variant in ("affinity", "replicated"):
            members, member_off, L = place_hash(adm_keys, adm_k, row, R, cold, cand.place_seed)
        else:
            members, member_off, L = place_lpt(adm_keys, adm_k, row, R, cold)
        plans[(w, c)] = dict(adm_keys=adm_keys, adm_k=adm_k, cold=cold, clamped=clamped,
                             members=members, member_off=member_off, L=L, n_window=n_w)
    return plans


def run(wl, lru: Optional[List[np.ndarray]] = None, counts_prev: Optional[np.ndarray] = None,
        timings: Optional[dict] = None, dispatch: str = "static") -> Dict:
    """Count -> plan -> route -> replay over ``wl`` (a workload.Workload).

    ``counts_prev`` (one row) stands in for the window before interval 0 when a
    stream is processed in chunks; ``lru`` is the carried replay state per
    candidate; ``dispatch`` is "static" (interval-start planned loads) or "live"
    (running loads within each interval).  Returns counts, plans, dest [P][n], stats [J][P][R][4] (or
    [bins][P][R][4] with ``wl.stat_offsets``), lru, and ``win_of[j][c]``, the window
    of candidate c's plan in interval j.
    """
    t0 = time.perf_counter()
    counts, _ = count_rates(wl.keys, wl.offsets, wl.num_keys)
    t1 = time.perf_counter()
    J, P, R = wl.J, wl.P, wl.R
    if counts_prev is None:
        src = counts
        if wl.plan_windows is None:
            win_of = [[plan_window(j)] * P for j in range(J)]
        else:
            win_of = [[int(wl.plan_windows[j][c]) for c in range(P)] for j in range(J)]
    else:
        if wl.plan_windows is not None:
            raise ValueError("a stream processed in chunks plans every interval from the window before it")
        src = np.concatenate([counts_prev.reshape(1, -1), counts], axis=0)
        win_of = [[j] * P for j in range(J)]  # interval j uses row j of src = counts of interval j-1
    needed = sorted({(win_of[j][c], c) for j in range(J) for c in range(P)})
    plans = build_plans(src, R, wl.candidates, needed)
    t2 = time.perf_counter()
    dest = np.zeros((P, wl.n), dtype=np.uint16)
    off = wl.offsets.astype(np.int64)
    for j in range(J):
        s, e = int(off[j]), int(off[j + 1])
        if e == s:
            continue
        for c in range(P):
            pl = plans[(win_of[j][c], c)]
            if dispatch == "live":
                dest[c, s:e] = route_live(wl.keys[s:e], wl.first_index + s, wl.seed, wl.num_keys, R,
                                          pl["adm_keys"], pl["member_off"], pl["members"])
            elif dispatch == "static":
                dest[c, s:e] = route(wl.keys[s:e], wl.first_index + s, wl.seed, wl.num_keys, R,
                                     pl["adm_keys"], pl["member_off"], pl["members"], pl["L"])
            else:
                raise ValueError(f"unknown dispatch {dispatch!r}")
    t3 = time.perf_counter()
    soff = wl.offsets if wl.stat_offsets is None else wl.stat_offsets
    stats = np.zeros((len(soff) - 1, P, R, 4), dtype=np.uint64)
    out_lru = []
    for c, cand in enumerate(wl.candidates):
        st, state = replay(wl.keys, wl.suffix, wl.prefix_len, dest[c], soff, R, cand.W,
                           None if lru is None else lru[c])
        stats[:, c] = st
        out_lru.append(state)
    t4 = time.perf_counter()
    if timings is not None:
        timings.update(count=t1 - t0, plan=t2 - t1, route=t3 - t2, replay=t4 - t3, n_plans=len(plans))
    return dict(counts=counts, plans=plans, win_of=win_of, dest=dest, stats=stats, lru=out_lru)
