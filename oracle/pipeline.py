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

``threads`` > 1 runs independent units of the same definition on several host
threads (the C calls release the interpreter lock): counting by groups of whole
intervals or, within one interval, by request ranges with the integer rows summed;
plans by (window, candidate); routing by (interval, candidate, request range); the
replay by candidate.  Every unit calls the same single-threaded oracle function on its part
of the input, so the results do not depend on the thread count.

TEST INFRASTRUCTURE: see the package docstring.
"""
from __future__ import annotations

import os
import time
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, List, Optional, Tuple

import numpy as np

from . import admit, admit_affinity, count_rates, place_hash, place_lpt, replay, route, route_live


def plan_window(j: int) -> int:
    return max(j - 1, 0)


def build_plan(counts: np.ndarray, R: int, candidates, w: int, c: int) -> Dict:
    """The plan of candidate c built from counts row w (Eq. 1 admission and LPT, or an
    ablation variant's admission and placement)."""
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
    return dict(adm_keys=adm_keys, adm_k=adm_k, cold=cold, clamped=clamped,
                members=members, member_off=member_off, L=L, n_window=n_w)


def build_plans(counts: np.ndarray, R: int, candidates, pairs: List[Tuple[int, int]], threads: int = 1) -> Dict:
    """The plan of every (window, candidate) pair in ``pairs``: dict[(w, c)] -> plan dict."""
    pairs = list(pairs)
    if threads <= 1:
        built = [build_plan(counts, R, candidates, w, c) for w, c in pairs]
    else:
        with ThreadPoolExecutor(threads) as ex:
            built = list(ex.map(lambda wc: build_plan(counts, R, candidates, wc[0], wc[1]), pairs))
    return dict(zip(pairs, built))


def host_threads() -> int:
    """Host threads available to this process (its CPU affinity)."""
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        return os.cpu_count() or 1


def count_fanout(keys, offsets, K: int, threads: int) -> np.ndarray:
    """Counts per interval with ``threads`` units of the same counting function: with
    at least as many intervals as threads, each unit counts a contiguous group of whole
    intervals (its own rows); otherwise the stream is cut into request ranges whose rows
    are summed."""
    keys = np.ascontiguousarray(keys, dtype=np.uint32)
    off = np.asarray(offsets, dtype=np.uint64)
    n, J = keys.shape[0], off.shape[0] - 1
    if threads <= 1 or n < 2 * threads:
        return count_rates(keys, off, K)[0]
    if J >= threads:
        jc = sorted({int(x) for x in np.searchsorted(off.astype(np.int64), [n * t // threads for t in range(threads)])}
                    | {0, J})
        counts = np.zeros((J, K), dtype=np.uint32)

        def rows(g):
            j0, j1 = jc[g], jc[g + 1]
            s, e = int(off[j0]), int(off[j1])
            counts[j0:j1] = count_rates(keys[s:e], off[j0:j1 + 1] - off[j0], K)[0]

        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(rows, range(len(jc) - 1)))
        return counts
    cuts = [n * t // threads for t in range(threads + 1)]

    def part(t):
        s, e = cuts[t], cuts[t + 1]
        loc = (np.clip(off.astype(np.int64), s, e) - s).astype(np.uint64)
        return count_rates(keys[s:e], loc, K)[0]

    with ThreadPoolExecutor(threads) as ex:
        parts = list(ex.map(part, range(threads)))
    total = parts[0].astype(np.uint64)
    for p in parts[1:]:
        total += p
    return total.astype(np.uint32)


def run(wl, lru: Optional[List[np.ndarray]] = None, counts_prev: Optional[np.ndarray] = None,
        timings: Optional[dict] = None, dispatch: str = "static", threads: int = 1,
        piece: int = 1 << 22) -> Dict:
    """Count -> plan -> route -> replay over ``wl`` (a workload.Workload).

    ``counts_prev`` (one row) stands in for the window before interval 0 when a
    stream is processed in chunks; ``lru`` is the carried replay state per
    candidate; ``dispatch`` is "static" (interval-start planned loads) or "live"
    (running loads within each interval); ``threads`` fans independent units out
    over host threads (``piece`` = most requests one static routing unit takes).
    Returns counts, plans, dest [P][n], stats [J][P][R][4] (or [bins][P][R][4] with
    ``wl.stat_offsets``), lru, and ``win_of[j][c]``, the window of candidate c's plan in
    interval j.
    """
    t0 = time.perf_counter()
    counts = count_fanout(wl.keys, wl.offsets, wl.num_keys, threads)
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
    plans = build_plans(src, R, wl.candidates, needed, threads)
    t2 = time.perf_counter()
    if dispatch not in ("static", "live"):
        raise ValueError(f"unknown dispatch {dispatch!r}")
    dest = np.zeros((P, wl.n), dtype=np.uint16)
    off = wl.offsets.astype(np.int64)
    units = []  # (c, plan, s, e): route requests [s, e) of one interval with one plan
    for j in range(J):
        s, e = int(off[j]), int(off[j + 1])
        if e == s:
            continue
        for c in range(P):
            pl = plans[(win_of[j][c], c)]
            step = (e - s) if (dispatch == "live" or threads <= 1) else piece
            for a in range(s, e, step):  # live dispatch is one chain per interval
                units.append((c, pl, a, min(e, a + step)))

    def route_unit(u):
        c, pl, s, e = u
        if dispatch == "live":
            dest[c, s:e] = route_live(wl.keys[s:e], wl.first_index + s, wl.seed, wl.num_keys, R,
                                      pl["adm_keys"], pl["member_off"], pl["members"])
        else:
            dest[c, s:e] = route(wl.keys[s:e], wl.first_index + s, wl.seed, wl.num_keys, R,
                                 pl["adm_keys"], pl["member_off"], pl["members"], pl["L"])

    if threads <= 1:
        for u in units:
            route_unit(u)
    else:
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(route_unit, units))
    t3 = time.perf_counter()
    soff = wl.offsets if wl.stat_offsets is None else wl.stat_offsets
    stats = np.zeros((len(soff) - 1, P, R, 4), dtype=np.uint64)
    out_lru = [None] * P
    if threads <= 1:
        for c, cand in enumerate(wl.candidates):
            st, state = replay(wl.keys, wl.suffix, wl.prefix_len, dest[c], soff, R, cand.W,
                               None if lru is None else lru[c])
            stats[:, c] = st
            out_lru[c] = state
    else:
        for c, cand in enumerate(wl.candidates):
            out_lru[c] = None

        def replay_unit(c):
            st, state = replay(wl.keys, wl.suffix, wl.prefix_len, dest[c], soff, R, wl.candidates[c].W,
                               None if lru is None else lru[c])
            stats[:, c] = st
            out_lru[c] = state

        order = sorted(range(P), key=lambda c: -wl.candidates[c].W)  # longest units first
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(replay_unit, order))
    t4 = time.perf_counter()
    if timings is not None:
        timings.update(count=t1 - t0, plan=t2 - t1, route=t3 - t2, replay=t4 - t3, n_plans=len(plans), threads=threads)
    return dict(counts=counts, plans=plans, win_of=win_of, dest=dest, stats=stats, lru=out_lru)
