"""Pins for the oracle's LPT placement (Algorithm 1 placement loop, Section 3.1), CPU only."""
import heapq
import itertools

import numpy as np
from hypothesis import given, settings, strategies as st

import oracle


def _random_plan(seed, K, R, maxk):
    rng = np.random.default_rng(seed)
    row = rng.integers(1, 1000, size=K).astype(np.uint32)
    order = np.lexsort((np.arange(K), -row.astype(np.int64)))
    ks = rng.integers(1, maxk + 1, size=K).astype(np.uint32)
    return row, order.astype(np.uint32), np.minimum(ks, R)


@settings(max_examples=80, deadline=None)
@given(seed=st.integers(0, 10**6), K=st.integers(1, 40), R=st.integers(1, 12), maxk=st.integers(1, 5),
       cold=st.integers(0, 10**6))
def test_lpt_invariants(seed, K, R, maxk, cold):
    row, keys, ks = _random_plan(seed, K, R, maxk)
    members, off, L = oracle.place_lpt(keys, ks, row, R, cold)
    total = cold + int(row.sum())
    assert abs(L.sum() - total) <= 1e-12 * total + 1e-9           # planned loads sum to the window
    assert off[0] == 0 and np.array_equal(np.diff(off), ks)
    per_dest = np.full(R, cold / R)
    for a in range(K):
        m = members[off[a]:off[a + 1]]
        assert len(set(m.tolist())) == len(m) and m.max() < R        # distinct destinations
        per_dest[m] += row[keys[a]] / ks[a]                          # copies sum to the key's count
    assert np.allclose(per_dest, L, rtol=1e-12, atol=1e-9)


@settings(max_examples=80, deadline=None)
@given(seed=st.integers(0, 10**6), K=st.integers(1, 30), R=st.integers(1, 10), maxk=st.integers(1, 4),
       cold=st.integers(0, 5000))
def test_lpt_each_step_takes_k_smallest(seed, K, R, maxk, cold):
    # At every step the members are the k smallest (L, r) pairs (numpy lexsort), in that order.
    row, keys, ks = _random_plan(seed, K, R, maxk)
    members, off, L = oracle.place_lpt(keys, ks, row, R, cold)
    cur = np.full(R, np.float64(cold) / np.float64(R))
    for a in range(K):
        k = int(ks[a])
        want = np.lexsort((np.arange(R), cur))[:k]
        assert np.array_equal(members[off[a]:off[a + 1]], want)
        x = np.float64(row[keys[a]]) / np.float64(k)
        cur[want] = cur[want] + x
    assert np.array_equal(cur, L)                                     # bit-exact double arithmetic


def test_lpt_first_R_copies_fill_destinations_in_order():
    R = 9
    row = np.arange(100, 60, -1).astype(np.uint32)  # strictly decreasing, all positive
    keys = np.arange(len(row), dtype=np.uint32)
    ks = np.ones(len(row), np.uint32)
    members, off, L = oracle.place_lpt(keys, ks, row, R, 123)
    assert members[:R].tolist() == list(range(R))
    ks2 = np.array([3, 2, 4] + [1] * 5, np.uint32)
    members2, off2, _ = oracle.place_lpt(keys[:8], ks2, row, R, 0)
    assert members2[:R].tolist() == list(range(R))


def test_lpt_matches_heap_scheduler_for_single_copies():
    rng = np.random.default_rng(0)
    for _ in range(50):
        R = int(rng.integers(1, 20))
        K = int(rng.integers(1, 200))
        row = rng.integers(1, 10**6, size=K).astype(np.uint32)
        keys = np.lexsort((np.arange(K), -row.astype(np.int64))).astype(np.uint32)
        cold = int(rng.integers(0, 10**7))
        members, off, L = oracle.place_lpt(keys, np.ones(K, np.uint32), row, R, cold)
        h = [(np.float64(cold) / R, r) for r in range(R)]
        heapq.heapify(h)
        got = []
        for b in keys:
            l, r = heapq.heappop(h)
            got.append(r)
            heapq.heappush(h, (l + np.float64(row[b]), r))
        assert members.tolist() == got


def _opt_makespan(jobs, R):
    best = float("inf")
    for assign in itertools.product(range(R), repeat=len(jobs)):
        loads = [0.0] * R
        for j, r in zip(jobs, assign):
            loads[r] += j
        best = min(best, max(loads))
    return best


def test_lpt_graham_bound_single_copies():
    # Graham 1969: LPT makespan <= (4/3 - 1/(3R)) OPT on identical machines; a common
    # initial offset only shrinks the ratio.
    rng = np.random.default_rng(42)
    worst = 0.0
    for _ in range(120):
        R = int(rng.integers(2, 5))
        n = int(rng.integers(R + 1, 9))
        row = rng.integers(1, 60, size=n).astype(np.uint32)
        keys = np.lexsort((np.arange(n), -row.astype(np.int64))).astype(np.uint32)
        cold = int(rng.choice([0, 0, int(rng.integers(0, 200))]))
        _, _, L = oracle.place_lpt(keys, np.ones(n, np.uint32), row, R, cold)
        opt = _opt_makespan(row.astype(float).tolist(), R) + cold / R
        ratio = L.max() / opt
        worst = max(worst, ratio)
        assert ratio <= 4 / 3 - 1 / (3 * R) + 1e-12
    assert worst > 1.0  # the brute force found instances where LPT is not optimal


def test_lpt_graham_tight_instance():
    # The classic tight family: 2R+1 jobs 2R-1, 2R-1, 2R-2, 2R-2, ..., R+1, R+1, R, R, R.
    for R in (2, 3):
        jobs = []
        for v in range(2 * R - 1, R, -1):
            jobs += [v, v]
        jobs += [R, R, R]
        row = np.array(jobs, np.uint32)
        keys = np.arange(len(jobs), dtype=np.uint32)
        _, _, L = oracle.place_lpt(keys, np.ones(len(jobs), np.uint32), row, R, 0)
        assert L.max() == 4 * R - 1 and 3 * R == sum(jobs) / R       # LPT = 4R-1, OPT = 3R
