"""Pins for the oracle's rate counting and admission (Eq. 1, Algorithm 1), CPU only."""
import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle
from paper_2608_19677_amd import workload as wl


def test_counts_equal_bincount_per_interval():
    w = wl.small_random(11, num_keys=300, n=20_000, R=8, Ws=[4], J=7)
    counts, bad = oracle.count_rates(w.keys, w.offsets, w.num_keys)
    assert bad == 0
    off = w.offsets.astype(np.int64)
    for j in range(w.J):
        ref = np.bincount(w.keys[off[j]:off[j + 1]], minlength=w.num_keys)
        assert np.array_equal(counts[j], ref)
        assert counts[j].sum() == off[j + 1] - off[j]


def test_counts_skip_out_of_range_keys():
    keys = np.array([0, 5, 5, 9, 10, 4000000000], np.uint32)
    counts, bad = oracle.count_rates(keys, np.array([0, 6], np.uint64), 10)
    assert bad == 2 and counts[0, 5] == 2 and counts[0].sum() == 4


def test_counts_reject_bad_offsets():
    with pytest.raises(ValueError):
        oracle.count_rates(np.zeros(4, np.uint32), np.array([0, 3, 2, 4], np.uint64), 5)
    with pytest.raises(ValueError):
        oracle.count_rates(np.zeros(4, np.uint32), np.array([0, 3], np.uint64), 5)


# --- Eq. 1: k = max(1, ceil(lambda / q_cap)) with q_cap = q_num / q_den -------------

@pytest.mark.parametrize("q", [1, 7, 352, 100000])
def test_kb_integer_target_edges(q):
    R = 1000
    assert oracle.kb(q, q, 1, R) == 1          # c = q_cap -> exactly one destination
    assert oracle.kb(q + 1, q, 1, R) == 2      # just above -> two
    assert oracle.kb(1, q, 1, R) == 1          # far below -> max(1, .) keeps one
    assert oracle.kb(2 * q, q, 1, R) == 2
    assert oracle.kb(2 * q + 1, q, 1, R) == 3


@settings(max_examples=300, deadline=None)
@given(c=st.integers(1, 2**32 - 1), qn=st.integers(1, 2**62), qd=st.integers(1, 2**31 - 1),
       R=st.integers(1, 65535))
def test_kb_is_the_ceiling(c, qn, qd, R):
    k = oracle.kb(c, qn, qd, R)
    # exact rational ceiling characterisation: (m-1) q_num < c q_den <= m q_num
    m = max(1, -(-(c * qd) // qn))
    assert k == min(R, m)
    assert (m - 1) * qn < c * qd <= m * qn or (m == 1 and c * qd <= qn)


def test_kb_replication_whales():
    # 6 % of a window against a target of 0.4 x (window / 16): 0.06 / 0.025 = 2.4 -> 3
    n_w, R = 30_000, 16
    c = int(0.06 * n_w)
    assert oracle.kb(c, 2 * n_w, 5 * R, R) == 3


def _lexsort_order(row):
    nz = np.nonzero(row)[0]
    return nz[np.lexsort((nz, -row[nz].astype(np.int64)))]


@settings(max_examples=60, deadline=None)
@given(seed=st.integers(0, 10**6), K=st.integers(1, 60), R=st.integers(1, 9), W=st.integers(1, 6),
       n=st.integers(0, 400), a=st.integers(1, 5), b=st.integers(1, 5))
def test_admission_is_maximal_prefix_of_rate_order(seed, K, R, W, n, a, b):
    rng = np.random.default_rng(seed)
    p = rng.dirichlet(np.full(K, 0.3))
    row = np.bincount(rng.choice(K, size=n, p=p), minlength=K).astype(np.uint32)
    n_w = int(row.sum())
    if n_w == 0:
        return
    q_num, q_den = a * n_w, b * R
    keys, ks, cold, clamped = oracle.admit(row, R, W, n_w, q_num, q_den)
    order = _lexsort_order(row)
    A = len(keys)
    assert np.array_equal(keys, order[:A])                 # a prefix of (rate desc, key asc)
    C = R * W
    assert ks.sum() <= C
    for key, k in zip(keys, ks):
        m = max(1, -(-(int(row[key]) * q_den) // q_num))
        assert k == min(m, R)
    if A < len(order):                                     # the next key does not fit
        nxt = order[A]
        k_next = min(R, max(1, -(-(int(row[nxt]) * q_den) // q_num)))
        assert ks.sum() + k_next > C
    assert cold == n_w - int(row[keys].sum())
    assert np.all(row[keys] > 0)


def test_admission_all_k_one_is_top_c_by_lexsort():
    rng = np.random.default_rng(1)
    row = np.bincount(rng.integers(0, 500, size=3000), minlength=600).astype(np.uint32)
    n_w, R, W = int(row.sum()), 10, 7
    keys, ks, cold, _ = oracle.admit(row, R, W, n_w, n_w * 1000, 1, )  # q_cap huge -> k = 1
    assert np.all(ks == 1)
    assert np.array_equal(keys, _lexsort_order(row)[:R * W])


def test_admission_prefix_stop_not_skip():
    # second key needs 3 slots and does not fit in C = 4 after the first (3); a later k=1 key
    # would fit, but admission stops at the first key that does not.
    row = np.array([0, 30, 25, 1], np.uint32)
    n_w = int(row.sum())
    keys, ks, cold, _ = oracle.admit(row, 4, 1, n_w, 10, 1)  # q_cap = 10 -> k = 3, 3, 1
    assert keys.tolist() == [1] and ks.tolist() == [3] and cold == 26


def test_admission_k_clamped_to_R():
    row = np.array([1000, 1], np.uint32)
    keys, ks, cold, clamped = oracle.admit(row, 4, 10, 1001, 10, 1)
    assert ks.tolist() == [4, 1] and clamped == 1


def test_primary_shape_has_k_one_everywhere():
    # The 70B-like shape keeps every key below the mean per-destination load (Section 3.2).
    w = wl.llama70b(n=300_000)
    counts, _ = oracle.count_rates(w.keys, w.offsets, w.num_keys)
    for j in range(min(w.J, 4)):
        row = counts[j]
        n_w = int(row.sum())
        assert row.max() * w.R <= n_w
        keys, ks, cold, clamped = oracle.admit(row, w.R, 64, n_w, n_w, w.R)
        assert np.all(ks == 1) and clamped == 0
