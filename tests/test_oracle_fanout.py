"""The oracle driver's thread fan-out (independent units on host threads) gives exactly the
single-threaded results: counts, plans, destinations, statistics and carried LRU state."""
import numpy as np
import pytest

from oracle import pipeline as opipe
from paper_2608_19677_amd import workload as wl

CASES = [
    # one interval: counting splits the request range and sums the rows
    dict(seed=3, num_keys=400, n=30_000, R=30, Ws=[16, 40], J=1, hot=2, hot_share=0.3),
    # more intervals than threads: counting takes groups of whole intervals
    dict(seed=8, num_keys=400, n=30_000, R=4, Ws=[2, 50], J=20, hot=2, hot_share=0.9),
    # R > 64 and several load targets
    dict(seed=5, num_keys=3000, n=40_000, R=100, Ws=[8, 70], J=3, hot=3, hot_share=0.4, qs=[(1, 1), (4, 5)]),
    # many candidates (replay fans out over them)
    dict(seed=14, num_keys=300, n=20_000, R=8, Ws=list(range(1, 9)), J=2, qs=[(a, 8) for a in range(5, 9)], hot=1,
         hot_share=0.2),
]


def _same(a, b):
    for k in ("counts", "dest", "stats"):
        np.testing.assert_array_equal(a[k], b[k], err_msg=k)
    assert a["win_of"] == b["win_of"]
    assert a["plans"].keys() == b["plans"].keys()
    for key, pa in a["plans"].items():
        pb = b["plans"][key]
        for f in ("adm_keys", "adm_k", "members", "member_off"):
            np.testing.assert_array_equal(pa[f], pb[f], err_msg=f"{key} {f}")
        assert pa["L"].tobytes() == pb["L"].tobytes()
        assert (pa["cold"], pa["clamped"]) == (pb["cold"], pb["clamped"])
    for la, lb in zip(a["lru"], b["lru"]):
        np.testing.assert_array_equal(la, lb)


@pytest.mark.parametrize("case", CASES, ids=[f"f{c['seed']}" for c in CASES])
@pytest.mark.parametrize("threads", [2, 5])
def test_fanout_equals_single_thread(case, threads):
    w = wl.small_random(**case)
    _same(opipe.run(w), opipe.run(w, threads=threads, piece=777))


def test_fanout_live_dispatch_and_carried_state():
    w = wl.small_random(9, num_keys=500, n=25_000, R=16, Ws=[4, 24], J=4, hot=2, hot_share=0.5)
    lru = [np.arange(16 * c.W, dtype=np.uint32).reshape(16, c.W) % 500 for c in w.candidates]
    for c in range(len(lru)):  # a carried state has distinct keys per destination
        lru[c] = np.array([np.unique(r)[: w.candidates[c].W] for r in lru[c]], dtype=np.uint32)
    prev = np.bincount(w.keys[:5000], minlength=w.num_keys).astype(np.uint32)
    a = opipe.run(w, lru=lru, counts_prev=prev, dispatch="live")
    b = opipe.run(w, lru=lru, counts_prev=prev, dispatch="live", threads=3)
    _same(a, b)


def test_count_fanout_split_points():
    # every split of one interval into request ranges sums to the same row
    w = wl.small_random(21, num_keys=50, n=10_007, R=4, Ws=[2], J=1)
    ref = opipe.count_fanout(w.keys, w.offsets, w.num_keys, 1)
    for t in (2, 3, 7, 16):
        np.testing.assert_array_equal(opipe.count_fanout(w.keys, w.offsets, w.num_keys, t), ref)
    assert int(ref.sum()) == w.n
