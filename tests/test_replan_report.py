"""Host-side report of the replanning study (ratios of the library's integers), CPU only."""
from types import SimpleNamespace

import numpy as np
import pytest

from paper_2608_19677_amd.replan import churn_rates, summarize


def test_churn_rates_from_counts():
    # |S_p| = 6, |S_q| = 4, 3 pairs in common -> Jaccard 3 / 7; 5 and 4 admitted keys,
    # 3 in both -> warm-set Jaccard 3 / 6; one of the 3 changes k, two keep their set
    r = churn_rates([3, 3, 1, 2], 6, 4, 5, 4)
    assert r["cache_churn"] == pytest.approx(4 / 7)
    assert r["warm_set_churn"] == pytest.approx(0.5)
    assert r["count_churn"] == pytest.approx(1 / 3)
    assert r["moved"] == pytest.approx(1 / 3)
    assert churn_rates([0, 0, 0, 0], 0, 0, 0, 0) == dict(cache_churn=0.0, count_churn=0.0, warm_set_churn=0.0,
                                                         moved=0.0)


def test_summary_of_a_hand_made_run():
    # two intervals of 10 requests, statistics in bins of 5; candidate 1 holds the old plan
    # in interval 1. Columns: requests, hits, prefill tokens, hit prefix tokens.
    wl = SimpleNamespace(P=2, offsets=np.array([0, 10, 20]), stat_offsets=np.array([0, 5, 10, 15, 20]))
    stats = np.zeros((4, 2, 1, 4), dtype=np.uint64)
    stats[:2, :, 0] = [5, 4, 100, 400]                 # interval 0: same for both candidates
    stats[2, 0, 0] = [5, 1, 400, 100]                  # fresh, first bin after the install: 20 % token hit
    stats[3, 0, 0] = [5, 5, 0, 500]                    # fresh, rewarmed: 100 %
    stats[2, 1, 0] = [5, 4, 200, 300]                  # held plan: 60 %, then 60 %
    stats[3, 1, 0] = [5, 4, 200, 300]
    churn = np.array([[3, 3, 1, 2]], dtype=np.uint64)
    S = np.array([6, 6, 4, 6])
    A = np.array([5, 5, 4, 5])
    s = summarize(wl, stats, churn, S, A, [1])
    row = s["transitions"][0]
    assert row["transition"] == "0->1"
    assert row["fresh_hit"] == pytest.approx(600 / 1000) and row["held_hit"] == pytest.approx(600 / 1000)
    assert row["stale_loss_pts"] == pytest.approx(0.0)
    assert row["stale_loss_steady_pts"] == pytest.approx(40.0)     # second half: 100 % vs 60 %
    assert row["warmup_dip_pts"] == pytest.approx(40.0)            # first bin: 60 % vs 20 %
    assert row["warmup_dip_req_pts"] == pytest.approx(60.0)        # 4/5 vs 1/5 requests
    assert row["stale_loss_req_pts"] == pytest.approx(100 * (6 / 10 - 8 / 10))
    assert row["cache_churn"] == pytest.approx(4 / 7)               # plans 0 and 2
    assert s["mean"]["warmup_dip_pts"] == pytest.approx(40.0)


def test_summary_rejects_bins_that_straddle_an_interval():
    wl = SimpleNamespace(P=2, offsets=np.array([0, 10, 20]), stat_offsets=np.array([0, 7, 20]))
    stats = np.zeros((2, 2, 1, 4), dtype=np.uint64)
    with pytest.raises(ValueError):
        summarize(wl, stats, np.zeros((1, 4), np.uint64), np.zeros(4, int), np.zeros(4, int), [1])
