"""Pins for the replanning study's oracle parts (Section 5.4, Appendix E), CPU only:
the churn measures between plans, the drift generator, and plans taken from windows
named per (interval, candidate)."""
import numpy as np
import pytest

import oracle
from oracle import pipeline as opipe
from oracle import replan
from paper_2608_19677_amd import workload as wl_mod


def _plan(assign):
    """Plan dict from {key: [destinations in selection order]} in admission order."""
    keys = list(assign)
    off = np.concatenate([[0], np.cumsum([len(assign[b]) for b in keys])]).astype(np.uint32)
    mem = np.array([r for b in keys for r in assign[b]], dtype=np.uint16)
    return dict(adm_keys=np.array(keys, dtype=np.uint32), member_off=off, members=mem)


def test_hand_example():
    # S_a = {(5,0),(5,1),(7,2)}, S_b = {(5,1),(5,3),(5,4),(9,2)}: one common pair (5,1);
    # key 5 is the only key in both, its k goes 2 -> 3 and its set changes.
    a = _plan({5: [1, 0], 7: [2]})
    b = _plan({9: [2], 5: [4, 1, 3]})
    assert replan.plan_churn(a, b) == (1, 1, 1, 0)
    r = replan.churn_rates(a, b)
    assert r["cache_churn"] == pytest.approx(1 - 1 / 6)   # |S_a ∪ S_b| = 3 + 4 - 1
    assert r["count_churn"] == 1.0
    assert r["warm_set_churn"] == pytest.approx(1 - 1 / 3)  # keys {5, 7} vs {5, 9}
    assert r["moved"] == 1.0


def test_same_set_in_another_order_is_no_churn():
    # T(b) is a set: the selection order of the members does not matter
    a = _plan({3: [0, 2, 1], 8: [4]})
    b = _plan({8: [4], 3: [1, 0, 2]})
    assert replan.plan_churn(a, b) == (4, 2, 0, 2)
    assert replan.churn_rates(a, b)["cache_churn"] == 0.0


def test_disjoint_plans_churn_fully():
    a = _plan({1: [0], 2: [1, 2]})
    b = _plan({3: [0], 4: [1, 2]})
    assert replan.plan_churn(a, b) == (0, 0, 0, 0)
    r = replan.churn_rates(a, b)
    assert r["cache_churn"] == 1.0 and r["warm_set_churn"] == 1.0 and r["count_churn"] == 0.0


def _lpt_plan(row, R, W):
    n_w = int(row.sum())
    keys, ks, cold, _ = oracle.admit(row, R, W, n_w, n_w, R)
    mem, off, _ = oracle.place_lpt(keys, ks, row, R, cold)
    return dict(adm_keys=keys, adm_k=ks, member_off=off, members=mem)


def _dense(plan, K, R):
    m = np.zeros((K, R), dtype=bool)
    for a, b in enumerate(plan["adm_keys"]):
        m[b, plan["members"][plan["member_off"][a]:plan["member_off"][a + 1]]] = True
    return m


@pytest.mark.parametrize("seed", range(6))
def test_matches_dense_indicator_form(seed):
    # The same four numbers from K x R indicator matrices of the two plans (LPT plans of
    # a counts row and of a lognormally perturbed copy of it).
    rng = np.random.default_rng(seed)
    K, R, W = 300, 7, 6
    row = (np.minimum(rng.zipf(1.3, size=K), 10**5) - 1).astype(np.uint32) * 3
    row2 = np.rint(row * np.exp(0.3 * rng.standard_normal(K))).astype(np.uint32)
    pa, pb = _lpt_plan(row, R, W), _lpt_plan(row2, R, W)
    ma, mb = _dense(pa, K, R), _dense(pb, K, R)
    both = ma.any(1) & mb.any(1)
    expect = (int((ma & mb).sum()), int(both.sum()), int((both & (ma.sum(1) != mb.sum(1))).sum()),
              int((both & (ma == mb).all(1)).sum()))
    assert replan.plan_churn(pa, pb) == expect
    assert replan.plan_churn(pb, pa) == expect  # symmetric
    assert replan.plan_churn(pa, pa) == (int(ma.sum()), len(pa["adm_keys"]), 0, len(pa["adm_keys"]))


def test_single_destination_churn_is_warm_set_overlap():
    # R = 1: every admitted key sits on destination 0, so the common pairs are the keys
    # admitted by both plans and no key can change its count or its set.
    rng = np.random.default_rng(3)
    row = rng.integers(0, 50, size=400).astype(np.uint32)
    row2 = rng.integers(0, 50, size=400).astype(np.uint32)
    pa, pb = _lpt_plan(row, 1, 60), _lpt_plan(row2, 1, 60)
    common_keys = np.intersect1d(pa["adm_keys"], pb["adm_keys"]).size
    assert replan.plan_churn(pa, pb) == (common_keys, common_keys, 0, common_keys)


def test_drift_generator_is_a_lognormal_walk():
    w = wl_mod.drift(n_per=20_000, steps=4, bins_per_interval=10)
    sh = w.meta["shares"]
    assert w.J == 4 and w.n == 80_000 and w.P == 4
    assert np.array_equal(w.offsets, np.arange(5, dtype=np.uint64) * 20_000)
    assert w.stat_offsets.shape == (41,) and w.stat_offsets[-1] == w.n and np.all(np.diff(w.stat_offsets) == 2000)
    base = np.sort(sh[0])[::-1]
    assert base[0] == pytest.approx(0.003, rel=1e-9)  # the 70B-like cap
    for t in range(1, 4):
        step = np.log(sh[t] / sh[t - 1])
        assert np.std(step) == pytest.approx(0.3, rel=0.03)  # sigma; the mean only renormalises
    # candidate 0 is fresh; candidate t keeps window t-1 during interval t only
    pw = w.plan_windows
    assert pw.tolist() == [[0, 0, 0, 0], [1, 0, 1, 1], [2, 2, 1, 2], [3, 3, 3, 2]]


def test_stale_candidate_shares_fresh_history_until_its_boundary():
    # Candidate t routes exactly as candidate 0 before interval t, so its statistics
    # agree bin for bin up to the boundary; at interval t it uses candidate 0's plan of
    # interval t-1 (same window, same parameters) and the statistics diverge.
    w = wl_mod.drift(n_per=6_000, steps=3, num_keys=400, R=5, W=8, bins_per_interval=6)
    r = opipe.run(w)
    off = w.offsets.astype(np.int64)
    for t in (1, 2):
        s = int(off[t])
        assert np.array_equal(r["dest"][t, :s], r["dest"][0, :s])
        assert np.array_equal(r["stats"][: 6 * t, t], r["stats"][: 6 * t, 0])
        assert r["win_of"][t][t] == t - 1 and r["win_of"][t][0] == t
        pl_stale, pl_prev = r["plans"][(t - 1, t)], r["plans"][(t - 1, 0)]
        for k in ("adm_keys", "member_off", "members"):
            assert np.array_equal(pl_stale[k], pl_prev[k])
    # every request is counted once per candidate, in its own bin
    assert np.all(r["stats"][..., 0].sum(axis=(0, 2)) == w.n)
    assert np.array_equal(r["stats"][..., 0].sum(axis=(1, 2)), np.diff(w.stat_offsets) * w.P)
