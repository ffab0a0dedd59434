"""End-to-end properties of the oracle's driver on the named shapes (CPU only)."""
import numpy as np

import oracle
from oracle import pipeline
from paper_2608_19677_amd import workload as wl


def test_tiny_plan_properties():
    w = wl.tiny()
    r = pipeline.run(w)
    pl = r["plans"][(0, 0)]
    n_w = w.n
    assert abs(pl["L"].sum() - n_w) <= 1e-12 * n_w               # planned loads sum to the window
    assert pl["adm_k"].sum() <= w.R * w.candidates[0].W
    # routing the window the plan was built from: cold requests are exactly the cold count
    adm = np.zeros(w.num_keys, bool)
    adm[pl["adm_keys"]] = True
    assert int((~adm[w.keys]).sum()) == pl["cold"]
    # admitted keys only ever reach their members
    dest = r["dest"][0]
    for a in range(0, len(pl["adm_keys"]), 37):
        b = pl["adm_keys"][a]
        m = set(pl["members"][pl["member_off"][a]:pl["member_off"][a + 1]].tolist())
        assert set(dest[w.keys == b].tolist()) <= m
    st = r["stats"].sum(axis=(0, 1, 2))
    assert st[0] == w.n


def test_plan_carried_from_previous_window():
    w = wl.small_random(5, num_keys=200, n=30_000, R=6, Ws=[5, 9], J=5)
    r = pipeline.run(w)
    assert [w[0] for w in r["win_of"]] == [0, 0, 1, 2, 3]
    counts = r["counts"]
    for (win, c), pl in r["plans"].items():
        n_w = int(counts[win].sum())
        assert abs(pl["L"].sum() - n_w) <= 1e-9 * max(1, n_w)


def test_replication_shape_whales_get_three_copies():
    # 8 injected keys at 6 % against q_cap = 0.4 x mean: ceil(2.4) = 3 copies each; the
    # background head (about 8.2 %) needs 4 and the next background key 2.
    w = wl.replication(n=120_000)
    counts, _ = oracle.count_rates(w.keys, w.offsets, w.num_keys)
    for j in range(w.J):
        row = counts[j]
        n_w = int(row.sum())
        keys, ks, cold, clamped = oracle.admit(row, w.R, 128, n_w, 2 * n_w, 5 * w.R)
        assert ks[:10].tolist() == [4] + [3] * 8 + [2]
        assert ks.sum() <= w.R * 128 and clamped == 0
