"""Pins for the oracle's live-load dispatch (Section 3.1 "Placement and dispatch": the
least-loaded member of T(b) for admitted keys, power of two choices for the rest, on the
running per-destination loads of the interval) and the Gamma arrivals, CPU only."""
import numpy as np
import pytest

import oracle
from oracle import pipeline as opipe
from paper_2608_19677_amd import workload as wl_mod


def _plan(assign):
    keys = list(assign)
    off = np.concatenate([[0], np.cumsum([len(assign[b]) for b in keys])]).astype(np.uint32)
    mem = np.array([r for b in keys for r in assign[b]], dtype=np.uint16)
    return np.array(keys, dtype=np.uint32), off, mem


def test_all_destinations_as_members_is_round_robin():
    # one key replicated on every destination (members listed in any order): equal loads
    # tie to the lowest index, so the requests go 0, 1, ..., R-1, 0, 1, ...
    R = 7
    adm, off, mem = _plan({3: [4, 0, 6, 2, 1, 5, 3]})
    keys = np.full(50, 3, dtype=np.uint32)
    d = oracle.route_live(keys, 0, 1, 10, R, adm, off, mem)
    assert d.tolist() == [i % R for i in range(50)]


def test_single_copy_keys_always_go_to_their_member():
    adm, off, mem = _plan({1: [5], 2: [0]})
    keys = np.array([1, 2, 1, 1, 2, 1], dtype=np.uint32)
    d = oracle.route_live(keys, 0, 1, 10, 8, adm, off, mem)
    assert d.tolist() == [5, 0, 5, 5, 0, 5]


def test_one_destination():
    rng = np.random.default_rng(0)
    keys = rng.integers(0, 50, size=300).astype(np.uint32)
    adm, off, mem = _plan({3: [0], 9: [0]})
    assert np.all(oracle.route_live(keys, 0, 4, 50, 1, adm, off, mem) == 0)


def test_two_members_alternate_by_load():
    # members {2, 5}: the first request ties (lowest index 2), then each goes to the member
    # with fewer requests so far; single-copy traffic to 5 shifts the balance
    adm, off, mem = _plan({7: [5, 2], 8: [5]})
    keys = np.array([7, 7, 8, 8, 7, 7, 7], dtype=np.uint32)
    d = oracle.route_live(keys, 0, 1, 10, 6, adm, off, mem)
    # loads (2, 5): (0,0) -> 2; (1,0) -> 5; 8 -> 5 (1,2); 8 -> 5 (1,3); (1,3) -> 2;
    # (2,3) -> 2; (3,3) -> 2
    assert d.tolist() == [2, 5, 5, 5, 2, 2, 2]


def _check_decisions(keys, dest, R, adm, off, mem, h_of):
    """Every decision follows from the requests routed before it in the interval."""
    rank = {int(b): a for a, b in enumerate(adm)}
    load = np.zeros(R, dtype=np.int64)
    for i, (b, d) in enumerate(zip(keys.tolist(), dest.tolist())):
        if b in rank:
            a = rank[b]
            m = [int(x) for x in mem[off[a]:off[a + 1]]]
            best = min(m, key=lambda r: (load[r], r))
            assert d == best, i
        else:
            h = h_of(i)
            d1, d2 = ((h & 0xFFFF) * R) >> 16, ((h >> 16) * R) >> 16
            assert d in (d1, d2) and load[d] == min(load[d1], load[d2]), i
            if load[d1] == load[d2]:
                assert d == d1, i
        load[d] += 1


@pytest.mark.parametrize("seed", range(4))
def test_each_decision_is_least_loaded_at_its_time(seed):
    rng = np.random.default_rng(seed)
    K, R, n = 200, 9, 3000
    keys = rng.integers(0, K + 5, size=n).astype(np.uint32)  # a few keys out of range: cold
    adm_keys = rng.choice(K, size=40, replace=False)
    assign = {int(b): sorted(rng.choice(R, size=int(rng.integers(1, 4)), replace=False).tolist(),
                             key=lambda _: rng.random()) for b in adm_keys}
    adm, off, mem = _plan(assign)
    first, s = 1000, 77
    dest = oracle.route_live(keys, first, s, K, R, adm, off, mem)
    _check_decisions(keys, dest, R, adm, off, mem, lambda i: oracle.hash_(s, first + i))


def test_loads_restart_every_interval():
    # the oracle driver dispatches each interval from zero loads: interval j's destinations
    # equal a fresh call over that interval alone
    w = wl_mod.small_random(4, num_keys=300, n=20_000, R=12, Ws=[8], J=4, hot=3, hot_share=0.6)
    r = opipe.run(w, dispatch="live")
    off = w.offsets.astype(np.int64)
    for j in range(w.J):
        s, e = int(off[j]), int(off[j + 1])
        pl = r["plans"][(r["win_of"][j][0], 0)]
        alone = oracle.route_live(w.keys[s:e], w.first_index + s, w.seed, w.num_keys, w.R, pl["adm_keys"],
                                  pl["member_off"], pl["members"])
        assert np.array_equal(r["dest"][0, s:e], alone)
        _check_decisions(w.keys[s:e], alone, w.R, pl["adm_keys"], pl["member_off"], pl["members"],
                         lambda i, s=s: oracle.hash_(w.seed, w.first_index + s + i))


def test_live_power_of_two_balances_better_than_static_hashing():
    # cold-only traffic: the running-load choice keeps destinations within a few requests
    # of each other, plain hashing does not
    rng = np.random.default_rng(9)
    n, R = 20_000, 16
    keys = rng.integers(0, 1000, size=n).astype(np.uint32)
    empty = (np.zeros(0, np.uint32), np.zeros(1, np.uint32), np.zeros(0, np.uint16))
    live = np.bincount(oracle.route_live(keys, 0, 3, 1000, R, *empty), minlength=R)
    stat = np.bincount(oracle.route(keys, 0, 3, 1000, R, *empty, np.zeros(R)), minlength=R)
    assert live.max() - live.min() <= 3
    assert stat.max() - stat.min() > 3 * (live.max() - live.min())


def test_gamma_arrivals_have_the_requested_cv():
    rng = np.random.default_rng(1)
    gaps_cv = []
    for cv in (1.0, 1.9, 3.0):
        g = rng.gamma(1.0 / (cv * cv), (cv * cv) / 176.0, size=400_000)
        gaps_cv.append(g.std() / g.mean())
        assert g.mean() == pytest.approx(1 / 176.0, rel=0.02)
    assert gaps_cv == pytest.approx([1.0, 1.9, 3.0], rel=0.03)
    a, b = wl_mod.llama70b(n=300_000), wl_mod.llama70b_gamma(n=300_000)
    assert np.array_equal(a.keys, b.keys) and not np.array_equal(a.offsets, b.offsets)
    # counts per 60-s interval vary more under bursty arrivals (renewal process: the count
    # variance grows with CV^2)
    va = np.diff(a.offsets.astype(np.int64))[:-1].var()
    vb = np.diff(b.offsets.astype(np.int64))[:-1].var()
    assert vb > 2 * va
