"""GPU parity of the replay that keeps several small lists per wavefront (k_replay_grp).

Calls with one interval replay their candidates with W <= 16 slots by k_replay_grp (lane
groups of 8 lanes for W <= 8, 16 lanes for W <= 16, one segment each, initial state rebuilt
forward) once n times their number reaches a size threshold; these cases lower the
threshold to 0 so that they take that path, and restore it afterwards. The cases cover W from 1 to 16 next to larger lists in the same call, one
key and one destination, streams of many segments, streams with fewer distinct keys than W
(segments out of rebuild budget, replayed by the sequential pass), carried cache state
between chunks, out-of-range keys, and 1,024 destinations."""
import numpy as np
import pytest
import torch

from oracle import pipeline as opipe
from paper_2608_19677_amd import workload as wl_mod
from paper_2608_19677_amd.pipeline import Pipeline
from paper_2608_19677_amd import binding as B

from cr_check import compare_all, say

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def grouped_everywhere():
    B.cr_replay_set_group_min_records(0)
    yield
    B.cr_replay_set_group_min_records(B.GROUP_MIN_RECORDS_DEFAULT)

CASES = [
    # seed, K, n, R, Ws, hot, hot_share, qs
    (201, 50, 3000, 7, [4], 0, 0.0, [(1, 1)]),
    (202, 1, 5000, 1, [3], 0, 0.0, [(1, 1)]),
    (203, 200, 20_000, 30, [16, 9], 3, 0.5, [(1, 1), (2, 5)]),
    (204, 1000, 100_003, 64, [1, 2, 7, 8, 15, 16, 17, 64], 2, 0.3, [(1, 1)]),
    (205, 5000, 50_000, 1024, [8, 14], 4, 0.4, [(1, 1)]),
    (206, 300, 40_000, 65, [10], 0, 0.0, [(1, 1), (28, 35), (42, 35)]),
    (207, 100, 10, 30, [16], 0, 0.0, [(1, 1)]),
    (208, 400, 30_000, 4, [2, 5], 2, 0.9, [(1, 3)]),
    # long streams: every stream is many 1,024-record segments
    (209, 3000, 400_000, 8, [8, 14, 16], 2, 0.3, [(1, 1)]),
    # 12 keys over one destination with 13 to 16 slots: no rebuild finds W keys, every
    # segment from the third on goes to the sequential pass
    (210, 12, 200_000, 1, [13, 16], 0, 0.0, [(1, 1)]),
    # 30 keys over two destinations: budget exhausted in some segments only
    (211, 30, 300_000, 2, [8, 14], 2, 0.5, [(1, 1), (1, 2)]),
]


@pytest.mark.parametrize("case", CASES, ids=[f"g{c[0]}" for c in CASES])
def test_grouped_replay_parity(case):
    seed, K, n, R, Ws, hot, share, qs = case
    wl = wl_mod.small_random(seed, num_keys=K, n=n, R=R, Ws=Ws, J=1, hot=hot, hot_share=share, qs=qs)
    say(f"[case] grouped {wl.name} n={wl.n} K={wl.num_keys} R={wl.R} W={Ws}")
    gp = Pipeline(wl)
    gp.step()
    compare_all(wl, gp, gp.host(), opipe.run(wl))


def test_grouped_replay_out_of_range_keys():
    wl = wl_mod.small_random(212, num_keys=500, n=50_000, R=20, Ws=[6, 12, 40], J=1, hot=2, hot_share=0.3)
    keys = wl.keys.copy()
    rng = np.random.default_rng(5)
    keys[rng.integers(0, wl.n, size=300)] = wl.num_keys + 7
    wl.keys = keys
    say("[case] grouped lists with out-of-range keys")
    gp = Pipeline(wl)
    gp.step()
    h = gp.host()
    assert h["err"] & B.CR_ERR_KEY_RANGE
    orc = opipe.run(wl)
    np.testing.assert_array_equal(h["stats"], orc["stats"])
    for c, cand in enumerate(wl.candidates):
        np.testing.assert_array_equal(h["lru"][c, :, :cand.W], orc["lru"][c])


@pytest.mark.parametrize("cut", [170_003, 1_024 * 37])
def test_grouped_replay_carried_state(cut):
    # two chunks, the second starting from the first one's final cache state (with empty
    # slots where a stream saw fewer than W keys), equal the uninterrupted stream
    wl = wl_mod.small_random(213, num_keys=3000, n=300_000, R=40, Ws=[5, 16, 150], J=1, hot=2, hot_share=0.2)
    whole = Pipeline(wl)
    whole.step()
    hw = whole.host()

    def part(s, e, first):
        return wl_mod.Workload(name="part", num_keys=wl.num_keys, R=wl.R, candidates=wl.candidates,
                               keys=wl.keys[s:e], suffix=wl.suffix[s:e], prefix_len=wl.prefix_len,
                               offsets=np.array([0, e - s], dtype=np.uint64), seed=wl.seed, first_index=first)

    a, b = part(0, cut, 0), part(cut, wl.n, cut)
    say(f"[case] grouped lists, carried state at {cut}")
    pa = Pipeline(a)
    pa.step()
    pb = Pipeline(b, prev_counts=whole.counts[0].clone(), lru_in=pa.lru_out.clone())
    pb.step()
    torch.cuda.synchronize()
    hb = pb.host()
    orc_b = opipe.run(b, lru=[pa.host()["lru"][c, :, :cd.W] for c, cd in enumerate(b.candidates)],
                      counts_prev=hw["counts"][0])
    assert hb["err"] == 0
    np.testing.assert_array_equal(hb["stats"], orc_b["stats"])
    for c, cand in enumerate(b.candidates):
        np.testing.assert_array_equal(hb["lru"][c, :, :cand.W], orc_b["lru"][c])
