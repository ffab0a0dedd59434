"""Pins for the opaque-key remap (Appendix A.2 "Data handling": b may be salted or
ephemeral), CPU only: dense index = rank of the id's first occurrence."""
import numpy as np
import pytest

from oracle import keymap
from oracle import count_rates
from paper_2608_19677_amd import workload as wl_mod


@pytest.mark.parametrize("seed", range(5))
def test_dense_index_is_rank_of_first_occurrence(seed):
    # against numpy.unique: the distinct ids sorted by their first index get 0, 1, 2, ...
    rng = np.random.default_rng(seed)
    pool = rng.integers(0, 2**32 - 1, size=300, dtype=np.uint64).astype(np.uint32)
    ids = pool[rng.zipf(1.3, size=5000) % 300]
    dense, d = keymap.remap(ids)
    uniq, first = np.unique(ids, return_index=True)
    order = uniq[np.argsort(first)]
    assert [d[int(x)] for x in order] == list(range(len(order)))
    assert np.array_equal(dense, np.array([d[int(x)] for x in ids], dtype=np.uint32))
    # first occurrences appear in increasing dense order along the stream
    firsts = dense[np.sort(first)]
    assert np.array_equal(firsts, np.arange(len(order), dtype=np.uint32))


def test_reserved_and_unknown_ids():
    ids = np.array([7, 0xFFFFFFFF, 9, 7, 0xFFFFFFFF], dtype=np.uint32)
    dense, d = keymap.remap(ids)
    assert d == {7: 0, 9: 1}
    assert dense.tolist() == [0, keymap.NO_KEY, 1, 0, keymap.NO_KEY]
    assert keymap.lookup(d, [5, 9]).tolist() == [keymap.NO_KEY, 1]


def test_scatter_by_id():
    d = {40: 1, 10: 0, 30: 2}
    out = keymap.scatter(d, [30, 99, 10, 40], [300, 999, 100, 400], 4, fill=7)
    assert out.tolist() == [100, 400, 300, 7]


def test_salted_ids_are_distinct_and_counts_relabel():
    # the salted ids of distinct keys are distinct, and counting the remapped stream gives
    # the dense stream's counts with the columns relabelled by first appearance
    wl = wl_mod.small_random(3, num_keys=500, n=40_000, R=8, Ws=[8], J=4)
    op = wl_mod.opaque(wl)
    assert len(np.unique(op.attr_ids)) == wl.num_keys and not np.any(op.attr_ids == 0xFFFFFFFF)
    dense, d = keymap.remap(op.ids)
    c_dense, _ = count_rates(wl.keys, wl.offsets, wl.num_keys)
    c_remap, _ = count_rates(dense, wl.offsets, wl.num_keys)
    for b in np.unique(wl.keys).tolist():
        assert np.array_equal(c_remap[:, d[int(op.attr_ids[b])]], c_dense[:, b])
    plen = keymap.scatter(d, op.attr_ids, op.prefix_by_id, wl.num_keys)
    for b in np.unique(wl.keys).tolist():
        assert plen[d[int(op.attr_ids[b])]] == wl.prefix_len[b]
