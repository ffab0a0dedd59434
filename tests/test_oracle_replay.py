"""Pins for the oracle's LRU prefix-slot shadow replay (Section 3.2 shared cache), CPU only."""
import numpy as np
from hypothesis import given, settings, strategies as st

import oracle

EMPTY = oracle.EMPTY


def _stream(seed, n, K, R, zipf=1.0):
    rng = np.random.default_rng(seed)
    p = np.arange(1, K + 1, dtype=float) ** -zipf
    keys = rng.choice(K, size=n, p=p / p.sum()).astype(np.uint32)
    dest = rng.integers(0, R, size=n).astype(np.uint16)
    suffix = rng.integers(50, 401, size=n).astype(np.uint16)
    plen = rng.integers(1, 5000, size=K).astype(np.uint32)
    return keys, dest, suffix, plen


def _one(n):
    return np.array([0, n], np.uint64)


def _mattson_hits(keys, dest, W):
    """Brute force: request i hits iff its key was used at the same destination before and
    fewer than W distinct keys were used there since (LRU stack distance < W)."""
    hit = np.zeros(len(keys), bool)
    for i in range(len(keys)):
        d, b = dest[i], keys[i]
        seen = set()
        for t in range(i - 1, -1, -1):
            if dest[t] != d:
                continue
            if keys[t] == b:
                hit[i] = len(seen) < W
                break
            seen.add(int(keys[t]))
    return hit


@settings(max_examples=40, deadline=None)
@given(seed=st.integers(0, 10**6), n=st.integers(1, 300), K=st.integers(1, 25), R=st.integers(1, 4))
def test_replay_matches_stack_distance_brute_force(seed, n, K, R):
    keys, dest, suffix, plen = _stream(seed, n, K, R)
    prev = None
    for W in range(1, 9):
        stats, _ = oracle.replay(keys, suffix, plen, dest, _one(n), R, W)
        hit = _mattson_hits(keys, dest, W)
        for d in range(R):
            sel = dest == d
            s = stats[0, d]
            assert s[0] == sel.sum()
            assert s[1] == (hit & sel).sum()
            assert s[3] == plen[keys[hit & sel]].sum()
            assert s[2] == suffix[sel].sum(dtype=np.uint64) + plen[keys[~hit & sel]].sum(dtype=np.uint64)
        tot = stats[0, :, 1].sum()
        if prev is not None:
            assert tot >= prev  # LRU inclusion: hits never drop as W grows
        prev = tot


def test_replay_unbounded_slots_closed_form():
    keys, dest, suffix, plen = _stream(1, 20_000, 300, 7)
    stats, _ = oracle.replay(keys, suffix, plen, dest, _one(len(keys)), 7, 400)
    pairs = set(zip(dest.tolist(), keys.tolist()))
    assert stats[0, :, 1].sum() == len(keys) - len(pairs)
    want_prefill = int(suffix.sum(dtype=np.uint64)) + sum(int(plen[b]) for _, b in pairs)
    assert stats[0, :, 2].sum() == want_prefill


def test_replay_single_key_single_destination():
    n = 1000
    stats, state = oracle.replay(np.zeros(n, np.uint32), np.full(n, 60, np.uint16),
                                 np.array([777], np.uint32), np.zeros(n, np.uint16), _one(n), 1, 3)
    assert stats[0, 0, 1] == n - 1
    assert stats[0, 0, 2] == 60 * n + 777
    assert state[0].tolist() == [0, EMPTY, EMPTY]


def test_replay_one_slot_hits_on_repeat():
    keys, dest, suffix, plen = _stream(4, 5000, 6, 3)
    stats, _ = oracle.replay(keys, suffix, plen, dest, _one(len(keys)), 3, 1)
    hits = 0
    last = {}
    for b, d in zip(keys.tolist(), dest.tolist()):
        hits += last.get(d) == b
        last[d] = b
    assert stats[0, :, 1].sum() == hits


def test_replay_carried_state_equals_uninterrupted():
    keys, dest, suffix, plen = _stream(7, 30_000, 500, 5, zipf=0.9)
    n = len(keys)
    off = np.array([0, 9000, 9000, 21000, n], np.uint64)
    full, st_full = oracle.replay(keys, suffix, plen, dest, off, 5, 16)
    cut = 17_345
    a, st_a = oracle.replay(keys[:cut], suffix[:cut], plen, dest[:cut], np.array([0, 9000, 9000, cut], np.uint64), 5, 16)
    b, st_b = oracle.replay(keys[cut:], suffix[cut:], plen, dest[cut:], np.array([0, 21000 - cut, n - cut], np.uint64), 5, 16, st_a)
    assert np.array_equal(st_b, st_full)
    assert np.array_equal(full[:2], a[:2])
    assert np.array_equal(full[2], a[2] + b[0])
    assert np.array_equal(full[3], b[1])
    assert full[1].sum() == 0  # empty interval


def test_replay_final_state_is_most_recent_distinct_keys():
    keys, dest, suffix, plen = _stream(8, 3000, 50, 3)
    _, state = oracle.replay(keys, suffix, plen, dest, _one(len(keys)), 3, 6)
    for d in range(3):
        seq = keys[dest == d][::-1]
        want = []
        for b in seq.tolist():
            if b not in want:
                want.append(b)
            if len(want) == 6:
                break
        assert state[d, :len(want)].tolist() == want
