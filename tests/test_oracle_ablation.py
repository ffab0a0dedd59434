"""Pins for the component-ablation plan variants (Section 5.2, 8B component ablation table),
CPU only: affinity admission, hash placement, and the flat plan."""
import itertools

import numpy as np
import pytest
from scipy import stats as sps

import oracle
from oracle import pipeline as opipe
from paper_2608_19677_amd import workload as wl_mod


def test_place_u_is_a_permutation_of_destinations():
    # for a fixed key, u(b, .) is a bijection of 32-bit destinations: no ties among any R
    for seed, b in ((0, 0), (7, 12345), (3, 2**31 + 5)):
        us = [oracle.place_u(seed, b, r) for r in range(4096)]
        assert len(set(us)) == len(us)


def _members(b, k, R, seed, c=10):
    row = np.zeros(b + 1, dtype=np.uint32)
    row[b] = c
    mem, off, L = oracle.place_hash([b], [k], row, R, 0, seed)
    return mem[off[0]:off[1]].tolist(), L


def test_hash_members_are_the_k_smallest_hashes():
    # brute force over every destination: the k members are the k smallest (u, r), in order
    for b, k, R in ((3, 1, 7), (11, 4, 9), (100, 9, 9), (5, 1, 1), (42, 30, 64)):
        mem, _ = _members(b, k, R, seed=7)
        ranked = sorted(range(R), key=lambda r: (oracle.place_u(7, b, r), r))
        assert mem == ranked[:k]


def test_hash_members_do_not_depend_on_loads_or_counts():
    a, _ = _members(17, 3, 12, seed=7, c=5)
    b, _ = _members(17, 3, 12, seed=7, c=5000)
    assert a == b
    row = np.zeros(30, dtype=np.uint32)
    row[17], row[3] = 5, 999
    mem, off, _ = oracle.place_hash([3, 17], [2, 3], row, 12, 10_000, 7)  # another key placed first
    assert mem[off[1]:off[2]].tolist() == a


def test_single_copy_placement_is_uniform():
    # k = 1 over 40,000 keys and 16 destinations: chi-square against uniform
    R, n = 16, 40_000
    keys = np.arange(n, dtype=np.uint32)
    row = np.ones(n, dtype=np.uint32)
    mem, _, _ = oracle.place_hash(keys, np.ones(n, np.uint32), row, R, 0, 11)
    obs = np.bincount(mem, minlength=R)
    assert sps.chisquare(obs).pvalue > 1e-3


def test_pair_placement_is_uniform_over_pairs():
    # k = 2 over 6 destinations: all 15 unordered pairs equally likely
    R, n = 6, 30_000
    keys = np.arange(n, dtype=np.uint32)
    mem, off, _ = oracle.place_hash(keys, np.full(n, 2, np.uint32), np.ones(n, np.uint32), R, 0, 5)
    pairs = {p: 0 for p in itertools.combinations(range(R), 2)}
    for a in range(n):
        pairs[tuple(sorted(mem[off[a]:off[a + 1]].tolist()))] += 1
    assert sps.chisquare(list(pairs.values())).pvalue > 1e-3


def test_hash_placement_loads():
    # L = cold / R + sum of c / k over the keys placed on r, in admission order; every key's
    # k members are distinct; the loads sum to the window
    rng = np.random.default_rng(4)
    K, R = 200, 9
    row = rng.integers(1, 500, size=K).astype(np.uint32)
    keys = rng.permutation(K).astype(np.uint32)[:120]
    ks = rng.integers(1, R + 1, size=120).astype(np.uint32)
    cold = 777
    mem, off, L = oracle.place_hash(keys, ks, row, R, cold, 3)
    ref = np.full(R, cold / R)
    for a, b in enumerate(keys):
        m = mem[off[a]:off[a + 1]]
        assert len(set(m.tolist())) == ks[a]
        for r in m:
            ref[r] = ref[r] + row[b] / ks[a]
    assert np.array_equal(L, ref)  # same additions in the same order
    assert L.sum() == pytest.approx(cold + int(row[keys].sum()), rel=1e-12)
    # k = R takes every destination, R = 1 only destination 0
    m_all, _ = _members(9, 9, 9, seed=1)
    assert sorted(m_all) == list(range(9))
    assert _members(9, 1, 1, seed=1)[0] == [0]


def test_affinity_admission_is_top_C_and_the_k1_case_of_eq1():
    # one slot per key: the first min(C, nnz) keys by (count desc, key asc); it equals Eq. 1
    # admission whenever q_cap is at least the largest count (every k = 1)
    rng = np.random.default_rng(8)
    for trial in range(20):
        K, R, W = 300, int(rng.integers(1, 9)), int(rng.integers(1, 40))
        row = (rng.integers(0, 6, size=K) * rng.integers(0, 2, size=K)).astype(np.uint32)
        n_w = int(row.sum())
        adm, ks, cold = oracle.admit_affinity(row, R, W, n_w)
        nz = [b for b in range(K) if row[b]]
        nz.sort(key=lambda b: (-int(row[b]), b))
        assert adm.tolist() == nz[: R * W] and np.all(ks == 1)
        assert cold == n_w - int(row[adm].sum())
        if n_w:
            a2, k2, cold2, _ = oracle.admit(row, R, W, n_w, int(row.max()) * R, R)
            assert np.array_equal(a2, adm) and np.all(k2 == 1) and cold2 == cold


def test_flat_plan_is_plain_hashing():
    # the flat plan admits nothing and has uniform loads, so power of two choices always ties
    # and keeps the first draw d1 = ((h & 0xFFFF) * R) >> 16
    w = wl_mod.small_random(3, num_keys=300, n=20_000, R=11, Ws=[8], J=3)
    w.candidates = [wl_mod.Candidate(8, variant="flat")]
    r = opipe.run(w)
    for pl in r["plans"].values():
        assert len(pl["adm_keys"]) == 0 and pl["cold"] == pl["n_window"]
        assert np.all(pl["L"] == pl["L"][0])
    h = np.array([oracle.hash_(w.seed, w.first_index + i) for i in range(w.n)], dtype=np.uint64)
    assert np.array_equal(r["dest"][0], ((h & 0xFFFF) * w.R) >> 16)


def test_ablation_stages_share_admission():
    # replicated and full admit the same keys with the same k (Eq. 1) and differ only in
    # placement; affinity admits at least as many keys, all with k = 1; hash placement puts a
    # key on the same destinations in every window
    w = wl_mod.ablation(n=300_000)
    r = opipe.run(w)
    for (win, c), pl in r["plans"].items():
        if c == 2:
            full = r["plans"][(win, 3)]
            assert np.array_equal(pl["adm_keys"], full["adm_keys"]) and np.array_equal(pl["adm_k"], full["adm_k"])
        if c == 1:
            assert np.all(pl["adm_k"] == 1) and len(pl["adm_keys"]) >= len(r["plans"][(win, 3)]["adm_keys"])
    p0, p1 = r["plans"][(0, 1)], r["plans"][(1, 1)]
    common = np.intersect1d(p0["adm_keys"], p1["adm_keys"])
    m0 = dict(zip(p0["adm_keys"].tolist(), p0["members"].tolist()))
    m1 = dict(zip(p1["adm_keys"].tolist(), p1["members"].tolist()))
    assert common.size > 100 and all(m0[b] == m1[b] for b in common.tolist())
