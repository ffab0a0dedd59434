"""Pins for the oracle's counter-based hash and its dispatch rule (CPU only)."""
import os

import numpy as np
import pytest

import oracle

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _rotl(x, r):
    return ((x << r) | (x >> (32 - r))) & 0xFFFFFFFF


def _murmur3_with_oracle_finalizer(data: bytes, seed: int) -> int:
    """MurmurHash3_x86_32 body; the final avalanche step is the ORACLE's fmix32."""
    c1, c2 = 0xCC9E2D51, 0x1B873593
    h = seed & 0xFFFFFFFF
    nb = len(data) // 4
    for i in range(nb):
        k = int.from_bytes(data[4 * i:4 * i + 4], "little")
        k = _rotl((k * c1) & 0xFFFFFFFF, 15)
        k = (k * c2) & 0xFFFFFFFF
        h = _rotl(h ^ k, 13)
        h = (h * 5 + 0xE6546B64) & 0xFFFFFFFF
    tail = data[4 * nb:]
    k = 0
    if len(tail) >= 3:
        k ^= tail[2] << 16
    if len(tail) >= 2:
        k ^= tail[1] << 8
    if len(tail) >= 1:
        k ^= tail[0]
        k = _rotl((k * c1) & 0xFFFFFFFF, 15)
        h ^= (k * c2) & 0xFFFFFFFF
    return oracle.fmix32(h ^ len(data))


def _rows(name):
    with open(os.path.join(GOLD, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                yield line.split()


def test_fmix32_against_published_murmur3_vectors():
    n = 0
    for data, seed, want in _rows("murmur3_x86_32.txt"):
        b = b"" if data == "-" else bytes.fromhex(data)
        assert _murmur3_with_oracle_finalizer(b, int(seed, 16)) == int(want, 16), (data, seed)
        n += 1
    assert n >= 10


def test_hash_golden_vectors():
    for seed, i, want in _rows("hash_vectors.txt"):
        assert oracle.hash_(int(seed), int(i)) == int(want, 16)


def test_hash_inner_term_constant_below_2_32():
    # The high word of the index only enters through the inner term.
    assert oracle.hash_(1, 5) != oracle.hash_(1, 5 + (1 << 32))
    assert oracle.hash_(3, 0) != oracle.hash_(3 + (1 << 32), 0)


def _plan(adm_keys, ks, R, L):
    off = np.concatenate([[0], np.cumsum(ks)]).astype(np.uint32)
    members = np.zeros(int(off[-1]), dtype=np.uint16)
    for a, k in enumerate(ks):  # arbitrary distinct members for routing-only tests
        members[off[a]:off[a + 1]] = (np.arange(k) * 3 + a) % R
    return np.asarray(adm_keys, np.uint32), off, members, np.asarray(L, np.float64)


def test_empty_plan_routes_to_first_draw_uniformly():
    # Equal loads: every comparison ties, so dest = d1 = ((h & 0xFFFF) * R) >> 16.
    R, n = 16, 200_000
    keys = np.zeros(n, np.uint32)
    ak, off, mem, L = _plan([], [], R, np.full(R, 7.0))
    dest = oracle.route(keys, 0, 1, 4, R, ak, off, mem, L)
    h = np.array([oracle.hash_(1, i) for i in range(2000)], dtype=np.uint64)
    d1 = ((h & 0xFFFF) * R) >> 16
    assert np.array_equal(dest[:2000], d1.astype(np.uint16))
    cnt = np.bincount(dest, minlength=R)
    chi2 = ((cnt - n / R) ** 2 / (n / R)).sum()
    assert chi2 < 45.0  # 15 dof, p ~ 1e-4


def test_p2c_rank_distribution():
    # Strictly ordered loads: P(dest has load rank j) = (2(R-j)-1)/R^2 (two draws with replacement).
    R, n = 16, 400_000
    order = np.random.default_rng(5).permutation(R)
    L = np.empty(R)
    L[order] = np.arange(R) * 1.5 + 1.0  # order[j] has the j-th smallest load
    ak, off, mem, _ = _plan([], [], R, L)
    dest = oracle.route(np.zeros(n, np.uint32), 0, 9, 4, R, ak, off, mem, L)
    cnt = np.bincount(dest, minlength=R)[order]
    p = np.array([(2 * (R - j) - 1) / R ** 2 for j in range(R)])
    chi2 = ((cnt - n * p) ** 2 / (n * p)).sum()
    assert chi2 < 45.0


def test_admitted_requests_land_in_their_member_set():
    R, K = 12, 40
    rng = np.random.default_rng(3)
    ak = np.array([5, 17, 2, 30], np.uint32)
    ks = [1, 3, 12, 2]
    off = np.concatenate([[0], np.cumsum(ks)]).astype(np.uint32)
    mem = np.concatenate([rng.permutation(R)[:k] for k in ks]).astype(np.uint16)
    L = rng.random(R)
    keys = rng.integers(0, K, size=50_000).astype(np.uint32)
    dest = oracle.route(keys, 123, 77, K, R, ak, off, mem, L)
    for a, b in enumerate(ak):
        sel = keys == b
        allowed = set(mem[off[a]:off[a + 1]].tolist())
        assert set(dest[sel].tolist()) == allowed  # every member is used, nothing else
    # k = R: members are picked uniformly by the high hash half
    sel = keys == 2
    cnt = np.bincount(dest[sel], minlength=R)
    e = sel.sum() / R
    assert ((cnt - e) ** 2 / e).sum() < 40.0


def test_out_of_range_key_goes_cold():
    R = 8
    ak, off, mem, L = _plan([1], [1], R, np.arange(R, dtype=float))
    d_bad = oracle.route(np.array([99], np.uint32), 0, 1, 10, R, ak, off, mem, L)
    d_cold = oracle.route(np.array([3], np.uint32), 0, 1, 10, R, ak, off, mem, L)
    assert d_bad[0] == d_cold[0]


def test_dispatch_uses_the_documented_hash_bits():
    # From the golden H(1, 0) = 0xd5aad292: low half 0xd292, high half 0xd5aa.
    # R = 30: d1 = (0xd292 * 30) >> 16 = 24, d2 = (0xd5aa * 30) >> 16 = 25.
    # Admitted key with k = 30 members [0..29]: member index (0xd5aa * 30) >> 16 = 25;
    # with k = 7: (0xd5aa * 7) >> 16 = 5.
    R = 30
    h = 0xD5AAD292
    assert ((h & 0xFFFF) * R) >> 16 == 24 and ((h >> 16) * R) >> 16 == 25
    L_d2_wins = np.zeros(R)
    L_d2_wins[24] = 1.0
    ak, off, mem, _ = _plan([], [], R, L_d2_wins)
    assert oracle.route(np.array([3], np.uint32), 0, 1, 10, R, ak, off, mem, L_d2_wins)[0] == 25
    L_d1_wins = np.zeros(R)
    L_d1_wins[25] = 1.0
    assert oracle.route(np.array([3], np.uint32), 0, 1, 10, R, ak, off, mem, L_d1_wins)[0] == 24
    members = np.arange(100, 130, dtype=np.uint16) % R
    for k, want in ((30, 25), (7, 5)):
        offk = np.array([0, k], np.uint32)
        members_k = np.roll(np.arange(R, dtype=np.uint16), -3)[:k]
        d = oracle.route(np.array([3], np.uint32), 0, 1, 10, R, np.array([3], np.uint32), offk,
                         members_k, np.zeros(R))
        assert d[0] == members_k[want]
