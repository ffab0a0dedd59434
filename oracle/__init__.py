"""CPU oracle for the CacheRoute planner and shadow replay -- TEST INFRASTRUCTURE.

Thin ctypes wrapper over ``libcr_oracle.so`` (plain C, ``cr_oracle.c``) plus the
oracle's own driver (``pipeline.py``).  Only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may import
this package; the device path never does, and this package never imports the
device path.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Tuple

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "cr_oracle.c")
LIB = os.environ.get("CR_ORACLE_LIB") or os.path.join(HERE, "libcr_oracle.so")
EMPTY = 0xFFFFFFFF

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (no FMA contraction, IEEE double)."""
    if force or not os.path.exists(LIB):
        tmp = LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
                               "-Wall", "-Wextra", "-fPIC", "-shared", SRC, "-o", tmp])
        os.replace(tmp, LIB)
    return LIB


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build(force=True)
        L = ctypes.CDLL(LIB)
        P = ctypes.c_void_p
        u32, u64 = ctypes.c_uint32, ctypes.c_uint64
        L.cro_count_rates.argtypes = [P, u64, P, u32, u32, P, P]
        L.cro_kb.argtypes = [u32, u64, u64, u32, P]
        L.cro_kb.restype = u32
        L.cro_admit.argtypes = [P, u32, u32, u32, u64, u64, u64, P, P, P, P, P]
        L.cro_place_lpt.argtypes = [P, P, u32, P, u32, u64, P, P, P]
        L.cro_fmix32.argtypes = [u32]
        L.cro_fmix32.restype = u32
        L.cro_hash.argtypes = [u64, u64]
        L.cro_hash.restype = u32
        L.cro_route.argtypes = [P, u64, u64, u64, u32, u32, P, u32, P, P, P, P, P]
        L.cro_route_live.argtypes = [P, u64, u64, u64, u32, u32, P, u32, P, P, P, P]
        L.cro_place_u.argtypes = [u32, u32, u32]
        L.cro_place_u.restype = u32
        L.cro_place_hash.argtypes = [P, P, u32, P, u32, u64, u32, P, P, P]
        L.cro_replay.argtypes = [P, P, P, u32, P, u64, P, u32, u32, u32, P, P, P]
        for f in (L.cro_count_rates, L.cro_admit, L.cro_place_lpt, L.cro_place_hash, L.cro_route, L.cro_route_live,
                  L.cro_replay):
            f.restype = ctypes.c_int
        _lib = L
    return _lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=dtype)


def _check(rc: int, what: str):
    if rc != 0:
        raise ValueError(f"oracle {what} failed with status {rc}")


def count_rates(keys, offsets, K: int) -> Tuple[np.ndarray, int]:
    keys = _c(keys, np.uint32)
    offsets = _c(offsets, np.uint64)
    J = offsets.shape[0] - 1
    counts = np.zeros((J, K), dtype=np.uint32)
    bad = np.zeros(1, dtype=np.uint64)
    _check(lib().cro_count_rates(_p(keys), keys.shape[0], _p(offsets), J, K, _p(counts), _p(bad)), "count")
    return counts, int(bad[0])


def kb(c: int, q_num: int, q_den: int, R: int) -> int:
    return int(lib().cro_kb(c, q_num, q_den, R, None))


def admit(counts_row, R: int, W: int, n_window: int, q_num: int, q_den: int):
    """Returns (adm_keys, adm_k, cold, n_clamped)."""
    row = _c(counts_row, np.uint32)
    cap = R * W
    keys = np.zeros(cap, dtype=np.uint32)
    ks = np.zeros(cap, dtype=np.uint32)
    A = np.zeros(1, dtype=np.uint32)
    cold = np.zeros(1, dtype=np.uint64)
    clamped = np.zeros(1, dtype=np.uint32)
    _check(lib().cro_admit(_p(row), row.shape[0], R, W, n_window, q_num, q_den, _p(keys), _p(ks),
                           _p(A), _p(cold), _p(clamped)), "admit")
    a = int(A[0])
    return keys[:a].copy(), ks[:a].copy(), int(cold[0]), int(clamped[0])


def place_lpt(adm_keys, adm_k, counts_row, R: int, cold: int):
    """Returns (members uint16[sum k], member_off uint32[A+1], L float64[R])."""
    adm_keys = _c(adm_keys, np.uint32)
    adm_k = _c(adm_k, np.uint32)
    row = _c(counts_row, np.uint32)
    A = adm_keys.shape[0]
    members = np.zeros(max(1, int(adm_k.sum())), dtype=np.uint16)
    off = np.zeros(A + 1, dtype=np.uint32)
    L = np.zeros(R, dtype=np.float64)
    _check(lib().cro_place_lpt(_p(adm_keys), _p(adm_k), A, _p(row), R, cold, _p(members), _p(off), _p(L)),
           "place_lpt")
    return members[: int(off[A])].copy(), off, L


def admit_affinity(counts_row, R: int, W: int, n_window: int):
    """Admission of the ablation's affinity stage (Section 5.2): every key takes one slot,
    so the admitted keys are the first min(C, nnz) nonzero keys by (count desc, key asc).
    Returns (adm_keys, adm_k, cold)."""
    row = np.asarray(counts_row, dtype=np.int64)
    nz = np.nonzero(row)[0]
    order = nz[np.lexsort((nz, -row[nz]))]
    adm = order[: R * W].astype(np.uint32)
    cold = int(n_window) - int(row[adm].sum())
    return adm, np.ones(adm.shape[0], dtype=np.uint32), cold


def place_u(seed: int, b: int, r: int) -> int:
    return int(lib().cro_place_u(seed & 0xFFFFFFFF, b & 0xFFFFFFFF, r & 0xFFFFFFFF))


def place_hash(adm_keys, adm_k, counts_row, R: int, cold: int, seed: int):
    """Hash placement (ablation): returns (members, member_off, L) like place_lpt."""
    adm_keys = _c(adm_keys, np.uint32)
    adm_k = _c(adm_k, np.uint32)
    row = _c(counts_row, np.uint32)
    A = adm_keys.shape[0]
    members = np.zeros(max(1, int(adm_k.sum())), dtype=np.uint16)
    off = np.zeros(A + 1, dtype=np.uint32)
    L = np.zeros(R, dtype=np.float64)
    _check(lib().cro_place_hash(_p(adm_keys), _p(adm_k), A, _p(row), R, cold, seed & 0xFFFFFFFF, _p(members),
                                _p(off), _p(L)), "place_hash")
    return members[: int(off[A])].copy(), off, L


def fmix32(x: int) -> int:
    return int(lib().cro_fmix32(x & 0xFFFFFFFF))


def hash_(seed: int, i: int) -> int:
    return int(lib().cro_hash(seed, i))


def route(keys, first_index: int, seed: int, K: int, R: int, adm_keys, member_off, members, L):
    keys = _c(keys, np.uint32)
    adm_keys = _c(adm_keys, np.uint32)
    member_off = _c(member_off, np.uint32)
    members = _c(members if len(members) else np.zeros(1), np.uint16)
    L = _c(L, np.float64)
    dest = np.zeros(keys.shape[0], dtype=np.uint16)
    bad = np.zeros(1, dtype=np.uint64)
    _check(lib().cro_route(_p(keys), keys.shape[0], first_index, seed, K, R, _p(adm_keys),
                           adm_keys.shape[0], _p(member_off), _p(members), _p(L), _p(dest), _p(bad)),
           "route")
    return dest


def route_live(keys, first_index: int, seed: int, K: int, R: int, adm_keys, member_off, members):
    """Live-load dispatch of ONE control interval (loads start at zero)."""
    keys = _c(keys, np.uint32)
    adm_keys = _c(adm_keys, np.uint32)
    member_off = _c(member_off, np.uint32)
    members = _c(members if len(members) else np.zeros(1), np.uint16)
    dest = np.zeros(keys.shape[0], dtype=np.uint16)
    bad = np.zeros(1, dtype=np.uint64)
    _check(lib().cro_route_live(_p(keys), keys.shape[0], first_index, seed, K, R, _p(adm_keys),
                                adm_keys.shape[0], _p(member_off), _p(members), _p(dest), _p(bad)), "route_live")
    return dest


def replay(keys, suffix, prefix_len, dest, offsets, R: int, W: int, lru: Optional[np.ndarray] = None):
    """Returns (stats uint64[J][R][4], lru uint32[R][W]); ``lru`` is carried state (MRU first)."""
    keys = _c(keys, np.uint32)
    suffix = _c(suffix, np.uint16)
    plen = _c(prefix_len, np.uint32)
    dest = _c(dest, np.uint16)
    offsets = _c(offsets, np.uint64)
    J = offsets.shape[0] - 1
    state = np.full((R, W), EMPTY, dtype=np.uint32) if lru is None else _c(lru, np.uint32).copy()
    stats = np.zeros((J, R, 4), dtype=np.uint64)
    bad = np.zeros(1, dtype=np.uint64)
    _check(lib().cro_replay(_p(keys), _p(suffix), _p(plen), plen.shape[0], _p(dest), keys.shape[0],
                            _p(offsets), J, R, W, _p(state), _p(stats), _p(bad)), "replay")
    return stats, state
