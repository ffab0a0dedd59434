"""Helpers for GPU-vs-oracle parity tests: run the device path through the C ABI and
the CPU oracle on the same seeded inputs and compare element by element."""
from __future__ import annotations

import sys

import numpy as np

import oracle
from oracle import pipeline as opipe

L_TOL = 1e-9  # absolute tolerance on planned loads; the design reproduces them bit for bit


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def compare_plan(gpl: dict, opl: dict, where: str):
    np.testing.assert_array_equal(gpl["adm_keys"], opl["adm_keys"], err_msg=f"{where}: admitted keys")
    np.testing.assert_array_equal(gpl["adm_k"], opl["adm_k"], err_msg=f"{where}: k")
    np.testing.assert_array_equal(gpl["member_off"], opl["member_off"], err_msg=f"{where}: member offsets")
    np.testing.assert_array_equal(gpl["members"], opl["members"], err_msg=f"{where}: members")
    assert gpl["cold"] == opl["cold"], where
    assert gpl["clamped"] == opl["clamped"], where
    assert np.max(np.abs(gpl["L"] - opl["L"]), initial=0.0) <= L_TOL, f"{where}: loads"
    assert np.array_equal(gpl["L"].view(np.uint64), opl["L"].view(np.uint64)), f"{where}: loads not bit-identical"


def compare_all(wl, gp, h: dict, orc: dict):
    """Full element-by-element comparison of a device pipeline run with the oracle's:
    every (plan group, candidate) the device routes with against the oracle's plan for
    the same interval and candidate."""
    assert h["err"] == 0, f"device error word {h['err']:#x}"
    np.testing.assert_array_equal(h["counts"], orc["counts"], err_msg="counts")
    seen = set()
    for j in range(wl.J):
        g = gp.gmap_host[j]
        for c in range(wl.P):
            if (g, c) in seen:
                continue
            seen.add((g, c))
            w = orc["win_of"][j][c]
            compare_plan(gp.plan_of(h, g, c), orc["plans"][(w, c)], f"interval {j} cand {c} (window {w})")
    np.testing.assert_array_equal(h["dest"], orc["dest"], err_msg="dest")
    np.testing.assert_array_equal(h["stats"], orc["stats"], err_msg="replay stats")
    for c, cand in enumerate(wl.candidates):
        np.testing.assert_array_equal(h["lru"][c, :, : cand.W], orc["lru"][c], err_msg=f"lru cand {c}")
        assert np.all(h["lru"][c, :, cand.W:] == oracle.EMPTY)
