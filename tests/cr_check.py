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


def compare_all(wl, gp, h: dict, orc: dict, win_to_group=None):
    """Full element-by-element comparison of a device pipeline run with the oracle's."""
    assert h["err"] == 0, f"device error word {h['err']:#x}"
    np.testing.assert_array_equal(h["counts"], orc["counts"], err_msg="counts")
    for (w, c), opl in orc["plans"].items():
        g = w if win_to_group is None else win_to_group[w]
        compare_plan(gp.plan_of(h, g, c), opl, f"plan window {w} cand {c}")
    np.testing.assert_array_equal(h["dest"], orc["dest"], err_msg="dest")
    np.testing.assert_array_equal(h["stats"], orc["stats"], err_msg="replay stats")
    for c, cand in enumerate(wl.candidates):
        np.testing.assert_array_equal(h["lru"][c, :, : cand.W], orc["lru"][c], err_msg=f"lru cand {c}")
        assert np.all(h["lru"][c, :, cand.W:] == oracle.EMPTY)
