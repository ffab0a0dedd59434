"""GPU parity for the component-ablation plan variants (Section 5.2, 8B component ablation
table): flat, affinity (k = 1, hash placement), replicated (Eq. 1, hash placement) and the
full method replayed as candidates of one stream, against the CPU oracle element by element."""
import numpy as np
import pytest

from oracle import pipeline as opipe
from paper_2608_19677_amd import workload as wl_mod
from paper_2608_19677_amd.pipeline import Pipeline
from paper_2608_19677_amd.report import ablation_summary

from cr_check import compare_all, say

pytestmark = pytest.mark.gpu

ALL = ("flat", "affinity", "replicated", "full")


def _run(wl):
    say(f"[case] {wl.name} n={wl.n} J={wl.J} K={wl.num_keys} R={wl.R} P={wl.P} "
        f"variants={[c.variant for c in wl.candidates]}")
    gp = Pipeline(wl)
    gp.step()
    h = gp.host()
    orc = opipe.run(wl)
    compare_all(wl, gp, h, orc)
    return gp, h, orc


def test_ablation_full_size_parity():
    # the injected-whale stream (2e7 requests, 667 intervals, 16 x 128 slots, q_cap = 0.4 x mean)
    # under the four stages: 2,664 plans
    gp, h, orc = _run(wl_mod.ablation())
    s = ablation_summary(gp.wl, h["stats"], h["load"], gp.gmap_host)
    rows = {r["variant"]: r for r in s["candidates"]}
    say(f"[ablation] {rows}")
    assert rows["flat"]["planned_imbalance"] == 1.0
    assert rows["affinity"]["planned_imbalance"] > rows["replicated"]["planned_imbalance"] > \
        rows["full"]["planned_imbalance"]
    assert rows["affinity"]["kv_hit"] > rows["flat"]["kv_hit"]


@pytest.mark.parametrize("case", [
    # seed, K, n, R, Ws, J, hot, hot_share, qs
    (1, 300, 40_000, 7, [8], 4, 3, 0.5, [(1, 1)]),
    (2, 2000, 60_000, 100, [4, 20], 3, 6, 0.6, [(1, 2)]),      # two lane slots per wavefront
    (3, 500, 30_000, 1, [40], 2, 0, 0.0, [(1, 1)]),              # one destination
    (4, 800, 50_000, 16, [2], 3, 2, 0.9, [(1, 20)]),             # k clamped to R
    (5, 5000, 80_000, 1024, [3], 2, 8, 0.5, [(1, 1)]),           # 16 lane slots
    (6, 60, 5_000, 30, [16], 5, 0, 0.0, [(1, 1)]),               # everything admitted
], ids=lambda c: f"a{c[0]}")
def test_variant_parity(case):
    seed, K, n, R, Ws, J, hot, share, qs = case
    wl = wl_mod.small_random(seed, num_keys=K, n=n, R=R, Ws=Ws, J=J, hot=hot, hot_share=share, qs=qs)
    base = wl.candidates
    wl.candidates = [wl_mod.Candidate(c.W, c.a, c.b, v, 11 + i) for c in base for i, v in enumerate(ALL)]
    _run(wl)
