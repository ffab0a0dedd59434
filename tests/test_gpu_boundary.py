"""GPU tests of the boundary's helper calls through the C ABI: the one-slice count
(cr_count_slice) against the oracle's counting, cr_lru_reset, and plan specs given with an
absolute N_w against the relative form (CR_WINDOW_SUM) the pipeline uses."""
import numpy as np
import pytest
import torch

import oracle
from oracle import pipeline as opipe
from paper_2608_19677_amd import binding as B
from paper_2608_19677_amd import workload as wl_mod
from paper_2608_19677_amd.pipeline import Pipeline

from cr_check import compare_all, say

pytestmark = pytest.mark.gpu

SLICES = [
    # n, K, zipf s, offset of the keys in their buffer (4-byte words: misaligned tiles)
    (1, 7, 1.0, 0),
    (4095, 1000, 1.1, 0),            # one partial tile
    (4096 * 3 + 17, 33_000, 0.9, 1),  # two buckets, ragged tail, unaligned rows
    (1_000_000, 100_003, 0.9, 0),     # four buckets, the last one short
    (3_000_000, 1_000_000, 0.9, 0),   # the sweep's key space
    (2_000_000, 1 << 23, 0.5, 3),     # 256 buckets (the maximum)
]


@pytest.mark.parametrize("case", SLICES, ids=[f"n{c[0]}_K{c[1]}" for c in SLICES])
def test_count_slice_matches_oracle(case):
    n, K, s, shift = case
    say(f"[case] count slice n={n} K={K} shift={shift}")
    rng = np.random.default_rng(n ^ K)
    p = wl_mod.zipf_probs(min(K, 1 << 20), s)
    keys = (rng.permutation(K)[:p.shape[0]][wl_mod.CategoricalSampler(p).sample(rng, n)]).astype(np.uint32)
    keys[rng.integers(0, n, size=min(n, 5))] = np.uint32(K + 3)  # out of range: skipped, flagged
    buf = torch.zeros(n + 4, dtype=torch.int32, device="cuda")
    buf[shift:shift + n] = torch.from_numpy(keys.view(np.int32)).cuda()
    d_keys = buf[shift:shift + n]
    base = rng.integers(0, 5, size=K).astype(np.uint32)  # counts accumulate onto what is there
    counts = torch.from_numpy(base.view(np.int32)).cuda()
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = torch.empty(B.cr_count_slice_workspace_bytes(n, K), dtype=torch.uint8, device="cuda")
    B.cr_count_slice(d_keys, K, counts, err, ws, n=n)
    got = counts.cpu().numpy().view(np.uint32)
    want, nbad = oracle.count_rates(keys, np.array([0, n], np.uint64), K)
    np.testing.assert_array_equal(got, base + want[0])
    assert nbad > 0 and int(err.item()) & B.CR_ERR_KEY_RANGE
    # a second slice adds on
    err.zero_()
    B.cr_count_slice(d_keys, K, counts, err, ws, n=n)
    np.testing.assert_array_equal(counts.cpu().numpy().view(np.uint32), base + 2 * want[0])


def test_lru_reset():
    P, R, W = 3, 70, 40
    lru = torch.randint(0, 1000, (P, R, W), dtype=torch.int32, device="cuda")
    assert B.cr_lru_state_bytes(P, R, W) == lru.numel() * 4
    B.cr_lru_reset(lru, P, R, W)
    assert np.all(lru.cpu().numpy().view(np.uint32) == B.CR_EMPTY_SLOT)


def test_absolute_and_relative_targets_agree():
    # a spec with n_window = the window's request count and q = (a N_w, b R) builds the same
    # plans as n_window = CR_WINDOW_SUM with q = (a, b); a wrong n_window is a spec error
    wl = wl_mod.small_random(61, num_keys=700, n=60_000, R=40, Ws=[12, 30], J=4, hot=2, hot_share=0.4,
                             qs=[(1, 1), (3, 4)])
    gp = Pipeline(wl)
    gp.step()
    ref = gp.host()
    compare_all(wl, gp, ref, opipe.run(wl))
    counts = gp.win_src.cpu().numpy().view(np.uint32)
    specs = []
    for g in range(gp.NG):
        for c, cand in enumerate(wl.candidates):
            w = gp.plan_window[g * gp.P + c]
            n_w = int(counts[w].sum(dtype=np.uint64))
            specs.append((w, cand.W, n_w, cand.a * n_w, cand.b * wl.R, 0, 0))
    ps = B.PlanSet(specs, gp.P, wl.R, gp.max_W, wl.num_keys, gp.NW, "cuda")
    ws = torch.empty(B.cr_admit_workspace_bytes(gp.NW, wl.R, gp.max_W), dtype=torch.uint8, device="cuda")
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    B.cr_admit(gp.win_src, ps.c, ws, err)
    B.cr_place_lpt(gp.win_src, ps.c)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    for name in ("num_admitted", "cold", "member_off", "members", "load"):
        a = getattr(ps, name).cpu().numpy()
        b = getattr(gp.plans, name).cpu().numpy()
        if name in ("member_off", "members"):
            for p in range(ps.num_plans):  # defined up to the used length
                A = int(ps.num_admitted[p].item())
                m = A + 1 if name == "member_off" else int(ps.member_off[p, A].item())
                np.testing.assert_array_equal(a[p, :m], b[p, :m], err_msg=f"{name} plan {p}")
        else:
            np.testing.assert_array_equal(a.view(np.uint8), b.view(np.uint8), err_msg=name)
    bad = list(specs)
    bad[1] = (bad[1][0], bad[1][1], bad[1][2] + 1) + bad[1][3:]
    ps2 = B.PlanSet(bad, gp.P, wl.R, gp.max_W, wl.num_keys, gp.NW, "cuda")
    B.cr_admit(gp.win_src, ps2.c, ws, err)
    torch.cuda.synchronize()
    assert int(err.item()) & B.CR_ERR_SPEC
    assert int(ps2.num_admitted[1].item()) == 0
