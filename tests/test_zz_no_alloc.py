"""cr_admit_noalloc (admission with the library's own device scratch instead of a caller
workspace) against cr_admit with a caller workspace, through the C ABI: two calls in a row,
the second with a smaller input, each compared with cr_admit on the same counts."""
import numpy as np
import pytest
import torch

from paper_2608_19677_amd import binding as B
from paper_2608_19677_amd import workload as wl_mod
from paper_2608_19677_amd.pipeline import Pipeline

from cr_check import say

pytestmark = pytest.mark.gpu


def _plans_host(ps):
    torch.cuda.synchronize()
    out = {}
    for name in ("n_order", "num_admitted", "cold", "clamped"):
        out[name] = getattr(ps, name).cpu().numpy().copy()
    for w in range(ps.num_windows):
        m = int(out["n_order"][w])
        out[f"order{w}"] = ps.order[w, :m].cpu().numpy().copy()
        out[f"order_count{w}"] = ps.order_count[w, :m].cpu().numpy().copy()
    for p in range(ps.num_plans):
        A = int(out["num_admitted"][p])
        out[f"member_off{p}"] = ps.member_off[p, :A + 1].cpu().numpy().copy()
    out["key_index"] = ps.key_index.cpu().numpy().copy()
    return out


def _admit_both(wl):
    gp = Pipeline(wl, group_tables=False)
    gp.count()
    specs = torch.empty_like(gp.plans.specs).copy_(gp.plans.specs)
    ref_ps = gp.plans
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    B.cr_admit(gp.win_src, ref_ps.c, gp.ws_admit, err)
    ref = _plans_host(ref_ps)
    assert int(err.item()) == 0
    # a second plan set with the same specs, admitted without a caller workspace
    raw = bytes(specs.cpu().numpy().tobytes())
    n_specs = len(raw) // 40
    spec_tuples = [B.CrPlanSpec.from_buffer_copy(raw[40 * i:40 * i + 40]) for i in range(n_specs)]
    ps = B.PlanSet([(s.window, s.W, s.n_window, s.q_num, s.q_den, s.variant, s.place_seed) for s in spec_tuples],
                   ref_ps.cands, ref_ps.R, ref_ps.max_W, ref_ps.num_keys, ref_ps.num_windows, "cuda")
    err2 = torch.zeros(1, dtype=torch.int32, device="cuda")
    B.cr_admit_noalloc(gp.win_src, ps.c, err2)
    got = _plans_host(ps)
    assert int(err2.item()) == 0
    assert ref.keys() == got.keys()
    for k in ref:
        np.testing.assert_array_equal(got[k], ref[k], err_msg=k)
    return gp


def test_noalloc_admit_equals_admit_two_calls():
    # 1: 50,000 keys (window sorts through the workspace), 1,024 destinations, 12 windows
    big = wl_mod.small_random(71, num_keys=50_000, n=400_000, R=1024, Ws=[8, 40], J=12, hot=4, hot_share=0.3,
                              qs=[(1, 1), (4, 5)])
    need = B.cr_admit_workspace_bytes(11, 1024, 40)
    say(f"[case] noalloc admit, first call: K=50000 R=1024 windows=11 workspace={need} B")
    assert need <= B.CR_ADMIT_SCRATCH_BYTES
    _admit_both(big)
    # 2: a smaller input right after (the array keeps the first call's contents)
    small = wl_mod.small_random(72, num_keys=40_000, n=30_000, R=30, Ws=[16], J=3, hot=2, hot_share=0.2)
    say("[case] noalloc admit, second call: K=40000 R=30 windows=2")
    _admit_both(small)


def test_noalloc_admit_rejects_beyond_scratch():
    # windows x R x max_W beyond the array: CR_ESIZE before anything is enqueued
    NW, R, W = 20, 1024, 512
    assert B.cr_admit_workspace_bytes(NW, R, W) > B.CR_ADMIT_SCRATCH_BYTES
    ps = B.PlanSet([(0, W, B.CR_WINDOW_SUM, 1, 1, 0, 0)], 1, R, W, 100, NW, "cuda")
    counts = torch.zeros((NW, 100), dtype=torch.int32, device="cuda")
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    rc = B.load().cr_admit_noalloc(counts.data_ptr(), __import__("ctypes").byref(ps.c), err.data_ptr(), None)
    assert rc == B.CR_ESIZE
