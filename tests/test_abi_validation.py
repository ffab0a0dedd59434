"""Argument validation of the C ABI: every malformed call returns its error code on the
host before anything is enqueued (runs without a GPU; no pointer is dereferenced)."""
import ctypes
import os

import pytest

from paper_2608_19677_amd import binding as B

FAKE = 0x10000  # never dereferenced: every call below fails validation first


def _gpu_visible() -> bool:
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:  # pragma: no cover
        return False


# Host-only checks: with a GPU visible a validation regression would launch a kernel on a
# fake address, so these run only where no GPU is present.
pytestmark = pytest.mark.skipif(_gpu_visible(), reason="host-side validation tests run without a GPU")


@pytest.fixture(scope="module")
def L():
    from paper_2608_19677_amd import build
    if not os.path.exists(build.LIB):
        build.build()
    return B.load()


def _set(**kw):
    f = dict(num_plans=2, cands=1, R=30, max_W=16, num_keys=100, num_windows=2)
    f.update(kw)
    ps = B.CrPlanSet(f["num_plans"], f["cands"], f["R"], f["max_W"], f["num_keys"], f["num_windows"],
                     *([FAKE] * 12))
    return ps


def test_count_rejects(L):
    assert L.cr_count_rates(FAKE, 10, FAKE, 0, 100, FAKE, FAKE, None) == B.CR_EINVAL      # J = 0
    assert L.cr_count_rates(FAKE, 10, FAKE, 1, 0, FAKE, FAKE, None) == B.CR_EINVAL        # no keys
    assert L.cr_count_rates(FAKE, 10, FAKE, 1, 0xFFFFFFFF, FAKE, FAKE, None) == B.CR_EINVAL
    assert L.cr_count_rates(None, 10, FAKE, 1, 100, FAKE, FAKE, None) == B.CR_EINVAL      # keys NULL
    assert L.cr_count_rates(FAKE + 2, 10, FAKE, 1, 100, FAKE, FAKE, None) == B.CR_EINVAL  # misaligned keys
    assert L.cr_count_rates(FAKE, 10, None, 1, 100, FAKE, FAKE, None) == B.CR_EINVAL
    assert L.cr_count_rates(FAKE, 10, FAKE, 1, 100, None, FAKE, None) == B.CR_EINVAL
    assert L.cr_count_rates(FAKE, 10, FAKE, 1, 100, FAKE, None, None) == B.CR_EINVAL


@pytest.mark.parametrize("kw", [dict(R=0), dict(R=1025), dict(max_W=0), dict(max_W=513), dict(cands=0),
                                dict(cands=257, num_plans=257), dict(num_plans=3, cands=2), dict(num_keys=0),
                                dict(num_windows=0), dict(num_plans=0)])
def test_plan_set_rejects(L, kw):
    ps = _set(**kw)
    assert L.cr_admit(FAKE, ctypes.byref(ps), FAKE, 1 << 40, FAKE, None) == B.CR_EINVAL
    assert L.cr_place_lpt(FAKE, ctypes.byref(ps), None) == B.CR_EINVAL
    assert L.cr_plan_churn(ctypes.byref(ps), FAKE, 1, FAKE, FAKE, None) == B.CR_EINVAL
    assert L.cr_place_hash(FAKE, ctypes.byref(ps), None) == B.CR_EINVAL


def test_place_hash_rejects(L):
    ps = _set()
    assert L.cr_place_hash(None, ctypes.byref(ps), None) == B.CR_EINVAL
    assert L.cr_place_hash(FAKE, None, None) == B.CR_EINVAL
    ps.members = None
    assert L.cr_place_hash(FAKE, ctypes.byref(ps), None) == B.CR_EINVAL


def test_churn_rejects(L):
    ps = _set()
    assert L.cr_plan_churn(ctypes.byref(ps), None, 1, FAKE, FAKE, None) == B.CR_EINVAL     # pairs NULL
    assert L.cr_plan_churn(ctypes.byref(ps), FAKE, 1, None, FAKE, None) == B.CR_EINVAL     # out NULL
    assert L.cr_plan_churn(ctypes.byref(ps), FAKE, 1, FAKE, None, None) == B.CR_EINVAL     # err NULL
    assert L.cr_plan_churn(None, FAKE, 1, FAKE, FAKE, None) == B.CR_EINVAL
    assert L.cr_plan_churn(ctypes.byref(ps), None, 0, None, FAKE, None) == B.CR_OK         # no pairs: no-op


def test_admit_workspace_too_small(L):
    ps = _set()
    need = L.cr_admit_workspace_bytes(2, 30, 16)
    assert L.cr_admit(FAKE, ctypes.byref(ps), FAKE, need - 1, FAKE, None) == B.CR_ESIZE
    assert L.cr_admit(FAKE, ctypes.byref(ps), None, need, FAKE, None) == B.CR_EINVAL
    ps.order_count = None
    assert L.cr_admit(FAKE, ctypes.byref(ps), FAKE, need, FAKE, None) == B.CR_EINVAL


@pytest.mark.parametrize("fn", ["cr_route", "cr_route_live"])
def test_route_rejects(L, fn):
    route = getattr(L, fn)
    ps = _set()
    assert route(FAKE, 10, 0, 1, FAKE, FAKE, 0, ctypes.byref(ps), FAKE, FAKE, None) == B.CR_EINVAL
    assert route(FAKE, 10, 0, 1, None, FAKE, 1, ctypes.byref(ps), FAKE, FAKE, None) == B.CR_EINVAL
    assert route(FAKE, 10, 0, 1, FAKE, None, 1, ctypes.byref(ps), FAKE, FAKE, None) == B.CR_EINVAL
    assert route(FAKE + 1, 10, 0, 1, FAKE, FAKE, 1, ctypes.byref(ps), FAKE, FAKE, None) == B.CR_EINVAL
    assert route(FAKE, 10, 0, 1, FAKE, FAKE, 1, ctypes.byref(ps), FAKE + 1, FAKE, None) == B.CR_EINVAL
    assert route(FAKE, 10, 0, 1, FAKE, FAKE, 1, None, FAKE, FAKE, None) == B.CR_EINVAL
    assert route(FAKE, 0, 0, 1, FAKE, FAKE, 1, ctypes.byref(ps), FAKE, FAKE, None) == B.CR_OK  # empty: no-op


def test_route_static_rejects_more(L):
    ps = _set()
    assert L.cr_route(FAKE, 10, 0, 1, FAKE, FAKE, 0, ctypes.byref(ps), FAKE, FAKE, None) == B.CR_EINVAL
    assert L.cr_route(FAKE, 10, 0, 1, None, FAKE, 1, ctypes.byref(ps), FAKE, FAKE, None) == B.CR_EINVAL
    assert L.cr_route(FAKE, 10, 0, 1, FAKE, None, 1, ctypes.byref(ps), FAKE, FAKE, None) == B.CR_EINVAL
    assert L.cr_route(FAKE + 1, 10, 0, 1, FAKE, FAKE, 1, ctypes.byref(ps), FAKE, FAKE, None) == B.CR_EINVAL
    bad = _set(R=2000)
    assert L.cr_route(FAKE, 10, 0, 1, FAKE, FAKE, 1, ctypes.byref(bad), FAKE, FAKE, None) == B.CR_EINVAL
    assert L.cr_route(FAKE, 0, 0, 1, FAKE, FAKE, 1, ctypes.byref(ps), FAKE, FAKE, None) == B.CR_OK  # empty: no-op


def _W(*v):
    return (ctypes.c_uint32 * len(v))(*v)


def test_replay_rejects(L):
    need = L.cr_replay_workspace_bytes(1000, 2, 30)
    ok = dict(keys=FAKE, suffix=FAKE, plen=FAKE, K=100, dest=FAKE, n=1000, off=FAKE, J=1, P=2, R=30,
              W=_W(16, 8), maxW=16, lin=None, lout=FAKE, stats=FAKE, ws=FAKE, wsb=need, err=FAKE)

    def call(**kw):
        a = dict(ok)
        a.update(kw)
        return L.cr_replay(a["keys"], a["suffix"], a["plen"], a["K"], a["dest"], a["n"], a["off"], a["J"], a["P"],
                           a["R"], a["W"], a["maxW"], a["lin"], a["lout"], a["stats"], a["ws"], a["wsb"], a["err"],
                           None)

    assert call(P=0) == B.CR_EINVAL
    assert call(P=257) == B.CR_EINVAL
    assert call(R=0) == B.CR_EINVAL
    assert call(J=0) == B.CR_EINVAL
    assert call(J=65536) == B.CR_EINVAL
    assert call(W=_W(16, 0)) == B.CR_EINVAL
    assert call(W=_W(16, 17)) == B.CR_EINVAL          # W above max_W
    assert call(maxW=513, W=_W(513, 8)) == B.CR_EINVAL
    assert call(wsb=need - 1) == B.CR_ESIZE
    assert call(lout=None) == B.CR_EINVAL
    assert call(lin=FAKE, lout=FAKE + 64) == B.CR_EINVAL  # overlapping carried state
    assert call(n=2**32) == B.CR_EINVAL
    assert call(K=0) == B.CR_EINVAL
    assert L.cr_replay_partition(FAKE, FAKE, FAKE, 1000, FAKE, 1, 2, 30, _W(16, 8), FAKE, need - 8, FAKE,
                                 None) == B.CR_ESIZE
    assert L.cr_replay_lru(FAKE, 100, 1000, 1, 2, 30, _W(16, 8), 8, None, FAKE, FAKE, FAKE, need, FAKE,
                           None) == B.CR_EINVAL  # max_W below a W


def test_keymap_rejects(L):
    tb = L.cr_keymap_bytes(100)
    ws = L.cr_keymap_workspace_bytes(1000)
    assert tb >= 16 * 200 and L.cr_keymap_bytes(1) >= 16 * 64
    assert L.cr_keymap_workspace_bytes(10**6) > ws > 0
    ok = (FAKE, 1000, 100, FAKE, tb, FAKE, ws, FAKE, FAKE, None)
    assert L.cr_keymap_build(*ok[:2], 0, *ok[3:]) == B.CR_EINVAL                    # capacity 0
    assert L.cr_keymap_build(*ok[:2], (1 << 28) + 1, *ok[3:]) == B.CR_EINVAL        # over the limit
    assert L.cr_keymap_build(*ok[:3], None, *ok[4:]) == B.CR_EINVAL                 # table NULL
    assert L.cr_keymap_build(*ok[:4], tb - 1, *ok[5:]) == B.CR_ESIZE                # table too small
    assert L.cr_keymap_build(*ok[:6], ws - 1, *ok[7:]) == B.CR_ESIZE                # workspace too small
    assert L.cr_keymap_build(None, *ok[1:]) == B.CR_EINVAL                          # ids NULL
    assert L.cr_keymap_build(FAKE + 2, *ok[1:]) == B.CR_EINVAL                      # misaligned ids
    assert L.cr_keymap_build(*ok[:7], None, *ok[8:]) == B.CR_EINVAL                 # num_keys NULL
    assert L.cr_keymap_build(*ok[:8], None, None) == B.CR_EINVAL                    # err NULL
    assert L.cr_keymap_lookup(FAKE, tb, 0, FAKE, 10, FAKE, None) == B.CR_EINVAL
    assert L.cr_keymap_lookup(FAKE, tb - 1, 100, FAKE, 10, FAKE, None) == B.CR_ESIZE
    assert L.cr_keymap_lookup(FAKE, tb, 100, None, 10, FAKE, None) == B.CR_EINVAL
    assert L.cr_keymap_lookup(FAKE, tb, 100, FAKE, 0, FAKE, None) == B.CR_OK        # empty: no-op
    assert L.cr_keymap_scatter(FAKE, tb, 100, FAKE, None, 5, FAKE, 10, None) == B.CR_EINVAL
    assert L.cr_keymap_scatter(FAKE, tb - 1, 100, FAKE, FAKE, 5, FAKE, 10, None) == B.CR_ESIZE
    assert L.cr_keymap_scatter(FAKE, tb, 100, FAKE, FAKE, 0, FAKE, 10, None) == B.CR_OK


def test_count_slice_rejects(L):
    ws = 1 << 40  # large enough: no call below reaches the size check by accident
    assert L.cr_count_slice(FAKE, 10, 0, FAKE, FAKE, FAKE, ws, None) == B.CR_EINVAL           # no keys
    assert L.cr_count_slice(FAKE, 10, 0xFFFFFFFF, FAKE, FAKE, FAKE, ws, None) == B.CR_EINVAL
    assert L.cr_count_slice(None, 10, 100, FAKE, FAKE, FAKE, ws, None) == B.CR_EINVAL         # keys NULL
    assert L.cr_count_slice(FAKE + 2, 10, 100, FAKE, FAKE, FAKE, ws, None) == B.CR_EINVAL     # misaligned
    assert L.cr_count_slice(FAKE, 10, 100, None, FAKE, FAKE, ws, None) == B.CR_EINVAL
    assert L.cr_count_slice(FAKE, 10, 100, FAKE, None, FAKE, ws, None) == B.CR_EINVAL
    assert L.cr_count_slice(FAKE, 10, 100, FAKE, FAKE, None, ws, None) == B.CR_EINVAL         # no workspace
    assert L.cr_count_slice(FAKE, 10, 1 << 30, FAKE, FAKE, FAKE, ws, None) == B.CR_EINVAL     # > 256 buckets
    need = L.cr_count_slice_workspace_bytes(10, 100)
    assert L.cr_count_slice(FAKE, 10, 100, FAKE, FAKE, FAKE, need - 1, None) == B.CR_ESIZE
    assert L.cr_count_slice(None, 0, 100, FAKE, FAKE, None, 0, None) == B.CR_OK                # empty slice


def test_lru_reset_rejects(L):
    assert L.cr_lru_reset(None, 1, 30, 16, None) == B.CR_EINVAL
    for P, R, W in [(0, 30, 16), (257, 30, 16), (1, 0, 16), (1, 1025, 16), (1, 30, 0), (1, 30, 513)]:
        assert L.cr_lru_reset(FAKE, P, R, W, None) == B.CR_EINVAL


def test_route_rejects_partial_group_tables(L):
    # the four group tables come together, group_dest, group_rank and group_multi 16-byte aligned
    keys = FAKE
    for wr, gd, gp, gm in [(FAKE, None, None, None), (FAKE, FAKE, None, FAKE), (None, FAKE, FAKE, FAKE),
                           (FAKE, FAKE, FAKE, None), (FAKE, FAKE + 8, FAKE, FAKE), (FAKE, FAKE, FAKE + 8, FAKE),
                           (FAKE, FAKE, FAKE, FAKE + 4)]:
        ps = _set(cands=2, num_plans=2)
        ps.window_rank, ps.group_dest, ps.group_rank, ps.group_multi = wr, gd, gp, gm
        assert L.cr_route(keys, 16, 0, 1, FAKE, FAKE, 1, ctypes.byref(ps), FAKE, FAKE, None) == B.CR_EINVAL
