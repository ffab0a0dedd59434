"""The C-ABI library loads on a CPU-only host and exports every entry point its header
declares (no compute calls here)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cr.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(cr_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib_path():
    from paper_2608_19677_amd import build
    if not os.path.exists(build.LIB):
        build.build()
    return build.LIB


def test_header_declares_the_five_calls():
    names = _declared()
    for f in ("cr_count_rates", "cr_admit", "cr_place_lpt", "cr_route", "cr_replay"):
        assert f in names


def test_library_exports_every_declared_symbol(lib_path):
    lib = ctypes.CDLL(lib_path)
    missing = [f for f in _declared() if not hasattr(lib, f)]
    assert not missing, missing


def test_binding_names_match_header(lib_path):
    from paper_2608_19677_amd import binding
    assert sorted(binding.EXPORTS) == _declared()
    for f in binding.EXPORTS:
        assert callable(getattr(binding, f))


def test_host_only_queries(lib_path):
    from paper_2608_19677_amd import binding
    assert binding.cr_version().startswith("cr ")
    a = binding.cr_admit_workspace_bytes(10, 30, 64)
    assert a >= 10 * 2 * 30 * 64 * 8
    r = binding.cr_replay_workspace_bytes(10**6, 2, 30)
    assert r >= 2 * 10**6 * 8
    assert binding.cr_replay_workspace_bytes(0, 1, 1) > 0
    # the grouped-replay size rule is host state only: setting and restoring it launches nothing
    binding.cr_replay_set_group_min_records(0)
    binding.cr_replay_set_group_min_records(binding.GROUP_MIN_RECORDS_DEFAULT)


def test_struct_layouts_match_header(lib_path):
    from paper_2608_19677_amd import binding
    assert ctypes.sizeof(binding.CrPlanSpec) == 40
    assert ctypes.sizeof(binding.CrPlanSet) == 6 * 4 + 16 * 8


def test_plan_sizes_follow_the_header_layouts(lib_path):
    # restated from the layouts documented in cr.h: C_max = R max_W, KW = ceil(K / 64),
    # NG = NP / cands, CS = cands rounded up to 8
    from paper_2608_19677_amd import binding
    for NP, cands, R, W, K, NW in [(1, 1, 30, 64, 20_000, 1), (948, 1, 30, 64, 20_000, 948),
                                   (64, 64, 1024, 512, 10**6, 1), (300, 100, 70, 60, 2000, 3)]:
        cm, KW, NG, CS = R * W, (K + 63) // 64, NP // cands, (cands + 7) // 8 * 8
        want = [NP * 40, NW * cm * 4, NW * cm * 4, NW * 4, NP * 4, NP * 8, NP * 4, NP * (cm + 1) * 4, NP * cm * 2,
                NP * R * 8, NP * KW * 16, NP * cm * 4, NW * K * 4, NG * cm * CS * 2, NG * R * CS * 2, NG * cm * CS * 4]
        assert binding.cr_plan_sizes(NP, cands, R, W, K, NW) == want


def test_workspace_and_state_sizes(lib_path):
    from paper_2608_19677_amd import binding
    for K, R, P, n in [(1000, 30, 1, 10**5), (10**6, 1024, 64, 10**8), (5, 1, 1, 0)]:
        ws = binding.cr_workspace_bytes(K, R, P, n)
        assert ws >= binding.cr_replay_workspace_bytes(n, P, R)
        assert ws >= binding.cr_count_slice_workspace_bytes(n, K)
    # the slice workspace holds the bucket-sorted keys: at least 4 B per request
    assert binding.cr_count_slice_workspace_bytes(10**8, 10**6) >= 4 * 10**8
    assert binding.cr_lru_state_bytes(64, 1024, 512) == 64 * 1024 * 512 * 4
    assert binding.cr_lru_state_bytes(1, 30, 16) == 30 * 16 * 4
