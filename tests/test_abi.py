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


def test_struct_layouts_match_header(lib_path):
    from paper_2608_19677_amd import binding
    assert ctypes.sizeof(binding.CrPlanSpec) == 40
    assert ctypes.sizeof(binding.CrPlanSet) == 6 * 4 + 15 * 8
