"""ctypes binding of libcr.so with the C ABI's names (argument marshalling only).

Every function takes torch tensors that already live on the GPU (device memory and
the current stream come from PyTorch) and passes their raw pointers to the library.
Integer buffers use torch's signed dtypes of the same width; the library reads them
as the unsigned types of the header. Nothing here computes any step of the path, and
there is no fallback: without the built library every call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch

from .build import LIB

CR_OK, CR_EINVAL, CR_ESIZE, CR_EHIP = 0, -1, -2, -3
CR_ERR_KEY_RANGE, CR_ERR_DEST_RANGE, CR_ERR_SPEC, CR_ERR_KEYMAP_FULL = 1, 2, 4, 8
CR_NO_KEY = 0xFFFFFFFF
CR_EMPTY_SLOT = 0xFFFFFFFF
CR_ROUTE_SINGLE = 0x80000000
CR_MAX_R, CR_MAX_W, CR_MAX_CANDS, CR_MAX_J = 1024, 512, 256, 65535
CR_ADMIT_SCRATCH_BYTES = 64 << 20

EXPORTS = ("cr_count_rates", "cr_count_slice_workspace_bytes", "cr_count_slice", "cr_admit_workspace_bytes",
           "cr_admit", "cr_admit_noalloc", "cr_plan_sizes", "cr_workspace_bytes", "cr_place_lpt", "cr_place_hash", "cr_route",
           "cr_route_live", "cr_plan_churn", "cr_keymap_bytes", "cr_keymap_workspace_bytes", "cr_keymap_build",
           "cr_keymap_lookup", "cr_keymap_scatter", "cr_replay_workspace_bytes", "cr_lru_state_bytes",
           "cr_lru_reset", "cr_replay", "cr_replay_partition", "cr_replay_lru", "cr_replay_set_group_min_records",
           "cr_version")
CR_WINDOW_SUM = 0xFFFFFFFFFFFFFFFF
CR_PLAN_BUFFERS = 16
CR_GROUP_MULTI, CR_GROUP_COLD = 0xFFFE, 0xFFFF

_u32, _u64, _P = ctypes.c_uint32, ctypes.c_uint64, ctypes.c_void_p


CR_PLAN_FULL, CR_PLAN_AFFINITY, CR_PLAN_REPLICATED, CR_PLAN_FLAT = 0, 1, 2, 3
PLAN_VARIANTS = {"full": CR_PLAN_FULL, "affinity": CR_PLAN_AFFINITY, "replicated": CR_PLAN_REPLICATED,
                 "flat": CR_PLAN_FLAT}


class CrPlanSpec(ctypes.Structure):
    _fields_ = [("window", _u32), ("W", _u32), ("n_window", _u64), ("q_num", _u64), ("q_den", _u64),
                ("variant", _u32), ("place_seed", _u32)]


class CrPlanSet(ctypes.Structure):
    _fields_ = [("num_plans", _u32), ("cands", _u32), ("R", _u32), ("max_W", _u32), ("num_keys", _u32),
                ("num_windows", _u32), ("specs", _P), ("order", _P), ("order_count", _P), ("n_order", _P),
                ("num_admitted", _P), ("cold", _P), ("clamped", _P), ("member_off", _P), ("members", _P),
                ("load", _P), ("key_index", _P), ("route", _P), ("window_rank", _P), ("group_dest", _P),
                ("group_rank", _P), ("group_multi", _P)]


class CrError(RuntimeError):
    pass


_lib = None


def load(path: Optional[str] = None):
    """Load libcr.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    p = path or LIB
    if not os.path.exists(p):
        raise CrError(f"{p} is missing: build it with paper_2608_19677_amd/build.py (no fallback exists)")
    L = ctypes.CDLL(p)
    L.cr_count_rates.argtypes = [_P, _u64, _P, _u32, _u32, _P, _P, _P]
    L.cr_replay_set_group_min_records.argtypes = [_u64]
    L.cr_replay_set_group_min_records.restype = None
    L.cr_count_slice_workspace_bytes.argtypes = [_u64, _u32]
    L.cr_count_slice_workspace_bytes.restype = ctypes.c_size_t
    L.cr_count_slice.argtypes = [_P, _u64, _u32, _P, _P, _P, ctypes.c_size_t, _P]
    L.cr_plan_sizes.argtypes = [_u32, _u32, _u32, _u32, _u32, _u32, ctypes.POINTER(ctypes.c_size_t)]
    L.cr_plan_sizes.restype = None
    L.cr_workspace_bytes.argtypes = [_u32, _u32, _u32, _u64]
    L.cr_workspace_bytes.restype = ctypes.c_size_t
    L.cr_lru_state_bytes.argtypes = [_u32, _u32, _u32]
    L.cr_lru_state_bytes.restype = ctypes.c_size_t
    L.cr_lru_reset.argtypes = [_P, _u32, _u32, _u32, _P]
    L.cr_admit_workspace_bytes.argtypes = [_u32, _u32, _u32]
    L.cr_admit_workspace_bytes.restype = ctypes.c_size_t
    L.cr_admit.argtypes = [_P, ctypes.POINTER(CrPlanSet), _P, ctypes.c_size_t, _P, _P]
    L.cr_admit_noalloc.argtypes = [_P, ctypes.POINTER(CrPlanSet), _P, _P]
    L.cr_place_lpt.argtypes = [_P, ctypes.POINTER(CrPlanSet), _P]
    L.cr_place_hash.argtypes = [_P, ctypes.POINTER(CrPlanSet), _P]
    L.cr_route.argtypes = [_P, _u64, _u64, _u64, _P, _P, _u32, ctypes.POINTER(CrPlanSet), _P, _P, _P]
    L.cr_keymap_bytes.argtypes = [_u32]
    L.cr_keymap_bytes.restype = ctypes.c_size_t
    L.cr_keymap_workspace_bytes.argtypes = [_u64]
    L.cr_keymap_workspace_bytes.restype = ctypes.c_size_t
    L.cr_keymap_build.argtypes = [_P, _u64, _u32, _P, ctypes.c_size_t, _P, ctypes.c_size_t, _P, _P, _P]
    L.cr_keymap_lookup.argtypes = [_P, ctypes.c_size_t, _u32, _P, _u64, _P, _P]
    L.cr_keymap_scatter.argtypes = [_P, ctypes.c_size_t, _u32, _P, _P, _u64, _P, _u32, _P]
    L.cr_route_live.argtypes = [_P, _u64, _u64, _u64, _P, _P, _u32, ctypes.POINTER(CrPlanSet), _P, _P, _P]
    L.cr_plan_churn.argtypes = [ctypes.POINTER(CrPlanSet), _P, _u32, _P, _P, _P]
    L.cr_replay_workspace_bytes.argtypes = [_u64, _u32, _u32]
    L.cr_replay_workspace_bytes.restype = ctypes.c_size_t
    L.cr_replay.argtypes = [_P, _P, _P, _u32, _P, _u64, _P, _u32, _u32, _u32, ctypes.POINTER(_u32), _u32, _P, _P,
                            _P, _P, ctypes.c_size_t, _P, _P]
    L.cr_replay_partition.argtypes = [_P, _P, _P, _u64, _P, _u32, _u32, _u32, ctypes.POINTER(_u32), _P,
                                      ctypes.c_size_t, _P, _P]
    L.cr_replay_lru.argtypes = [_P, _u32, _u64, _u32, _u32, _u32, ctypes.POINTER(_u32), _u32, _P, _P, _P, _P,
                                ctypes.c_size_t, _P, _P]
    L.cr_version.restype = ctypes.c_char_p
    for f in ("cr_count_rates", "cr_count_slice", "cr_lru_reset", "cr_admit", "cr_admit_noalloc", "cr_place_lpt", "cr_place_hash", "cr_route", "cr_route_live", "cr_plan_churn",
              "cr_keymap_build", "cr_keymap_lookup", "cr_keymap_scatter", "cr_replay",
              "cr_replay_partition", "cr_replay_lru"):
        getattr(L, f).restype = ctypes.c_int32
    _lib = L
    return L


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_cuda:
        raise CrError("libcr takes device tensors")
    if not t.is_contiguous():
        raise CrError("libcr takes contiguous tensors")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _check(rc: int, name: str):
    if rc != CR_OK:
        raise CrError(f"{name} returned {rc}")


def cr_version() -> str:
    return load().cr_version().decode()


def cr_count_rates(keys, off, J: int, num_keys: int, counts, err, stream=None, n: Optional[int] = None):
    n = keys.numel() if n is None else n
    _check(load().cr_count_rates(_ptr(keys), n, _ptr(off), J, num_keys, _ptr(counts), _ptr(err), _stream(stream)),
           "cr_count_rates")


def cr_count_slice_workspace_bytes(n: int, num_keys: int) -> int:
    return int(load().cr_count_slice_workspace_bytes(n, num_keys))


def cr_count_slice(keys, num_keys: int, counts, err, ws, stream=None, n: Optional[int] = None):
    n = keys.numel() if n is None else n
    _check(load().cr_count_slice(_ptr(keys), n, num_keys, _ptr(counts), _ptr(err), _ptr(ws), _nbytes(ws),
                                 _stream(stream)), "cr_count_slice")


def cr_plan_sizes(num_plans: int, cands: int, R: int, max_W: int, num_keys: int, num_windows: int):
    out = (ctypes.c_size_t * CR_PLAN_BUFFERS)()
    load().cr_plan_sizes(num_plans, cands, R, max_W, num_keys, num_windows, out)
    return [int(x) for x in out]


def cr_workspace_bytes(num_keys: int, R: int, P: int, max_n: int) -> int:
    return int(load().cr_workspace_bytes(num_keys, R, P, max_n))


def cr_lru_state_bytes(P: int, R: int, max_W: int) -> int:
    return int(load().cr_lru_state_bytes(P, R, max_W))


def cr_lru_reset(lru_state, P: int, R: int, max_W: int, stream=None):
    _check(load().cr_lru_reset(_ptr(lru_state), P, R, max_W, _stream(stream)), "cr_lru_reset")


def cr_admit_workspace_bytes(num_windows: int, R: int, max_W: int) -> int:
    return int(load().cr_admit_workspace_bytes(num_windows, R, max_W))


def cr_admit(counts, plans: CrPlanSet, ws, err, stream=None):
    _check(load().cr_admit(_ptr(counts), ctypes.byref(plans), _ptr(ws), ws.numel() * ws.element_size(), _ptr(err),
                           _stream(stream)), "cr_admit")


def cr_admit_noalloc(counts, plans: CrPlanSet, err, stream=None):
    _check(load().cr_admit_noalloc(_ptr(counts), ctypes.byref(plans), _ptr(err), _stream(stream)), "cr_admit_noalloc")


def cr_place_lpt(counts, plans: CrPlanSet, stream=None):
    _check(load().cr_place_lpt(_ptr(counts), ctypes.byref(plans), _stream(stream)), "cr_place_lpt")


def cr_place_hash(counts, plans: CrPlanSet, stream=None):
    _check(load().cr_place_hash(_ptr(counts), ctypes.byref(plans), _stream(stream)), "cr_place_hash")


def cr_route(keys, first_index: int, seed: int, off, gmap, J: int, plans: CrPlanSet, dest, err, stream=None,
             n: Optional[int] = None):
    n = keys.numel() if n is None else n
    _check(load().cr_route(_ptr(keys), n, first_index, seed, _ptr(off), _ptr(gmap), J, ctypes.byref(plans),
                           _ptr(dest), _ptr(err), _stream(stream)), "cr_route")


def cr_keymap_bytes(capacity: int) -> int:
    return int(load().cr_keymap_bytes(capacity))


def cr_keymap_workspace_bytes(n: int) -> int:
    return int(load().cr_keymap_workspace_bytes(n))


def _nbytes(t) -> int:
    return t.numel() * t.element_size()


def cr_keymap_build(ids, capacity: int, table, ws, num_keys, err, stream=None, n: Optional[int] = None):
    n = ids.numel() if n is None else n
    _check(load().cr_keymap_build(_ptr(ids), n, capacity, _ptr(table), _nbytes(table), _ptr(ws), _nbytes(ws),
                                  _ptr(num_keys), _ptr(err), _stream(stream)), "cr_keymap_build")


def cr_keymap_lookup(table, capacity: int, ids, dense, stream=None, n: Optional[int] = None):
    n = ids.numel() if n is None else n
    _check(load().cr_keymap_lookup(_ptr(table), _nbytes(table), capacity, _ptr(ids), n, _ptr(dense), _stream(stream)),
           "cr_keymap_lookup")


def cr_keymap_scatter(table, capacity: int, ids, values, out, stream=None):
    _check(load().cr_keymap_scatter(_ptr(table), _nbytes(table), capacity, _ptr(ids), _ptr(values), ids.numel(),
                                    _ptr(out), out.numel(), _stream(stream)), "cr_keymap_scatter")


def cr_route_live(keys, first_index: int, seed: int, off, gmap, J: int, plans: CrPlanSet, dest, err, stream=None,
                  n: Optional[int] = None):
    n = keys.numel() if n is None else n
    _check(load().cr_route_live(_ptr(keys), n, first_index, seed, _ptr(off), _ptr(gmap), J, ctypes.byref(plans),
                                _ptr(dest), _ptr(err), _stream(stream)), "cr_route_live")


def cr_plan_churn(plans: CrPlanSet, pairs, out, err, stream=None):
    """pairs: int32 [num_pairs, 2] plan indices; out: int64 [num_pairs, 4]."""
    num_pairs = pairs.shape[0]
    _check(load().cr_plan_churn(ctypes.byref(plans), _ptr(pairs), num_pairs, _ptr(out), _ptr(err), _stream(stream)),
           "cr_plan_churn")


def cr_replay_workspace_bytes(n: int, P: int, R: int) -> int:
    return int(load().cr_replay_workspace_bytes(n, P, R))


GROUP_MIN_RECORDS_DEFAULT = 1 << 25


def cr_replay_set_group_min_records(min_records: int) -> None:
    load().cr_replay_set_group_min_records(min_records)


def cr_replay(keys, suffix, prefix_len, num_keys: int, dest, off, J: int, P: int, R: int, W: Sequence[int],
              max_W: int, lru_in, lru_out, stats, ws, err, stream=None, n: Optional[int] = None):
    n = keys.numel() if n is None else n
    Wa = (_u32 * len(W))(*[int(x) for x in W])
    _check(load().cr_replay(_ptr(keys), _ptr(suffix), _ptr(prefix_len), num_keys, _ptr(dest), n, _ptr(off), J, P, R,
                            Wa, max_W, _ptr(lru_in), _ptr(lru_out), _ptr(stats), _ptr(ws),
                            ws.numel() * ws.element_size(), _ptr(err), _stream(stream)), "cr_replay")


def cr_replay_partition(keys, suffix, dest, off, J: int, P: int, R: int, W: Sequence[int], ws, err, stream=None,
                        n: Optional[int] = None):
    n = keys.numel() if n is None else n
    Wa = (_u32 * len(W))(*[int(x) for x in W])
    _check(load().cr_replay_partition(_ptr(keys), _ptr(suffix), _ptr(dest), n, _ptr(off), J, P, R, Wa, _ptr(ws),
                                      ws.numel() * ws.element_size(), _ptr(err), _stream(stream)),
           "cr_replay_partition")


def cr_replay_lru(prefix_len, num_keys: int, n: int, J: int, P: int, R: int, W: Sequence[int], max_W: int, lru_in,
                  lru_out, stats, ws, err, stream=None):
    Wa = (_u32 * len(W))(*[int(x) for x in W])
    _check(load().cr_replay_lru(_ptr(prefix_len), num_keys, n, J, P, R, Wa, max_W, _ptr(lru_in), _ptr(lru_out),
                                _ptr(stats), _ptr(ws), ws.numel() * ws.element_size(), _ptr(err), _stream(stream)),
           "cr_replay_lru")


class PlanSet:
    """Device buffers of a cr_plan_set (NP = NG * cands plans over num_windows rows).
    ``group_tables`` also allocates the optional group dispatch tables that let cr_route
    serve every candidate of a request from one row (candidates of a group must share
    their counting window)."""

    def __init__(self, specs, cands: int, R: int, max_W: int, num_keys: int, num_windows: int, device,
                 group_tables: bool = False):
        self.num_plans = len(specs)
        self.cands, self.R, self.max_W, self.num_keys, self.num_windows = cands, R, max_W, num_keys, num_windows
        cmax = R * max_W
        self.cmax = cmax
        NP, NW = self.num_plans, num_windows
        raw = (CrPlanSpec * NP)(*[CrPlanSpec(*s) for s in specs])
        host = torch.frombuffer(bytearray(bytes(raw)), dtype=torch.uint8)
        self.specs = host.to(device)
        i32 = dict(dtype=torch.int32, device=device)
        self.order = torch.empty((NW, cmax), **i32)
        self.order_count = torch.empty((NW, cmax), **i32)
        self.n_order = torch.empty(NW, **i32)
        self.num_admitted = torch.empty(NP, **i32)
        self.cold = torch.empty(NP, dtype=torch.int64, device=device)
        self.clamped = torch.empty(NP, **i32)
        self.member_off = torch.empty((NP, cmax + 1), **i32)
        self.members = torch.empty((NP, cmax), dtype=torch.int16, device=device)
        self.load = torch.empty((NP, R), dtype=torch.float64, device=device)
        self.key_index = torch.empty((NP, (num_keys + 63) // 64, 2), dtype=torch.int64, device=device)
        self.route = torch.empty((NP, cmax), **i32)
        self.window_rank = self.group_dest = self.group_rank = self.group_multi = None
        if group_tables:
            NG = NP // cands
            self.window_rank = torch.empty((NW, num_keys), **i32)
            self.group_dest = torch.empty((NG, cmax, group_row(cands)), dtype=torch.int16, device=device)
            self.group_rank = torch.empty((NG, R, group_row(cands)), dtype=torch.int16, device=device)
            self.group_multi = torch.empty((NG, cmax, group_row(cands)), **i32)
        self.c = CrPlanSet(NP, cands, R, max_W, num_keys, NW, _ptr(self.specs), _ptr(self.order),
                           _ptr(self.order_count), _ptr(self.n_order),
                           _ptr(self.num_admitted), _ptr(self.cold), _ptr(self.clamped), _ptr(self.member_off),
                           _ptr(self.members), _ptr(self.load), _ptr(self.key_index), _ptr(self.route),
                           _ptr(self.window_rank), _ptr(self.group_dest), _ptr(self.group_rank),
                           _ptr(self.group_multi))


def group_row(cands: int) -> int:
    """Entries per group_dest row: cands rounded up to a multiple of 8."""
    return (cands + 7) // 8 * 8


def group_table_bytes(NG: int, cands: int, R: int, max_W: int, num_keys: int, num_windows: int) -> int:
    """Bytes of the four group dispatch tables."""
    return (num_windows * num_keys * 4 + NG * R * max_W * group_row(cands) * 6
            + NG * R * group_row(cands) * 2)
