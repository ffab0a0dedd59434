"""Device-path driver: one pass of count -> plan -> route -> replay through libcr.

Semantics (the paper's statement of the loop, Sections 3.1-3.2):
* the counting windows are the control intervals; the plan in force during interval j
  is built from the counts of interval j-1 and stays fixed for the interval; interval 0
  has no earlier window and is planned from its own counts (or, for a stream processed
  in chunks, from the last window of the previous chunk);
* candidate (W, a, b) has C = R W warm slots and load target q_cap = (a/b) N_w / R,
  passed to the library as q_num = a N_w, q_den = b R;
* the replay's per-destination cache state is carried across intervals and chunks.

Inputs are uploaded once by ``prepare``; ``step`` only enqueues the five library calls
(plus clearing the accumulating outputs) on the current stream.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional

import numpy as np
import torch

from . import binding as B


@dataclass
class DeviceInputs:
    keys: torch.Tensor
    suffix: torch.Tensor
    prefix_len: torch.Tensor
    off: torch.Tensor
    off_host: np.ndarray


def upload(wl, device="cuda") -> DeviceInputs:
    def t(a, dt):
        return torch.from_numpy(np.ascontiguousarray(a).view(dt)).to(device)

    return DeviceInputs(keys=t(wl.keys, np.int32), suffix=t(wl.suffix, np.int16),
                        prefix_len=t(wl.prefix_len, np.int32), off=t(wl.offsets, np.int64),
                        off_host=np.asarray(wl.offsets, dtype=np.uint64))


class Pipeline:
    """All device buffers for one workload (or one chunk of a chunked stream)."""

    def __init__(self, wl, device="cuda", dev_in: Optional[DeviceInputs] = None,
                 prev_counts: Optional[torch.Tensor] = None, prev_n: int = 0,
                 lru_in: Optional[torch.Tensor] = None):
        self.wl = wl
        self.device = device
        self.inp = dev_in if dev_in is not None else upload(wl, device)
        J, K, R, P = wl.J, wl.num_keys, wl.R, wl.P
        self.J, self.K, self.R, self.P, self.n = J, K, R, P, wl.n
        self.Ws = [c.W for c in wl.candidates]
        self.max_W = max(self.Ws)
        sizes = np.diff(self.inp.off_host.astype(np.int64))
        i32 = dict(dtype=torch.int32, device=device)
        self.counts = torch.empty((J, K), **i32)
        self.err = torch.zeros(1, **i32)
        # plan windows: groups g = 0..NG-1, interval j -> group gmap[j]
        self.prev_counts = prev_counts
        if prev_counts is None:
            NG = max(J - 1, 1)
            self.win_src = self.counts[:NG]
            gmap = [max(j - 1, 0) for j in range(J)]
            n_win = [int(sizes[g]) for g in range(NG)]
        else:
            NG = J
            self.win_buf = torch.empty((J, K), **i32)
            self.win_src = self.win_buf
            gmap = list(range(J))
            n_win = [int(prev_n)] + [int(sizes[g]) for g in range(J - 1)]
        self.NG = NG
        self.gmap = torch.tensor(gmap, dtype=torch.int32, device=device)
        specs = []
        for g in range(NG):
            for cand in wl.candidates:
                specs.append((g, cand.W, n_win[g], cand.a * n_win[g], cand.b * R))
        self.plans = B.PlanSet(specs, P, R, self.max_W, K, NG, device)
        self.ws_admit = torch.empty(B.cr_admit_workspace_bytes(NG, R, self.max_W), dtype=torch.uint8, device=device)
        self.ws_replay = torch.empty(B.cr_replay_workspace_bytes(wl.n, P, R), dtype=torch.uint8, device=device)
        self.dest = torch.empty((P, max(wl.n, 1)), dtype=torch.int16, device=device)
        self.stats = torch.zeros((J, P, R, 4), dtype=torch.int64, device=device)
        self.lru_in = lru_in
        self.lru_out = torch.empty((P, R, self.max_W), **i32)

    # -- the five calls ----------------------------------------------------------------
    def count(self, stream=None):
        B.cr_count_rates(self.inp.keys, self.inp.off, self.J, self.K, self.counts, self.err, stream, n=self.n)
        if self.prev_counts is not None:
            self.win_buf[0].copy_(self.prev_counts)
            if self.J > 1:
                self.win_buf[1:].copy_(self.counts[: self.J - 1])

    def admit(self, stream=None):
        B.cr_admit(self.win_src, self.plans.c, self.ws_admit, self.err, stream)

    def place(self, stream=None):
        B.cr_place_lpt(self.win_src, self.plans.c, stream)

    def plan(self, stream=None):
        self.admit(stream)
        self.place(stream)

    def route(self, stream=None):
        B.cr_route(self.inp.keys, self.wl.first_index, self.wl.seed, self.inp.off, self.gmap, self.J, self.plans.c,
                   self.dest, self.err, stream, n=self.n)

    def partition(self, stream=None):
        B.cr_replay_partition(self.inp.keys, self.inp.suffix, self.dest, self.inp.off, self.J, self.P, self.R,
                              self.Ws, self.ws_replay, self.err, stream, n=self.n)

    def lru(self, stream=None):
        self.stats.zero_()
        B.cr_replay_lru(self.inp.prefix_len, self.K, self.n, self.J, self.P, self.R, self.Ws, self.max_W,
                        self.lru_in, self.lru_out, self.stats, self.ws_replay, self.err, stream)

    def replay(self, stream=None):
        self.stats.zero_()
        B.cr_replay(self.inp.keys, self.inp.suffix, self.inp.prefix_len, self.K, self.dest, self.inp.off, self.J,
                    self.P, self.R, self.Ws, self.max_W, self.lru_in, self.lru_out, self.stats, self.ws_replay,
                    self.err, stream, n=self.n)

    STAGES = ("count", "admit", "place", "route", "partition", "lru")

    def step(self, stream=None):
        for s in self.STAGES:
            getattr(self, s)(stream)

    # -- host views for checking -------------------------------------------------------
    def host(self) -> dict:
        torch.cuda.synchronize()
        u32 = lambda t: t.cpu().numpy().view(np.uint32)
        ps = self.plans
        return dict(counts=u32(self.counts), n_order=u32(ps.n_order), order=u32(ps.order),
                    num_admitted=u32(ps.num_admitted), cold=ps.cold.cpu().numpy().view(np.uint64),
                    clamped=u32(ps.clamped), member_off=u32(ps.member_off),
                    members=ps.members.cpu().numpy().view(np.uint16), load=ps.load.cpu().numpy(),
                    route=u32(ps.route), dest=self.dest[:, : self.n].cpu().numpy().view(np.uint16),
                    stats=self.stats.cpu().numpy().view(np.uint64), lru=u32(self.lru_out),
                    err=int(self.err.cpu().numpy().view(np.uint32)[0]))

    def plan_of(self, h: dict, g: int, c: int) -> dict:
        """Admitted keys, k and members of plan (group g, candidate c) from host views."""
        p = g * self.P + c
        A = int(h["num_admitted"][p])
        w = g
        mo = h["member_off"][p, : A + 1]
        return dict(adm_keys=h["order"][w, :A].copy(), adm_k=np.diff(mo).astype(np.uint32),
                    member_off=mo.copy(), members=h["members"][p, : int(mo[A]) if A else 0].copy(),
                    L=h["load"][p].copy(), cold=int(h["cold"][p]), clamped=int(h["clamped"][p]))
