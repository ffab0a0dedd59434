"""Device-path driver: one pass of count -> plan -> route -> replay through libcr.

Semantics (the paper's statement of the loop, Sections 3.1-3.2):
* the counting windows are the control intervals; the plan in force during interval j
  is built from the counts of interval j-1 and stays fixed for the interval; interval 0
  has no earlier window and is planned from its own counts (or, for a stream processed
  in chunks, from the last window of the previous chunk);
* candidate (W, a, b) has C = R W warm slots and load target q_cap = (a/b) N_w / R,
  passed to the library as q_num = a N_w, q_den = b R;
* the replay's per-destination cache state is carried across intervals and chunks;
* dispatch is static (interval-start planned loads, order independent) or live (running
  loads of the interval, one serial chain per interval and candidate);
* a workload may name the window of each (interval, candidate) plan itself, as the
  replanning study does (Section 5.4, Appendix E): one plan group per interval then,
  and replay statistics may be kept in bins finer than the intervals.

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

    GROUP_TABLE_BUDGET = 4 << 30  # bytes the optional group dispatch tables may take
    SLICE_MIN_KEYS = 100_000      # one-interval streams with this many keys use cr_count_slice

    def __init__(self, wl, device="cuda", dev_in: Optional[DeviceInputs] = None,
                 prev_counts: Optional[torch.Tensor] = None,
                 lru_in: Optional[torch.Tensor] = None, dispatch: str = "static",
                 group_tables: Optional[bool] = None):
        if dispatch not in ("static", "live"):
            raise ValueError(f"unknown dispatch {dispatch!r}")
        self.dispatch = dispatch
        self.wl = wl
        self.device = device
        self.inp = dev_in if dev_in is not None else upload(wl, device)
        J, K, R, P = wl.J, wl.num_keys, wl.R, wl.P
        self.J, self.K, self.R, self.P, self.n = J, K, R, P, wl.n
        self.Ws = [c.W for c in wl.candidates]
        self.max_W = max(self.Ws)
        i32 = dict(dtype=torch.int32, device=device)
        self.err = torch.zeros(1, **i32)
        # plan groups g = 0..NG-1 (interval j -> group gmap[j]); window[g][c] = counts row
        # that candidate c's plan of group g is built from
        self.prev_counts = prev_counts
        pw = getattr(wl, "plan_windows", None)
        if prev_counts is None and pw is None:
            self.counts = torch.empty((J, K), **i32)
            NG = max(J - 1, 1)
            self.win_src = self.counts[:NG]
            gmap = [max(j - 1, 0) for j in range(J)]
            window = [[g] * P for g in range(NG)]
        elif prev_counts is None:
            self.counts = torch.empty((J, K), **i32)
            NG = J
            self.win_src = self.counts
            gmap = list(range(J))
            window = [[int(pw[j][c]) for c in range(P)] for j in range(J)]
            if any(not 0 <= w < J for row in window for w in row):
                raise ValueError("plan_windows names a window outside the stream")
        else:
            if pw is not None:
                raise ValueError("a stream processed in chunks plans every interval from the window before it")
            # row 0 holds the previous chunk's last window, rows 1..J this chunk's counts,
            # so that window g (the plan of interval g) is row g with no copy of the rest
            self.cbuf = torch.empty((J + 1, K), **i32)
            self.counts = self.cbuf[1:]
            NG = J
            self.win_src = self.cbuf[:J]
            gmap = list(range(J))
            window = [[g] * P for g in range(NG)]
        self.NG = NG
        self.gmap_host = gmap
        self.gmap = torch.tensor(gmap, dtype=torch.int32, device=device)
        self.plan_window = [window[g][c] for g in range(NG) for c in range(P)]  # by plan p = g * P + c
        # N_w of every window is its counts row's sum, taken on the device (CR_WINDOW_SUM), and
        # q_cap = (a / b) N_w / R is given relative to the mean per-destination load
        specs = []
        for g in range(NG):
            for c, cand in enumerate(wl.candidates):
                w = window[g][c]
                v = B.PLAN_VARIANTS[getattr(cand, "variant", "full")]
                specs.append((w, cand.W, B.CR_WINDOW_SUM, cand.a, cand.b, v, getattr(cand, "place_seed", 0)))
        # hash-placed ablation stages need cr_place_hash after cr_place_lpt
        self.hash_placed = any(getattr(c, "variant", "full") in ("affinity", "replicated") for c in wl.candidates)
        self.NW = self.win_src.shape[0]  # counts rows the plans are built from
        # Group dispatch tables (one row per request for all candidates) need every
        # candidate of a group to plan from the same window; by default they are used for
        # groups of at least 8 candidates (rows are padded to a multiple of 8) when they fit
        # the budget.
        shared = all(len(set(window[g])) == 1 for g in range(NG))
        if group_tables is None:
            group_tables = (P >= 8 and shared and dispatch == "static" and
                            B.group_table_bytes(NG, P, R, self.max_W, K, self.NW) <= self.GROUP_TABLE_BUDGET)
        elif group_tables and not shared:
            raise ValueError("group dispatch tables need every candidate of a group to share its window")
        self.group_tables = bool(group_tables)
        self.plans = B.PlanSet(specs, P, R, self.max_W, K, self.NW, device, group_tables=self.group_tables)
        self.ws_admit = torch.empty(B.cr_admit_workspace_bytes(self.NW, R, self.max_W), dtype=torch.uint8,
                                    device=device)
        self.ws_replay = torch.empty(B.cr_replay_workspace_bytes(wl.n, P, R), dtype=torch.uint8, device=device)
        # one interval over a key space beyond LDS: counted as one slice (no global atomics)
        self.slice_count = J == 1 and K >= self.SLICE_MIN_KEYS and wl.n > 0
        self.ws_count = (torch.empty(B.cr_count_slice_workspace_bytes(wl.n, K), dtype=torch.uint8, device=device)
                         if self.slice_count else None)
        self.dest = torch.empty((P, max(wl.n, 1)), dtype=torch.int16, device=device)
        soff = getattr(wl, "stat_offsets", None)
        if soff is None:
            self.stat_off, self.JS = self.inp.off, J
        else:
            soff = np.asarray(soff, dtype=np.uint64)
            if soff.ndim != 1 or soff.shape[0] < 2 or soff[0] != 0 or soff[-1] != wl.n or np.any(np.diff(soff.astype(np.int64)) < 0):
                raise ValueError("stat_offsets must rise from 0 to n")
            self.stat_off = torch.from_numpy(soff.view(np.int64).copy()).to(device)
            self.JS = soff.shape[0] - 1
        self.stats = torch.zeros((self.JS, P, R, 4), dtype=torch.int64, device=device)
        self.churn_pairs = None
        self.churn_out = None
        self.lru_in = lru_in
        self.lru_out = torch.empty((P, R, self.max_W), **i32)
        self.first_index = wl.first_index  # global index of the chunk's first request

    def set_inputs(self, dev_in: DeviceInputs):
        """Point the pipeline at another chunk's device inputs (same sizes and intervals)."""
        if dev_in.keys.numel() != self.inp.keys.numel() or not np.array_equal(dev_in.off_host, self.inp.off_host):
            raise ValueError("a chunk must have the same length and interval offsets as the pipeline's")
        if self.stat_off is self.inp.off:
            self.stat_off = dev_in.off
        self.inp = dev_in

    # -- the five calls ----------------------------------------------------------------
    def count(self, stream=None):
        if self.slice_count:
            self.counts.zero_()
            B.cr_count_slice(self.inp.keys, self.K, self.counts, self.err, self.ws_count, stream, n=self.n)
        else:
            B.cr_count_rates(self.inp.keys, self.inp.off, self.J, self.K, self.counts, self.err, stream, n=self.n)
        if self.prev_counts is not None:
            self.cbuf[0].copy_(self.prev_counts)

    def admit(self, stream=None):
        B.cr_admit(self.win_src, self.plans.c, self.ws_admit, self.err, stream)

    def place(self, stream=None):
        B.cr_place_lpt(self.win_src, self.plans.c, stream)
        if self.hash_placed:
            B.cr_place_hash(self.win_src, self.plans.c, stream)

    def plan(self, stream=None):
        self.admit(stream)
        self.place(stream)

    def route(self, stream=None):
        fn = B.cr_route_live if self.dispatch == "live" else B.cr_route
        fn(self.inp.keys, self.first_index, self.wl.seed, self.inp.off, self.gmap, self.J, self.plans.c, self.dest,
           self.err, stream, n=self.n)

    def partition(self, stream=None):
        B.cr_replay_partition(self.inp.keys, self.inp.suffix, self.dest, self.stat_off, self.JS, self.P, self.R,
                              self.Ws, self.ws_replay, self.err, stream, n=self.n)
        self.stats.zero_()  # cr_replay_lru accumulates into it (cleared here so that lru is one kernel)

    def lru(self, stream=None):
        B.cr_replay_lru(self.inp.prefix_len, self.K, self.n, self.JS, self.P, self.R, self.Ws, self.max_W,
                        self.lru_in, self.lru_out, self.stats, self.ws_replay, self.err, stream)

    def replay(self, stream=None):
        self.stats.zero_()
        B.cr_replay(self.inp.keys, self.inp.suffix, self.inp.prefix_len, self.K, self.dest, self.stat_off, self.JS,
                    self.P, self.R, self.Ws, self.max_W, self.lru_in, self.lru_out, self.stats, self.ws_replay,
                    self.err, stream, n=self.n)

    def set_churn_pairs(self, pairs):
        """Plan pairs (p, q), p = group * P + candidate, whose churn ``churn`` measures."""
        pr = np.asarray(pairs, dtype=np.int64).reshape(-1, 2)
        if pr.size and (pr.min() < 0 or pr.max() >= self.plans.num_plans):
            raise ValueError("churn pair names a plan outside the set")
        self.churn_pairs = torch.from_numpy(pr.astype(np.int32)).to(self.device)
        self.churn_out = torch.empty((pr.shape[0], 4), dtype=torch.int64, device=self.device)

    def churn(self, stream=None):
        B.cr_plan_churn(self.plans.c, self.churn_pairs, self.churn_out, self.err, stream)

    STAGES = ("count", "admit", "place", "route", "partition", "lru")

    def step(self, stream=None):
        for s in self.STAGES:
            getattr(self, s)(stream)

    def capture(self):
        """Record one step as a HIP graph (every library call only enqueues kernels on the
        current stream, and the statistics are cleared by a fill kernel, not a memset)."""
        side = torch.cuda.Stream(device=self.device)
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            self.step()
        torch.cuda.current_stream().wait_stream(side)
        self.graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(self.graph):
            self.step()
        return self.graph

    def replay_graph(self):
        self.graph.replay()

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
                    err=int(self.err.cpu().numpy().view(np.uint32)[0]),
                    churn=None if self.churn_out is None else self.churn_out.cpu().numpy().view(np.uint64))

    def plan_of(self, h: dict, g: int, c: int) -> dict:
        """Admitted keys, k and members of plan (group g, candidate c) from host views."""
        p = g * self.P + c
        A = int(h["num_admitted"][p])
        w = self.plan_window[p]
        mo = h["member_off"][p, : A + 1]
        return dict(adm_keys=h["order"][w, :A].copy(), adm_k=np.diff(mo).astype(np.uint32),
                    member_off=mo.copy(), members=h["members"][p, : int(mo[A]) if A else 0].copy(),
                    L=h["load"][p].copy(), cold=int(h["cold"][p]), clamped=int(h["clamped"][p]))


class ChunkStream:
    """Consecutive chunks of one request stream through the path, two HIP streams deep.

    Chunk k (the workload's requests again, at global indices k*n .. k*n + n - 1) is
    counted, planned, routed and partitioned on the plan stream; chunk k-1's LRU replay
    runs on the replay stream from the end of chunk k's admission, beside chunk k's
    placement, routing and partition. `flush()` enqueues the last chunk's replay, which has
    no next chunk to wait for. Chunk k >= 1 plans its first interval from chunk
    k-1's last window and starts its replay from chunk k-1's final cache state, so the
    results are those of processing the chunks one after another. Chunk 0 has its own
    buffers; later chunks alternate between two sets, and a chunk's partition waits for
    the replay of the chunk that used its set before it. Both streams have the default
    priority.
    """

    def __init__(self, wl, device="cuda"):
        self.wl = wl
        self.n = wl.n
        self.inp = upload(wl, device)
        self.first = Pipeline(wl, device, self.inp)
        self.slots = [Pipeline(wl, device, self.inp, prev_counts=self.first.counts[wl.J - 1],
                               lru_in=self.first.lru_out) for _ in range(2)]
        self.s_plan = torch.cuda.Stream(device=device)
        self.s_rep = torch.cuda.Stream(device=device)
        self.ev_part = {}
        self.ev_rep = {}
        self.k = 0
        self.pending = None  # chunk whose replay is not enqueued yet

    def pipe(self, k: int) -> Pipeline:
        return self.first if k == 0 else self.slots[(k - 1) % 2]

    def _run(self, p, stage, stream, timers):
        if timers is None:
            getattr(p, stage)()
            return
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        getattr(p, stage)()
        b.record(stream)
        timers.setdefault(stage, []).append((a, b))

    def _replay(self, after, timers):
        """Enqueue the pending chunk's replay on the replay stream, after its partition and
        (if given) the event `after`."""
        j = self.pending
        if j is None:
            return
        with torch.cuda.stream(self.s_rep):
            self.s_rep.wait_event(self.ev_part.pop(j))
            if after is not None:
                self.s_rep.wait_event(after)
            self._run(self.pipe(j), "lru", self.s_rep, timers)
            ev = torch.cuda.Event()
            ev.record(self.s_rep)
            self.ev_rep[j] = ev
        self.pending = None

    def enqueue(self, timers=None):
        """Enqueue the next chunk. `timers`, if given, maps stage -> list of (start, end)
        events recorded on the stream the stage runs on. The previous chunk's replay is
        enqueued once this chunk's admission is queued, so that it runs beside this chunk's
        placement, routing and partition (placement is a few hundred latency-bound
        wavefronts that leave most of the chip idle) rather than ahead of its counting."""
        k = self.k
        p = self.pipe(k)
        p.first_index = self.wl.first_index + k * self.n
        if k:
            prev = self.pipe(k - 1)
            p.prev_counts = prev.counts[self.wl.J - 1]
            p.lru_in = prev.lru_out
        with torch.cuda.stream(self.s_plan):
            for stage in ("count", "admit"):
                self._run(p, stage, self.s_plan, timers)
            adm = torch.cuda.Event()
            adm.record(self.s_plan)
        self._replay(adm, timers)
        with torch.cuda.stream(self.s_plan):
            for stage in ("place", "route"):
                self._run(p, stage, self.s_plan, timers)
            if k >= 3:  # this buffer set was last replayed by chunk k-2
                self.s_plan.wait_event(self.ev_rep.pop(k - 2))
            self._run(p, "partition", self.s_plan, timers)
            ev = torch.cuda.Event()
            ev.record(self.s_plan)
            self.ev_part[k] = ev
        self.pending = k
        self.k += 1
        return p

    def flush(self, timers=None):
        """Enqueue the last chunk's replay (it has no next chunk to wait for)."""
        self._replay(None, timers)

    def capture(self):
        """Record the steady state as two HIP graphs, one per buffer set. Graph x runs the
        next chunk into set x (count and admission, then placement, routing and partition)
        and, forked onto the replay stream after the admission, the replay of the chunk
        before it, which sits in the other set; the replay stream joins the capture stream
        at the end. Graph launches on one stream run one after another, which orders each
        partition after the replay that last used its set. Replaying the graphs in turn
        continues the chunk sequence; each graph keeps the global indices of the chunk it
        was recorded with. Returns the chunk indices the two graphs were recorded for."""
        while self.k < 3:
            self.enqueue()
        torch.cuda.synchronize()  # chunk k-1's replay is left pending: the first graph runs it
        self.graphs = []
        recorded = []
        for _ in range(2):
            k = self.k
            p, prev = self.pipe(k), self.pipe(k - 1)
            p.first_index = self.wl.first_index + k * self.n
            p.prev_counts = prev.counts[self.wl.J - 1]
            p.lru_in = prev.lru_out
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                cap = torch.cuda.current_stream()
                p.count()
                p.admit()
                self.s_rep.wait_stream(cap)
                with torch.cuda.stream(self.s_rep):
                    prev.lru()
                p.place()
                p.route()
                p.partition()
                cap.wait_stream(self.s_rep)
            self.graphs.append(g)
            recorded.append(k)
            self.k += 1
        self.pending = None
        self.turn = 0
        return recorded

    def replay_graph(self):
        """One step of the captured steady state: the next graph in turn."""
        self.graphs[self.turn].replay()
        self.turn ^= 1

    def graph_pending(self) -> "Pipeline":
        """The buffer set whose chunk was planned by the last graph replay and has not been
        replayed yet (the next graph, or `replay_pending`, replays it)."""
        return self.pipe(self.k - 1 - self.turn)

    def replay_pending(self):
        """Replay, eagerly on the current stream, the chunk the last graph planned."""
        self.graph_pending().lru()


class ChunkStream3:
    """Consecutive chunks of one request stream, three HIP streams deep.

    A chunk goes through four stages: count, admission (with the window sort), B (placement,
    routing and partition) and the LRU replay. Step s runs, at the same time, the admission
    of chunk s on one stream, B of chunk s-1 on a second, and on the third the replay of chunk
    s-2 followed by the count of chunk s+1 (the count is bandwidth-bound and the replay
    vector-bound, and the admission, which waits on the chip's largest blocks, then has a
    stream to itself). A chunk's buffers are in use from its count (step k-1) to its replay
    (step k+2), so chunks 1, 2, ... take four buffer sets in turn (chunk 0 has its own) and
    the work of a step touches four disjoint sets. Eager enqueues order each stage after
    the stages it reads (count(k) before admit(k) before B(k) before replay(k)) and after the
    last users of its set (B of chunk k-4 before count(k) and admit(k), the replay of chunk
    k-4 before B(k)); captured steps run one after another, which gives the same order.
    Chunk k >= 1 plans its first interval from chunk k-1's last window and starts its
    replay from chunk k-1's final cache state, as if the chunks ran one by one.
    """

    NSETS = 4

    def __init__(self, wl, device="cuda"):
        self.wl = wl
        self.n = wl.n
        self.inp = upload(wl, device)
        self.first = Pipeline(wl, device, self.inp)
        self.slots = [Pipeline(wl, device, self.inp, prev_counts=self.first.counts[wl.J - 1],
                               lru_in=self.first.lru_out) for _ in range(self.NSETS)]
        self.streams = [torch.cuda.Stream(device=device) for _ in range(3)]
        self.ev = {}  # (stage, chunk) -> event recorded after that stage
        self.s = 0    # next step
        self.limit = 1 << 62  # chunks from this one on are not started (set by drain)

    def pipe(self, k: int) -> Pipeline:
        return self.first if k == 0 else self.slots[(k - 1) % self.NSETS]

    STAGES = {"count": ("count",), "admit": ("admit",), "B": ("place", "route", "partition"), "lru": ("lru",)}

    def _stage(self, name, k, stream, waits, timers, capturing=False):
        if k < 0 or k >= self.limit:
            return
        p = self.pipe(k)
        with torch.cuda.stream(stream):
            if not capturing:
                for key in waits:
                    e = self.ev.get(key)
                    if e is not None:
                        stream.wait_event(e)
            if name == "count":
                p.first_index = self.wl.first_index + k * self.n
                if k:
                    prev = self.pipe(k - 1)
                    p.prev_counts = prev.counts[self.wl.J - 1]
                    p.lru_in = prev.lru_out
            for stage in self.STAGES[name]:
                if timers is None:
                    getattr(p, stage)()
                else:
                    a = torch.cuda.Event(enable_timing=True)
                    b = torch.cuda.Event(enable_timing=True)
                    a.record(stream)
                    getattr(p, stage)()
                    b.record(stream)
                    timers.setdefault(stage, []).append((a, b))
            if not capturing:
                e = torch.cuda.Event()
                e.record(stream)
                self.ev[(name, k)] = e

    def _enqueue_step(self, s, timers, capturing=False):
        sa, sb, sc = self.streams
        if s == 0:  # chunk 0's count has no step before it
            self._stage("count", 0, sc, [], timers, capturing)
        self._stage("admit", s, sa, [("count", s), ("B", s - 4)], timers, capturing)
        self._stage("B", s - 1, sb, [("admit", s - 1), ("lru", s - 5)], timers, capturing)
        self._stage("lru", s - 2, sc, [("B", s - 2)], timers, capturing)
        self._stage("count", s + 1, sc, [("B", s - 3)], timers, capturing)

    def step(self, timers=None):
        """Enqueue step s. Returns the chunk whose replay this step enqueued (None if none)."""
        s = self.s
        self._enqueue_step(s, timers)
        # events no later enqueue waits for: count(k) is read at step k, admit(k) at k+1,
        # B(k) at steps k+2 .. k+4, lru(k) at step k+5
        for key in (("count", s), ("admit", s - 1), ("B", s - 4), ("lru", s - 5)):
            self.ev.pop(key, None)
        self.s += 1
        return self.pipe(s - 2) if 0 <= s - 2 < self.limit else None

    def drain(self, timers=None):
        """Finish the chunks already admitted (no new chunk is admitted)."""
        self.limit = self.s
        while self.s < self.limit + 2:
            self.step(timers)

    def capture(self):
        """Record the steady state as four HIP graphs (one per step modulo 4), each with the
        three streams forked from the capture stream and joined at the end. Returns the step
        numbers the graphs were recorded for."""
        while self.s < 5:
            self.step()
        torch.cuda.synchronize()
        self.ev.clear()
        self.graphs = []
        recorded = []
        for _ in range(self.NSETS):
            s = self.s
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                cap = torch.cuda.current_stream()
                for st in self.streams:
                    st.wait_stream(cap)
                self._enqueue_step(s, None, capturing=True)
                for st in self.streams:
                    cap.wait_stream(st)
            self.graphs.append(g)
            recorded.append(s)
            self.s += 1
        self.turn = 0
        return recorded

    def replay_graph(self):
        """One step of the captured steady state: the next graph in turn."""
        self.graphs[self.turn].replay()
        self.turn = (self.turn + 1) % self.NSETS


class ChunkChain:
    """Consecutive chunks of one request stream, each with its own inputs, through two
    buffer sets on one stream. Step s runs chunk s: the inputs of ``chunks[s % len]`` at
    global indices s * n .. s * n + n - 1, every interval planned from the window before
    it (chunk s's first interval from chunk s-1's last window; chunk 0's from its own
    first window) and the replay started from chunk s-1's final cache state (empty for
    chunk 0). Every chunk must have the same length and intervals (every window's N_w is
    taken on the device, so the plan specs of the two buffer sets fit every chunk). This is
    how the large sweep streams 1e9 requests as ten 1e8-request chunks.

    With ``overlap`` (the default) a chunk's count, plans, routing and partition run on one
    HIP stream (F) and its replay on a second (L). Step s enqueues on F the count and plans
    of chunk s+1 (chunk 0's front half comes first in step 0), on L the replay of chunk s,
    and on F the routing and partition of chunk s+1, which then run while chunk s is
    replayed. The replay of chunk s waits for its own partition and for the plans of chunk
    s+1: the count and plan kernels are short, latency-bound launches of few blocks, and
    under a replay that keeps every wavefront slot busy they waited up to 13 ms each for
    room, while alone on the chip they take about 10 ms together (the chunk step measured
    146-148 -> 140-142 ms on the large sweep). The partition of chunk s+1 (which rewrites
    the buffer set's records and clears its statistics) waits for the replay of chunk s-1 on
    the same set; everything else a chunk reads was written earlier on its own stream. A
    chunk's results stay in its buffer set until the next step is enqueued. Without
    ``overlap`` every call goes to the caller's stream in order."""

    def __init__(self, chunks, device="cuda", overlap: bool = True):
        self.chunks = list(chunks)
        w0 = self.chunks[0]
        for w in self.chunks[1:]:
            if (w.n, w.num_keys, w.R, w.P) != (w0.n, w0.num_keys, w0.R, w0.P) or \
                    not np.array_equal(np.asarray(w.offsets), np.asarray(w0.offsets)):
                raise ValueError("chunks of a chain must have the same shape and intervals")
        if w0.plan_windows is not None or getattr(w0, "stat_offsets", None) is not None:
            raise ValueError("a chain plans every interval from the window before it")
        self.n = w0.n
        self.inputs = [upload(w, device) for w in self.chunks]
        self.sets = [Pipeline(w0, device, self.inputs[0], prev_counts=torch.empty(0), lru_in=None) for _ in range(2)]
        self.s = 0
        self.overlap = overlap
        if overlap:  # both at the default priority
            self.front = torch.cuda.Stream(device=device)
            self.back = torch.cuda.Stream(device=device)
            self.replayed = [None, None]  # per buffer set: event after its last replay
            self.parted = [None, None]  # per buffer set: event after its last partition
            self.ahead = False  # chunk s's front half is already enqueued

    def pipe(self, s: int) -> Pipeline:
        return self.sets[s % 2]

    def prepare(self, s: int) -> Pipeline:
        """Set up buffer set s % 2 for chunk s (no launches)."""
        p = self.pipe(s)
        p.set_inputs(self.inputs[s % len(self.inputs)])
        p.first_index = s * self.n
        if s == 0:
            p.prev_counts = p.counts[0]  # plan chunk 0's first interval from its own window
            p.lru_in = None
        else:
            prev = self.pipe(s - 1)
            p.prev_counts = prev.counts[prev.J - 1]
            p.lru_in = prev.lru_out
        return p

    def step(self, timers=None, stream=None, on_done=None) -> Pipeline:
        """Enqueue chunk s; returns its buffer set. ``timers`` maps stage -> list of (start,
        end) events. ``on_done(p)`` is called with the set after its replay has been
        enqueued, on the stream that replays it and before the set can be reused, so that
        it may enqueue copies of the chunk's results there. With ``overlap`` the work goes
        to the chain's own streams, after what the caller's stream has enqueued so far (and
        includes the next chunk's front half); synchronize the device (or ``join``) before
        reading results on the host, and read them before the next step."""
        p = self.prepare(self.s)

        def run(q, stage, st):
            if timers is None:
                getattr(q, stage)()
                return
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record(st)
            getattr(q, stage)()
            b.record(st)
            timers.setdefault(stage, []).append((a, b))

        if not self.overlap:
            st = stream if stream is not None else torch.cuda.current_stream()
            for stage in Pipeline.STAGES:
                run(p, stage, st)
            if on_done is not None:
                on_done(p)
            self.s += 1
            return p
        cur = stream if stream is not None else torch.cuda.current_stream()
        F, L = self.front, self.back
        F.wait_stream(cur)
        L.wait_stream(cur)

        def front_plans(q):  # count and plans of a chunk, on F
            with torch.cuda.stream(F):
                for stage in ("count", "admit", "place"):
                    run(q, stage, F)

        def front_rest(q, k):  # routing and partition of a chunk (buffer set k), on F
            with torch.cuda.stream(F):
                run(q, "route", F)
                if self.replayed[k] is not None:
                    F.wait_event(self.replayed[k])  # the last replay on this set is done with it
                run(q, "partition", F)
                ev = torch.cuda.Event()
                ev.record(F)
                self.parted[k] = ev

        k = self.s % 2
        if not self.ahead:  # the first step: chunk s's own front half
            front_plans(p)
            front_rest(p, k)
        nxt = self.prepare(self.s + 1)  # the other buffer set, for chunk s+1
        front_plans(nxt)
        planned = torch.cuda.Event()
        planned.record(F)
        with torch.cuda.stream(L):
            L.wait_event(self.parted[k])
            L.wait_event(planned)
            run(p, "lru", L)
            if on_done is not None:
                on_done(p)
            ev = torch.cuda.Event()
            ev.record(L)
            self.replayed[k] = ev
        front_rest(nxt, 1 - k)
        self.ahead = True
        self.s += 1
        return p

    def join(self, stream=None):
        """Make ``stream`` (default: the current one) wait for everything enqueued so far."""
        if self.overlap:
            st = stream if stream is not None else torch.cuda.current_stream()
            st.wait_stream(self.front)
            st.wait_stream(self.back)
