"""Benchmark: count -> plan -> route -> LRU replay on one MI355X, plus the CPU oracle baseline.

Default (--workload sweep): the large sweep, 1e9 requests streamed as ten 1e8-request
chunks (one control interval each) over 1,000,000 keys with Zipf(0.9) popularity and 1,024
destinations, with 64 candidate plans (8 warm-slot budgets x 8 load targets) replayed in
parallel. A step is one chunk: counting, one window sort shared by the 64 admissions, LPT
for all 64 plans, routing of every request under every plan, the partition and the replay,
with the plan taken from the previous chunk's window and every cache state carried. The
default 10 timed steps are one pass over the 1e9-request stream. The chunks are generated
and uploaded before timing; per-stage times are HIP events on the stream the library uses.

Other workloads (--workload llama70b|tiny|replication|burst|drift|ablation|llama70b_gamma)
keep their schedules: by default (--schedule overlap) consecutive batches run as chunks of
one stream, three HIP streams deep (step s counts and admits chunk s, places, routes and
partitions chunk s-1 and replays chunk s-2), timed as replays of that steady state captured
as HIP graphs; --schedule overlap2 is two streams deep; --schedule serial runs every step
from scratch on one stream; --eager times plain launches. --workload drift times the
replanning study, --workload ablation the component ablation; --dispatch live routes by
running loads within each interval; --opaque remaps salted 32-bit ids on the device.

The oracle baseline runs the C oracle with its units fanned out over every host thread
this process may use, on a bounded sample (stated in the line). Prints ONE JSON line.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--schedule ...]
                  [--dispatch static|live] [--opaque] [--no-cpu-baseline] [--cpu-threads N]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E
TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "llama70b_hbm_traffic.md")
KERNEL_SOURCE = {"k_count": "cr_count.hip", "k_sort": "cr_plan.hip", "k_admit": "cr_plan.hip", "k_lpt": "cr_plan.hip",
                 "k_route": "cr_route.hip", "k_part": "cr_replay.hip", "k_scan": "cr_replay.hip",
                 "k_seg": "cr_replay.hip", "k_replay": "cr_replay.hip"}
# 32-bit integer VALU: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz = 39,322 G lane-ops/s.
ALU_PEAK_GOPS = 256 * 4 * 16 * 2.4


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed steps (default: 10 for the sweep, one pass over its 1e9 requests; 20 otherwise)")
    ap.add_argument("--warmup", type=int, default=None, help="untimed steps first (default: 2 sweep, 3 otherwise)")
    ap.add_argument("--workload", default="sweep")
    ap.add_argument("--sweep-serial", action="store_true",
                    help="sweep: every call on one stream in order (kernels alone on the chip, for profiles)")
    ap.add_argument("--sweep-chunks", type=int, default=0,
                    help="sweep: distinct 1e8-request chunks generated and cycled through (default all ten; fewer "
                         "only shortens set-up, for example under a profiler)")
    ap.add_argument("--cpu-threads", type=int, default=0,
                    help="host threads for the oracle baseline (default: every core this process may use)")
    ap.add_argument("--schedule", default="overlap", choices=("overlap", "overlap2", "serial"),
                    help="overlap: consecutive chunks of one stream three HIP streams deep, step s counting and "
                         "admitting chunk s, placing, routing and partitioning chunk s-1 and replaying chunk s-2 "
                         "(cache state and last window carried); overlap2: two streams deep, chunk k placed, "
                         "routed and partitioned while chunk k-1 replays; serial: every step is the whole "
                         "workload from scratch on one stream. The drift study, live dispatch and --opaque run "
                         "serial")
    ap.add_argument("--dispatch", default="static", choices=("static", "live"),
                    help="static: order-independent dispatch on interval-start planned loads; live: least-loaded "
                         "member and power of two choices on the running loads of each interval")
    ap.add_argument("--opaque", action="store_true",
                    help="keys arrive as salted 32-bit ids: every step first builds the device directory and "
                         "remaps the stream to dense keys (timed as stage 'remap')")
    ap.add_argument("--eager", action="store_true",
                    help="time eager launches instead of replays of the step captured as one HIP graph (the "
                         "per-stage times always come from an eager pass; studies and --opaque run eagerly)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-alone", action="store_true",
                    help="sweep: skip timing count and routing alone after the timed steps (keeps a kernel trace "
                         "to the steps' own launches)")
    ap.add_argument("--no-unbatched", action="store_true",
                    help="skip the single unbatched plan build (keeps a kernel trace to the step's own launches)")
    ap.add_argument("--copy-ceiling", action="store_true",
                    help="time plain device-to-device copies that move the count's and routing's "
                         "algorithmic bytes at the 70B-like and sweep sizes, print one JSON line and exit")
    ap.add_argument("--calib-copy-mb", type=int, default=0,
                    help="after timing, copy this many MiB device-to-device once (a plain copy kernel of known "
                         "size, to scale the FETCH_SIZE / WRITE_SIZE counters)")
    return ap.parse_args()


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch of `kernel` from the committed FETCH_SIZE / WRITE_SIZE summary
    (70B-like workload only), or None when the kernel's sources changed since then."""
    import hashlib
    if workload != "llama70b" or not os.path.exists(TRAFFIC_PROFILE):
        return None
    rec = None
    with open(TRAFFIC_PROFILE) as f:
        for line in f:
            if line.startswith("traffic-json: "):
                rec = json.loads(line[len("traffic-json: "):])
    if rec is None or kernel not in rec["bytes_per_launch"]:
        return None
    src = next((v for k, v in KERNEL_SOURCE.items() if kernel.startswith(k)), None)
    if src is None:
        return None
    for rel in ("paper_2608_19677_amd/csrc/" + src, "paper_2608_19677_amd/csrc/cr_common.h"):
        with open(os.path.join(ROOT, rel), "rb") as f:
            if hashlib.sha256(f.read()).hexdigest() != rec["sources_sha256"].get(rel):
                return None
    return rec["bytes_per_launch"][kernel]


def one_plan_build_us(wl, pipe, torch, reps=20, cand=None):
    """One unbatched plan build: cr_admit + cr_place_lpt for a single plan (the first
    interval's window; the first candidate unless `cand` is given), timed with events on the
    current stream."""
    from paper_2608_19677_amd import binding as B
    cand = wl.candidates[0] if cand is None else cand
    n_win = int(wl.offsets[1] - wl.offsets[0])
    ps = B.PlanSet([(0, cand.W, n_win, cand.a * n_win, cand.b * wl.R)], 1, wl.R, cand.W, wl.num_keys, 1,
                   pipe.device)
    ws = torch.empty(B.cr_admit_workspace_bytes(1, wl.R, cand.W), dtype=torch.uint8, device=pipe.device)
    err = torch.zeros(1, dtype=torch.int32, device=pipe.device)
    row = pipe.counts[0:1]
    stream = torch.cuda.current_stream()
    for _ in range(3):
        B.cr_admit(row, ps.c, ws, err, None)
        B.cr_place_lpt(row, ps.c, None)
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(reps):
        B.cr_admit(row, ps.c, ws, err, None)
        B.cr_place_lpt(row, ps.c, None)
    b.record(stream)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    return a.elapsed_time(b) * 1e3 / reps


def describe(name, wl):
    return {
        "workload": {
            "llama70b": "70B-like: 20,000 keys Zipf(1.0) capped at 0.3% share; 1e7 requests, 176 QPS, "
                        "60-s intervals; 30 destinations x 64 LRU slots; q_cap = mean load",
            "tiny": "Tiny: 1,000 keys Zipf(1.1); 1e5 requests, one interval; 30 x 16 slots",
            "replication": "Replication stress: 5,000 Zipf(1.1) + 8 keys at 6%; 2e7 requests, 60-s intervals; "
                           "16 x 128 slots; q_cap = 0.4 x mean",
            "burst": "Burst: 50,000 keys Zipf(1.2), 5% keys 10x for 20 s; 5e7 requests, 100 x 10-s intervals; "
                     "64 x 64 slots",
            "ablation": "Component ablation: 5,000 Zipf(1.1) + 8 keys at 6%; 2e7 requests, 60-s intervals; "
                        "16 x 128 slots; q_cap = 0.4 x mean; candidates flat, affinity (k = 1, hash placement), "
                        "replicated (Eq. 1, hash placement), full (Eq. 1, LPT)",
            "drift": "Replanning under drift: 70B-like keys, lognormal random walk sigma 0.3 over 6 intervals "
                     "of 1e6 requests; 6 candidates (fresh plan, and the plan held one interval at each "
                     "boundary); 30 x 64 slots; 600 statistics bins; churn of consecutive fresh plans",
        }.get(name, name),
        "requests": wl.n, "intervals": wl.J, "plan_builds": None, "keys": wl.num_keys, "destinations": wl.R,
        "slots": [c.W for c in wl.candidates], "candidates": wl.P,
    }


def run_sweep(args):
    """The large sweep: ten 1e8-request chunks (1,000,000 keys, Zipf 0.9, R = 1,024, 64
    candidate plans), one chunk per step through ChunkChain: count, admission for all 64
    candidates from one window sort, LPT, routing of every candidate through the group
    tables, partition and replay, with the plan taken from the previous chunk's window and
    the cache state carried; chunk s+1's front half runs on a second HIP stream while chunk s
    is replayed. Step s runs the inputs of chunk s mod 10 at global indices s * 1e8 onwards.
    The chunks are generated and uploaded before timing; the timed region starts and ends
    with the device idle, so its K steps are K whole chunks."""
    import numpy as np
    import torch

    from paper_2608_19677_amd import workload
    from paper_2608_19677_amd.pipeline import ChunkChain, Pipeline

    steps = 10 if args.steps is None else args.steps
    warmup = 2 if args.warmup is None else args.warmup
    nchunks = args.sweep_chunks or workload.SWEEP_CHUNKS
    chunks = [workload.sweep_chunk(k) for k in range(nchunks)]
    w0 = chunks[0]
    torch.cuda.set_device(0)
    chain = ChunkChain(chunks, device="cuda:0", overlap=not args.sweep_serial)
    for _ in range(warmup):
        chain.step()
    torch.cuda.synchronize()
    ev = {}
    t0 = time.perf_counter()
    last = None
    for _ in range(steps):
        last = chain.step(timers=ev)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / steps
    stage_ms = {s: float(np.mean([a.elapsed_time(b) for a, b in ev[s]])) for s in Pipeline.STAGES}
    err = int(last.err.cpu().numpy().view(np.uint32)[0])
    assert err == 0, f"device error word {err:#x}"
    n, P, R = w0.n, w0.P, w0.R
    st = last.stats.cpu().numpy().view(np.uint64).sum(axis=(0, 2)).astype(np.float64)  # [P][4]
    hit = st[:, 1] / st[:, 0]
    Ws = np.array([c.W for c in w0.candidates], dtype=np.float64)
    # replay: per record a W-slot compare, and on a miss a W-wide reduction for the victim
    lru_work = float(np.sum(n * Ws * (2.0 - hit)))
    kern = {
        "count": dict(kernel="k_count_*", bound="hbm", unit="GB/s", work=4.0 * n, peak=HBM_PEAK_GBS),
        "route": dict(kernel="k_route_group<true,1> + group tables", bound="hbm", unit="GB/s",
                      work=(4.0 + 2.0 * P) * n, peak=HBM_PEAK_GBS),
        "lru": dict(kernel="k_replay<1..8> (one cr_replay_lru call)", bound="alu", unit="Glane-op/s",
                    work=lru_work, peak=ALU_PEAK_GOPS),
    }
    for k, v in kern.items():
        v["ms"] = stage_ms[k]
        v["achieved"] = v["work"] / (stage_ms[k] * 1e-3) / 1e9
        v["frac"] = v["achieved"] / v["peak"]
    # Under the default schedule the count and routing events also time the wait for room on a
    # chip the replay of the previous chunk fills. After the timed steps each call runs again
    # on the idle device (same inputs; counts into a scratch row, routing rewrites the same
    # destinations), for their own rooflines.
    from paper_2608_19677_amd import binding as B
    scratch = torch.zeros_like(last.counts)

    def alone(fn, reps=5):
        ts = []
        for _ in range(reps):
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b))
        return float(np.median(ts))

    if not args.no_alone:
        if last.slice_count:
            count_alone = alone(lambda: B.cr_count_slice(last.inp.keys, last.K, scratch, last.err, last.ws_count,
                                                         None, n=last.n))
        else:
            count_alone = alone(lambda: B.cr_count_rates(last.inp.keys, last.inp.off, last.J, last.K, scratch,
                                                         last.err, None, n=last.n))
        for k, ms in (("count", count_alone), ("route", alone(last.route))):
            v = kern[k]
            v["ms_alone"] = ms
            v["achieved_alone"] = v["work"] / (ms * 1e-3) / 1e9
            v["frac_alone"] = v["achieved_alone"] / v["peak"]
        err = int(last.err.cpu().numpy().view(np.uint32)[0])
        assert err == 0, f"device error word {err:#x} after the calls alone"
    d = kern["lru"]
    out = {
        "metric": "requests/sec through count+route+LRU replay",
        "value": n / (ms_step * 1e-3),
        "unit": "requests/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32",
        "data": "synthetic",
        "config": {
            "workload": "Large sweep: 1,000,000 keys Zipf(0.9); 1e9 requests streamed in ten 1e8-request chunks "
                        "(one control interval each); 1,024 destinations; 64 candidate plans = 8 warm-slot budgets "
                        "(8..512 per destination) x 8 load targets (0.8..1.2 x mean), replayed in parallel",
            "requests_per_step": n, "chunks": workload.SWEEP_CHUNKS, "keys": w0.num_keys, "destinations": R,
            "slots": sorted({c.W for c in w0.candidates}), "candidates": P, "plan_builds_per_step": P,
            "schedule": "chunk chain, one stream" if args.sweep_serial else
                        "chunk chain, two HIP streams (count, plans, routing, partition of chunk s+1 "
                        "under the replay of chunk s)", "dispatch": "static", "launch": "eager",
        },
        "roofline": {"bound": d["bound"], "achieved": d["achieved"], "peak": d["peak"], "unit": d["unit"],
                     "frac": d["frac"], "traffic": sweep_traffic(), "kernel": d["kernel"]},
        "request_plans_per_s": n * P / (ms_step * 1e-3),
        "us_per_plan_build": (stage_ms["admit"] + stage_ms["place"]) * 1e3 / P,
        "stage_ms": stage_ms,
        "kernels": {k: {kk: vv for kk, vv in v.items() if kk != "work"} for k, v in kern.items()},
        "hbm_frac": ({"count": kern["count"]["frac_alone"], "route": kern["route"]["frac_alone"],
                      "measured": "each call alone on the idle device after the timed steps"} if not args.no_alone else
                     {"count": kern["count"]["frac"], "route": kern["route"]["frac"],
                      "measured": "HIP events of the timed steps"}),
        "hit_rate": {"min": float(hit.min()), "max": float(hit.max())},
    }
    if args.calib_copy_mb:
        nb = args.calib_copy_mb << 20
        src = torch.empty(nb, dtype=torch.uint8, device="cuda:0")
        dst = torch.empty_like(src)
        src.fill_(1)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        out["calib_copy_bytes"] = nb
    if not args.no_unbatched:
        # one plan alone: the largest budget (W = 512, C = 524,288) at the mean load target
        big = max(w0.candidates, key=lambda c: (c.W, -abs(c.a - c.b)))
        out["us_one_plan_build"] = one_plan_build_us(w0, last, torch, cand=big)
        out["one_plan_build"] = f"W = {big.W}, q_cap = {big.a}/{big.b} x mean, window of {w0.n:,} requests"
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = sweep_cpu_baseline(args, chunks[0])
    return out


def check_graph_errors(gs):
    """The device error words of every buffer set a captured schedule used (they accumulate
    over the replays): zero, or the bench stops."""
    import numpy as np
    for p in [gs.first] + list(gs.slots):
        e = int(p.err.cpu().numpy().view(np.uint32)[0])
        assert e == 0, f"device error word {e:#x} after the graph replays"


def sweep_traffic():
    """HBM bytes per replay stage from the committed counter summary of the sweep, or None
    when the replay's sources changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "sweep_counters.md")
    if not os.path.exists(path):
        return None
    rec = None
    with open(path) as f:
        for line in f:
            if line.startswith("traffic-json: "):
                rec = json.loads(line[len("traffic-json: "):])
    if rec is None or "lru" not in rec.get("bytes_per_step", {}):
        return None
    for rel, sha in rec["sources_sha256"].items():
        with open(os.path.join(ROOT, rel), "rb") as f:
            if hashlib.sha256(f.read()).hexdigest() != sha:
                return None
    return rec["bytes_per_step"]["lru"]


def sweep_cpu_baseline(args, w0):
    """The oracle, fanned out over this host's threads, on one chunk of the sweep: chunk 0
    (1e8 requests, one window) through count, 64 plans, routing and replay of every
    candidate, timed end to end (about 15 s on 16 threads)."""
    from oracle import pipeline as opipe
    S = int(w0.n)
    ws = w0
    threads = args.cpu_threads or opipe.host_threads()
    tm = {}
    t = time.perf_counter()
    opipe.run(ws, threads=threads, timings=tm)
    sec = time.perf_counter() - t
    return {"value": S / sec, "unit": "requests/s", "cores": threads, "kind": "oracle",
            "sample": f"sweep chunk 0 ({S:,} requests, one window), all 64 candidates "
                      f"(count, plans, route, replay), {sec:.1f} s on {threads} host threads; stages (s) "
                      + ", ".join(f"{k} {v:.2f}" for k, v in tm.items() if k in ("count", "plan", "route", "replay"))}


def copy_ceiling():
    """Plain device-to-device copies (the runtime's copy kernel behind torch's copy_) that move
    as many bytes as the count and routing kernels' algorithmic traffic at the sizes they run
    at: half read, half written. What a copy of that size reaches is a practical ceiling for
    an HBM-bound kernel moving the same bytes in one launch."""
    import numpy as np
    import torch
    torch.cuda.set_device(0)
    cases = [("count, 70B-like: 1e7 requests x 4 B", 40e6), ("route, 70B-like: 1e7 x (4 + 2) B", 60e6),
             ("count, sweep chunk: 1e8 x 4 B", 4e8), ("route, sweep chunk: 1e8 x (4 + 2 x 64) B", 13.2e9)]
    out = []
    for name, moved in cases:
        nb = int(moved) // 2
        src = torch.empty(nb, dtype=torch.uint8, device="cuda:0")
        src.fill_(1)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        ts = []
        for _ in range(20 if moved < 1e9 else 5):
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record()
            dst.copy_(src)
            b.record()
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b))
        ms = float(np.median(ts))
        out.append({"case": name, "bytes_moved": 2 * nb, "us_events": ms * 1e3,
                    "frac_of_8TB_s": 2 * nb / (ms * 1e-3) / (HBM_PEAK_GBS * 1e9)})
        del src, dst
    return {"copy_ceiling": out, "peak_GB_s": HBM_PEAK_GBS}


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "one GPU only: the path runs on a single MI355X and has no multi-GPU "
                                   "sharding", "n_gpus": args.gpus}), flush=True)
        sys.exit(2)
    if args.copy_ceiling:
        print(json.dumps(copy_ceiling()), flush=True)
        return
    if args.workload == "sweep":
        from paper_2608_19677_amd import build as hip_build
        if not os.path.exists(hip_build.LIB):
            hip_build.build()
        print(json.dumps(run_sweep(args)), flush=True)
        return
    if args.steps is None:
        args.steps = 20
    if args.warmup is None:
        args.warmup = 3
    import numpy as np
    import torch

    from paper_2608_19677_amd import build as hip_build
    if not os.path.exists(hip_build.LIB):
        hip_build.build()
    from paper_2608_19677_amd import workload
    from paper_2608_19677_amd.pipeline import ChunkStream, ChunkStream3, Pipeline

    wl = workload.CONFIGS[args.workload]()
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    study = None
    stages = Pipeline.STAGES
    if args.workload == "drift":
        from paper_2608_19677_amd.replan import DriftStudy
        study = DriftStudy(wl, device="cuda:0")
        stages = DriftStudy.STAGES
        args.schedule = "serial"  # its plans come from named windows, not from the previous chunk
    if args.dispatch == "live":
        args.schedule = "serial"
    remap = None
    if args.opaque:
        if study is not None:
            raise SystemExit("--opaque runs the plain path only")
        from paper_2608_19677_amd.keymap import KeyMap, to_device
        from paper_2608_19677_amd.pipeline import DeviceInputs
        args.schedule = "serial"
        op = workload.opaque(wl)
        km = KeyMap(wl.num_keys, device="cuda:0")
        d_ids = to_device(op.ids, "cuda:0")
        dense = torch.empty_like(d_ids)
        plen = torch.zeros(wl.num_keys, dtype=torch.int32, device="cuda:0")
        km_err = torch.zeros(1, dtype=torch.int32, device="cuda:0")
        km.build(d_ids, km_err)
        km.scatter(to_device(op.attr_ids, "cuda:0"), to_device(op.prefix_by_id, "cuda:0"), plen)
        dev_in = DeviceInputs(keys=dense, suffix=torch.from_numpy(wl.suffix.view(np.int16)).to(dev), prefix_len=plen,
                              off=torch.from_numpy(wl.offsets.view(np.int64)).to(dev),
                              off_host=wl.offsets.astype(np.uint64))

        class _Remap:
            def remap(self, stream=None):
                km.build(d_ids, km_err, stream)
                km.lookup(d_ids, dense, stream)

        remap = _Remap()
        stages = ("remap",) + tuple(stages)
    ev = {s: [] for s in stages}
    if args.schedule == "serial":
        if remap is not None:
            gp = Pipeline(wl, device="cuda:0", dev_in=dev_in, dispatch=args.dispatch)
            gp.remap = remap.remap
        else:
            gp = study.pipe if study is not None else Pipeline(wl, device="cuda:0", dispatch=args.dispatch)
        stream = torch.cuda.current_stream()
        for _ in range(args.warmup):
            for s in stages:
                getattr(gp, s)()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            for s in stages:
                a = torch.cuda.Event(enable_timing=True)
                b = torch.cuda.Event(enable_timing=True)
                a.record(stream)
                getattr(gp, s)()
                b.record(stream)
                ev[s].append((a, b))
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        last = gp
        if not args.eager and study is None and remap is None:
            # the step as one HIP graph: replays replace the eager launches in the timed region
            gp.capture()
            for _ in range(args.warmup):
                gp.replay_graph()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(args.steps):
                gp.replay_graph()
            torch.cuda.synchronize()
            t1 = time.perf_counter()
    elif args.schedule == "overlap":
        cs = ChunkStream3(wl, device="cuda:0")
        for _ in range(args.warmup):
            cs.step()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            cs.step(timers=ev)
        cs.drain(timers=ev)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        last = cs.pipe(cs.limit - 1)
        if not args.eager:
            # the steady state as three HIP graphs (steps modulo 3), replayed in turn: each
            # replay counts and admits one chunk, places, routes and partitions the one before
            # and replays the one before that
            gs = ChunkStream3(wl, device="cuda:0")
            gs.capture()
            for _ in range(args.warmup):
                gs.replay_graph()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(args.steps):
                gs.replay_graph()
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            check_graph_errors(gs)
    else:
        cs = ChunkStream(wl, device="cuda:0")
        for _ in range(args.warmup):
            cs.enqueue()
        cs.flush()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            last = cs.enqueue(timers=ev)
        cs.flush(timers=ev)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        if not args.eager:
            # the steady state as two HIP graphs (one per buffer set), replayed in turn: each
            # replay plans, routes and partitions one chunk beside the previous chunk's replay
            gs = ChunkStream(wl, device="cuda:0")
            gs.capture()
            for _ in range(args.warmup):
                gs.replay_graph()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(args.steps):
                gs.replay_graph()
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            check_graph_errors(gs)
    n_plans = last.plans.num_plans
    ms_step = (t1 - t0) * 1e3 / args.steps
    one_build_us = None if args.no_unbatched else one_plan_build_us(wl, last, torch)
    stage_ms = {s: float(np.mean([a.elapsed_time(b) for a, b in ev[s]])) for s in stages}
    h = last.host()
    assert h["err"] == 0, f"device error word {h['err']:#x}"
    tot = h["stats"].sum(axis=(0, 2)).astype(np.float64)

    n, P, R = wl.n, wl.P, wl.R
    n_adm = int(h["member_off"][np.arange(n_plans), h["num_admitted"].astype(np.int64)].astype(np.int64).sum())
    # Algorithmic work per launch of the single-kernel calls (the statistics are cleared in
    # the partition stage; count, place, route and lru each launch exactly one kernel here).
    kern = {
        # counting reads every key once: 4 B per request
        "count": dict(kernel="k_count_*", bound="hbm", unit="GB/s", work=4.0 * n, peak=HBM_PEAK_GBS),
        "route": dict(kernel="k_route<true>" if args.dispatch == "static" else "k_route_live<%s>" % (
            "false" if R <= 64 else "true"), bound="hbm", unit="GB/s", work=(4.0 + 2.0 * P) * n, peak=HBM_PEAK_GBS),
        # LPT: every job copy is compared against the R destination loads.
        "place": dict(kernel="k_lpt_small", bound="alu", unit="Glane-op/s", work=float(n_adm) * R,
                      peak=ALU_PEAK_GOPS),
        # LRU: every request compares its key with the W slots and moves up to W of them one
        # place (a move-to-front list: one compare and one shift per slot).
        "lru": dict(kernel="k_replay<%d, %s, false>" % (lambda sl: (sl, "true" if sl >= 5 else "false"))(
                        max((c.W + 63) // 64 for c in wl.candidates)), bound="alu", unit="Glane-op/s",
                    work=float(sum(2.0 * c.W for c in wl.candidates)) * n, peak=ALU_PEAK_GOPS),
    }
    for k, v in kern.items():
        sec = stage_ms[k] * 1e-3
        v["ms"] = stage_ms[k]
        v["achieved"] = v["work"] / sec / 1e9
        v["frac"] = v["achieved"] / v["peak"]
    # Serial schedule: the stage with the longest time. Overlapped schedules: the replay, the
    # largest kernel by device time in their kernel traces; there a stage's HIP-event time
    # also counts the wait for room on a chip that the other streams' kernels fill.
    dominant = max(kern, key=lambda k: kern[k]["ms"]) if args.schedule == "serial" else "lru"
    d = kern[dominant]

    out = {
        "metric": "requests/sec through count+route+LRU replay",
        "value": n / (ms_step * 1e-3),
        "unit": "requests/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32",
        "data": "synthetic",
        "config": describe(args.workload, wl),
        "roofline": {"bound": d["bound"], "achieved": d["achieved"], "peak": d["peak"], "unit": d["unit"],
                     "frac": d["frac"], "traffic": measured_traffic(d["kernel"], args.workload),
                     "kernel": d["kernel"]},
        "us_per_plan_build": (stage_ms["admit"] + stage_ms["place"]) * 1e3 / n_plans,
        "us_one_plan_build": one_build_us,
        "stage_ms": stage_ms,
        "kernels": {k: {kk: vv for kk, vv in v.items() if kk != "work"} for k, v in kern.items()},
        "hbm_frac": {"count": kern["count"]["frac"], "route": kern["route"]["frac"]},
        "hit_rate": (tot[:, 1] / tot[:, 0]).tolist(),
    }
    out["config"]["plan_builds"] = n_plans
    out["config"]["schedule"] = args.schedule
    out["config"]["dispatch"] = args.dispatch
    out["config"]["launch"] = "eager" if (args.eager or study is not None or remap is not None) else "hip-graph"
    if remap is not None:
        torch.cuda.synchronize()
        assert int(km_err.item()) == 0
        out["config"]["keys"] = "salted 32-bit ids, remapped on the device every step"
        out["kernels"]["remap"] = {"ms": stage_ms["remap"], "kernel": "k_km_*",
                                   "achieved_GBps": 12.0 * n / (stage_ms["remap"] * 1e-3) / 1e9}
    if study is not None:
        out["study"] = study.summary()
        out["kernels"]["churn"] = {"ms": stage_ms["churn"], "kernel": "k_plan_churn"}
    if args.workload == "ablation":
        from paper_2608_19677_amd.report import ablation_summary
        out["study"] = ablation_summary(wl, h["stats"], h["load"], last.gmap_host)

    if args.calib_copy_mb:
        nb = args.calib_copy_mb << 20
        src = torch.empty(nb, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        src.fill_(1)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        out["calib_copy_bytes"] = nb

    if not args.no_cpu_baseline:
        from oracle import pipeline as opipe
        threads = args.cpu_threads or opipe.host_threads()
        times = []
        t_start = time.perf_counter()
        while True:
            s = time.perf_counter()
            opipe.run(wl, dispatch=args.dispatch, threads=threads)
            times.append(time.perf_counter() - s)
            if time.perf_counter() - t_start > args.cpu_seconds or len(times) >= 10:
                break
        med = float(np.median(times))
        out["cpu_baseline"] = {"value": n / med, "unit": "requests/s", "cores": threads, "kind": "oracle",
                               "sample": f"the full workload, {len(times)} passes, median "
                                         f"{med:.3f} s per pass (C oracle, units fanned out over {threads} "
                                         f"host threads)"}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
