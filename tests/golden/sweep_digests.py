"""Writes ``sweep_digests.json``: digests of the CPU oracle's results on the large sweep.

The sweep is 1e9 requests in ten 1e8-request chunks (each chunk one control interval),
1,000,000 keys with Zipf(0.9) popularity, 1,024 destinations and 64 candidate plans
(8 warm-slot budgets x 8 load targets).  Chunk k is planned from the counts of chunk
k-1 (chunk 0 from its own) and every candidate's per-destination LRU state is carried
from chunk to chunk.  The oracle's full results (12.8 GB of destinations per chunk)
are too large to store, so this script stores a 64-bit xxh3 digest of every array the
device path must reproduce, plus a few plain totals for reading:

  per chunk:      counts row
  per candidate:  admitted keys, member offsets, members, planned loads (raw f64
                  bytes), A, sum of k, cold, clamped count, destinations of every request,
                  replay statistics [R][4], final LRU state [R][W], and the summed
                  statistics {requests, hits, prefill, hit_prefix}.

Only the input generator and ``oracle/`` are used; the device path is never imported.
Run from the repository root (about 15 minutes on 8 host threads):

    python tests/golden/sweep_digests.py [--chunks 10] [--threads N]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import xxhash

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "sweep_digests.json")


def digest(a) -> str:
    """xxh3-64 of an array's bytes in C order (little endian)."""
    return xxhash.xxh3_64_hexdigest(np.ascontiguousarray(a).tobytes())


def candidate_record(plan: dict, dest: np.ndarray, stats: np.ndarray, lru: np.ndarray) -> dict:
    A = int(plan["adm_keys"].shape[0])
    return dict(
        A=A, sum_k=int(plan["member_off"][A]), cold=int(plan["cold"]), clamped=int(plan["clamped"]),
        adm_keys=digest(plan["adm_keys"].astype(np.uint32)),
        member_off=digest(plan["member_off"][:A + 1].astype(np.uint32)),
        members=digest(plan["members"].astype(np.uint16)),
        load=digest(plan["L"].astype(np.float64)),
        dest=digest(dest.astype(np.uint16)),
        stats=digest(stats.astype(np.uint64)),
        lru=digest(lru.astype(np.uint32)),
        totals=[int(x) for x in stats.sum(axis=0)],
    )


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--chunks", type=int, default=10)
    ap.add_argument("--threads", type=int, default=0)
    args = ap.parse_args()
    import oracle
    from oracle import pipeline as opipe
    from paper_2608_19677_amd import workload

    threads = args.threads or opipe.host_threads()
    rec = dict(
        workload="sweep: 1e6 keys Zipf(0.9), 1e8-request chunks, R = 1024, 64 candidates "
                 "(W in 8..512 log-even x q_cap = (28+2m)/35 of the mean load), hash seed 1, workload seed 2",
        numpy=np.__version__, chunk_n=100_000_000, chunks=[],
    )
    prev_counts = None
    lru = None
    for k in range(args.chunks):
        t0 = time.time()
        w = workload.sweep_chunk(k)
        R, P = w.R, w.P
        counts = opipe.count_fanout(w.keys, w.offsets, w.num_keys, threads)
        src = counts if prev_counts is None else prev_counts[None, :]
        plans = opipe.build_plans(src, R, w.candidates, [(0, c) for c in range(P)], threads)
        if lru is None:
            lru = [np.full((R, c.W), oracle.EMPTY, dtype=np.uint32) for c in w.candidates]
        cands = [None] * P

        def unit(c):
            pl = plans[(0, c)]
            dest = oracle.route(w.keys, w.first_index, w.seed, w.num_keys, R, pl["adm_keys"], pl["member_off"],
                                pl["members"], pl["L"])
            st, state = oracle.replay(w.keys, w.suffix, w.prefix_len, dest, w.offsets, R, w.candidates[c].W, lru[c])
            lru[c] = state
            cands[c] = candidate_record(pl, dest, st[0], state)

        order = sorted(range(P), key=lambda c: -w.candidates[c].W)
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(unit, order))
        rec["chunks"].append(dict(chunk=k, first_index=int(w.first_index), counts=digest(counts[0]), cands=cands))
        prev_counts = counts[0]
        print(f"chunk {k}: {time.time() - t0:.1f} s, threads {threads}", flush=True)
        with open(OUT + ".tmp", "w") as f:
            json.dump(rec, f, indent=0, separators=(",", ":"))
        os.replace(OUT + ".tmp", OUT)


if __name__ == "__main__":
    main()
