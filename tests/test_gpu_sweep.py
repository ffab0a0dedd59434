"""GPU parity on the large sweep at full size: 1e9 requests in ten 1e8-request chunks,
1,000,000 keys, R = 1,024, 64 candidate plans, run through ``ChunkChain`` exactly as
``bench.py`` runs it (two buffer sets, plans from the previous chunk's window, LRU state
carried from chunk to chunk).

Every array the path produces is compared with the CPU oracle through the xxh3-64 digests
that ``tests/golden/sweep_digests.py`` (oracle only) stored: counts, and for every chunk and
candidate the admitted keys in order, member offsets, members, planned loads (raw bits),
A, cold, clamp count, all 1e8 destinations, the replay statistics of every destination and
the final LRU state of every destination."""
import json
import os

import numpy as np
import pytest
import torch
import xxhash

from paper_2608_19677_amd import workload as wl_mod
from paper_2608_19677_amd.pipeline import ChunkChain

from cr_check import say

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "sweep_digests.json")


def _digest(a) -> str:
    return xxhash.xxh3_64_hexdigest(np.ascontiguousarray(a).tobytes())


def _u(t, dt):
    return t.cpu().numpy().view(dt)


def check_chunk(p, ck, where):
    """Mismatches between buffer set p (a chunk just run) and the chunk's stored digests."""
    torch.cuda.synchronize()
    bad = []
    if int(_u(p.err, np.uint32)[0]) != 0:
        bad.append(f"{where}: device error word {int(_u(p.err, np.uint32)[0]):#x}")
    if _digest(_u(p.counts[0], np.uint32)) != ck["counts"]:
        bad.append(f"{where}: counts")
    ps = p.plans
    A_all = _u(ps.num_admitted, np.uint32)
    cold = _u(ps.cold, np.uint64)
    clamped = _u(ps.clamped, np.uint32)
    for c, oc in enumerate(ck["cands"]):
        A = int(A_all[c])
        w = p.plan_window[c]
        mo = _u(ps.member_off[c, :A + 1], np.uint32)
        got = dict(
            A=A, sum_k=int(mo[A]), cold=int(cold[c]), clamped=int(clamped[c]),
            adm_keys=_digest(_u(ps.order[w, :A], np.uint32)), member_off=_digest(mo),
            members=_digest(_u(ps.members[c, :int(mo[A])], np.uint16)),
            load=_digest(ps.load[c].cpu().numpy()),
            dest=_digest(_u(p.dest[c, :p.n], np.uint16)),
            stats=_digest(_u(p.stats[0, c], np.uint64)),
            lru=_digest(_u(p.lru_out[c, :, :p.Ws[c]], np.uint32)),
        )
        for key, val in got.items():
            if val != oc[key]:
                bad.append(f"{where} cand {c}: {key} {val} != oracle {oc[key]}")
        tot = [int(x) for x in _u(p.stats[0, c], np.uint64).sum(axis=0)]
        if tot != oc["totals"]:
            bad.append(f"{where} cand {c}: totals {tot} != oracle {oc['totals']}")
    return bad


@pytest.mark.timeout(1100)
def test_sweep_full_stream_matches_oracle():
    rec = json.load(open(GOLDEN))
    assert rec["numpy"] == np.__version__, "inputs would differ: regenerate tests/golden/sweep_digests.json"
    chunks = [wl_mod.sweep_chunk(k) for k in range(len(rec["chunks"]))]
    say(f"[case] sweep chain: {len(chunks)} chunks of {chunks[0].n}, P={chunks[0].P}, R={chunks[0].R}")
    chain = ChunkChain(chunks, device="cuda")
    assert all(p.group_tables for p in chain.sets)
    bad = []
    for k, ck in enumerate(rec["chunks"]):
        p = chain.step()
        assert p.first_index == ck["first_index"]
        bad += check_chunk(p, ck, f"chunk {k}")
        say(f"[chunk {k}] mismatches so far: {len(bad)}")
    assert not bad, "\n".join(bad[:40])
