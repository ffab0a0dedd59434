"""GPU parity: the HIP path through the C ABI against the CPU oracle, element by element.

Bit-exact: counts, admitted keys in order, k, member lists, cold counts, clamp counts,
per-request destinations, per-(interval, candidate, destination) replay statistics and
the carried LRU state. Planned loads: within 1e-9 absolute and, by design, bit-identical.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import pipeline as opipe
from paper_2608_19677_amd import workload as wl_mod
from paper_2608_19677_amd.pipeline import ChunkStream, ChunkStream3, Pipeline

from cr_check import compare_all, compare_plan, say

pytestmark = pytest.mark.gpu


def _run(wl, group_tables=None):
    say(f"[case] {wl.name} n={wl.n} J={wl.J} K={wl.num_keys} R={wl.R} P={wl.P} "
        f"W={[c.W for c in wl.candidates]} group_tables={group_tables}")
    gp = Pipeline(wl, group_tables=group_tables)
    if group_tables is not None:
        assert gp.group_tables == group_tables
    gp.step()
    h = gp.host()
    orc = opipe.run(wl)
    compare_all(wl, gp, h, orc)
    return gp, h, orc


SMALL = [
    # seed, K, n, R, Ws, J, hot, hot_share, qs
    (1, 50, 3000, 7, [4], 3, 0, 0.0, [(1, 1)]),
    (2, 1, 5000, 1, [3], 1, 0, 0.0, [(1, 1)]),
    (3, 200, 20000, 30, [16], 5, 3, 0.5, [(1, 1), (2, 5)]),
    (4, 1000, 100_003, 64, [64, 65, 130, 300, 512], 4, 2, 0.3, [(1, 1)]),
    (5, 5000, 50_000, 1024, [8, 100], 2, 4, 0.4, [(1, 1)]),
    (6, 300, 40_000, 65, [10], 9, 0, 0.0, [(1, 1), (28, 35), (42, 35)]),
    (7, 100, 10, 30, [16], 3, 0, 0.0, [(1, 1)]),
    (8, 400, 30_000, 4, [2, 50], 20, 2, 0.9, [(1, 3)]),
    (9, 2000, 77_777, 16, [128], 6, 8, 0.48, [(2, 5)]),
    (10, 64, 4096, 128, [1, 63, 64], 2, 0, 0.0, [(1, 1)]),
    (11, 300, 20_000, 2, [8, 30], 3, 2, 0.5, [(1, 1)]),         # two destinations: one exchange per merge
    (12, 600, 40_000, 33, [6, 12], 4, 3, 0.4, [(1, 2)]),        # 31 idle lanes in the 64-lane merge
    # 40 keys over two destinations, W = 64 and 48: every segment's rebuild runs through full
    # 64-record batches to the start of the stream without filling the list, so repeated keys
    # are written past q and must be cleared before the replay and the final state
    (13, 40, 20_000, 2, [64, 48], 3, 0, 0.0, [(1, 1)]),
    # 100 keys over two destinations with 130 to 512 slots: the blocked lists never fill,
    # every rebuild reaches the start of the stream with several registers in use
    (14, 100, 30_000, 2, [130, 300, 512], 3, 0, 0.0, [(1, 1)]),
    # 2,000 keys spread thin over 5 destinations, 65 to 257 slots: deep hits and misses in
    # every register, lists filled past one register
    (15, 2000, 60_000, 5, [65, 129, 257], 4, 0, 0.0, [(1, 1)]),
    # 50 keys, one destination, 1e6 requests, every list class: no rebuild ever finds W
    # distinct keys, so every segment from the ninth on runs out of its rebuild budget and
    # is replayed by its stream's sequential pass
    (16, 50, 1_000_000, 1, [60, 100, 200, 512], 5, 0, 0.0, [(1, 1)]),
    # 60 keys over three destinations: long streams, budget exhausted in most segments
    (17, 60, 300_000, 3, [64, 300], 7, 2, 0.5, [(1, 1), (1, 2)]),
    # every list size from 2 to 8 registers, full ones (W = 64 SL) among them: 3,000 keys
    # over six destinations fill every list
    (18, 3000, 120_000, 6, [192, 193, 320, 321, 384, 385, 448, 449], 3, 2, 0.3, [(1, 1)]),
    # 80 keys over two destinations with 150 to 420 slots: no rebuild of the 3- to 7-register
    # lists finds W keys, so their streams go through the sequential pass
    (19, 80, 400_000, 2, [150, 310, 350, 420], 3, 0, 0.0, [(1, 1)]),
]


@pytest.mark.parametrize("case", SMALL, ids=[f"s{c[0]}" for c in SMALL])
def test_small_random_parity(case):
    seed, K, n, R, Ws, J, hot, share, qs = case
    wl = wl_mod.small_random(seed, num_keys=K, n=n, R=R, Ws=Ws, J=J, hot=hot, hot_share=share, qs=qs)
    _run(wl)


MULTI = [c for c in SMALL if len(c[4]) * len(c[8]) > 1]


@pytest.mark.parametrize("case", MULTI, ids=[f"s{c[0]}" for c in MULTI])
@pytest.mark.parametrize("group_tables", [False, True])
def test_multi_candidate_route_paths(case, group_tables):
    # several candidates per plan group: cr_route with the group dispatch tables (one row
    # per request for all candidates) and with the per-plan tables only
    seed, K, n, R, Ws, J, hot, share, qs = case
    wl = wl_mod.small_random(seed, num_keys=K, n=n, R=R, Ws=Ws, J=J, hot=hot, hot_share=share, qs=qs)
    _run(wl, group_tables=group_tables)


def test_group_tables_many_candidates():
    # 100 candidates: two P2C words per destination pair and a padded row (CS = 104)
    Ws = [3, 9, 17, 33, 60]
    qs = [(a, 10) for a in range(5, 25)]
    wl = wl_mod.small_random(15, num_keys=2000, n=30_000, R=70, Ws=Ws, J=3, qs=qs, hot=3, hot_share=0.4)
    _run(wl, group_tables=True)


def test_tiny_intervals_parity():
    # Thousands of intervals of a few requests each (many empty): a 1024-request route block
    # spans hundreds of interval boundaries, and the partition and replay cross one in
    # almost every 64-request chunk.
    _run(wl_mod.small_random(11, num_keys=500, n=50_000, R=30, Ws=[16], J=8000, hot=2, hot_share=0.2))


def test_out_of_range_keys_parity():
    # Keys >= num_keys are not counted, are dispatched as cold, are skipped by the replay
    # and set CR_ERR_KEY_RANGE; everything else matches the oracle.
    wl = wl_mod.small_random(12, num_keys=300, n=30_000, R=16, Ws=[8, 32], J=4, hot=2, hot_share=0.3)
    rng = np.random.default_rng(5)
    bad = rng.choice(wl.n, size=400, replace=False)
    wl.keys = wl.keys.copy()
    wl.keys[bad] = (wl.num_keys + rng.integers(0, 1000, size=bad.size)).astype(np.uint32)
    wl.keys[bad[:5]] = np.uint32(0xFFFFFFFF)
    say(f"[case] out-of-range keys n={wl.n} bad={bad.size}")
    gp = Pipeline(wl)
    gp.step()
    h = gp.host()
    assert h["err"] & 1, "CR_ERR_KEY_RANGE not set"
    h["err"] = 0
    compare_all(wl, gp, h, opipe.run(wl))


def test_empty_stream_parity():
    wl = wl_mod.small_random(13, num_keys=100, n=0, R=8, Ws=[4], J=3)
    _run(wl)


def test_max_candidates_parity():
    # 256 candidate plans (the ABI's maximum) replayed at once
    Ws = list(range(1, 17))
    qs = [(a, 8) for a in range(5, 21)]
    _run(wl_mod.small_random(14, num_keys=300, n=20_000, R=8, Ws=Ws, J=2, qs=qs, hot=1, hot_share=0.2))


def test_tiny_shape_parity():
    gp, h, orc = _run(wl_mod.tiny())
    pl = gp.plan_of(h, 0, 0)
    assert len(pl["adm_keys"]) > 400 and pl["adm_k"].max() > 1


@pytest.mark.timeout(900)
def test_llama70b_shape_full_parity():
    gp, h, orc = _run(wl_mod.llama70b())
    assert h["num_admitted"].max() > 0
    assert np.all(np.diff(h["member_off"][:, :2], axis=1) <= 1)  # every k is 1 on this shape


@pytest.mark.timeout(900)
def test_replication_shape_full_parity():
    gp, h, orc = _run(wl_mod.replication())
    ks = gp.plan_of(h, 3, 0)["adm_k"]
    assert ks[:10].tolist() == [4] + [3] * 8 + [2]


@pytest.mark.timeout(900)
def test_burst_shape_full_parity():
    _run(wl_mod.burst())


def test_chunked_stream_equals_whole_stream():
    # Two chunks split at an interval boundary, the second planned from the first chunk's
    # last window and starting from its carried cache state, equal the uninterrupted run.
    wl = wl_mod.small_random(21, num_keys=3000, n=200_000, R=40, Ws=[24, 200], J=6, hot=2, hot_share=0.2)
    say(f"[case] chunked n={wl.n} J={wl.J}")
    whole = Pipeline(wl)
    whole.step()
    hw = whole.host()
    cut_j = 3
    cut = int(wl.offsets[cut_j])

    def part(s, e, js, je, first):
        off = (wl.offsets[js:je + 1] - wl.offsets[js]).astype(np.uint64)
        return wl_mod.Workload(name="part", num_keys=wl.num_keys, R=wl.R, candidates=wl.candidates,
                               keys=wl.keys[s:e], suffix=wl.suffix[s:e], prefix_len=wl.prefix_len, offsets=off,
                               seed=wl.seed, first_index=first)

    a = part(0, cut, 0, cut_j, 0)
    b = part(cut, wl.n, cut_j, wl.J, cut)
    pa = Pipeline(a)
    pa.step()
    pb = Pipeline(b, prev_counts=pa.counts[a.J - 1].clone(), lru_in=pa.lru_out.clone())
    pb.step()
    ha, hb = pa.host(), pb.host()
    np.testing.assert_array_equal(np.concatenate([ha["dest"], hb["dest"]], axis=1), hw["dest"])
    np.testing.assert_array_equal(np.concatenate([ha["stats"], hb["stats"]], axis=0), hw["stats"])
    np.testing.assert_array_equal(hb["lru"], hw["lru"])
    # and the second chunk's plans equal the oracle's chunked driver
    orc_b = opipe.run(b, lru=[ha["lru"][c, :, :cd.W] for c, cd in enumerate(b.candidates)],
                      counts_prev=ha["counts"][a.J - 1])
    assert hb["err"] == 0
    for (w, c), opl in orc_b["plans"].items():
        compare_plan(pb.plan_of(hb, w, c), opl, f"chunk plan {w}/{c}")
    np.testing.assert_array_equal(hb["stats"], orc_b["stats"])
    np.testing.assert_array_equal(hb["dest"], orc_b["dest"])


def test_repeat_runs_are_identical():
    wl = wl_mod.small_random(31, num_keys=800, n=120_000, R=30, Ws=[32, 96], J=4, hot=3, hot_share=0.3)
    say(f"[case] determinism n={wl.n}")
    gp = Pipeline(wl)
    gp.step()
    h1 = gp.host()
    gp.step()
    h2 = gp.host()
    for k in ("counts", "order", "members", "load", "route", "dest", "stats", "lru"):
        assert np.array_equal(np.asarray(h1[k]).view(np.uint8), np.asarray(h2[k]).view(np.uint8)), k


def _chunk_chain(wl, firsts):
    """Host results of chunks run one by one, chunk i with the global indices of chunk
    firsts[i], each planned from the previous chunk's last window with its cache state."""
    import dataclasses
    ref, prev = [], None
    for f in firsts:
        wk = dataclasses.replace(wl, first_index=wl.first_index + f * wl.n)
        if prev is None:
            p = Pipeline(wk)
        else:
            p = Pipeline(wk, prev_counts=prev.counts[wl.J - 1].clone(), lru_in=prev.lru_out.clone())
        p.step()
        ref.append(p.host())
        prev = p
    return ref


def _same(h, ref, keys, msg):
    assert h["err"] == 0, msg
    for key in keys:
        np.testing.assert_array_equal(np.asarray(h[key]), np.asarray(ref[key]), err_msg=f"{msg} {key}")


def test_three_stream_chunk_pipeline_equals_serial():
    # ChunkStream3 runs, per step, the admission of chunk s, placement + routing + partition
    # of chunk s-1, and the replay of chunk s-2 followed by the count of chunk s+1, on three
    # streams over four buffer sets; seven chunks enqueued without host synchronisation,
    # then drained, must equal the chunks run one after another (the last three chunks'
    # buffer sets are compared)
    wl = wl_mod.small_random(44, num_keys=1800, n=130_000, R=30, Ws=[48], J=5, hot=2, hot_share=0.3)
    say(f"[case] three-stream chunks n={wl.n} J={wl.J}")
    cs = ChunkStream3(wl)
    for _ in range(7):
        cs.step()
    cs.drain()
    torch.cuda.synchronize()
    ref = _chunk_chain(wl, list(range(7)))
    for k in (4, 5, 6):
        pk = cs.pipe(k)
        h = pk.host()
        _same(h, ref[k], ("counts", "load", "dest", "stats", "lru"), f"chunk {k}")
        for g in range(pk.NG):
            for c in range(pk.P):
                compare_plan(pk.plan_of(h, g, c), pk.plan_of(ref[k], g, c), f"chunk {k} plan {g}/{c}")


def test_three_stream_chunk_graphs_equal_eager_chunks():
    # the steady state captured as four HIP graphs (steps 5 .. 8), replayed in turn eight
    # times with eager reads in between; after replay r (step 5 + r) chunk 4 + r is planned,
    # routed and partitioned and chunk 3 + r replayed, each equal to the serial chain.
    # Routing is the only stage that reads the global indices, and each graph keeps those
    # of the chunk it routed when it was recorded (chunks 4 .. 7 in turn)
    wl = wl_mod.small_random(45, num_keys=1500, n=120_000, R=30, Ws=[32], J=4, hot=2, hot_share=0.3)
    say(f"[case] three-stream chunk graphs n={wl.n} J={wl.J}")
    cs = ChunkStream3(wl)
    steps = cs.capture()
    assert steps == [5, 6, 7, 8]
    ref = _chunk_chain(wl, [0, 1, 2, 3, 4, 5, 6, 7, 4, 5, 6, 7])
    for r in range(8):
        cs.replay_graph()
        torch.cuda.synchronize()
        _same(cs.pipe(4 + r).host(), ref[4 + r], ("counts", "load", "dest"), f"replay {r} chunk {4 + r}")
        _same(cs.pipe(3 + r).host(), ref[3 + r], ("stats", "lru"), f"replay {r} chunk {3 + r}")


def test_two_stream_chunk_graphs_equal_eager_chunks():
    # the steady state of the two-stream schedule captured as two HIP graphs (one per buffer
    # set), replayed in turn four times with eager reads and synchronisations in between;
    # every replay's planned chunk and every replayed chunk must equal a serial chain of
    # eager chunks with the same global indices (each graph keeps the indices of the chunk
    # it was recorded with) and the carried cache state
    import dataclasses
    wl = wl_mod.small_random(43, num_keys=1500, n=120_000, R=30, Ws=[32], J=4, hot=2, hot_share=0.3)
    say(f"[case] two-stream chunk graphs n={wl.n} J={wl.J}")
    cs = ChunkStream(wl)
    k0, k1 = cs.capture()
    firsts = [0, 1, 2, k0, k1, k0, k1]  # chunk index whose global indices each chunk uses
    ref, prev = [], None
    for f in firsts:
        wk = dataclasses.replace(wl, first_index=wl.first_index + f * wl.n)
        if prev is None:
            p = Pipeline(wk)
        else:
            p = Pipeline(wk, prev_counts=prev.counts[wl.J - 1].clone(), lru_in=prev.lru_out.clone())
        p.step()
        ref.append(p.host())
        prev = p
    for r in range(4):
        cs.replay_graph()
        torch.cuda.synchronize()
        planned = cs.graph_pending()  # chunk 3 + r, planned by this replay
        h = planned.host()
        assert h["err"] == 0
        for key in ("counts", "load", "dest"):
            np.testing.assert_array_equal(np.asarray(h[key]), np.asarray(ref[3 + r][key]), err_msg=f"replay {r} {key}")
        if r:  # the chunk planned by the previous replay has been replayed by this one
            done = cs.pipe(cs.k - 1 - (cs.turn ^ 1))
            hd = done.host()
            for key in ("stats", "lru"):
                np.testing.assert_array_equal(np.asarray(hd[key]), np.asarray(ref[2 + r][key]),
                                              err_msg=f"replay {r} chunk {2 + r} {key}")
    cs.replay_pending()
    torch.cuda.synchronize()
    hl = cs.graph_pending().host()
    for key in ("stats", "lru"):
        np.testing.assert_array_equal(np.asarray(hl[key]), np.asarray(ref[6][key]), err_msg=f"last chunk {key}")


def test_two_stream_chunk_schedule_equals_serial():
    # ChunkStream plans chunk k on one stream while chunk k-1 replays on another, reusing
    # two buffer sets; five chunks enqueued with no host synchronisation must equal the
    # chunks run one after another (plans from the previous chunk's last window, cache
    # state carried). Buffer sets are reused, so the last two chunks are the ones compared.
    import dataclasses
    wl = wl_mod.small_random(41, num_keys=2000, n=150_000, R=30, Ws=[64], J=5, hot=2, hot_share=0.3)
    say(f"[case] two-stream chunks n={wl.n} J={wl.J}")
    n_chunks = 5
    cs = ChunkStream(wl)
    for _ in range(n_chunks):
        cs.enqueue()
    cs.flush()
    torch.cuda.synchronize()
    prev, ref = None, []
    for k in range(n_chunks):
        wk = dataclasses.replace(wl, first_index=wl.first_index + k * wl.n)
        if prev is None:
            p = Pipeline(wk)
        else:
            p = Pipeline(wk, prev_counts=prev.counts[wl.J - 1].clone(), lru_in=prev.lru_out.clone())
        p.step()
        ref.append(p.host())
        prev = p
    for k in (n_chunks - 2, n_chunks - 1):
        pk = cs.pipe(k)
        h = pk.host()
        assert h["err"] == 0
        for key in ("counts", "load", "dest", "stats", "lru"):
            np.testing.assert_array_equal(np.asarray(h[key]), np.asarray(ref[k][key]), err_msg=f"chunk {k} {key}")
        for g in range(pk.NG):  # order and members are defined up to their used lengths
            for c in range(pk.P):
                compare_plan(pk.plan_of(h, g, c), pk.plan_of(ref[k], g, c), f"chunk {k} plan {g}/{c}")


@pytest.mark.timeout(900)
def test_sweep_chunks_sampled_parity():
    # The 1,024-destination sweep at its full chunk size (1e8 requests, 64 candidates):
    # counts exact; sampled candidates' plans and routing exact for every request; replay
    # exact on a sample of destinations (the per-destination caches are independent).
    from paper_2608_19677_amd import binding as B
    say("[case] sweep chunk 0, n=1e8, P=64, R=1024")
    w0 = wl_mod.sweep_chunk(0)
    gp = Pipeline(w0)
    gp.step()
    torch.cuda.synchronize()
    err = int(gp.err.cpu().numpy().view(np.uint32)[0])
    assert err == 0
    counts = gp.counts.cpu().numpy().view(np.uint32)
    ocounts, _ = oracle.count_rates(w0.keys, w0.offsets, w0.num_keys)
    np.testing.assert_array_equal(counts, ocounts)
    row = ocounts[0]
    n_w = int(row.sum())
    R = w0.R
    stats = gp.stats.cpu().numpy().view(np.uint64)
    lru = gp.lru_out.cpu().numpy().view(np.uint32)
    dsample = np.array([0, 1, 511, 1023] + list(range(200, 204)))
    for c in (0, 7, 27, 63):
        cand = w0.candidates[c]
        say(f"[case] sweep cand {c} W={cand.W} q={cand.a}/{cand.b}")
        keys, ks, cold, clamped = oracle.admit(row, R, cand.W, n_w, cand.a * n_w, cand.b * R)
        members, moff, L = oracle.place_lpt(keys, ks, row, R, cold)
        h = dict(num_admitted=gp.plans.num_admitted.cpu().numpy().view(np.uint32),
                 order=gp.plans.order.cpu().numpy().view(np.uint32),
                 member_off=gp.plans.member_off[c:c + 1].cpu().numpy().view(np.uint32),
                 members=gp.plans.members[c:c + 1].cpu().numpy().view(np.uint16),
                 load=gp.plans.load[c:c + 1].cpu().numpy(),
                 cold=gp.plans.cold[c:c + 1].cpu().numpy().view(np.uint64),
                 clamped=gp.plans.clamped[c:c + 1].cpu().numpy().view(np.uint32))
        A = int(h["num_admitted"][c])
        mo = h["member_off"][0, :A + 1]
        gpl = dict(adm_keys=h["order"][0, :A], adm_k=np.diff(mo).astype(np.uint32), member_off=mo,
                   members=h["members"][0, :int(mo[A])], L=h["load"][0], cold=int(h["cold"][0]),
                   clamped=int(h["clamped"][0]))
        compare_plan(gpl, dict(adm_keys=keys, adm_k=ks, member_off=moff, members=members, L=L, cold=cold,
                               clamped=clamped), f"sweep cand {c}")
        dest_o = oracle.route(w0.keys, w0.first_index, w0.seed, w0.num_keys, R, keys, moff, members, L)
        dest_g = gp.dest[c].cpu().numpy().view(np.uint16)
        np.testing.assert_array_equal(dest_g, dest_o, err_msg=f"dest cand {c}")
        sel = np.isin(dest_o, dsample)
        st, state = oracle.replay(w0.keys[sel], w0.suffix[sel], w0.prefix_len, dest_o[sel],
                                  np.array([0, int(sel.sum())], np.uint64), R, cand.W)
        np.testing.assert_array_equal(stats[0, c, dsample], st[0, dsample], err_msg=f"stats cand {c}")
        np.testing.assert_array_equal(lru[c, dsample, :cand.W], state[dsample])
    # every request is accounted for once per candidate
    assert np.all(stats[0, :, :, 0].sum(axis=1) == w0.n)


LIVE = [
    # seed, K, n, R, Ws, J, hot, hot_share, qs
    (41, 300, 30_000, 7, [8], 4, 3, 0.5, [(1, 1)]),
    (42, 2000, 80_000, 30, [16, 64], 6, 5, 0.4, [(1, 1), (1, 4)]),   # k > 1 members, two candidates
    (43, 500, 20_000, 1, [40], 3, 0, 0.0, [(1, 1)]),                # one destination
    (44, 5000, 60_000, 100, [4], 3, 8, 0.5, [(1, 1)]),              # counts in LDS (R > 64)
    (45, 100, 10, 30, [16], 3, 0, 0.0, [(1, 1)]),                   # intervals shorter than a batch
    (46, 800, 40_000, 16, [2], 2, 2, 0.9, [(1, 20)]),               # k clamped to R
]


@pytest.mark.parametrize("case", LIVE, ids=[f"l{c[0]}" for c in LIVE])
def test_live_dispatch_parity(case):
    # live-load dispatch: every decision on the running loads of its interval
    seed, K, n, R, Ws, J, hot, share, qs = case
    wl = wl_mod.small_random(seed, num_keys=K, n=n, R=R, Ws=Ws, J=J, hot=hot, hot_share=share, qs=qs)
    say(f"[case] live {wl.name} n={wl.n} J={wl.J} R={wl.R} P={wl.P}")
    gp = Pipeline(wl, dispatch="live")
    gp.step()
    compare_all(wl, gp, gp.host(), opipe.run(wl, dispatch="live"))


def test_live_dispatch_70b_gamma_full_parity():
    # the 70B-like stream with Gamma (CV 1.9) arrivals, 1e7 requests, live dispatch
    wl = wl_mod.llama70b_gamma()
    say(f"[case] live {wl.name} n={wl.n} J={wl.J}")
    gp = Pipeline(wl, dispatch="live")
    gp.step()
    compare_all(wl, gp, gp.host(), opipe.run(wl, dispatch="live"))


def test_graph_replays_equal_eager_steps():
    # one step captured as a HIP graph and replayed three times, with eager work between the
    # replays; every replay must reproduce the eager step exactly
    wl = wl_mod.small_random(51, num_keys=900, n=150_000, R=30, Ws=[32, 64], J=6, hot=3, hot_share=0.3)
    say(f"[case] graph n={wl.n} J={wl.J} P={wl.P}")
    gp = Pipeline(wl)
    gp.step()
    ref = gp.host()
    other = Pipeline(wl_mod.small_random(52, num_keys=300, n=40_000, R=16, Ws=[8], J=3))
    gp.capture()
    torch.cuda.synchronize()
    for r in range(3):
        other.step()  # eager work between replays
        gp.err.zero_()
        gp.dest.zero_()
        gp.stats.fill_(7)
        gp.replay_graph()
        h = gp.host()
        for k in ("counts", "order", "num_admitted", "members", "load", "route", "dest", "stats", "lru"):
            assert np.array_equal(np.asarray(h[k]).view(np.uint8), np.asarray(ref[k]).view(np.uint8)), (r, k)
        assert h["err"] == 0
    compare_all(wl, gp, h, opipe.run(wl))
