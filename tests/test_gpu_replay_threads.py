"""Replay calls from two host threads at once.

cr_replay_lru hands its list sizes' launches to two side streams per device that every call
on the device shares, and a host mutex orders the calls while they enqueue. Two host threads
run whole steps (count, plans, routing, partition, replay) of two different sweep-shaped
workloads (64 candidates, W 8..512, 64 destinations) on their own HIP streams at the same
time, three rounds each; every round's statistics and final cache state must equal the same
workload's step run alone on one thread, bit for bit."""
import threading

import numpy as np
import pytest
import torch

from paper_2608_19677_amd import workload as wl_mod
from paper_2608_19677_amd.pipeline import Pipeline

from cr_check import say

pytestmark = pytest.mark.gpu


def _snap(p):
    return (p.stats.cpu().numpy().copy(), p.lru_out.cpu().numpy().copy(),
            int(p.err.cpu().numpy().view(np.uint32)[0]))


def test_replay_from_two_host_threads():
    wls = [wl_mod.sweep_chunk(k, chunk_n=400_000, num_keys=60_000, R=64) for k in (0, 1)]
    say(f"[case] two host threads, {len(wls)} workloads of {wls[0].n} requests x {wls[0].P} plans")
    torch.cuda.set_device(0)
    pipes = [Pipeline(w, device="cuda") for w in wls]
    ref = []
    for p in pipes:  # each workload alone: every step starts from empty caches
        p.step()
        torch.cuda.synchronize()
        ref.append(_snap(p))
    streams = [torch.cuda.Stream() for _ in pipes]  # default priority
    rounds = 3
    got = [[] for _ in pipes]
    errors = []
    barrier = threading.Barrier(len(pipes), timeout=120)

    def work(i):
        try:
            torch.cuda.set_device(0)
            with torch.cuda.stream(streams[i]):
                for _ in range(rounds):
                    barrier.wait()  # both threads enqueue their steps at the same time
                    pipes[i].step()
                    streams[i].synchronize()
                    got[i].append(_snap(pipes[i]))
        except BaseException as e:  # reported by the main thread
            errors.append(e)
            barrier.abort()

    threads = [threading.Thread(target=work, args=(i,)) for i in range(len(pipes))]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=300)
    assert not any(t.is_alive() for t in threads), "a replay thread did not finish"
    assert not errors, errors
    for i, (s0, l0, e0) in enumerate(ref):
        assert e0 == 0
        assert len(got[i]) == rounds
        assert s0[0, :, :, 0].sum() == wls[i].P * wls[i].n  # every request counted once per plan
        for r, (s1, l1, e1) in enumerate(got[i]):
            assert e1 == 0, (i, r, e1)
            np.testing.assert_array_equal(s1, s0, err_msg=f"workload {i} round {r} stats")
            np.testing.assert_array_equal(l1, l0, err_msg=f"workload {i} round {r} cache state")
