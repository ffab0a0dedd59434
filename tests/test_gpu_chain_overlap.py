"""The two-stream chunk chain equals the one-stream chain.

``ChunkChain`` overlaps chunk s+1's count, plans, routing and partition (one HIP stream)
with chunk s's replay (a second stream) over two buffer sets. Five chunks of a smaller
sweep-shaped stream (64 candidates, W 8..512, 64 destinations) are enqueued back to back
without synchronizing; each chunk's statistics, final cache state and error word are copied
on the replay stream as soon as its replay is enqueued (before its buffer set can be
reused), and compared with the same chunks run one stream in order. Both with and without
the grouped replay of the small caches."""
import numpy as np
import pytest
import torch

from paper_2608_19677_amd import binding as B
from paper_2608_19677_amd import workload as wl_mod
from paper_2608_19677_amd.pipeline import ChunkChain

from cr_check import say

pytestmark = pytest.mark.gpu


def _run(chunks, overlap, steps):
    chain = ChunkChain(chunks, device="cuda", overlap=overlap)
    out = []

    def keep(p):
        out.append((p.stats.clone(), p.lru_out.clone(), p.err.clone()))

    for _ in range(steps):
        chain.step(on_done=keep)
    torch.cuda.synchronize()
    return [(s.cpu().numpy(), l.cpu().numpy(), int(e.cpu().numpy().view(np.uint32)[0])) for s, l, e in out]


@pytest.mark.parametrize("grouped", [False, True], ids=["one-list-per-wavefront", "grouped"])
def test_two_stream_chain_equals_one_stream(grouped):
    chunks = [wl_mod.sweep_chunk(k, chunk_n=400_000, num_keys=60_000, R=64) for k in range(3)]
    say(f"[case] chain overlap, grouped={grouped}: 5 steps over {len(chunks)} chunks of {chunks[0].n}")
    B.cr_replay_set_group_min_records(0 if grouped else 1 << 62)
    try:
        ref = _run(chunks, overlap=False, steps=5)
        got = _run(chunks, overlap=True, steps=5)
    finally:
        B.cr_replay_set_group_min_records(B.GROUP_MIN_RECORDS_DEFAULT)
    for k, ((s0, l0, e0), (s1, l1, e1)) in enumerate(zip(ref, got)):
        assert e0 == 0 and e1 == 0, (k, e0, e1)
        np.testing.assert_array_equal(s1, s0, err_msg=f"chunk {k} stats")
        np.testing.assert_array_equal(l1, l0, err_msg=f"chunk {k} cache state")
        assert s0[0, :, :, 0].sum() == chunks[0].P * chunks[0].n  # every request counted once per plan
