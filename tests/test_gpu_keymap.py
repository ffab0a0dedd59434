"""GPU parity for the opaque-key directory (cr_keymap_*) against the oracle's remap, and
the whole path run on remapped keys against the oracle run on the oracle's remap."""
import numpy as np
import pytest
import torch

from oracle import keymap as okm
from oracle import pipeline as opipe
from paper_2608_19677_amd import binding as B
from paper_2608_19677_amd import workload as wl_mod
from paper_2608_19677_amd.keymap import KeyMap, to_device
from paper_2608_19677_amd.pipeline import DeviceInputs, Pipeline

from cr_check import compare_all, say

pytestmark = pytest.mark.gpu


def _remap_gpu(ids: np.ndarray, capacity: int):
    km = KeyMap(capacity)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    d_ids = to_device(ids)
    km.build(d_ids, err)
    dense = torch.empty_like(d_ids)
    km.lookup(d_ids, dense)
    torch.cuda.synchronize()
    return km, dense, int(km.num_keys.item()), int(err.item()) & 0xFFFFFFFF


@pytest.mark.parametrize("case", [(1, 5000, 300), (2, 200_000, 20_000), (3, 1, 1), (4, 100_003, 100_003)],
                         ids=["zipf", "many", "one", "all-distinct"])
def test_keymap_matches_first_occurrence(case):
    seed, n, distinct = case
    rng = np.random.default_rng(seed)
    pool = np.unique(rng.integers(0, 2**32 - 1, size=distinct * 2, dtype=np.uint64).astype(np.uint32))[:distinct]
    pool = rng.permutation(pool)
    idx = rng.zipf(1.2, size=n) % len(pool) if case[0] != 4 else rng.permutation(n) % len(pool)
    ids = pool[idx].astype(np.uint32)
    say(f"[case] keymap n={n} distinct<={len(pool)}")
    km, dense, nk, err = _remap_gpu(ids, len(pool))
    ref, d = okm.remap(ids)
    assert err == 0 and nk == len(d)
    assert np.array_equal(dense.cpu().numpy().view(np.uint32), ref)


def test_keymap_reserved_unknown_and_overflow():
    ids = np.array([5, 0xFFFFFFFF, 6, 5, 7], dtype=np.uint32)
    say("[case] keymap reserved id")
    km, dense, nk, err = _remap_gpu(ids, 8)
    assert err & B.CR_ERR_KEY_RANGE and nk == 3
    assert dense.cpu().numpy().view(np.uint32).tolist() == [0, B.CR_NO_KEY, 1, 0, 2]
    probe = to_device(np.array([6, 8, 0xFFFFFFFF], dtype=np.uint32))
    out = torch.empty_like(probe)
    km.lookup(probe, out)
    assert out.cpu().numpy().view(np.uint32).tolist() == [1, B.CR_NO_KEY, B.CR_NO_KEY]
    # more distinct ids than the capacity: flagged
    many = np.arange(1, 300, dtype=np.uint32) * 7919
    say("[case] keymap overflow")
    _, _, nk2, err2 = _remap_gpu(many, 100)
    assert err2 & B.CR_ERR_KEYMAP_FULL and nk2 > 100


def test_opaque_70b_path_parity():
    # the 70B-like stream with salted ids: directory, lookup and prefix scatter on the device,
    # then the unchanged path on the dense keys, against the oracle on its own remap
    wl = wl_mod.llama70b()
    op = wl_mod.opaque(wl)
    cap = wl.num_keys
    say(f"[case] opaque 70b n={wl.n}")
    km, dense, nk, err = _remap_gpu(op.ids, cap)
    ref, d = okm.remap(op.ids)
    assert err == 0 and nk == len(d)
    assert np.array_equal(dense.cpu().numpy().view(np.uint32), ref)
    plen = torch.zeros(cap, dtype=torch.int32, device="cuda")
    km.scatter(to_device(op.attr_ids), to_device(op.prefix_by_id), plen)
    plen_ref = okm.scatter(d, op.attr_ids, op.prefix_by_id, cap)
    assert np.array_equal(plen.cpu().numpy().view(np.uint32), plen_ref)
    wr = wl_mod.Workload(name="opaque70b", num_keys=cap, R=wl.R, candidates=wl.candidates, keys=ref, suffix=wl.suffix,
                         prefix_len=plen_ref, offsets=wl.offsets, seed=wl.seed)
    dev = DeviceInputs(keys=dense, suffix=torch.from_numpy(wl.suffix.view(np.int16)).cuda(), prefix_len=plen,
                       off=torch.from_numpy(wl.offsets.view(np.int64)).cuda(), off_host=wl.offsets.astype(np.uint64))
    gp = Pipeline(wr, dev_in=dev)
    gp.step()
    compare_all(wr, gp, gp.host(), opipe.run(wr))
