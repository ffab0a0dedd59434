"""Seeded synthetic request streams for the CacheRoute planner and shadow replay.

This module produces inputs only.  It draws keys, prefix lengths, suffix lengths
and arrival-derived interval boundaries; it computes nothing the routing method
computes (no counts, no admission, no placement, no hashing, no cache model).
Both the CPU oracle's tests and the device path consume the arrays it returns.

The paper's workloads are de-identified telemetry aggregates that are not
public; the shapes below stand in for them:

* per-key popularity is Zipf(s) over ``num_keys`` keys with a seeded
  rank-to-key permutation (keys are opaque dense ids, Appendix A.2);
* the 70B-like shape caps every key's share at 0.3 % by water-filling, the
  paper's top-key bound for its primary aggregate (Section 2.1, Table 7);
* prefix lengths are per key, lognormal around a median; suffix lengths are
  uniform integers in [50, 400] per request;
* arrivals are exponential at a fixed QPS and cut into control intervals of a
  fixed length; the burst shape uses piecewise-constant interval sizes.

Every stream is drawn from its own ``SeedSequence`` child so one chunk of a
large stream can be generated without the others.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import numpy as np

# Stream tags for SeedSequence children (fixed forever: changing them changes inputs).
_S_PERM, _S_PREFIX, _S_KEYS, _S_SUFFIX, _S_ARRIVAL, _S_BURST, _S_DRIFT = 1, 2, 3, 4, 5, 6, 7

SUFFIX_LO, SUFFIX_HI = 50, 400


VARIANTS = ("full", "affinity", "replicated", "flat")


@dataclass
class Candidate:
    """One candidate plan: W warm slots per destination and load target
    q_cap = (a / b) x (mean per-destination load of the window). ``variant`` names a stage
    of the component ablation (Section 5.2): "full" (the method), "affinity" (one copy
    per key, hash placement), "replicated" (Eq. 1 copies, hash placement) or "flat"
    (nothing admitted); ``place_seed`` seeds the hash placement."""

    W: int
    a: int = 1
    b: int = 1
    variant: str = "full"
    place_seed: int = 0


@dataclass
class Workload:
    name: str
    num_keys: int
    R: int
    candidates: List[Candidate]
    keys: np.ndarray          # uint32 [N]
    suffix: np.ndarray        # uint16 [N]
    prefix_len: np.ndarray    # uint32 [num_keys]
    offsets: np.ndarray       # uint64 [J+1], interval boundaries, offsets[0] = 0
    seed: int = 1             # P2C / hash seed
    first_index: int = 0      # global index of keys[0] in the whole stream
    meta: dict = field(default_factory=dict)
    # plan_windows[j][c]: the counting window whose counts build candidate c's plan for
    # interval j (None = window j-1, and window 0 for interval 0)
    plan_windows: Optional[np.ndarray] = None
    # finer boundaries for the replay statistics (None = the control intervals)
    stat_offsets: Optional[np.ndarray] = None

    @property
    def n(self) -> int:
        return int(self.keys.shape[0])

    @property
    def J(self) -> int:
        return int(self.offsets.shape[0] - 1)

    @property
    def P(self) -> int:
        return len(self.candidates)


def _rng(seed: int, tag: int, stream: int, sub: int = 0, *more: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, tag, stream, sub, *more])))


def _tag(name: str) -> int:
    return sum((i + 1) * ord(c) for i, c in enumerate(name)) & 0xFFFF


def zipf_probs(num_ranks: int, s: float) -> np.ndarray:
    """p_r proportional to r^-s for ranks r = 1..num_ranks (float64, sums to 1)."""
    w = np.arange(1, num_ranks + 1, dtype=np.float64) ** (-float(s))
    return w / w.sum()


def water_fill(p_sorted_desc: np.ndarray, cap: float) -> np.ndarray:
    """Cap every share at ``cap`` and rescale the uncapped tail so the total stays 1."""
    p = np.asarray(p_sorted_desc, dtype=np.float64)
    tail = np.cumsum(p[::-1])[::-1]  # tail[t] = sum_{r >= t} p[r]
    for t in range(p.shape[0]):
        scale = (1.0 - t * cap) / tail[t]
        if p[t] * scale <= cap:
            out = p.copy()
            out[:t] = cap
            out[t:] *= scale
            return out / out.sum()
    raise ValueError("cap too small for the number of keys")


class CategoricalSampler:
    """Inverse-CDF sampler with a guide table (Chen's method) for large key sets."""

    def __init__(self, probs: np.ndarray, guide_factor: int = 4):
        p = np.asarray(probs, dtype=np.float64)
        cdf = np.cumsum(p)
        cdf /= cdf[-1]
        cdf[-1] = 1.0
        self.cdf = cdf
        g = max(16, guide_factor * p.shape[0])
        self.G = g
        self.guide = np.searchsorted(cdf, np.arange(g + 1, dtype=np.float64) / g, side="right")
        self.guide = np.minimum(self.guide, p.shape[0] - 1).astype(np.int64)

    def sample(self, rng: np.random.Generator, n: int, block: int = 1 << 24) -> np.ndarray:
        out = np.empty(n, dtype=np.int64)
        for s in range(0, n, block):
            e = min(n, s + block)
            u = rng.random(e - s)
            idx = self.guide[(u * self.G).astype(np.int64)]
            # advance while cdf[idx] <= u (answer = first index with cdf > u)
            todo = np.nonzero(self.cdf[idx] <= u)[0]
            while todo.size:
                idx[todo] += 1
                np.minimum(idx, self.cdf.shape[0] - 1, out=idx)
                keep = self.cdf[idx[todo]] <= u[todo]
                keep &= idx[todo] < self.cdf.shape[0] - 1
                todo = todo[keep]
            out[s:e] = idx
        return out


def _prefix_lengths(seed: int, tag: int, num_keys: int, median: float, sigma: float) -> np.ndarray:
    z = _rng(seed, tag, _S_PREFIX).standard_normal(num_keys)
    v = np.rint(median * np.exp(sigma * z))
    return np.maximum(1, v).astype(np.uint32)


def _suffixes(rng: np.random.Generator, n: int) -> np.ndarray:
    return rng.integers(SUFFIX_LO, SUFFIX_HI + 1, size=n, dtype=np.int64).astype(np.uint16)


def _exp_intervals(rng: np.random.Generator, n: int, qps: float, interval_s: Optional[float],
                   cv: Optional[float] = None) -> np.ndarray:
    """Inter-arrivals at ``qps``: exponential, or Gamma with coefficient of variation ``cv``
    (shape 1 / cv^2, same mean; Section 5.4 "Arrival burstiness"); offsets of fixed-length
    control intervals."""
    if interval_s is None:
        return np.array([0, n], dtype=np.uint64)
    if cv is None:
        gaps = rng.exponential(1.0 / qps, size=n)
    else:
        gaps = rng.gamma(1.0 / (cv * cv), (cv * cv) / qps, size=n)
    t = np.cumsum(gaps)
    j = np.floor(t / interval_s).astype(np.int64)
    J = int(j[-1]) + 1 if n else 1
    off = np.searchsorted(j, np.arange(J + 1), side="left").astype(np.uint64)
    off[-1] = n
    return off


def synthetic(name: str, *, num_keys: int, n: int, R: int, candidates: Sequence[Candidate],
              probs_by_rank: np.ndarray, qps: float = 100.0, interval_s: Optional[float] = None,
              prefix_median: float = 2000.0, prefix_sigma: float = 0.5, seed: int = 2,
              p2c_seed: int = 1, cv: Optional[float] = None) -> Workload:
    """A stationary stream: keys iid from ``probs_by_rank`` through a seeded permutation."""
    tag = _tag(name)
    perm = _rng(seed, tag, _S_PERM).permutation(num_keys)
    sampler = CategoricalSampler(probs_by_rank)
    ranks = sampler.sample(_rng(seed, tag, _S_KEYS), n)
    keys = perm[ranks].astype(np.uint32)
    suffix = _suffixes(_rng(seed, tag, _S_SUFFIX), n)
    offsets = _exp_intervals(_rng(seed, tag, _S_ARRIVAL), n, qps, interval_s, cv)
    plen = _prefix_lengths(seed, tag, num_keys, prefix_median, prefix_sigma)
    return Workload(name=name, num_keys=num_keys, R=R, candidates=list(candidates), keys=keys,
                    suffix=suffix, prefix_len=plen, offsets=offsets, seed=p2c_seed,
                    meta=dict(qps=qps, interval_s=interval_s, seed=seed, cv=cv))


# ---------------------------------------------------------------------------
# The five named shapes.
# ---------------------------------------------------------------------------

def tiny(seed: int = 2, n: int = 100_000) -> Workload:
    """1,000 keys, Zipf 1.1, 100 QPS exponential arrivals, one control interval,
    30 destinations x 16 LRU slots, prefixes lognormal(2000, 0.5)."""
    return synthetic("tiny", num_keys=1000, n=n, R=30, candidates=[Candidate(16)],
                     probs_by_rank=zipf_probs(1000, 1.1), qps=100.0, interval_s=None,
                     prefix_median=2000.0, prefix_sigma=0.5, seed=seed)


def llama70b(seed: int = 2, n: int = 10_000_000, cv: Optional[float] = None) -> Workload:
    """20,000 keys, Zipf 1.0 water-filled to a 0.3 % top share, 176 QPS,
    60-s control intervals, 30 destinations x 64 slots, prefixes lognormal(3000, 0.7).
    ``cv`` replaces the exponential gaps by Gamma gaps of that coefficient of variation
    (the same keys; only the interval boundaries move)."""
    p = water_fill(zipf_probs(20_000, 1.0), 0.003)
    return synthetic("llama70b", num_keys=20_000, n=n, R=30, candidates=[Candidate(64)],
                     probs_by_rank=p, qps=176.0, interval_s=60.0,
                     prefix_median=3000.0, prefix_sigma=0.7, seed=seed, cv=cv)


def llama70b_gamma(seed: int = 2, n: int = 10_000_000) -> Workload:
    """The 70B-like stream with Gamma arrivals matched to the workload's marginal
    inter-arrival CV of 1.9 (Section 5.4 "Arrival burstiness")."""
    wl = llama70b(seed, n, cv=1.9)
    wl.name = "llama70b_gamma"
    return wl


def replication(seed: int = 2, n: int = 20_000_000) -> Workload:
    """5,000 Zipf-1.1 background keys carrying 52 % plus 8 injected keys at 6 % each;
    500 QPS, 60-s intervals, 16 destinations x 128 slots; load target 0.4 x mean."""
    bg = zipf_probs(5000, 1.1) * 0.52
    p = np.concatenate([np.full(8, 0.06), bg])  # ranks 1..8 are the injected keys
    return synthetic("replication", num_keys=5008, n=n, R=16, candidates=[Candidate(128, 2, 5)],
                     probs_by_rank=p, qps=500.0, interval_s=60.0, seed=seed)


def ablation(seed: int = 2, n: int = 20_000_000, place_seed: int = 7) -> Workload:
    """The component ablation (Section 5.2, 8B component ablation table) on the
    injected-whale stream of ``replication``: the same requests replayed under four
    candidates that add the method's parts one at a time, load balancing alone (flat),
    + affinity (one copy per key, hash placement), + replication (Eq. 1, hash placement)
    and + LPT (the method), all with 128 slots per destination and q_cap = 0.4 x mean."""
    wl = replication(seed, n)
    wl.name = "ablation"
    wl.candidates = [Candidate(128, 2, 5, v, place_seed) for v in ("flat", "affinity", "replicated", "full")]
    return wl


def burst(seed: int = 2, n: int = 50_000_000, J: int = 100, num_keys: int = 50_000,
          R: int = 64, W: int = 64, burst_frac: float = 0.05, burst_mult: float = 10.0,
          burst_len: int = 2) -> Workload:
    """50,000 keys, Zipf 1.2, 100 ten-second intervals; a random 5 % of keys get a
    10x weight for two consecutive intervals; interval sizes follow total weight."""
    name = "burst"
    tag = _tag(name)
    perm = _rng(seed, tag, _S_PERM).permutation(num_keys)
    base = np.empty(num_keys)
    base[perm] = zipf_probs(num_keys, 1.2)  # per key id
    brng = _rng(seed, tag, _S_BURST)
    nb = int(round(burst_frac * num_keys))
    bkeys = brng.choice(num_keys, size=nb, replace=False)
    bstart = brng.integers(0, J - burst_len + 1, size=nb)
    mult = np.ones((J, num_keys))
    for t in range(burst_len):
        mult[bstart + t, bkeys] = burst_mult
    wj = (mult * base[None, :]).sum(axis=1)
    share = wj / wj.sum() * n
    nj = np.floor(share).astype(np.int64)
    rem = n - int(nj.sum())
    order = np.argsort(-(share - nj), kind="stable")
    nj[order[:rem]] += 1
    offsets = np.zeros(J + 1, dtype=np.uint64)
    offsets[1:] = np.cumsum(nj)
    keys = np.empty(n, dtype=np.uint32)
    krng = _rng(seed, tag, _S_KEYS)
    for j in range(J):
        pj = mult[j] * base
        s = CategoricalSampler(pj / pj.sum(), guide_factor=2)
        keys[int(offsets[j]):int(offsets[j + 1])] = s.sample(krng, int(nj[j])).astype(np.uint32)
    suffix = _suffixes(_rng(seed, tag, _S_SUFFIX), n)
    plen = _prefix_lengths(seed, tag, num_keys, 2000.0, 0.5)
    return Workload(name=name, num_keys=num_keys, R=R, candidates=[Candidate(W)], keys=keys,
                    suffix=suffix, prefix_len=plen, offsets=offsets, seed=1,
                    meta=dict(interval_s=10.0, seed=seed, burst_keys=bkeys, burst_start=bstart))


def drift(seed: int = 2, n_per: int = 1_000_000, steps: int = 6, sigma: float = 0.3,
          num_keys: int = 20_000, R: int = 30, W: int = 64, bins_per_interval: int = 100) -> Workload:
    """Rate drift (Section 5.4, Appendix E): the 70B-like key distribution evolves for
    ``steps`` intervals by a lognormal random walk, w_t(b) = w_{t-1}(b) exp(sigma z),
    z ~ N(0, 1) per key and step, starting from the base shares; interval t draws
    ``n_per`` keys iid from w_t / sum(w_t).

    Candidates (all W slots, q_cap = mean load) differ only in the window their plans
    come from: candidate 0 is fresh (interval j uses window j's own counts, the rate
    vector of that interval); candidate t >= 1 is the same except that interval t keeps
    the plan of window t-1, so it shares candidate 0's history up to the boundary and
    stays warm after it. Replay statistics are kept in ``bins_per_interval`` equal bins
    per interval so the rewarming transient after each install is visible."""
    name = "drift"
    tag = _tag(name)
    perm = _rng(seed, tag, _S_PERM).permutation(num_keys)
    w = np.empty(num_keys)
    w[perm] = water_fill(zipf_probs(num_keys, 1.0), 0.003)  # per key id
    zr = _rng(seed, tag, _S_DRIFT)
    krng = _rng(seed, tag, _S_KEYS)
    n = n_per * steps
    keys = np.empty(n, dtype=np.uint32)
    shares = np.empty((steps, num_keys))
    for t in range(steps):
        if t:
            w = w * np.exp(sigma * zr.standard_normal(num_keys))
        shares[t] = w / w.sum()
        keys[t * n_per:(t + 1) * n_per] = CategoricalSampler(shares[t]).sample(krng, n_per).astype(np.uint32)
    offsets = (np.arange(steps + 1, dtype=np.uint64) * np.uint64(n_per))
    bins = np.linspace(0, n, steps * bins_per_interval + 1)
    stat_offsets = np.rint(bins).astype(np.uint64)
    pw = np.tile(np.arange(steps, dtype=np.int64)[:, None], (1, steps))
    for t in range(1, steps):
        pw[t, t] = t - 1
    suffix = _suffixes(_rng(seed, tag, _S_SUFFIX), n)
    plen = _prefix_lengths(seed, tag, num_keys, 3000.0, 0.7)
    return Workload(name=name, num_keys=num_keys, R=R, candidates=[Candidate(W) for _ in range(steps)],
                    keys=keys, suffix=suffix, prefix_len=plen, offsets=offsets, seed=1,
                    meta=dict(seed=seed, sigma=sigma, shares=shares, bins_per_interval=bins_per_interval),
                    plan_windows=pw, stat_offsets=stat_offsets)


SWEEP_W = (8, 14, 26, 48, 86, 156, 283, 512)


def sweep_candidates() -> List[Candidate]:
    """8 warm-slot budgets (log-even 8..512) x 8 load targets (0.8..1.2 x mean)."""
    return [Candidate(W, 28 + 2 * m, 35) for W in SWEEP_W for m in range(8)]


SWEEP_CHUNKS = 10          # 1e9 requests in ten 1e8-request chunks (= control intervals)
SWEEP_SUBBLOCKS = 16       # each chunk is drawn as 16 independently seeded sub-blocks


def _sweep_tables(seed: int, num_keys: int, _cache: dict = {}):
    """The sweep's rank -> key permutation and Zipf(0.9) sampler (cached: 1e6 keys)."""
    ck = (seed, num_keys)
    if ck not in _cache:
        perm = _rng(seed, _tag("sweep"), _S_PERM).permutation(num_keys).astype(np.uint32)
        _cache.clear()
        _cache[ck] = (perm, CategoricalSampler(zipf_probs(num_keys, 0.9)))
    return _cache[ck]


def sweep_chunk(chunk: int, seed: int = 2, chunk_n: int = 100_000_000, num_keys: int = 1_000_000,
                R: int = 1024, candidates: Optional[List[Candidate]] = None,
                threads: Optional[int] = None) -> Workload:
    """One 1e8-request chunk (= one control interval) of the 1e9-request sweep:
    1,000,000 keys, Zipf 0.9, 1,024 destinations, 64 candidate plans.

    The chunk is cut into ``SWEEP_SUBBLOCKS`` equal sub-blocks, each with its own seed
    (seed, tag, stream, chunk, sub-block), so the sub-blocks can be drawn by several
    threads at once; the result does not depend on ``threads``."""
    name = "sweep"
    tag = _tag(name)
    perm, sampler = _sweep_tables(seed, num_keys)
    keys = np.empty(chunk_n, dtype=np.uint32)
    suffix = np.empty(chunk_n, dtype=np.uint16)
    bounds = [b * chunk_n // SWEEP_SUBBLOCKS for b in range(SWEEP_SUBBLOCKS + 1)]

    def fill(b: int) -> None:
        s, e = bounds[b], bounds[b + 1]
        ranks = sampler.sample(_rng(seed, tag, _S_KEYS, chunk, b), e - s)
        keys[s:e] = perm[ranks]
        suffix[s:e] = _rng(seed, tag, _S_SUFFIX, chunk, b).integers(SUFFIX_LO, SUFFIX_HI + 1, size=e - s,
                                                                    dtype=np.uint16)

    nt = threads if threads is not None else min(16, os.cpu_count() or 1)
    if nt <= 1:
        for b in range(SWEEP_SUBBLOCKS):
            fill(b)
    else:
        with ThreadPoolExecutor(nt) as ex:
            list(ex.map(fill, range(SWEEP_SUBBLOCKS)))
    plen = _prefix_lengths(seed, tag, num_keys, 2000.0, 0.5)
    return Workload(name=name, num_keys=num_keys, R=R,
                    candidates=candidates if candidates is not None else sweep_candidates(),
                    keys=keys, suffix=suffix, prefix_len=plen,
                    offsets=np.array([0, chunk_n], dtype=np.uint64), seed=1,
                    first_index=chunk * chunk_n, meta=dict(chunk=chunk, seed=seed))


CONFIGS = {
    "tiny": tiny,
    "llama70b": llama70b,
    "replication": replication,
    "burst": burst,
    "drift": drift,
    "ablation": ablation,
    "llama70b_gamma": llama70b_gamma,
}


@dataclass
class OpaqueStream:
    """A request stream whose keys are opaque 32-bit ids, with the per-key prefix lengths
    given by id (including ids that never appear in the stream)."""

    ids: np.ndarray           # uint32 [N], never 0xFFFFFFFF
    attr_ids: np.ndarray      # uint32 [K] every key's id
    prefix_by_id: np.ndarray  # uint32 [K] prefix length of attr_ids[x]


def opaque(wl: Workload, salt: int = 0x5EED1234) -> OpaqueStream:
    """Salted ids for a workload's dense keys (Appendix A.2: keys may be salted): a fixed
    odd-multiplier bijection of the 32-bit key space, xor a salt. The ids carry no order
    of the dense keys; 0xFFFFFFFF is never produced."""
    def salted(b: np.ndarray) -> np.ndarray:
        x = (b.astype(np.uint64) * np.uint64(0x9E3779B1) + np.uint64(salt)) & np.uint64(0xFFFFFFFF)
        x = x.astype(np.uint32) ^ np.uint32((salt * 0x632BE5AB) & 0xFFFFFFFF)
        return x

    all_ids = salted(np.arange(wl.num_keys, dtype=np.uint32))
    if np.any(all_ids == 0xFFFFFFFF):
        raise ValueError("salt maps a key to the reserved id; choose another salt")
    return OpaqueStream(ids=all_ids[wl.keys], attr_ids=all_ids, prefix_by_id=wl.prefix_len.copy())


def small_random(seed: int, *, num_keys: int, n: int, R: int, Ws: Sequence[int],
                 J: int = 1, zipf_s: float = 1.1, qs: Sequence[Tuple[int, int]] = ((1, 1),),
                 hot: int = 0, hot_share: float = 0.0) -> Workload:
    """Small random stream for parity and property tests: Zipf keys, optional
    injected hot keys, J intervals of random (possibly empty) sizes."""
    rng = _rng(seed, 77, 0)
    p = zipf_probs(num_keys, zipf_s)
    if hot:
        p = p * (1.0 - hot_share)
        p[:hot] += hot_share / hot
        p /= p.sum()
    perm = rng.permutation(num_keys)
    ranks = CategoricalSampler(p).sample(rng, n)
    keys = perm[ranks].astype(np.uint32)
    suffix = _suffixes(rng, n)
    cuts = np.sort(rng.integers(0, n + 1, size=J - 1)) if J > 1 else np.zeros(0, dtype=np.int64)
    offsets = np.concatenate([[0], cuts, [n]]).astype(np.uint64)
    plen = np.maximum(1, np.rint(2000 * np.exp(0.5 * rng.standard_normal(num_keys)))).astype(np.uint32)
    cands = [Candidate(W, a, b) for W in Ws for (a, b) in qs]
    return Workload(name=f"small{seed}", num_keys=num_keys, R=R, candidates=cands, keys=keys,
                    suffix=suffix, prefix_len=plen, offsets=offsets, seed=int(rng.integers(0, 2**63)))
