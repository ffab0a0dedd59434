"""Churn between two plans, as the replanning study measures it -- TEST INFRASTRUCTURE.

Definitions (Section 5.4 and Appendix E, table of replan measurements):

* a plan's assignment set is S = {(b, r) : r in T(b)} over its admitted keys b;
  cache churn between consecutive plans is one minus the Jaccard index of their
  assignment sets, 1 - |S ∩ S'| / |S ∪ S'|;
* count churn is the share of keys whose assignment count k_b changes.  The paper
  does not say over which keys; the reading here is the keys admitted by both plans
  (a key that enters or leaves the warm set has no count on one side).

``plan_churn`` returns the four integers both the oracle and the device report, in
plain Python sets; the ratios follow from them and the plans' sizes.  Plans are the
oracle's plan dicts (adm_keys, member_off, members).
"""
from __future__ import annotations

from typing import Dict, Set, Tuple


def assignment(plan: dict) -> Dict[int, Set[int]]:
    """T(b) of every admitted key b, as a set of destinations."""
    off = plan["member_off"]
    mem = plan["members"]
    return {int(b): {int(r) for r in mem[int(off[a]):int(off[a + 1])]} for a, b in enumerate(plan["adm_keys"])}


def plan_churn(pa: dict, pb: dict) -> Tuple[int, int, int, int]:
    """(|S_a ∩ S_b|, keys admitted by both, of those the keys whose k differs,
    of those the keys whose destination set is the same)."""
    ta, tb = assignment(pa), assignment(pb)
    sa = {(b, r) for b, t in ta.items() for r in t}
    sb = {(b, r) for b, t in tb.items() for r in t}
    both = ta.keys() & tb.keys()
    k_changed = sum(1 for b in both if len(ta[b]) != len(tb[b]))
    same = sum(1 for b in both if ta[b] == tb[b])
    return len(sa & sb), len(both), k_changed, same


def churn_rates(pa: dict, pb: dict) -> Dict[str, float]:
    """Cache churn (1 - Jaccard of assignment sets), count churn, warm-set churn
    (1 - Jaccard of admitted key sets) and the share of common keys that moved."""
    common, both, k_changed, same = plan_churn(pa, pb)
    na, nb = int(pa["member_off"][len(pa["adm_keys"])]), int(pb["member_off"][len(pb["adm_keys"])])
    ka, kb_ = len(pa["adm_keys"]), len(pb["adm_keys"])
    union = na + nb - common
    kunion = ka + kb_ - both
    return dict(cache_churn=1.0 - common / union if union else 0.0,
                count_churn=k_changed / both if both else 0.0,
                warm_set_churn=1.0 - both / kunion if kunion else 0.0,
                moved=1.0 - same / both if both else 0.0)
