"""Orchestrator planners, stated plainly -- TEST INFRASTRUCTURE ONLY.

Only tests/ may import this module.  It restates, from the paper's description
of the load-balancing orchestrator (Sec. 3.3), the two planning rules the
library implements natively, with exact rational arithmetic:

* Resource partitioning plan: DP groups per policy version in proportion to
  the version's workload (active and pending requests).  Reading taken where
  the text is silent: a version with work keeps at least one group (no request
  is stranded, no trajectory abandoned); the rest are apportioned by the
  largest-remainder (Hamilton) method; equal remainders favour the newer
  version (the plan shrinks legacy versions and grows the latest); with no
  work at all, every group goes to the latest version.
* Staleness-aware data supplementation: the latest version is given prompts
  first, up to what its rollout batch still needs and its idle slots hold;
  legacy versions are given only prompts that fill their residual idle slots.
"""
from __future__ import annotations

from fractions import Fraction
from typing import List, Sequence


def partition(workload: Sequence[int], n_groups: int) -> List[int]:
    """Target DP groups per version (index order = age, last = latest)."""
    n = len(workload)
    if n < 1 or n_groups < 1 or any(w < 0 for w in workload):
        raise ValueError("bad arguments")
    busy = [v for v in range(n) if workload[v] > 0]
    if len(busy) > n_groups:
        raise ValueError("more versions with work than groups")
    groups = [0] * n
    if not busy:
        groups[-1] = n_groups
        return groups
    total = sum(workload)
    spare = n_groups - len(busy)
    quota = {v: Fraction(workload[v] * spare, total) for v in busy}
    for v in busy:
        groups[v] = 1 + int(quota[v])            # floor of a non-negative quota
    left = n_groups - sum(groups)
    # the `left` largest fractional parts, newer version first on ties
    order = sorted(busy, key=lambda v: (quota[v] - int(quota[v]), v), reverse=True)
    for v in order[:left]:
        groups[v] += 1
    return groups


def supplement(groups: Sequence[int], active: Sequence[int], slots_per_group: int,
               latest_quota: int) -> List[int]:
    """Prompts to inject per version (last = latest)."""
    if len(groups) != len(active) or not groups or slots_per_group < 1 or latest_quota < 0:
        raise ValueError("bad arguments")
    out = []
    for v, (g, a) in enumerate(zip(groups, active)):
        idle = max(0, g * slots_per_group - a)
        out.append(min(idle, latest_quota) if v == len(groups) - 1 else idle)
    return out
