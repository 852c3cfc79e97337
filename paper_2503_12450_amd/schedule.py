"""LazyMAR's step schedule (host logic).

Sec. 4.1: with 64 decoding steps caching starts at the 5th step with a
period tau = 9; with 32 steps it starts at the 4th with tau = 5.  Sec. 1 and
Fig. 3: the steps before the start, and the first step of every period, run
in full (every token, both guidance pathways) and refill the token cache and
the condition cache; the other steps of a period reuse them.

Reading of the period rule: steps are numbered 1..K; step s is a full step
when s < start or (s - start) % tau == 0, a cached step otherwise.  For the
guidance pathways two rules are offered:
  "paper"     every cached step runs the conditional pathway only and
              reuses the stored residual (Eq. 10);
  "alternate" cached steps at odd offsets from the last refresh run the
              conditional pathway only (reuse), those at even offsets run
              both pathways with the token cache and store a fresh residual.
"""
from __future__ import annotations

import dataclasses
from typing import List

FULL = "full"
CACHED = "cached"
BOTH = "both"
COND = "cond"
STORE = "store"
REUSE = "reuse"


@dataclasses.dataclass(frozen=True)
class StepPlan:
    step: int        # 1-based decoding step
    mode: str        # FULL or CACHED
    branches: str    # BOTH or COND
    cfg: str         # STORE or REUSE


def lazymar_schedule(n_steps: int = 64, start: int = 5, tau: int = 9, cfg: str = "paper") -> List[StepPlan]:
    if n_steps < 1 or start < 1 or tau < 1:
        raise ValueError("n_steps, start and tau must be >= 1")
    if cfg not in ("paper", "alternate"):
        raise ValueError(cfg)
    plans = []
    for s in range(1, n_steps + 1):
        if s < start or (s - start) % tau == 0:
            plans.append(StepPlan(s, FULL, BOTH, STORE))
            continue
        offset = (s - start) % tau
        if cfg == "alternate" and offset % 2 == 0:
            plans.append(StepPlan(s, CACHED, BOTH, STORE))
        else:
            plans.append(StepPlan(s, CACHED, COND, REUSE))
    return plans


def counts(plans: List[StepPlan]):
    full = sum(p.mode == FULL for p in plans)
    cached_cond = sum(p.mode == CACHED and p.branches == COND for p in plans)
    cached_both = sum(p.mode == CACHED and p.branches == BOTH for p in plans)
    return full, cached_cond, cached_both
