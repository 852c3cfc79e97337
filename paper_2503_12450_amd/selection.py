"""Token-selection rules of the paper's strategy comparison (Table 3) that
choose the computed rows on the host.

The similarity-based rules run on the device inside the step
(MAR_TOKEN_CACHED computes the least similar rows, strategy V;
MAR_TOKEN_CACHED_MOST_SIMILAR the most similar ones, strategy IV).  The
rules below depend on the sampler's state or on random draws instead of the
block P-1 value rows, so they produce index arrays that the step takes as
given rows (MAR_TOKEN_GIVEN):

  random_rows        strategy III: the cached (and so the computed) tokens
                     drawn uniformly at random, from the caller's generator;
  observation_rows   strategies I and II (Sec. 3.2, token types): compute
                     the tokens already decoded ("predicted"), caching the
                     undecoded ones (I), or the reverse (II).

Every rule returns int32 [n_slots, n], each row strictly ascending, exactly
n tokens per slot.  The paper does not say how a token-type rule meets a
fixed budget n; here the tokens of the type to compute come first, lowest
index first, then the other type, lowest index first.
"""
from __future__ import annotations

import numpy as np

COMPUTE_DECODED = "decoded"      # strategy I: cache the not-yet-decoded tokens
COMPUTE_UNDECODED = "undecoded"  # strategy II: cache the decoded tokens


def _check(n_slots: int, seq: int, n: int) -> None:
    if n_slots < 0 or seq < 1 or not 0 <= n <= seq:
        raise ValueError(f"need n_slots >= 0, seq >= 1 and 0 <= n <= seq (got {n_slots}, {seq}, {n})")


def random_rows(n_slots: int, seq: int, n: int, rng: np.random.Generator) -> np.ndarray:
    """n distinct tokens per slot, uniformly at random, ascending."""
    _check(n_slots, seq, n)
    out = np.empty((n_slots, n), dtype=np.int32)
    for b in range(n_slots):
        out[b] = np.sort(rng.choice(seq, size=n, replace=False))
    return out


def observation_rows(decoded, n: int, compute: str) -> np.ndarray:
    """Token-type selection: `decoded` is bool [n_slots, seq], True for the
    tokens the sampler has already predicted; `compute` names the type to
    compute (COMPUTE_DECODED or COMPUTE_UNDECODED).  The n computed tokens
    are those of that type, lowest index first, filled up with the other
    type, lowest index first."""
    decoded = np.asarray(decoded, dtype=bool)
    if decoded.ndim != 2:
        raise ValueError("decoded must be [n_slots, seq]")
    n_slots, seq = decoded.shape
    _check(n_slots, seq, n)
    if compute not in (COMPUTE_DECODED, COMPUTE_UNDECODED):
        raise ValueError(f"compute must be {COMPUTE_DECODED!r} or {COMPUTE_UNDECODED!r}")
    want = decoded if compute == COMPUTE_DECODED else ~decoded
    out = np.empty((n_slots, n), dtype=np.int32)
    for b in range(n_slots):
        order = np.concatenate([np.flatnonzero(want[b]), np.flatnonzero(~want[b])])
        out[b] = np.sort(order[:n])
    return out
