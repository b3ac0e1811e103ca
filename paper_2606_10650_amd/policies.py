"""Fixed state-merging policies, as decision schedules for the override path.

The paper contrasts information-aware merging with fixed schedules: blocking
and merging every K tokens (Sec. 3.1, motivation) and the Fenwick-tree buckets
of log-linear attention (Sec. 2.3), and compares their prefill throughput and
memory with a single-state model (Sec. 4.3, Fig. 3).  Each schedule here is a
pair of override arrays (boundary_override, merge_override; -1 = decide) that
dla_prefill and dla_decode_step take, so that every policy runs on the same
kernels and the same cache, and differs from DLA only in where states open and
which adjacent pair Alg. 2 merges when the cache is full.  These functions
decide nothing from the data: they compute no score and touch no state.

  * single_state: the base model's one gated state (C = 1).
  * every_k: a state opens every K tokens; when the cache is full the two
    oldest states merge, so the cache holds one summary of the distant past
    and the C - 1 most recent blocks.
  * log_linear: a state opens at every token and, when the cache is full, the
    oldest adjacent pair of equal token counts merges, with capacity
    C = ceil(log2(T)) + 1, the bucket count of Sec. 2.3 at the last token.  State sizes are
    then powers of two, non-increasing from the oldest state, and the most
    recent tokens keep states of their own: the Fenwick decomposition's fine
    resolution near the current position and coarse resolution far from it.
    Alg. 2 merges one pair per opened state, so where the Fenwick counter
    carries through several buckets at one token, the schedule carries one
    bucket per token.
"""
from __future__ import annotations

import numpy as np


def log_linear_capacity(T: int) -> int:
    """Bucket count ceil(log2(t + 1)) + 1 of the Fenwick decomposition of the
    prefix [0, t] of T = t + 1 tokens (in integers: (T - 1).bit_length() + 1)."""
    return max(T - 1, 0).bit_length() + 1


def single_state(T: int):
    """C = 1: one state absorbs every token (returns C and the overrides)."""
    return 1, np.full(T, -1, np.int8), np.full(T, -1, np.int32)


def every_k(T: int, K: int, C: int, t0: int = 0):
    """A boundary at every token t with (t0 + t) % K == 0, and a merge of the
    two oldest states (index 0) whenever a boundary finds the cache full.
    t0: tokens absorbed before (for a continuation)."""
    t = np.arange(T) + t0
    b = np.where(t % K == 0, 1, 0).astype(np.int8)
    m = np.zeros(T, np.int32)   # honoured only at a boundary with a full cache
    return C, b, m


def log_linear(T: int, C: int = None):
    """A boundary at every token; at a full cache the oldest adjacent pair of
    equal token counts merges (the pair of smallest combined count when no two
    are equal).  Returns C and the overrides."""
    C = log_linear_capacity(T) if C is None else C
    b = np.ones(T, np.int8)
    m = np.full(T, -1, np.int32)
    sizes = []
    for t in range(T):
        if C > 1 and len(sizes) == C:
            i = next((j for j in range(C - 1) if sizes[j] == sizes[j + 1]), None)
            if i is None:
                i = min(range(C - 1), key=lambda j: (sizes[j] + sizes[j + 1], j))
            sizes[i] += sizes[i + 1]
            del sizes[i + 1]
            m[t] = i
        if C > 1 or not sizes:
            sizes.append(1)
        else:
            sizes[-1] += 1
    return C, b, m


POLICIES = ("single_state", "every_k", "log_linear", "dla")


def schedule(policy: str, T: int, C_dla: int = 30, K: int = 64):
    """(C, boundary_override, merge_override) of a policy for T tokens; the
    overrides are None for DLA's own decisions."""
    if policy == "single_state":
        return single_state(T)
    if policy == "every_k":
        return every_k(T, K, C_dla)
    if policy == "log_linear":
        return log_linear(T)
    if policy == "dla":
        return C_dla, None, None
    raise ValueError(policy)
