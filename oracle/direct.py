"""Direct evaluation of the DLA readout and state cache from a run's decisions.

TEST INFRASTRUCTURE: only tests/, the smoke check and the benchmark's CPU
baseline leg may import this module.  It shares no code with the HIP path.

Given the boundary decisions b_t and merge indices of a run (from the float64
oracle's decisions mode, which scores against the newest state only), every
state of the cache is a contiguous range of tokens: a boundary opens a state
at its token, and a capacity merge of Alg. 2 joins the ranges of two adjacent
states.  The definitions then fix everything else directly, token by token:

  * the state over a token range R at token t (Sec. 2.1 gated linear attention
    with every state decaying by the same gate, the reading the oracle takes):
        S_R(t) = sum_{s in R, s <= t} exp(G_t - G_s) k_s v_s^T,  G_t = sum_{r<=t} g_r;
  * the readout (eq. capacity_bounded_output):
        o_t = sum_j lambda[t][j] S_j(t)^T q_t,
    j running over the states after token t in chronological order.

Both are O(t d) per output token and O(T d_k d_v) for the final cache, so
sampled outputs of full-size workloads can be checked without replaying the
per-token decay of every state.  The test-suite pins this module to the C
oracle's full mode on small inputs.
"""
from __future__ import annotations

import numpy as np


def state_starts(b, merge, C: int, upto: int, starts0=None):
    """First token of every state after token `upto` (inclusive), replaying the
    boundaries and Alg. 2 merges on range starts.  starts0: the states present
    before token 0 (their first tokens, negative for tokens of earlier calls)."""
    starts = list(starts0 or [])
    for t in range(upto + 1):
        if b[t]:
            if len(starts) == C:
                i = int(merge[t])
                if not 0 <= i <= C - 2:
                    raise ValueError(f"t={t}: capacity merge with index {i}")
                del starts[i + 1]   # the ranges of states i and i + 1 join
            starts.append(t)
    return starts


def starts_timeline(b, merge, C: int, tokens):
    """state_starts for each token of the sorted list `tokens`, in one pass."""
    out = {}
    want = sorted(set(int(t) for t in tokens))
    starts = []
    k = 0
    for t in range(len(b)):
        if b[t]:
            if len(starts) == C:
                i = int(merge[t])
                if not 0 <= i <= C - 2:
                    raise ValueError(f"t={t}: capacity merge with index {i}")
                del starts[i + 1]
            starts.append(t)
        while k < len(want) and want[k] == t:
            out[t] = list(starts)
            k += 1
        if k == len(want):
            break
    return out


def outputs_at(q, k, v, g, lam, b, merge, C: int, tokens, batch: int = 64):
    """o_t for each t in `tokens` of one head (q, k: [T, d_k]; v: [T, d_v];
    g: [T]; lam: [T, C] or None; float64, finite), straight from the
    definitions: o_t = sum_{s <= t} lambda[t][j_t(s)] exp(G_t - G_s) (q_t . k_s) v_s,
    j_t(s) the chronological index at token t of the state holding token s.
    Tokens are evaluated `batch` at a time as one masked product."""
    G = np.cumsum(np.asarray(g, np.float64))
    toks = [int(t) for t in tokens]
    tl = starts_timeline(b, merge, C, toks)
    out = np.zeros((len(toks), v.shape[1]))
    for i0 in range(0, len(toks), batch):
        tb = np.array(toks[i0:i0 + batch])
        tmax = int(tb.max())
        s = np.arange(tmax + 1)
        causal = s[None, :] <= tb[:, None]
        W = (q[tb] @ k[: tmax + 1].T) * np.exp(np.where(causal, G[tb][:, None] - G[None, s],
                                                        -np.inf))
        if lam is not None:
            for r, t in enumerate(tb):
                slot = np.searchsorted(np.array(tl[int(t)]), s, side="right") - 1
                W[r] *= lam[t, np.clip(slot, 0, C - 1)]
        out[i0:i0 + len(tb)] = np.where(causal, W, 0.0) @ v[: tmax + 1]
    return out


def final_states(k, v, g, b, merge, C: int):
    """The cache after the last token of one head: m, the token count and the
    true (decayed) state of every state, chronological (states [C, d_k, d_v],
    entries past m zero)."""
    T = len(b)
    G = np.cumsum(np.asarray(g, np.float64))
    starts = state_starts(b, merge, C, T - 1)
    ends = starts[1:] + [T]
    S = np.zeros((C, k.shape[1], v.shape[1]))
    n = np.zeros(C, np.int64)
    for j, (a, e) in enumerate(zip(starts, ends)):
        f = np.exp(G[T - 1] - G[a:e])
        S[j] = (k[a:e] * f[:, None]).T @ v[a:e]
        n[j] = e - a
    return len(starts), n, S
