"""Pins for the float64 oracle: checks against what the paper and the
mathematics fix, independent of the oracle's own code.

Each pin is a function ``pin_xxx(lib_path=None)`` that raises AssertionError
when the oracle disagrees.  test_oracle_pins.py runs them on the oracle;
test_oracle_mutants.py runs them on deliberately broken copies of the oracle
and requires every broken copy to fail at least one pin.

What pins what (paper passages in brackets):
  * gated linear attention, parallel form (QK^T (.) decay mask) V  [Sec. 2.1,
    eq. linear_attn_parallel]: readout with lambda = 1 for any tau, C, and the
    sum of all cached states;
  * one state per token (tau <= 0, C >= T) equals lambda-weighted masked
    attention, C = 1 equals lambda_0-weighted linear attention  [Sec. 3.2,
    eq. capacity_bounded_output];
  * brute force on membership lists: Alg. 2 replayed on lists of token ids
    with a scalar argmin, outputs as sums over member tokens  [Alg. 2, Sec. 3.2];
  * closed forms of the score: identical tokens, orthogonal keys, scalar states
    (sign flips), scale invariance, 0 <= I <= 2, and the rank-one expansion of
    the score  [eq. importance_score, RMSNorm remark of Sec. 3.1];
  * hand-computed merge schedules on scalar states  (tests/golden/), including
    the near-tie margins of the parity protocol and the merge override;
  * conservation (counts, scores, states) and C-independence of boundaries;
  * the delta-rule form (Gated DeltaNet, Sec. 2.2, eq. delta_rule_rnn): C = 1
    is the textbook recurrence, a unit key with step 1 is overwritten with its
    value, step 0 writes nothing, and with boundaries and merges every state is
    the sum of its ranges' own recurrences (Alg. 2 replayed on membership lists).
"""
from __future__ import annotations

import json
import os

import numpy as np

from oracle import OracleCache, oracle_forward
from paper_2606_10650_amd.workloads import WORKLOADS, make_inputs, to_f64

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


# ----------------------------------------------------------------------------
# independent helpers (no oracle code)
# ----------------------------------------------------------------------------

def cum_gate(g):
    return np.cumsum(np.asarray(g, np.float64), axis=-1)


def decay_mask(G):
    """D[t, s] = exp(G_t - G_s) for s <= t, else 0 (G inclusive cumulative)."""
    T = G.shape[0]
    D = np.exp(np.minimum(G[:, None] - G[None, :], 0.0))
    return np.tril(D) * np.tri(T)


def gated_linear_attention(q, k, v, g):
    """Textbook parallel form O = (Q K^T (.) M_decay) V of one head."""
    D = decay_mask(cum_gate(g))
    return ((q @ k.T) * D) @ v


def replay_membership(b, merge, C):
    """Replay the recorded decisions on lists of token ids (Alg. 2 with the
    merges given).  Returns, per token t, the slots as lists of token ids."""
    slots, hist = [], []
    for t in range(len(b)):
        if b[t]:
            if len(slots) == C:
                i = int(merge[t])
                assert 0 <= i <= C - 2, f"t={t}: capacity reached but merge index {i}"
                slots[i] = slots[i] + slots[i + 1]
                del slots[i + 1]
            else:
                assert merge[t] == -1, f"t={t}: merge {merge[t]} below capacity"
            slots.append([t])
        else:
            assert slots, "first token must open a state"
            assert merge[t] == -1
            slots[-1].append(t)
        assert len(slots) <= C
        hist.append([list(s) for s in slots])
    return hist


def brute_outputs(q, k, v, g, lam, hist):
    """o_t = sum_j lam[t, j] sum_{s in slot j} exp(G_t - G_s) (q_t . k_s) v_s."""
    G = cum_gate(g)
    T = q.shape[0]
    out = np.zeros((T, v.shape[1]))
    for t in range(T):
        for j, members in enumerate(hist[t]):
            s = np.array(members)
            w = np.exp(G[t] - G[s]) * (k[s] @ q[t])
            lj = 1.0 if lam is None else lam[t, j]
            out[t] += lj * (w @ v[s])
    return out


def brute_term_magnitudes(q, k, v, g, lam, hist):
    """sum_j |lam[t, j]| ||S_j(t)||_F ||q_t||, S_j(t) = sum over the slot's
    members of exp(G_t - G_s) k_s v_s^T."""
    G = cum_gate(g)
    T = q.shape[0]
    mag = np.zeros(T)
    for t in range(T):
        for j, members in enumerate(hist[t]):
            s = np.array(members)
            Sj = (k[s] * np.exp(G[t] - G[s])[:, None]).T @ v[s]
            lj = 1.0 if lam is None else lam[t, j]
            mag[t] += abs(lj) * np.linalg.norm(Sj)
        mag[t] *= np.linalg.norm(q[t])
    return mag


def rms_sq_norm(x2, D, eps_rms):
    """||N(X)||^2 for ||X||^2 = x2 under RMSNorm over D entries."""
    return x2 / (x2 / D + eps_rms)


def score_rank_one(kt, vt, Sbar, eps, eps_rms):
    """Score of token state k v^T against state Sbar via the rank-one expansion
    ||N(s) - N(S)||^2 = a/rs^2 + b/rS^2 - 2 k^T S v/(rs rS)."""
    D = Sbar.size
    a = float(kt @ kt) * float(vt @ vt)
    b = float((Sbar * Sbar).sum())
    c = float(kt @ Sbar @ vt)
    rs = np.sqrt(a / D + eps_rms)
    rS = np.sqrt(b / D + eps_rms)
    num = max(0.0, a / rs**2 + b / rS**2 - 2.0 * c / (rs * rS))
    return np.sqrt(num) / (np.sqrt(b) / rS + eps)


def f64_inputs(name, **kw):
    w = WORKLOADS[name].replace(**kw) if kw else WORKLOADS[name]
    x = make_inputs(w)
    f = lambda a: to_f64(a, w.dtype)
    return w, f(x["q"]), f(x["k"]), f(x["v"]), x["g"].astype(np.float64), f(x["lam"])


# ----------------------------------------------------------------------------
# pins
# ----------------------------------------------------------------------------

def pin_lambda_one_is_gated_linear_attention(lib_path=None):
    """lambda = 1: the sum over states is the single gated state for any tau, C."""
    w, q, k, v, g, _ = f64_inputs("cfg1", T=192)
    ref = np.stack([gated_linear_attention(q[h], k[h], v[h], g[h]) for h in range(len(q))])
    for C, tau in ((8, 0.5), (3, 0.5), (1, 0.5), (4, 0.0), (2, 0.3)):
        r = oracle_forward(k, v, g, C, tau, q=q, lib_path=lib_path)
        err = np.abs(r["out"] - ref).max() / np.abs(ref).max()
        assert err < 1e-12, f"C={C} tau={tau}: rel err {err}"


def pin_single_state_and_one_state_per_token(lib_path=None):
    """C = 1 or tau = inf: o_t = lam_{t,0} q_t^T P_t.  tau <= 0 with C >= T:
    o_t = sum_s lam_{t,s} exp(G_t - G_s) (q_t . k_s) v_s."""
    w, q, k, v, g, _ = f64_inputs("cfg1", T=96)
    rng = np.random.default_rng(7)
    T = q.shape[1]
    lam = 1.0 + 0.5 * rng.standard_normal((q.shape[0], T, T))
    for h in range(q.shape[0]):
        base = gated_linear_attention(q[h], k[h], v[h], g[h])
        for C, tau in ((1, 0.5), (5, np.inf)):
            r = oracle_forward(k[h:h + 1], v[h:h + 1], g[h:h + 1], C, tau, q=q[h:h + 1],
                               lam=lam[h:h + 1, :, :C], want_mag=True, lib_path=lib_path)
            ref = lam[h, :, :1] * base
            assert np.abs(r["out"][0] - ref).max() < 1e-12 * np.abs(ref).max(), (C, tau)
            # a single state, the gated state P_t: |lam_0| ||P_t||_F ||q_t||
            G = cum_gate(g[h])
            P = [(k[h, :t + 1] * np.exp(G[t] - G[:t + 1])[:, None]).T @ v[h, :t + 1]
                 for t in range(T)]
            ref_mag = np.array([abs(lam[h, t, 0]) * np.linalg.norm(P[t]) * np.linalg.norm(q[h, t])
                                for t in range(T)])
            assert np.abs(r["mag"][0] - ref_mag).max() < 1e-12 * ref_mag.max(), (C, tau)
            assert r["b"][0, 0] == 1 and r["b"][0, 1:].sum() == 0
        r = oracle_forward(k[h:h + 1], v[h:h + 1], g[h:h + 1], T, 0.0, q=q[h:h + 1],
                           lam=lam[h:h + 1], lib_path=lib_path)
        D = decay_mask(cum_gate(g[h]))
        ref = ((q[h] @ k[h].T) * D * lam[h]) @ v[h]
        assert np.abs(r["out"][0] - ref).max() < 1e-12 * np.abs(ref).max()
        assert r["b"][0].all() and (r["merge"][0] == -1).all()


def pin_brute_force_membership(lib_path=None):
    """Tiny inputs: outputs and merges equal a replay of Alg. 2 on lists of token
    ids with a scalar argmin over (sum of scores)/(count)."""
    for name, kw, C in (("cfg1", dict(T=160, dk=8, dv=8, n_seg=12), 4),
                        ("cfg1_iid", dict(T=48, dk=4, dv=4), 3),
                        ("cfg1", dict(T=64, dk=4, dv=6, n_seg=9), 2),
                        ("cfg1", dict(T=80, dk=6, dv=4, n_seg=20, rho2=0.9), 5)):
        w, q, k, v, g, lam = f64_inputs(name, C=C, **kw)
        r = oracle_forward(k, v, g, C, w.tau, q=q, lam=lam, want_mag=True, lib_path=lib_path)
        for h in range(q.shape[0]):
            b, merge, score = r["b"][h], r["merge"][h], r["score"][h]
            hist = replay_membership(b, merge, C)
            out = brute_outputs(q[h], k[h], v[h], g[h], lam[h], hist)
            err = np.abs(out - r["out"][h]).max() / np.abs(out).max()
            assert err < 1e-11, f"{name} C={C}: brute-force output rel err {err}"
            # the scale of the readout's terms: sum_j |lambda_{t,j}| ||S_j||_F ||q_t||
            mag = brute_term_magnitudes(q[h], k[h], v[h], g[h], lam[h], hist)
            merr = np.abs(mag - r["mag"][h]).max() / mag.max()
            assert merr < 1e-11, f"{name} C={C}: term magnitudes rel err {merr}"
            assert (r["mag"][h] >= np.linalg.norm(r["out"][h], axis=-1) * (1 - 1e-12)).all()
            # independent scalar Alg. 2 on membership lists
            prev = []
            for t in range(len(b)):
                if b[t] and len(prev) == C:
                    dens = [(sum(score[prev[i]]) + sum(score[prev[i + 1]])) /
                            (len(prev[i]) + len(prev[i + 1])) for i in range(C - 1)]
                    order = sorted(range(C - 1), key=lambda i: (dens[i], i))
                    close = len(order) > 1 and dens[order[1]] - dens[order[0]] <= 1e-9 * abs(
                        dens[order[0]])
                    if not close:
                        assert merge[t] == order[0], f"t={t}: merge {merge[t]} vs {order[0]}"
                prev = hist[t]
            # m_t and counts
            assert all(len(hist[t]) == r["m"][h, t] for t in range(len(b)))


def pin_score_identical_tokens(lib_path=None):
    """Identical tokens, no decay: the newest state after n tokens is n s, so
    I_{n+1} = sqrt(a) |1/r_1 - n/r_n| / (n sqrt(a)/r_n + eps) with
    r_x = sqrt(x^2 a / D + eps_rms).  eps_rms is chosen comparable to a/D so
    that its handling matters."""
    dk, dv, T = 3, 2, 7
    kv = np.array([0.3, -0.2, 0.1])
    vv = np.array([0.05, 0.02])
    a = float(kv @ kv) * float(vv @ vv)
    D = dk * dv
    eps, eps_rms = 1e-3, a / D
    k = np.tile(kv, (1, T, 1))
    v = np.tile(vv, (1, T, 1))
    g = np.zeros((1, T))
    r = oracle_forward(k, v, g, 4, 10.0, lib_path=lib_path, eps=eps, eps_rms=eps_rms, full=True,
                       q=np.ones((1, T, dk)))
    r1 = np.sqrt(a / D + eps_rms)
    for t in range(1, T):
        n = t
        rn = np.sqrt(n * n * a / D + eps_rms)
        ref = np.sqrt(a) * abs(1.0 / r1 - n / rn) / (n * np.sqrt(a) / rn + eps)
        assert abs(r["score"][0, t] - ref) < 1e-12, (t, r["score"][0, t], ref)
    assert r["score"][0, 0] == 0.0 and r["b"][0, 0] == 1 and r["b"][0, 1:].sum() == 0


def pin_score_orthogonal_key(lib_path=None):
    """A key orthogonal to every key of the newest state gives k^T S v = 0, so
    I = sqrt(|N(s)|^2 + |N(S)|^2) / (|N(S)| + eps); decay enters through S."""
    dk, dv = 4, 3
    k = np.array([[[1.0, 0, 0, 0], [0.6, 0.8, 0, 0], [0, 0, 1.0, 0], [0.8, 0, 0, 0.6]]])
    v = np.array([[[1.0, 2.0, -1.0], [0.5, 1.0, 0.5], [-1.0, 0.3, 2.0], [0.2, 0.2, 0.2]]])
    g = np.array([[0.0, -0.3, -0.7, -0.1]])
    eps, eps_rms = 1e-4, 0.05
    D = dk * dv
    bo = np.array([[-1, 0, 1, 0]], np.int8)   # tokens 0-1 form one state, 2 opens one
    r = oracle_forward(k, v, g, 3, 0.5, lib_path=lib_path, eps=eps, eps_rms=eps_rms,
                       b_override=bo, q=np.ones((1, 4, dk)))
    # token 2 against the decayed state of tokens 0, 1
    S = np.exp(g[0, 1] + g[0, 2]) * np.outer(k[0, 0], v[0, 0]) + np.exp(g[0, 2]) * np.outer(
        k[0, 1], v[0, 1])
    s = np.outer(k[0, 2], v[0, 2])
    ns2 = rms_sq_norm((s * s).sum(), D, eps_rms)
    nS2 = rms_sq_norm((S * S).sum(), D, eps_rms)
    ref = np.sqrt(ns2 + nS2) / (np.sqrt(nS2) + eps)
    assert abs(r["score"][0, 2] - ref) < 1e-12, (r["score"][0, 2], ref)
    # token 3 against the single-token state of token 2 (k orthogonal again)
    S = np.exp(g[0, 3]) * s
    s = np.outer(k[0, 3], v[0, 3])
    ns2 = rms_sq_norm((s * s).sum(), D, eps_rms)
    nS2 = rms_sq_norm((S * S).sum(), D, eps_rms)
    ref3 = np.sqrt(ns2 + nS2) / (np.sqrt(nS2) + eps)
    assert abs(r["score"][0, 3] - ref3) < 1e-12, (r["score"][0, 3], ref3)


def pin_score_rank_one_expansion(lib_path=None):
    """Every score equals the rank-one expansion of the definition, evaluated on
    the decayed newest state rebuilt from the replayed membership lists."""
    w, q, k, v, g, lam = f64_inputs("cfg1", T=96, dk=8, dv=8, n_seg=6)
    eps, eps_rms = 1e-3, 2e-3
    r = oracle_forward(k, v, g, 4, w.tau, q=q, lam=lam[:, :, :4], eps=eps, eps_rms=eps_rms,
                       lib_path=lib_path)
    G = cum_gate(g)
    for h in range(q.shape[0]):
        hist = replay_membership(r["b"][h], r["merge"][h], 4)
        for t in range(1, q.shape[1]):
            newest = hist[t - 1][-1]
            S = sum(np.exp(G[h, t] - G[h, s]) * np.outer(k[h, s], v[h, s]) for s in newest)
            ref = score_rank_one(k[h, t], v[h, t], S, eps, eps_rms)
            assert abs(r["score"][h, t] - ref) < 1e-10, (h, t, r["score"][h, t], ref)
            assert r["b"][h, t] == (1 if r["score"][h, t] >= w.tau else 0)


def pin_scalar_states_sign_flips(lib_path=None):
    """d_k = d_v = 1, eps = eps_rms = 0: N(x) = sign(x), so I = 0 when the token
    state has the sign of the newest state and 2 otherwise.  Two schedules worked
    out by hand in tests/golden/: sign flips with tau = 1 (merges at index 0 and
    1), and tau = 2 (the equality case of I >= tau) with exactly tied densities."""
    for fixture in ("scalar_sign_flips.json", "scalar_ties.json"):
        with open(os.path.join(GOLDEN, fixture)) as fh:
            gold = json.load(fh)
        kk = np.array(gold["k"], np.float64)[None, :, None]
        vv = np.array(gold["v"], np.float64)[None, :, None]
        g = np.array(gold["g"], np.float64)[None, :]
        q = np.ones_like(kk)
        lam = np.tile(np.array(gold["lambda_row"], np.float64), (1, kk.shape[1], 1))
        r = oracle_forward(kk, vv, g, gold["C"], gold["tau"], q=q, lam=lam, eps=0.0,
                           eps_rms=0.0, lib_path=lib_path)
        assert r["score"][0].tolist() == gold["score"], (fixture, r["score"][0].tolist())
        assert r["b"][0].tolist() == gold["b"], (fixture, r["b"][0].tolist())
        assert r["merge"][0].tolist() == gold["merge"], (fixture, r["merge"][0].tolist())
        assert r["m"][0].tolist() == gold["m"], (fixture, r["m"][0].tolist())
        c = r["cache"]
        m = int(c.m[0])
        assert c.n[0, :m].tolist() == gold["final_n"], (fixture, c.n[0].tolist())
        assert c.ibar[0, :m].tolist() == gold["final_ibar"], (fixture, c.ibar[0].tolist())
        assert np.allclose(c.S[0, :m, 0, 0], gold["final_S"], rtol=0, atol=1e-12), fixture
        assert np.allclose(r["out"][0, :, 0], gold["out"], rtol=0, atol=1e-12), fixture


def pin_score_scale_invariance_and_range(lib_path=None):
    """With eps = eps_rms = 0 the score is invariant to positive scaling of all
    values or all keys; with eps > 0 it stays in [0, 2)."""
    w, q, k, v, g, _ = f64_inputs("cfg1_iid", T=64, dk=8, dv=8)
    w2, q2, k2, v2, g2, _ = f64_inputs("cfg1", T=64, dk=8, dv=8, n_seg=4)
    for (kk, vv, gg) in ((k, v, g), (k2, v2, g2)):
        r0 = oracle_forward(kk, vv, gg, 4, 0.5, eps=0.0, eps_rms=0.0, full=False,
                            lib_path=lib_path)
        r1 = oracle_forward(kk * 3.7, vv * 0.01, gg, 4, 0.5, eps=0.0, eps_rms=0.0, full=False,
                            lib_path=lib_path)
        assert np.abs(r0["score"] - r1["score"]).max() < 1e-12
        r2 = oracle_forward(kk, vv, gg, 4, 0.5, full=False, lib_path=lib_path)
        assert r2["score"].min() >= 0.0 and r2["score"].max() < 2.0
    # opposite states give the maximum 2/(1+eps) ... with eps = 0 exactly 2
    kk = np.array([[[1.0, 0.0], [1.0, 0.0]]])
    vv = np.array([[[0.5, 0.5], [-1.0, -1.0]]])
    r = oracle_forward(kk, vv, np.zeros((1, 2)), 2, 0.5, eps=0.0, eps_rms=0.0, full=False,
                       lib_path=lib_path)
    assert abs(r["score"][0, 1] - 2.0) < 1e-15


def pin_conservation(lib_path=None):
    """Counts, scores and states are conserved by merging: sum_j n_j = t,
    sum_j Ibar_j = sum_s I_s, m_t = min(#boundaries, C), #merges =
    max(0, #boundaries - C), and sum_j S_j equals the single gated state."""
    for name, C in (("cfg1", 3), ("cfg1_iid", 8), ("cfg1", 8)):
        w, q, k, v, g, lam = f64_inputs(name, T=256)
        r = oracle_forward(k, v, g, C, w.tau, q=q, lam=lam[:, :, :C], lib_path=lib_path)
        c = r["cache"]
        G = cum_gate(g)
        T = q.shape[1]
        for h in range(q.shape[0]):
            m = c.m[h]
            assert m == min(int(r["b"][h].sum()), C)
            assert int((r["merge"][h] >= 0).sum()) == max(0, int(r["b"][h].sum()) - C)
            assert c.n[h, :m].sum() == T and (c.n[h, :m] > 0).all()
            assert abs(c.ibar[h, :m].sum() - r["score"][h].sum()) < 1e-9
            P = np.einsum("s,sa,sb->ab", np.exp(G[h, -1] - G[h]), k[h], v[h])
            assert np.abs(c.S[h, :m].sum(0) - P).max() < 1e-12 * np.abs(P).max()
            mt = np.minimum(np.cumsum(r["b"][h]), C)
            assert (r["m"][h] == mt).all()


def pin_boundaries_independent_of_capacity(lib_path=None):
    """Capacity merges never touch the newest state, so b and I are the same
    for every C >= 2; decisions mode agrees with full mode."""
    w, q, k, v, g, lam = f64_inputs("cfg1", T=384, n_seg=30, rho2=0.9)
    ref = oracle_forward(k, v, g, 2, w.tau, q=q, lam=lam[:, :, :2], lib_path=lib_path)
    for C in (3, 8, 384):
        lamC = np.ones((q.shape[0], q.shape[1], C))
        r = oracle_forward(k, v, g, C, w.tau, q=q, lam=lamC, lib_path=lib_path)
        assert (r["b"] == ref["b"]).all() and np.array_equal(r["score"], ref["score"])
        rd = oracle_forward(k, v, g, C, w.tau, full=False, lib_path=lib_path)
        assert (rd["b"] == r["b"]).all() and (rd["merge"] == r["merge"]).all()
        assert np.abs(rd["score"] - r["score"]).max() < 1e-12


def pin_continuation(lib_path=None):
    """prefill(x[:T]) equals prefill(x[:T1]) followed by prefill(x[T1:]) on the
    returned cache."""
    w, q, k, v, g, lam = f64_inputs("cfg1", T=200, n_seg=10)
    C = 4
    lam = lam[:, :, :C]
    full = oracle_forward(k, v, g, C, w.tau, q=q, lam=lam, lib_path=lib_path)
    for T1 in (1, 77, 199):
        a = oracle_forward(k[:, :T1], v[:, :T1], g[:, :T1], C, w.tau, q=q[:, :T1],
                           lam=lam[:, :T1], lib_path=lib_path)
        b = oracle_forward(k[:, T1:], v[:, T1:], g[:, T1:], C, w.tau, q=q[:, T1:],
                           lam=lam[:, T1:], cache=a["cache"], lib_path=lib_path)
        assert (np.concatenate([a["b"], b["b"]], 1) == full["b"]).all()
        assert (np.concatenate([a["merge"], b["merge"]], 1) == full["merge"]).all()
        o = np.concatenate([a["out"], b["out"]], 1)
        assert np.abs(o - full["out"]).max() < 1e-12 * np.abs(full["out"]).max()


def _golden_value(x):
    return np.inf if x == "inf" else float(x)


def pin_margins_and_merge_overrides(lib_path=None):
    """The near-tie margins the parity protocol reads and the merge override,
    against a schedule worked out by hand (tests/golden/scalar_margins.json;
    Sec. 3.1 boundary indicator, Alg. 2 / Sec. 3.2 lowest-density merge):
    margin_b = |I - tau| for a freely decided boundary (infinite when forced or
    at the first token), margin_m = (d2 - d1) / d1 over the two lowest pair
    densities of a freely decided capacity merge (infinite otherwise), the
    override honoured only at a capacity merge, and an out-of-range override
    rejected."""
    with open(os.path.join(GOLDEN, "scalar_margins.json")) as fh:
        gold = json.load(fh)
    kk = np.array(gold["k"], np.float64)[None, :, None]
    vv = np.array(gold["v"], np.float64)[None, :, None]
    g = np.array(gold["g"], np.float64)[None, :]
    T = kk.shape[1]
    q = np.ones_like(kk)
    lam = np.tile(np.array(gold["lambda_row"], np.float64), (1, T, 1))
    bo = np.array(gold["boundary_override"], np.int8)[None, :]
    mo = np.array(gold["merge_override"], np.int32)[None, :]
    r = oracle_forward(kk, vv, g, gold["C"], gold["tau"], q=q, lam=lam, eps=0.0, eps_rms=0.0,
                       b_override=bo, m_override=mo, lib_path=lib_path)
    assert r["score"][0].tolist() == gold["score"], r["score"][0].tolist()
    assert r["b"][0].tolist() == gold["b"], r["b"][0].tolist()
    assert r["merge"][0].tolist() == gold["merge"], r["merge"][0].tolist()
    assert r["m"][0].tolist() == gold["m"], r["m"][0].tolist()
    for key in ("margin_b", "margin_m"):
        exp = np.array([_golden_value(x) for x in gold[key]])
        got = r[key][0]
        assert (np.isinf(exp) == np.isinf(got)).all(), (key, got.tolist())
        fin = np.isfinite(exp)
        assert np.abs(got[fin] - exp[fin]).max() < 1e-12, (key, got.tolist())
    c = r["cache"]
    m = int(c.m[0])
    assert c.n[0, :m].tolist() == gold["final_n"], c.n[0].tolist()
    assert c.ibar[0, :m].tolist() == gold["final_ibar"], c.ibar[0].tolist()
    assert np.allclose(c.S[0, :m, 0, 0], gold["final_S"], rtol=0, atol=1e-12)
    assert np.allclose(r["out"][0, :, 0], gold["out"], rtol=0, atol=1e-12)
    # an override outside [0, C - 2] at a capacity merge is an error
    for case in gold["bad_merge_override_cases"]:
        bad = mo.copy()
        bad[0, case["t"]] = case["value"]
        try:
            oracle_forward(kk, vv, g, gold["C"], gold["tau"], eps=0.0, eps_rms=0.0,
                           b_override=bo, m_override=bad, full=False, lib_path=lib_path)
        except ValueError:
            continue
        raise AssertionError(f"merge override {case['value']} at t={case['t']} accepted")


def pin_margin_b_chord_distance(lib_path=None):
    """With d_k = 1, d_v = 2 and eps = eps_rms = 0, RMSNorm scales a state to
    norm sqrt(2) along its direction, so the score is the chord distance
    |u - w| = 2 sin(theta / 2) between the unit directions of the token value
    and of the newest state (Sec. 3.1).  Replaying the boundary rule with that
    closed form on random angles fixes every score, boundary and the margin
    |I - tau| of each free decision; C = 2 (one candidate pair, so no tie is
    possible) gives an infinite merge margin at every merge."""
    rng = np.random.default_rng(5)
    T, tau = 120, 1.2
    phi = rng.uniform(0.0, 2.0 * np.pi, T)
    amp = rng.uniform(0.5, 2.0, T)
    v = np.stack([amp * np.cos(phi), amp * np.sin(phi)], axis=1)[None]
    k = np.ones((1, T, 1))
    g = np.zeros((1, T))
    for C in (T, 2):
        r = oracle_forward(k, v, g, C, tau, eps=0.0, eps_rms=0.0, full=False,
                           lib_path=lib_path)
        newest = None
        for t in range(T):
            if newest is None:
                exp_I, exp_b = 0.0, 1
            else:
                u = v[0, t] / np.linalg.norm(v[0, t])
                w = newest / np.linalg.norm(newest)
                exp_I = float(np.linalg.norm(u - w))
                exp_b = 1 if exp_I >= tau else 0
            assert abs(r["score"][0, t] - exp_I) < 1e-12, (C, t, r["score"][0, t], exp_I)
            assert r["b"][0, t] == exp_b, (C, t)
            if t == 0:
                assert np.isinf(r["margin_b"][0, t])
            else:
                assert abs(r["margin_b"][0, t] - abs(exp_I - tau)) < 1e-12, (C, t)
            newest = v[0, t].copy() if exp_b else newest + v[0, t]
        merges = r["merge"][0] >= 0
        if C == 2:
            assert merges.any() and np.isinf(r["margin_m"][0][merges]).all()
        else:
            assert not merges.any()
        assert np.isinf(r["margin_m"][0][~merges]).all()


def pin_direct_evaluation_matches_the_recurrence(lib_path=None):
    """The direct evaluator (oracle/direct.py: states as decayed sums over
    their token ranges, the readout of eq. capacity_bounded_output evaluated
    per token) agrees with the token-by-token recurrence on the recurrence's
    own decisions: sampled outputs and the final cache, with merges, ragged
    decays, lambda and C = 1."""
    from oracle import direct
    for name, kw, C in (("cfg1", dict(T=300, n_seg=20, rho2=0.9), 4),
                        ("cfg1_iid", dict(T=200), 6),
                        ("cfg1", dict(T=150), 1)):
        w, q, k, v, g, lam = f64_inputs(name, C=C, **kw)
        lam = lam[:, :, :C]
        r = oracle_forward(k, v, g, C, w.tau, q=q, lam=lam, lib_path=lib_path)
        T = q.shape[1]
        tokens = [0, 1, T // 3, T // 2 + 1, T - 2, T - 1]
        for h in range(q.shape[0]):
            o = direct.outputs_at(q[h], k[h], v[h], g[h], lam[h], r["b"][h], r["merge"][h], C,
                                  tokens)
            ref = r["out"][h, tokens]
            assert np.abs(o - ref).max() < 1e-11 * max(np.abs(ref).max(), 1e-30), (name, h)
            m, n, S = direct.final_states(k[h], v[h], g[h], r["b"][h], r["merge"][h], C)
            c = r["cache"]
            assert m == c.m[h] and (n[:m] == c.n[h, :m]).all(), (name, h)
            assert np.abs(S[:m] - c.S[h, :m]).max() < 1e-11 * np.abs(c.S[h, :m]).max()


# ----------------------------------------------------------------------------
# the delta-rule form (Gated DeltaNet base model, Sec. 2.2, eq. delta_rule_rnn)
# ----------------------------------------------------------------------------

def gated_deltanet(q, k, v, g, beta):
    """Textbook recurrence of one head, S = sum k v^T orientation:
    S_t = exp(g_t) (I - beta_t k_t k_t^T) S_{t-1} + beta_t k_t v_t^T, o_t = S_t^T q_t."""
    dk, dv = k.shape[1], v.shape[1]
    S = np.zeros((dk, dv))
    out = np.zeros((len(k), dv))
    for t in range(len(k)):
        A = np.exp(g[t]) * (np.eye(dk) - beta[t] * np.outer(k[t], k[t]))
        S = A @ S + beta[t] * np.outer(k[t], v[t])
        out[t] = S.T @ q[t]
    return out, S


def delta_range_states(k, v, g, beta, b, upto):
    """The state of every token range (a run of tokens opened by a boundary) at
    token `upto`: the delta-rule recurrence over the range's own tokens, then
    decay only once the range is closed.  Returns {first token: state}."""
    G = cum_gate(g)
    dk, dv = k.shape[1], v.shape[1]
    starts = [t for t in range(upto + 1) if b[t] or t == 0]
    out = {}
    for i, a in enumerate(starts):
        e = (starts[i + 1] - 1) if i + 1 < len(starts) else upto
        S = beta[a] * np.outer(k[a], v[a])
        for s in range(a + 1, e + 1):
            S = np.exp(g[s]) * (S - beta[s] * np.outer(k[s], k[s] @ S)) + beta[s] * np.outer(k[s], v[s])
        out[a] = np.exp(G[upto] - G[e]) * S
    return out


def _delta_inputs(name, T, C, seed, **kw):
    w, q, k, v, g, lam = f64_inputs(name, T=T, **kw)
    beta = np.random.default_rng(seed).uniform(0.05, 1.0, size=g.shape)
    return w, q, k, v, g, lam[:, :, :C], beta


def pin_delta_single_state_is_gated_deltanet(lib_path=None):
    """C = 1 with lambda = 1: the layer is the Gated DeltaNet recurrence (the
    first token's write opens the one state, every later token accumulates)."""
    w, q, k, v, g, _, beta = _delta_inputs("cfg1", 160, 1, 3)
    r = oracle_forward(k, v, g, 1, w.tau, q=q, beta=beta, lib_path=lib_path)
    for h in range(len(q)):
        ref, S = gated_deltanet(q[h], k[h], v[h], g[h], beta[h])
        assert np.abs(r["out"][h] - ref).max() < 1e-11 * np.abs(ref).max(), h
        assert np.abs(r["cache"].S[h, 0] - S).max() < 1e-11 * np.abs(S).max(), h


def pin_delta_rule_overwrites_a_unit_key(lib_path=None):
    """beta = 1 and a unit key: after the token, the accumulating state maps that
    key to exactly its value (S^T k = v), whatever it held before."""
    w, q, k, v, g, _, beta = _delta_inputs("cfg1", 64, 4, 5)
    beta[:] = 0.3
    beta[:, -1] = 1.0
    k[:, -1] /= np.linalg.norm(k[:, -1], axis=-1, keepdims=True)   # exactly unit in float64
    r = oracle_forward(k, v, g, 4, 1e30, q=q, beta=beta, lib_path=lib_path)
    for h in range(len(q)):
        assert r["cache"].m[h] == 1
        got = r["cache"].S[h, 0].T @ k[h, -1]
        assert np.abs(got - v[h, -1]).max() < 1e-12 * np.abs(v[h, -1]).max(), h


def pin_delta_zero_step_writes_nothing(lib_path=None):
    """beta = 0: no token writes anything, so every state and output is 0."""
    w, q, k, v, g, lam, beta = _delta_inputs("cfg1", 80, 4, 7)
    r = oracle_forward(k, v, g, 4, w.tau, q=q, lam=lam, beta=np.zeros_like(beta),
                       lib_path=lib_path)
    assert np.abs(r["out"]).max() == 0.0 and np.abs(r["cache"].S).max() == 0.0


def pin_delta_ranges_and_merges(lib_path=None):
    """With boundaries and capacity merges: each state is the sum of the token
    ranges merged into it (Alg. 2 replayed on membership lists), each range the
    delta-rule recurrence over its own tokens while it was the newest state and
    decayed only after it closed; outputs as in eq. capacity_bounded_output."""
    for name, T, C, kw in (("cfg1", 140, 4, dict(n_seg=12, rho2=0.9)), ("cfg1_iid", 60, 3, {})):
        w, q, k, v, g, lam, beta = _delta_inputs(name, T, C, 11, **kw)
        r = oracle_forward(k, v, g, C, w.tau, q=q, lam=lam, beta=beta, lib_path=lib_path)
        for h in range(len(q)):
            b, mg = r["b"][h], r["merge"][h]
            assert (mg >= 0).sum() > 0, "the case must merge"
            hist = replay_membership(b, mg, C)
            for t in (0, 1, T // 2, T - 1):
                rs = delta_range_states(k[h], v[h], g[h], beta[h], b, t)
                o = np.zeros(v.shape[2])
                for j, slot in enumerate(hist[t]):
                    Sj = sum(rs[a] for a in slot if a in rs)
                    o += lam[h, t, j] * (Sj.T @ q[h, t])
                ref = r["out"][h, t]
                assert np.abs(o - ref).max() < 1e-10 * max(np.abs(ref).max(), 1e-30), (name, h, t)
            rs = delta_range_states(k[h], v[h], g[h], beta[h], b, T - 1)
            for j, slot in enumerate(hist[T - 1]):
                Sj = sum(rs[a] for a in slot if a in rs)
                assert np.abs(Sj - r["cache"].S[h, j]).max() < 1e-10 * np.abs(Sj).max(), (name, h, j)


def pin_delta_decisions_mode(lib_path=None):
    """The decisions mode (newest state only) takes the full mode's decisions
    with the delta rule too."""
    w, q, k, v, g, lam, beta = _delta_inputs("cfg1", 200, 4, 13, n_seg=10)
    full = oracle_forward(k, v, g, 4, w.tau, q=q, lam=lam, beta=beta, lib_path=lib_path)
    dec = oracle_forward(k, v, g, 4, w.tau, beta=beta, full=False, lib_path=lib_path)
    assert np.array_equal(full["b"], dec["b"]) and np.array_equal(full["merge"], dec["merge"])
    assert np.abs(full["score"] - dec["score"]).max() < 1e-12


def pin_delta_pseudo_values(lib_path=None):
    """The exported write vectors u_t (each token adds k_t u_t^T): at C = 1
    they are beta_t (v_t - (exp(g_t) S_{t-1})^T k_t) of the textbook Gated
    DeltaNet states (beta_t v_t at the first token); with boundaries and
    merges, the direct evaluator given u in place of v reproduces the delta
    recurrence's outputs and final cache in decisions mode too."""
    from oracle import direct
    w, q, k, v, g, _, beta = _delta_inputs("cfg1", 120, 1, 17)
    r = oracle_forward(k, v, g, 1, w.tau, q=q, beta=beta, want_u=True, lib_path=lib_path)
    for h in range(len(q)):
        dk, dv = k.shape[2], v.shape[2]
        S = np.zeros((dk, dv))
        for t in range(q.shape[1]):
            want = beta[h, t] * (v[h, t] - (np.exp(g[h, t]) * S).T @ k[h, t])
            assert np.abs(r["u"][h, t] - want).max() < 1e-12 * max(np.abs(want).max(), 1e-30)
            A = np.exp(g[h, t]) * (np.eye(dk) - beta[h, t] * np.outer(k[h, t], k[h, t]))
            S = A @ S + beta[h, t] * np.outer(k[h, t], v[h, t])
    for name, T, C, kw in (("cfg1", 220, 4, dict(n_seg=14, rho2=0.9)), ("cfg1_iid", 70, 3, {})):
        w, q, k, v, g, lam, beta = _delta_inputs(name, T, C, 19, **kw)
        r = oracle_forward(k, v, g, C, w.tau, q=q, lam=lam, beta=beta, want_u=True,
                           lib_path=lib_path)
        dec = oracle_forward(k, v, g, C, w.tau, beta=beta, full=False, want_u=True,
                             lib_path=lib_path)
        assert np.abs(r["u"] - dec["u"]).max() < 1e-12 * np.abs(r["u"]).max()
        tokens = [0, 1, T // 3, T // 2 + 1, T - 2, T - 1]
        for h in range(len(q)):
            assert (r["merge"][h] >= 0).sum() > 0, "the case must merge"
            o = direct.outputs_at(q[h], k[h], r["u"][h], g[h], lam[h], r["b"][h], r["merge"][h], C,
                                  tokens)
            ref = r["out"][h, tokens]
            assert np.abs(o - ref).max() < 1e-10 * max(np.abs(ref).max(), 1e-30), (name, h)
            m, n, S = direct.final_states(k[h], r["u"][h], g[h], r["b"][h], r["merge"][h], C)
            c = r["cache"]
            assert m == c.m[h] and (n[:m] == c.n[h, :m]).all(), (name, h)
            assert np.abs(S[:m] - c.S[h, :m]).max() < 1e-10 * np.abs(c.S[h, :m]).max(), (name, h)


ALL_PINS = [
    pin_lambda_one_is_gated_linear_attention,
    pin_single_state_and_one_state_per_token,
    pin_brute_force_membership,
    pin_score_identical_tokens,
    pin_score_orthogonal_key,
    pin_score_rank_one_expansion,
    pin_scalar_states_sign_flips,
    pin_score_scale_invariance_and_range,
    pin_conservation,
    pin_boundaries_independent_of_capacity,
    pin_continuation,
    pin_margins_and_merge_overrides,
    pin_margin_b_chord_distance,
    pin_direct_evaluation_matches_the_recurrence,
    pin_delta_single_state_is_gated_deltanet,
    pin_delta_rule_overwrites_a_unit_key,
    pin_delta_zero_step_writes_nothing,
    pin_delta_ranges_and_merges,
    pin_delta_decisions_mode,
    pin_delta_pseudo_values,
]
