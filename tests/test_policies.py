"""Fixed state-merging policies (every-K blocking, log-linear buckets, single
state) as override schedules: the shapes they give the cache, checked by
running the float64 oracle with the schedule as its overrides."""
import math

import numpy as np
import pytest

from oracle import oracle_forward
from paper_2606_10650_amd import policies as P


def _run(T, C, b, m, heads=2, seed=0, dk=8, dv=4):
    rng = np.random.default_rng(seed)
    k = rng.standard_normal((heads, T, dk))
    v = rng.standard_normal((heads, T, dv))
    g = -0.05 * rng.random((heads, T))
    bo = None if b is None else np.broadcast_to(b, (heads, T)).copy()
    mo = None if m is None else np.broadcast_to(m, (heads, T)).copy()
    return oracle_forward(k, v, g, C, 0.5, full=False, b_override=bo, m_override=mo)


def _sizes_timeline(C, b, m):
    """Token counts of the states after every token, replaying the schedule."""
    sizes, out = [], []
    for t in range(len(b)):
        if b[t] == 1 or not sizes:
            if len(sizes) == C:
                i = int(m[t])
                sizes[i] += sizes[i + 1]
                del sizes[i + 1]
            sizes.append(1)
        else:
            sizes[-1] += 1
        out.append(list(sizes))
    return out


def test_log_linear_capacity_is_the_bucket_count():
    # L = ceil(log2(t + 1)) + 1 buckets for a prefix of t + 1 tokens (Sec. 2.3)
    assert [P.log_linear_capacity(T) for T in (1, 2, 3, 4, 7, 8, 128, 65536)] == \
        [1, 2, 3, 3, 4, 4, 8, 17]
    assert P.log_linear_capacity(2 ** 29) == 30   # the paper's maximum of 30 states


@pytest.mark.parametrize("T", [1, 2, 3, 17, 64, 128, 300, 1000])
def test_log_linear_buckets_are_powers_of_two_finest_at_the_present(T):
    C, b, m = P.log_linear(T)
    assert C == P.log_linear_capacity(T)
    assert (b == 1).all()
    for t, s in enumerate(_sizes_timeline(C, b, m)):
        assert sum(s) == t + 1
        assert len(s) == min(t + 1, C)
        assert all(x & (x - 1) == 0 for x in s), (t, s)          # powers of two
        assert all(s[i] >= s[i + 1] for i in range(len(s) - 1)), (t, s)  # coarse to fine
        assert s[-1] == 1                                         # the newest token alone
        assert s[0] <= 2 ** int(math.floor(math.log2(t + 1)))


def test_log_linear_matches_the_fenwick_buckets_at_powers_of_two():
    # At T = 2^n tokens the prefix splits into the current token and buckets of
    # 1, 2, 4, ..., 2^(n-1) tokens: L = n + 1 buckets (Sec. 2.3).
    for n in (1, 4, 7, 10, 12):
        T = 2 ** n
        C, b, m = P.log_linear(T)
        assert C == n + 1
        assert _sizes_timeline(C, b, m)[-1] == [2 ** e for e in range(n - 1, -1, -1)] + [1]


@pytest.mark.parametrize("T", [5, 64, 200])
def test_log_linear_schedule_through_the_oracle(T):
    C, b, m = P.log_linear(T)
    ref = _run(T, C, b, m)
    want = _sizes_timeline(C, b, m)[-1]
    for h in range(2):
        assert (ref["b"][h, 1:] == 1).all()
        assert np.array_equal(ref["merge"][h], m), "merges follow the schedule"
        assert ref["m"][h, -1] == len(want)
        assert list(ref["cache"].n[h, :len(want)]) == want
        assert not np.isfinite(ref["margin_b"][h]).any()   # nothing decided from the data
        assert not np.isfinite(ref["margin_m"][h]).any()


@pytest.mark.parametrize("T,K,C", [(200, 16, 5), (64, 64, 30), (1000, 64, 30), (130, 8, 2)])
def test_every_k_keeps_recent_blocks_and_one_summary(T, K, C):
    C, b, m = P.every_k(T, K, C)
    assert np.array_equal(np.flatnonzero(b == 1), np.arange(0, T, K))
    ref = _run(T, C, b, m)
    nblk = -(-T // K)
    for h in range(2):
        n = list(ref["cache"].n[h, :ref["m"][h, -1]])
        if nblk <= C:
            want = [K] * (nblk - 1) + [T - K * (nblk - 1)]
        else:
            # the oldest state summarises everything before the C - 1 newest blocks
            last = T - K * (nblk - 1)
            want = [T - K * (C - 2) - last] + [K] * (C - 2) + [last]
        assert n == want, (n, want)
        merges = ref["merge"][h][ref["merge"][h] >= 0]
        assert (merges == 0).all() and len(merges) == max(0, nblk - C)


def test_every_k_continuation_offsets_the_blocks():
    _, b0, _ = P.every_k(100, 16, 4)
    _, b1, _ = P.every_k(60, 16, 4, t0=100)
    assert np.array_equal(np.concatenate([b0, b1]), P.every_k(160, 16, 4)[1])


def test_single_state_is_the_base_model():
    C, b, m = P.single_state(50)
    ref = _run(50, C, b, m)
    assert C == 1 and (ref["m"][:, -1] == 1).all() and (ref["cache"].n[:, 0] == 50).all()


def test_schedule_dispatch():
    assert P.schedule("dla", 100)[1:] == (None, None)
    assert P.schedule("log_linear", 128)[0] == 8
    assert P.schedule("every_k", 128, C_dla=30, K=64)[0] == 30
    with pytest.raises(ValueError):
        P.schedule("fenwick", 10)
