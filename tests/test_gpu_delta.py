"""GPU parity of the Gated DeltaNet form (delta rule on the newest state, step
sizes beta; Sec. 2.2, eq. delta_rule_rnn): dla_decode_step_delta and
dla_prefill_delta through the C ABI against the float64 oracle given the same
beta.  Decisions bit-exact with near ties pinned, outputs and final cache
within the tolerances of the gated form."""
import numpy as np
import pytest

from oracle import oracle_forward
from tests import harness as H
from paper_2606_10650_amd.workloads import WORKLOADS, make_inputs, make_beta

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _oracle(w, x, beta, b_override=None, m_override=None):
    xf = H.f64(x, w)
    return oracle_forward(xf["k"], xf["v"], xf["g"], w.C, w.tau, q=xf["q"], lam=xf.get("lam"),
                          beta=beta.astype(np.float64), b_override=b_override,
                          m_override=m_override, want_mag=True)


def _case(w, mode, state_dtype=0, no_lambda=False, pool_budget_log2=0):
    """mode: 'prefill' (dla_prefill_delta) or 'decode' (T steps of
    dla_decode_step_delta)."""
    torch = _torch()
    from paper_2606_10650_amd import dla
    x = make_inputs(w)
    if no_lambda:
        del x["lam"]
    beta = make_beta(w)
    ref = _oracle(w, x, beta)
    bo, mo, nb, nm = H.near_tie_overrides(ref, what=f"delta {mode} {w.label}")
    q, k, v, g, lam = H.inputs_to_device(w, x, w.B, w.H)
    shp = (w.B, w.H, w.T)
    bt = torch.from_numpy(beta).reshape(shp).cuda()
    bo_d = torch.from_numpy(bo).reshape(shp).cuda()
    mo_d = torch.from_numpy(mo).reshape(shp).cuda()
    cache = dla.cache_alloc(w.B, w.H, w.C, w.dk, w.dv, state_dtype=state_dtype)
    if mode == "prefill":
        out, b, mi, sc = dla.prefill_delta(cache, q, k, v, g, bt, lam, tau=w.tau,
                                           boundary_override=bo_d, merge_override=mo_d,
                                           pool_budget_log2=pool_budget_log2)
    else:
        outs, bs, ms, ss = [], [], [], []
        for t in range(w.T):
            sl = lambda a: None if a is None else a[:, :, t].contiguous()
            o, bb, mm, s_ = dla.decode_step_delta(cache, sl(q), sl(k), sl(v), sl(g), sl(bt), sl(lam),
                                                  tau=w.tau, boundary_override=sl(bo_d),
                                                  merge_override=sl(mo_d))
            outs.append(o); bs.append(bb); ms.append(mm); ss.append(s_)
        out, b, mi, sc = (torch.stack(z, 2) for z in (outs, bs, ms, ss))
    torch.cuda.synchronize()
    nh = w.B * w.H
    H.assert_decisions(b.cpu().numpy().reshape(nh, -1), mi.cpu().numpy().reshape(nh, -1), ref,
                       w.label)
    serr = np.abs(sc.cpu().numpy().reshape(nh, -1) - ref["score"]).max()
    assert serr < H.DELTA_B / 10, f"score error {serr}"
    sb = state_dtype == dla.DLA_BF16
    tol = H.TOL["bf16"] if (w.dtype == "bf16" or sb) else H.TOL["f32"]
    rel = H.assert_outputs(out.float().cpu().numpy().reshape(nh, w.T, w.dv), ref["out"], tol,
                           w.label, mag=ref["mag"], mag_tol=H.state_mag_tol(sb, w.dk))
    srel = H.assert_cache(dla.cache_export(cache), ref["cache"], H.STATE_TOL[sb], what=w.label)
    assert dla.cache_flags(cache) == 0
    print(f"[delta-ok] {mode} {w.label} near={nb}+{nm} boundaries={int(ref['b'].sum())} "
          f"merges={int((ref['merge'] >= 0).sum())} max_rel_out={rel:.2e} "
          f"max_rel_state={srel:.2e}", flush=True)


@pytest.mark.parametrize("mode", ["decode", "prefill"])
def test_delta_matches_oracle_f32(mode):
    _case(WORKLOADS["cfg1"].replace(T=240, n_seg=8), mode)


@pytest.mark.parametrize("mode", ["decode", "prefill"])
def test_delta_matches_oracle_bf16(mode):
    _case(WORKLOADS["cfg2"].replace(B=1, H=2, T=400, C=4), mode)


def test_delta_every_token_a_boundary_and_merge():
    _case(WORKLOADS["cfg1_iid"].replace(T=120), "prefill")


def test_delta_single_state_is_gated_deltanet():
    """C = 1: every token after the first accumulates under the delta rule."""
    _case(WORKLOADS["cfg2"].replace(B=1, H=2, T=300, C=1), "prefill")


def test_delta_mixed_head_dims_and_no_lambda():
    _case(WORKLOADS["cfg2"].replace(B=2, H=1, T=150, C=5, dk=128, dv=64), "prefill")
    _case(WORKLOADS["cfg2"].replace(B=1, H=2, T=150, C=5, dk=64, dv=128), "decode", no_lambda=True)


def test_delta_bf16_state_storage():
    _case(WORKLOADS["cfg2"].replace(B=1, H=2, T=300, C=6), "prefill", state_dtype=1)


def test_delta_one_workgroup_per_head():
    """1024 heads: the decode step runs one workgroup per head (no split), and
    the prefill's scan one workgroup per head."""
    from paper_2606_10650_amd import dla
    w = WORKLOADS["cfg1"].replace(B=64, H=16, T=24, C=4)
    assert dla.lib() and w.B * w.H >= 1024
    _case(w, "decode")
    _case(w.replace(T=300), "prefill")


def test_delta_prefill_long_bf16():
    """Spans and bursts over 2600 tokens: several chunks of the update and
    readout stages, merges at a full cache of 24."""
    _case(WORKLOADS["cfg3"].replace(B=1, H=2, T=2600, C=24), "prefill")


def test_delta_prefill_long_f32():
    _case(WORKLOADS["cfg1"].replace(T=1500, n_seg=24, C=8), "prefill")


def test_delta_prefill_small_pool_budget():
    """A state-copy budget of 8 MiB splits the stages into segments of a
    chunk or two."""
    from paper_2606_10650_amd import dla
    w = WORKLOADS["cfg3"].replace(B=1, H=2, T=2600, C=24)
    c = dla.cache_alloc(w.B, w.H, w.C, w.dk, w.dv)
    assert dla.delta_workspace_bytes(c, w.T, pool_budget_log2=23) < dla.delta_workspace_bytes(c, w.T)
    _case(w, "prefill", pool_budget_log2=23)


def test_delta_prefill_split_then_decode():
    """Two prefill calls and then decode steps continue one sequence: the
    second call starts from the cache (and the newest state) the first left,
    and the steps from the second's, against one oracle run."""
    torch = _torch()
    from paper_2606_10650_amd import dla
    w = WORKLOADS["cfg2"].replace(B=1, H=2, T=900, C=10)
    T1, T2 = 333, 850
    x = make_inputs(w)
    beta = make_beta(w)
    ref = _oracle(w, x, beta)
    bo, mo, nb, nm = H.near_tie_overrides(ref, what="delta split")
    q, k, v, g, lam = H.inputs_to_device(w, x, w.B, w.H)
    shp = (w.B, w.H, w.T)
    bt = torch.from_numpy(beta).reshape(shp).cuda()
    bo_d = torch.from_numpy(bo).reshape(shp).cuda()
    mo_d = torch.from_numpy(mo).reshape(shp).cuda()
    cache = dla.cache_alloc(w.B, w.H, w.C, w.dk, w.dv)
    parts = []
    for a0, a1 in ((0, T1), (T1, T2)):
        sl = lambda z: z[:, :, a0:a1].contiguous()
        parts.append(dla.prefill_delta(cache, sl(q), sl(k), sl(v), sl(g), sl(bt), sl(lam),
                                       tau=w.tau, boundary_override=sl(bo_d),
                                       merge_override=sl(mo_d)))
    for t in range(T2, w.T):
        sl = lambda z: z[:, :, t].contiguous()
        o, bb, mm, s_ = dla.decode_step_delta(cache, sl(q), sl(k), sl(v), sl(g), sl(bt), sl(lam),
                                              tau=w.tau, boundary_override=sl(bo_d),
                                              merge_override=sl(mo_d))
        parts.append((o.unsqueeze(2), bb.unsqueeze(2), mm.unsqueeze(2), s_.unsqueeze(2)))
    torch.cuda.synchronize()
    out, b, mi, sc = (torch.cat([p_[i] for p_ in parts], 2) for i in range(4))
    nh = w.B * w.H
    H.assert_decisions(b.cpu().numpy().reshape(nh, -1), mi.cpu().numpy().reshape(nh, -1), ref,
                       "delta split")
    rel = H.assert_outputs(out.float().cpu().numpy().reshape(nh, w.T, w.dv), ref["out"],
                           H.TOL["bf16"], "delta split", mag=ref["mag"], mag_tol=0.0)
    srel = H.assert_cache(dla.cache_export(cache), ref["cache"], H.STATE_TOL[False],
                          what="delta split")
    assert dla.cache_flags(cache) == 0
    print(f"[delta-ok] split {T1}+{T2 - T1}+{w.T - T2} near={nb}+{nm} max_rel_out={rel:.2e} "
          f"max_rel_state={srel:.2e}", flush=True)


def test_delta_prefill_skip_readout_and_refusals():
    """SKIP_READOUT builds the same cache; a missing beta, a short workspace
    and an unaligned one are refused before any work."""
    torch = _torch()
    import ctypes
    from paper_2606_10650_amd import dla
    w = WORKLOADS["cfg2"].replace(B=1, H=2, T=700, C=8)
    x = make_inputs(w)
    beta = make_beta(w)
    ref = _oracle(w, x, beta)
    bo, mo, nb, nm = H.near_tie_overrides(ref, what="delta skip")
    q, k, v, g, lam = H.inputs_to_device(w, x, w.B, w.H)
    shp = (w.B, w.H, w.T)
    bt = torch.from_numpy(beta).reshape(shp).cuda()
    cache = dla.cache_alloc(w.B, w.H, w.C, w.dk, w.dv)
    dla.prefill_delta(cache, None, k, v, g, bt, None, tau=w.tau, skip_readout=True,
                      boundary_override=torch.from_numpy(bo).reshape(shp).cuda(),
                      merge_override=torch.from_numpy(mo).reshape(shp).cuda())
    torch.cuda.synchronize()
    H.assert_cache(dla.cache_export(cache), ref["cache"], H.STATE_TOL[False], what="delta skip")
    L = dla.lib()
    p = dla._params(w.tau, 1e-6, 1e-6, False)
    need = dla.delta_workspace_bytes(cache, w.T)
    ws = torch.empty(need + 512, dtype=torch.uint8, device="cuda")
    out = torch.empty((w.B, w.H, w.T, w.dv), dtype=k.dtype, device="cuda")
    def call(beta_ptr, wptr, wbytes):
        return L.dla_prefill_delta(ctypes.byref(cache.desc), dla._ptr(cache.buf), dla._ptr(q),
                                   dla._ptr(k), dla._ptr(v), dla._ptr(g), beta_ptr, dla._ptr(lam),
                                   w.T, dla.DLA_BF16, ctypes.byref(p), dla._ptr(out), dla.DLA_BF16,
                                   None, None, None, None, None, wptr, wbytes, dla._stream(q.device))
    before = cache.buf.clone()
    assert call(None, dla._ptr(ws), need) == dla.DLA_ERR_INVALID_ARG
    assert call(dla._ptr(bt), dla._ptr(ws), need - 1) == dla.DLA_ERR_WORKSPACE
    assert call(dla._ptr(bt), ctypes.c_void_p(ws.data_ptr() + 128), need) == dla.DLA_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert torch.equal(before, cache.buf)


def test_delta_prefill_full_size_sampled_heads():
    """The delta form at the 16k-token workload's full size (B=4, H=16,
    T=16384, C=128), the call the benchmark times.  Six heads spread over batch
    and head: every decision and score, the outputs of four windows and the
    final cache, against the oracle's decisions mode with its write vectors u
    and the direct evaluation over them (both pinned to the delta
    recurrence)."""
    torch = _torch()
    from oracle import OracleCache, direct
    from paper_2606_10650_amd import dla
    from tests.test_gpu_full_size import spread_heads, windows
    w = WORKLOADS["cfg3"]
    nh = w.B * w.H
    heads = spread_heads(w.B, w.H, 6)
    x = make_inputs(w)
    beta = make_beta(w)
    xs = H.f64({key: x[key][heads] for key in ("q", "k", "v", "lam", "g")}, w)
    dec = oracle_forward(xs["k"], xs["v"], xs["g"], w.C, w.tau, beta=beta[heads].astype(np.float64),
                         full=False, want_u=True)
    bo_s, mo_s, nb, nm = H.near_tie_overrides(dec, what=f"delta {w.label} full size")
    bo = np.full((nh, w.T), -1, np.int8)
    mo = np.full((nh, w.T), -1, np.int32)
    bo[heads], mo[heads] = bo_s, mo_s
    q, k, v, g, lam = H.inputs_to_device(w, x, w.B, w.H)
    del x
    shp = (w.B, w.H, w.T)
    cache = dla.cache_alloc(w.B, w.H, w.C, w.dk, w.dv)
    out, b, mi, sc = dla.prefill_delta(cache, q, k, v, g, torch.from_numpy(beta).reshape(shp).cuda(),
                                       lam, tau=w.tau,
                                       boundary_override=torch.from_numpy(bo).reshape(shp).cuda(),
                                       merge_override=torch.from_numpy(mo).reshape(shp).cuda())
    torch.cuda.synchronize()
    H.assert_decisions(b.cpu().numpy().reshape(nh, w.T)[heads],
                       mi.cpu().numpy().reshape(nh, w.T)[heads], dec, w.label)
    serr = np.abs(sc.cpu().numpy().reshape(nh, w.T)[heads] - dec["score"]).max()
    assert serr < H.DELTA_B / 10, f"score error {serr}"
    # windows inside a chunk (512 tokens), across the start of a later segment
    # of the pipelined call, the last segment's first tokens and the end
    seg_starts = dla.prefill_segment_starts(cache, w.T, torch.bfloat16)
    toks, wins = windows(w.T, 512, seg_starts)
    og = out.float().reshape(nh, w.T, w.dv)[heads][:, toks].cpu().numpy()
    del q, k, v, g, lam, out
    oc = OracleCache.empty(len(heads), w.C, w.dk, w.dv)
    ref_o = np.zeros((len(heads), len(toks), w.dv))
    for i in range(len(heads)):
        u = dec["u"][i]
        ref_o[i] = direct.outputs_at(xs["q"][i], xs["k"][i], u, xs["g"][i], xs["lam"][i],
                                     dec["b"][i], dec["merge"][i], w.C, toks)
        m, n, S = direct.final_states(xs["k"][i], u, xs["g"][i], dec["b"][i], dec["merge"][i], w.C)
        assert m == dec["cache"].m[i] and (n[:m] == dec["cache"].n[i, :m]).all()
        oc.m[i], oc.n[i], oc.S[i] = m, n, S
        oc.ibar[i] = dec["cache"].ibar[i]
    rel = H.assert_outputs(og, ref_o, H.TOL[w.dtype], f"delta {w.label} windows {wins}")
    exp = dla.cache_export(cache, heads=heads)
    H.assert_cache(exp, oc, 1e-4, what=f"delta {w.label}")
    print(f"[delta-full-ok] {w.label} heads={heads} near={nb}+{nm} "
          f"boundaries={int(dec['b'].sum())} merges={int((dec['merge'] >= 0).sum())} "
          f"segments={len(seg_starts)} windows={wins} max_rel_out={rel:.2e} "
          f"max_score_err={serr:.2e}", flush=True)


def _random_cases(n, seed):
    """Seeded shape mixes for the delta form: head counts off the 8-head
    groups of the update and readout grids, token counts around the 64-token
    staging rounds and the readout chunks, capacities from 1 to past 128, all
    head sizes, both input types, with and without lambda, both state types;
    decode runs the shorter ones step by step.  i.i.d. tokens keep capacities
    up to 33: at 130 their merge densities tie too often for the harness's
    bound on near-tie pins."""
    rng = np.random.default_rng(seed)
    structures = ["cuts", "geom", "spans_bursts", "iid"]
    cases = []
    for i in range(n):
        dtype = ["f32", "bf16"][i % 2]
        mode = "decode" if i % 4 == 3 else "prefill"
        rl = 256 if dtype == "f32" else 512
        choices = [1, 63, 64, 65, 130] if mode == "decode" else [1, 63, 65, rl - 1, rl + 1, 2 * rl + 37]
        T = int(rng.choice(choices))
        dk, dv = [(64, 64), (128, 128), (64, 128), (128, 64)][int(rng.integers(4))]
        C = int(rng.choice([1, 2, 3, 7, 33, 130]))
        B, Hh = int(rng.choice([1, 2, 3])), int(rng.choice([1, 3, 5]))
        st = structures[int(rng.integers(len(structures)))]
        if st == "iid":
            C = min(C, 33)
        w = WORKLOADS["cfg1"].replace(
            name=f"delta_random{i}", B=B, H=Hh, T=T, dk=dk, dv=dv, C=C, dtype=dtype,
            tau=round(float(rng.uniform(0.1, 0.9)), 2), seed=2000 + i, structure=st,
            n_seg=max(1, T // 50), mean_len=40.0, span_mean=200.0, burst_mean=8.0,
            g_lo=float(rng.choice([-0.05, -0.01])))
        cases.append((w, mode, bool(rng.integers(2)), (i // 2) % 2))
    return cases


@pytest.mark.parametrize("w,mode,no_lambda,state_dtype", _random_cases(16, 20261203),
                         ids=[f"delta_random{i}" for i in range(16)])
def test_delta_random_shapes(w, mode, no_lambda, state_dtype):
    _case(w, mode, state_dtype=state_dtype, no_lambda=no_lambda)


def _bits_equal(a, b):
    torch = _torch()
    if a.dtype in (torch.bfloat16, torch.float16):
        return torch.equal(a.view(torch.int16), b.view(torch.int16))
    if a.dtype == torch.float32:
        return torch.equal(a.view(torch.int32), b.view(torch.int32))
    return torch.equal(a, b)


@pytest.mark.parametrize("case", ["bf16_ragged", "f32", "continuation", "small_budgets"])
def test_delta_pipelined_matches_serial(case):
    """The delta form's pipelined prefill (scan segments on a second stream,
    each resuming from the carry of the one before) gives bit-identical
    outputs, exports and caches to the serial one: ragged last chunk, float32
    inputs (256-token chunks), a continuation on a non-empty cache, and small
    state-copy budgets that split both calls into many segments, differently."""
    torch = _torch()
    from paper_2606_10650_amd import dla
    budgets = (0, 0)
    cut = None
    if case == "bf16_ragged":
        w = WORKLOADS["cfg3"].replace(B=1, H=3, T=2600, C=24, span_mean=200.0)
    elif case == "f32":
        w = WORKLOADS["cfg1"].replace(T=1000)
    elif case == "continuation":
        w, cut = WORKLOADS["cfg2"].replace(B=1, H=2, T=2900, C=16), 1100
    else:
        # 4 heads x 128 states x 32 KiB: 16 MiB of copies per chunk; budgets of
        # 64 MiB (pipelined) and 32 MiB (serial)
        w = WORKLOADS["cfg3"].replace(B=1, H=4, T=5000)
        budgets = (26, 25)
    x = make_inputs(w)
    beta = make_beta(w)
    q, k, v, g, lam = H.inputs_to_device(w, x, w.B, w.H)
    bt = torch.from_numpy(beta).reshape(w.B, w.H, w.T).cuda()
    cuts = [0, w.T] if cut is None else [0, cut, w.T]
    res = {}
    for serial in (False, True):
        kb = budgets[1 if serial else 0]
        cache = dla.cache_alloc(w.B, w.H, w.C, w.dk, w.dv)
        outs = []
        for a, b in zip(cuts[:-1], cuts[1:]):
            sl = lambda t: t[:, :, a:b].contiguous()
            nseg = dla.prefill_segments(cache, b - a, k.dtype, serial=serial, pool_budget_log2=kb)
            o, bd, mi, sc = dla.prefill_delta(cache, sl(q), sl(k), sl(v), sl(g), sl(bt), sl(lam),
                                              tau=w.tau, serial=serial, pool_budget_log2=kb)
            torch.cuda.synchronize()
            outs.append((o.cpu(), bd.cpu(), mi.cpu(), sc.cpu(), nseg))
        res[serial] = (outs, dla.cache_export(cache))
    (op, cp), (os_, cs) = res[False], res[True]
    print(f"[delta-pipe] {case} segments pipelined={[o[4] for o in op]} serial={[o[4] for o in os_]}",
          flush=True)
    # (the counts are dla_prefill's plan; the delta call splits a shared pool's
    # call into at least as many segments)
    assert any(o[4] > 1 for o in op)
    for a, b in zip(op, os_):
        for ta, tb in zip(a[:4], b[:4]):
            assert _bits_equal(ta, tb), case
    for key in cp:
        assert np.array_equal(cp[key], cs[key]), (case, key)
    assert int(os_[-1][1].sum()) > 1
