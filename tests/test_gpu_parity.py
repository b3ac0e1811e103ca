"""GPU parity: the HIP path (through the C ABI) against the float64 oracle on
the same seeded inputs.  Decisions bit-exact (near ties pinned to the oracle's
choice), outputs within 1e-4 (float32 inputs) or 2e-2 (bfloat16 inputs)
relative, final cache states within 1e-4, token counts exact."""
import numpy as np
import pytest

from oracle import oracle_forward
from tests import harness as H
from paper_2606_10650_amd.workloads import WORKLOADS, make_inputs, make_decode_tokens

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _dla():
    from paper_2606_10650_amd import dla
    return dla


def _report(tag, **kw):
    print(f"[{tag}] " + " ".join(f"{k}={v}" for k, v in kw.items()), flush=True)


def _prefill_case(w, C=None, tau=None, T_split=None, out_dtype=None, no_lambda=False,
                  state_dtype=0):
    """state_dtype: DLA_F32 (0) or DLA_BF16 (1) storage of the cache's states."""
    torch = _torch()
    dla = _dla()
    C = C or w.C
    tau = w.tau if tau is None else tau
    w = w.replace(C=C, tau=tau)
    x = make_inputs(w)
    if no_lambda:
        del x["lam"]  # every state weighted 1, on both sides
    ref = H.run_oracle(w, x)
    bo, mo, nb, nm = H.near_tie_overrides(ref, what=w.label)
    _report("prefill", case=w.label, near_b=nb, near_m=nm, boundaries=int(ref["b"].sum()),
            merges=int((ref["merge"] >= 0).sum()))
    q, k, v, g, lam = H.inputs_to_device(w, x, w.B, w.H)
    cache = dla.cache_alloc(w.B, w.H, C, w.dk, w.dv, state_dtype=state_dtype)
    shp = (w.B, w.H, w.T)
    bo_d = torch.from_numpy(bo).reshape(shp).cuda()
    mo_d = torch.from_numpy(mo).reshape(shp).cuda()
    if T_split is None:
        out, b, mi, sc = dla.prefill(cache, q, k, v, g, lam, tau=tau, boundary_override=bo_d,
                                     merge_override=mo_d, out_dtype=out_dtype)
    else:
        parts = []
        s0 = 0
        for s1 in list(T_split) + [w.T]:
            sl = slice(s0, s1)
            parts.append(dla.prefill(cache, q[:, :, sl].contiguous(), k[:, :, sl].contiguous(),
                                     v[:, :, sl].contiguous(), g[:, :, sl].contiguous(),
                                     lam[:, :, sl].contiguous(), tau=tau,
                                     boundary_override=bo_d[:, :, sl].contiguous(),
                                     merge_override=mo_d[:, :, sl].contiguous()))
            s0 = s1
        out, b, mi, sc = (torch.cat([p[i] for p in parts], dim=2) for i in range(4))
    torch.cuda.synchronize()
    nh = w.B * w.H
    H.assert_decisions(b.cpu().numpy().reshape(nh, -1), mi.cpu().numpy().reshape(nh, -1), ref,
                       w.label)
    serr = np.abs(sc.cpu().numpy().reshape(nh, -1) - ref["score"]).max()
    assert serr < H.DELTA_B / 10, f"score error {serr}"
    if out_dtype is not None:
        assert out.dtype == out_dtype
    # a bfloat16 input, output or state storage sets the tolerance
    sb = state_dtype == dla.DLA_BF16
    tol = H.TOL["bf16"] if (w.dtype == "bf16" or out.dtype == torch.bfloat16 or sb) else H.TOL["f32"]
    rel = H.assert_outputs(out.float().cpu().numpy().reshape(nh, w.T, w.dv), ref["out"], tol,
                           w.label, mag=ref["mag"], mag_tol=H.state_mag_tol(sb, w.dk))
    exp = dla.cache_export(cache)
    srel = H.assert_cache(exp, ref["cache"], H.STATE_TOL[sb], what=w.label)
    assert (exp["tokens"] == w.T).all()
    _report("prefill-ok", case=w.label, state="bf16" if sb else "f32", max_score_err=f"{serr:.2e}",
            max_rel_out=f"{rel:.2e}", max_rel_state=f"{srel:.2e}")


def test_prefill_cfg1():
    _prefill_case(WORKLOADS["cfg1"])


def test_prefill_cfg1_iid_merges_every_token():
    _prefill_case(WORKLOADS["cfg1_iid"])


def test_prefill_cfg1_capacity_one_and_threshold_zero():
    _prefill_case(WORKLOADS["cfg1"], C=1)
    _prefill_case(WORKLOADS["cfg1"].replace(T=300), C=300, tau=0.0)


def test_prefill_bf16_geometric_segments_ragged():
    # cfg2 distributions at a size the oracle finishes in seconds: 1000 tokens
    # (7 chunks + a ragged tail of 104), capacity reached
    _prefill_case(WORKLOADS["cfg2"].replace(B=1, H=4, T=1000, C=12))


def test_prefill_bf16_spans_and_bursts():
    _prefill_case(WORKLOADS["cfg3"].replace(B=1, H=3, T=2600, C=24, span_mean=200.0))


def test_prefill_bf16_many_segments_slow_decay():
    _prefill_case(WORKLOADS["cfg4"].replace(B=1, H=2, T=3000, C=40, n_seg=200))


def test_prefill_mixed_head_dims():
    _prefill_case(WORKLOADS["cfg2"].replace(B=1, H=2, T=700, C=9, dk=64, dv=128))
    _prefill_case(WORKLOADS["cfg2"].replace(B=2, H=1, T=500, C=7, dk=128, dv=64))


def test_prefill_f32_head_dim_128():
    # float32 inputs at d = 128 (the scan reads its row-major copies)
    _prefill_case(WORKLOADS["cfg1"].replace(T=600, dk=128, dv=128))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_prefill_largest_capacity(dtype):
    # C = 1024 with every token a boundary: merges start after 1024 tokens
    w = WORKLOADS["cfg1" if dtype == "f32" else "cfg2"].replace(B=1, H=1, T=1100, dk=128, dv=128)
    _prefill_case(w, C=1024, tau=0.0)


def test_prefill_without_lambda():
    # no readout weights: every live state counts with weight 1
    _prefill_case(WORKLOADS["cfg2"].replace(B=1, H=2, T=900, C=10), no_lambda=True)
    _prefill_case(WORKLOADS["cfg1"].replace(T=500), no_lambda=True)


def test_prefill_threshold_never_reached():
    # only the first token opens a state; every later token joins it, so each
    # chunk's state list holds one state
    _prefill_case(WORKLOADS["cfg2"].replace(B=1, H=2, T=1100, C=8), tau=1e30)


def test_prefill_mixed_output_types():
    # bfloat16 inputs with float32 outputs, and float32 inputs with bfloat16 outputs
    torch = _torch()
    _prefill_case(WORKLOADS["cfg2"].replace(B=1, H=2, T=700, C=9), out_dtype=torch.float32)
    _prefill_case(WORKLOADS["cfg1"].replace(T=400), out_dtype=torch.bfloat16)


def test_prefill_continuation():
    _prefill_case(WORKLOADS["cfg2"].replace(B=1, H=2, T=900, C=10), T_split=[1, 300, 301, 640])
    _prefill_case(WORKLOADS["cfg1_iid"].replace(T=200), T_split=[57, 128])


def test_decode_steps_from_empty_match_oracle():
    """T decode steps from an empty cache equal the oracle's recurrence."""
    torch = _torch()
    dla = _dla()
    for w in (WORKLOADS["cfg1"].replace(T=256), WORKLOADS["cfg1_iid"].replace(T=96),
              WORKLOADS["cfg2"].replace(B=1, H=2, T=200, C=6)):
        x = make_inputs(w)
        ref = H.run_oracle(w, x)
        bo, mo, nb, nm = H.near_tie_overrides(ref, what=f"decode {w.label}")
        _report("decode", case=w.label, near_b=nb, near_m=nm)
        q, k, v, g, lam = H.inputs_to_device(w, x, w.B, w.H)
        cache = dla.cache_alloc(w.B, w.H, w.C, w.dk, w.dv)
        bo_d = torch.from_numpy(bo).reshape(w.B, w.H, w.T).cuda()
        mo_d = torch.from_numpy(mo).reshape(w.B, w.H, w.T).cuda()
        outs, bs, ms, ss = [], [], [], []
        for t in range(w.T):
            o, b, mi, sc = dla.decode_step(cache, q[:, :, t].contiguous(), k[:, :, t].contiguous(),
                                           v[:, :, t].contiguous(), g[:, :, t].contiguous(),
                                           lam[:, :, t].contiguous(),
                                           boundary_override=bo_d[:, :, t].contiguous(),
                                           merge_override=mo_d[:, :, t].contiguous())
            outs.append(o)
            bs.append(b)
            ms.append(mi)
            ss.append(sc)
        torch.cuda.synchronize()
        nh = w.B * w.H
        out = torch.stack(outs, 2).float().cpu().numpy().reshape(nh, w.T, w.dv)
        b = torch.stack(bs, 2).cpu().numpy().reshape(nh, w.T)
        mi = torch.stack(ms, 2).cpu().numpy().reshape(nh, w.T)
        H.assert_decisions(b, mi, ref, w.label)
        H.assert_outputs(out, ref["out"], H.TOL[w.dtype], w.label)
        H.assert_cache(dla.cache_export(cache), ref["cache"], 1e-4, what=w.label)


def test_decode_without_lambda():
    """Decode steps from an empty cache with no readout weights (every live
    state counts with weight 1) equal the oracle's recurrence."""
    torch = _torch()
    dla = _dla()
    w = WORKLOADS["cfg2"].replace(B=1, H=2, T=150, C=6)
    x = make_inputs(w)
    del x["lam"]
    ref = H.run_oracle(w, x)
    bo, mo, _, _ = H.near_tie_overrides(ref, what="decode, no lambda")
    q, k, v, g, lam = H.inputs_to_device(w, x, w.B, w.H)
    assert lam is None
    cache = dla.cache_alloc(w.B, w.H, w.C, w.dk, w.dv)
    bo_d = torch.from_numpy(bo).reshape(w.B, w.H, w.T).cuda()
    mo_d = torch.from_numpy(mo).reshape(w.B, w.H, w.T).cuda()
    outs, bs, ms = [], [], []
    for t in range(w.T):
        o, b, mi, _ = dla.decode_step(cache, q[:, :, t].contiguous(), k[:, :, t].contiguous(),
                                      v[:, :, t].contiguous(), g[:, :, t].contiguous(), None,
                                      boundary_override=bo_d[:, :, t].contiguous(),
                                      merge_override=mo_d[:, :, t].contiguous())
        outs.append(o)
        bs.append(b)
        ms.append(mi)
    torch.cuda.synchronize()
    nh = w.B * w.H
    H.assert_decisions(torch.stack(bs, 2).cpu().numpy().reshape(nh, w.T),
                       torch.stack(ms, 2).cpu().numpy().reshape(nh, w.T), ref, "decode, no lambda")
    H.assert_outputs(torch.stack(outs, 2).float().cpu().numpy().reshape(nh, w.T, w.dv), ref["out"],
                     H.TOL[w.dtype], "decode, no lambda")
    H.assert_cache(dla.cache_export(cache), ref["cache"], 1e-4, what="decode, no lambda")


def _decode_case(w, T1=0, label=None, state_dtype=0):
    """Prefill of the first T1 tokens (none for T1 = 0), then one decode step per
    remaining token; every decision, output and the final cache against the
    oracle over all tokens.  state_dtype: storage of the cache's states."""
    torch = _torch()
    dla = _dla()
    label = label or w.label
    sb = state_dtype == dla.DLA_BF16
    x = make_inputs(w)
    ref = H.run_oracle(w, x)
    bo, mo, _, _ = H.near_tie_overrides(ref, what=label)
    q, k, v, g, lam = H.inputs_to_device(w, x, w.B, w.H)
    shp = (w.B, w.H, w.T)
    bo_d = torch.from_numpy(bo).reshape(shp).cuda()
    mo_d = torch.from_numpy(mo).reshape(shp).cuda()
    cache = dla.cache_alloc(w.B, w.H, w.C, w.dk, w.dv, state_dtype=state_dtype)
    outs, bs, ms = [], [], []
    if T1 > 0:
        sl = slice(0, T1)
        o1, b1, m1, _ = dla.prefill(cache, q[:, :, sl].contiguous(), k[:, :, sl].contiguous(),
                                    v[:, :, sl].contiguous(), g[:, :, sl].contiguous(),
                                    lam[:, :, sl].contiguous(), tau=w.tau,
                                    boundary_override=bo_d[:, :, sl].contiguous(),
                                    merge_override=mo_d[:, :, sl].contiguous())
        outs.append(o1)
        bs.append(b1)
        ms.append(m1)
    for t in range(T1, w.T):
        o, b, mi, _ = dla.decode_step(cache, q[:, :, t].contiguous(), k[:, :, t].contiguous(),
                                      v[:, :, t].contiguous(), g[:, :, t].contiguous(),
                                      lam[:, :, t].contiguous(), tau=w.tau,
                                      boundary_override=bo_d[:, :, t].contiguous(),
                                      merge_override=mo_d[:, :, t].contiguous())
        outs.append(o.unsqueeze(2))
        bs.append(b.unsqueeze(2))
        ms.append(mi.unsqueeze(2))
    torch.cuda.synchronize()
    nh = w.B * w.H
    H.assert_decisions(torch.cat(bs, 2).cpu().numpy().reshape(nh, -1),
                       torch.cat(ms, 2).cpu().numpy().reshape(nh, -1), ref, label)
    rel = H.assert_outputs(torch.cat(outs, 2).float().cpu().numpy().reshape(nh, w.T, w.dv),
                           ref["out"], H.TOL["bf16" if sb else w.dtype], label, mag=ref["mag"],
                           mag_tol=H.state_mag_tol(sb, w.dk))
    srel = H.assert_cache(dla.cache_export(cache), ref["cache"], H.STATE_TOL[sb], what=label)
    _report("decode-ok", case=label, state="bf16" if sb else "f32", max_rel_out=f"{rel:.2e}",
            max_rel_state=f"{srel:.2e}")


def test_decode_edge_shapes():
    # mixed head dimensions
    _decode_case(WORKLOADS["cfg2"].replace(B=1, H=2, T=120, C=5, dk=64, dv=128), label="decode dk64 dv128")
    _decode_case(WORKLOADS["cfg2"].replace(B=2, H=1, T=90, C=4, dk=128, dv=64), label="decode dk128 dv64")
    # C = 1: a single state absorbs every token after the first
    _decode_case(WORKLOADS["cfg1"].replace(T=80, C=1), label="decode C=1")
    # the largest capacity, full, with a merge at every step
    _decode_case(WORKLOADS["cfg2"].replace(B=1, H=1, T=1040, C=1024, tau=0.0), T1=1030,
                 label="decode C=1024")


@pytest.mark.parametrize("case", ["bf16_ragged", "spans_bursts", "f32_inputs", "continuation",
                                  "capacity_one", "threshold_zero"])
def test_prefill_bf16_state_storage(case):
    """bfloat16 storage of the closed states (the newest state stays float32):
    decisions bit-exact, outputs and final cache states within the bfloat16
    tolerance."""
    bf = 1  # DLA_BF16
    if case == "bf16_ragged":
        _prefill_case(WORKLOADS["cfg2"].replace(B=1, H=4, T=1000, C=12), state_dtype=bf)
    elif case == "spans_bursts":
        _prefill_case(WORKLOADS["cfg3"].replace(B=1, H=3, T=2600, C=24, span_mean=200.0),
                      state_dtype=bf)
    elif case == "f32_inputs":
        _prefill_case(WORKLOADS["cfg1"].replace(T=600), state_dtype=bf)
    elif case == "continuation":
        _prefill_case(WORKLOADS["cfg2"].replace(B=1, H=2, T=2900, C=16), T_split=[1, 700, 701, 1600],
                      state_dtype=bf)
    elif case == "capacity_one":
        _prefill_case(WORKLOADS["cfg2"].replace(B=1, H=2, T=1100), C=1, state_dtype=bf)
    else:
        _prefill_case(WORKLOADS["cfg2"].replace(B=1, H=2, T=700), C=64, tau=0.0, state_dtype=bf)


def test_decode_bf16_state_storage():
    """Decode with bfloat16 storage: from an empty cache (several workgroups
    per head), after a prefill, at C = 1, with steep decay and a merge at every
    step, and at the largest capacity."""
    bf = 1  # DLA_BF16
    _decode_case(WORKLOADS["cfg2"].replace(B=1, H=2, T=200, C=6), label="decode bf16 empty",
                 state_dtype=bf)
    _decode_case(WORKLOADS["cfg2"].replace(B=1, H=2, T=1300, C=12), T1=1100,
                 label="decode bf16 after prefill", state_dtype=bf)
    _decode_case(WORKLOADS["cfg1"].replace(T=80, C=1), label="decode bf16 C=1", state_dtype=bf)
    _decode_case(WORKLOADS["cfg2"].replace(B=1, H=2, T=2600, C=16, g_lo=-0.2, tau=0.0), T1=2400,
                 label="decode bf16 far-apart frames", state_dtype=bf)
    _decode_case(WORKLOADS["cfg2"].replace(B=1, H=1, T=1040, C=1024, tau=0.0), T1=1030,
                 label="decode bf16 C=1024", state_dtype=bf)


def test_decode_merges_states_of_far_apart_frames():
    """Regression: a decode-step merge whose left state was rewritten more
    recently than its right neighbour.  The merged state was rebased to the
    right state's (older) frame with a factor exp(F_right - F_left) > 1, which
    overflows once the frames lie more than ~88 nats apart.  Steep decay
    (g ~ U(-0.2, 0)) over a 2400-token prefill spreads the frames by hundreds
    of nats; tau = 0 then merges at every decode step."""
    _decode_case(WORKLOADS["cfg2"].replace(B=1, H=2, T=2600, C=16, g_lo=-0.2, tau=0.0), T1=2400,
                 label="decode merges, far-apart frames")


@pytest.mark.parametrize("out_f32", [False, True])
def test_prefill_then_decode_continuation(out_f32):
    """prefill(T1) followed by decode steps equals the oracle over all tokens
    (bfloat16 inputs; outputs in bfloat16, or in float32)."""
    torch = _torch()
    dla = _dla()
    w = WORKLOADS["cfg2"].replace(B=1, H=2, T=420, C=8)
    x = make_inputs(w)
    ref = H.run_oracle(w, x)
    bo, mo, _, _ = H.near_tie_overrides(ref, what="prefill+decode")
    q, k, v, g, lam = H.inputs_to_device(w, x, w.B, w.H)
    bo_d = torch.from_numpy(bo).reshape(1, 2, w.T).cuda()
    mo_d = torch.from_numpy(mo).reshape(1, 2, w.T).cuda()
    T1 = 389
    od = torch.float32 if out_f32 else None
    cache = dla.cache_alloc(w.B, w.H, w.C, w.dk, w.dv)
    o1, b1, m1, _ = dla.prefill(cache, q[:, :, :T1].contiguous(), k[:, :, :T1].contiguous(),
                                v[:, :, :T1].contiguous(), g[:, :, :T1].contiguous(),
                                lam[:, :, :T1].contiguous(), boundary_override=bo_d[:, :, :T1].contiguous(),
                                merge_override=mo_d[:, :, :T1].contiguous(), out_dtype=od)
    outs, bs, ms = [o1], [b1], [m1]
    for t in range(T1, w.T):
        o, b, mi, _ = dla.decode_step(cache, q[:, :, t].contiguous(), k[:, :, t].contiguous(),
                                      v[:, :, t].contiguous(), g[:, :, t].contiguous(),
                                      lam[:, :, t].contiguous(),
                                      boundary_override=bo_d[:, :, t].contiguous(),
                                      merge_override=mo_d[:, :, t].contiguous(), out_dtype=od)
        assert o.dtype == (od or torch.bfloat16)
        outs.append(o.unsqueeze(2))
        bs.append(b.unsqueeze(2))
        ms.append(mi.unsqueeze(2))
    torch.cuda.synchronize()
    out = torch.cat(outs, 2).float().cpu().numpy().reshape(2, w.T, w.dv)
    H.assert_decisions(torch.cat(bs, 2).cpu().numpy().reshape(2, -1),
                       torch.cat(ms, 2).cpu().numpy().reshape(2, -1), ref, "prefill+decode")
    H.assert_outputs(out, ref["out"], H.TOL[w.dtype], "prefill+decode")
    H.assert_cache(dla.cache_export(cache), ref["cache"], 1e-4, what="prefill+decode")


def test_forced_overrides_match_oracle():
    """Random forced boundaries and merge indices take the same path on both sides."""
    torch = _torch()
    dla = _dla()
    w = WORKLOADS["cfg2"].replace(B=1, H=2, T=600, C=6)
    x = make_inputs(w)
    rng = np.random.default_rng(11)
    bo = np.where(rng.random((2, w.T)) < 0.08, 1, -1).astype(np.int8)
    bo[rng.random((2, w.T)) < 0.05] = 0
    mo = np.where(rng.random((2, w.T)) < 0.5, rng.integers(0, w.C - 1, (2, w.T)), -1).astype(np.int32)
    ref = H.run_oracle(w, x, b_override=bo, m_override=mo)
    bo2, mo2, _, _ = H.near_tie_overrides(ref, bo, mo, what="forced overrides")
    q, k, v, g, lam = H.inputs_to_device(w, x, w.B, w.H)
    cache = dla.cache_alloc(w.B, w.H, w.C, w.dk, w.dv)
    out, b, mi, sc = dla.prefill(cache, q, k, v, g, lam,
                                 boundary_override=torch.from_numpy(bo2).reshape(1, 2, -1).cuda(),
                                 merge_override=torch.from_numpy(mo2).reshape(1, 2, -1).cuda())
    torch.cuda.synchronize()
    H.assert_decisions(b.cpu().numpy().reshape(2, -1), mi.cpu().numpy().reshape(2, -1), ref, "forced")
    H.assert_outputs(out.float().cpu().numpy().reshape(2, w.T, w.dv), ref["out"], H.TOL["bf16"],
                     "forced")
    assert dla.cache_flags(cache) == 0


def test_bad_merge_override_sets_flag_and_is_ignored():
    torch = _torch()
    dla = _dla()
    w = WORKLOADS["cfg1_iid"].replace(T=40)
    x = make_inputs(w)
    ref = H.run_oracle(w, x)
    bo, mo, _, _ = H.near_tie_overrides(ref, what="bad merge override")
    mo[:, 20] = 99   # out of range: decided freely, flag raised
    q, k, v, g, lam = H.inputs_to_device(w, x, w.B, w.H)
    cache = dla.cache_alloc(w.B, w.H, w.C, w.dk, w.dv)
    out, b, mi, sc = dla.prefill(cache, q, k, v, g, lam,
                                 boundary_override=torch.from_numpy(bo).reshape(1, 2, -1).cuda(),
                                 merge_override=torch.from_numpy(mo).reshape(1, 2, -1).cuda())
    torch.cuda.synchronize()
    H.assert_decisions(b.cpu().numpy().reshape(2, -1), mi.cpu().numpy().reshape(2, -1), ref, "bad")
    assert dla.cache_flags(cache) == dla.DLA_FLAG_BAD_MERGE_OVERRIDE
    assert dla.cache_flags(cache) == 0   # cleared by the read


def test_skip_readout_builds_the_same_cache():
    torch = _torch()
    dla = _dla()
    w = WORKLOADS["cfg2"].replace(B=1, H=2, T=530, C=7)
    x = make_inputs(w)
    ref = H.run_oracle(w, x)
    bo, mo, _, _ = H.near_tie_overrides(ref, what="skip readout")
    q, k, v, g, lam = H.inputs_to_device(w, x, w.B, w.H)
    cache = dla.cache_alloc(w.B, w.H, w.C, w.dk, w.dv)
    _, b, mi, _ = dla.prefill(cache, None, k, v, g, None, skip_readout=True,
                              boundary_override=torch.from_numpy(bo).reshape(1, 2, -1).cuda(),
                              merge_override=torch.from_numpy(mo).reshape(1, 2, -1).cuda())
    torch.cuda.synchronize()
    H.assert_decisions(b.cpu().numpy().reshape(2, -1), mi.cpu().numpy().reshape(2, -1), ref, "skip")
    H.assert_cache(dla.cache_export(cache), ref["cache"], 1e-4, what="skip")


def _run_modes(w, x, T_split=None, budgets=(0, 0)):
    """Prefill the same inputs twice, pipelined and serial (optionally as two
    calls split at T_split), and return both runs' outputs, exports, caches
    and the pipelined run's readout-launch event count.  budgets: the state-copy
    budgets (log2 bytes, 0 = default) of the pipelined and the serial run."""
    torch = _torch()
    dla = _dla()
    q, k, v, g, lam = H.inputs_to_device(w, x, w.B, w.H)
    cuts = [0, w.T] if T_split is None else [0, T_split, w.T]
    res = {}
    for serial in (False, True):
        kb = budgets[1 if serial else 0]
        cache = dla.cache_alloc(w.B, w.H, w.C, w.dk, w.dv)
        outs = []
        for a, b in zip(cuts[:-1], cuts[1:]):
            sl = lambda t: t[:, :, a:b].contiguous()
            rev = None
            nseg = dla.prefill_segments(cache, b - a, k.dtype, serial=serial, pool_budget_log2=kb)
            if not serial:
                rev = [torch.cuda.Event(enable_timing=True) for _ in range(2 * nseg)]
            o, bd, mi, sc = dla.prefill(cache, sl(q), sl(k), sl(v), sl(g), sl(lam), tau=w.tau,
                                        serial=serial, readout_events=rev, pool_budget_log2=kb)
            torch.cuda.synchronize()
            outs.append((o.cpu(), bd.cpu(), mi.cpu(), sc.cpu()))
            if rev is not None:
                # every readout launch of the call is bracketed by a pair of events
                for i in range(nseg):
                    assert rev[2 * i].elapsed_time(rev[2 * i + 1]) > 0.0
        res[serial] = (outs, dla.cache_export(cache))
    return res


@pytest.mark.parametrize("case", ["bf16_ragged", "bf16_three_chunks", "f32", "continuation",
                                  "bf16_16k", "bf16_64k", "small_budgets"])
def test_pipelined_prefill_matches_serial(case):
    """The pipelined prefill (scan segments on a second stream, resuming from
    the scan carry) gives bit-identical outputs, exports and cache to the serial
    one: ragged last chunk, fewer chunks than segments, float32 inputs (256-token
    chunks), a continuation on a non-empty cache, the 16k-token shape (one
    shared pool), the 64k-token workload (segments that restart their pool,
    serial and pipelined), and small state-copy budgets that split both calls
    into many segments, differently."""
    budgets = (0, 0)
    if case == "bf16_ragged":
        w, cut = WORKLOADS["cfg3"].replace(B=1, H=3, T=2600, C=24, span_mean=200.0), None
    elif case == "bf16_three_chunks":
        w, cut = WORKLOADS["cfg2"].replace(B=1, H=2, T=1100, C=12), None
    elif case == "f32":
        w, cut = WORKLOADS["cfg1"].replace(T=1000), None
    elif case == "continuation":
        w, cut = WORKLOADS["cfg2"].replace(B=1, H=2, T=2900, C=16), 1100
    elif case == "bf16_16k":
        w, cut = WORKLOADS["cfg3"].replace(B=1, H=4), None
    elif case == "small_budgets":
        # 4 heads x 128 states x 32 KiB: 16 MiB of copies per chunk; budgets of
        # 64 MiB (pipelined) and 32 MiB (serial) give segments of 4 and 2 chunks
        w, cut = WORKLOADS["cfg3"].replace(B=1, H=4, T=9000), None
        budgets = (26, 25)
    else:
        # 64k tokens at C = 256: the state copies exceed the pool budget, so
        # both calls run segments that restart their pool (4 serial, 6
        # pipelined), each starting with copies of the states present
        w, cut = WORKLOADS["cfg4"], None
    _report("pipe-vs-serial", case=case, T=w.T, C=w.C, dtype=w.dtype)
    x = make_inputs(w)
    res = _run_modes(w, x, cut, budgets)
    (op, cp), (os_, cs) = res[False], res[True]
    for a, b in zip(op, os_):
        for ta, tb in zip(a, b):
            assert torch_equal_bits(ta, tb), case
    for key in cp:
        assert np.array_equal(cp[key], cs[key]), (case, key)
    # the inputs open states after the first token, so the scan carry matters
    assert int(os_[-1][1].sum()) > 1


def test_pipelined_prefill_on_user_streams_and_threads():
    """A pipelined prefill enqueued on a stream the caller created, and two
    pipelined prefills on separate caches from two host threads at once (each
    thread has its own second stream and events), match the same prefill on
    the default stream bit for bit."""
    import threading
    torch = _torch()
    dla = _dla()
    w = WORKLOADS["cfg2"].replace(B=1, H=2, T=2100, C=12)
    x = make_inputs(w)
    q, k, v, g, lam = H.inputs_to_device(w, x, w.B, w.H)
    assert dla.prefill_segments(dla.cache_alloc(w.B, w.H, w.C, w.dk, w.dv), w.T, k.dtype) > 1

    def run():
        cache = dla.cache_alloc(w.B, w.H, w.C, w.dk, w.dv)
        o, b, m, sc = dla.prefill(cache, q, k, v, g, lam, tau=w.tau)
        return cache, o, b, m, sc

    ref = run()
    torch.cuda.synchronize()
    ref_cache = dla.cache_export(ref[0])

    def check(res, what):
        for ta, tb in zip(res[1:], ref[1:]):
            assert torch_equal_bits(ta.cpu(), tb.cpu()), what
        ce = dla.cache_export(res[0])
        for key in ce:
            assert np.array_equal(ce[key], ref_cache[key]), (what, key)

    st = torch.cuda.Stream()
    st.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(st):
        res = run()
    st.synchronize()
    check(res, "user stream")

    out = [None, None]
    err = []

    def worker(i):
        try:
            s2 = torch.cuda.Stream()
            s2.wait_stream(torch.cuda.default_stream())
            with torch.cuda.stream(s2):
                out[i] = run()
            s2.synchronize()
        except Exception as e:  # reported below, on the main thread
            err.append(e)

    ths = [threading.Thread(target=worker, args=(i,)) for i in range(2)]
    for t in ths:
        t.start()
    for t in ths:
        t.join(timeout=120)
    assert not err, err
    for i in range(2):
        check(out[i], f"thread {i}")


def torch_equal_bits(a, b):
    torch = _torch()
    if a.dtype in (torch.bfloat16, torch.float16):
        return torch.equal(a.view(torch.int16), b.view(torch.int16))
    if a.dtype == torch.float32:
        return torch.equal(a.view(torch.int32), b.view(torch.int32))
    return torch.equal(a, b)


def _random_cases(n, seed):
    """Seeded mixes of the shape parameters the kernels branch on: head counts
    that are not a multiple of the 8-head workgroup groups, token counts at and
    around the 64-token scan blocks and the readout chunks (256 tokens for
    float32 inputs, 512 for bfloat16), capacities from 1 to past the 128-state
    DPP range, both head sizes and both input types, with and without lambda,
    float32 or bfloat16 state storage."""
    rng = np.random.default_rng(seed)
    structures = ["cuts", "geom", "spans_bursts", "iid"]
    cases = []
    for i in range(n):
        dtype = ["f32", "bf16"][i % 2]
        rl = 256 if dtype == "f32" else 512
        T = int(rng.choice([1, 63, 64, 65, rl - 1, rl, rl + 1, 2 * rl + 37, 3 * rl - 5]))
        dk, dv = [(64, 64), (128, 128), (64, 128), (128, 64)][int(rng.integers(4))]
        C = int(rng.choice([1, 2, 3, 7, 33, 130]))
        B, Hh = int(rng.choice([1, 2, 3])), int(rng.choice([1, 3, 5]))
        st = structures[int(rng.integers(len(structures)))]
        w = WORKLOADS["cfg1"].replace(
            name=f"random{i}", B=B, H=Hh, T=T, dk=dk, dv=dv, C=C, dtype=dtype,
            tau=round(float(rng.uniform(0.1, 0.9)), 2), seed=1000 + i, structure=st,
            n_seg=max(1, T // 50), mean_len=40.0, span_mean=200.0, burst_mean=8.0,
            g_lo=float(rng.choice([-0.05, -0.01])))
        cases.append((w, bool(rng.integers(2)), (i // 2) % 2))
    return cases


@pytest.mark.parametrize("w,no_lambda,state_dtype", _random_cases(24, 20261202),
                         ids=[f"random{i}" for i in range(24)])
def test_prefill_random_shapes(w, no_lambda, state_dtype):
    _prefill_case(w, no_lambda=no_lambda, state_dtype=state_dtype)


def _random_decode_cases(n, seed):
    """Seeded mixes for decode: head counts from 1 (the step split over up to
    16 workgroups per head) to 15, capacities 1 to 130, all head sizes, both
    input and state types, steps from an empty cache or after a prefill."""
    rng = np.random.default_rng(seed)
    structures = ["cuts", "geom", "spans_bursts", "iid"]
    cases = []
    for i in range(n):
        dtype = ["f32", "bf16"][i % 2]
        dk, dv = [(64, 64), (128, 128), (64, 128), (128, 64)][int(rng.integers(4))]
        C = int(rng.choice([1, 2, 3, 7, 33, 130]))
        B, Hh = int(rng.choice([1, 2, 3])), int(rng.choice([1, 3, 5]))
        st = structures[int(rng.integers(len(structures)))]
        if st == "iid":
            C = min(C, 7)  # (i.i.d. tokens merging at larger capacities tie densities
            # too often for the harness's bound on near-tie pins)
        T1 = int(rng.choice([0, 1, 70, 300]))
        T = T1 + int(rng.integers(1, 60))
        w = WORKLOADS["cfg1"].replace(
            name=f"decode_random{i}", B=B, H=Hh, T=T, dk=dk, dv=dv, C=C, dtype=dtype,
            tau=round(float(rng.uniform(0.1, 0.9)), 2), seed=3000 + i, structure=st,
            n_seg=max(1, T // 40), mean_len=30.0, span_mean=120.0, burst_mean=6.0,
            g_lo=float(rng.choice([-0.05, -0.01])))
        cases.append((w, T1, (i // 2) % 2))
    return cases


@pytest.mark.parametrize("w,T1,state_dtype", _random_decode_cases(12, 20261205),
                         ids=[f"decode_random{i}" for i in range(12)])
def test_decode_random_shapes(w, T1, state_dtype):
    _decode_case(w, T1=T1, state_dtype=state_dtype)
