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


def _case(w, mode, state_dtype=0, no_lambda=False):
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
                                           boundary_override=bo_d, merge_override=mo_d)
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
    """1024 heads: the step runs one workgroup per head (no split)."""
    from paper_2606_10650_amd import dla
    w = WORKLOADS["cfg1"].replace(B=64, H=16, T=40, C=4)
    assert dla.lib() and w.B * w.H >= 1024
    _case(w, "prefill")
