"""GPU parity of the fixed state-merging policies (every-K blocking, log-linear
buckets, single state) driven through the override path: the same kernels as
DLA, with every decision fixed by the schedule, against the float64 oracle
given the same schedule.  Layer shape of a Mamba-2 head (d_k = 128 state
size, d_v = 64 head dimension)."""
import numpy as np
import pytest

from tests import harness as H
from paper_2606_10650_amd import policies as P
from paper_2606_10650_amd.workloads import WORKLOADS, make_inputs

pytestmark = pytest.mark.gpu

MAMBA = WORKLOADS["cfg2"].replace(B=1, H=2, dk=128, dv=64, tau=0.6)


def _torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _schedule(policy, T, C_dla, K):
    C, b, m = P.schedule(policy, T, C_dla=C_dla, K=K)
    return C, b, m


def _check(dla, torch, w, x, ref, cache, out, b, mi, sb, what):
    nh = w.B * w.H
    H.assert_decisions(b.cpu().numpy().reshape(nh, -1), mi.cpu().numpy().reshape(nh, -1), ref, what)
    rel = H.assert_outputs(out.float().cpu().numpy().reshape(nh, w.T, w.dv), ref["out"],
                           H.TOL["bf16"], what, mag=ref["mag"], mag_tol=H.state_mag_tol(sb, w.dk))
    srel = H.assert_cache(dla.cache_export(cache), ref["cache"], H.STATE_TOL[sb], what=what)
    assert dla.cache_flags(cache) == 0
    print(f"[policy-ok] {what} states={int(ref['m'][0, -1])} max_rel_out={rel:.2e} "
          f"max_rel_state={srel:.2e}", flush=True)


@pytest.mark.parametrize("policy", ["single_state", "every_k", "log_linear"])
@pytest.mark.parametrize("state", ["f32", "bf16"])
def test_policy_prefill_matches_oracle(policy, state):
    torch = _torch()
    from paper_2606_10650_amd import dla
    T = 1100
    C, b, m = _schedule(policy, T, C_dla=8, K=64)
    w = MAMBA.replace(T=T, C=C)
    x = make_inputs(w)
    nh = w.B * w.H
    bo = np.broadcast_to(b, (nh, T)).copy()
    mo = np.broadcast_to(m, (nh, T)).copy()
    ref = H.run_oracle(w, x, b_override=bo, m_override=mo)
    sd = dla.DLA_BF16 if state == "bf16" else dla.DLA_F32
    q, k, v, g, lam = H.inputs_to_device(w, x, w.B, w.H)
    cache = dla.cache_alloc(w.B, w.H, C, w.dk, w.dv, state_dtype=sd)
    out, bb, mi, _ = dla.prefill(cache, q, k, v, g, lam, tau=w.tau,
                                 boundary_override=torch.from_numpy(bo).reshape(1, 2, T).cuda(),
                                 merge_override=torch.from_numpy(mo).reshape(1, 2, T).cuda())
    torch.cuda.synchronize()
    _check(dla, torch, w, x, ref, cache, out, bb, mi, sd == dla.DLA_BF16,
           f"{policy} prefill C{C} {state} states")


@pytest.mark.parametrize("policy", ["every_k", "log_linear"])
def test_policy_prefill_then_decode(policy):
    """A schedule for T0 + steps tokens: the prefill takes its first T0
    decisions, every decode step the next one."""
    torch = _torch()
    from paper_2606_10650_amd import dla
    T0, steps = 700, 90
    T = T0 + steps
    C, b, m = _schedule(policy, T, C_dla=6, K=32)
    w = MAMBA.replace(T=T, C=C)
    x = make_inputs(w)
    nh = w.B * w.H
    bo = torch.from_numpy(np.broadcast_to(b, (nh, T)).copy()).reshape(1, 2, T).cuda()
    mo = torch.from_numpy(np.broadcast_to(m, (nh, T)).copy()).reshape(1, 2, T).cuda()
    ref = H.run_oracle(w, x, b_override=bo.cpu().numpy().reshape(nh, T),
                       m_override=mo.cpu().numpy().reshape(nh, T))
    q, k, v, g, lam = H.inputs_to_device(w, x, w.B, w.H)
    cache = dla.cache_alloc(w.B, w.H, C, w.dk, w.dv)
    sl = slice(0, T0)
    o1, b1, m1, _ = dla.prefill(cache, q[:, :, sl].contiguous(), k[:, :, sl].contiguous(),
                                v[:, :, sl].contiguous(), g[:, :, sl].contiguous(),
                                lam[:, :, sl].contiguous(), tau=w.tau,
                                boundary_override=bo[:, :, sl].contiguous(),
                                merge_override=mo[:, :, sl].contiguous())
    outs, bs, ms = [o1], [b1], [m1]
    for t in range(T0, T):
        o, bt, mt, _ = dla.decode_step(cache, q[:, :, t].contiguous(), k[:, :, t].contiguous(),
                                       v[:, :, t].contiguous(), g[:, :, t].contiguous(),
                                       lam[:, :, t].contiguous(), tau=w.tau,
                                       boundary_override=bo[:, :, t].contiguous(),
                                       merge_override=mo[:, :, t].contiguous())
        outs.append(o.unsqueeze(2))
        bs.append(bt.unsqueeze(2))
        ms.append(mt.unsqueeze(2))
    torch.cuda.synchronize()
    _check(dla, torch, w, x, ref, cache, torch.cat(outs, 2), torch.cat(bs, 2), torch.cat(ms, 2),
           False, f"{policy} prefill {T0} + {steps} decode steps C{C}")
