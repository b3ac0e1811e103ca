"""dla_prefill_static, the prefill entry point that allocates nothing (its
workspace is the library's static device scratch), against dla_prefill with
a workspace argument and serial stages: bit-identical outputs, exports and
cache, on two calls in a row, the second with a smaller input; a call whose
workspace exceeds the scratch is refused before any device work."""
import numpy as np
import pytest

from tests import harness as H
from paper_2606_10650_amd.workloads import WORKLOADS, make_inputs

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _bits(t):
    torch = _torch()
    if t.dtype in (torch.bfloat16, torch.float16):
        return t.view(torch.int16)
    if t.dtype == torch.float32:
        return t.view(torch.int32)
    return t


def test_static_scratch_prefill_matches_workspace_prefill():
    torch = _torch()
    from paper_2606_10650_amd import dla
    for w in (WORKLOADS["cfg2"].replace(B=1, H=4, T=1500, C=16),
              WORKLOADS["cfg2"].replace(B=1, H=2, T=700, C=16)):
        x = make_inputs(w)
        q, k, v, g, lam = H.inputs_to_device(w, x, w.B, w.H)
        shp = (w.B, w.H, w.T)
        res = []
        for static in (True, False):
            cache = dla.cache_alloc(w.B, w.H, w.C, w.dk, w.dv)
            out = torch.empty((w.B, w.H, w.T, w.dv), dtype=torch.bfloat16, device="cuda")
            bnd = torch.empty(shp, dtype=torch.int8, device="cuda")
            mrg = torch.empty(shp, dtype=torch.int32, device="cuda")
            scr = torch.empty(shp, dtype=torch.float32, device="cuda")
            if static:
                dla.prefill_static(cache, q, k, v, g, lam, tau=w.tau, out=out, boundary=bnd,
                                   merge_idx=mrg, score=scr)
            else:
                dla.prefill(cache, q, k, v, g, lam, tau=w.tau, out=out, boundary=bnd,
                            merge_idx=mrg, score=scr, serial=True)
            torch.cuda.synchronize()
            res.append((out, bnd, mrg, scr, dla.cache_export(cache)))
        (a, b) = res
        for ta, tb in zip(a[:4], b[:4]):
            assert torch.equal(_bits(ta), _bits(tb)), w.label
        for key in a[4]:
            assert np.array_equal(a[4][key], b[4][key]), (w.label, key)
        assert int(b[1].sum()) > w.H   # states opened after the first tokens
    # too large for the scratch: refused with DLA_ERR_WORKSPACE, nothing enqueued
    big = WORKLOADS["cfg3"].replace(B=1, H=16, T=16384)
    cache = dla.cache_alloc(big.B, big.H, big.C, big.dk, big.dv)
    need = dla.workspace_bytes(cache, big.T, torch.bfloat16, serial=True)
    assert need > dla.STATIC_SCRATCH_BYTES
    kk = torch.zeros((1, 16, big.T, 128), dtype=torch.bfloat16, device="cuda")
    gg = torch.zeros((1, 16, big.T), dtype=torch.float32, device="cuda")
    before = cache.buf.clone()
    with pytest.raises(dla.DLAError) as e:
        dla.prefill_static(cache, kk, kk, kk, gg, None, out=torch.empty_like(kk))
    assert e.value.status == dla.DLA_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert torch.equal(cache.buf, before)
