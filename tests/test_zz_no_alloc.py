"""The allocation-free Hessian entry point (realq_hessian_accum_noalloc) against the allocating
one (realq_hessian_accum), through the C ABI, on two calls in a row with the second input smaller,
and its size limit."""
import numpy as np
import pytest

import synth
from tests import parity as P

pytestmark = pytest.mark.gpu


def _both(rq, ctx, L, use_s):
    import torch
    Xh = torch.from_numpy(np.ascontiguousarray(L.Xhat, dtype=np.float32)).to(torch.bfloat16).cuda()
    s = torch.from_numpy(np.ascontiguousarray(L.s, dtype=np.float32)).cuda() if use_s else None
    n = Xh.shape[1]
    ref = torch.zeros((n, n), dtype=torch.float64, device="cuda")
    got = torch.full((n, n), 0.5, dtype=torch.float64, device="cuda")   # accumulates onto what is there
    rq.hessian_accum(ctx, Xh, s, ref)
    rq.hessian_accum_noalloc(ctx, Xh, s, got)
    torch.cuda.synchronize()
    return ref.cpu().numpy() + 0.5, got.cpu().numpy()


def test_noalloc_hessian_matches_the_allocating_entry_point(rq, ctx):
    print("\n[gpu-case] hessian noalloc: 5000 x 4096 with s, then 700 x 640 without", flush=True)
    # n = 4096 stages 2048 tokens per chunk, so 5000 tokens take three chunks, the last ragged
    a = synth.make_module("single_512", m=8, n=4096, T=5000, seed=3)
    ref, got = _both(rq, ctx, a, True)
    err = P.rel_fro(got, ref)
    print("rel Frobenius (s, 3 chunks)", err, flush=True)
    assert err <= 1e-6 and err <= P.HESS_RTOL
    b = synth.make_module("single_512", m=8, n=640, T=700, seed=4)
    ref, got = _both(rq, ctx, b, False)
    err = P.rel_fro(got, ref)
    print("rel Frobenius (no s, one chunk)", err, flush=True)
    assert err <= 1e-6
    assert np.array_equal(got, got.T)


def test_noalloc_hessian_rejects_too_many_columns(rq, ctx):
    """n above the scratch limit is refused on the host before anything is launched."""
    import torch
    n = 32769
    Xh = torch.zeros((8, n), dtype=torch.bfloat16, device="cuda")
    H = torch.zeros((1, 1), dtype=torch.float64, device="cuda")   # never touched: the call returns first
    with pytest.raises(rq.RealqError) as ei:
        ctx.check(rq.lib().realq_hessian_accum_noalloc(ctx.h, rq._ptr(Xh), None, 8, n, rq._ptr(H)))
    assert ei.value.code == -2
    assert "scratch limit" in str(ei.value)
