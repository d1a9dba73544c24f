"""The no-allocation entry point (crf_inside_fwd_bwd_cky_noalloc) through the
C ABI, against the entry point it is a variant of (crf_inside_fwd_bwd_cky,
which the parity tests hold to the oracle) and against the oracle itself.

Two calls in a row share the library's static scratch: the first on the
5,000-sentence mixed batch (its 99-word sentence keeps a CKY split table in
the workspace), the second on a smaller batch whose 200-word sentence keeps
both charts there; then the first plan again.  A plan that needs more
workspace than the scratch holds is rejected before any launch.
"""
import ctypes

import numpy as np
import pytest

from oracle import oracle as orc
from paper_2008_03736_amd import binding as B
from paper_2008_03736_amd import workloads as W

pytestmark = pytest.mark.gpu

SCRATCH_WS = (8 << 20) - 256


@pytest.fixture(scope="module")
def torch():
    import torch as _t

    if not _t.cuda.is_available():
        pytest.fail("GPU tests need a ROCm device")
    B.load()
    return _t


def _outputs(torch, plan, s, fill):
    t = torch
    R = 2 * (plan.n1 - 1) - 1
    return (t.full((plan.B,), fill, dtype=t.float32, device=s.device), t.full_like(s, fill),
            t.full((plan.B, R, 2), 7, dtype=t.int32, device=s.device),
            t.full((plan.B,), fill, dtype=t.float32, device=s.device))


def _call(torch, fn, plan, s, grad, outs):
    lz, mu, sp, be = outs
    stream = torch.cuda.current_stream(s.device).cuda_stream
    fn(plan._handle, s.data_ptr(), None if grad is None else grad.data_ptr(), lz.data_ptr(), mu.data_ptr(),
       sp.data_ptr(), be.data_ptr(), stream)


def _run_both(torch, batch, grad=None):
    dev = torch.device("cuda", 0)
    s = torch.from_numpy(batch.scores).to(dev)
    g = None if grad is None else torch.tensor(grad, dtype=torch.float32, device=dev)
    plan = B.Plan(batch.lengths, n1=batch.n1, device=dev)
    assert plan.info["workspace_bytes"] <= SCRATCH_WS
    ref = _outputs(torch, plan, s, -3.0)
    got = _outputs(torch, plan, s, -3.0)
    _call(torch, B.crf_inside_fwd_bwd_cky, plan, s, g, ref)
    _call(torch, B.crf_inside_fwd_bwd_cky_noalloc, plan, s, g, got)
    torch.cuda.synchronize()
    return plan, s, g, [x.cpu().numpy() for x in ref], [x.cpu().numpy() for x in got]


def _same(ref, got):
    for name, a, b in zip(("logZ", "marginals", "spans", "best"), ref, got):
        assert np.array_equal(a, b), f"{name} differs from crf_inside_fwd_bwd_cky"


def _against_oracle(batch, got, grad=None):
    lz, mu, sp, be = got
    lz_ref, mu_ref = orc.marginals(batch.scores, batch.lengths, grad=grad, threads=16)
    assert np.all(np.abs(lz - lz_ref) <= 1e-5 * np.maximum(1.0, np.abs(lz_ref)))
    v = W.valid_mask(batch.lengths, batch.n1)
    assert np.max(np.abs(mu[v] - mu_ref[v])) <= 1e-4
    assert np.all(mu[~v] == np.float32(-3.0))          # padding untouched
    sp_ref, be_ref = orc.cky(batch.scores, batch.lengths, threads=16)
    assert np.array_equal(sp, sp_ref)
    assert np.array_equal(be, be_ref.astype(np.float32))


def test_noalloc_matches_fused_call_twice_in_a_row(torch):
    big = W.make("mixed")
    plan1, s1, _, ref1, got1 = _run_both(torch, big)
    assert plan1.info["split_ws_count"] >= 1            # the scratch is really used
    _same(ref1, got1)
    _against_oracle(big, got1)

    small = W.custom([200, 97, 5, 30, 1, 64], seed=77, sd=2.0)
    grad = [1.0, 0.5, 2.0, -1.0, 1.0, 3.0]
    plan2, _, _, ref2, got2 = _run_both(torch, small, grad=grad)
    assert plan2.info["spill_count"] == 1 and plan2.info["cky_spill_count"] == 1
    _same(ref2, got2)
    _against_oracle(small, got2, grad=grad)

    # the first plan again, after the scratch held the second call's charts
    again = _outputs(torch, plan1, s1, -3.0)
    _call(torch, B.crf_inside_fwd_bwd_cky_noalloc, plan1, s1, None, again)
    torch.cuda.synchronize()
    _same(ref1, [x.cpu().numpy() for x in again])
    plan1.close()
    plan2.close()


def test_noalloc_rejects_plan_beyond_scratch(torch):
    b = W.make("stress")                                # 64 sentences of 256 words: ~68 MB of workspace
    dev = torch.device("cuda", 0)
    s = torch.from_numpy(b.scores).to(dev)
    with B.Plan(b.lengths, n1=b.n1, device=dev) as plan:
        assert plan.info["workspace_bytes"] > SCRATCH_WS
        outs = _outputs(torch, plan, s, -3.0)
        with pytest.raises(B.CrfError) as ei:
            _call(torch, B.crf_inside_fwd_bwd_cky_noalloc, plan, s, None, outs)
        assert ei.value.status == B.CRF_EINVAL
        assert "static scratch" in str(ei.value)
        torch.cuda.synchronize()
        assert torch.all(outs[0] == -3.0)                # nothing was launched


def test_noalloc_rejects_bad_arguments(torch):
    dummy = ctypes.c_void_p(0x1000)
    lib = B.load()
    assert lib.crf_inside_fwd_bwd_cky_noalloc(None, dummy, None, dummy, dummy, dummy, None, None) == B.CRF_EINVAL
