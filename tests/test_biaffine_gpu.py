"""GPU parity of the biaffine span scorer (Sec. 2.2, Eq. biaffine) through
the C ABI against the float64 oracle.

The inputs are bf16; the GPU forms u = [r^l;1]^T W in fp32 on the matrix
cores, keeps it as bf16 hi + lo parts (a relative residue of at most 2^-16),
and sums u . r^r in fp32.  So |gpu - oracle| <= 2^-12 * sum_c |u_c| |r^r_c|
(the oracle's bound), a 16x margin over that residue and fp32 rounding of
sums of at most 512 terms.
"""
import numpy as np
import pytest

from oracle import biaffine as obi
from paper_2008_03736_amd import binding as B
from paper_2008_03736_amd import workloads as W

pytestmark = pytest.mark.gpu

REL = 2.0 ** -12


@pytest.fixture(scope="module")
def torch():
    import torch as _t

    if not _t.cuda.is_available():
        pytest.fail("GPU tests need a ROCm device")
    B.load()
    return _t


def run(torch, inp, ldw=None):
    dev = torch.device("cuda", 0)
    d, L = inp.d, inp.num_labels
    ldw = ldw or ((d + 1 + 3) // 4 * 4)
    w = np.zeros((L, d, ldw), np.uint16)
    w[:, :, : d + 1] = inp.wt
    w[:, :, d + 1:] = 0x7FC0                      # NaN bit patterns past the bias: never read
    t = lambda a: torch.from_numpy(a.view(np.int16)).to(dev)
    with B.Plan(inp.lengths, n1=inp.n1, device=dev) as plan:
        s = plan.biaffine_scores(t(inp.rl), t(inp.rr), t(w))
        torch.cuda.synchronize()
    return s.cpu().numpy()


def check(got, inp):
    ref, bound = obi.biaffine(inp.rl, inp.rr, inp.wt, inp.lengths)
    v = W.valid_mask(inp.lengths, inp.n1)
    if got.ndim == 4:
        v4 = np.broadcast_to(v[..., None], got.shape)
    else:
        v4 = v
    err = np.abs(got[v4].astype(np.float64) - ref[v4])
    ratio = float((err / (REL * bound[v4] + 1e-30)).max())
    assert ratio <= 1.0, f"error {ratio:.2f} x the bound"
    assert np.isnan(got[~v4]).all(), "cells outside the valid triangle written"
    return float(err.max())


@pytest.mark.parametrize("d", [500, 100, 4, 64, 508, 124, 128, 252, 256])
def test_biaffine_span_scores(torch, d):
    # lengths across the packing (short sentences packed into one tile) and
    # the blocking (sentences of 64 or more fence posts), d = 500 (the
    # paper's), 100 (its label scorer), the limits, and the K paddings'
    # edges: d + 1 just under and over 128 and 256, which put the appended
    # 1 (and the end of W's rows) in the third or fourth quarter of K, the
    # quarter each wavefront of the first product takes
    lengths = [1, 2, 5, 30, 62, 63, 64, 99, 130, 20, 7]
    inp = W.biaffine_inputs(lengths, d, seed=d)
    worst = check(run(torch, inp), inp)
    print(f"d = {d}: max |error| {worst:.2e}")


def test_biaffine_label_scores(torch):
    # one W per label (d = 100, L = 26: the labelled workload's label count)
    inp = W.biaffine_inputs([3, 17, 40, 70], 100, labels=26, seed=9)
    check(run(torch, inp, ldw=104), inp)


def test_biaffine_mixed_batch_sample(torch):
    # the 5,000-sentence mixed batch's lengths at d = 500, checked on a sample
    # of sentences (the oracle's loops over all would take minutes)
    m = W.make("mixed")
    inp = W.biaffine_inputs(m.lengths, 500, seed=1)
    got = run(torch, inp)
    order = np.argsort(-m.lengths, kind="stable")
    idx = np.unique(np.concatenate([order[:6], order[-6:], np.arange(0, m.B, 211)]))
    sub = W.BiaffineInputs(inp.lengths[idx], inp.rl[idx], inp.rr[idx], inp.wt)
    check(got[idx], sub)


@pytest.mark.parametrize("d,ldw,labels", [(100, 112, 3), (64, 68, 2), (500, 520, 1), (12, 20, 5)])
def test_biaffine_row_strides(torch, d, ldw, labels):
    # weight rows wider than d + 1 (NaN padding never read), on both load
    # widths: 16-byte pieces when ldw is a multiple of 8, 8-byte ones else
    inp = W.biaffine_inputs([1, 9, 40, 66], d, labels=labels, seed=ldw)
    check(run(torch, inp, ldw=ldw), inp)
