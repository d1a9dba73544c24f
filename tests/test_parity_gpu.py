"""GPU parity: the HIP library against the float64 oracle, through the C ABI.

Tolerances (fp32 path vs float64 oracle):
  log Z      |gpu - oracle| <= 1e-5 * max(1, |oracle|)
  marginals  |gpu - oracle| <= 1e-4 on every valid cell
  CKY        spans identical (ties: lowest split), best == float32(oracle best)
The CKY chart is float64 on both sides with the same association order, so the
trees and scores must agree bit for bit.
"""
import numpy as np
import pytest

from oracle import oracle as orc
from paper_2008_03736_amd import binding as B
from paper_2008_03736_amd import workloads as W

pytestmark = pytest.mark.gpu

LOGZ_RTOL = 1e-5
MARG_ATOL = 1e-4
ORACLE_THREADS = 16


@pytest.fixture(scope="module")
def torch():
    import torch as _t

    if not _t.cuda.is_available():
        pytest.fail("GPU tests need a ROCm device")
    B.load()
    return _t


def gpu_run(torch, batch, flags=0, grad=None, decode=True, marg_fill=0.0):
    dev = torch.device("cuda", 0)
    s = torch.from_numpy(batch.scores).to(dev)
    with B.Plan(batch.lengths, n1=batch.n1, num_labels=batch.num_labels, flags=flags,
                device=dev) as plan:
        g = None if grad is None else torch.from_numpy(np.asarray(grad, np.float32)).to(dev)
        marg = torch.full_like(s, marg_fill)
        lz, marg = plan.inside_fwd_bwd(s, grad_logZ=g, marginals=marg)
        lz_only = plan.inside_fwd(s)
        out = {"logZ": lz, "marg": marg, "logZ_fwd": lz_only, "info": plan.info}
        if decode and batch.num_labels == 1:
            spans, best = plan.cky_decode(s)
            out["spans"], out["best"] = spans, best
            # the fused launch (inside, marginals and CKY together) that the
            # benchmark times, on its own outputs
            pm = torch.full_like(s, marg_fill)
            plz, pm, psp, pbe = plan.parse(s, grad_logZ=g, marginals=pm)
            out.update(p_logZ=plz, p_marg=pm, p_spans=psp, p_best=pbe)
        torch.cuda.synchronize()
    return {k: (v.cpu().numpy() if hasattr(v, "cpu") else v) for k, v in out.items()}


def check_logz(gpu, ref):
    err = np.abs(gpu.astype(np.float64) - ref)
    bound = LOGZ_RTOL * np.maximum(1.0, np.abs(ref))
    bad = np.nonzero(err > bound)[0]
    assert bad.size == 0, f"logZ mismatch at {bad[:5]}: gpu {gpu[bad[:5]]} ref {ref[bad[:5]]}"


def check_marg(gpu, ref, lengths, n1, labeled=False):
    v = W.valid_mask(np.asarray(lengths), n1)
    if labeled:
        v = np.broadcast_to(v[..., None], gpu.shape)
    err = np.abs(gpu[v].astype(np.float64) - ref[v])
    worst = float(err.max()) if err.size else 0.0
    assert worst <= MARG_ATOL, f"max |marginal error| {worst:.3e}"
    return worst


def check_cky(spans, best, batch, ref=None):
    spans_ref, best_ref = ref if ref is not None else orc.cky(batch.scores, batch.lengths, threads=ORACLE_THREADS)
    bad = np.nonzero((spans != spans_ref).any(axis=(1, 2)))[0]
    assert bad.size == 0, f"trees differ for sentences {bad[:10]}"
    assert np.array_equal(best, best_ref.astype(np.float32))
    return spans_ref, best_ref


def full_check(torch, batch, flags=0, grad=None, decode=True):
    """Every entry point against the oracle: inside_fwd, inside_fwd_bwd,
    cky_decode, and the fused parse launch (each on its own outputs)."""
    out = gpu_run(torch, batch, flags=flags, grad=grad, decode=decode)
    lz, mu = orc.marginals(batch.scores, batch.lengths, grad=grad, threads=ORACLE_THREADS)
    check_logz(out["logZ"], lz)
    check_logz(out["logZ_fwd"], lz)
    worst = check_marg(out["marg"], mu, batch.lengths, batch.n1)
    if decode:
        ref = check_cky(out["spans"], out["best"], batch)
        check_logz(out["p_logZ"], lz)
        worst = max(worst, check_marg(out["p_marg"], mu, batch.lengths, batch.n1))
        check_cky(out["p_spans"], out["p_best"], batch, ref)
    return out, worst


# --------------------------------------------------------------------------
# Workloads


def test_tiny(torch):
    full_check(torch, W.make("tiny"))


def test_mixed_full_batch(torch):
    # the 5,000-sentence batch in the launch configuration the benchmark times
    b = W.make("mixed")
    out, worst = full_check(torch, b)
    print(f"mixed: max |marginal error| {worst:.2e}, lds {out['info']['lds_count']}")


def test_longer_full_batch(torch):
    b = W.make("longer")
    full_check(torch, b)


def test_stress_full_batch(torch):
    # n = 256, sd 3, 5% of spans at -1e4: workspace-chart kernels
    b = W.make("stress")
    out, worst = full_check(torch, b)
    assert out["info"]["spill_count"] == b.B
    print(f"stress: max |marginal error| {worst:.2e}")


def check_labeled_chunks(out, b, chunk=125):
    """All sentences of a labelled batch against the oracle, a chunk of
    sentences at a time (each re-padded to its own longest sentence)."""
    worst = 0.0
    for c0 in range(0, b.B, chunk):
        idx = np.arange(c0, min(b.B, c0 + chunk))
        sub = W.subset(b, idx)
        lz, mu = orc.labeled(sub.scores, sub.lengths, threads=ORACLE_THREADS)
        check_logz(out["logZ"][idx], lz)
        check_logz(out["logZ_fwd"][idx], lz)
        n1 = sub.n1
        worst = max(worst, check_marg(out["marg"][idx][:, :n1, :n1], mu, sub.lengths, n1, labeled=True))
    return worst


def test_labeled_full_batch(torch):
    # all 1,000 sentences of the labelled batch (L = 26)
    b = W.make("labeled")
    out = gpu_run(torch, b, decode=False)
    worst = check_labeled_chunks(out, b)
    # label marginals sum to the span marginal, which is 1 on forced spans
    for bi in range(4):
        n = int(b.lengths[bi])
        assert abs(out["marg"][bi, 0, n].sum() - 1.0) < 1e-5
    print(f"labeled: max |marginal error| {worst:.2e}")


@pytest.mark.parametrize("labels", [33, 64, 138, 139])
def test_labeled_many_labels(torch, labels):
    # more than 32 labels per span: the label log-sum-exp and the per-label
    # marginals run in blocks of 32 (the second and later blocks, even and
    # odd counts); 138 is the size of the paper's CNF label set for English
    b = W.custom([1, 2, 5, 17, 40, 41, 64], seed=300 + labels, sd=1.0, labels=labels)
    out = gpu_run(torch, b, decode=False)
    worst = check_labeled_chunks(out, b, chunk=b.B)
    print(f"L = {labels}: max |marginal error| {worst:.2e}")


@pytest.mark.parametrize("spill", [False, True])
def test_labeled_in_bundle_boundary(torch, spill):
    # sentences on both sides of the longest length whose bundles read their
    # label scores and write their per-label marginals themselves (48 words),
    # and the same batch with every chart in the workspace, where the label
    # work always runs chip-wide; NaN-filled outputs show any cell left unwritten
    b = W.custom([1, 3, 47, 48, 49, 50, 48, 2], seed=77, sd=1.0, labels=5)
    flags = B.CRF_FORCE_SPILL if spill else 0
    out = gpu_run(torch, b, flags=flags, decode=False, marg_fill=float("nan"))
    assert out["info"]["spill_count"] == (b.B if spill else 0)
    worst = check_labeled_chunks(out, b, chunk=b.B)
    print(f"labelled around the in-bundle cutoff (spill={spill}): max |marginal error| {worst:.2e}")


# --------------------------------------------------------------------------
# Edge cases


def test_short_and_padded(torch):
    # n = 1 and n = 2 (only forced spans), a sentence at full padding, extra
    # padding beyond the longest sentence
    b = W.custom([1, 2, 3, 1, 7, 2, 12], seed=3, sd=1.5, n1=16)
    full_check(torch, b)
    b = W.custom([15, 1, 15], seed=4, sd=1.0, n1=16)
    full_check(torch, b)


@pytest.mark.parametrize("sd,mean", [(10.0, 0.0), (1.0, -60.0), (1.0, 60.0)])
def test_scores_beyond_the_linear_range(torch, sd, mean):
    # sd 10: a spread that a float32 chart of exp2 values cannot hold past a
    # few words -- the sweeps detect it and redo those bundles in the log
    # domain, on LDS charts (n <= 142) and workspace charts alike (every
    # sentence but the 3-word one, measured with a build that skips the redo).
    # Offsets of +-60 nats stay in the linear domain: the per-sentence shift,
    # seeded from the scores' mean, absorbs them.
    b = W.custom([3, 17, 40, 99, 130, 150], seed=78, sd=sd)
    v = W.valid_mask(b.lengths, b.n1)
    b.scores[v] += np.float32(mean)
    full_check(torch, b)


def test_all_zero_scores(torch):
    # every tree ties: right-branching tree, Catalan-ratio marginals
    b = W.custom([1, 2, 5, 40, 99], sd=0.0)
    full_check(torch, b)


def test_integer_scores_ties(torch):
    b = W.custom(list(range(2, 60)) * 2, seed=5, integer=(-2, 2))
    full_check(torch, b)


def test_force_spill_matches(torch):
    b = W.custom([1, 2, 9, 33, 70, 130], seed=6, sd=2.0)
    full_check(torch, b, flags=B.CRF_FORCE_SPILL)
    out_s = gpu_run(torch, b, flags=B.CRF_FORCE_SPILL)
    out_l = gpu_run(torch, b)
    assert out_s["info"]["spill_count"] == b.B
    assert np.array_equal(out_s["spans"], out_l["spans"])


def test_upstream_gradient(torch):
    b = W.custom([4, 17, 30], seed=8, sd=1.0)
    full_check(torch, b, grad=[2.0, -0.5, 0.0])


def test_padding_untouched_and_order(torch):
    # outputs outside the valid triangle keep the caller's values; sentence
    # order is preserved whatever the internal schedule
    rng = np.random.default_rng(10)
    lengths = rng.permutation(np.array([3, 50, 1, 20, 77, 8, 2, 64]))
    b = W.custom(lengths, seed=11, sd=2.0)
    out = gpu_run(torch, b, marg_fill=123.5)
    v = W.valid_mask(b.lengths, b.n1)
    assert np.all(out["marg"][~v] == np.float32(123.5))
    lz, mu = orc.marginals(b.scores, b.lengths)
    check_logz(out["logZ"], lz)
    check_marg(out["marg"], mu, b.lengths, b.n1)


def test_deterministic(torch):
    b = W.custom([5, 33, 90, 120], seed=12, sd=2.0)
    o1 = gpu_run(torch, b)
    o2 = gpu_run(torch, b)
    for k in ("logZ", "marg", "spans", "best"):
        assert np.array_equal(o1[k], o2[k], equal_nan=True), k


def test_labeled_small(torch):
    b = W.custom([1, 2, 6, 13], seed=13, sd=1.0, labels=7)
    out = gpu_run(torch, b, decode=False)
    lz, mu = orc.labeled(b.scores, b.lengths)
    check_logz(out["logZ"], lz)
    check_marg(out["marg"], mu, b.lengths, b.n1, labeled=True)


@pytest.mark.parametrize("offset", [0, 1])
@pytest.mark.parametrize("labels", [6, 7])
def test_labeled_alignment(torch, offset, labels):
    # labelled scores and marginals 8-byte aligned (offset 0) or only 4-byte
    # aligned (offset 1 float), with an even and an odd label count: the
    # 8-byte label accesses are taken only for even counts on aligned
    # tensors, and every case gives the same results, both in the bundles
    # that do their own label work and in the chip-wide label passes
    b = W.custom([5, 12, 30, 31, 49, 60], seed=41 + labels, sd=1.0, labels=labels)
    dev = torch.device("cuda", 0)
    size = b.scores.size
    s = torch.empty(size + 1, dtype=torch.float32, device=dev)[offset:offset + size].view(b.scores.shape)
    s.copy_(torch.from_numpy(b.scores))
    m = torch.full((size + 1,), float("nan"), dtype=torch.float32, device=dev)[offset:offset + size].view(b.scores.shape)
    with B.Plan(b.lengths, n1=b.n1, num_labels=b.num_labels, device=dev) as plan:
        lz, mu_gpu = plan.inside_fwd_bwd(s, marginals=m)
        torch.cuda.synchronize()
    lz_ref, mu_ref = orc.labeled(b.scores, b.lengths)
    check_logz(lz.cpu().numpy(), lz_ref)
    check_marg(mu_gpu.cpu().numpy(), mu_ref, b.lengths, b.n1, labeled=True)


@pytest.mark.parametrize("name", ["tiny", "mixed"])
def test_fused_call_matches_separate_calls(torch, name):
    # one launch for inside + reverse + CKY gives the separate calls' bits
    b = W.make(name)
    dev = torch.device("cuda", 0)
    s = torch.from_numpy(b.scores).to(dev)
    with B.Plan(b.lengths, device=dev) as plan:
        lz1, mu1 = plan.inside_fwd_bwd(s)
        sp1, be1 = plan.cky_decode(s)
        lz2, mu2, sp2, be2 = plan.parse(s)
        torch.cuda.synchronize()
    assert torch.equal(lz1, lz2) and torch.equal(mu1, mu2)
    assert torch.equal(sp1, sp2) and torch.equal(be1, be2)


def test_decode_rejects_labeled_plan(torch):
    b = W.custom([3], seed=1, labels=2)
    dev = torch.device("cuda", 0)
    s = torch.from_numpy(b.scores).to(dev)
    with B.Plan(b.lengths, num_labels=2, device=dev) as plan:
        with pytest.raises(B.CrfError) as ei:
            plan.cky_decode(s)
        assert ei.value.status == B.CRF_EUNSUPPORTED
        with pytest.raises(B.CrfError) as ei:
            plan.parse(s)
        assert ei.value.status == B.CRF_EUNSUPPORTED


def test_autograd_function(torch):
    b = W.custom([6, 11], seed=14, sd=1.0)
    dev = torch.device("cuda", 0)
    s = torch.from_numpy(b.scores).to(dev).requires_grad_(True)
    with B.Plan(b.lengths, device=dev) as plan:
        lz = B.log_partition(s, plan)
        (lz * torch.tensor([1.0, 3.0], device=dev)).sum().backward()
    _, mu = orc.marginals(b.scores, b.lengths, grad=[1.0, 3.0])
    check_marg(s.grad.cpu().numpy(), mu, b.lengths, b.n1)


def test_step_shape_boundaries(torch):
    # lengths on both sides of every change of step shape (split counts 1, 2,
    # 3, 5, 9, 17, 33, 49, 65, 97, 129), the last length whose CKY chart fits
    # in LDS (142) and the first that does not (143)
    lengths = [2, 3, 4, 5, 6, 9, 10, 17, 18, 33, 34, 49, 50, 65, 66, 97, 98, 129, 130, 142, 143]
    b = W.custom(lengths, seed=21, sd=2.0)
    out, worst = full_check(torch, b)
    assert out["info"]["spill_count"] >= 1
    print(f"shape boundaries: max |marginal error| {worst:.2e}")


def test_many_short_sentences(torch):
    # large bundles of short sentences: the depth-first tree walk
    b = W.custom([12] * 700 + [7] * 300 + [3] * 50, seed=22, sd=2.0)
    full_check(torch, b)


@pytest.mark.parametrize("n,count", [(9, 4), (12, 33), (14, 16), (14, 40), (17, 32), (20, 20), (22, 8),
                                     (30, 8), (45, 4), (56, 3), (98, 1)])
def test_bundle_counts_and_chart_strides(torch, n, count):
    # `count` sentences of n words, which the plan puts in one bundle when the
    # batch's total work is large (the 99-word sentences make it so), with
    # counts of various factors of two: the inside chart strides depend on
    # both (strict and loose layouts, spans interleaved across half-wavefronts
    # or side by side, rows changing inside a half).
    b = W.custom([n] * count + [99] * 200, seed=100 + n + count, sd=2.0)
    full_check(torch, b)


def test_longest_sentence(torch):
    # the longest sentence the library accepts, on the workspace kernels
    b = W.custom([1023], seed=23, sd=1.0)
    out, worst = full_check(torch, b)
    assert out["info"]["spill_count"] == 1
    print(f"n = 1023: max |marginal error| {worst:.2e}")


def test_workspace_teams(torch):
    # 16 sentences of 150..256 words: few enough that the workspace launches
    # split each sentence pass over a team of 8 (fused, 32 passes) or 16
    # workgroups of one XCD, several teams per XCD; every entry point against
    # the oracle
    lengths = [int(x) for x in np.random.default_rng(25).integers(150, 257, size=16)]
    b = W.custom(lengths, seed=25, sd=2.0)
    out, worst = full_check(torch, b)
    assert out["info"]["spill_count"] == b.B
    print(f"teams: max |marginal error| {worst:.2e}")


def test_workspace_teams_bit_identical(torch):
    # teams split each step's lanes over workgroups but keep every span's
    # arithmetic: every workspace entry point gives the same bits as with one
    # workgroup per sentence pass (CRF_NO_TEAMS), LDS bundles beside them
    b = W.custom([256, 201, 150, 143, 30, 7], seed=26, sd=2.0)
    gold, _ = orc.cky(b.scores, b.lengths)
    dev = torch.device("cuda", 0)
    s = torch.from_numpy(b.scores).to(dev)
    g = torch.from_numpy(np.ascontiguousarray(gold, np.int32)).to(dev)
    grad = torch.tensor([1.0, -0.5, 2.0, 0.25, 1.0, 3.0], dtype=torch.float32, device=dev)

    def run(flags):
        with B.Plan(b.lengths, n1=b.n1, flags=flags, device=dev) as plan:
            outs = [plan.inside_fwd(s), *plan.inside_fwd_bwd(s, grad_logZ=grad), *plan.cky_decode(s),
                    *plan.parse(s), *plan.mbr_decode(s), *plan.gold_loss(s, g, grad_loss=grad)]
            torch.cuda.synchronize()
            info = plan.info
        return [x.cpu().numpy() for x in outs], info

    teams, info_t = run(0)
    lone, info_l = run(B.CRF_NO_TEAMS)
    assert info_t["spill_count"] == 4 and info_l["spill_count"] == 4
    for i, (x, y) in enumerate(zip(teams, lone)):
        assert np.array_equal(x, y, equal_nan=True), f"output {i} differs between teams and lone workgroups"
    assert np.all(np.isfinite(teams[0]))


def test_split_tables_in_workspace(torch):
    # sentences whose CKY chart leaves no room in half a CU for the split
    # table keep it in global memory; a longer one moves every bundle to a
    # whole CU
    b = W.custom([97, 97, 98, 99, 99, 120, 3, 40], seed=24, sd=2.0)
    full_check(torch, b)


@pytest.mark.parametrize("name", ["tiny", "mixed"])
def test_fused_repeat_launches(torch, name):
    # the fused kernel's workgroups pull bundles from a counter that the last
    # claim resets: back-to-back launches on one plan give the same bits
    b = W.make(name)
    dev = torch.device("cuda", 0)
    s = torch.from_numpy(b.scores).to(dev)
    with B.Plan(b.lengths, device=dev) as plan:
        lz0, mu0 = plan.inside_fwd_bwd(s)
        sp0, be0 = plan.cky_decode(s)
        outs = [plan.parse(s) for _ in range(4)]
        torch.cuda.synchronize()
    for lz, mu, sp, be in outs:
        assert torch.equal(lz, lz0) and torch.equal(mu, mu0)
        assert torch.equal(sp, sp0) and torch.equal(be, be0)
