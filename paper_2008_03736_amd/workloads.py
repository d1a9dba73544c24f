"""Seeded synthetic inputs shaped like treebank batches.

This module only draws random numbers; it holds none of the CRF arithmetic.
It serves both the GPU tests/benchmark and the float64 oracle checks.

The paper measures on PTB/CTB (Sec. 4.1, Table 1), licensed treebanks that are
not available here.  These batches stand in for them: per-sentence span
scores for a two-stage bracketing model (Sec. 2.1), or labelled span scores
for the one-stage variant (Sec. 4.2), with sentence lengths drawn from a
lognormal shaped like treebank length distributions.

Layout: ``scores[b, i, j]`` (``[b, i, j, l]`` when labelled) is s(i,j) for
fence posts 0 <= i < j <= lengths[b]; every other cell holds NaN so that a
kernel reading outside the valid triangle is caught.

Draw order for a named workload (fresh ``numpy.random.default_rng(seed)``):
lengths, then the score tensor, then (stress only) the near-forbidden mask.
"""
from dataclasses import dataclass
import math

import numpy as np

FORBIDDEN = -1.0e4


@dataclass
class Batch:
    name: str
    lengths: np.ndarray      # int32 [B]
    scores: np.ndarray       # float32 [B, N1, N1] or [B, N1, N1, L]
    sd: float

    @property
    def B(self):
        return int(self.lengths.shape[0])

    @property
    def n1(self):
        return int(self.scores.shape[1])

    @property
    def num_labels(self):
        return int(self.scores.shape[3]) if self.scores.ndim == 4 else 1


# name -> (B, length law, length params, score sd, labels, forbidden fraction)
WORKLOADS = {
    # 32 sentences, lengths uniform in [5, 40], s ~ N(0, 1)
    "tiny": dict(B=32, law="uniform", lo=5, hi=40, sd=1.0, labels=1, forbid=0.0),
    # 5,000 sentences, lognormal lengths mean 25 sd 12 clipped to [2, 140], s ~ N(0, 2)
    "mixed": dict(B=5000, law="lognormal", mean=25.0, std=12.0, lo=2, hi=140, sd=2.0,
                  labels=1, forbid=0.0),
    # 2,000 sentences, lognormal mean 28 sd 16 clipped to [2, 240], s ~ N(0, 2)
    "longer": dict(B=2000, law="lognormal", mean=28.0, std=16.0, lo=2, hi=240, sd=2.0,
                   labels=1, forbid=0.0),
    # 1,000 sentences, lengths as "mixed", labelled s(i,j,l) ~ N(0, 1), L = 26
    "labeled": dict(B=1000, law="lognormal", mean=25.0, std=12.0, lo=2, hi=140, sd=1.0,
                    labels=26, forbid=0.0),
    # 64 sentences of 256 words, s ~ N(0, 3), 5% of valid spans at -1e4
    "stress": dict(B=64, law="fixed", n=256, sd=3.0, labels=1, forbid=0.05),
}


def lognormal_lengths(rng, B, mean, std, lo, hi):
    """Lengths whose lognormal law has the given mean and sd, rounded and clipped."""
    var_ln = math.log1p((std / mean) ** 2)
    mu_ln = math.log(mean) - var_ln / 2.0
    x = rng.lognormal(mu_ln, math.sqrt(var_ln), size=B)
    return np.clip(np.rint(x), lo, hi).astype(np.int32)


def valid_mask(lengths, n1):
    """Boolean [B, N1, N1]: True where 0 <= i < j <= lengths[b]."""
    idx = np.arange(n1)
    upper = idx[:, None] < idx[None, :]
    inside = idx[None, None, :] <= lengths[:, None, None]
    return upper[None, :, :] & inside


def make(name, seed=0):
    """The named workload at ``seed``."""
    cfg = WORKLOADS[name]
    rng = np.random.default_rng(seed)
    if cfg["law"] == "uniform":
        lengths = rng.integers(cfg["lo"], cfg["hi"] + 1, size=cfg["B"]).astype(np.int32)
    elif cfg["law"] == "lognormal":
        lengths = lognormal_lengths(rng, cfg["B"], cfg["mean"], cfg["std"], cfg["lo"], cfg["hi"])
    else:
        lengths = np.full(cfg["B"], cfg["n"], np.int32)
    return scores_for(name, lengths, rng, cfg["sd"], cfg["labels"], cfg["forbid"])


def scores_for(name, lengths, rng, sd, labels=1, forbid=0.0, n1=None):
    """Draw N(0, sd^2) float32 scores for the given lengths; poison padding with NaN."""
    lengths = np.asarray(lengths, np.int32)
    B = lengths.shape[0]
    n1 = int(lengths.max()) + 1 if n1 is None else int(n1)
    shape = (B, n1, n1) if labels == 1 else (B, n1, n1, labels)
    scores = rng.standard_normal(shape, dtype=np.float32)
    scores *= np.float32(sd)
    valid = valid_mask(lengths, n1)
    if forbid > 0.0:
        hit = rng.random((B, n1, n1)) < forbid
        scores[hit & valid] = np.float32(FORBIDDEN)
    scores[~valid] = np.nan
    return Batch(name, lengths, scores, float(sd))


def custom(lengths, seed=0, sd=1.0, labels=1, forbid=0.0, n1=None, integer=None):
    """Ad-hoc batch for edge cases.

    ``integer=(lo, hi)`` draws integer scores in [lo, hi] (exact ties);
    ``sd=0`` gives all-zero scores.
    """
    rng = np.random.default_rng(seed)
    lengths = np.asarray(lengths, np.int32)
    if integer is None:
        return scores_for("custom", lengths, rng, sd, labels, forbid, n1)
    B = lengths.shape[0]
    n1 = int(lengths.max()) + 1 if n1 is None else int(n1)
    shape = (B, n1, n1) if labels == 1 else (B, n1, n1, labels)
    scores = rng.integers(integer[0], integer[1] + 1, size=shape).astype(np.float32)
    scores[~valid_mask(lengths, n1)] = np.nan
    return Batch("custom", lengths, scores, float(max(abs(integer[0]), abs(integer[1]))))


def subset(batch, idx):
    """Sentences ``idx`` of a batch, re-padded to their own maximum length."""
    idx = np.asarray(idx)
    lengths = batch.lengths[idx]
    n1 = int(lengths.max()) + 1
    scores = np.ascontiguousarray(batch.scores[idx][:, :n1, :n1])
    return Batch(batch.name, lengths, scores, batch.sd)


# --------------------------------------------------------------------------
# Boundary representations for the biaffine span scorer (Sec. 2.2,
# Eq. biaffine), stored as bfloat16 bit patterns (uint16).


def to_bf16(x):
    """float32 array -> bfloat16 bit patterns (uint16), rounded to nearest even."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    b = b + (np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1)))
    return (b >> np.uint32(16)).astype(np.uint16)


def from_bf16(h):
    """bfloat16 bit patterns (uint16) -> float32."""
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclass
class BiaffineInputs:
    lengths: np.ndarray      # int32 [B]
    rl: np.ndarray           # uint16 (bf16) [B, N1, d]: left boundary representations r^l_i
    rr: np.ndarray           # uint16 (bf16) [B, N1, d]: right boundary representations r^r_j
    wt: np.ndarray           # uint16 (bf16) [L, d, d+1]: wt[l, c, a] = W_l[a, c]; a = d is the bias row

    @property
    def B(self):
        return int(self.lengths.shape[0])

    @property
    def n1(self):
        return int(self.rl.shape[1])

    @property
    def d(self):
        return int(self.rl.shape[2])

    @property
    def num_labels(self):
        return int(self.wt.shape[0])


def biaffine_inputs(lengths, d, labels=1, seed=0, score_sd=2.0, n1=None):
    """Seeded representations and weights: r ~ N(0,1), W ~ N(0, (score_sd/d)^2),
    so that a span score sums d products of d products and has sd about
    score_sd (as the span scores of the CRF workloads).  Rows past each
    sentence hold NaN (never read).  Draw order: rl, rr, wt."""
    rng = np.random.default_rng(seed)
    lengths = np.asarray(lengths, np.int32)
    B = lengths.shape[0]
    n1 = int(lengths.max()) + 1 if n1 is None else int(n1)
    rl = rng.standard_normal((B, n1, d), dtype=np.float32)
    rr = rng.standard_normal((B, n1, d), dtype=np.float32)
    wt = rng.standard_normal((labels, d, d + 1), dtype=np.float32) * np.float32(score_sd / d)
    rows = np.arange(n1)[None, :] > lengths[:, None]
    rl[rows] = np.nan
    rr[rows] = np.nan
    return BiaffineInputs(lengths, to_bf16(rl), to_bf16(rr), to_bf16(wt))
