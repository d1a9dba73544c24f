"""Brute-force enumeration of binary bracketings (test infrastructure only).

For tiny sentences this computes every quantity straight from its definition
by listing all legal trees -- no dynamic programming at all:

  * a legal tree over n words is a binary bracketing: 2n-1 fence-post spans,
    all n width-1 spans and the root among them (Sec. 2.1; Fig. 1b shows a
    5-word CNF tree with 9 constituents);
  * s(x,y) = sum of the span scores of y                    (Eq. tree-score)
  * Z = sum over trees of exp(s(x,y)), p(y|x) = exp(s)/Z      (Eq. tree-prob)
  * p((i,j)|x) = sum of p(y|x) over trees containing (i,j)  (Eq. partial-derivative)
  * the best tree maximises s(x,y)                           (Eq. tree-argmax)
  * one-stage labelled score: sum of s(i,j,l) over labelled spans (Eq. tree-label-score)
  * gold-tree loss -log p(y|x) = log Z - s(x,y)              (Eq. bracket-loss)
  * MBR decoding: the tree maximising the sum of its spans' marginals (Sec. 3.3)
  * labelling: each span of a tree takes its best label      (Eq. label-argmax)

Ties between best trees are resolved by the lowest split point, which on
exactly representable scores is the optimal tree whose preorder sequence of
split points is lexicographically smallest.
"""
import itertools
import math


def trees(i, j):
    """Yield (spans_in_preorder, splits_in_preorder) for every bracketing of (i, j)."""
    if j - i == 1:
        yield [(i, j)], []
        return
    for k in range(i + 1, j):
        for ls, lk in trees(i, k):
            for rs, rk in trees(k, j):
                yield [(i, j)] + ls + rs, [k] + lk + rk


def _lse(vals):
    m = max(vals)
    return m + math.log(sum(math.exp(v - m) for v in vals))


def enumerate_all(s, n):
    """All trees of an n-word sentence with their scores; ``s[i][j]`` is s(i,j)."""
    out = []
    for spans, splits in trees(0, n):
        out.append((sum(float(s[i][j]) for i, j in spans), spans, splits))
    return out


def log_z(s, n):
    return _lse([t[0] for t in enumerate_all(s, n)])


def marginals(s, n):
    """{(i,j): p((i,j)|x)} for every span 0 <= i < j <= n."""
    all_t = enumerate_all(s, n)
    lz = _lse([t[0] for t in all_t])
    mu = {(i, j): 0.0 for i in range(n) for j in range(i + 1, n + 1)}
    for score, spans, _ in all_t:
        p = math.exp(score - lz)
        for sp in spans:
            mu[sp] += p
    return mu


def best_tree(s, n):
    """(best score, preorder spans) with the lowest-split tie rule."""
    all_t = enumerate_all(s, n)
    top = max(t[0] for t in all_t)
    cands = [t for t in all_t if t[0] == top]
    cands.sort(key=lambda t: t[2])
    return top, cands[0][1]


def labeled(s4, n, L):
    """One-stage labelled CRF by enumerating trees and label assignments.

    Returns (log Z, {(i,j,l): p((i,j,l)|x)}).
    """
    scored = []
    for spans, _ in trees(0, n):
        for labels in itertools.product(range(L), repeat=len(spans)):
            tot = sum(float(s4[i][j][l]) for (i, j), l in zip(spans, labels))
            scored.append((tot, spans, labels))
    lz = _lse([t[0] for t in scored])
    mu = {(i, j, l): 0.0 for i in range(n) for j in range(i + 1, n + 1) for l in range(L)}
    for tot, spans, labels in scored:
        p = math.exp(tot - lz)
        for (i, j), l in zip(spans, labels):
            mu[(i, j, l)] += p
    return lz, mu


def loss(s, n, gold):
    """-log p(y|x) for the gold tree y (a list of spans), by enumeration."""
    lz = log_z(s, n)
    return lz - sum(float(s[i][j]) for i, j in gold)


def best_labeled_tree(s4, n, L):
    """(best score, preorder spans, labels) over every tree and labelling.

    Among optimal labelled trees, the one whose preorder split sequence is
    lexicographically smallest, then whose preorder label sequence is.
    """
    cands = []
    for spans, splits in trees(0, n):
        for labels in itertools.product(range(L), repeat=len(spans)):
            tot = sum(float(s4[i][j][l]) for (i, j), l in zip(spans, labels))
            cands.append((tot, splits, labels, spans))
    top = max(c[0] for c in cands)
    opt = sorted((c for c in cands if c[0] == top), key=lambda c: (c[1], c[2]))
    return top, opt[0][3], list(opt[0][2])


def mbr_tree(s, n):
    """MBR decoding by enumeration: (best, preorder spans, gap to the runner-up)
    of the tree maximising the sum of its spans' marginals."""
    mu = marginals(s, n)
    scored = sorted(((sum(mu[sp] for sp in spans), spans) for spans, _ in trees(0, n)),
                    key=lambda t: -t[0])
    gap = scored[0][0] - scored[1][0] if len(scored) > 1 else float("inf")
    return scored[0][0], scored[0][1], gap
