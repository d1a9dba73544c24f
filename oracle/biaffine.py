"""Float64 oracle of the biaffine span scorer (test infrastructure only).

Sec. 2.2, Eq. biaffine: a candidate span (i,j) of a sentence is scored from
the left boundary representation of fence post i and the right one of fence
post j,

    s(i,j) = [r^l_i ; 1]^T W r^r_j,

with W of (d+1) x d entries: the appended 1 makes W's last row a bias on the
right representation (the equation's bracket appends 1 to the left vector
only).  Label scores use one such W per label (the label-scoring paragraph
of Sec. 2.2): s(i,j,l) = [r^l_i ; 1]^T W_l r^r_j.

Inputs are bfloat16 bit patterns (uint16), widened to float64 here; the
products and sums are float64 matrix products of the widened values.  Only
cells 0 <= i < j <= n_b are produced; the rest are NaN.
"""
import numpy as np


def _f64(h):
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def biaffine(rl, rr, wt, lengths):
    """(scores, bound): scores [B,N1,N1] (one W) or [B,N1,N1,L], and the
    float64 bound sum_c |u_ic| |r^r_jc| (u = [r^l_i;1]^T W, per label) that a
    rounding analysis scales into a tolerance."""
    rl, rr, wt = _f64(rl), _f64(rr), _f64(wt)
    lengths = np.asarray(lengths)
    B, N1, d = rl.shape
    L = wt.shape[0]
    out = np.full((B, N1, N1, L), np.nan)
    bound = np.full((B, N1, N1, L), np.nan)
    for b in range(B):
        n = int(lengths[b])
        a = np.concatenate([rl[b, :n + 1], np.ones((n + 1, 1))], axis=1)    # [r^l_i ; 1]
        r = rr[b, :n + 1]
        for l in range(L):
            W = wt[l].T                                                     # (d+1) x d
            u = a @ W
            s = u @ r.T
            m = np.abs(u) @ np.abs(r).T
            iu = np.triu_indices(n + 1, 1)
            out[b][iu + (l,)] = s[iu]
            bound[b][iu + (l,)] = m[iu]
    if L == 1:
        return out[..., 0], bound[..., 0]
    return out, bound
