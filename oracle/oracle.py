"""ctypes binding of the float64 C oracle (test infrastructure only).

Every function takes the same inputs as the GPU library -- a float32 score
block ``[B, N1, N1]`` (``[B, N1, N1, L]`` for labels) and int32 lengths -- and
returns float64 results computed by ``crf_oracle.c``.  Only cells
``0 <= i < j <= n_b`` of the scores are read; outputs outside that triangle are
NaN so a test cannot mistake them for results.
"""
import ctypes
import os

import numpy as np

from . import build as _build

_lib = None


def lib():
    """Load (building if needed) ``libcrforacle.so``."""
    global _lib
    if _lib is None:
        path = _build.LIB
        if not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(_build.SRC):
            _build.build()
        L = ctypes.CDLL(path)
        P = ctypes.c_void_p
        i = ctypes.c_int
        L.orc_logz.argtypes = [i, i, P, P, P, i]
        L.orc_marginals.argtypes = [i, i, P, P, P, P, P, i, i]
        L.orc_cky.argtypes = [i, i, P, P, P, P, i]
        L.orc_labeled.argtypes = [i, i, i, P, P, P, P, P, i]
        L.orc_loss.argtypes = [i, i, P, P, P, P, P, P, i]
        L.orc_labeled_cky.argtypes = [i, i, i, P, P, P, P, P, i]
        L.orc_label_spans.argtypes = [i, i, i, P, P, P, P, i]
        for f in (L.orc_logz, L.orc_marginals, L.orc_cky, L.orc_labeled, L.orc_loss, L.orc_labeled_cky,
                  L.orc_label_spans):
            f.restype = ctypes.c_int
        _lib = L
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _prep(scores, lengths, labeled=False):
    s = np.ascontiguousarray(scores, dtype=np.float32)
    n = np.ascontiguousarray(lengths, dtype=np.int32)
    if s.ndim != (4 if labeled else 3) or s.shape[1] != s.shape[2] or s.shape[0] != n.shape[0]:
        raise ValueError(f"bad shapes scores={s.shape} lengths={n.shape}")
    return s, n


def _check(rc):
    if rc != 0:
        raise RuntimeError(f"oracle returned status {rc}")


def logz(scores, lengths, threads=1):
    """log Z(x) per sentence (Eq. tree-prob via Algorithm 1), float64 [B]."""
    s, n = _prep(scores, lengths)
    out = np.empty(s.shape[0], np.float64)
    _check(lib().orc_logz(s.shape[0], s.shape[1], _ptr(n), _ptr(s), _ptr(out), threads))
    return out


def marginals(scores, lengths, grad=None, method="adjoint", threads=1, out=None):
    """(log Z [B], marginals [B,N1,N1]) in float64.

    ``method='adjoint'`` differentiates the inside recursion (Sec. 3.2);
    ``method='outside'`` runs the classical log-space outside pass.  The two
    are independent derivations of Eq. partial-derivative.  ``out`` may supply
    a float64 [B,N1,N1] buffer for the marginals (its invalid cells are left
    as they are).
    """
    s, n = _prep(scores, lengths)
    B, ld = s.shape[0], s.shape[1]
    g = None if grad is None else np.ascontiguousarray(grad, dtype=np.float64)
    lz = np.empty(B, np.float64)
    if out is None:
        mu = np.full((B, ld, ld), np.nan, np.float64)
    else:
        if out.shape != (B, ld, ld) or out.dtype != np.float64 or not out.flags.c_contiguous:
            raise ValueError("out must be a C-contiguous float64 [B, N1, N1] array")
        mu = out
    code = {"adjoint": 0, "outside": 1}[method]
    _check(lib().orc_marginals(B, ld, _ptr(n), _ptr(s), _ptr(g), _ptr(lz), _ptr(mu), code, threads))
    return lz, mu


def cky(scores, lengths, threads=1):
    """(spans int32 [B, 2(N1-1)-1, 2] in preorder, padded with -1; best [B])."""
    s, n = _prep(scores, lengths)
    B, ld = s.shape[0], s.shape[1]
    spans = np.empty((B, 2 * (ld - 1) - 1, 2), np.int32)
    best = np.empty(B, np.float64)
    _check(lib().orc_cky(B, ld, _ptr(n), _ptr(s), _ptr(spans), _ptr(best), threads))
    return spans, best


def labeled(scores, lengths, grad=None, want_marginals=True, threads=1):
    """One-stage labelled CRF (Eq. tree-label-score): (log Z [B], mu [B,N1,N1,L] or None)."""
    s, n = _prep(scores, lengths, labeled=True)
    B, ld, L = s.shape[0], s.shape[1], s.shape[3]
    g = None if grad is None else np.ascontiguousarray(grad, dtype=np.float64)
    lz = np.empty(B, np.float64)
    mu = np.full((B, ld, ld, L), np.nan, np.float64) if want_marginals else None
    _check(lib().orc_labeled(B, ld, L, _ptr(n), _ptr(s), _ptr(g), _ptr(lz), _ptr(mu), threads))
    return lz, mu


def _rows(spans, B, ld):
    sp = np.ascontiguousarray(spans, dtype=np.int32)
    if sp.shape != (B, 2 * (ld - 1) - 1, 2):
        raise ValueError(f"span lists must be int32 [{B}, {2 * (ld - 1) - 1}, 2], got {sp.shape}")
    return sp


def loss(scores, lengths, gold, grad=None, threads=1):
    """Gold-tree CRF loss (Sec. 2.3, Eq. bracket-loss) and its gradient.

    ``gold`` is an int32 [B, 2(N1-1)-1, 2] span list whose first 2n_b-1 rows
    are the gold tree of sentence b.  Returns (loss [B] = log Z - s(x,y),
    gradient [B, N1, N1] = grad[b] * (p((i,j)|x) - 1[(i,j) in y]) on valid
    cells, NaN elsewhere), float64.
    """
    s, n = _prep(scores, lengths)
    B, ld = s.shape[0], s.shape[1]
    gy = _rows(gold, B, ld)
    g = None if grad is None else np.ascontiguousarray(grad, dtype=np.float64)
    out = np.empty(B, np.float64)
    gr = np.full((B, ld, ld), np.nan, np.float64)
    _check(lib().orc_loss(B, ld, _ptr(n), _ptr(s), _ptr(gy), _ptr(g), _ptr(out), _ptr(gr), threads))
    return out, gr


def labeled_cky(scores, lengths, threads=1):
    """One-stage labelled decoding (Sec. 4.2, Eq. tree-label-score): (spans
    int32 [B, 2(N1-1)-1, 2] preorder padded with -1, labels int32
    [B, 2(N1-1)-1] padded with -1, best [B] float64)."""
    s, n = _prep(scores, lengths, labeled=True)
    B, ld, L = s.shape[0], s.shape[1], s.shape[3]
    spans = np.empty((B, 2 * (ld - 1) - 1, 2), np.int32)
    labels = np.empty((B, 2 * (ld - 1) - 1), np.int32)
    best = np.empty(B, np.float64)
    _check(lib().orc_labeled_cky(B, ld, L, _ptr(n), _ptr(s), _ptr(spans), _ptr(labels), _ptr(best), threads))
    return spans, labels, best


def label_spans(label_scores, lengths, spans, threads=1):
    """Labelling stage (Sec. 2.1, Eq. label-argmax) on given trees: int32
    [B, 2(N1-1)-1], the lowest argmax label of every row that is a span of its
    sentence, -1 for every other row."""
    s, n = _prep(label_scores, lengths, labeled=True)
    B, ld, L = s.shape[0], s.shape[1], s.shape[3]
    sp = _rows(spans, B, ld)
    labels = np.empty((B, 2 * (ld - 1) - 1), np.int32)
    _check(lib().orc_label_spans(B, ld, L, _ptr(n), _ptr(s), _ptr(sp), _ptr(labels), threads))
    return labels


def mbr(scores, lengths, threads=1, marginals_f32=None):
    """MBR decoding (Sec. 3.3): the CKY tree with the span marginals
    p((i,j)|x) in place of the span scores.  The marginals are those of
    ``marginals`` rounded to float32 (the precision in which a decoder
    receives them), or ``marginals_f32`` when given; the CKY chart over them
    is float64 (``cky``).  Returns (spans, best, marginals_f32)."""
    if marginals_f32 is None:
        _, mu = marginals(scores, lengths, threads=threads)
        mu32 = mu.astype(np.float32)
    else:
        mu32 = np.ascontiguousarray(marginals_f32, dtype=np.float32)
    spans, best = cky(mu32, lengths, threads=threads)
    return spans, best, mu32
