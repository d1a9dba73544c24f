"""ctypes binding of ``libcrfinside.so`` (C ABI in ``include/crf_inside.h``).

Argument marshalling only: every step of the computation runs in the HIP
library.  PyTorch supplies device memory and the current HIP stream.

The raw entry points keep the C names (``crf_plan_create``, ``crf_inside_fwd``,
``crf_inside_bwd``, ``crf_inside_fwd_bwd``, ``crf_cky_decode``, ...) and take
integer device pointers.  :class:`Plan` wraps them for torch tensors.

There is no fallback: if the library is missing, :func:`load` raises.
"""
import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libcrfinside.so")

CRF_OK, CRF_EINVAL, CRF_ENOMEM, CRF_EHIP, CRF_EUNSUPPORTED = 0, 1, 2, 3, 4
CRF_MAX_LEN = 1023
CRF_MAX_LABELS = 4096
CRF_FORCE_SPILL = 0x1
CRF_NO_TEAMS = 0x2

# Every function the C header declares, with its ctypes signature.
_P = ctypes.c_void_p
_I32 = ctypes.c_int32
SIGNATURES = {
    "crf_plan_create": (ctypes.c_int, [ctypes.POINTER(_P), _P, _I32, _I32, _I32, ctypes.c_uint32]),
    "crf_plan_destroy": (ctypes.c_int, [_P]),
    "crf_plan_info": (ctypes.c_int, [_P, _P]),
    "crf_inside_fwd": (ctypes.c_int, [_P, _P, _P, _P]),
    "crf_inside_bwd": (ctypes.c_int, [_P, _P, _P, _P, _P]),
    "crf_inside_fwd_bwd": (ctypes.c_int, [_P, _P, _P, _P, _P, _P]),
    "crf_cky_decode": (ctypes.c_int, [_P, _P, _P, _P, _P]),
    "crf_inside_fwd_bwd_cky": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P, _P]),
    "crf_inside_fwd_bwd_cky_noalloc": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P, _P]),
    "crf_mbr_decode": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P]),
    "crf_gold_loss": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P]),
    "crf_cky_decode_labeled": (ctypes.c_int, [_P, _P, _P, _P, _P, _P]),
    "crf_label_spans": (ctypes.c_int, [_P, _P, _I32, _P, _P, _P]),
    "crf_biaffine_scores": (ctypes.c_int, [_P, _P, _P, _P, _I32, _I32, _I32, _P, _P]),
    "crf_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "crf_last_error": (ctypes.c_char_p, []),
}


class PlanStats(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32),
        ("n1", ctypes.c_int32),
        ("num_labels", ctypes.c_int32),
        ("max_len", ctypes.c_int32),
        ("lds_count", ctypes.c_int32),
        ("spill_count", ctypes.c_int32),
        ("workspace_bytes", ctypes.c_int64),
        ("lds_bytes_inside", ctypes.c_int32),
        ("lds_bytes_cky", ctypes.c_int32),
        ("cky_spill_count", ctypes.c_int32),
        ("split_ws_count", ctypes.c_int32),
        ("workspace_users", ctypes.c_int32),
        ("fused_queue", ctypes.c_int32),
        ("mbr_fused", ctypes.c_int32),
    ]


class CrfError(RuntimeError):
    def __init__(self, status, where):
        lib = load()
        msg = lib.crf_last_error().decode() or lib.crf_status_string(status).decode()
        super().__init__(f"{where}: status {status} ({lib.crf_status_string(status).decode()}): {msg}")
        self.status = status


_lib = None


def load(path=LIB_PATH):
    """Load the HIP library (once).  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(path):
            raise RuntimeError(
                f"{path} is missing: build it with __graft_entry__.build() "
                "(or python paper_2008_03736_amd/build.py); there is no fallback")
        lib = ctypes.CDLL(path)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def _check(status, where):
    if status != CRF_OK:
        raise CrfError(status, where)


# --------------------------------------------------------------------------
# Raw entry points (C names, integer pointers).

def crf_plan_create(lengths_ptr, batch, n1, num_labels=1, flags=0):
    plan = _P()
    _check(load().crf_plan_create(ctypes.byref(plan), lengths_ptr, batch, n1, num_labels, flags),
           "crf_plan_create")
    return plan


def crf_plan_destroy(plan):
    _check(load().crf_plan_destroy(plan), "crf_plan_destroy")


def crf_plan_info(plan):
    st = PlanStats()
    _check(load().crf_plan_info(plan, ctypes.byref(st)), "crf_plan_info")
    return {k: getattr(st, k) for k, _ in PlanStats._fields_}


def crf_inside_fwd(plan, scores, logZ, stream):
    _check(load().crf_inside_fwd(plan, scores, logZ, stream), "crf_inside_fwd")


def crf_inside_bwd(plan, scores, grad_logZ, marginals, stream):
    _check(load().crf_inside_bwd(plan, scores, grad_logZ, marginals, stream), "crf_inside_bwd")


def crf_inside_fwd_bwd(plan, scores, grad_logZ, logZ, marginals, stream):
    _check(load().crf_inside_fwd_bwd(plan, scores, grad_logZ, logZ, marginals, stream),
           "crf_inside_fwd_bwd")


def crf_cky_decode(plan, scores, spans, best, stream):
    _check(load().crf_cky_decode(plan, scores, spans, best, stream), "crf_cky_decode")


def crf_inside_fwd_bwd_cky(plan, scores, grad_logZ, logZ, marginals, spans, best, stream):
    _check(load().crf_inside_fwd_bwd_cky(plan, scores, grad_logZ, logZ, marginals, spans, best,
                                         stream), "crf_inside_fwd_bwd_cky")


def crf_inside_fwd_bwd_cky_noalloc(plan, scores, grad_logZ, logZ, marginals, spans, best, stream):
    _check(load().crf_inside_fwd_bwd_cky_noalloc(plan, scores, grad_logZ, logZ, marginals, spans, best,
                                                 stream), "crf_inside_fwd_bwd_cky_noalloc")


def crf_mbr_decode(plan, scores, logZ, marginals, spans, best, stream):
    _check(load().crf_mbr_decode(plan, scores, logZ, marginals, spans, best, stream), "crf_mbr_decode")


def crf_gold_loss(plan, scores, gold_spans, grad_loss, loss, grad_scores, stream):
    _check(load().crf_gold_loss(plan, scores, gold_spans, grad_loss, loss, grad_scores, stream), "crf_gold_loss")


def crf_cky_decode_labeled(plan, scores, spans, labels, best, stream):
    _check(load().crf_cky_decode_labeled(plan, scores, spans, labels, best, stream), "crf_cky_decode_labeled")


def crf_label_spans(plan, label_scores, num_labels, spans, labels, stream):
    _check(load().crf_label_spans(plan, label_scores, num_labels, spans, labels, stream), "crf_label_spans")


def crf_biaffine_scores(plan, rl, rr, w, d, ldw, num_labels, scores, stream):
    _check(load().crf_biaffine_scores(plan, rl, rr, w, d, ldw, num_labels, scores, stream),
           "crf_biaffine_scores")


def crf_status_string(status):
    return load().crf_status_string(status).decode()


def crf_last_error():
    return load().crf_last_error().decode()


# --------------------------------------------------------------------------
# Torch-tensor wrapper.

def _stream_ptr(torch, device):
    return torch.cuda.current_stream(device).cuda_stream


class Plan:
    """A batch shape: sentence lengths, padded side N1, label count.

    Tensors passed to the methods must be contiguous float32 on the plan's
    device with shape ``[B, N1, N1]`` (``[B, N1, N1, L]`` when labelled).
    """

    def __init__(self, lengths, n1=None, num_labels=1, flags=0, device=None):
        import numpy as np
        import torch

        self._torch = torch
        lens = np.ascontiguousarray(np.asarray(lengths, dtype=np.int32))
        if lens.ndim != 1:
            raise ValueError("lengths must be 1-D")
        self.lengths = lens
        self.B = int(lens.shape[0])
        self.n1 = int(lens.max()) + 1 if n1 is None else int(n1)
        self.L = int(num_labels)
        self.device = torch.device("cuda", torch.cuda.current_device()) if device is None else torch.device(device)
        self._handle = None
        with torch.cuda.device(self.device):
            self._handle = crf_plan_create(lens.ctypes.data, self.B, self.n1, self.L, flags)

    def close(self):
        if self._handle is not None:
            with self._torch.cuda.device(self.device):
                crf_plan_destroy(self._handle)
            self._handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    @property
    def info(self):
        return crf_plan_info(self._handle)

    # shape / dtype checks (host side only)
    def _scores(self, scores):
        t = self._torch
        shape = (self.B, self.n1, self.n1) if self.L == 1 else (self.B, self.n1, self.n1, self.L)
        if tuple(scores.shape) != shape or scores.dtype != t.float32 or not scores.is_contiguous():
            raise ValueError(f"scores must be contiguous float32 {shape}, got "
                             f"{tuple(scores.shape)} {scores.dtype}")
        if scores.device != self.device:
            raise ValueError(f"scores on {scores.device}, plan on {self.device}")
        return scores.data_ptr()

    def _vec(self, v, name):
        """Pointer of a float32 [B] vector.  Outputs and inputs alike must be
        contiguous: a pointer into a temporary copy would let the kernel write
        results that the caller never sees."""
        if v is None:
            return None
        if tuple(v.shape) != (self.B,) or v.dtype != self._torch.float32 or v.device != self.device:
            raise ValueError(f"{name} must be float32 [{self.B}] on {self.device}")
        if not v.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
        return v.data_ptr()

    def inside_fwd(self, scores, logZ=None):
        """log Z per sentence (float32 [B])."""
        t = self._torch
        sp = self._scores(scores)
        if logZ is None:
            logZ = t.empty(self.B, dtype=t.float32, device=self.device)
        crf_inside_fwd(self._handle, sp, self._vec(logZ, "logZ"), _stream_ptr(t, self.device))
        return logZ

    def inside_fwd_bwd(self, scores, grad_logZ=None, logZ=None, marginals=None):
        """(log Z, marginals).  Only valid cells of ``marginals`` are written;
        a fresh buffer is zero-filled first."""
        t = self._torch
        sp = self._scores(scores)
        if logZ is None:
            logZ = t.empty(self.B, dtype=t.float32, device=self.device)
        if marginals is None:
            marginals = t.zeros_like(scores)
        elif tuple(marginals.shape) != tuple(scores.shape) or not marginals.is_contiguous():
            raise ValueError("marginals must be a contiguous tensor shaped like scores")
        crf_inside_fwd_bwd(self._handle, sp, self._vec(grad_logZ, "grad_logZ"),
                           self._vec(logZ, "logZ"), marginals.data_ptr(),
                           _stream_ptr(t, self.device))
        return logZ, marginals

    def inside_bwd(self, scores, grad_logZ=None, marginals=None):
        t = self._torch
        sp = self._scores(scores)
        if marginals is None:
            marginals = t.zeros_like(scores)
        elif tuple(marginals.shape) != tuple(scores.shape) or not marginals.is_contiguous():
            raise ValueError("marginals must be a contiguous tensor shaped like scores")
        crf_inside_bwd(self._handle, sp, self._vec(grad_logZ, "grad_logZ"), marginals.data_ptr(),
                       _stream_ptr(t, self.device))
        return marginals

    def parse(self, scores, grad_logZ=None, logZ=None, marginals=None, spans=None, best=None):
        """inside_fwd_bwd and cky_decode in one launch:
        (logZ, marginals, spans, best)."""
        t = self._torch
        sp = self._scores(scores)
        R = 2 * (self.n1 - 1) - 1
        if logZ is None:
            logZ = t.empty(self.B, dtype=t.float32, device=self.device)
        if marginals is None:
            marginals = t.zeros_like(scores)
        elif tuple(marginals.shape) != tuple(scores.shape) or not marginals.is_contiguous():
            raise ValueError("marginals must be a contiguous tensor shaped like scores")
        if spans is None:
            spans = t.empty((self.B, R, 2), dtype=t.int32, device=self.device)
        elif tuple(spans.shape) != (self.B, R, 2) or spans.dtype != t.int32 or not spans.is_contiguous():
            raise ValueError(f"spans must be contiguous int32 [{self.B}, {R}, 2]")
        if best is None:
            best = t.empty(self.B, dtype=t.float32, device=self.device)
        crf_inside_fwd_bwd_cky(self._handle, sp, self._vec(grad_logZ, "grad_logZ"),
                               self._vec(logZ, "logZ"), marginals.data_ptr(), spans.data_ptr(),
                               self._vec(best, "best"), _stream_ptr(t, self.device))
        return logZ, marginals, spans, best

    def _spans_out(self, spans):
        t = self._torch
        R = 2 * (self.n1 - 1) - 1
        if spans is None:
            return t.empty((self.B, R, 2), dtype=t.int32, device=self.device)
        if tuple(spans.shape) != (self.B, R, 2) or spans.dtype != t.int32 or not spans.is_contiguous():
            raise ValueError(f"spans must be contiguous int32 [{self.B}, {R}, 2]")
        if spans.device != self.device:
            raise ValueError(f"spans on {spans.device}, plan on {self.device}")
        return spans

    def _labels_out(self, labels):
        t = self._torch
        R = 2 * (self.n1 - 1) - 1
        if labels is None:
            return t.empty((self.B, R), dtype=t.int32, device=self.device)
        if tuple(labels.shape) != (self.B, R) or labels.dtype != t.int32 or not labels.is_contiguous():
            raise ValueError(f"labels must be contiguous int32 [{self.B}, {R}]")
        if labels.device != self.device:
            raise ValueError(f"labels on {labels.device}, plan on {self.device}")
        return labels

    def mbr_decode(self, scores, logZ=None, marginals=None, spans=None, best=None):
        """MBR decoding (Sec. 3.3): (logZ, marginals, spans, best), the trees
        decoded by CKY over the marginals."""
        t = self._torch
        sp = self._scores(scores)
        if logZ is None:
            logZ = t.empty(self.B, dtype=t.float32, device=self.device)
        if marginals is None:
            marginals = t.zeros_like(scores)
        elif tuple(marginals.shape) != tuple(scores.shape) or not marginals.is_contiguous():
            raise ValueError("marginals must be a contiguous tensor shaped like scores")
        spans = self._spans_out(spans)
        if best is None:
            best = t.empty(self.B, dtype=t.float32, device=self.device)
        crf_mbr_decode(self._handle, sp, self._vec(logZ, "logZ"), marginals.data_ptr(), spans.data_ptr(),
                       self._vec(best, "best"), _stream_ptr(t, self.device))
        return logZ, marginals, spans, best

    def gold_loss(self, scores, gold_spans, grad_loss=None, loss=None, grad_scores=None):
        """Gold-tree CRF loss (Sec. 2.3, Eq. bracket-loss): (loss [B],
        gradient shaped like scores, valid cells only; a fresh buffer is
        zero-filled)."""
        t = self._torch
        sp = self._scores(scores)
        R = 2 * (self.n1 - 1) - 1
        if (tuple(gold_spans.shape) != (self.B, R, 2) or gold_spans.dtype != t.int32
                or not gold_spans.is_contiguous() or gold_spans.device != self.device):
            raise ValueError(f"gold_spans must be contiguous int32 [{self.B}, {R}, 2] on {self.device}")
        if loss is None:
            loss = t.empty(self.B, dtype=t.float32, device=self.device)
        if grad_scores is None:
            grad_scores = t.zeros_like(scores)
        elif tuple(grad_scores.shape) != tuple(scores.shape) or not grad_scores.is_contiguous():
            raise ValueError("grad_scores must be a contiguous tensor shaped like scores")
        crf_gold_loss(self._handle, sp, gold_spans.data_ptr(), self._vec(grad_loss, "grad_loss"),
                      self._vec(loss, "loss"), grad_scores.data_ptr(), _stream_ptr(t, self.device))
        return loss, grad_scores

    def cky_decode_labeled(self, scores, spans=None, labels=None, best=None):
        """One-stage labelled decoding (Sec. 4.2): (spans, labels, best)."""
        t = self._torch
        sp = self._scores(scores)
        spans = self._spans_out(spans)
        labels = self._labels_out(labels)
        if best is None:
            best = t.empty(self.B, dtype=t.float32, device=self.device)
        crf_cky_decode_labeled(self._handle, sp, spans.data_ptr(), labels.data_ptr(), self._vec(best, "best"),
                               _stream_ptr(t, self.device))
        return spans, labels, best

    def label_spans(self, label_scores, spans, labels=None):
        """Labelling stage (Sec. 2.1, Eq. label-argmax) of given trees:
        label_scores [B, N1, N1, L'] float32 (any L'), spans as cky_decode
        writes them; returns int32 [B, 2(N1-1)-1]."""
        t = self._torch
        if (label_scores.dim() != 4 or tuple(label_scores.shape[:3]) != (self.B, self.n1, self.n1)
                or label_scores.dtype != t.float32 or not label_scores.is_contiguous()
                or label_scores.device != self.device):
            raise ValueError(f"label_scores must be contiguous float32 [{self.B}, {self.n1}, {self.n1}, L]")
        spans = self._spans_out(spans)
        labels = self._labels_out(labels)
        crf_label_spans(self._handle, label_scores.data_ptr(), int(label_scores.shape[3]), spans.data_ptr(),
                        labels.data_ptr(), _stream_ptr(t, self.device))
        return labels

    def biaffine_scores(self, rl, rr, w, scores=None):
        """Span (or label) scores from boundary representations (Sec. 2.2,
        Eq. biaffine).  rl, rr: bf16 bit patterns as int16/uint16 tensors
        [B, N1, d]; w: [L, d, ldw] (W transposed, bias at index d).  Returns
        float32 [B, N1, N1] (L = 1) or [B, N1, N1, L]; a fresh buffer is
        NaN-filled, and only valid cells are written."""
        t = self._torch
        if rl.dim() != 3 or tuple(rl.shape[:2]) != (self.B, self.n1) or tuple(rr.shape) != tuple(rl.shape):
            raise ValueError(f"rl and rr must be [{self.B}, {self.n1}, d]")
        d = int(rl.shape[2])
        if w.dim() != 3 or int(w.shape[1]) != d:
            raise ValueError("w must be [L, d, ldw]")
        for x in (rl, rr, w):
            if x.dtype not in (t.int16, t.uint16) or not x.is_contiguous() or x.device != self.device:
                raise ValueError("rl, rr and w must be contiguous 16-bit tensors on the plan's device")
        L = int(w.shape[0])
        shape = (self.B, self.n1, self.n1) if L == 1 else (self.B, self.n1, self.n1, L)
        if scores is None:
            scores = t.full(shape, float("nan"), dtype=t.float32, device=self.device)
        elif tuple(scores.shape) != shape or scores.dtype != t.float32 or not scores.is_contiguous():
            raise ValueError(f"scores must be contiguous float32 {shape}")
        crf_biaffine_scores(self._handle, rl.data_ptr(), rr.data_ptr(), w.data_ptr(), d, int(w.shape[2]), L,
                            scores.data_ptr(), _stream_ptr(t, self.device))
        return scores

    def cky_decode(self, scores, spans=None, best=None):
        """(spans int32 [B, 2(N1-1)-1, 2] preorder padded with -1, best float32 [B])."""
        t = self._torch
        sp = self._scores(scores)
        R = 2 * (self.n1 - 1) - 1
        if spans is None:
            spans = t.empty((self.B, R, 2), dtype=t.int32, device=self.device)
        elif tuple(spans.shape) != (self.B, R, 2) or spans.dtype != t.int32 or not spans.is_contiguous():
            raise ValueError(f"spans must be contiguous int32 [{self.B}, {R}, 2]")
        if best is None:
            best = t.empty(self.B, dtype=t.float32, device=self.device)
        crf_cky_decode(self._handle, sp, spans.data_ptr(), self._vec(best, "best"),
                       _stream_ptr(t, self.device))
        return spans, best


def log_partition(scores, plan):
    """Differentiable log Z: backward returns the span marginals times the
    upstream gradient (Sec. 3.2, Eq. partial-derivative)."""
    import torch

    class _LogZ(torch.autograd.Function):
        @staticmethod
        def forward(ctx, s):
            ctx.save_for_backward(s)
            return plan.inside_fwd(s)

        @staticmethod
        def backward(ctx, g):
            (s,) = ctx.saved_tensors
            g = g.float().contiguous()   # held by this frame until the call has been enqueued
            return plan.inside_bwd(s, grad_logZ=g)

    return _LogZ.apply(scores)
