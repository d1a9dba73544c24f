"""The C ABI without a GPU: the library loads, exports every declared symbol,
and rejects bad arguments on the host before any HIP call."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2008_03736_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "crf_inside.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(crf_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B.LIB_PATH):
        pytest.fail("libcrfinside.so is not built (run __graft_entry__.build())")
    return B.load()


def test_header_and_binding_agree():
    assert _declared_functions() == sorted(B.SIGNATURES)


def test_every_declared_symbol_is_exported(lib):
    for name in _declared_functions():
        assert hasattr(lib, name), name


def test_constants_match_header():
    text = open(HEADER).read()
    assert f"#define CRF_MAX_LEN {B.CRF_MAX_LEN}" in text
    assert f"#define CRF_MAX_LABELS {B.CRF_MAX_LABELS}" in text
    assert f"#define CRF_FORCE_SPILL 0x{B.CRF_FORCE_SPILL:x}u" in text
    assert f"#define CRF_NO_TEAMS 0x{B.CRF_NO_TEAMS:x}u" in text
    for name, val in [("CRF_OK", 0), ("CRF_EINVAL", 1), ("CRF_ENOMEM", 2), ("CRF_EHIP", 3),
                      ("CRF_EUNSUPPORTED", 4)]:
        assert re.search(rf"\b{name} = {val}\b", text)


def test_status_strings(lib):
    assert B.crf_status_string(0) == "success"
    assert B.crf_status_string(1) == "invalid argument"
    assert B.crf_status_string(4) == "unsupported"
    assert B.crf_status_string(99) == "unknown status"


def _create(lib, lengths, batch, n1, labels=1, flags=0, out=True):
    arr = None if lengths is None else np.ascontiguousarray(lengths, np.int32)
    plan = ctypes.c_void_p(12345)
    rc = lib.crf_plan_create(ctypes.byref(plan) if out else None,
                             None if arr is None else arr.ctypes.data, batch, n1, labels, flags)
    return rc, plan


@pytest.mark.parametrize(
    "lengths,batch,n1,labels,flags,needle",
    [
        (None, 1, 4, 1, 0, "lengths_host"),
        ([3], 0, 4, 1, 0, "batch"),
        ([3], -5, 4, 1, 0, "batch"),
        ([3], 1, 1, 1, 0, "n1"),
        ([3], 1, 1025, 1, 0, "n1"),
        ([0], 1, 4, 1, 0, "lengths[0]"),
        ([4], 1, 4, 1, 0, "lengths[0]"),
        ([2, -1], 2, 4, 1, 0, "lengths[1]"),
        ([3], 1, 4, 0, 0, "num_labels"),
        ([3], 1, 4, 4097, 0, "num_labels"),
        ([3], 1, 4, 1, 0x8, "flags"),
    ],
)
def test_plan_create_rejects_bad_arguments(lib, lengths, batch, n1, labels, flags, needle):
    rc, plan = _create(lib, lengths, batch, n1, labels, flags)
    assert rc == B.CRF_EINVAL
    assert plan.value is None          # *out is cleared on failure
    assert needle in B.crf_last_error()


def test_plan_create_null_out(lib):
    rc, _ = _create(lib, [3], 1, 4, out=False)
    assert rc == B.CRF_EINVAL and "out" in B.crf_last_error()


def test_compute_calls_reject_null_plan(lib):
    dummy = ctypes.c_void_p(0x1000)
    assert lib.crf_inside_fwd(None, dummy, dummy, None) == B.CRF_EINVAL
    assert lib.crf_inside_bwd(None, dummy, None, dummy, None) == B.CRF_EINVAL
    assert lib.crf_inside_fwd_bwd(None, dummy, None, dummy, dummy, None) == B.CRF_EINVAL
    assert lib.crf_cky_decode(None, dummy, dummy, None, None) == B.CRF_EINVAL
    assert lib.crf_inside_fwd_bwd_cky(None, dummy, None, dummy, dummy, dummy, None, None) == B.CRF_EINVAL
    assert lib.crf_inside_fwd_bwd_cky_noalloc(None, dummy, None, dummy, dummy, dummy, None, None) == B.CRF_EINVAL
    assert lib.crf_plan_info(None, None) == B.CRF_EINVAL
    assert lib.crf_plan_destroy(None) == B.CRF_OK


def test_python_wrapper_raises_with_message(lib):
    arr = np.array([5, 0], np.int32)
    with pytest.raises(B.CrfError, match=r"lengths\[1\] = 0"):
        B.crf_plan_create(arr.ctypes.data, 2, 6)


def test_product_package_never_touches_the_oracle():
    pkg = os.path.join(ROOT, "paper_2008_03736_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".cpp", ".h")):
                text = open(os.path.join(dirpath, f)).read()
                assert "oracle" not in text.lower() or f == "workloads.py", f
                assert "import oracle" not in text and "from oracle" not in text, f


def test_ceilings_library_exports_its_header():
    # the microbenchmark library behind bench.py --ceilings
    from paper_2008_03736_amd import ceilings as C

    text = open(os.path.join(ROOT, "include", "crf_ceilings.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    declared = sorted(set(re.findall(r"\b(crf_[a-z_]+)\s*\(", text)))
    assert declared == sorted(C.SIGNATURES)
    if not os.path.exists(C.LIB_PATH):
        pytest.fail("libcrfceilings.so is not built (run __graft_entry__.build())")
    lib = C.load()
    for name in declared:
        assert hasattr(lib, name), name
    # bad arguments are rejected before any launch (no GPU needed)
    assert lib.crf_ceiling_run(9, 1, 64, 1, None, None) != 0
    assert lib.crf_ceiling_run(0, 1, 100, 1, None, None) != 0
