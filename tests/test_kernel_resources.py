"""Register budgets of the HIP kernels, from the resource report that the
build writes beside the library (the compiler's per-kernel figures).

A kernel that runs out of registers spills to scratch memory: the spill
reloads then sit on the sweeps' dependent chain of steps and the spills add
HBM traffic (label code once compiled into the shared inside body pushed
every inside kernel past its 128 VGPRs and slowed the fused launch by a
fifth).  These tests hold every kernel to the scratch it uses now, so such a
change fails on the CPU, at build time, rather than in a profile."""
import csv
import os

import pytest

from paper_2008_03736_amd import build as BLD

# scratch bytes per lane each kernel may use; every other kernel none.  The
# fused and MBR kernels (both the inside and the CKY body in one persistent
# kernel) sit at 128 VGPRs with nothing spilled, since log Z is taken without
# a float64 log, whose coefficients a persistent loop would keep in registers
# (each spilled dword was stored once per lane, 1 MB of HBM writes per
# launch).  Only two team builds of the workspace kernels spill (their team
# state and job loop beside two full sweeps); they run on launches of a few
# long sentences, whose time is set by memory round trips.
ALLOWED_SCRATCH = {"spill_parse_kernel<true>": 72, "loss_kernel<true, true>": 20}
# every kernel the library launches (short names)
# (the workspace kernels come in a lone-workgroup and a team build: the
# last template argument)
EXPECTED = [
    "inside_kernel<false, false, false, false>", "inside_kernel<true, false, false, false>",
    "inside_kernel<false, false, true, false>", "inside_kernel<true, false, true, false>",
    "inside_kernel<false, true, false, false>", "inside_kernel<true, true, false, false>",
    "inside_kernel<false, true, false, true>", "inside_kernel<true, true, false, true>",
    "cky_kernel<false, false, false>", "cky_kernel<false, true, false>",
    "cky_kernel<true, false, false>", "cky_kernel<true, true, false>",
    "cky_kernel<true, false, true>", "cky_kernel<true, true, true>",
    "loss_kernel<false, false>", "loss_kernel<true, false>", "loss_kernel<true, true>",
    "parse_kernel", "spill_parse_kernel<false>", "spill_parse_kernel<true>", "mbr_kernel",
    "label_reduce_kernel", "label_expand_kernel", "label_spans_kernel",
]


def short(name):
    name = name.replace("crf::(anonymous namespace)::", "").replace("crf::", "")
    if name.startswith("void "):
        name = name[5:]
    return name.split("(")[0]


@pytest.fixture(scope="module")
def report():
    if not os.path.exists(BLD.RESOURCES):
        pytest.fail("no kernel resource report: build the library (__graft_entry__.build())")
    with open(BLD.RESOURCES) as f:
        rows = list(csv.DictReader(f, delimiter="\t"))
    return {short(r["kernel"]): r for r in rows}


def test_report_lists_every_kernel(report):
    missing = [k for k in EXPECTED if k not in report]
    assert not missing, f"kernels missing from the resource report: {missing}"
    assert any(k.startswith("biaffine_kernel<") for k in report)


def test_no_kernel_spills_beyond_its_budget(report):
    over = []
    for k, r in report.items():
        scratch = int(r["ScratchSize [bytes/lane]"])
        if scratch > ALLOWED_SCRATCH.get(k, 0):
            over.append(f"{k}: {scratch} bytes/lane of scratch ({r['VGPRs Spill']} VGPRs spilled)")
    assert not over, "kernels spill to scratch: " + "; ".join(over)


def test_inside_kernels_keep_their_occupancy(report):
    # the forward-only inside kernels fit five waves per SIMD, the others four
    for k in ("inside_kernel<false, false, false, false>", "inside_kernel<false, false, true, false>"):
        assert int(report[k]["Occupancy [waves/SIMD]"]) >= 5, k
    for k in ("inside_kernel<true, false, false, false>", "inside_kernel<true, false, true, false>", "parse_kernel"):
        assert int(report[k]["Occupancy [waves/SIMD]"]) >= 4, k
