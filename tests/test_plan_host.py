"""Host logic of the plan (crf_plan.cpp), built for the CPU with stub HIP
allocation calls (tests/plan_host_stub.cpp) and checked on synthetic batches:
every sentence in exactly one inside and one CKY bundle, each bundle within
the launch's LDS, the chart layouts' stride congruences (the condition under
which the sweeps' LDS reads are bank-conflict free), and the fused queue.
"""
import os
import shutil
import subprocess

import numpy as np
import pytest

from paper_2008_03736_amd import workloads as W

HERE = os.path.dirname(os.path.abspath(__file__))
ROCM_INCLUDE = "/opt/rocm/include"


@pytest.fixture(scope="module")
def harness(tmp_path_factory):
    cxx = shutil.which("g++")
    if cxx is None or not os.path.isdir(ROCM_INCLUDE):
        pytest.skip("needs g++ and the HIP headers")
    out = str(tmp_path_factory.mktemp("plan") / "plan_host")
    # host code only (g++, no GPU code): built with the address and
    # undefined-behaviour sanitizers, which abort the run on a finding
    cmd = [cxx, "-O1", "-g", "-std=c++17", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-fno-omit-frame-pointer", "-D__HIP_PLATFORM_AMD__", "-I" + ROCM_INCLUDE,
           "-I" + os.path.join(HERE, "..", "include"), "-o", out, os.path.join(HERE, "plan_host_stub.cpp")]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    return out


def plan_of(harness, tmp_path, lengths, labels=None, flags=0):
    f = tmp_path / "lengths.txt"
    f.write_text("\n".join(str(int(v)) for v in lengths))
    args = [harness, str(f), str(labels if labels is not None else 1), str(flags)]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    res = subprocess.run(args, capture_output=True, text=True, env=env)
    assert res.returncode == 0, res.stdout[-2000:] + res.stderr[-4000:]
    assert "runtime error" not in res.stderr and "AddressSanitizer" not in res.stderr, res.stderr[-4000:]
    head, recs = None, []
    for line in res.stdout.splitlines():
        t = line.split()
        if t[0] == "P":
            head = dict(zip(["n_mix", "grid", "lds_in", "lds_ck", "half_cu"], map(int, t[1:])))
        elif t[0] == "W":
            head.update(zip(["spill", "cky_spill", "split_ws", "ws_users", "ws_bytes", "fused_queue"],
                            map(int, t[1:])))
        elif t[0] == "R":
            v = list(map(int, t[1:]))
            recs.append(dict(kind=v[0], n=v[1], count=v[2], split_ws=v[3], strict=v[4], ld=v[5], cs=v[6],
                             e=v[7], bytes=v[8], ids=v[9:]))
        elif t[0] == "I":
            v = list(map(int, t[1:]))
            recs.append(dict(kind=1, n=v[0], count=v[1], ids=v[2:]))
        elif t[0] == "Q":
            head.update(zip(["team_cap", "team_area"], map(int, t[1:])))
        elif t[0] == "T":
            v = list(map(int, t[1:]))
            head["n1"] = v[0]
            head.setdefault("tiles", []).append(v[1:])
        elif t[0] == "M":
            v = list(map(int, t[1:]))
            head.setdefault("mbr", []).append(dict(n=v[0], count=v[1], split_ws=v[2], inside_strict=v[3],
                                                   cky_strict=v[4], grid=v[5], lds=v[6], inside_bytes=v[7],
                                                   ids=v[8:]))
    return head, recs


def check_plan(head, recs, lengths):
    lengths = np.asarray(lengths)
    assert head["n_mix"] == len(recs)
    # one workgroup slot per CU per bundle LDS that fits (256 CUs, 160 KiB each)
    per_cu = min(4, max(1, 163840 // max(head["lds_in"], head["lds_ck"])))
    assert head["grid"] == min(len(recs), 256 * per_cu)
    for kind in (0, 1):
        ids = [i for r in recs if r["kind"] == kind for i in r["ids"]]
        assert sorted(ids) == list(range(len(lengths))), "every sentence once per kind"
    for r in recs:
        assert r["count"] == len(r["ids"]) >= 1
        assert all(lengths[i] == r["n"] for i in r["ids"])
        n, nb, ld, cs = r["n"], r["count"], r["ld"], r["cs"]
        if r["kind"] == 1:
            assert ld >= n + 1 and 2 * ld * ld <= cs < 2 * ld * ld + 32
            assert 0 < r["bytes"] <= head["lds_in"] <= 2 * head["half_cu"] + 256
            if r["strict"] and r["e"] == 0 and not (nb >= 32 and nb % 4 == 0):
                # span g's runs start at sigma g (mod 32): cs = sigma odd, ld = nb sigma
                assert cs % 2 == 1 and (ld - nb * cs) % 32 == 0, r
        else:
            assert ld >= n + 1 and cs % 8 == 0 and cs >= 8 * ld * ld
            u = cs // 8
            if r["strict"] and not (nb >= 16 and nb % 4 == 0):
                assert u % 2 == 1 and (ld + 1 - nb * u) % 16 == 0, r
            elif not r["strict"]:
                assert u % 2 == 1 and ld % 2 == 0


@pytest.mark.parametrize("name", ["tiny", "mixed", "longer"])
def test_plan_of_workloads(harness, tmp_path, name):
    b = W.make(name)
    head, recs = plan_of(harness, tmp_path, b.lengths)
    check_plan(head, recs, b.lengths)
    if name == "longer":
        # sentences of more than 99 words need a whole CU in either layout:
        # the launch runs one workgroup per CU, and those bundles take the
        # strict layout there
        assert head["lds_in"] > head["half_cu"]
        assert all(r["strict"] for r in recs if r["kind"] == 1 and r["n"] > 99)
    if name == "mixed":
        assert head["lds_in"] <= head["half_cu"]
        # both layouts occur, and most bundles take the strict one
        for kind in (0, 1):
            flags = [r["strict"] for r in recs if r["kind"] == kind]
            assert 0 < sum(flags) and sum(flags) > len(flags) // 2


@pytest.mark.parametrize("seed", range(6))
def test_plan_of_random_batches(harness, tmp_path, seed):
    rng = np.random.default_rng(seed)
    lengths = rng.integers(1, 100, size=int(rng.integers(1, 3000)))
    head, recs = plan_of(harness, tmp_path, lengths)
    check_plan(head, recs, lengths)


@pytest.mark.parametrize("n,count", [(9, 4), (14, 40), (17, 32), (20, 20), (30, 8), (45, 4), (99, 1)])
def test_plan_of_one_length(harness, tmp_path, n, count):
    lengths = [n] * count + [99] * 200
    head, recs = plan_of(harness, tmp_path, lengths)
    check_plan(head, recs, lengths)


@pytest.mark.parametrize("labels,seed", [(2, 0), (7, 1), (32, 2), (33, 3), (100, 4)])
def test_plan_of_labelled_batches(harness, tmp_path, labels, seed):
    # labelled plans run inside bundles only (no fused queue); each sentence
    # in exactly one bundle of sentences of its own length
    rng = np.random.default_rng(seed)
    lengths = rng.integers(1, 100, size=int(rng.integers(1, 2000)))
    head, recs = plan_of(harness, tmp_path, lengths, labels)
    assert head["n_mix"] == 0 and recs
    ids = [i for r in recs for i in r["ids"]]
    assert sorted(ids) == list(range(len(lengths)))
    for r in recs:
        assert r["count"] == len(r["ids"]) >= 1
        assert all(lengths[i] == r["n"] for i in r["ids"])


def test_workspace_users_reported(harness, tmp_path):
    # The mixed batch keeps every chart in LDS, yet its 99-word sentence's CKY
    # split table lives in the plan's workspace: plan info must count it as a
    # workspace user (calls on one plan are stream-ordered for that reason).
    b = W.make("mixed")
    head, _ = plan_of(harness, tmp_path, b.lengths)
    assert head["spill"] == 0 and head["cky_spill"] == 0
    long_ones = int(np.sum(b.lengths >= 97))
    assert long_ones >= 1
    assert head["split_ws"] == long_ones and head["ws_users"] == long_ones
    assert head["ws_bytes"] > 0 and head["fused_queue"] == 1
    # a batch of short sentences uses no workspace at all
    head, _ = plan_of(harness, tmp_path, [5, 9, 30, 60] * 10)
    assert head["ws_users"] == 0 and head["ws_bytes"] == 0
    # sentences past the LDS limit use it for both charts
    head, _ = plan_of(harness, tmp_path, [200, 150, 10])
    assert head["spill"] == 2 and head["cky_spill"] == 2 and head["ws_users"] == 2


def test_team_area_only_with_workspace_sentences(harness, tmp_path):
    # the team area (and the device's capacity for workspace workgroups: the
    # stub's 256 CUs, one workgroup each) exists exactly when some sentence's
    # chart is in the workspace
    head, _ = plan_of(harness, tmp_path, [200, 150, 10])
    assert head["team_area"] == 1 and head["team_cap"] == 256
    head, _ = plan_of(harness, tmp_path, W.make("mixed").lengths)
    assert head["team_area"] == 0
    # CRF_NO_TEAMS (0x2): workspace sentences, no team area
    head, _ = plan_of(harness, tmp_path, [200, 150, 10], flags=2)
    assert head["team_area"] == 0 and head["spill"] == 2


def test_step_shape_runs(harness):
    # shape_run_end, the closed form the sweeps use to run a shape's steps as
    # one loop, agrees with step_shape_k for every step up to 5000 splits:
    # the shape holds from K to the run's end and changes there
    res = subprocess.run([harness, "runs"], capture_output=True, text=True)
    assert res.returncode == 0 and res.stdout.strip() == "RUNS OK", res.stdout[-500:]


def test_team_launch_shapes(harness):
    # Every workspace launch shape: a team of k (a power of two in
    # [kTeamMinK, kTeamMaxK] = [8, 16]) per job, m = ceil(jobs / 8) teams per
    # XCD, the grid 8 m k within what the device holds at once; otherwise a
    # workgroup per job.  Teams whenever the device has room for k >= 8.
    res = subprocess.run([harness, "teams"], capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-2000:]
    rows = [tuple(map(int, l.split()[1:])) for l in res.stdout.splitlines() if l.startswith("S ")]
    assert len(rows) == 8 * 301
    for jobs, cap, k, grid in rows:
        m = -(-jobs // 8)
        if k == 1:
            assert grid == jobs
            assert jobs == 0 or 8 * m * 8 > cap        # no room for teams of 8
        else:
            assert k in (8, 16) and grid == 8 * m * k <= cap
            assert 8 * m >= jobs and 8 * m <= 1024    # a team per job, within the team area
            assert k == 16 or 8 * m * 16 > cap        # the largest team that fits
    assert any(k > 1 for _, _, k, _ in rows)
    assert res.stdout.splitlines()[-1] == "N 1 5"     # no team area: a workgroup per job


@pytest.mark.parametrize("name", ["tiny", "mixed", "longer"])
def test_mbr_bundles(harness, tmp_path, name):
    # MBR bundles: every sentence in exactly one, of its own length, within
    # the launch's LDS with either chart; split tables of long sentences in
    # the workspace; one workgroup slot per CU per bundle LDS that fits
    b = W.make(name)
    head, _ = plan_of(harness, tmp_path, b.lengths)
    mb = head["mbr"]
    ids = sorted(i for r in mb for i in r["ids"])
    assert ids == list(range(b.B))
    lds = mb[0]["lds"]
    for r in mb:
        assert r["count"] == len(r["ids"]) and all(b.lengths[i] == r["n"] for i in r["ids"])
        assert r["inside_bytes"] <= lds
        assert (r["split_ws"] >= 0) == (r["n"] >= 97)
        assert r["grid"] == min(len(mb), 256 * min(4, max(1, 163840 // lds)))
    if name == "mixed":
        assert lds <= head["half_cu"]          # two workgroups per CU


def test_mbr_not_fused_when_all_in_workspace(harness, tmp_path):
    head, _ = plan_of(harness, tmp_path, [200, 150])
    assert "mbr" not in head


def check_tiles(head, lengths, rows=64):
    """The scorer's tiles cover every valid cell (i < j <= n_b) of every
    sentence exactly once; a tile's rows and columns are fence posts of the
    batch (or -1); a tile that packs whole sentences uses its fence posts as
    both its rows and its columns."""
    lengths = np.asarray(lengths, np.int64)
    n1 = head["n1"]
    t = np.asarray(head["tiles"], np.int64)
    assert t.shape[1] == 2 * rows
    r, c = t[:, :rows], t[:, rows:]
    for ids in (r, c):
        v = ids[ids >= 0]
        assert np.all(v % n1 <= lengths[v // n1]), "a tile names a fence post past its sentence"
    rr = np.repeat(r[:, :, None], rows, axis=2)
    cc = np.repeat(c[:, None, :], rows, axis=1)
    ok = (rr >= 0) & (cc >= 0) & (rr // n1 == cc // n1) & (rr % n1 < cc % n1)
    cells = rr[ok] * n1 + cc[ok] % n1                       # (b n1 + i) n1 + j
    got = np.bincount(cells, minlength=len(lengths) * n1 * n1)
    b, i, j = np.unravel_index(np.arange(len(lengths) * n1 * n1), (len(lengths), n1, n1))
    want = ((i < j) & (j <= lengths[b])).astype(np.int64)
    assert np.array_equal(got, want), "valid cells covered exactly once, nothing else"
    # a sentence of up to rows - 1 words sits whole in one tile, whose rows
    # are also its columns
    short = np.flatnonzero(lengths + 1 <= rows)
    for k in range(len(t)):
        row = r[k][r[k] >= 0]
        for b in np.unique(row // n1):
            if lengths[b] + 1 <= rows:
                assert np.array_equal(np.sort(row[row // n1 == b] % n1), np.arange(lengths[b] + 1)), (k, b)
                assert np.array_equal(r[k], c[k])
    seen = np.unique(r[r >= 0] // n1)
    assert np.all(np.isin(short, seen))
    tile_idx = np.arange(len(t))[:, None].repeat(rows, 1)
    pairs = np.unique(np.stack([tile_idx[r >= 0], r[r >= 0] // n1], -1), axis=0)   # (tile, sentence)
    tiles_of = np.bincount(pairs[:, 1], minlength=len(lengths))
    assert np.all(tiles_of[short] == 1), "a short sentence in more than one tile"


@pytest.mark.parametrize("name", ["tiny", "mixed", "longer", "stress"])
def test_biaffine_tiles_cover_every_cell_once(harness, tmp_path, name):
    lengths = W.make(name, 0).lengths
    head, _ = plan_of(harness, tmp_path, lengths)
    check_tiles(head, lengths)


def test_biaffine_tiles_edge_lengths(harness, tmp_path):
    # one word, exactly a tile's rows (63 words: 64 fence posts), one past it,
    # two and three blocks, and many short sentences that fill tiles unevenly
    lengths = [1, 63, 64, 127, 128, 129, 200, 2, 3, 5, 7, 11, 13] + [4] * 40
    head, _ = plan_of(harness, tmp_path, lengths)
    check_tiles(head, lengths)
