"""bench.py's host-side arithmetic on CPU: the algorithmic work model behind
every roofline fraction it reports, the source hash that decides whether the
stored HBM-traffic figures still describe the kernels, and its refusal to run
on more than one GPU."""
import hashlib
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_work_model_counts_splits_and_spans():
    # T: the split points over every span of width >= 2 (one per inside term);
    # P: the spans 0 <= i < j <= n -- counted by enumeration
    lengths = np.array([1, 2, 3, 5, 9, 17, 40], np.int32)
    T = sum(1 for n in lengths for i in range(n + 1) for j in range(i + 2, n + 1) for _ in range(i + 1, j))
    P = sum(1 for n in lengths for i in range(n + 1) for _ in range(i + 1, n + 1))
    wm = bench.work_model(lengths)
    assert wm["T"] == T and wm["P"] == P
    # bytes: scores in and marginals out (fp32), log Z; CKY: scores in,
    # 2n-1 spans of two int32, best
    assert wm["bytes_inside"] == 8 * P + 4 * len(lengths)
    assert wm["bytes_cky"] == 4 * P + 8 * int((2 * lengths.astype(np.int64) - 1).sum()) + 4 * len(lengths)
    # a transcendental priced at 2 slots instead of 4 lowers the inside count
    assert bench.work_model(lengths, trans_slots=2)["slots_inside"] < wm["slots_inside"]
    # labels add per-label work on every span
    assert bench.work_model(lengths, labels=26)["slots_inside"] > wm["slots_inside"]


def test_strip_comments_keeps_code_and_literals():
    src = 'int a = 1; // one\n/* two\n lines */ int b = 2;\nconst char *s = "// not a comment /* nor this */";\n' \
          "char c = '/'; char d = '\\''; const char *e = \"q\\\"// still a string\"; // gone"
    out = bench.strip_comments(src)
    assert "one" not in out and "two" not in out and "gone" not in out
    assert '"// not a comment /* nor this */"' in out
    assert "char c = '/';" in out and "char d = '\\'';" in out
    assert '"q\\"// still a string"' in out
    assert out.startswith("int a = 1; int b = 2;")


def test_source_hash_ignores_comments_and_layout_only():
    code = "int f(int x) {\n    return x + 1;   // add one\n}\n"
    same = "/* header */\nint f(int x) { return x + 1; }\n\n// trailing\n"
    other = "int f(int x) { return x + 2; }"
    h = lambda s: hashlib.sha256(bench.strip_comments(s).encode()).hexdigest()
    assert h(code) == h(same) != h(other)
    # the repository's own hash is well formed and stable across calls
    assert len(bench.source_sha16()) == 16 and bench.source_sha16() == bench.source_sha16()


def test_stored_traffic_is_reported_only_for_its_source():
    name, entry = next(iter(bench.MEASURED_TRAFFIC.items()))
    got, profile = bench.measured_traffic(name)
    if entry["source_sha16"] == bench.source_sha16():
        assert got == entry["bytes"] and os.path.exists(os.path.join(ROOT, profile))
    else:
        assert got is None and profile is None
    assert bench.measured_traffic("no such workload") == (None, None)


def test_more_than_one_gpu_is_refused():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=300)
    assert res.returncode == 2
    assert "one GPU only" in res.stderr
