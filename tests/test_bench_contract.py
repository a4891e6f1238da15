"""The parts of bench.py's contract that need no GPU: the one-GPU refusal, the digest
that ties a committed counter summary to the kernel sources it was taken on, and the
committed summaries themselves (CPU)."""
import glob
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode != 0
    assert "one GPU" in r.stdout + r.stderr
    assert not any(line.startswith("{") for line in r.stdout.splitlines())  # no bench line


def test_code_digest_ignores_comments_and_indentation(tmp_path):
    a, b, c = tmp_path / "a.hip", tmp_path / "b.hip", tmp_path / "c.hip"
    a.write_text("int f(int x) {\n  return x + 1;  // one more\n}\n")
    b.write_text("/* the same code */\nint f(int x) {\n\n        return x + 1;\n}\n")
    c.write_text("int f(int x) {\n  return x + 2;\n}\n")
    rel = lambda p: os.path.relpath(p, tmp_path)
    da = bench.code_sha256(str(tmp_path), [rel(a)])
    assert da == bench.code_sha256(str(tmp_path), [rel(b)])
    assert da != bench.code_sha256(str(tmp_path), [rel(c)])


def test_committed_counter_summaries_parse():
    hbm = sorted(glob.glob(os.path.join(ROOT, "profiles", "*_hbm_counters.txt")))
    sq = sorted(glob.glob(os.path.join(ROOT, "profiles", "*_sq_counters.txt")))
    assert hbm and sq
    for path in hbm + sq:
        fields = {}
        for line in open(path):
            if ":" in line and not line.startswith(" "):
                k, v = line.split(":", 1)
                fields[k.strip()] = v.strip()
        rels = fields["sources"].split()
        assert rels and all(os.path.exists(os.path.join(ROOT, r)) for r in rels), path
        assert len(fields["sources_code_sha256"]) == 64, path
        if path in hbm:
            for k in ("fetch_kib_per_dispatch", "fetch_scale", "write_kib_per_dispatch", "write_scale"):
                assert float(fields[k]) > 0, (path, k)
        else:
            for k in ("mfma_busy", "lds_busy", "wave_wait"):
                assert 0.0 <= float(fields[k]) <= 1.0, (path, k)
