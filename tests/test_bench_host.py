"""bench.py's host-side helpers, on the CPU: the code hash that ties the committed
counter summaries to the kernel source they were taken on, and the one-GPU rule."""

import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _write(path, text):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w") as f:
        f.write(text)
    return path


def test_comment_and_layout_edits_keep_the_code_hash(tmp_path):
    a = _write(str(tmp_path / "a.hip"), "int f(int x) {\n  return x + 1;  // one more\n}\n")
    b = _write(str(tmp_path / "b.hip"), "/* a header\n   over two lines */\nint f(int x) {\n\n    return x + 1;\n}\n")
    c = _write(str(tmp_path / "c.hip"), "int f(int x) {\n  return x + 2;  // one more\n}\n")
    assert bench.code_hash(a) == bench.code_hash(b)
    assert bench.code_hash(a) != bench.code_hash(c)


def test_comment_markers_inside_literals_are_code():
    assert bench.code_only('const char* s = "a//b";  // gone') == 'const char* s = "a//b";'
    assert bench.code_only("char c = '/'; /* gone */ char d = '*';") == "char c = '/';   char d = '*';"
    assert bench.code_only('const char* e = "q\\"//";') == 'const char* e = "q\\"//";'


def test_traffic_is_read_only_for_the_current_kernel_source(tmp_path, monkeypatch):
    src = _write(str(tmp_path / "paper_2609_32278_amd" / "csrc" / "kvx_attn.hip"), "__global__ void k() {}\n")
    summary = str(tmp_path / "profiles" / "extend_attn_wide70b_hbm_counters.md")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    h = bench.code_hash(src)
    assert h == bench.attn_source_hash("wide70b")
    line = "kernel code sha256[:16] (source without comments and blank lines): `{}` (store: `0000000000000000`)"
    _write(summary, line.format(h) + "\n\nHBM bytes per launch (scaled): `3.5e+11`\n")
    assert bench.traffic_from_profiles("wide70b") == 3.5e11
    _write(src, "__global__ void k() { int x = 0; }\n")  # the kernel changed: the counters are stale
    assert bench.traffic_from_profiles("wide70b") is None


def test_committed_summaries_name_a_hash_in_the_current_format():
    import glob
    for path in glob.glob(os.path.join(ROOT, "profiles", "*_hbm_counters.md")):
        text = open(path).read()
        assert "kernel code sha256[:16] (source without comments and blank lines): `" in text, path


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       timeout=300, cwd=ROOT)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)
