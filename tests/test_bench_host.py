"""Host logic of bench.py (no GPU): the one-GPU contract and the rule that a
committed counter reading is used only for the workload and the kernel
sources it was taken on."""
import importlib.util
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)


def test_source_hash_ignores_comments_and_layout_only():
    b = _bench()
    code = "int f(int x)\n{\n    return x + 1;   // add one\n}\n"
    assert b._code_only(code) == b._code_only("/* a\n block */ int f(int x) {\n return x + 1; }")
    assert b._code_only(code) != b._code_only(code.replace("x + 1", "x + 2"))


def test_counter_reading_only_for_its_workload_and_sources(tmp_path, monkeypatch):
    b = _bench()
    rec = json.load(open(os.path.join(ROOT, "profiles", "traffic.json")))
    cls = "attn_decode"
    # the committed record belongs to the default workload
    assert rec["workload"] == b.DEFAULT_WORKLOAD
    # a copy under another root: same record, then a stale source hash, then another workload
    prof = tmp_path / "profiles"
    prof.mkdir()
    csrc = tmp_path / "paper_2606_18967_amd" / "csrc"
    csrc.mkdir(parents=True)
    for f in b.SOURCES_OF_CLASS[cls]:
        (csrc / f).write_text(open(os.path.join(ROOT, "paper_2606_18967_amd", "csrc", f)).read())
    monkeypatch.setattr(b, "ROOT", str(tmp_path))
    (prof / "traffic.json").write_text(json.dumps(rec))
    want = rec["detail"][cls]["bytes"]
    if rec["detail"][cls]["sources"] == b.kernel_sources_hash(b.SOURCES_OF_CLASS[cls]):
        assert b.measured_traffic(cls) == want
    # a comment-only edit keeps the reading; a code edit voids it
    src = csrc / b.SOURCES_OF_CLASS[cls][-1]
    rec["detail"][cls]["sources"] = b.kernel_sources_hash(b.SOURCES_OF_CLASS[cls])
    (prof / "traffic.json").write_text(json.dumps(rec))
    assert b.measured_traffic(cls) == want
    src.write_text(src.read_text() + "\n// a note\n")
    assert b.measured_traffic(cls) == want
    src.write_text(src.read_text() + "\nstatic int extra_symbol_for_the_test;\n")
    assert b.measured_traffic(cls) is None
    # another workload key never takes it
    rec["detail"][cls]["sources"] = b.kernel_sources_hash(b.SOURCES_OF_CLASS[cls])
    (prof / "traffic.json").write_text(json.dumps(rec))
    assert b.measured_traffic(cls, b.workload_key("L4_8B", 64, 2048, 4, "w4", 0)) is None
    assert b.measured_traffic(cls) == want
