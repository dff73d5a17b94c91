"""bench.py's command line on the host (no GPU): the one-GPU guard and the
sweep's output handling, with the GPU measurement itself replaced by a stub."""
import importlib.util
import json
import os
import subprocess
import sys
import types

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench_module():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 2
    assert "--gpus must be 1" in r.stderr
    assert r.stdout == ""


def test_sweep_lines_go_to_stdout_and_the_named_file(tmp_path, capsys):
    bench = _bench_module()
    recs = [{"M": 1, "K": 1024, "N": 1024}, {"M": 16, "K": 2048, "N": 2048}]
    bench.sweep_records = lambda Ms, Ks, reps, sink: [sink(r) for r in recs]
    out = tmp_path / "sub" / "sweep.jsonl"
    bench.run_sweep(types.SimpleNamespace(sweep_m="", sweep_k="", sweep_out=str(out)))
    assert [json.loads(l) for l in out.read_text().splitlines()] == recs
    assert [json.loads(l) for l in capsys.readouterr().out.splitlines()] == recs


def test_sweep_without_a_file_writes_stdout_only(tmp_path, capsys, monkeypatch):
    bench = _bench_module()
    recs = [{"M": 256, "K": 4096, "N": 4096}]
    bench.sweep_records = lambda Ms, Ks, reps, sink: [sink(r) for r in recs]
    monkeypatch.chdir(tmp_path)
    bench.run_sweep(types.SimpleNamespace(sweep_m="", sweep_k="", sweep_out=""))
    assert [json.loads(l) for l in capsys.readouterr().out.splitlines()] == recs
    assert list(tmp_path.iterdir()) == []
