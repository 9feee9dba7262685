"""bench.py's output contract, on short runs called in-process (no child process).

GPU: each memory form, and the configuration form's graph-replay mode, prints one JSON line
with the fields the measurement needs. CPU: more than one GPU is refused with exit status 2.
"""
import json
import sys

import pytest

import bench

TOP = ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
       "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config", "roofline",
       "stages", "finite")
ROOF = ("bound", "achieved", "peak", "unit", "frac", "traffic")

CASES = {
    "config_tiny": ["--config", "tiny", "--steps", "1", "--warmup", "1", "--no-cpu-baseline"],
    "config_tiny_graph": ["--config", "tiny", "--steps", "2", "--warmup", "1",
                          "--no-cpu-baseline", "--graph"],
    "swiglu": ["--memory", "swiglu", "--segments", "4", "--steps", "1", "--warmup", "1",
               "--no-cpu-baseline"],
}


def _run(monkeypatch, capsys, argv):
    monkeypatch.setattr(sys, "argv", ["bench.py", *argv])
    bench.main()
    lines = [ln for ln in capsys.readouterr().out.splitlines() if ln.strip()]
    return json.loads(lines[-1])


@pytest.mark.gpu
@pytest.mark.parametrize("name", list(CASES))
def test_bench_prints_one_json_line(monkeypatch, capsys, name):
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    print(f"[bench] {name}", flush=True)
    d = _run(monkeypatch, capsys, CASES[name])
    missing = [k for k in TOP if k not in d] + [k for k in ROOF if k not in d["roofline"]]
    assert not missing, missing
    assert d["value"] > 0 and d["ms_per_step"] > 0 and d["finite"]
    assert d["n_gpus"] == 1 and d["higher_is_better"] is True
    assert "workload" in d["config"]
    assert 0 < d["roofline"]["frac"] < 1


def test_more_than_one_gpu_is_refused(monkeypatch, capsys):
    monkeypatch.setattr(sys, "argv", ["bench.py", "--gpus", "2"])
    with pytest.raises(SystemExit) as e:
        bench.main()
    assert e.value.code == 2
    assert "one GPU" in capsys.readouterr().err
