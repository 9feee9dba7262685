"""bench.py's output contract, on short runs called in-process (no child process).

GPU: each memory form, and the configuration form's graph-replay mode, prints one JSON line
with the fields the measurement needs. CPU: more than one GPU is refused with exit status 2, and
the algorithmic FLOPs and bytes the roofline divides by match their closed forms.
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


# ---- the algorithmic work the roofline divides by (host logic only)

def test_segment_flops_are_the_closed_form():
    """FWD1 + FWD2 + BWD + UPD of one segment are 2 L T (2 d h + 3 h D + d D) FLOPs: for the
    8B-class shape 2^32 per context token."""
    from paper_2608_17616_amd import configs
    for cfg in (configs.TINY, configs.ONE_B, configs.THREE_B, configs.EIGHT_B):
        w = bench.stage_work(cfg, 64)
        L, d, h, D, T = cfg.n_layers, cfg.d_model, cfg.d_hidden, cfg.d_out, cfg.seg_len
        seg = sum(w[k][0] for k in ("xt", "fwd1", "fwd2", "bwd", "upd"))
        assert seg == 2 * L * T * (2 * d * h + 3 * h * D + d * D)
    assert sum(bench.stage_work(configs.EIGHT_B, 64)[k][0]
               for k in ("fwd1", "fwd2", "bwd", "upd")) / configs.EIGHT_B.seg_len == 2 ** 32


def test_paper_optimizer_bytes_over_one_call():
    """With S segments per call, the renormalisation's per-launch average times S is the row
    scales of every segment plus one rescaling of both weights and their copies, and the
    updates carry the copies of the other S - 1 segments."""
    from paper_2608_17616_amd import configs
    for act in ("bf16", "f32"):
        cfg = configs.ONE_B.with_(optimizer="paper", act_dtype=act)
        L, d, h, D = cfg.n_layers, cfg.d_model, cfg.d_hidden, cfg.d_out
        E = 2 if act == "bf16" else 4
        one = bench.stage_work(cfg, 64, per_call=1)
        for S in (2, 5, 64):
            many = bench.stage_work(cfg, 64, per_call=S)
            scales = L * 4 * (h * d + D * h) // 64
            assert many["renorm"][1] * S == pytest.approx(
                one["renorm"][1] + (S - 1) * scales, rel=1e-12)
            copies_w1 = L * h * d * (E if act == "bf16" else 0)
            copies_w2 = L * D * h * 2 * E
            assert (many["upd"][1] - one["upd"][1]) * S == pytest.approx((S - 1) * copies_w1,
                                                                         rel=1e-12)
            assert (many["bwd"][1] - one["bwd"][1]) * S == pytest.approx((S - 1) * copies_w2,
                                                                         rel=1e-12)
            for k in ("fwd1", "fwd2", "bwd", "upd"):
                assert many[k][0] == one[k][0]


def test_block_form_flops():
    """The block form's FLOPs per segment, averaged over a block of B segments: the step's own
    plus the corrections 2 T kp (3 h + 2 D) with kp = T (B - 1) / 2, plus the block's share of
    the token Gram matrix."""
    from paper_2608_17616_amd import configs
    cfg = configs.STRESS
    L, d, h, D, T = cfg.n_layers, cfg.d_model, cfg.d_hidden, cfg.d_out, cfg.seg_len
    B = 8
    w = bench.stage_work(cfg, 64, blk=B)
    bt = B * T
    own = 2 * L * T * (2 * d * h + 3 * h * D + d * D)
    corr = L * 2 * T * (T * (B - 1) / 2) * (3 * h + 2 * D)
    gram = L * 2 * bt * bt * d
    per_segment = (w["bfwd"][0] + w["bupd"][0]) / B + w["bseq"][0]
    assert per_segment == pytest.approx(own + corr + gram / B, rel=1e-12)
