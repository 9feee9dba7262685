"""HIP-graph capture of the segment step.

The segment calls enqueue kernels only: no allocation, no memset and no host synchronisation.
A caller can therefore capture them in a graph and replay it, copying each new segment into
the captured input buffer first. Every replay here is checked bitwise against the same
segments run eagerly on a second handle over the same initial state. Eager work and
synchronisations run between the replays.

The configuration-form handle alternates two copies of W2^T between consecutive segments: the
backward reads the copy of the previous weights while the update writes the next one. Its graph
therefore captures two consecutive segment calls. The paper-form handle keeps no such state
and captures one.
"""
import numpy as np
import pytest

from paper_2608_17616_amd import configs, inputs, mone
from gpu_helpers import DeviceProblem

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

GRAPH_BF16 = configs.MoneConfig("graph_bf16", n_layers=3, d_model=128, d_hidden=192, d_kv=64,
                                seg_len=160, n_context=960, act_dtype="bf16", lr=5e-2)
# 64-token segments in fp32: the forward launches split their contraction (partial sums in the
# workspace, then a fixed-order reduction)
GRAPH_SHORT = configs.MoneConfig("graph_short_f32", n_layers=3, d_model=512, d_hidden=384,
                                 d_kv=128, seg_len=64, n_context=384, act_dtype="f32", lr=2e-2)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    mone.lib()


@pytest.mark.parametrize("cfg", [GRAPH_BF16, GRAPH_SHORT], ids=lambda c: c.name)
def test_config_form_segment_pairs_replay_bitwise(cfg):
    print(f"[graph] config form {cfg.name}", flush=True)
    prob = DeviceProblem(cfg, [0])
    segs = [prob.segment(s) for s in range(6)]
    w1e, w2e = prob.w1.clone(), prob.w2.clone()
    eager = mone.TtlSession(cfg, prob.wkv, w1e, w2e)
    w1g, w2g = prob.w1.clone(), prob.w2.clone()
    sess = mone.TtlSession(cfg, prob.wkv, w1g, w2g)
    x0, x1 = torch.empty_like(segs[0]), torch.empty_like(segs[0])
    torch.cuda.synchronize()  # the handles' set-up work is done before the capture
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        sess.segment(x0)
        sess.segment(x1)
    torch.cuda.synchronize()
    assert torch.equal(w1g, prob.w1) and torch.equal(w2g, prob.w2)  # capture ran nothing
    for r in range(3):
        x0.copy_(segs[2 * r])
        x1.copy_(segs[2 * r + 1])
        g.replay()
        eager.segment(segs[2 * r])
        eager.segment(segs[2 * r + 1])
        torch.cuda.synchronize()
        assert torch.equal(w1g, w1e) and torch.equal(w2g, w2e), f"replay {r}"
        assert not torch.equal(w1g, prob.w1)
        float((w1g.abs().sum() + w2g.abs().sum()).item())  # eager work between replays
    # the graph leaves the handle's state consistent for eager calls that follow
    x = prob.segment(6)
    sess.segment(x)
    eager.segment(x)
    torch.cuda.synchronize()
    assert torch.equal(w1g, w1e) and torch.equal(w2g, w2e)
    assert np.allclose(sess.loss(), eager.loss(), rtol=0, atol=0)
    sess.close()
    eager.close()


GRAPH_BLOCK = configs.MoneConfig("graph_block_bf16", n_layers=3, d_model=192, d_hidden=320,
                                 d_kv=64, seg_len=64, n_context=1024, act_dtype="bf16", lr=2e-2,
                                 block_tokens=512)


def test_block_form_replays_bitwise():
    # mone_ttl_segments in the block form: 16 segments = two blocks of 8, so the W2^T copies
    # alternate twice per call and the captured call can be replayed as it is
    cfg = GRAPH_BLOCK
    print(f"[graph] block form {cfg.name}", flush=True)
    prob = DeviceProblem(cfg, [])
    T, S = cfg.seg_len, 16
    ctx = [torch.cat([prob.segment(16 * r + s, record=False) for s in range(S)], dim=1)
           for r in range(3)]
    w1e, w2e = prob.w1.clone(), prob.w2.clone()
    eager = mone.TtlSession(cfg, prob.wkv, w1e, w2e)
    w1g, w2g = prob.w1.clone(), prob.w2.clone()
    sess = mone.TtlSession(cfg, prob.wkv, w1g, w2g)
    xg = torch.empty_like(ctx[0])
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        sess.segments(xg)
    torch.cuda.synchronize()
    assert torch.equal(w1g, prob.w1) and torch.equal(w2g, prob.w2)  # capture ran nothing
    for r in range(3):
        xg.copy_(ctx[r])
        g.replay()
        eager.segments(ctx[r])
        torch.cuda.synchronize()
        assert torch.equal(w1g, w1e) and torch.equal(w2g, w2e), f"replay {r}"
        assert np.array_equal(sess.loss(), eager.loss())
        float((w1g.abs().sum() + w2g.abs().sum()).item())  # eager work between replays
    sess.close()
    eager.close()


def _sw_session(cfg):
    from test_gpu_swiglu import SwProblem
    return SwProblem(cfg)


@pytest.mark.parametrize("cfg", [
    configs.SW_TINY.with_(name="graph_sw_f32_paper", optimizer="paper"),
    configs.SW_TINY.with_(name="graph_sw_bf16_sgd", act_dtype="bf16"),
], ids=lambda c: c.name)
def test_paper_form_segment_replays_bitwise(cfg):
    print(f"[graph] paper form {cfg.name}", flush=True)
    pe, pg = _sw_session(cfg), _sw_session(cfg)
    L, n = cfg.n_layers, cfg.seg_len
    act = torch.bfloat16 if cfg.act_dtype == "bf16" else torch.float32

    def seg(s):
        xs = np.stack([inputs.segment_x(cfg, l, s, n) for l in range(L)])
        return torch.from_numpy(xs).to("cuda", act)

    xg = torch.empty(L, n, cfg.d_model, dtype=act, device="cuda")
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        pg.sess.segment(xg, n)
    torch.cuda.synchronize()
    for s in range(4):
        xg.copy_(seg(s))
        g.replay()
        pe.segment(s, n)
        torch.cuda.synchronize()
        for m in range(3):
            assert torch.equal(pg.w[m], pe.w[m]), f"segment {s}, matrix {m}"
            if pe.opt is not None:
                assert torch.equal(pg.mom[m], pe.mom[m]), f"segment {s}, momentum {m}"
        float(sum(w.abs().sum() for w in pg.w).item())  # eager work between replays
    assert np.array_equal(pg.sess.loss(), pe.sess.loss())
    pg.sess.close()
    pe.sess.close()


def test_paper_form_multi_batch_call_replays_bitwise():
    # one mone_swiglu_segments call of 6 segments in batches of 2: the preprocessing runs on the
    # handle's internal stream, forked from and joined to the captured stream
    cfg = configs.SW_TINY.with_(name="graph_sw_multi", optimizer="paper", prep_segments=2)
    print(f"[graph] paper form multi-batch call {cfg.name}", flush=True)
    pe, pg = _sw_session(cfg), _sw_session(cfg)
    L, T, S = cfg.n_layers, cfg.seg_len, 6
    act = torch.bfloat16 if cfg.act_dtype == "bf16" else torch.float32
    xg = torch.empty(L, S * T, cfg.d_model, dtype=act, device="cuda")
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        pg.sess.segments(xg)
    torch.cuda.synchronize()
    for m in range(3):
        assert torch.equal(pg.w[m], pg.w0[m])  # capture ran nothing
    for r in range(3):
        x = pe.segments(r * S, S)
        xg.copy_(x)
        g.replay()
        torch.cuda.synchronize()
        for m in range(3):
            assert torch.equal(pg.w[m], pe.w[m]), f"replay {r}, matrix {m}"
            assert torch.equal(pg.mom[m], pe.mom[m]), f"replay {r}, momentum {m}"
        assert np.array_equal(pg.sess.loss(), pe.sess.loss())
        float(sum(w.abs().sum() for w in pg.w).item())  # eager work between replays
    pg.sess.close()
    pe.sess.close()
