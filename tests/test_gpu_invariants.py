"""GPU invariants of the TTL path that need no oracle: they hold bitwise.

  * lr = 0 leaves the fast weights bitwise unchanged (Eq. update with a zero step);
  * an empty segment is a no-op;
  * two identical runs give bitwise-identical weights (no order-dependent reductions);
  * perturbing one layer's hidden states changes no other layer (Sec. 3.4, layer locality);
  * the read is idempotent and leaves the weights unchanged (Eq. read; Sec. 3.4);
  * a run split across handles (checkpoint the weights, create a new handle on the copy,
    continue) equals the one-shot run (incremental extension of the final state);
  * segment order matters, and the read of a longer query batch is chunked correctly.
"""
import numpy as np
import pytest

import oracle as orc
from paper_2608_17616_amd import configs, mone
from tests.gpu_helpers import DeviceProblem, rel_l2

pytestmark = pytest.mark.gpu

SMALL = configs.MoneConfig("inv_bf16", n_layers=3, d_model=128, d_hidden=192, d_kv=64,
                           seg_len=160, n_context=640, act_dtype="bf16", lr=5e-2)
SMALL_F32 = SMALL.with_(name="inv_f32", act_dtype="f32")
# 64-token segments: the forward launches split their contraction over several workgroups
# per tile (2 for Z = X W1^T, 2 for the two-part K2, one split straddling its part boundary)
SHORT_F32 = configs.MoneConfig("inv_short_f32", n_layers=3, d_model=512, d_hidden=384,
                               d_kv=128, seg_len=64, n_context=256, act_dtype="f32", lr=2e-2)


@pytest.fixture(scope="module")
def torch():
    t = pytest.importorskip("torch")
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    mone.lib()
    return t


def _run(cfg, segs, prob=None, lr=None, checked=(0,)):
    cfg = cfg if lr is None else cfg.with_(lr=lr)
    prob = prob or DeviceProblem(cfg, checked)
    w1, w2 = prob.w1.clone(), prob.w2.clone()
    sess = mone.TtlSession(cfg, prob.wkv, w1, w2)
    for x in segs:
        sess.segment(x)
    return sess, w1, w2


@pytest.mark.parametrize("cfg", [SMALL, SMALL_F32], ids=lambda c: c.name)
def test_lr_zero_and_empty_segment_leave_weights_bitwise(torch, cfg):
    print(f"[inv] lr0 {cfg.name}", flush=True)
    prob = DeviceProblem(cfg, [0])
    segs = [prob.segment(s) for s in range(3)]
    sess, w1, w2 = _run(cfg, segs, prob, lr=0.0)
    torch.cuda.synchronize()
    assert torch.equal(w1, prob.w1) and torch.equal(w2, prob.w2)
    sess.close()
    sess, w1, w2 = _run(cfg, [], prob)
    mone.mone_ttl_segment(sess.handle, segs[0], 0)
    torch.cuda.synchronize()
    assert torch.equal(w1, prob.w1) and torch.equal(w2, prob.w2)
    with pytest.raises(mone.MoneError) as e:
        sess.loss()
    assert e.value.code == mone.MONE_ESTATE
    sess.close()


@pytest.mark.parametrize("cfg", [SMALL, SMALL_F32, SHORT_F32], ids=lambda c: c.name)
def test_runs_are_deterministic_and_layers_independent(torch, cfg):
    print(f"[inv] determinism/locality {cfg.name}", flush=True)
    prob = DeviceProblem(cfg, [0])
    segs = [prob.segment(s) for s in range(4)]
    s1, a1, a2 = _run(cfg, segs, prob)
    s2, b1, b2 = _run(cfg, segs, prob)
    pert = [x.clone() for x in segs]
    for x in pert:
        x[1] = x[1] * 0.5 + 0.25
    s3, c1, c2 = _run(cfg, pert, prob)
    torch.cuda.synchronize()
    assert torch.equal(a1, b1) and torch.equal(a2, b2)
    for l in (0, 2):
        assert torch.equal(a1[l], c1[l]) and torch.equal(a2[l], c2[l])
    assert not torch.equal(a1[1], c1[1])
    for s in (s1, s2, s3):
        s.close()


@pytest.mark.parametrize("cfg", [SMALL, SMALL_F32], ids=lambda c: c.name)
def test_read_is_idempotent_and_read_only(torch, cfg):
    print(f"[inv] read {cfg.name}", flush=True)
    prob = DeviceProblem(cfg, [0])
    segs = [prob.segment(s) for s in range(2)]
    sess, w1, w2 = _run(cfg, segs, prob)
    xq, _ = prob.query(q=50)
    kv1 = torch.empty(cfg.n_layers, 50, cfg.d_out, dtype=torch.float32, device="cuda")
    kv2 = torch.empty_like(kv1)
    torch.cuda.synchronize()
    w1c, w2c = w1.clone(), w2.clone()
    sess.memory_kv(xq, kv1)
    sess.memory_kv(xq, kv2)
    torch.cuda.synchronize()
    assert torch.equal(kv1, kv2)
    assert torch.equal(w1, w1c) and torch.equal(w2, w2c)
    # more segments may follow a read (incremental extension) and equal a run without it
    x2 = prob.segment(2)
    sess.segment(x2)
    ref, r1, r2 = _run(cfg, segs + [x2], prob)
    torch.cuda.synchronize()
    assert torch.equal(w1, r1) and torch.equal(w2, r2)
    sess.close()
    ref.close()
    # bf16 output equals the fp32 output rounded to bf16
    kvb = torch.empty(cfg.n_layers, 50, cfg.d_out, dtype=torch.bfloat16, device="cuda")
    sess2, _, _ = _run(cfg, segs, prob)
    sess2.memory_kv(xq, kvb)
    torch.cuda.synchronize()
    assert torch.equal(kvb, kv1.to(torch.bfloat16))
    sess2.close()


@pytest.mark.parametrize("cfg", [SMALL, SMALL_F32], ids=lambda c: c.name)
def test_split_run_equals_one_shot(torch, cfg):
    print(f"[inv] split {cfg.name}", flush=True)
    prob = DeviceProblem(cfg, [0])
    segs = [prob.segment(s) for s in range(5)]
    full, f1, f2 = _run(cfg, segs, prob)
    part, p1, p2 = _run(cfg, segs[:2], prob)
    torch.cuda.synchronize()
    ck1, ck2 = p1.clone(), p2.clone()      # checkpoint = a copy of the fast weights
    part.close()
    resumed = mone.TtlSession(cfg, prob.wkv, ck1, ck2)
    for x in segs[2:]:
        resumed.segment(x)
    torch.cuda.synchronize()
    assert torch.equal(ck1, f1) and torch.equal(ck2, f2)
    full.close()
    resumed.close()


def test_segment_order_matters(torch):
    cfg = SMALL_F32
    prob = DeviceProblem(cfg, [0])
    s0, s1 = prob.segment(0), prob.segment(1)
    a, a1, a2 = _run(cfg, [s0, s1], prob)
    b, b1, b2 = _run(cfg, [s1, s0], prob)
    torch.cuda.synchronize()
    diff = (a2 - b2).norm().item()
    step = (a2 - prob.w2).norm().item()
    assert diff > 1e-3 * step
    a.close()
    b.close()


@pytest.mark.parametrize("cfg", [SMALL, SMALL_F32], ids=lambda c: c.name)
def test_long_query_batch_is_chunked(torch, cfg):
    # q larger than the workspace's row capacity (seg_len rounded up to 256) runs in chunks
    print(f"[inv] long query {cfg.name}", flush=True)
    prob = DeviceProblem(cfg, [0, 2])
    segs = [prob.segment(s) for s in range(2)]
    sess, w1, w2 = _run(cfg, segs, prob, checked=(0, 2))
    q = 600
    xq, hxq = prob.query(q=q)
    kv = torch.empty(cfg.n_layers, q, cfg.d_out, dtype=torch.float32, device="cuda")
    sess.memory_kv(xq, kv)
    torch.cuda.synchronize()
    w1h, w2h, kvh = w1.cpu().numpy(), w2.cpu().numpy(), kv.cpu().numpy()
    bar = 1e-4 if cfg.act_dtype == "f32" else 2e-2
    for l in (0, 2):
        ref = orc.memory_kv(hxq[l], w1h[l], w2h[l])
        assert rel_l2(kvh[l], ref) <= bar
    sess.close()
