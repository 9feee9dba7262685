"""GPU parity of memory injection into attention (mone_memory_attention) against the CPU
oracle: on the GPU's own memory K/V rows (the attention step alone), and end to end from the
oracle's memory state after a few TTL segments.  Bars: 1e-4 (fp32 output), 2e-2 (bf16)."""
import numpy as np
import pytest

import oracle as orc
from paper_2608_17616_amd import configs, mone
from tests.gpu_helpers import DeviceProblem, rel_l2

pytestmark = pytest.mark.gpu

C = configs.MoneConfig
# (config, checked layers, segments, q, n_heads, n_kv_heads)
CASES = {
    "tiny_f32": (configs.TINY.with_(n_layers=2), [0, 1], 2, 37, 4, 2),
    "ragged_bf16": (C("attn_bf16", n_layers=3, d_model=192, d_hidden=320, d_kv=64, seg_len=200,
                      n_context=400, act_dtype="bf16", lr=2e-2), [2], 2, 64, 2, 1),
    "8b_bf16": (configs.EIGHT_B.with_(name="8b_attn", n_layers=2), [1], 1, 64, 32, 8),
    "wide_head_f32": (C("attn_wide", n_layers=1, d_model=128, d_hidden=128, d_kv=256,
                        seg_len=64, n_context=64, act_dtype="f32", lr=1e-2), [0], 1, 9, 3, 1),
}


@pytest.fixture(scope="module")
def torch_cuda():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    mone.lib()
    return torch


@pytest.mark.parametrize("name", list(CASES))
@pytest.mark.parametrize("out_bf16", [False, True], ids=["out_f32", "out_bf16"])
def test_memory_attention_matches_oracle(torch_cuda, name, out_bf16):
    torch = torch_cuda
    cfg, checked, segs, q, hq, hkv = CASES[name]
    print(f"[attn] case={name} q={q} heads={hq}/{hkv} out_bf16={out_bf16}", flush=True)
    prob = DeviceProblem(cfg, checked)
    sess = mone.TtlSession(cfg, prob.wkv, prob.w1, prob.w2)
    for s in range(segs):
        sess.segment(prob.segment(s))
    xq, hxq = prob.query(q=q)
    L, D, dkv = cfg.n_layers, cfg.d_out, cfg.d_kv
    dh = dkv // hkv
    kv = torch.empty(L, q, D, dtype=torch.float32, device="cuda")
    sess.memory_kv(xq, kv)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(7)
    act = prob.act
    qh = torch.randn(L, q, hq * dh, generator=gen, device="cuda").to(act)
    kh = torch.randn(L, q, hkv * dh, generator=gen, device="cuda").to(act)
    vh = torch.randn(L, q, hkv * dh, generator=gen, device="cuda").to(act)
    out = torch.empty(L, q, hq * dh, dtype=torch.bfloat16 if out_bf16 else torch.float32,
                      device="cuda")
    mone.mone_memory_attention(sess.handle, qh, kh, vh, kv, mone.MONE_F32, q, hq, hkv, out,
                               mone.MONE_BF16 if out_bf16 else mone.MONE_F32)
    torch.cuda.synchronize()
    sess.close()
    bar = 2e-2 if out_bf16 else 1e-4
    outh = out.float().cpu().numpy()
    qn, kn, vn, kvn = (t.float().cpu().numpy() for t in (qh, kh, vh, kv))
    for l in range(L):
        e_step = rel_l2(outh[l], orc.memory_attention(qn[l], kn[l], vn[l], kvn[l], hq, hkv))
        msg = f"  layer {l}: attention on the GPU's memory rows {e_step:.2e}"
        assert e_step <= bar, e_step
        if l in checked:
            hs = prob.host[l]
            o1, o2, _ = orc.ttl_run(hs["x"], hs["w1"], hs["w2"], hs["wkv"], cfg.lr, cfg.loss)
            kv_o = orc.memory_kv(hxq[l], o1, o2)
            e_end = rel_l2(outh[l], orc.memory_attention(qn[l], kn[l], vn[l], kv_o, hq, hkv))
            msg += f"; end to end {e_end:.2e}"
            assert e_end <= max(bar, 2e-2 if cfg.act_dtype == "bf16" else 1e-4), e_end
        print(msg, flush=True)


def test_memory_attention_of_no_rows_is_a_no_op(torch_cuda):
    torch = torch_cuda
    cfg = configs.TINY
    prob = DeviceProblem(cfg, [])
    sess = mone.TtlSession(cfg, prob.wkv, prob.w1, prob.w2)
    out = torch.full((1, 4, 128), 3.0, device="cuda")
    mone.mone_memory_attention(sess.handle, out, out, out, out, mone.MONE_F32, 0, 2, 2, out,
                               mone.MONE_F32)
    torch.cuda.synchronize()
    sess.close()
    assert bool((out == 3.0).all())


def test_memory_attention_rejects_bad_arguments(torch_cuda):
    torch = torch_cuda
    cfg = configs.TINY  # d_kv = 128
    prob = DeviceProblem(cfg, [])
    sess = mone.TtlSession(cfg, prob.wkv, prob.w1, prob.w2)
    buf = torch.zeros(1 << 16, device="cuda")
    Lb = mone.lib()
    H = sess.handle
    p = buf.data_ptr()
    bad = [
        (p, p, p, p, 0, -1, 2, 1, p, 0),      # negative q
        (p, p, p, p, 2, 4, 2, 1, p, 0),       # kv dtype
        (p, p, p, p, 0, 4, 2, 1, p, 5),       # out dtype
        (p, p, p, p, 0, 4, 3, 2, p, 0),       # heads not a multiple
        (p, p, p, p, 0, 4, 3, 3, p, 0),       # 3 does not divide d_kv = 128
        (None, p, p, p, 0, 4, 2, 1, p, 0),    # NULL
        (p + 4, p, p, p, 0, 4, 2, 1, p, 0),   # misaligned
    ]
    for args in bad:
        assert Lb.mone_memory_attention(H, *args, None) == mone.MONE_EINVAL, args
    # head width above 256 is outside the kernel's limits
    wide = configs.MoneConfig("w", n_layers=1, d_model=64, d_hidden=64, d_kv=512, seg_len=64,
                              n_context=64, act_dtype="f32", lr=0.0)
    pw = DeviceProblem(wide, [])
    sw = mone.TtlSession(wide, pw.wkv, pw.w1, pw.w2)
    assert Lb.mone_memory_attention(sw.handle, p, p, p, p, 0, 4, 1, 1, p, 0,
                                    None) == mone.MONE_EUNSUPPORTED
    sw.close()
    sess.close()
