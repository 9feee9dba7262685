"""GPU parity of mone_ttl_segments (several consecutive segments in one call) against the CPU
oracle's sequential run, and against the one-segment-per-call path.

With plain SGD on a squared-error loss and segments of a multiple of 64 tokens up to 256, the
call runs blocks of 512 / T segments in the block form: each segment's step at the block's
starting weights plus the earlier segments' updates, entered through T x T token products
(exact algebra of the sequential chain of Sec. 3.4, summed in another order).  Other settings
run segment by segment.  Bars as everywhere: relative L2 1e-4 (fp32 activations), 2e-2 (bf16),
per layer on W_S, W_S - W_0 and the read; row and 64 x 64 tile errors within 5x the bar.
"""
import numpy as np
import pytest

import oracle as orc
from paper_2608_17616_amd import configs, mone
from tests.gpu_helpers import LOCAL_FACTOR, DeviceProblem, local_rel_max, rel_l2

pytestmark = pytest.mark.gpu

C = configs.MoneConfig
SMALL_BF16 = C("small_bf16", n_layers=3, d_model=192, d_hidden=320, d_kv=64, seg_len=64,
               n_context=64 * 13, act_dtype="bf16", lr=2e-2, block_tokens=512)
# name -> (config, checked layers, segments)
CASES = {
    # T = 128: blocks of 4 segments; 7 segments = a block of 4 and one of 3
    "tiny_f32": (configs.TINY.with_(name="tiny_f32", block_tokens=512), [0], 7),
    # T = 64: blocks of 8; 13 = 8 + 5
    "small_bf16": (SMALL_BF16, [0, 2], 13),
    "small_f32": (SMALL_BF16.with_(name="small_f32", act_dtype="f32"), [0, 2], 13),
    "small_mean_f32": (SMALL_BF16.with_(name="small_mean_f32", act_dtype="f32",
                                        loss="mse_mean", lr=1.0), [1], 9),
    # T = 64 in blocks of 4 (256 tokens)
    "small_b4_bf16": (SMALL_BF16.with_(name="small_b4_bf16", block_tokens=256), [1], 10),
    # T = 192: blocks of 2 (384 tokens); 5 = 2 + 2 + 1 (the last one alone)
    "t192_f32": (C("t192_f32", n_layers=2, d_model=256, d_hidden=384, d_kv=128, seg_len=192,
                   n_context=960, act_dtype="f32", lr=1e-2, block_tokens=384), [0, 1], 5),
    # T = 256 in blocks of 4 (1024 tokens, the library's default size there); 9 = 4 + 4 + 1
    "t256_bf16": (C("t256_bf16", n_layers=2, d_model=256, d_hidden=512, d_kv=128, seg_len=256,
                    n_context=2304, act_dtype="bf16", lr=1e-2, block_tokens=1024), [0, 1], 9),
    # T = 128 in blocks of 8 (1024 tokens, the default size there); 10 = 8 + 2
    "t128_f32": (C("t128_f32", n_layers=2, d_model=256, d_hidden=384, d_kv=64, seg_len=128,
                   n_context=1280, act_dtype="f32", lr=1e-2, block_tokens=1024), [0, 1], 10),
    # T = 512 in blocks of 2 (1024 tokens)
    "t512_bf16": (C("t512_bf16", n_layers=2, d_model=256, d_hidden=512, d_kv=128, seg_len=512,
                    n_context=2560, act_dtype="bf16", lr=1e-2, block_tokens=1024), [1], 5),
    # not in the block form: segment by segment
    "nip_bf16": (SMALL_BF16.with_(name="nip_bf16", loss="nip", lr=5e-3, block_tokens=0),
                 [0, 2], 10),
    "t100_bf16": (SMALL_BF16.with_(name="t100_bf16", seg_len=100, n_context=1000,
                                   block_tokens=0), [0], 6),
    "small_none_bf16": (SMALL_BF16.with_(name="small_none_bf16", block_tokens=-1), [0], 9),
    # the 64-token workload: 16 layers, 2048 -> 2048 -> 1024; 64 segments = 8 blocks of 512
    # tokens (the library's choice for it)
    "stress": (configs.STRESS, [0, 15], 64),
}


def tol(cfg):
    return 1e-4 if cfg.act_dtype == "f32" else 2e-2


@pytest.fixture(scope="module")
def torch_cuda():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    mone.lib()
    return torch


def _context(torch, prob, S):
    """Segments 0..S-1 as one [L, S*T, d] tensor (each layer's part of the context in one
    piece), recording the checked layers' host copies."""
    cfg = prob.cfg
    T = cfg.seg_len
    x = torch.empty(cfg.n_layers, S * T, cfg.d_model, dtype=prob.act, device="cuda")
    for s in range(S):
        x[:, s * T:(s + 1) * T] = prob.segment(s)
    return x


@pytest.mark.parametrize("name", list(CASES))
def test_segments_match_oracle(torch_cuda, name):
    torch = torch_cuda
    cfg, checked, S = CASES[name]
    print(f"[segments] case={name} L={cfg.n_layers} d={cfg.d_model} h={cfg.d_hidden} "
          f"D={cfg.d_out} T={cfg.seg_len} S={S} act={cfg.act_dtype} loss={cfg.loss}", flush=True)
    prob = DeviceProblem(cfg, checked)
    x = _context(torch, prob, S)
    sess = mone.TtlSession(cfg, prob.wkv, prob.w1, prob.w2)
    sess.segments(x)
    loss = sess.loss()
    xq, hxq = prob.query()
    kv = torch.empty(cfg.n_layers, cfg.n_query, cfg.d_out, dtype=torch.float32, device="cuda")
    sess.memory_kv(xq, kv)
    torch.cuda.synchronize()
    w1, w2, kvh = prob.w1.cpu().numpy(), prob.w2.cpu().numpy(), kv.cpu().numpy()
    assert np.isfinite(w1).all() and np.isfinite(w2).all()
    sess.close()
    bar = tol(cfg)
    for l in checked:
        hs = prob.host[l]
        o1, o2, losses = orc.ttl_run(hs["x"], hs["w1"], hs["w2"], hs["wkv"], cfg.lr, cfg.loss)
        okv = orc.memory_kv(hxq[l], o1, o2)
        errs = dict(W1=rel_l2(w1[l], o1), W2=rel_l2(w2[l], o2),
                    dW1=rel_l2(w1[l] - hs["w1"], o1 - hs["w1"]),
                    dW2=rel_l2(w2[l] - hs["w2"], o2 - hs["w2"]), KV=rel_l2(kvh[l], okv),
                    loss=abs(loss[l] - losses[-1]) / abs(losses[-1]))
        loc = max(local_rel_max(w1[l] - hs["w1"], o1 - hs["w1"]),
                  local_rel_max(w2[l] - hs["w2"], o2 - hs["w2"]), local_rel_max(kvh[l], okv))
        print(f"  layer {l}: " + " ".join(f"{k} {v:.2e}" for k, v in errs.items()) +
              f" local {loc:.2e}", flush=True)
        assert max(errs.values()) <= bar, errs
        assert loc <= LOCAL_FACTOR * bar, loc


def test_segments_continue_the_chain_across_calls(torch_cuda):
    # segments, then one segment alone, then segments again: one chain, equal to the oracle
    torch = torch_cuda
    cfg = SMALL_BF16
    prob = DeviceProblem(cfg, [1])
    x1 = _context(torch, prob, 11)       # a block of 8 and one of 3
    x2 = prob.segment(11)                # one segment alone
    x3 = torch.empty(cfg.n_layers, 9 * cfg.seg_len, cfg.d_model, dtype=prob.act, device="cuda")
    for s in range(9):
        x3[:, s * cfg.seg_len:(s + 1) * cfg.seg_len] = prob.segment(12 + s)
    sess = mone.TtlSession(cfg, prob.wkv, prob.w1, prob.w2)
    sess.segments(x1)
    sess.segment(x2)
    sess.segments(x3[:, :4 * cfg.seg_len], 4)  # a view: layer stride of the whole tensor
    sess.segments(x3[:, 4 * cfg.seg_len:], 5)
    torch.cuda.synchronize()
    w1, w2 = prob.w1[1].cpu().numpy(), prob.w2[1].cpu().numpy()
    sess.close()
    hs = prob.host[1]
    o1, o2, _ = orc.ttl_run(hs["x"], hs["w1"], hs["w2"], hs["wkv"], cfg.lr, cfg.loss)
    d1 = rel_l2(w1 - hs["w1"], o1 - hs["w1"])
    d2 = rel_l2(w2 - hs["w2"], o2 - hs["w2"])
    print(f"  21 segments over four calls: dW1 {d1:.2e} dW2 {d2:.2e}", flush=True)
    assert d1 <= tol(cfg) and d2 <= tol(cfg)


def test_segments_argument_checks(torch_cuda):
    torch = torch_cuda
    cfg = SMALL_BF16
    prob = DeviceProblem(cfg, [])
    sess = mone.TtlSession(cfg, prob.wkv, prob.w1, prob.w2)
    x = torch.zeros(cfg.n_layers, 2 * cfg.seg_len, cfg.d_model, dtype=prob.act, device="cuda")
    before = prob.w1.clone()
    mone.mone_ttl_segments(sess.handle, x, x.stride(0), 0)  # no segments: nothing happens
    with pytest.raises(mone.MoneError):
        mone.mone_ttl_segments(sess.handle, x, x.stride(0) - 1, 2)  # layer stride too small
    with pytest.raises(mone.MoneError):
        mone.mone_ttl_segments(sess.handle, x, x.stride(0), -1)
    with pytest.raises(mone.MoneError):
        mone.mone_ttl_segments(sess.handle, None, x.stride(0), 1)
    torch.cuda.synchronize()
    assert torch.equal(before, prob.w1)
    sess.close()


def test_full_stress_context_block_form_against_per_segment_path(torch_cuda):
    # all 8192 segments of 64 tokens at the real shape: the block form against the
    # one-segment-per-call path from the same inputs (both checked against the oracle on
    # prefixes above), and bitwise repeatable
    torch = torch_cuda
    cfg = configs.STRESS
    S, T, L = cfg.n_segments, cfg.seg_len, cfg.n_layers
    print(f"[segments] full stress context: {S} segments, {L} layers", flush=True)
    chunk = 1024  # segments per call (each layer's slice in one piece)
    prob = DeviceProblem(cfg, [])
    w1_0, w2_0 = prob.w1.clone(), prob.w2.clone()
    gen = torch.Generator(device="cuda")

    def draw(c):
        gen.manual_seed(4321 + c)
        x = torch.empty(L, chunk * T, cfg.d_model, dtype=torch.float32, device="cuda")
        x.normal_(generator=gen)
        return x.to(prob.act)

    def run(block):
        prob.w1.copy_(w1_0)
        prob.w2.copy_(w2_0)
        sess = mone.TtlSession(cfg, prob.wkv, prob.w1, prob.w2)
        for c in range(S // chunk):
            x = draw(c)
            if block:
                sess.segments(x)
            else:
                for s in range(chunk):
                    sess.segment(x[:, s * T:(s + 1) * T].contiguous())
            torch.cuda.synchronize()
            print(f"  {'block form' if block else 'per segment'}: {(c + 1) * chunk} of {S}",
                  flush=True)
        sess.close()
        return prob.w1.clone(), prob.w2.clone()

    b1, b2 = run(True)
    assert bool(torch.isfinite(b1).all()) and bool(torch.isfinite(b2).all())
    p1, p2 = run(False)
    r1, r2 = run(True)
    assert torch.equal(b1, r1) and torch.equal(b2, r2)
    bar = tol(cfg)
    for l in (0, L - 1):
        w10, w20 = w1_0[l].cpu().numpy(), w2_0[l].cpu().numpy()
        e = (rel_l2(b1[l].cpu().numpy() - w10, p1[l].cpu().numpy() - w10),
             rel_l2(b2[l].cpu().numpy() - w20, p2[l].cpu().numpy() - w20))
        drift = float(np.linalg.norm(b1[l].cpu().numpy() - w10) / np.linalg.norm(w10))
        print(f"  layer {l}: block form vs per segment: dW1 {e[0]:.2e} dW2 {e[1]:.2e} "
              f"(|W1_S - W1_0|/|W1_0| {drift:.1e}); repeat bitwise equal", flush=True)
        assert max(e) <= bar
