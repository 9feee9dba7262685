"""The no-allocation step (mone_ttl_step_noalloc) against the handle path (mone_ttl_init +
mone_ttl_segment) on the same inputs: two calls in a row, the second with fewer tokens, each
compared after the call.  The static workspace keeps the previous call's contents, so the
second call also checks that every call clears what must start at zero."""
import numpy as np
import pytest

from paper_2608_17616_amd import configs, mone
from tests.gpu_helpers import DeviceProblem, rel_l2

pytestmark = pytest.mark.gpu

RAGGED_BF16 = configs.MoneConfig("ragged_bf16", n_layers=3, d_model=192, d_hidden=320, d_kv=64,
                                 seg_len=200, n_context=1000, act_dtype="bf16", lr=2e-2)
CASES = {
    "tiny": (configs.TINY, [128, 77]),
    "ragged_bf16": (RAGGED_BF16, [200, 137]),
    "nip_bf16": (RAGGED_BF16.with_(name="nip_bf16", loss="nip", lr=5e-3), [200, 64]),
}


@pytest.fixture(scope="module")
def torch_cuda():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    mone.lib()
    return torch


@pytest.mark.parametrize("name", list(CASES))
def test_noalloc_step_matches_handle_path(torch_cuda, name):
    torch = torch_cuda
    cfg, ns = CASES[name]
    print(f"[noalloc] case={name} L={cfg.n_layers} d={cfg.d_model} h={cfg.d_hidden} "
          f"D={cfg.d_out} T={cfg.seg_len} tokens={ns} act={cfg.act_dtype}", flush=True)
    assert mone.mone_ttl_workspace_bytes(mone.config_from(cfg)) <= 64 << 20
    prob = DeviceProblem(cfg, [])
    xs = [prob.segment(s, n, record=False) for s, n in enumerate(ns)]
    w1a, w2a = prob.w1.clone(), prob.w2.clone()
    w1b, w2b = prob.w1.clone(), prob.w2.clone()
    sess = mone.TtlSession(cfg, prob.wkv, w1a, w2a)
    c = mone.config_from(cfg)
    bar = 1e-4 if cfg.act_dtype == "f32" else 2e-2
    for i, (x, n) in enumerate(zip(xs, ns)):
        sess.segment(x, n)
        torch.cuda.synchronize()
        free0 = torch.cuda.mem_get_info()[0]
        mone.mone_ttl_step_noalloc(c, prob.wkv, w1b, w2b, x, n)
        torch.cuda.synchronize()
        free1 = torch.cuda.mem_get_info()[0]
        # no device allocation by the call (the static array was loaded with the library's
        # code by the handle path's first launch)
        assert free1 >= free0 - (1 << 20), (free0, free1)
        errs = [rel_l2(w1b.cpu().numpy(), w1a.cpu().numpy()),
                rel_l2(w2b.cpu().numpy(), w2a.cpu().numpy()),
                rel_l2((w1b - prob.w1).cpu().numpy(), (w1a - prob.w1).cpu().numpy()),
                rel_l2((w2b - prob.w2).cpu().numpy(), (w2a - prob.w2).cpu().numpy())]
        same = bool(torch.equal(w1a, w1b) and torch.equal(w2a, w2b))
        print(f"  call {i + 1} (n={n}): W1 {errs[0]:.2e} W2 {errs[1]:.2e} dW1 {errs[2]:.2e} "
              f"dW2 {errs[3]:.2e} bitwise={same}", flush=True)
        assert max(errs) <= bar, errs
        assert bool(torch.isfinite(w1b).all())
    sess.close()
    assert float((w1b - prob.w1).abs().max()) > 0  # the steps did move the weights
