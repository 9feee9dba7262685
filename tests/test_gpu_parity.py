"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on the same seeded inputs.

The GPU always runs every layer of the configuration as one grouped launch per stage, at the
real shape; the oracle recomputes a subset of layers, which is exact because a layer's update
depends on nothing outside it (layer-localised gradients, Sec. 3.4).  Compared per checked
layer: the final fast weights W1_S and W2_S, their change W_S - W_0 (so that a small update
cannot pass on the weights alone), the memory read K/V on a query batch, and the last
segment's loss.

Bars (relative L2 error, per layer and tensor): 1e-4 with fp32 activations, 2e-2 with bf16
activations.  The change of the weights and the read are also held row by row and 64 x 64 tile
by tile, each against its own norm, to 5x the bar, so that one wrong row or one wrong column
chunk of an output tile cannot hide in a whole-tensor norm.

Segments and checked layers follow the parity protocol for the large workloads: 1B-class the
whole context on layers {0, 15}; 3B-class the first 8 segments on layers {0, 13, 27}; 8B-class
the first 4 on {0, 15, 31}; 64-token segments the first 256 on {0, 15}, with the error reported
after 16, 64 and 256 segments; then full-length runs checked on sampled outputs.
"""
import numpy as np
import pytest

import oracle as orc
from paper_2608_17616_amd import configs, mone
from tests.gpu_helpers import LOCAL_FACTOR, DeviceProblem, local_rel_max, rel_l2

pytestmark = pytest.mark.gpu

C = configs.MoneConfig
RAGGED_F32 = C("ragged_f32", n_layers=3, d_model=192, d_hidden=320, d_kv=64, seg_len=200,
               n_context=1000, act_dtype="f32", lr=2e-2)
RAGGED_BF16 = RAGGED_F32.with_(name="ragged_bf16", act_dtype="bf16")
MEAN_F32 = RAGGED_F32.with_(name="mean_f32", loss="mse_mean", lr=1.0)
NIP_F32 = RAGGED_F32.with_(name="nip_f32", loss="nip", lr=5e-3)
NIP_BF16 = NIP_F32.with_(name="nip_bf16", act_dtype="bf16")
# segments of at most 64 tokens in fp32, shaped so that the forward launches and the read's
# first GEMM split their contraction (one split of K2 straddles its two parts)
SHORT_F32 = C("short_f32", n_layers=3, d_model=512, d_hidden=384, d_kv=128, seg_len=64,
              n_context=234, act_dtype="f32", lr=2e-2)

# name -> (config, checked layers, tokens per segment)
CASES = {
    "tiny": (configs.TINY, [0], [128] * 8),
    "ragged_f32": (RAGGED_F32, [0, 2], [200, 137, 64, 1, 200, 77]),
    "ragged_bf16": (RAGGED_BF16, [0, 2], [200, 137, 64, 1, 200, 77]),
    "mean_f32": (MEAN_F32, [1], [200, 150, 200]),
    "nip_f32": (NIP_F32, [0, 2], [200, 137, 64, 1, 200, 77]),
    "nip_bf16": (NIP_BF16, [0, 2], [200, 137, 64, 1, 200, 77]),
    "1b_nip": (configs.ONE_B.with_(name="1b_nip", loss="nip", lr=1e-3), [0, 15], [512] * 4),
    "1b": (configs.ONE_B, [0, 15], [512] * 4),
    "1b_f32": (configs.ONE_B.with_(name="1b_f32", act_dtype="f32"), [0, 15], [512] * 2),
    "3b": (configs.THREE_B, [0, 13, 27], [1024] * 8),
    "8b": (configs.EIGHT_B, [0, 15, 31], [2048] * 4),
    "short_f32": (SHORT_F32, [0, 2], [64, 64, 37, 64, 5]),
    # the longest supported segment, then a ragged one (1024-step weight-gradient contractions)
    "longest_f32": (C("longest_f32", n_layers=2, d_model=64, d_hidden=128, d_kv=64,
                      seg_len=65536, n_context=105536, act_dtype="f32", lr=1e-2), [0, 1],
                    [65536, 40000]),
    # the negative inner product: K2 is the targets alone (one K part), split in two
    "short_nip_f32": (SHORT_F32.with_(name="short_nip_f32", loss="nip", lr=5e-3), [0, 2],
                      [64, 64, 37, 64, 5]),
    # 256 x 256 tiles for FWD1 and BWD (contractions of 2048 tokens or more, 288 tiles) with
    # ragged token extents: partial tiles of the backward's packed SiLU' prefetch
    "big_tile_ragged_bf16": (C("big_tile_ragged_bf16", n_layers=8, d_model=256, d_hidden=1024,
                               d_kv=128, seg_len=2304, n_context=6912, act_dtype="bf16",
                               lr=2e-3), [0, 7], [2304, 2100, 2250]),
    "big_tile_ragged_f32": (C("big_tile_ragged_f32", n_layers=8, d_model=256, d_hidden=1024,
                              d_kv=128, seg_len=2304, n_context=6912, act_dtype="f32",
                              lr=2e-3), [0, 7], [2304, 2100, 2250]),
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


@pytest.mark.parametrize("name", list(CASES))
def test_ttl_and_read_match_oracle(torch_cuda, name):
    torch = torch_cuda
    cfg, checked, ns = CASES[name]
    print(f"[parity] case={name} L={cfg.n_layers} d={cfg.d_model} h={cfg.d_hidden} "
          f"D={cfg.d_out} T={cfg.seg_len} segs={len(ns)} act={cfg.act_dtype}", flush=True)
    prob = DeviceProblem(cfg, checked)
    sess = mone.TtlSession(cfg, prob.wkv, prob.w1, prob.w2)
    for s, n in enumerate(ns):
        sess.segment(prob.segment(s, n), n)
    gpu_loss = sess.loss()
    xq, hxq = prob.query(q=cfg.n_query)
    kv = torch.empty(cfg.n_layers, cfg.n_query, cfg.d_out, dtype=torch.float32, device="cuda")
    sess.memory_kv(xq, kv)
    torch.cuda.synchronize()
    w1 = prob.w1.cpu().numpy()
    w2 = prob.w2.cpu().numpy()
    kvh = kv.cpu().numpy()
    sess.close()

    bar = tol(cfg)
    for l in checked:
        hs = prob.host[l]
        o1, o2, losses = orc.ttl_run(hs["x"], hs["w1"], hs["w2"], hs["wkv"], cfg.lr, cfg.loss)
        e1, e2 = rel_l2(w1[l], o1), rel_l2(w2[l], o2)
        d1 = rel_l2(w1[l] - hs["w1"], o1 - hs["w1"])
        d2 = rel_l2(w2[l] - hs["w2"], o2 - hs["w2"])
        okv = orc.memory_kv(hxq[l], o1, o2)
        ekv = rel_l2(kvh[l], okv)
        eloss = abs(gpu_loss[l] - losses[-1]) / abs(losses[-1])
        loc = max(local_rel_max(w1[l] - hs["w1"], o1 - hs["w1"]),
                  local_rel_max(w2[l] - hs["w2"], o2 - hs["w2"]), local_rel_max(kvh[l], okv))
        print(f"  layer {l}: W1 {e1:.2e} W2 {e2:.2e} dW1 {d1:.2e} dW2 {d2:.2e} KV {ekv:.2e} "
              f"loss {eloss:.2e} local {loc:.2e} "
              f"(|dW1|/|W1| {np.linalg.norm(o1 - hs['w1']) / np.linalg.norm(hs['w1']):.1e})",
              flush=True)
        assert e1 <= bar and e2 <= bar, (e1, e2)
        assert d1 <= bar and d2 <= bar, (d1, d2)
        assert ekv <= bar, ekv
        assert eloss <= bar, eloss
        assert loc <= LOCAL_FACTOR * bar, loc


def test_stress_prefix_error_growth(torch_cuda):
    # 64-token segments: the first 256 of the context on layers {0, 15}; the change of the
    # weights against the oracle after 16, 64 and 256 sequential bf16 steps.
    torch = torch_cuda
    cfg = configs.STRESS
    checked = [0, 15]
    marks = (16, 64, 256)
    print(f"[parity] stress prefix: {marks[-1]} segments of {cfg.seg_len} tokens, "
          f"{cfg.n_layers} layers", flush=True)
    prob = DeviceProblem(cfg, checked)
    sess = mone.TtlSession(cfg, prob.wkv, prob.w1, prob.w2)
    snaps = {}
    for s in range(marks[-1]):
        sess.segment(prob.segment(s))
        if s + 1 in marks:
            torch.cuda.synchronize()
            snaps[s + 1] = {l: (prob.w1[l].cpu().numpy(), prob.w2[l].cpu().numpy())
                            for l in checked}
    sess.close()
    bar = tol(cfg)
    for l in checked:
        hs = prob.host[l]
        w1, w2 = hs["w1"].astype(np.float64), hs["w2"].astype(np.float64)
        done = 0
        for m in marks:
            w1, w2, _ = orc.ttl_run(hs["x"][done:m], w1, w2, hs["wkv"], cfg.lr, cfg.loss)
            done = m
            g1, g2 = snaps[m][l]
            d1 = rel_l2(g1 - hs["w1"], w1 - hs["w1"])
            d2 = rel_l2(g2 - hs["w2"], w2 - hs["w2"])
            loc = max(local_rel_max(g1 - hs["w1"], w1 - hs["w1"]),
                      local_rel_max(g2 - hs["w2"], w2 - hs["w2"]))
            print(f"  layer {l} after {m:4d} segments: dW1 {d1:.2e} dW2 {d2:.2e} "
                  f"W1 {rel_l2(g1, w1):.2e} W2 {rel_l2(g2, w2):.2e} local {loc:.2e}", flush=True)
            assert d1 <= bar and d2 <= bar, (m, d1, d2)
            assert loc <= LOCAL_FACTOR * bar, (m, loc)


# ------------------------------------------------------------------------------------------
# Full-length runs, in the launch configuration the benchmark times (all layers, every segment
# of the context).  The oracle cannot replay a whole 8B-class context, so it checks sampled
# outputs it can compute one by one: the last segment's step from the GPU's own state after
# all earlier segments, and the read of the GPU's final state.

def _full_run_last_step(torch, cfg, checked):
    prob = DeviceProblem(cfg, checked)
    sess = mone.TtlSession(cfg, prob.wkv, prob.w1, prob.w2)
    S = cfg.n_segments
    for s in range(S - 1):
        sess.segment(prob.segment(s, record=False))
        if (s + 1) % 1024 == 0:
            torch.cuda.synchronize()
            print(f"  {s + 1} of {S} segments", flush=True)
    torch.cuda.synchronize()
    before = {l: (prob.w1[l].cpu().numpy(), prob.w2[l].cpu().numpy()) for l in checked}
    sess.segment(prob.segment(S - 1))
    loss = sess.loss()
    xq, hxq = prob.query()
    kv = torch.empty(cfg.n_layers, cfg.n_query, cfg.d_out, dtype=torch.float32, device="cuda")
    sess.memory_kv(xq, kv)
    torch.cuda.synchronize()
    after = {l: (prob.w1[l].cpu().numpy(), prob.w2[l].cpu().numpy()) for l in checked}
    assert bool(torch.isfinite(prob.w1).all()) and bool(torch.isfinite(prob.w2).all())
    kvh = kv.cpu().numpy()
    sess.close()
    bar = tol(cfg)
    for l in checked:
        hs = prob.host[l]
        w1p, w2p = before[l]
        o1, o2, ls = orc.ttl_step(hs["x"][-1], w1p, w2p, hs["wkv"], cfg.lr, cfg.loss)
        d1 = rel_l2(after[l][0] - w1p, o1 - w1p)
        d2 = rel_l2(after[l][1] - w2p, o2 - w2p)
        ekv = rel_l2(kvh[l], orc.memory_kv(hxq[l], after[l][0], after[l][1]))
        eloss = abs(loss[l] - ls) / ls
        loc = max(local_rel_max(after[l][0] - w1p, o1 - w1p),
                  local_rel_max(after[l][1] - w2p, o2 - w2p))
        drift = np.linalg.norm(after[l][0] - hs["w1"]) / np.linalg.norm(hs["w1"])
        print(f"  layer {l}: last-step dW1 {d1:.2e} dW2 {d2:.2e} KV {ekv:.2e} loss {eloss:.2e} "
              f"local {loc:.2e} (|W1_S - W1_0|/|W1_0| {drift:.1e} after {S} segments)",
              flush=True)
        assert d1 <= bar and d2 <= bar and ekv <= bar and eloss <= bar
        assert loc <= LOCAL_FACTOR * bar
    return prob


def test_full_context_8b_last_step_and_read(torch_cuda):
    print("[parity] full 8B-class context: 64 segments, all 32 layers", flush=True)
    _full_run_last_step(torch_cuda, configs.EIGHT_B, [0, 31])


def test_full_context_stress_last_step_read_and_determinism(torch_cuda):
    # all 8192 segments of 64 tokens: the last step against the oracle from the GPU's own state,
    # finite weights, and a second run from the same inputs bitwise equal to the first
    torch = torch_cuda
    cfg = configs.STRESS
    print(f"[parity] full stress context: {cfg.n_segments} segments, all {cfg.n_layers} layers",
          flush=True)
    first = _full_run_last_step(torch, cfg, [0, 15])
    w1a, w2a = first.w1.clone(), first.w2.clone()
    del first
    prob = DeviceProblem(cfg, [0, 15])  # same seeds: the same weights and inputs
    sess = mone.TtlSession(cfg, prob.wkv, prob.w1, prob.w2)
    for s in range(cfg.n_segments):
        sess.segment(prob.segment(s, record=s == cfg.n_segments - 1))
    torch.cuda.synchronize()
    sess.close()
    assert torch.equal(prob.w1, w1a) and torch.equal(prob.w2, w2a)
    print("  second run bitwise equal", flush=True)


def test_full_context_1b_every_segment(torch_cuda):
    # 1B-class: the oracle replays the whole 64-segment context for two layers.
    torch = torch_cuda
    cfg = configs.ONE_B
    print("[parity] full 1B-class context: 64 segments, all 16 layers", flush=True)
    prob = DeviceProblem(cfg, [0, 15])
    sess = mone.TtlSession(cfg, prob.wkv, prob.w1, prob.w2)
    for s in range(cfg.n_segments):
        sess.segment(prob.segment(s))
    torch.cuda.synchronize()
    w1, w2 = prob.w1.cpu().numpy(), prob.w2.cpu().numpy()
    sess.close()
    for l in (0, 15):
        hs = prob.host[l]
        o1, o2, _ = orc.ttl_run(hs["x"], hs["w1"], hs["w2"], hs["wkv"], cfg.lr, cfg.loss)
        errs = (rel_l2(w1[l], o1), rel_l2(w2[l], o2), rel_l2(w1[l] - hs["w1"], o1 - hs["w1"]),
                rel_l2(w2[l] - hs["w2"], o2 - hs["w2"]))
        print(f"  layer {l}: W1 {errs[0]:.2e} W2 {errs[1]:.2e} dW1 {errs[2]:.2e} "
              f"dW2 {errs[3]:.2e}", flush=True)
        assert max(errs) <= tol(cfg)
