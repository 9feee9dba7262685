"""GPU parity of the paper-form memory (SwiGLU per fast-weight head) against the oracle.

Every layer's inputs come from the keyed generator, so the oracle sees the same numbers; the
checked layers are compared element by element through relative L2 errors of the final fast
weights, of their change over the run (W_S - W_0, so a small update cannot pass on the weights
alone) and, with the paper's optimiser, of the momenta, plus the per-layer segment loss.
Bars: 1e-4 in fp32 mode, 2e-2 in bf16 mode.  The loss is a sum of signed terms that can
nearly cancel (rounding the keys, values and weights to bf16 alone moves one such loss by 15%),
so in bf16 mode its bar is absolute, relative to the size of its terms: |L_gpu - L| <=
1e-2 * (1/n) sum |v * y| (elementwise), a few bf16 roundings (2^-9 each) per term.
"""
import numpy as np
import pytest

from paper_2608_17616_amd import configs, inputs, mone
import oracle.swiglu_memory as sw
from gpu_helpers import rel_l2

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _host_layer(cfg, l):
    proj = inputs.sw_layer_proj(cfg, l)
    scale, shift = inputs.sw_layer_affine(cfg, l)
    fast = inputs.sw_layer_fast(cfg, l)
    return proj, scale, shift, fast


class SwProblem:
    """Device state of a paper-form run with every layer drawn from the keyed generator."""

    def __init__(self, cfg):
        self.cfg = cfg
        L, d = cfg.n_layers, cfg.d_model
        self.act = torch.bfloat16 if cfg.act_dtype == "bf16" else torch.float32
        host = [_host_layer(cfg, l) for l in range(L)]
        self.host = host
        dev = "cuda"
        self.proj = torch.from_numpy(np.stack([h[0] for h in host])).to(dev, self.act)
        self.k_scale = torch.from_numpy(np.stack([h[1] for h in host])).to(dev)
        self.k_shift = torch.from_numpy(np.stack([h[2] for h in host])).to(dev)
        self.w = [torch.from_numpy(np.stack([h[3][m] for h in host])).to(dev) for m in range(3)]
        self.w0 = [w.clone() for w in self.w]
        self.opt = None
        if cfg.optimizer == "paper":
            meta = [inputs.layer_meta(cfg, l) for l in range(L)]
            self.meta = [(m[0].astype(np.float64), float(m[1]), m[2].astype(np.float64),
                          float(m[3])) for m in meta]
            u = torch.from_numpy(np.stack([m[0] for m in meta])).to(dev)
            bu = torch.tensor([float(m[1]) for m in meta], dtype=torch.float32, device=dev)
            v = torch.from_numpy(np.stack([m[2] for m in meta])).to(dev)
            bv = torch.tensor([float(m[3]) for m in meta], dtype=torch.float32, device=dev)
            self.mom = [torch.zeros_like(w) for w in self.w]
            self.opt = (u, bu, v, bv, *self.mom)
        self.sess = mone.SwigluSession(cfg, self.proj, self.k_scale, self.k_shift, *self.w,
                                       opt=self.opt)
        self.segs = []

    def segment(self, s, n):
        cfg = self.cfg
        xs = [inputs.segment_x(cfg, l, s, n) for l in range(cfg.n_layers)]
        self.segs.append(xs)
        x = torch.from_numpy(np.stack(xs)).to("cuda", self.act)
        self.sess.segment(x, n)
        return x

    def segments(self, s0, S):
        """Segments s0 .. s0+S-1 (whole) through one mone_swiglu_segments call, the context
        of each layer in one piece [L, S*T, d]."""
        cfg = self.cfg
        T = cfg.seg_len
        xs = [[inputs.segment_x(cfg, l, s0 + s, T) for l in range(cfg.n_layers)]
              for s in range(S)]
        self.segs.extend(xs)
        x = torch.from_numpy(np.stack([np.concatenate([xs[s][l] for s in range(S)])
                                       for l in range(cfg.n_layers)])).to("cuda", self.act)
        self.sess.segments(x)
        return x

    def frozen(self, l):
        proj, scale, shift, _ = self.host[l]
        d = self.cfg.d_model
        return dict(p_k=proj[:d].astype(np.float64), p_v=proj[d:].astype(np.float64),
                    scale=scale.astype(np.float64), shift=shift.astype(np.float64))

    def oracle(self, l, upto=None):
        cfg = self.cfg
        segs = [xs[l].astype(np.float64) for xs in self.segs[:upto]]
        meta = self.meta[l] if cfg.optimizer == "paper" else None
        return sw.swiglu_run(segs, self.host[l][3], self.frozen(l), cfg.lr, cfg.n_heads,
                             cfg.optimizer, meta, cfg.rope_base)

    def loss_scale(self, l):
        """(1/n) sum |v * y| over the last segment at the weights it started from."""
        cfg = self.cfg
        prev, _, _ = self.oracle(l, upto=-1)
        x = self.segs[-1][l].astype(np.float64)
        k, v = sw.layer_keys_values(x, self.frozen(l), cfg.n_heads, base=cfg.rope_base)
        return float(np.sum(np.abs(v * sw.memory_read(k, prev))) / x.shape[0])


def _check(p, layers, tol, loss_tol):
    torch.cuda.synchronize()
    got = [w.cpu().numpy().astype(np.float64) for w in p.w]
    w0 = [w.cpu().numpy().astype(np.float64) for w in p.w0]
    loss = p.sess.loss()
    errs = {}
    for l in layers:
        fast, mom, losses = p.oracle(l)
        for m, name in enumerate(("w_in", "w_gate", "w_out")):
            errs[f"{name}[{l}]"] = rel_l2(got[m][l], fast[m])
            errs[f"d{name}[{l}]"] = rel_l2(got[m][l] - w0[m][l], fast[m] - w0[m][l])
            if mom is not None:
                errs[f"mom_{name}[{l}]"] = rel_l2(p.mom[m][l].cpu().numpy(), mom[m])
        den = abs(losses[-1]) if p.cfg.act_dtype == "f32" else p.loss_scale(l)
        errs[f"loss[{l}]"] = abs(loss[l] - losses[-1]) / max(den, 1e-30)
    print("max errors:", {k: f"{v:.2e}" for k, v in sorted(errs.items(), key=lambda t: -t[1])[:4]})
    bad = {k: v for k, v in errs.items() if v > (loss_tol if k.startswith("loss") else tol)}
    assert not bad, f"{bad} (all: {errs})"
    return errs


@pytest.mark.parametrize("optimizer", ["sgd", "paper"])
def test_tiny_f32_ragged(optimizer):
    cfg = configs.SW_TINY.with_(optimizer=optimizer)
    p = SwProblem(cfg)
    for s, n in enumerate([128, 100, 37]):
        p.segment(s, n)
    _check(p, range(cfg.n_layers), 1e-4, 1e-4)


@pytest.mark.parametrize("optimizer", ["sgd", "paper"])
def test_tiny_bf16(optimizer):
    cfg = configs.SW_TINY.with_(act_dtype="bf16", optimizer=optimizer)
    p = SwProblem(cfg)
    for s, n in enumerate([128, 128, 77]):
        p.segment(s, n)
    _check(p, range(cfg.n_layers), 2e-2, 1e-2)


@pytest.mark.parametrize("optimizer", ["sgd", "paper"])
def test_paper_shape_bf16(optimizer):
    """The paper's shape (24 layers, 4 heads of 224, 512-token segments) on 3 segments, the
    first and last layers checked."""
    cfg = configs.SW_PAPER.with_(optimizer=optimizer)
    p = SwProblem(cfg)
    for s in range(3):
        p.segment(s, cfg.seg_len)
    _check(p, [0, cfg.n_layers - 1], 2e-2, 1e-2)


@pytest.mark.parametrize("d_head,optimizer", [(96, "paper"), (96, "sgd"), (48, "sgd"),
                                              (48, "paper")])
def test_fp32_odd_head_width_and_short_segments(d_head, optimizer):
    """A head width that is not a multiple of 64 (padded contraction) and segments shorter than
    one K step.  With SGD the update's row chunks are split (columns 4q.. and 32+4q..): at 96
    the second half of every last-segment chunk is outside the row, at 48 only that of lanes
    4..7, so a lane pair's exchanged bf16 copy store is masked on one side."""
    n_heads = 192 // d_head
    cfg = configs.SwigluConfig(f"sw_odd{d_head}_{optimizer}", n_layers=1, d_model=192,
                               n_heads=n_heads, d_head=d_head, seg_len=300, n_context=900,
                               act_dtype="f32", lr=2.0, optimizer=optimizer)
    p = SwProblem(cfg)
    for s, n in enumerate([300, 5, 259]):
        p.segment(s, n)
    _check(p, [0], 1e-4, 1e-4)


def test_fp32_longest_segment():
    """The longest supported segment (65536 tokens: RoPE positions up to 65535, 1024-step
    weight-gradient contractions), then a ragged one."""
    cfg = configs.SwigluConfig("sw_long", n_layers=1, d_model=128, n_heads=2, d_head=64,
                               seg_len=65536, n_context=105536, act_dtype="f32", lr=1.0,
                               optimizer="paper")
    p = SwProblem(cfg)
    for s, n in enumerate([65536, 40000]):
        p.segment(s, n)
    _check(p, [0], 1e-4, 1e-4)


def test_empty_segment_is_a_no_op_and_loss_needs_a_segment():
    cfg = configs.SW_TINY
    p = SwProblem(cfg)
    with pytest.raises(mone.MoneError) as ei:
        p.sess.loss()
    assert ei.value.code == mone.MONE_ESTATE
    x = torch.zeros(cfg.n_layers, 1, cfg.d_model, device="cuda")
    p.sess.segment(x, 0)
    torch.cuda.synchronize()
    for w, w0 in zip(p.w, p.w0):
        assert torch.equal(w, w0)


# ---------------------------------------------------------------- the read and attention

def _reader(p, d_kv):
    cfg = p.cfg
    rds = [inputs.sw_layer_reader(cfg, l, d_kv) for l in range(cfg.n_layers)]
    dev = {k: torch.from_numpy(np.stack([r[k] for r in rds])).to("cuda") for k in rds[0]}
    dev["p_q"] = dev["p_q"].to(p.act)
    dev["w_kv"] = dev["w_kv"].to(p.act)
    c = mone.swiglu_reader(dev["p_q"], dev["q_scale"], dev["q_shift"], dev["rms_w"],
                           dev["gate_w"], dev["gate_b"], dev["w_kv"], d_kv)
    return rds, dev, c


@pytest.mark.parametrize("case", ["f32_sgd", "bf16_paper", "paper_shape"])
def test_read_and_attention(case):
    """mone_swiglu_read at the GPU's current weights against the oracle's read on the same
    weights (and, end to end, on the oracle's own weights), then mone_swiglu_attention with
    those memory rows against the attention oracle."""
    import oracle as orc
    if case == "paper_shape":
        cfg, d_kv, q, hq, hkv, layers = configs.SW_PAPER, 128, 64, 14, 2, [0, 23]
    else:
        cfg = configs.SW_TINY.with_(act_dtype="f32" if case == "f32_sgd" else "bf16",
                                    optimizer="sgd" if case == "f32_sgd" else "paper")
        d_kv, q, hq, hkv, layers = 64, 50, 4, 1, [0, 1]
    tol = 1e-4 if cfg.act_dtype == "f32" else 2e-2
    p = SwProblem(cfg)
    for s in range(2):
        p.segment(s, cfg.seg_len)
    rds, dev, crd = _reader(p, d_kv)
    L, d = cfg.n_layers, cfg.d_model
    xq_h = [inputs.query_x(cfg, l, q) for l in range(L)]
    xq = torch.from_numpy(np.stack(xq_h)).to("cuda", p.act)
    kv = torch.empty(L, q, 2 * d_kv, dtype=torch.float32, device="cuda")
    p.sess.read(crd, xq, kv)
    rng = np.random.default_rng(5)
    dh = d_kv // hkv
    att = [rng.standard_normal((L, q, w)).astype(np.float32) for w in (hq * dh, hkv * dh,
                                                                        hkv * dh)]
    qh, kh, vh = (torch.from_numpy(a).to("cuda", p.act) for a in att)
    out = torch.empty(L, q, hq * dh, dtype=torch.float32, device="cuda")
    mone.mone_swiglu_attention(p.sess.handle, d_kv, qh, kh, vh, kv, mone.MONE_F32, q, hq, hkv,
                               out, mone.MONE_F32)
    torch.cuda.synchronize()
    got_w = [w.cpu().numpy().astype(np.float64) for w in p.w]
    kv_h = kv.cpu().numpy().astype(np.float64)
    out_h = out.cpu().numpy().astype(np.float64)
    att_h = [torch.from_numpy(a).to(p.act).float().numpy().astype(np.float64) for a in att]
    errs = {}
    for l in layers:
        fast_gpu = tuple(w[l] for w in got_w)
        h = sw.memory_tokens(xq_h[l], fast_gpu, rds[l], cfg.n_heads, cfg.rope_base)
        want = sw.memory_kv(h, rds[l]["w_kv"])
        errs[f"kv[{l}]"] = rel_l2(kv_h[l], want)
        fast_orc, _, _ = p.oracle(l)
        h2 = sw.memory_tokens(xq_h[l], fast_orc, rds[l], cfg.n_heads, cfg.rope_base)
        errs[f"kv_end_to_end[{l}]"] = rel_l2(kv_h[l], sw.memory_kv(h2, rds[l]["w_kv"]))
        want_out = orc.memory_attention(att_h[0][l], att_h[1][l], att_h[2][l], want, hq, hkv)
        errs[f"attn[{l}]"] = rel_l2(out_h[l], want_out)
    print("max errors:", {k: f"{v:.2e}" for k, v in sorted(errs.items(), key=lambda t: -t[1])[:4]})
    bad = {k: v for k, v in errs.items() if v > tol}
    assert not bad, f"{bad} (all: {errs})"


def test_read_argument_checks():
    cfg = configs.SW_TINY
    p = SwProblem(cfg)
    _, _, crd = _reader(p, 64)
    kv = torch.empty(cfg.n_layers, 4, 128, device="cuda")
    xq = torch.zeros(cfg.n_layers, 4, cfg.d_model, device="cuda")
    with pytest.raises(mone.MoneError) as ei:
        mone.mone_swiglu_read(p.sess.handle, crd, xq, 257, kv, mone.MONE_F32)
    assert ei.value.code == mone.MONE_EUNSUPPORTED  # above seg_len rounded up to 256
    bad = mone.mone_swiglu_reader(crd.proj_q, crd.q_scale, crd.q_shift, crd.rms_w, crd.gate_w,
                                  crd.gate_b, crd.w_kv, 96)
    with pytest.raises(mone.MoneError) as ei:
        mone.mone_swiglu_read(p.sess.handle, bad, xq, 4, kv, mone.MONE_F32)
    assert ei.value.code == mone.MONE_EUNSUPPORTED
    with pytest.raises(mone.MoneError) as ei:
        mone.mone_swiglu_read(p.sess.handle, None, xq, 4, kv, mone.MONE_F32)
    assert ei.value.code == mone.MONE_EINVAL
    mone.mone_swiglu_read(p.sess.handle, crd, None, 0, None, mone.MONE_F32)  # q = 0: no-op


def test_stage_timing_and_mask():
    """Every stage of a step is timed once per segment; with a mask only the masked stage."""
    cfg = configs.SW_TINY.with_(optimizer="paper")
    p = SwProblem(cfg)
    h = p.sess.handle
    mone.mone_swiglu_set_stage_timing(h, 64)
    p.segment(0, cfg.seg_len)
    t = mone.mone_swiglu_stage_times(h)
    for st in ("rate", "proj", "keys", "da", "fwd", "upd"):
        assert t[st][1] == 1 and t[st][0] > 0, (st, t[st])
    assert t["qproj"][1] == 0
    mone.mone_swiglu_set_stage_timing(h, 64, 1 << mone.SW_STAGES.index("upd"))
    p.segment(1, cfg.seg_len)
    p.segment(2, 50)
    t = mone.mone_swiglu_stage_times(h)
    assert t["upd"][1] == 2 and all(v[1] == 0 for k, v in t.items() if k != "upd")
    mone.mone_swiglu_set_stage_timing(h, 0)  # off
    p.segment(3, cfg.seg_len)
    assert all(v[1] == 0 for v in mone.mone_swiglu_stage_times(h).values())


def test_deterministic_and_resumable():
    """Two runs from the same state are bitwise identical, and a run split across handles (a
    checkpoint of the weights and the momenta, resumed by a new handle) equals the one-shot
    run: the renormalisation targets are the resumed weights' row norms, which the
    renormalisation keeps equal to the initial ones (up to its rounding)."""
    cfg = configs.SW_TINY.with_(act_dtype="bf16", optimizer="paper")
    runs = []
    for _ in range(2):
        p = SwProblem(cfg)
        for s in range(4):
            p.segment(s, cfg.seg_len)
        torch.cuda.synchronize()
        runs.append([w.clone() for w in p.w] + [m.clone() for m in p.mom])
    for a, b in zip(*runs):
        assert torch.equal(a, b)
    # split: 2 segments, checkpoint, new handle on the copies, 2 more segments
    p = SwProblem(cfg)
    for s in range(2):
        p.segment(s, cfg.seg_len)
    torch.cuda.synchronize()
    ck_w = [w.clone() for w in p.w]
    ck_m = [m.clone() for m in p.mom]
    p.sess.close()
    opt = p.opt[:4] + tuple(ck_m)
    sess = mone.SwigluSession(cfg, p.proj, p.k_scale, p.k_shift, *ck_w, opt=opt)
    for s in range(2, 4):
        xs = [inputs.segment_x(cfg, l, s) for l in range(cfg.n_layers)]
        sess.segment(torch.from_numpy(np.stack(xs)).to("cuda", p.act))
    torch.cuda.synchronize()
    for got, want in zip(ck_w + ck_m, runs[0]):
        err = float((got - want).norm() / want.norm())
        assert err < 1e-5, err


def test_full_context_paper_shape_last_step():
    """The paper's shape over a whole 128K-token context (256 segments) with the paper's
    optimiser: the last step, from the GPU's own state before it, against the oracle's step on
    that state (first and last layers), and every row norm still at its initial value."""
    cfg = configs.SW_PAPER.with_(optimizer="paper")
    p = SwProblem(cfg)
    L, T, d, H = cfg.n_layers, cfg.seg_len, cfg.d_model, cfg.n_heads
    gen = torch.Generator(device="cuda")
    gen.manual_seed(7)
    x = torch.empty(L, T, d, dtype=p.act, device="cuda")
    for _ in range(cfg.n_segments - 1):
        inputs.device_normal_(x, 1.0, gen)
        p.sess.segment(x, T)
    torch.cuda.synchronize()
    snap_w = [w.cpu().numpy().astype(np.float64) for w in p.w]
    snap_m = [m.cpu().numpy().astype(np.float64) for m in p.mom]
    checked = [0, L - 1]
    inputs.device_normal_(x, 1.0, gen)
    xh = {}
    for l in checked:
        xh[l] = inputs.segment_x(cfg, l, cfg.n_segments - 1)
        x[l].copy_(torch.from_numpy(xh[l]))
    p.sess.segment(x, T)
    torch.cuda.synchronize()
    got_w = [w.cpu().numpy().astype(np.float64) for w in p.w]
    got_m = [m.cpu().numpy().astype(np.float64) for m in p.mom]
    w0 = [w.cpu().numpy().astype(np.float64) for w in p.w0]
    errs = {}
    for l in checked:
        fast = tuple(w[l] for w in snap_w)
        mom = tuple(m[l] for m in snap_m)
        norms0 = sw.initial_norms(tuple(w[l] for w in w0))
        new, new_m, _, _ = sw.paper_step(xh[l].astype(np.float64), fast, mom, p.frozen(l),
                                         p.meta[l], norms0, cfg.lr, H, cfg.rope_base)
        for k, name in enumerate(("w_in", "w_gate", "w_out")):
            errs[f"{name}[{l}]"] = rel_l2(got_w[k][l], new[k])
            errs[f"d{name}[{l}]"] = rel_l2(got_w[k][l] - fast[k], new[k] - fast[k])
            errs[f"mom_{name}[{l}]"] = rel_l2(got_m[k][l], new_m[k])
    print("max errors:", {k: f"{v:.2e}" for k, v in sorted(errs.items(), key=lambda t: -t[1])[:4]})
    assert max(errs.values()) < 2e-2, errs
    for k in range(3):  # row norms over every layer and head after the whole context
        n_end = np.linalg.norm(got_w[k], axis=-1)
        n_0 = np.linalg.norm(w0[k], axis=-1)
        assert np.max(np.abs(n_end - n_0) / n_0) < 1e-4



def test_full_context_one_multi_segment_call():
    """The benchmark's call at the paper's shape: the whole 128K-token context (256 segments)
    through one mone_swiglu_segments call, 32 batches whose preprocessing runs beside the memory
    steps, bitwise equal to one call per segment on the same inputs; the last of those steps
    against the oracle's step from the GPU's own state before it (first and last layers)."""
    cfg = configs.SW_PAPER.with_(optimizer="paper")
    L, T, d, H, S = cfg.n_layers, cfg.seg_len, cfg.d_model, cfg.n_heads, cfg.n_segments
    a, b = SwProblem(cfg), SwProblem(cfg)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(11)
    ctx = inputs.device_normal_(torch.empty(L, S * T, d, dtype=a.act, device="cuda"), 1.0, gen)
    checked = [0, L - 1]
    xh = {}
    for l in checked:  # the last segment of the checked layers from the host generator
        xh[l] = inputs.segment_x(cfg, l, S - 1)
        ctx[l, (S - 1) * T:].copy_(torch.from_numpy(xh[l]))
    print(f"[swiglu] one call of {S} segments", flush=True)
    a.sess.segments(ctx)
    for s in range(S - 1):
        b.sess.segment(ctx[:, s * T:(s + 1) * T].contiguous(), T)
    torch.cuda.synchronize()
    snap_w = [w.cpu().numpy().astype(np.float64) for w in b.w]
    snap_m = [m.cpu().numpy().astype(np.float64) for m in b.mom]
    b.sess.segment(ctx[:, (S - 1) * T:].contiguous(), T)
    torch.cuda.synchronize()
    for m in range(3):
        assert torch.equal(a.w[m], b.w[m]) and torch.equal(a.mom[m], b.mom[m]), m
        assert bool(torch.isfinite(a.w[m]).all())
    assert np.array_equal(a.sess.loss(), b.sess.loss())
    got_w = [w.cpu().numpy().astype(np.float64) for w in a.w]
    got_m = [m.cpu().numpy().astype(np.float64) for m in a.mom]
    w0 = [w.cpu().numpy().astype(np.float64) for w in a.w0]
    errs = {}
    for l in checked:
        fast = tuple(w[l] for w in snap_w)
        mom = tuple(m[l] for m in snap_m)
        norms0 = sw.initial_norms(tuple(w[l] for w in w0))
        new, new_m, _, _ = sw.paper_step(xh[l].astype(np.float64), fast, mom, a.frozen(l),
                                         a.meta[l], norms0, cfg.lr, H, cfg.rope_base)
        for k, name in enumerate(("w_in", "w_gate", "w_out")):
            errs[f"d{name}[{l}]"] = rel_l2(got_w[k][l] - fast[k], new[k] - fast[k])
            errs[f"mom_{name}[{l}]"] = rel_l2(got_m[k][l], new_m[k])
    print("max errors:", {k: f"{v:.2e}" for k, v in sorted(errs.items(), key=lambda t: -t[1])[:4]})
    assert max(errs.values()) < 2e-2, errs

# ------------------------------------------------------------------------------------------
# Several segments per call (mone_swiglu_segments): the weight-independent preprocessing of up
# to prep_segments segments runs as one batch; each segment's memory step follows in order.

@pytest.mark.parametrize("optimizer", ["sgd", "paper"])
def test_segments_tiny_f32(optimizer):
    # 11 segments: a batch of 8 (the default) and one of 3
    cfg = configs.SW_TINY.with_(optimizer=optimizer)
    p = SwProblem(cfg)
    p.segments(0, 11)
    _check(p, range(cfg.n_layers), 1e-4, 1e-4)


def test_segments_tiny_bf16_batches_of_3_then_single_then_batch():
    cfg = configs.SW_TINY.with_(name="sw_tiny_b3", act_dtype="bf16", optimizer="paper",
                                prep_segments=3)
    p = SwProblem(cfg)
    p.segments(0, 5)                 # 3 + 2
    p.segment(5, cfg.seg_len)        # one call per segment in between
    p.segments(6, 3)
    _check(p, range(cfg.n_layers), 2e-2, 1e-2)


def test_segments_odd_head_width_f32():
    cfg = configs.SwigluConfig("sw_odd_seg", n_layers=1, d_model=192, n_heads=2, d_head=96,
                               seg_len=192, n_context=960, act_dtype="f32", lr=2.0,
                               optimizer="paper", prep_segments=2)
    p = SwProblem(cfg)
    p.segments(0, 5)                 # 2 + 2 + 1
    _check(p, [0], 1e-4, 1e-4)


def test_segments_paper_shape_bf16():
    cfg = configs.SW_PAPER.with_(optimizer="paper")
    p = SwProblem(cfg)
    p.segments(0, 10)                # 8 + 2
    _check(p, [0, cfg.n_layers - 1], 2e-2, 1e-2)


@pytest.mark.parametrize("act", ["f32", "bf16"])
def test_segments_bitwise_equal_to_one_call_per_segment(act):
    # the batch computes every token's preprocessing with the same arithmetic as one segment
    cfg = configs.SW_TINY.with_(name=f"sw_tiny_{act}", act_dtype=act, optimizer="paper")
    a, b = SwProblem(cfg), SwProblem(cfg)
    a.segments(0, 6)
    for s in range(6):
        b.segment(s, cfg.seg_len)
    torch.cuda.synchronize()
    for m in range(3):
        assert torch.equal(a.w[m], b.w[m]) and torch.equal(a.mom[m], b.mom[m]), m
    assert np.array_equal(a.sess.loss(), b.sess.loss())


@pytest.mark.parametrize("act,optimizer", [("f32", "paper"), ("bf16", "paper"),
                                           ("bf16", "sgd")])
def test_segments_overlapped_batches_bitwise(act, optimizer):
    # 11 segments in batches of 2: six batches, whose preprocessing runs on the handle's own
    # stream one batch ahead and alternates between two sets of copies; every set is reused
    # while later segments are still queued, so a missing wait would change the result
    cfg = configs.SW_TINY.with_(name=f"sw_tiny_ov_{act}_{optimizer}", act_dtype=act,
                                optimizer=optimizer, prep_segments=2)
    a, b = SwProblem(cfg), SwProblem(cfg)
    a.segments(0, 11)
    for s in range(11):
        b.segment(s, cfg.seg_len)
    torch.cuda.synchronize()
    def same():
        for m in range(3):
            assert torch.equal(a.w[m], b.w[m]), m
            if a.opt is not None:
                assert torch.equal(a.mom[m], b.mom[m]), m
    same()
    assert np.array_equal(a.sess.loss(), b.sess.loss())
    a.segments(11, 3)                # a second call on the same handle: 2 + 1
    for s in range(11, 14):
        b.segment(s, cfg.seg_len)
    torch.cuda.synchronize()
    same()
    _check(a, range(cfg.n_layers), 1e-4 if act == "f32" else 2e-2, 1e-4 if act == "f32" else 1e-2)
