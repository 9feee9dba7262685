#!/usr/bin/env python3
"""Throughput of the MoNe test-time-learning hot path on one MI355X.

One step = the whole hot path over one synthetic context: every segment of the context goes
through one mone_ttl_segments call (all layers, grouped launches; short segments in the block
form, the others one by one; --call segment issues one call per segment), then mone_memory_kv
reads the final state on a query batch.  The default workload is the 8B-class shape: 32 layers, d = h = 4096,
D = 2048 (8 KV heads x 128 for K and for V), T = 2048, N = 131072 context tokens
(64 segments), Q = 64 query tokens, bf16 activations, fp32 fast weights, lr 1e-3.

The context is resident in HBM before timing starts (64 distinct segments, 32 GiB).  Inputs
are seeded synthetic Gaussians: x ~ N(0, 1), W_k, W_v, W1 ~ N(0, 1/d), W2 ~ N(0, 1/h), drawn
on the GPU with torch's generator.

Prints one JSON line.  Kernel durations come from HIP events the library records on the launch
stream: around every stage during one untimed profiling step after the warmup ("stages"), and
around the dominant stage only during the timed steps ("roofline"), so that event records between
the other kernels do not slow the timed work.  The CPU baseline times the CPU
oracle (float64 NumPy, as it stands) on one layer over as many segments as fit in about
--cpu-seconds, scaled to all layers.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "context tokens/sec of test-time learning (all layers); % bf16 MFMA peak"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3     # MI355X dense fp32 matrix
PEAK_HBM_GBS = 8000.0


def block_segments(cfg):
    """Segments per block of mone_ttl_segments' block form for this configuration (1: the
    segments run one by one), by the rule the library's header states."""
    T = cfg.seg_len
    if cfg.block_tokens < 0 or not (cfg.optimizer == "sgd" and cfg.loss in ("mse_sum", "mse_mean")
                                    and T % 64 == 0):
        return 1
    if cfg.block_tokens > 0:
        return cfg.block_tokens // T
    weights = cfg.n_layers * cfg.d_hidden * (cfg.d_model + cfg.d_out)
    return min(8, 1024 // T) if T <= 256 and weights >= 1 << 24 else 1


def stage_work(cfg, q, blk=1, per_call=1):
    """Algorithmic FLOPs and bytes of one launch of each stage (all layers).  With the block
    form (blk segments per block) the staging and the block stages cover a block of blk*T
    tokens, and BSEQ one segment (its corrections averaged over the block).  With the paper's
    optimiser and per_call segments per call, the renormalisation pass runs once per call (the
    other segments' updates write the weight copies instead); the figures are averages per
    launch."""
    L, d, h, D, T = cfg.n_layers, cfg.d_model, cfg.d_hidden, cfg.d_out, cfg.seg_len
    E = 2 if cfg.act_dtype == "bf16" else 4
    hkv = max(1, cfg.d_kv // 128)
    hq, dh = 4 * hkv, cfg.d_kv // hkv
    # causal scores and weighted sums over q query keys and q memory keys per query row
    attn = (L * hq * 2 * (q * (q + 1)) * 2 * dh,
            L * q * ((hq + 2 * hkv) * dh * E + D * 4 + hq * dh * 4))
    if blk > 1:
        bt = blk * T
        kp = T * (blk - 1) / 2  # earlier segments' tokens, averaged over the block
        return {
            "xt": (0, L * bt * d * E * 2),
            "bfwd": (L * (2 * bt * d * (h + D) + 2 * bt * bt * d),
                     L * (E * (bt * d + h * d + D * d + bt * bt) + 4 * bt * (h + D))),
            "bseq": (L * (4 * T * h * D + 2 * T * kp * (3 * h + 2 * D)),
                     L * (2 * D * h * E + T * (8 * h + 8 * D + E * (5 * h + 3 * D)))),
            "bupd": (L * 2 * bt * (D * h + h * d),
                     L * (8 * (D * h + h * d) + E * (2 * D * h + h * d)
                          + E * bt * (D + 2 * h + d))),
            "kv1": (L * 2 * q * d * h, L * (q * d + h * d + q * h) * E),
            "kv2": (L * 2 * q * h * D, L * (q * h + D * h) * E + L * q * D * 4),
            "attn": attn,
        }
    if cfg.optimizer == "paper":
        # momentum read-modify-write in the update epilogues; the copies move to RENORM, except
        # between the segments of one call (written by the updates, renormalised once per call)
        cp1 = E if cfg.act_dtype == "bf16" else 0
        defer = (per_call - 1) / per_call
        return {
            "xt": (0, L * T * d * E * 2),
            "rate": (L * 4 * T * d, L * (T * d * E + 2 * d * 4 + T * 4)),
            "fwd1": (L * 2 * T * d * h, L * (T * d + h * d + T * h * 3) * E),
            "fwd2": (L * 2 * T * D * (h + d), L * ((T * h + D * h + T * d + D * d + 2 * T * D) * E
                                                   + T * 4)),
            "bwd": (L * (2 * T * D * h + 2 * T * D * h),
                    L * ((T * D + h * D + 2 * T * h + D * T + h * T) * E
                         + D * h * (16 + 2 * E * defer))),
            "upd": (L * 2 * T * h * d, L * ((h * T + d * T) * E + h * d * (16 + cp1 * defer))),
            # every segment: the row scales from the row-segment sums of squares; once per
            # call: the rescaled masters and their copies
            "renorm": (0, L * (4 * (h * d + D * h) // 64
                               + (h * d * (8 + cp1) + D * h * (8 + 2 * E)) * (1 - defer))),
            "kv1": (L * 2 * q * d * h, L * (q * d + h * d + q * h) * E),
            "kv2": (L * 2 * q * h * D, L * (q * h + D * h) * E + L * q * D * 4),
            "attn": attn,
        }
    fwd2 = (L * 2 * T * D * (h + d), L * (T * h + D * h + T * d + D * d + 2 * T * D) * E)
    if cfg.loss == "nip":  # the targets alone
        fwd2 = (L * 2 * T * D * d, L * (T * d + D * d + 2 * T * D) * E)
    return {
        "xt": (0, L * T * d * E * 2),
        "fwd1": (L * 2 * T * d * h, L * (T * d + h * d + T * h * 3) * E),
        "fwd2": fwd2,
        # backward (G W2 -> dZ^T) and the W2 update (G^T A) share one launch
        "bwd": (L * (2 * T * D * h + 2 * T * D * h),
                L * ((T * D + h * D + 2 * T * h + D * T + h * T) * E + D * h * 8)),
        # W1 update (dZ^T X)
        "upd": (L * 2 * T * h * d, L * ((h * T + d * T) * E + h * d * 8)),
        "kv1": (L * 2 * q * d * h, L * (q * d + h * d + q * h) * E),
        "kv2": (L * 2 * q * h * D, L * (q * h + D * h) * E + L * q * D * 4),
        "attn": attn,
    }


def counted_traffic(stage, record="hbm_traffic_8b.json"):
    """Per-launch HBM bytes of `stage` from a committed counter summary under profiles/, or
    None when the kernel sources have changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", record)
    try:
        with open(path) as f:
            rec = json.load(f)
        h = hashlib.sha256()
        for src in rec["sources"]:
            with open(os.path.join(ROOT, src), "rb") as f:
                h.update(f.read())
        if h.hexdigest() != rec["source_sha256"] or stage not in rec["per_launch"]:
            return None
        t = rec["per_launch"][stage]
        return {"read_bytes": round(t["fetch_bytes"]), "write_bytes": round(t["write_bytes"])}
    except (OSError, KeyError, ValueError):
        return None


class _HostThreads:
    """The oracle's BLAS thread count for the CPU baseline: the host's share of cores for this
    job (the affinity mask, capped by OMP_NUM_THREADS), set for the duration of the block."""

    def __enter__(self):
        self.affinity = len(os.sched_getaffinity(0))
        env = os.environ.get("OMP_NUM_THREADS", "")
        self.cores = min(self.affinity, int(env)) if env.isdigit() and int(env) > 0 \
            else self.affinity
        try:
            from threadpoolctl import threadpool_limits
            self._lim = threadpool_limits(limits=self.cores, user_api="blas")
        except Exception:  # pragma: no cover
            self._lim = None
        return self

    def __exit__(self, *exc):
        if self._lim is not None:
            self._lim.restore_original_limits()
        return False

    def record(self, value, t, done, cfg):
        return {"value": value, "unit": "tokens/s", "cores": int(self.cores), "kind": "oracle",
                "sample": f"layer 0, {done} consecutive segments of T={cfg.seg_len} tokens "
                          f"({t:.1f} s, float64 NumPy), scaled to {cfg.n_layers} layers",
                "affinity_cores": int(self.affinity), "cpu_model": _cpu_model()}


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(cfg, w1, w2, wkv, xs, budget_s, meta=None):
    import numpy as np

    import oracle as orc
    with _HostThreads() as ht:
        w1 = np.asarray(w1, np.float64)
        w2 = np.asarray(w2, np.float64)
        if meta is not None:
            norms0 = (orc.row_norms(w1), orc.row_norms(w2))
            m1, m2 = np.zeros_like(w1), np.zeros_like(w2)
        done, t0 = 0, time.perf_counter()
        while True:
            x = xs[done % len(xs)]
            if meta is None:
                w1, w2, _ = orc.ttl_step(x, w1, w2, wkv, cfg.lr, cfg.loss)
            else:
                w1, w2, m1, m2, _, _ = orc.paper_step(x, w1, w2, m1, m2, wkv, meta, norms0,
                                                      cfg.lr, cfg.loss)
            done += 1
            if time.perf_counter() - t0 >= budget_s or done >= 64:
                break
        t = time.perf_counter() - t0
        return ht.record(done * cfg.seg_len / t / cfg.n_layers, t, done, cfg)


def sw_stage_work(cfg, prep=1):
    """Algorithmic FLOPs and bytes of one launch of each stage of the paper-form memory (all
    layers and heads; B = L H head problems of d_h x d_h; T tokens).  RATE, PROJ and KEYS
    launches cover `prep` segments at a time."""
    L, d, H, dh, T = cfg.n_layers, cfg.d_model, cfg.n_heads, cfg.d_head, cfg.seg_len
    g = prep
    E = 2 if cfg.act_dtype == "bf16" else 4
    B = L * H
    paper = cfg.optimizer == "paper"
    # the three masters are read and written in fp32 and their MFMA copies written (+ the
    # momentum's read and write with the paper's optimiser, whose row renormalisation happens
    # in the same epilogue)
    upd_w = 3 * dh * dh * (8 + E + (8 if paper else 0))
    return {
        "rate": (g * L * 4 * T * d, g * L * (T * d * E + 2 * d * 4 + T * 4)),
        # the projections with the elementwise preprocessing fused: X and P in; K', dY0 and
        # dY^T out
        "proj": (g * L * 2 * T * 2 * d * d, L * (4 * g * T * d + 2 * d * d) * E),
        # K' in; K and K^T out
        "keys": (0, 3 * g * L * T * d * E),
        "da": (B * 2 * T * dh * dh, B * (dh * dh + 2 * T * dh) * E),
        "fwd": (B * 2 * T * 2 * dh * dh, B * (2 * dh * dh + 5 * T * dh) * E + L * T * 4),
        "upd": (B * 2 * T * 3 * dh * dh, B * (5 * dh * T * E + upd_w)),
    }


def sw_read_work(cfg, q, d_kv, hq, hkv):
    """Algorithmic FLOPs and bytes of the read's stages (all layers and heads; q query tokens;
    attention with hq query heads and hkv key/value heads of width d_kv / hkv)."""
    L, d, H, dh = cfg.n_layers, cfg.d_model, cfg.n_heads, cfg.d_head
    E = 2 if cfg.act_dtype == "bf16" else 4
    B, D, ah = L * H, 2 * d_kv, d_kv // hkv
    return {
        "qproj": (L * 2 * q * d * (d + H), L * ((2 * q * d + d * d) * E + H * d * 4)),
        "qkeys": (0, 3 * L * q * d * E),
        "qfwd": (B * 2 * q * 2 * dh * dh, B * (2 * q * dh + 2 * dh * dh) * E),
        "qout": (B * 2 * q * dh * dh, B * (2 * q * dh + dh * dh) * E + B * dh * dh * 4),
        "qkv": (L * 2 * q * d * D, L * ((q * d + D * d) * E + q * D * 4)),
        "attn": (L * hq * 2 * (q * (q + 1)) * 2 * ah,
                 L * q * ((hq + 2 * hkv) * ah * E + D * 4 + hq * ah * 4)),
    }


def roofline(kernel, flops, nbytes, seconds, peak_tflops):
    """Roofline entry of one launch: the bound is the resource nearest its peak (MFMA for a
    contraction that keeps the matrix cores busy, HBM for one whose epilogue traffic dominates)."""
    tf = flops / seconds / 1e12
    gb = nbytes / seconds / 1e9
    if flops > 0 and tf / peak_tflops >= gb / PEAK_HBM_GBS:
        return {"kernel": kernel, "bound": "mfma", "achieved": round(tf, 1), "peak": peak_tflops,
                "unit": "TFLOP/s", "frac": round(tf / peak_tflops, 4), "traffic": None}
    return {"kernel": kernel, "bound": "hbm", "achieved": round(gb, 1), "peak": PEAK_HBM_GBS,
            "unit": "GB/s", "frac": round(gb / PEAK_HBM_GBS, 4), "traffic": None}


def timed_steps(step, steps, set_timing, stage_times, names, records_per_step):
    """Run one profiling step with every stage bracketed by HIP events (the per-stage breakdown
    and the dominant stage), then time exactly `steps` steps with events around the dominant
    stage only, so that event records between the other kernels do not slow the timed work.
    Returns (elapsed seconds of the timed steps, per-stage (ms, launches) of the profiling step,
    dominant stage, its (ms, launches) over the timed steps)."""
    import torch
    set_timing(records_per_step, 0xFFFFFFFF)
    step()
    torch.cuda.synchronize()
    prof = stage_times()
    dom = max((n for n in prof if prof[n][1]), key=lambda n: prof[n][0])
    set_timing(steps * records_per_step, 1 << names.index(dom))
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    return elapsed, prof, dom, stage_times()[dom]


def stage_table(stimes, work):
    """Per-stage average launch time and algorithmic rates."""
    stages = {}
    for name, (ms, cnt) in stimes.items():
        if cnt == 0:
            continue
        fl, by = work[name]
        avg_s = ms / cnt / 1e3
        stages[name] = {"launches": cnt, "avg_ms": round(ms / cnt, 4),
                        "tflops": round(fl / avg_s / 1e12, 1),
                        "gbs": round(by / avg_s / 1e9, 1)}
    return stages


def sw_cpu_baseline(cfg, host, xs, budget_s, meta):
    import numpy as np

    import oracle.swiglu_memory as sw
    with _HostThreads() as ht:
        proj, scale, shift, fast = host
        d = cfg.d_model
        frozen = dict(p_k=proj[:d], p_v=proj[d:], scale=scale, shift=shift)
        fast = tuple(np.asarray(w, np.float64) for w in fast)
        if meta is not None:
            norms0 = sw.initial_norms(fast)
            mom = tuple(np.zeros_like(w) for w in fast)
        done, t0 = 0, time.perf_counter()
        while True:
            x = xs[done % len(xs)]
            if meta is None:
                fast, _ = sw.sgd_step(x, fast, frozen, cfg.lr, cfg.n_heads, cfg.rope_base)
            else:
                fast, mom, _, _ = sw.paper_step(x, fast, mom, frozen, meta, norms0, cfg.lr,
                                                cfg.n_heads, cfg.rope_base)
            done += 1
            if time.perf_counter() - t0 >= budget_s or done >= 256:
                break
        t = time.perf_counter() - t0
        return ht.record(done * cfg.seg_len / t / cfg.n_layers, t, done, cfg)


def run_swiglu(args):
    """The paper-form memory (SwiGLU per fast-weight head) at the paper's shape: one step is
    every segment of the context through one mone_swiglu_segments call (all layers and heads;
    --call segment: one call per segment)."""
    import numpy as np
    import torch

    from paper_2608_17616_amd import configs, inputs, mone

    cfg = configs.SW_CONFIGS[args.config if args.config in configs.SW_CONFIGS
                             else "sw_qwen0.5b"].with_(optimizer=args.optimizer,
                                                       prep_segments=args.prep_segments)
    L, d, H, dh, T = cfg.n_layers, cfg.d_model, cfg.n_heads, cfg.d_head, cfg.seg_len
    S = args.segments or cfg.n_segments
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    act = torch.bfloat16 if cfg.act_dtype == "bf16" else torch.float32
    gen = torch.Generator(device=dev)
    gen.manual_seed(cfg.seed)
    f32 = torch.float32
    proj = inputs.device_normal_(torch.empty(L, 2 * d, d, dtype=act, device=dev),
                                 1 / np.sqrt(d), gen)
    k_scale = inputs.device_normal_(torch.empty(L, d, dtype=f32, device=dev), 0.1, gen) + 1.0
    k_shift = inputs.device_normal_(torch.empty(L, d, dtype=f32, device=dev), 0.1, gen)
    w = [inputs.device_normal_(torch.empty(L, H, dh, dh, dtype=f32, device=dev),
                               1 / np.sqrt(dh), gen) for _ in range(3)]
    # each layer's part of the context in one piece: token t of segment s at ctx[l, s*T + t]
    ctx = torch.empty(L, S * T, d, dtype=act, device=dev)
    for s in range(S):
        inputs.device_normal_(ctx[:, s * T:(s + 1) * T], 1.0, gen)
    opt = None
    if cfg.optimizer == "paper":
        opt = (inputs.device_normal_(torch.empty(L, d, dtype=f32, device=dev), 1 / np.sqrt(d),
                                     gen),
               torch.full((L,), inputs.B_U, dtype=f32, device=dev),
               inputs.device_normal_(torch.empty(L, d, dtype=f32, device=dev), 1 / np.sqrt(d),
                                     gen),
               torch.full((L,), inputs.B_V, dtype=f32, device=dev),
               *(torch.zeros_like(t) for t in w))
    n_cpu = 0 if args.no_cpu_baseline else min(S, 4)
    cpu_in = None
    if n_cpu:
        host = (proj[0].double().cpu().numpy(), k_scale[0].double().cpu().numpy(),
                k_shift[0].double().cpu().numpy(), tuple(t[0].double().cpu().numpy() for t in w))
        cpu_in = (host, [ctx[0, s * T:(s + 1) * T].double().cpu().numpy()
                         for s in range(n_cpu)])

    # the read: Q query tokens through the memory (Qwen2.5-0.5B's attention: 14 query heads and
    # 2 key/value heads of 64, d_kv = 128), then the memory-injected attention
    Q, d_kv, hq, hkv = cfg.n_query, 128, 14, 2
    ah = d_kv // hkv
    xq = inputs.device_normal_(torch.empty(L, Q, d, dtype=act, device=dev), 1.0, gen)
    rd = dict(p_q=inputs.device_normal_(torch.empty(L, d, d, dtype=act, device=dev),
                                        1 / np.sqrt(d), gen),
              q_scale=inputs.device_normal_(torch.empty(L, d, dtype=f32, device=dev), 0.1,
                                            gen) + 1.0,
              q_shift=inputs.device_normal_(torch.empty(L, d, dtype=f32, device=dev), 0.1, gen),
              rms_w=inputs.device_normal_(torch.empty(L, d, dtype=f32, device=dev), 0.1,
                                          gen) + 1.0,
              gate_w=inputs.device_normal_(torch.empty(L, H, d, dtype=f32, device=dev),
                                           1 / np.sqrt(d), gen),
              gate_b=inputs.device_normal_(torch.empty(L, H, dtype=f32, device=dev), 0.1, gen),
              w_kv=inputs.device_normal_(torch.empty(L, 2 * d_kv, d, dtype=act, device=dev),
                                         1 / np.sqrt(d), gen))
    crd = mone.swiglu_reader(rd["p_q"], rd["q_scale"], rd["q_shift"], rd["rms_w"],
                             rd["gate_w"], rd["gate_b"], rd["w_kv"], d_kv)
    kv = torch.empty(L, Q, 2 * d_kv, dtype=f32, device=dev)
    aq = inputs.device_normal_(torch.empty(L, Q, hq * ah, dtype=act, device=dev), 1.0, gen)
    ak = inputs.device_normal_(torch.empty(L, Q, hkv * ah, dtype=act, device=dev), 1.0, gen)
    av = inputs.device_normal_(torch.empty(L, Q, hkv * ah, dtype=act, device=dev), 1.0, gen)
    aout = torch.empty(L, Q, hq * ah, dtype=f32, device=dev)

    stream = torch.cuda.current_stream(dev)
    sess = mone.SwigluSession(cfg, proj, k_scale, k_shift, *w, opt=opt, stream=stream)
    Hd = sess.handle
    sptr = stream.cuda_stream

    lstride = ctx.stride(0)
    # segments per preprocessing batch, as the library's header states the default
    prep = 1 if args.call == "segment" else (
        cfg.prep_segments if cfg.prep_segments > 0 else (8 if T % 64 == 0 else 1))

    def step():
        if args.call == "segments":
            mone.mone_swiglu_segments(Hd, ctx, lstride, S, sptr)
        else:
            for s in range(S):
                mone.mone_swiglu_segments(Hd, ctx[:, s * T:], lstride, 1, sptr)
        mone.mone_swiglu_read(Hd, crd, xq, Q, kv, mone.MONE_F32, sptr)
        mone.mone_swiglu_attention(Hd, d_kv, aq, ak, av, kv, mone.MONE_F32, Q, hq, hkv, aout,
                                   mone.MONE_F32, sptr)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    if args.calib_copy_mib:
        src = torch.empty(args.calib_copy_mib << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    elapsed, stimes, dom, (dms, dcnt) = timed_steps(
        step, args.steps, lambda n, m: mone.mone_swiglu_set_stage_timing(Hd, n, m),
        lambda: mone.mone_swiglu_stage_times(Hd), mone.SW_STAGES, S * 6 + 6)
    finite = all(bool(torch.isfinite(t).all().item()) for t in w + [kv, aout])
    sess.close()

    tokens = args.steps * S * T
    value = tokens / elapsed
    flop_tok = cfg.flops_per_token()
    peak = PEAK_BF16_TFLOPS if cfg.act_dtype == "bf16" else PEAK_F32_TFLOPS
    work = dict(sw_stage_work(cfg, prep), **sw_read_work(cfg, Q, d_kv, hq, hkv))
    stages = stage_table(stimes, work)
    dfl, dby = work[dom]
    davg = dms / dcnt / 1e3
    kname = {"keys": "sw_keys_kernel", "rate": "rate_kernel"}.get(dom, f"gemm_nt_kernel ({dom})")
    roof = roofline(kname, dfl, dby, davg, peak)
    counted = (counted_traffic(dom, "hbm_traffic_sw_qwen0.5b.json")
               if cfg.name == "sw_qwen0.5b" and cfg.optimizer == "paper" else None)
    if counted:
        roof["traffic"] = counted["read_bytes"] + counted["write_bytes"]
        roof["traffic_detail"] = dict(counted, algorithmic_bytes=dby,
                                      source="profiles/hbm_traffic_sw_qwen0.5b.json")
    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": cfg.act_dtype, "data": "synthetic",
        "config": {"workload": f"paper-form SwiGLU memory TTL ({cfg.name}): L={L} d={d} "
                               f"H={H} d_h={dh} T={T} N={S * T} ({S} segments), "
                               f"{'paper optimiser' if cfg.optimizer == 'paper' else 'SGD'}"
                               f" + read Q={Q} + attention ({hq}/{hkv} heads of {ah})",
                   "n_layers": L, "d_model": d, "n_heads": H, "d_head": dh, "seg_len": T,
                   "n_context": S * T, "n_query": Q, "d_kv": d_kv, "lr": cfg.lr,
                   "optimizer": cfg.optimizer, "loss": "nip"},
        "mfma_pct": round(100.0 * value * flop_tok / (peak * 1e12), 2),
        "flop_per_token": flop_tok,
        "roofline": roof,
        "stages": stages,
        "stage_timing": "stages: one untimed profiling step, every stage timed; roofline: the "
                        "dominant stage over the timed steps",
        "finite": finite,
    }
    if cpu_in is not None:
        meta = None
        if opt is not None:
            meta = (opt[0][0].double().cpu().numpy(), float(opt[1][0]),
                    opt[2][0].double().cpu().numpy(), float(opt[3][0]))
        out["cpu_baseline"] = sw_cpu_baseline(cfg, *cpu_in, args.cpu_seconds, meta)
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", default="8b")
    ap.add_argument("--segments", type=int, default=0,
                    help="context segments per step (default: the workload's N / T)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="also run one device copy of this size (HBM counter calibration)")
    ap.add_argument("--loss", default=None, choices=("mse_sum", "mse_mean", "nip"),
                    help="override the configuration's loss (nip: the paper's negative inner "
                         "product, whose step skips the output layer's forward)")
    ap.add_argument("--optimizer", default=None, choices=("sgd", "paper"),
                    help="SGD or the paper's optimiser (per-token rates, momentum, row "
                         "renormalisation); default: SGD for the configurations' memory, the "
                         "paper's optimiser for the paper-form memory (whose negative inner "
                         "product loss is unbounded below: plain SGD lets the weights grow "
                         "without limit over a long context)")
    ap.add_argument("--graph", action="store_true",
                    help="configurations' memory: capture one whole step (its segment calls, "
                         "the read and the attention) in a HIP graph and time its replays; the "
                         "segment count must be even (the W2^T copies alternate per segment)")
    ap.add_argument("--call", default="segments", choices=("segments", "segment"),
                    help="configurations' memory: the whole context through one "
                         "mone_ttl_segments call (default; the block form for short segments), "
                         "or one call per segment")
    ap.add_argument("--block-tokens", type=int, default=0,
                    help="configurations' memory: tokens per block of the block form (0: the "
                         "library's choice, -1: none)")
    ap.add_argument("--prep-segments", type=int, default=0,
                    help="paper-form memory: segments per preprocessing batch (0: the "
                         "library's choice)")
    ap.add_argument("--memory", default="config", choices=("config", "swiglu"),
                    help="config: the configurations' 2-layer memory (default); swiglu: the "
                         "paper-form SwiGLU memory per fast-weight head at the paper's shape")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: --gpus {args.gpus} is not supported: this build measures one GPU "
              "(the path would shard by layers with no communication during TTL).",
              file=sys.stderr, flush=True)
        sys.exit(2)
    if args.memory == "swiglu":
        args.optimizer = args.optimizer or "paper"
        run_swiglu(args)
        return
    args.optimizer = args.optimizer or "sgd"

    import numpy as np
    import torch

    from paper_2608_17616_amd import configs, inputs, mone

    cfg = configs.CONFIGS[args.config].with_(optimizer=args.optimizer,
                                             block_tokens=args.block_tokens)
    if args.loss:
        cfg = cfg.with_(loss=args.loss)
    L, d, h, D, T, Q = (cfg.n_layers, cfg.d_model, cfg.d_hidden, cfg.d_out, cfg.seg_len,
                        cfg.n_query)
    S = args.segments or cfg.n_segments
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    act = torch.bfloat16 if cfg.act_dtype == "bf16" else torch.float32
    gen = torch.Generator(device=dev)
    gen.manual_seed(cfg.seed)

    w1 = inputs.device_normal_(torch.empty(L, h, d, dtype=torch.float32, device=dev),
                               1 / np.sqrt(d), gen)
    w2 = inputs.device_normal_(torch.empty(L, D, h, dtype=torch.float32, device=dev),
                               1 / np.sqrt(h), gen)
    wkv = inputs.device_normal_(torch.empty(L, D, d, dtype=act, device=dev), 1 / np.sqrt(d), gen)
    # each layer's part of the context in one piece: token t of segment s of layer l at
    # ctx[l, s*T + t]
    ctx = torch.empty(L, S * T, d, dtype=act, device=dev)
    for s in range(S):
        inputs.device_normal_(ctx[:, s * T:(s + 1) * T], 1.0, gen)
    xq = inputs.device_normal_(torch.empty(L, Q, d, dtype=act, device=dev), 1.0, gen)
    kv = torch.empty(L, Q, D, dtype=torch.float32, device=dev)
    # memory injection into attention after the read: grouped-query heads of width 128 (64 when
    # d_kv is smaller), four query heads per key/value head
    hkv = max(1, cfg.d_kv // 128)
    hq = 4 * hkv
    dh = cfg.d_kv // hkv
    aq = inputs.device_normal_(torch.empty(L, Q, hq * dh, dtype=act, device=dev), 1.0, gen)
    ak = inputs.device_normal_(torch.empty(L, Q, hkv * dh, dtype=act, device=dev), 1.0, gen)
    av = inputs.device_normal_(torch.empty(L, Q, hkv * dh, dtype=act, device=dev), 1.0, gen)
    aout = torch.empty(L, Q, hq * dh, dtype=torch.float32, device=dev)
    # CPU-baseline sample: layer 0 of the same workload, before any step changes the state
    n_cpu = 0 if args.no_cpu_baseline else min(S, 4)
    cpu_in = None
    if n_cpu:
        cpu_in = (w1[0].double().cpu().numpy(), w2[0].double().cpu().numpy(),
                  wkv[0].double().cpu().numpy(),
                  [ctx[0, s * T:(s + 1) * T].double().cpu().numpy() for s in range(n_cpu)])

    opt = None
    if cfg.optimizer == "paper":
        opt = (inputs.device_normal_(torch.empty(L, d, dtype=torch.float32, device=dev),
                                     1 / np.sqrt(d), gen),
               torch.full((L,), inputs.B_U, dtype=torch.float32, device=dev),
               inputs.device_normal_(torch.empty(L, d, dtype=torch.float32, device=dev),
                                     1 / np.sqrt(d), gen),
               torch.full((L,), inputs.B_V, dtype=torch.float32, device=dev),
               torch.zeros(L, h, d, dtype=torch.float32, device=dev),
               torch.zeros(L, D, h, dtype=torch.float32, device=dev))
    stream = torch.cuda.current_stream(dev)
    sess = mone.TtlSession(cfg, wkv, w1, w2, stream, opt=opt)
    H = sess.handle
    sptr = stream.cuda_stream

    lstride = ctx.stride(0)
    blk = block_segments(cfg) if args.call == "segments" else 1

    def step(sp=sptr):
        if args.call == "segments":
            mone.mone_ttl_segments(H, ctx, lstride, S, sp)
        else:
            for s in range(S):
                mone.mone_ttl_segments(H, ctx[:, s * T:], lstride, 1, sp)
        mone.mone_memory_kv(H, xq, Q, kv, mone.MONE_F32, sp)
        mone.mone_memory_attention(H, aq, ak, av, kv, mone.MONE_F32, Q, hq, hkv, aout,
                                   mone.MONE_F32, sp)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    graph = None
    if args.graph:
        # the W2^T copies alternate per block (per segment outside the block form)
        if (S // blk + (1 if S % blk else 0)) % 2:
            print("bench.py: --graph needs an even number of blocks (segments outside the "
                  "block form)", file=sys.stderr, flush=True)
            sys.exit(2)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):  # timing hooks are off here
            step(torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
    if args.calib_copy_mib:
        nb = args.calib_copy_mib << 20
        src = torch.empty(nb, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    if graph is None:
        elapsed, stimes, dom, (dms, dcnt) = timed_steps(
            step, args.steps, lambda n, m: mone.mone_ttl_set_stage_timing(H, n, m),
            lambda: mone.mone_ttl_stage_times(H), mone.STAGES, S * 7 + 3)
    else:
        # the stage table and the roofline come from one eager profiling step; the timed steps
        # are replays of the captured step
        mone.mone_ttl_set_stage_timing(H, S * 7 + 3, 0xFFFFFFFF)
        step()
        torch.cuda.synchronize()
        stimes = mone.mone_ttl_stage_times(H)
        mone.mone_ttl_set_stage_timing(H, 0, 0)
        dom = max((n for n in stimes if stimes[n][1]), key=lambda n: stimes[n][0])
        dms, dcnt = stimes[dom]
        t0 = time.perf_counter()
        for _ in range(args.steps):
            graph.replay()
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
    finite = bool(torch.isfinite(w1).all().item() and torch.isfinite(w2).all().item()
                  and torch.isfinite(kv).all().item())
    sess.close()

    tokens = args.steps * S * T
    value = tokens / elapsed
    flop_tok = cfg.flops_per_token()
    peak = PEAK_BF16_TFLOPS if cfg.act_dtype == "bf16" else PEAK_F32_TFLOPS
    mfma_pct = 100.0 * value * flop_tok / (peak * 1e12)
    work = stage_work(cfg, Q, blk, S if args.call == "segments" else 1)
    stages = stage_table(stimes, work)
    dfl, dby = work[dom]
    davg = dms / dcnt / 1e3
    roof = roofline(f"gemm_nt_kernel ({dom})" if dfl > 0 else dom, dfl, dby, davg, peak)
    counted = (counted_traffic(dom) if (args.config == "8b" and cfg.optimizer == "sgd" and S >= 1)
               else None)
    if counted:
        roof["traffic"] = counted["read_bytes"] + counted["write_bytes"]
        roof["traffic_detail"] = dict(counted, algorithmic_bytes=dby,
                                      source="profiles/hbm_traffic_8b.json")

    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": cfg.act_dtype, "data": "synthetic",
        "config": {"workload": f"{cfg.name}-class TTL: L={L} d={d} h={h} D={D} T={T} "
                               f"N={S * T} ({S} segments) + read Q={Q}"
                               + (", paper optimiser" if cfg.optimizer == "paper" else "")
                               + (f", loss {cfg.loss}" if args.loss else "")
                               + (", HIP graph replay" if graph is not None else "")
                               + (f", block form ({blk} segments per block)" if blk > 1
                                  else ""),
                   "n_layers": L, "d_model": d, "d_hidden": h, "d_out": D, "seg_len": T,
                   "n_context": S * T, "n_query": Q, "lr": cfg.lr, "optimizer": cfg.optimizer,
                   "loss": cfg.loss},
        "mfma_pct": round(mfma_pct, 2),
        "flop_per_token": flop_tok,
        "roofline": roof,
        "stages": stages,
        "stage_timing": ("stages: one untimed profiling step, every stage timed; roofline: the "
                         "dominant stage over the timed steps") if graph is None else
                        ("timed steps: replays of the step captured in a HIP graph; stages and "
                         "roofline: one eager profiling step, every stage timed"),
        "finite": finite,
    }
    if cpu_in is not None:
        meta = None
        if opt is not None:
            meta = (opt[0][0].double().cpu().numpy(), float(opt[1][0]),
                    opt[2][0].double().cpu().numpy(), float(opt[3][0]))
        out["cpu_baseline"] = cpu_baseline(cfg, *cpu_in, args.cpu_seconds, meta)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
