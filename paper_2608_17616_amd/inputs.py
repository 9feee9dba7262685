"""Seeded synthetic inputs for the MoNe TTL hot path.

This module holds input generation only and none of the method's arithmetic: both the CPU
oracle's callers and the GPU path's callers draw their inputs here, so the two sides see the
same numbers.

Keyed generator: every block is drawn from its own NumPy PCG64 stream keyed by
``(seed, kind, layer, index)``, so any layer or segment can be generated on its own (a parity
test can check a subset of layers of a full-size run, and a segment can be regenerated without
drawing the ones before it).  Draws are float64 standard normals, scaled, cast to float32, and,
for bf16 activations, rounded to the nearest bf16 (ties to even).

Distributions (the workloads' stated defaults):
  x, x_q ~ N(0, 1)                           segment and query hidden states, per layer
  W_k, W_v ~ N(0, 1/d)   stacked as W_kv = [W_k; W_v], shape [2*d_kv, d]
  W1 ~ N(0, 1/d)         shape [h, d]      (variance 1/fan_in)
  W2 ~ N(0, 1/h)         shape [2*d_kv, h] (variance 1/fan_in)
Paper-form (SwiGLU per head) memory, per layer:
  P_k, P_v ~ N(0, 1/d)   key and value projections, stacked as [P_k; P_v], shape [2d, d]
  s = 1 + 0.1 N(0, 1), b = 0.1 N(0, 1)    the keys' per-channel affine step, shape [d] each
  W_in, W_gate, W_out ~ N(0, 1/d_h)       fast weights, shape [H, d_h, d_h] each
Read of the paper-form memory, per layer:
  P_q ~ N(0, 1/d)                          query projection, shape [d, d]
  s_q = 1 + 0.1 N(0, 1), b_q = 0.1 N(0, 1) the queries' affine step, shape [d] each
  w_rms = 1 + 0.1 N(0, 1)                  RMSNorm weight, shape [d]
  a ~ N(0, 1/d), c = 0.1 N(0, 1)           gate vectors [H, d] and biases [H]
  W_k, W_v ~ N(0, 1/d)                     the backbone's key/value maps, [2 d_kv, d]
Meta-parameters of the paper's optimiser (trained offline in the paper; synthetic here):
  u, v ~ N(0, 1/d)       rate and decay projections, shape [d] each
  b_u = log(e - 1)       so that softplus(b_u) = 1: rates average about lr
  b_v = 0                decays average about 1/2
"""
from __future__ import annotations

import numpy as np

KIND_WK, KIND_WV, KIND_W1, KIND_W2, KIND_X, KIND_XQ, KIND_U, KIND_V = range(8)
KIND_PK, KIND_PV, KIND_KSCALE, KIND_KSHIFT, KIND_WIN, KIND_WGATE, KIND_WOUT = range(8, 15)
KIND_PQ, KIND_QSCALE, KIND_QSHIFT, KIND_RMSW, KIND_GATEW, KIND_GATEB, KIND_BWK, KIND_BWV = range(15, 23)
B_U = float(np.log(np.e - 1.0))
B_V = 0.0


def normal(seed: int, kind: int, layer: int, index: int, shape, std: float) -> np.ndarray:
    rng = np.random.default_rng([int(seed), int(kind), int(layer), int(index)])
    return (rng.standard_normal(shape) * std).astype(np.float32)


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); returns the raw uint16 patterns.

    Inputs are finite Gaussian draws, so no NaN/Inf handling is needed.
    """
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def bf16_widen(bits: np.ndarray) -> np.ndarray:
    """Exact float32 value of raw bf16 patterns."""
    return (bits.astype(np.uint32) << 16).view(np.float32)


def act_round(a: np.ndarray, act_dtype: str) -> np.ndarray:
    """Activation-dtype values as float32 (bf16: nearest bf16, widened exactly)."""
    if act_dtype == "f32":
        return a
    if act_dtype == "bf16":
        return bf16_widen(bf16_bits(a))
    raise ValueError(act_dtype)


def layer_wkv(cfg, layer: int) -> np.ndarray:
    """Frozen [W_k; W_v] of one layer, [2*d_kv, d], float32 (bf16-representable in bf16 mode)."""
    d = cfg.d_model
    wk = normal(cfg.seed, KIND_WK, layer, 0, (cfg.d_kv, d), 1.0 / np.sqrt(d))
    wv = normal(cfg.seed, KIND_WV, layer, 0, (cfg.d_kv, d), 1.0 / np.sqrt(d))
    return act_round(np.concatenate([wk, wv], axis=0), cfg.act_dtype)


def layer_w1(cfg, layer: int) -> np.ndarray:
    """Initial fast weight W1 (W_in) of one layer, [h, d], float32."""
    return normal(cfg.seed, KIND_W1, layer, 0, (cfg.d_hidden, cfg.d_model),
                  1.0 / np.sqrt(cfg.d_model))


def layer_w2(cfg, layer: int) -> np.ndarray:
    """Initial fast weight W2 (W_out) of one layer, [2*d_kv, h], float32."""
    return normal(cfg.seed, KIND_W2, layer, 0, (cfg.d_out, cfg.d_hidden),
                  1.0 / np.sqrt(cfg.d_hidden))


def layer_meta(cfg, layer: int):
    """Optimiser meta-parameters of one layer: (u [d], b_u, v [d], b_v), float32 vectors."""
    d = cfg.d_model
    u = normal(cfg.seed, KIND_U, layer, 0, (d,), 1.0 / np.sqrt(d))
    v = normal(cfg.seed, KIND_V, layer, 0, (d,), 1.0 / np.sqrt(d))
    return u, np.float32(B_U), v, np.float32(B_V)


def sw_layer_proj(cfg, layer: int) -> np.ndarray:
    """Frozen [P_k; P_v] of one layer of the paper-form memory, [2d, d], float32."""
    d = cfg.d_model
    pk = normal(cfg.seed, KIND_PK, layer, 0, (d, d), 1.0 / np.sqrt(d))
    pv = normal(cfg.seed, KIND_PV, layer, 0, (d, d), 1.0 / np.sqrt(d))
    return act_round(np.concatenate([pk, pv], axis=0), cfg.act_dtype)


def sw_layer_affine(cfg, layer: int):
    """The keys' per-channel scale and shift of one layer, [d] float32 each."""
    d = cfg.d_model
    scale = (1.0 + normal(cfg.seed, KIND_KSCALE, layer, 0, (d,), 0.1)).astype(np.float32)
    shift = normal(cfg.seed, KIND_KSHIFT, layer, 0, (d,), 0.1)
    return scale, shift


def sw_layer_fast(cfg, layer: int):
    """Initial (W_in, W_gate, W_out) of one layer, [H, d_h, d_h] float32 each."""
    shape, std = (cfg.n_heads, cfg.d_head, cfg.d_head), 1.0 / np.sqrt(cfg.d_head)
    return tuple(normal(cfg.seed, k, layer, 0, shape, std)
                 for k in (KIND_WIN, KIND_WGATE, KIND_WOUT))


def sw_layer_reader(cfg, layer: int, d_kv: int) -> dict:
    """The read's frozen parameters of one layer of the paper-form memory (float32; the
    projections bf16-representable in bf16 mode)."""
    d, H, sd = cfg.d_model, cfg.n_heads, 1.0 / np.sqrt(cfg.d_model)
    r = lambda kind, shape, std: normal(cfg.seed, kind, layer, 0, shape, std)  # noqa: E731
    wk, wv = r(KIND_BWK, (d_kv, d), sd), r(KIND_BWV, (d_kv, d), sd)
    return dict(p_q=act_round(r(KIND_PQ, (d, d), sd), cfg.act_dtype),
                q_scale=(1.0 + r(KIND_QSCALE, (d,), 0.1)).astype(np.float32),
                q_shift=r(KIND_QSHIFT, (d,), 0.1),
                rms_w=(1.0 + r(KIND_RMSW, (d,), 0.1)).astype(np.float32),
                gate_w=r(KIND_GATEW, (H, d), sd), gate_b=r(KIND_GATEB, (H,), 0.1),
                w_kv=act_round(np.concatenate([wk, wv], axis=0), cfg.act_dtype))


def segment_x(cfg, layer: int, s: int, n_tokens: int | None = None) -> np.ndarray:
    """Hidden states of segment s (0-based) at one layer, [n_tokens, d], float32."""
    n = cfg.seg_len if n_tokens is None else n_tokens
    return act_round(normal(cfg.seed, KIND_X, layer, s, (n, cfg.d_model), 1.0), cfg.act_dtype)


def query_x(cfg, layer: int, q: int | None = None, index: int = 0) -> np.ndarray:
    """Query-side memory input of one layer, [q, d], float32."""
    q = cfg.n_query if q is None else q
    return act_round(normal(cfg.seed, KIND_XQ, layer, index, (q, cfg.d_model), 1.0),
                     cfg.act_dtype)


def device_normal_(t, std: float, generator):
    """Fill a device tensor in place with N(0, std^2) draws rounded to its dtype.

    Used for benchmark inputs too large to draw on the host in reasonable time; the draws are
    seeded through ``generator`` (a torch.Generator on the tensor's device).
    """
    import torch
    if t.dtype == torch.float32:
        t.normal_(0.0, std, generator=generator)
    else:
        tmp = torch.empty(t.shape, dtype=torch.float32, device=t.device)
        tmp.normal_(0.0, std, generator=generator)
        t.copy_(tmp)
    return t
